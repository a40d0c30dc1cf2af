// Thread-local last-error message and status helpers shared by the ABI files.
#pragma once
#include <hip/hip_runtime.h>

#include <string>

namespace tps {

int set_error(int code, const std::string& msg);
int clear_error();
const char* last_error();

// Map a HIP status to TPS_EHIP with context; TPS_OK on success.
int check_hip(hipError_t e, const char* what);

}  // namespace tps
