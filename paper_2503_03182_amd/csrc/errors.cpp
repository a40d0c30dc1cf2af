// Thread-local error message behind tps_last_error().
#include "errors.h"

#include "../../include/tpstage.h"

namespace tps {

static thread_local std::string g_last_error;

int set_error(int code, const std::string& msg) {
  g_last_error = msg;
  return code;
}

int clear_error() {
  g_last_error.clear();
  return TPS_OK;
}

const char* last_error() { return g_last_error.c_str(); }

int check_hip(hipError_t e, const char* what) {
  if (e == hipSuccess) return TPS_OK;
  return set_error(TPS_EHIP, std::string(what) + ": " + hipGetErrorString(e));
}

}  // namespace tps

extern "C" const char* tps_last_error(void) { return tps::last_error(); }
