// Host-only stand-in (see hip_runtime.h in this directory).
#pragma once
#include "hip_runtime.h"

hipError_t hipExtStreamCreateWithCUMask(hipStream_t* s, uint32_t cu_mask_size, const uint32_t* cu_mask);
