// Expansion of quantized weight reloads: FP8 E4M3 codes with one f32 scale
// per matrix row -> bf16 weights, w = bf16(decode(q) * scale) (round to
// nearest even).  E4M3: 1 sign bit, 4 exponent bits with bias 7, 3 mantissa
// bits; exponent field 0 holds the subnormals f * 2^-9; the all-ones pattern
// S.1111.111 is NaN (the host quantizer never produces it).  HBM-bound: one
// byte read and two written per weight, eight weights per thread.
#include <hip/hip_runtime.h>

#include "kernels.h"
#include "tps_device.h"

namespace tps {

namespace {

__device__ __forceinline__ float e4m3_decode(uint32_t c) {
  const uint32_t s = (c & 0x80u) << 24;
  const uint32_t e = (c >> 3) & 0xFu, f = c & 7u;
  if (e == 0xFu && f == 7u) return __uint_as_float(s | 0x7FC00000u);
  if (e == 0u) return __uint_as_float(s | __float_as_uint((float)f * 0.001953125f));   // f * 2^-9
  return __uint_as_float(s | ((e + 120u) << 23) | (f << 20));                           // (1 + f/8) 2^(e-7)
}

__global__ __launch_bounds__(256) void dequant_fp8_rows_kernel(const uint2* __restrict__ q,
                                                               const float* __restrict__ scale, int64_t cols,
                                                               int64_t chunks, bf16x8* __restrict__ out) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < chunks; i += (int64_t)gridDim.x * blockDim.x) {
    const uint2 c = q[i];
    const float sc = scale[(i * 8) / cols];
    bf16x8 v;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      frag_at(v, k) = (bf16)(e4m3_decode((c.x >> (8 * k)) & 0xFFu) * sc);
      frag_at(v, 4 + k) = (bf16)(e4m3_decode((c.y >> (8 * k)) & 0xFFu) * sc);
    }
    out[i] = v;
  }
}

}  // namespace

hipError_t dequant_fp8_rows_launch(const void* q, const float* scale, int64_t rows, int64_t cols, void* out,
                                   hipStream_t st) {
  if (rows <= 0 || cols <= 0) return hipSuccess;
  if (cols % 8) return hipErrorInvalidValue;
  const int64_t chunks = rows * cols / 8;
  const int64_t blocks = std::min<int64_t>((chunks + 255) / 256, 4096);
  hipLaunchKernelGGL(dequant_fp8_rows_kernel, dim3((unsigned)blocks), dim3(256), 0, st, static_cast<const uint2*>(q),
                     scale, cols, chunks, static_cast<bf16x8*>(out));
  return hipGetLastError();
}

}  // namespace tps
