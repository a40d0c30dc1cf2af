// AdamW on the device for the layers whose model state T-Offload keeps on the
// GPU (the shallow ones, whose update would otherwise sit between two
// iterations): the host update's arithmetic (host_optim.cpp) with the same
// f32 operations in the same order, no contraction into fused multiply-adds
// and correctly rounded division and square root, so the two paths give the
// same bits.  HBM-bound: 16 bytes read and 12 + sizeof(storage) written per
// parameter, four parameters per thread.
#include <hip/hip_runtime.h>

#include "kernels.h"
#include "tps_device.h"

namespace tps {

namespace {

struct Coef {
  float b1, b2, eps, lr_c, inv_bc2_sqrt, wd_c;
};

template <typename T>
__device__ __forceinline__ float adamw_one(float& w, float& m, float& v, float g, const Coef& c) {
#pragma clang fp contract(off)
  const float mi = c.b1 * m + (1.f - c.b1) * g;
  const float vi = c.b2 * v + (1.f - c.b2) * g * g;
  m = mi;
  v = vi;
  const float denom = __builtin_sqrtf(vi) * c.inv_bc2_sqrt + c.eps;
  w = w - c.lr_c * mi / denom - c.wd_c * w;
  return w;
}

// n4 groups of four parameters (16-byte accesses), then the n % 4 tail
template <typename T>
__global__ __launch_bounds__(256) void adamw_kernel(float* __restrict__ w, float* __restrict__ m,
                                                    float* __restrict__ v, const float* __restrict__ g,
                                                    T* __restrict__ out, int64_t n, Coef c) {
  const int64_t n4 = n / 4;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n4; i += stride) {
    f32x4 wv = reinterpret_cast<const f32x4*>(w)[i];
    f32x4 mv = reinterpret_cast<const f32x4*>(m)[i];
    f32x4 vv = reinterpret_cast<const f32x4*>(v)[i];
    const f32x4 gv = reinterpret_cast<const f32x4*>(g)[i];
    T o[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      float wk = wv[k], mk = mv[k], vk = vv[k];
      o[k] = from_f32<T>(adamw_one<T>(wk, mk, vk, gv[k], c));
      wv[k] = wk;
      mv[k] = mk;
      vv[k] = vk;
    }
    reinterpret_cast<f32x4*>(w)[i] = wv;
    reinterpret_cast<f32x4*>(m)[i] = mv;
    reinterpret_cast<f32x4*>(v)[i] = vv;
#pragma unroll
    for (int k = 0; k < 4; ++k) out[4 * i + k] = o[k];
  }
  for (int64_t i = 4 * n4 + (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) {
    float wk = w[i], mk = m[i], vk = v[i];
    out[i] = from_f32<T>(adamw_one<T>(wk, mk, vk, g[i], c));
    w[i] = wk;
    m[i] = mk;
    v[i] = vk;
  }
}

}  // namespace

hipError_t adamw_launch(int dtype, int64_t n, float* w, float* m, float* v, const float* g, void* out,
                        const float c[6], hipStream_t st) {
  if (n <= 0) return hipSuccess;
  if (!w || !m || !v || !g || !out || !c) return hipErrorInvalidValue;
  // the 16-byte path needs 16-byte aligned f32 blocks
  if (((uintptr_t)w | (uintptr_t)m | (uintptr_t)v | (uintptr_t)g) & 15u) return hipErrorInvalidValue;
  const Coef k{c[0], c[1], c[2], c[3], c[4], c[5]};
  const int64_t blocks = std::min<int64_t>((n / 4 + 255) / 256 + 1, 8192);
  if (dtype == TPS_BF16)
    hipLaunchKernelGGL(adamw_kernel<bf16>, dim3((unsigned)blocks), dim3(256), 0, st, w, m, v, g,
                       static_cast<bf16*>(out), n, k);
  else
    hipLaunchKernelGGL(adamw_kernel<float>, dim3((unsigned)blocks), dim3(256), 0, st, w, m, v, g,
                       static_cast<float*>(out), n, k);
  return hipGetLastError();
}

}  // namespace tps
