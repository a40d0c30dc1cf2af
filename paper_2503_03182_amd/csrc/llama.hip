// Element-wise kernels of the LLAMA-style layer: rotary position embedding
// (and its table), SwiGLU forward and backward, and the fold of per-query-
// head key/value gradients of grouped-query attention.  All HBM-bound:
// 16-byte accesses, one thread per 8 elements, no reductions across threads.
#include "kernels.h"
#include "tps_device.h"

namespace tps {

namespace {

// cos and sin of pos * base^(-2 i / d) for pos < s, i < d / 2, evaluated in
// double and rounded once to f32: table[pos][i] cos, table[s + pos][i] sin.
__global__ __launch_bounds__(256) void rope_table_kernel(int s, int half, double log_base_over_half,
                                                         float* __restrict__ table) {
  const int64_t k = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (k >= (int64_t)s * half) return;
  const int pos = (int)(k / half), i = (int)(k % half);
  const double ang = (double)pos * exp(-(double)i * log_base_over_half);
  table[k] = (float)cos(ang);
  table[(int64_t)s * half + k] = (float)sin(ang);
}

// One thread turns 8 pairs (x_i, x_{i + d/2}), i = i0 .. i0 + 7, of one head
// of one row by +angle (or -angle: the transposed rotation of a gradient).
// Columns [0, n_rot * d) of each row are rotated.
__global__ __launch_bounds__(256) void rope_kernel(bf16* __restrict__ x, int64_t ld, int rows, int s, int n_rot,
                                                   int d, const float* __restrict__ table, float sign) {
  const int half = d / 2, per_head = half / 8;
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t per_row = (int64_t)n_rot * per_head;
  if (t >= (int64_t)rows * per_row) return;
  const int row = (int)(t / per_row);
  const int r = (int)(t % per_row);
  const int head = r / per_head, i0 = (r % per_head) * 8;
  const int pos = row % s;
  bf16* lo_p = x + (int64_t)row * ld + (int64_t)head * d + i0;
  bf16* hi_p = lo_p + half;
  const Vec16<bf16> lo = load16(lo_p), hi = load16(hi_p);
  const float* cp = table + (int64_t)pos * half + i0;
  const float* sp = table + (int64_t)s * half + (int64_t)pos * half + i0;
  const f32x4 c0 = *reinterpret_cast<const f32x4*>(cp), c1 = *reinterpret_cast<const f32x4*>(cp + 4);
  const f32x4 s0 = *reinterpret_cast<const f32x4*>(sp), s1 = *reinterpret_cast<const f32x4*>(sp + 4);
  Vec16<bf16> nlo, nhi;
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const float c = j < 4 ? c0[j] : c1[j - 4];
    const float sn = sign * (j < 4 ? s0[j] : s1[j - 4]);
    const float a = to_f32(lo.get(j)), b = to_f32(hi.get(j));
    nlo.set(j, from_f32<bf16>(a * c - b * sn));
    nhi.set(j, from_f32<bf16>(b * c + a * sn));
  }
  store16(lo_p, nlo);
  store16(hi_p, nhi);
}

__device__ __forceinline__ float sigmoid(float z) { return 1.0f / (1.0f + expf(-z)); }

// g[t][j] = SiLU(u[t][j]) * u[t][f + j]
__global__ __launch_bounds__(256) void swiglu_kernel(const bf16* __restrict__ u, bf16* __restrict__ g, int rows,
                                                     int f) {
  const int per_row = f / 8;
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (t >= (int64_t)rows * per_row) return;
  const int row = (int)(t / per_row), c = (int)(t % per_row) * 8;
  const bf16* ur = u + (int64_t)row * 2 * f;
  const Vec16<bf16> a = load16(ur + c), b = load16(ur + f + c);
  Vec16<bf16> o;
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const float z = to_f32(a.get(j));
    o.set(j, from_f32<bf16>(z * sigmoid(z) * to_f32(b.get(j))));
  }
  store16(g + (int64_t)row * f + c, o);
}

// du[t][j] = dg * up * sigma (1 + gate (1 - sigma)), du[t][f + j] = dg * SiLU(gate)
__global__ __launch_bounds__(256) void swiglu_bwd_kernel(const bf16* __restrict__ dg, const bf16* __restrict__ u,
                                                         bf16* __restrict__ du, int rows, int f) {
  const int per_row = f / 8;
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (t >= (int64_t)rows * per_row) return;
  const int row = (int)(t / per_row), c = (int)(t % per_row) * 8;
  const bf16* ur = u + (int64_t)row * 2 * f;
  const Vec16<bf16> a = load16(ur + c), b = load16(ur + f + c), d = load16(dg + (int64_t)row * f + c);
  Vec16<bf16> ga, gb;
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const float z = to_f32(a.get(j)), up = to_f32(b.get(j)), dd = to_f32(d.get(j));
    const float sg = sigmoid(z);
    ga.set(j, from_f32<bf16>(dd * up * sg * (1.0f + z * (1.0f - sg))));
    gb.set(j, from_f32<bf16>(dd * z * sg));
  }
  bf16* dr = du + (int64_t)row * 2 * f;
  store16(dr + c, ga);
  store16(dr + f + c, gb);
}

// Key/value head kv of row t gets the sum, in ascending query-head order, of
// the dK (dV) of its grp query heads from the workspace ws [T][2 nh d] (dK
// of head n at columns n d, dV at nh d + n d); dqkv rows hold q | k | v with
// nh, nkv, nkv heads.
__global__ __launch_bounds__(256) void gqa_fold_kernel(const bf16* __restrict__ ws, bf16* __restrict__ dqkv, int rows,
                                                       int nh, int nkv, int d) {
  const int per_row = 2 * nkv * d / 8;   // 8-column chunks of the k and v blocks
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (t >= (int64_t)rows * per_row) return;
  const int row = (int)(t / per_row), c = (int)(t % per_row) * 8;
  const int part = c / (nkv * d);          // 0: k, 1: v
  const int cc = c % (nkv * d);
  const int kv = cc / d, e = cc % d;
  const int grp = nh / nkv;
  const bf16* src = ws + (int64_t)row * 2 * nh * d + (int64_t)part * nh * d + (int64_t)kv * grp * d + e;
  float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  for (int j = 0; j < grp; ++j) {
    const Vec16<bf16> v = load16(src + (int64_t)j * d);
#pragma unroll
    for (int k = 0; k < 8; ++k) acc[k] += to_f32(v.get(k));
  }
  Vec16<bf16> o;
#pragma unroll
  for (int k = 0; k < 8; ++k) o.set(k, from_f32<bf16>(acc[k]));
  store16(dqkv + (int64_t)row * (nh + 2 * nkv) * d + (int64_t)nh * d + c, o);
}

unsigned blocks_for(int64_t threads) { return (unsigned)((threads + 255) / 256); }

}  // namespace

hipError_t rope_table_launch(int s, int d, float base, float* table, hipStream_t st) {
  if (s <= 0) return hipSuccess;
  if (d % 16 != 0 || !(base > 1.0f)) return hipErrorInvalidValue;
  const int half = d / 2;
  hipLaunchKernelGGL(rope_table_kernel, dim3(blocks_for((int64_t)s * half)), dim3(256), 0, st, s, half,
                     log((double)base) / (double)half, table);
  return hipGetLastError();
}

hipError_t rope_launch(void* x, int64_t ld, int rows, int s, int n_rot, int d, const float* table, int inverse,
                       hipStream_t st) {
  if (rows <= 0 || n_rot <= 0) return hipSuccess;
  if (d % 16 != 0 || ld % 8 != 0) return hipErrorInvalidValue;
  const int64_t threads = (int64_t)rows * n_rot * (d / 16);
  hipLaunchKernelGGL(rope_kernel, dim3(blocks_for(threads)), dim3(256), 0, st, (bf16*)x, ld, rows, s, n_rot, d, table,
                     inverse ? -1.0f : 1.0f);
  return hipGetLastError();
}

hipError_t swiglu_launch(int rows, int f, const void* u, void* g, hipStream_t st) {
  if (rows <= 0) return hipSuccess;
  if (f % 8 != 0) return hipErrorInvalidValue;
  hipLaunchKernelGGL(swiglu_kernel, dim3(blocks_for((int64_t)rows * (f / 8))), dim3(256), 0, st, (const bf16*)u,
                     (bf16*)g, rows, f);
  return hipGetLastError();
}

hipError_t swiglu_bwd_launch(int rows, int f, const void* dg, const void* u, void* du, hipStream_t st) {
  if (rows <= 0) return hipSuccess;
  if (f % 8 != 0) return hipErrorInvalidValue;
  hipLaunchKernelGGL(swiglu_bwd_kernel, dim3(blocks_for((int64_t)rows * (f / 8))), dim3(256), 0, st,
                     (const bf16*)dg, (const bf16*)u, (bf16*)du, rows, f);
  return hipGetLastError();
}

hipError_t gqa_fold_launch(const void* ws, void* dqkv, int rows, int nh, int nkv, int d, hipStream_t st) {
  if (rows <= 0) return hipSuccess;
  if (nkv <= 0 || nh % nkv != 0 || d % 8 != 0) return hipErrorInvalidValue;
  hipLaunchKernelGGL(gqa_fold_kernel, dim3(blocks_for((int64_t)rows * (2 * nkv * d / 8))), dim3(256), 0, st,
                     (const bf16*)ws, (bf16*)dqkv, rows, nh, nkv, d);
  return hipGetLastError();
}

}  // namespace tps
