// Device-side building blocks shared by the gfx950 kernels: storage types,
// 32x32 MFMA wrappers, vector memory helpers and wavefront reductions.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace tps {

typedef __bf16 bf16;
typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(16))) float f32x16;
typedef __attribute__((ext_vector_type(4))) float f32x4;
typedef __attribute__((ext_vector_type(4))) uint32_t u32x4;
typedef __attribute__((ext_vector_type(2))) uint32_t u32x2;

constexpr int kWave = 64;

// ---------------------------------------------------------------------------
// 32x32 MFMA tile: D[32,32] += A[32,K] * B[K,32] with K = 2 * KPL.
// Lane l supplies A[l % 32][(l / 32) * KPL + i] and B[(l / 32) * KPL + i][l % 32]
// for i < KPL; result register j of lane l holds D[row_of(j, l)][l % 32].
// bf16: v_mfma_f32_32x32x16_bf16 (KPL 8);  f32: v_mfma_f32_32x32x2f32 (KPL 1).
// ---------------------------------------------------------------------------
template <typename T> struct Mma;

template <> struct Mma<bf16> {
  static constexpr int KPL = 8;
  typedef bf16x8 Frag;
  static __device__ __forceinline__ f32x16 run(const Frag& a, const Frag& b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
  }
};

template <> struct Mma<float> {
  static constexpr int KPL = 1;
  typedef float Frag;
  static __device__ __forceinline__ f32x16 run(const Frag& a, const Frag& b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
  }
};

__device__ __forceinline__ int acc_row(int j, int lane) {
  return ((j >> 2) << 3) + ((lane >> 5) << 2) + (j & 3);
}

// Element i of a fragment.
__device__ __forceinline__ bf16& frag_at(bf16x8& f, int i) { return reinterpret_cast<bf16*>(&f)[i]; }
__device__ __forceinline__ float& frag_at(float& f, int) { return f; }

// ---------------------------------------------------------------------------
// Conversions (round to nearest even on store).
// ---------------------------------------------------------------------------
template <typename T> __device__ __forceinline__ T from_f32(float v);
template <> __device__ __forceinline__ float from_f32<float>(float v) { return v; }
template <> __device__ __forceinline__ bf16 from_f32<bf16>(float v) { return (bf16)v; }
__device__ __forceinline__ float to_f32(float v) { return v; }
__device__ __forceinline__ float to_f32(bf16 v) { return (float)v; }

// 16-byte vector of storage elements.
template <typename T> struct Vec16 {
  static constexpr int N = 16 / sizeof(T);
  u32x4 raw;
  __device__ __forceinline__ T get(int i) const { return reinterpret_cast<const T*>(&raw)[i]; }
  __device__ __forceinline__ void set(int i, T v) { reinterpret_cast<T*>(&raw)[i] = v; }
};

template <typename T>
__device__ __forceinline__ Vec16<T> load16(const T* p) {
  Vec16<T> v;
  v.raw = *reinterpret_cast<const u32x4*>(p);
  return v;
}
template <typename T>
__device__ __forceinline__ void store16(T* p, const Vec16<T>& v) {
  *reinterpret_cast<u32x4*>(p) = v.raw;
}
template <typename T>
__device__ __forceinline__ Vec16<T> zero16() {
  Vec16<T> v;
  v.raw = u32x4{0u, 0u, 0u, 0u};
  return v;
}

// ---------------------------------------------------------------------------
// Fixed-order (butterfly) wavefront reductions: every lane ends with the same
// value, and the association order depends only on the lane count.
// ---------------------------------------------------------------------------
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, kWave);
  return v;
}
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v = fmaxf(v, __shfl_xor(v, off, kWave));
  return v;
}

// ---------------------------------------------------------------------------
// GeLU (erf form) and its derivative, f32.  erf follows Abramowitz & Stegun,
// Handbook of Mathematical Functions, formula 7.1.26 (|error| <= 1.5e-7 for
// all x): erf(x) = 1 - (a1 t + ... + a5 t^5) exp(-x^2), t = 1 / (1 + p x),
// x >= 0, odd extension.  Branch-free, one reciprocal and one exp2; the
// absolute error is far below the bf16 rounding of the results.  Every kernel
// that produces GeLU(u) uses these, so a recomputed g is bit-identical.
// ---------------------------------------------------------------------------
struct ErfParts {
  float erf;    // erf(x)
  float gauss;  // exp(-x^2)
};
__device__ __forceinline__ ErfParts erf_as(float x) {
  const float ax = __builtin_fabsf(x);
  const float t = __builtin_amdgcn_rcpf(__builtin_fmaf(0.3275911f, ax, 1.0f));
  float p = 1.061405429f;
  p = __builtin_fmaf(p, t, -1.453152027f);
  p = __builtin_fmaf(p, t, 1.421413741f);
  p = __builtin_fmaf(p, t, -0.284496736f);
  p = __builtin_fmaf(p, t, 0.254829592f);
  p *= t;
  const float e = __builtin_amdgcn_exp2f(-ax * ax * 1.4426950408889634f);
  return {__builtin_copysignf(__builtin_fmaf(-p, e, 1.0f), x), e};
}
__device__ __forceinline__ float gelu_f(float u) {
  return 0.5f * u * (1.0f + erf_as(u * 0.70710678118654752f).erf);
}
// GeLU'(u) = Phi(u) + u phi(u), phi(u) = exp(-u^2 / 2) / sqrt(2 pi)
__device__ __forceinline__ float gelu_grad_f(float u) {
  const ErfParts e = erf_as(u * 0.70710678118654752f);
  return 0.5f * (1.0f + e.erf) + u * 0.39894228040143268f * e.gauss;
}

}  // namespace tps
