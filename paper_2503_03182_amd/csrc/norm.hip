// HBM-bound kernels of the stage: LayerNorm forward/backward, fixed-order
// column reductions (bias, gain and shift gradients), GeLU recompute and a
// zero fill.  16-byte vector accesses; one 256-thread workgroup per row for
// the row-wise kernels, reductions butterfly-within-wave then in wave order.
#include "kernels.h"
#include "tps_device.h"
#include "ws.h"

namespace tps {

namespace {


__device__ __forceinline__ float block_sum(float v, float* red) {
  v = wave_sum(v);
  const int wave = threadIdx.x >> 6;
  __syncthreads();
  if ((threadIdx.x & 63) == 0) red[wave] = v;
  __syncthreads();
  return ((red[0] + red[1]) + red[2]) + red[3];
}

// RMS: no centring and no shift (mean taken as 0, beta unused)
template <typename T, int NC, bool RMS = false>
__global__ __launch_bounds__(256) void ln_fwd_kernel(const T* __restrict__ x, const T* __restrict__ gamma,
                                                     const T* __restrict__ beta, float eps, T* __restrict__ out,
                                                     float* __restrict__ mean, float* __restrict__ rstd,
                                                     int rows, int cols) {
  constexpr int VEC = 16 / sizeof(T);
  __shared__ float red[4];
  const int row = blockIdx.x;
  const T* xr = x + (int64_t)row * cols;
  float v[NC][VEC];
  float s = 0.f;
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    const int col = (threadIdx.x + c * 256) * VEC;
    if (col < cols) {
      const Vec16<T> t = load16(xr + col);
#pragma unroll
      for (int i = 0; i < VEC; ++i) v[c][i] = to_f32(t.get(i));
    } else {
#pragma unroll
      for (int i = 0; i < VEC; ++i) v[c][i] = 0.f;
    }
#pragma unroll
    for (int i = 0; i < VEC; ++i) s += v[c][i];
  }
  const float mu = RMS ? 0.f : block_sum(s, red) / (float)cols;
  float ss = 0.f;
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    const int col = (threadIdx.x + c * 256) * VEC;
    if (col < cols) {
#pragma unroll
      for (int i = 0; i < VEC; ++i) {
        const float d = v[c][i] - mu;
        ss += d * d;
      }
    }
  }
  const float var = block_sum(ss, red) / (float)cols;
  const float rs = 1.0f / sqrtf(var + eps);
  T* orow = out + (int64_t)row * cols;
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    const int col = (threadIdx.x + c * 256) * VEC;
    if (col < cols) {
      const Vec16<T> g = load16(gamma + col);
      Vec16<T> b;
      if constexpr (!RMS) b = load16(beta + col);
      Vec16<T> o;
#pragma unroll
      for (int i = 0; i < VEC; ++i) {
        const float n = (v[c][i] - mu) * rs * to_f32(g.get(i));
        o.set(i, from_f32<T>(RMS ? n : n + to_f32(b.get(i))));
      }
      store16(orow + col, o);
    }
  }
  if (threadIdx.x == 0) {
    if (mean) mean[row] = mu;
    if (rstd) rstd[row] = rs;
  }
}

template <typename T, int NC, bool RMS = false>
__global__ __launch_bounds__(256) void ln_bwd_kernel(const T* __restrict__ dout, const T* __restrict__ x,
                                                     const float* __restrict__ mean, const float* __restrict__ rstd,
                                                     const T* __restrict__ gamma, const T* __restrict__ resid,
                                                     T* __restrict__ dx, int rows, int cols) {
  constexpr int VEC = 16 / sizeof(T);
  __shared__ float red[4];
  const int row = blockIdx.x;
  const float mu = RMS ? 0.f : mean[row], rs = rstd[row];
  const T* xr = x + (int64_t)row * cols;
  const T* dr = dout + (int64_t)row * cols;
  float zh[NC][VEC], gv[NC][VEC];
  float s1 = 0.f, s2 = 0.f;
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    const int col = (threadIdx.x + c * 256) * VEC;
    if (col < cols) {
      const Vec16<T> xv = load16(xr + col), dv = load16(dr + col), g = load16(gamma + col);
#pragma unroll
      for (int i = 0; i < VEC; ++i) {
        zh[c][i] = (to_f32(xv.get(i)) - mu) * rs;
        gv[c][i] = to_f32(dv.get(i)) * to_f32(g.get(i));
        s1 += gv[c][i];
        s2 += gv[c][i] * zh[c][i];
      }
    } else {
#pragma unroll
      for (int i = 0; i < VEC; ++i) zh[c][i] = gv[c][i] = 0.f;
    }
  }
  const float m1 = RMS ? 0.f : block_sum(s1, red) / (float)cols;
  const float m2 = block_sum(s2, red) / (float)cols;
  T* o = dx + (int64_t)row * cols;
  const T* rr = resid ? resid + (int64_t)row * cols : nullptr;
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    const int col = (threadIdx.x + c * 256) * VEC;
    if (col < cols) {
      Vec16<T> r;
      if (rr) r = load16(rr + col);
      Vec16<T> w;
#pragma unroll
      for (int i = 0; i < VEC; ++i) {
        float val = rs * (gv[c][i] - m1 - zh[c][i] * m2);
        if (rr) val += to_f32(r.get(i));
        w.set(i, from_f32<T>(val));
      }
      store16(o + col, w);
    }
  }
}

// Wave-per-row LayerNorm for rows of NV * 512 bf16 (lane l holds the 8-column
// chunks l, l + 64, ...): reductions are wave butterflies only, four rows per
// 256-thread workgroup.  Rows of 4096 columns and more stay in registers as
// packed bf16 and each pass converts them again: settle() between passes
// keeps the compiler from holding the f32 values of one pass for the next,
// which at 8192 columns took every register of the SIMD and left one or two
// waves per SIMD to hide the HBM latency.  The operations are those of the
// source either way; only the compiler's pairing of multiplies and adds into
// FMAs may differ (one bf16 ulp in one element of 33.5M seen in the RMS
// backward at 4096 x 8192).
template <int NV>
__device__ __forceinline__ void settle(Vec16<bf16> (&v)[NV]) {
#pragma unroll
  for (int c = 0; c < NV; ++c) asm volatile("" : "+v"(v[c].raw));
}
// rows this wide keep only the packed row live across passes
template <int NV> constexpr bool kWideRow = NV >= 8;

template <int NV, bool RMS = false>
__global__ __launch_bounds__(256) void ln_fwd_wave_kernel(const bf16* __restrict__ x, const bf16* __restrict__ gamma,
                                                          const bf16* __restrict__ beta, float eps,
                                                          bf16* __restrict__ out, float* __restrict__ mean,
                                                          float* __restrict__ rstd, int rows, int cols) {
  const int lane = threadIdx.x & 63;
  const int row = blockIdx.x * 4 + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);   // wave-uniform
  if (row >= rows) return;
  const bf16* xr = x + (int64_t)row * cols;
  Vec16<bf16> xv[NV];
#pragma unroll
  for (int c = 0; c < NV; ++c) xv[c] = load16(xr + (c * 64 + lane) * 8);
  float s = 0.f;
  if constexpr (!RMS) {
#pragma unroll
    for (int c = 0; c < NV; ++c)
#pragma unroll
      for (int i = 0; i < 8; ++i) s += to_f32(xv[c].get(i));
  }
  const float mu = RMS ? 0.f : wave_sum(s) / (float)cols;
  if constexpr (kWideRow<NV>) settle(xv);
  float ss = 0.f;
#pragma unroll
  for (int c = 0; c < NV; ++c)
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const float d = to_f32(xv[c].get(i)) - mu;
      ss += d * d;
    }
  const float rs = 1.0f / sqrtf(wave_sum(ss) / (float)cols + eps);
  if constexpr (kWideRow<NV>) settle(xv);
  bf16* orow = out + (int64_t)row * cols;
#pragma unroll
  for (int c = 0; c < NV; ++c) {
    const int col = (c * 64 + lane) * 8;
    const Vec16<bf16> g = load16(gamma + col);
    Vec16<bf16> b;
    if constexpr (!RMS) b = load16(beta + col);
    Vec16<bf16> o;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const float n = (to_f32(xv[c].get(i)) - mu) * rs * to_f32(g.get(i));
      o.set(i, from_f32<bf16>(RMS ? n : n + to_f32(b.get(i))));
    }
    store16(orow + col, o);
  }
  if (lane == 0) {
    if (mean) mean[row] = mu;
    if (rstd) rstd[row] = rs;
  }
}

template <int NV, bool RMS = false>
__global__ __launch_bounds__(256) void ln_bwd_wave_kernel(const bf16* __restrict__ dout, const bf16* __restrict__ x,
                                                          const float* __restrict__ mean,
                                                          const float* __restrict__ rstd,
                                                          const bf16* __restrict__ gamma,
                                                          const bf16* __restrict__ resid, bf16* __restrict__ dx,
                                                          int rows, int cols) {
  const int lane = threadIdx.x & 63;
  const int row = blockIdx.x * 4 + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);   // wave-uniform
  if (row >= rows) return;
  const float mu = RMS ? 0.f : mean[row], rs = rstd[row];
  const bf16* xr = x + (int64_t)row * cols;
  const bf16* dr = dout + (int64_t)row * cols;
  // narrower rows load the residual gradient with the row; wide rows load it
  // chunk by chunk in the output pass
  constexpr bool WIDE = kWideRow<NV>;
  Vec16<bf16> xv[NV], dv[NV], rv[WIDE ? 1 : NV];
#pragma unroll
  for (int c = 0; c < NV; ++c) {
    const int col = (c * 64 + lane) * 8;
    xv[c] = load16(xr + col);
    dv[c] = load16(dr + col);
    if constexpr (!WIDE) {
      if (resid) rv[c] = load16(resid + (int64_t)row * cols + col);
    }
  }
  float s1 = 0.f, s2 = 0.f;
#pragma unroll
  for (int c = 0; c < NV; ++c) {
    const Vec16<bf16> g = load16(gamma + (c * 64 + lane) * 8);
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const float gv = to_f32(dv[c].get(i)) * to_f32(g.get(i));
      s1 += gv;
      s2 += gv * ((to_f32(xv[c].get(i)) - mu) * rs);
    }
  }
  const float m1 = RMS ? 0.f : wave_sum(s1) / (float)cols;
  const float m2 = wave_sum(s2) / (float)cols;
  if constexpr (WIDE) {
    settle(xv);
    settle(dv);
  }
  bf16* o = dx + (int64_t)row * cols;
#pragma unroll
  for (int c = 0; c < NV; ++c) {
    const int col = (c * 64 + lane) * 8;
    const Vec16<bf16> g = load16(gamma + col);
    if constexpr (WIDE) rv[0] = resid ? load16(resid + (int64_t)row * cols + col) : zero16<bf16>();
    const Vec16<bf16>& r = rv[WIDE ? 0 : c];
    Vec16<bf16> w;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const float gv = to_f32(dv[c].get(i)) * to_f32(g.get(i));
      const float zh = (to_f32(xv[c].get(i)) - mu) * rs;
      float val = rs * (gv - m1 - zh * m2);
      if (resid) val += to_f32(r.get(i));
      w.set(i, from_f32<bf16>(val));
    }
    store16(o + col, w);
  }
}

// Wave-per-row launch for bf16 rows of a multiple of 512 columns (up to 8192);
// returns false when the shape needs the block-per-row kernels.
#define TPS_WAVE_ROW_DISPATCH(KERNEL, FLAG, rows, cols, st, ...)                                       \
  ([&]() -> bool {                                                                                  \
    if ((cols) % 512 != 0 || (cols) > 8192) return false;                                            \
    const dim3 grid_(((rows) + 3) / 4), block_(256);                                                 \
    switch ((cols) / 512) {                                                                          \
      case 1: hipLaunchKernelGGL((KERNEL<1, FLAG>), grid_, block_, 0, st, __VA_ARGS__, rows, cols); break;   \
      case 2: hipLaunchKernelGGL((KERNEL<2, FLAG>), grid_, block_, 0, st, __VA_ARGS__, rows, cols); break;   \
      case 4: hipLaunchKernelGGL((KERNEL<4, FLAG>), grid_, block_, 0, st, __VA_ARGS__, rows, cols); break;   \
      case 8: hipLaunchKernelGGL((KERNEL<8, FLAG>), grid_, block_, 0, st, __VA_ARGS__, rows, cols); break;   \
      case 10: hipLaunchKernelGGL((KERNEL<10, FLAG>), grid_, block_, 0, st, __VA_ARGS__, rows, cols); break; \
      case 16: hipLaunchKernelGGL((KERNEL<16, FLAG>), grid_, block_, 0, st, __VA_ARGS__, rows, cols); break; \
      default: return false;                                                                         \
    }                                                                                                \
    return true;                                                                                     \
  }())

// Pass 1 of a column reduction: block (column group of 64, row segment).
// Thread (row lane rl, chunk cc) sums rows rl, rl+32, ... of the segment for
// 8 columns; the 32 row lanes are then added in ascending order.
// k = 0: sum x (or dout); k = 1 (LN mode): sum dout * (xin - mean) * rstd.
// The segment's sum of column c for output k goes to
// dst[segment * seg_stride + k * k_stride + c], stored (ACC false) or added
// to what is there (ACC true: one owner per element, so calls in stream order
// accumulate in a fixed order).
// MODE 2 (RMS): one output, sum dout * x * rstd (no centring).
template <typename T, int MODE, bool ACC>
__global__ __launch_bounds__(256) void colsum_part_kernel(const T* __restrict__ x, int64_t ldx,
                                                          const T* __restrict__ xin, const float* __restrict__ mean,
                                                          const float* __restrict__ rstd, float* __restrict__ dst,
                                                          int64_t seg_stride, int64_t k_stride, int rows, int cols,
                                                          int seg_rows) {
  constexpr int VEC = 16 / sizeof(T);
  constexpr int COLS = 8 * VEC;                 // columns per block
  constexpr bool LN = MODE == 1, ZH = MODE != 0;
  __shared__ float red[LN ? 2 : 1][32][COLS + 1];
  const int cc = threadIdx.x & 7, rl = threadIdx.x >> 3;
  const int col = blockIdx.x * COLS + cc * VEC;
  const int r0 = blockIdx.y * seg_rows, r1 = min(rows, r0 + seg_rows);
  float a[VEC], z[VEC];
#pragma unroll
  for (int i = 0; i < VEC; ++i) a[i] = z[i] = 0.f;
  if (col < cols) {
    // rows rl, rl + 32, ... of the segment, UNR loads in flight; the sum of
    // each lane runs in ascending row order
    constexpr int UNR = 4;
    for (int r = r0 + rl; r < r1; r += 32 * UNR) {
      Vec16<T> v[UNR], xv[UNR];
      float mu[UNR], rs[UNR];
#pragma unroll
      for (int u = 0; u < UNR; ++u) {
        const int ru = r + 32 * u;
        if (ru < r1) {
          v[u] = load16(x + (int64_t)ru * ldx + col);
          if constexpr (ZH) {
            xv[u] = load16(xin + (int64_t)ru * cols + col);
            mu[u] = LN ? mean[ru] : 0.f;
            rs[u] = rstd[ru];
          }
        }
      }
#pragma unroll
      for (int u = 0; u < UNR; ++u) {
        if (r + 32 * u < r1) {
          if constexpr (LN) {
#pragma unroll
            for (int i = 0; i < VEC; ++i) {
              const float d = to_f32(v[u].get(i));
              a[i] += d;
              z[i] += d * ((to_f32(xv[u].get(i)) - mu[u]) * rs[u]);
            }
          } else if constexpr (ZH) {
#pragma unroll
            for (int i = 0; i < VEC; ++i) a[i] += to_f32(v[u].get(i)) * (to_f32(xv[u].get(i)) * rs[u]);
          } else {
#pragma unroll
            for (int i = 0; i < VEC; ++i) a[i] += to_f32(v[u].get(i));
          }
        }
      }
    }
  }
#pragma unroll
  for (int i = 0; i < VEC; ++i) {
    red[0][rl][cc * VEC + i] = a[i];
    if constexpr (LN) red[1][rl][cc * VEC + i] = z[i];
  }
  __syncthreads();
  const int nk = LN ? 2 : 1;
  if (threadIdx.x < COLS * nk) {
    const int k = threadIdx.x / COLS, c = threadIdx.x % COLS;
    const int gc = blockIdx.x * COLS + c;
    float acc = 0.f;
    for (int i = 0; i < 32; ++i) acc += red[k][i][c];
    if (gc < cols) {
      float* d = dst + (int64_t)blockIdx.y * seg_stride + k * k_stride + gc;
      if constexpr (ACC) *d += acc;
      else *d = acc;
    }
  }
}

// Pass 2: out_k[c] += sum over segments in ascending order.
__global__ __launch_bounds__(256) void colsum_final_kernel(const float* __restrict__ ws, int parts, int nk,
                                                           int cols, float* __restrict__ out0,
                                                           float* __restrict__ out1) {
  const int c = blockIdx.x * 256 + threadIdx.x;
  if (c >= cols) return;
  // all partials are loaded before the (ascending, fixed-order) adds, so the
  // loads are in flight together; parts <= 16
  float p0[16], p1[16];
#pragma unroll
  for (int p = 0; p < 16; ++p) {
    p0[p] = p < parts ? ws[((int64_t)p * nk) * cols + c] : 0.f;
    p1[p] = (p < parts && nk == 2) ? ws[((int64_t)p * nk + 1) * cols + c] : 0.f;
  }
  float s0 = 0.f, s1 = 0.f;
#pragma unroll
  for (int p = 0; p < 16; ++p) {
    if (p < parts) {
      s0 += p0[p];
      s1 += p1[p];
    }
  }
  if (out0) out0[c] += s0;
  if (nk == 2 && out1) out1[c] += s1;
}

// Sums the segment partials of each column of a partial block (columns in
// ranges m.c0[r] .. m.c0[r+1], range r owned by the f32 vector at grads +
// m.goff[r]) in ascending segment order, adds them to that vector and clears
// the partials.
__global__ __launch_bounds__(256) void colsum_finalize_kernel(ColMap m, float* __restrict__ part, int segs,
                                                              int64_t seg_stride, float* __restrict__ grads,
                                                              int overwrite) {
  const int c = blockIdx.x * 256 + threadIdx.x;
  if (c >= m.c0[m.n]) return;
  int r = 0;
  while (r + 1 < m.n && c >= m.c0[r + 1]) ++r;
  float v[16];
#pragma unroll
  for (int i = 0; i < 16; ++i) v[i] = i < segs ? part[(int64_t)i * seg_stride + c] : 0.f;
  float acc = 0.f;
#pragma unroll
  for (int i = 0; i < 16; ++i)
    if (i < segs) acc += v[i];
  for (int i = 16; i < segs; ++i) acc += part[(int64_t)i * seg_stride + c];
  for (int i = 0; i < segs; ++i) part[(int64_t)i * seg_stride + c] = 0.f;
  float* gp = grads + m.goff[r] + (c - m.c0[r]);
  *gp = (overwrite ? 0.f : *gp) + acc;
}

template <typename T>
__global__ __launch_bounds__(256) void gelu_kernel(const T* __restrict__ u, T* __restrict__ g, int64_t n) {
  constexpr int VEC = 16 / sizeof(T);
  const int64_t i = ((int64_t)blockIdx.x * 256 + threadIdx.x) * VEC;
  if (i + VEC <= n) {
    const Vec16<T> v = load16(u + i);
    Vec16<T> w;
#pragma unroll
    for (int k = 0; k < VEC; ++k) w.set(k, from_f32<T>(gelu_f(to_f32(v.get(k)))));
    store16(g + i, w);
  } else {
    for (int64_t k = i; k < n; ++k) g[k] = from_f32<T>(gelu_f(to_f32(u[k])));
  }
}

// out[c][r] = in[r][c] over 64 x 64 tiles through LDS; rows, cols multiples of 8.
template <typename T>
__global__ __launch_bounds__(256) void transpose_kernel(const T* __restrict__ in, int64_t ldi, T* __restrict__ out,
                                                        int64_t ldo, int rows, int cols) {
  constexpr int VEC = 16 / sizeof(T);
  __shared__ T tile[64][64 + 1];
  const int r0 = blockIdx.y * 64, c0 = blockIdx.x * 64;
  for (int v = threadIdx.x; v < 64 * 64 / VEC; v += 256) {
    const int r = v / (64 / VEC), c = (v % (64 / VEC)) * VEC;
    if (r0 + r < rows && c0 + c < cols) {
      const Vec16<T> x = load16(in + (int64_t)(r0 + r) * ldi + c0 + c);
#pragma unroll
      for (int i = 0; i < VEC; ++i) tile[r][c + i] = x.get(i);
    }
  }
  __syncthreads();
  for (int v = threadIdx.x; v < 64 * 64 / VEC; v += 256) {
    const int c = v / (64 / VEC), r = (v % (64 / VEC)) * VEC;
    if (c0 + c < cols && r0 + r < rows) {
      Vec16<T> y;
#pragma unroll
      for (int i = 0; i < VEC; ++i) y.set(i, tile[r + i][c]);
      store16(out + (int64_t)(c0 + c) * ldo + r0 + r, y);
    }
  }
}

__global__ __launch_bounds__(256) void fill_bytes_kernel(u32x4* p, uint64_t n16, uint8_t* tail, uint32_t ntail,
                                                         uint32_t word) {
  const uint64_t i = (uint64_t)blockIdx.x * 256 + threadIdx.x;
  const uint64_t stride = (uint64_t)gridDim.x * 256;
  for (uint64_t k = i; k < n16; k += stride) p[k] = u32x4{word, word, word, word};
  if (i < ntail) tail[i] = (uint8_t)word;
}

// Per-row kernels are instantiated for NC 16-byte chunks per thread.
#define TPS_ROW_DISPATCH(KERNEL, T, FLAG, rows, cols, st, ...)                                     \
  do {                                                                                           \
    constexpr int VEC_ = 16 / sizeof(T);                                                         \
    const int nc_ = (cols + 256 * VEC_ - 1) / (256 * VEC_);                                      \
    dim3 grid_(rows), block_(256);                                                               \
    if (nc_ <= 1) hipLaunchKernelGGL((KERNEL<T, 1, FLAG>), grid_, block_, 0, st, __VA_ARGS__, rows, cols);       \
    else if (nc_ <= 2) hipLaunchKernelGGL((KERNEL<T, 2, FLAG>), grid_, block_, 0, st, __VA_ARGS__, rows, cols);  \
    else if (nc_ <= 4) hipLaunchKernelGGL((KERNEL<T, 4, FLAG>), grid_, block_, 0, st, __VA_ARGS__, rows, cols);  \
    else if (nc_ <= 8) hipLaunchKernelGGL((KERNEL<T, 8, FLAG>), grid_, block_, 0, st, __VA_ARGS__, rows, cols);  \
    else hipLaunchKernelGGL((KERNEL<T, 16, FLAG>), grid_, block_, 0, st, __VA_ARGS__, rows, cols);               \
  } while (0)

template <typename T>
hipError_t colsum_typed(int rows, int cols, const void* x, int64_t ldx, const void* xin, const float* mean,
                        const float* rstd, float* out0, float* out1, float* ws, int mode, hipStream_t st) {
  constexpr int VEC = 16 / sizeof(T);
  const int seg = (int)colsum_seg_rows(rows);
  const int parts = (int)colsum_segments(rows);
  dim3 grid((cols + 8 * VEC - 1) / (8 * VEC), parts);
  const int64_t nk = mode == 1 ? 2 : 1;
  const T* xi = static_cast<const T*>(mode ? xin : nullptr);
  if (mode == 1)
    hipLaunchKernelGGL((colsum_part_kernel<T, 1, false>), grid, dim3(256), 0, st, static_cast<const T*>(x), ldx, xi,
                       mean, rstd, ws, nk * cols, (int64_t)cols, rows, cols, seg);
  else if (mode == 2)
    hipLaunchKernelGGL((colsum_part_kernel<T, 2, false>), grid, dim3(256), 0, st, static_cast<const T*>(x), ldx, xi,
                       mean, rstd, ws, nk * cols, (int64_t)cols, rows, cols, seg);
  else
    hipLaunchKernelGGL((colsum_part_kernel<T, 0, false>), grid, dim3(256), 0, st, static_cast<const T*>(x), ldx, xi,
                       mean, rstd, ws, nk * cols, (int64_t)cols, rows, cols, seg);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(colsum_final_kernel, dim3((cols + 255) / 256), dim3(256), 0, st, ws, parts, (int)nk,
                     cols, out0, out1);
  return hipGetLastError();
}

// Pass 1 only, accumulating into a caller's partial block.
template <typename T>
hipError_t colsum_acc_typed(int rows, int cols, const void* x, int64_t ldx, const void* xin, const float* mean,
                            const float* rstd, float* part0, int64_t k_stride, int64_t seg_stride, int mode,
                            hipStream_t st) {
  constexpr int VEC = 16 / sizeof(T);
  const int seg = (int)colsum_seg_rows(rows);
  const int parts = (int)colsum_segments(rows);
  dim3 grid((cols + 8 * VEC - 1) / (8 * VEC), parts);
  const T* xi = static_cast<const T*>(mode ? xin : nullptr);
  if (mode == 1)
    hipLaunchKernelGGL((colsum_part_kernel<T, 1, true>), grid, dim3(256), 0, st, static_cast<const T*>(x), ldx, xi,
                       mean, rstd, part0, seg_stride, k_stride, rows, cols, seg);
  else if (mode == 2)
    hipLaunchKernelGGL((colsum_part_kernel<T, 2, true>), grid, dim3(256), 0, st, static_cast<const T*>(x), ldx, xi,
                       mean, rstd, part0, seg_stride, k_stride, rows, cols, seg);
  else
    hipLaunchKernelGGL((colsum_part_kernel<T, 0, true>), grid, dim3(256), 0, st, static_cast<const T*>(x), ldx, xi,
                       mean, rstd, part0, seg_stride, k_stride, rows, cols, seg);
  return hipGetLastError();
}

}  // namespace

uint64_t colsum_ws_bytes(int64_t rows, int64_t cols) { return colsum_ws_elems(rows, cols) * 4; }

hipError_t colsum_acc_launch(int dtype, int rows, int cols, const void* x, int64_t ldx, float* part,
                             int64_t seg_stride, hipStream_t st) {
  if (rows == 0) return hipSuccess;
  if (dtype == TPS_BF16)
    return colsum_acc_typed<bf16>(rows, cols, x, ldx, nullptr, nullptr, nullptr, part, 0, seg_stride, 0, st);
  return colsum_acc_typed<float>(rows, cols, x, ldx, nullptr, nullptr, nullptr, part, 0, seg_stride, 0, st);
}

hipError_t colsum_finalize_launch(const ColMap& m, float* part, int segs, int64_t seg_stride, float* grads,
                                  hipStream_t st, int overwrite) {
  const int cols = m.c0[m.n];
  if (cols == 0) return hipSuccess;
  hipLaunchKernelGGL(colsum_finalize_kernel, dim3((cols + 255) / 256), dim3(256), 0, st, m, part, segs, seg_stride,
                     grads, overwrite);
  return hipGetLastError();
}

hipError_t layernorm_fwd_launch(int dtype, int rows, int cols, const void* x, const void* gamma,
                                const void* beta, float eps, void* out, float* mean, float* rstd,
                                hipStream_t st) {
  if (rows == 0) return hipSuccess;
  if (dtype == TPS_BF16) {
    if (!TPS_WAVE_ROW_DISPATCH(ln_fwd_wave_kernel, false, rows, cols, st, (const bf16*)x, (const bf16*)gamma,
                               (const bf16*)beta, eps, (bf16*)out, mean, rstd))
      TPS_ROW_DISPATCH(ln_fwd_kernel, bf16, false, rows, cols, st, (const bf16*)x, (const bf16*)gamma, (const bf16*)beta,
                       eps, (bf16*)out, mean, rstd);
  } else
    TPS_ROW_DISPATCH(ln_fwd_kernel, float, false, rows, cols, st, (const float*)x, (const float*)gamma,
                     (const float*)beta, eps, (float*)out, mean, rstd);
  return hipGetLastError();
}

hipError_t layernorm_bwd_launch(int dtype, int rows, int cols, const void* dout, const void* x,
                                const float* mean, const float* rstd, const void* gamma,
                                const void* resid, void* dx, float* dgamma, float* dbeta,
                                float* ws, hipStream_t st) {
  if (rows == 0) return hipSuccess;
  if (dtype == TPS_BF16) {
    if (!TPS_WAVE_ROW_DISPATCH(ln_bwd_wave_kernel, false, rows, cols, st, (const bf16*)dout, (const bf16*)x, mean, rstd,
                               (const bf16*)gamma, (const bf16*)resid, (bf16*)dx))
      TPS_ROW_DISPATCH(ln_bwd_kernel, bf16, false, rows, cols, st, (const bf16*)dout, (const bf16*)x, mean, rstd,
                       (const bf16*)gamma, (const bf16*)resid, (bf16*)dx);
  } else
    TPS_ROW_DISPATCH(ln_bwd_kernel, float, false, rows, cols, st, (const float*)dout, (const float*)x, mean, rstd,
                     (const float*)gamma, (const float*)resid, (float*)dx);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || (dgamma == nullptr && dbeta == nullptr)) return e;
  // dbeta = sum dout (k = 0), dgamma = sum dout * zhat (k = 1)
  if (dtype == TPS_BF16)
    return colsum_typed<bf16>(rows, cols, dout, cols, x, mean, rstd, dbeta, dgamma, ws, 1, st);
  return colsum_typed<float>(rows, cols, dout, cols, x, mean, rstd, dbeta, dgamma, ws, 1, st);
}

hipError_t layernorm_bwd_acc_launch(int dtype, int rows, int cols, const void* dout, const void* x,
                                    const float* mean, const float* rstd, const void* gamma, const void* resid,
                                    void* dx, float* part_dbeta, int64_t k_stride, int64_t seg_stride,
                                    hipStream_t st) {
  if (rows == 0) return hipSuccess;
  hipError_t e = layernorm_bwd_launch(dtype, rows, cols, dout, x, mean, rstd, gamma, resid, dx, nullptr, nullptr,
                                      nullptr, st);
  if (e != hipSuccess) return e;
  if (dtype == TPS_BF16)
    return colsum_acc_typed<bf16>(rows, cols, dout, cols, x, mean, rstd, part_dbeta, k_stride, seg_stride, 1, st);
  return colsum_acc_typed<float>(rows, cols, dout, cols, x, mean, rstd, part_dbeta, k_stride, seg_stride, 1, st);
}

hipError_t colsum_launch(int dtype, int rows, int cols, const void* x, int64_t ldx, float* out,
                         float* ws, hipStream_t st) {
  if (rows == 0) return hipSuccess;
  if (dtype == TPS_BF16)
    return colsum_typed<bf16>(rows, cols, x, ldx, nullptr, nullptr, nullptr, out, nullptr, ws, 0, st);
  return colsum_typed<float>(rows, cols, x, ldx, nullptr, nullptr, nullptr, out, nullptr, ws, 0, st);
}

hipError_t gelu_launch(int dtype, int64_t n, const void* u, void* g, hipStream_t st) {
  if (n == 0) return hipSuccess;
  if (dtype == TPS_BF16) {
    const int64_t blocks = (n / 8 + 255) / 256 + 1;
    hipLaunchKernelGGL((gelu_kernel<bf16>), dim3((unsigned)blocks), dim3(256), 0, st, (const bf16*)u, (bf16*)g, n);
  } else {
    const int64_t blocks = (n / 4 + 255) / 256 + 1;
    hipLaunchKernelGGL((gelu_kernel<float>), dim3((unsigned)blocks), dim3(256), 0, st, (const float*)u, (float*)g, n);
  }
  return hipGetLastError();
}

hipError_t transpose_launch(int dtype, int rows, int cols, const void* in, int64_t ldi, void* out, int64_t ldo,
                            hipStream_t st) {
  if (rows == 0 || cols == 0) return hipSuccess;
  const dim3 grid((cols + 63) / 64, (rows + 63) / 64);
  if (dtype == TPS_BF16)
    hipLaunchKernelGGL((transpose_kernel<bf16>), grid, dim3(256), 0, st, (const bf16*)in, ldi, (bf16*)out, ldo, rows,
                       cols);
  else
    hipLaunchKernelGGL((transpose_kernel<float>), grid, dim3(256), 0, st, (const float*)in, ldi, (float*)out, ldo, rows,
                       cols);
  return hipGetLastError();
}

hipError_t rmsnorm_fwd_launch(int dtype, int rows, int cols, const void* x, const void* gamma, float eps, void* out,
                              float* rstd, hipStream_t st) {
  if (rows == 0) return hipSuccess;
  if (dtype == TPS_BF16) {
    if (!TPS_WAVE_ROW_DISPATCH(ln_fwd_wave_kernel, true, rows, cols, st, (const bf16*)x, (const bf16*)gamma,
                               (const bf16*)nullptr, eps, (bf16*)out, (float*)nullptr, rstd))
      TPS_ROW_DISPATCH(ln_fwd_kernel, bf16, true, rows, cols, st, (const bf16*)x, (const bf16*)gamma,
                       (const bf16*)nullptr, eps, (bf16*)out, (float*)nullptr, rstd);
  } else
    TPS_ROW_DISPATCH(ln_fwd_kernel, float, true, rows, cols, st, (const float*)x, (const float*)gamma,
                     (const float*)nullptr, eps, (float*)out, (float*)nullptr, rstd);
  return hipGetLastError();
}

namespace {
hipError_t rms_bwd_rows(int dtype, int rows, int cols, const void* dout, const void* x, const float* rstd,
                        const void* gamma, const void* resid, void* dx, hipStream_t st) {
  if (dtype == TPS_BF16) {
    if (!TPS_WAVE_ROW_DISPATCH(ln_bwd_wave_kernel, true, rows, cols, st, (const bf16*)dout, (const bf16*)x,
                               (const float*)nullptr, rstd, (const bf16*)gamma, (const bf16*)resid, (bf16*)dx))
      TPS_ROW_DISPATCH(ln_bwd_kernel, bf16, true, rows, cols, st, (const bf16*)dout, (const bf16*)x,
                       (const float*)nullptr, rstd, (const bf16*)gamma, (const bf16*)resid, (bf16*)dx);
  } else
    TPS_ROW_DISPATCH(ln_bwd_kernel, float, true, rows, cols, st, (const float*)dout, (const float*)x,
                     (const float*)nullptr, rstd, (const float*)gamma, (const float*)resid, (float*)dx);
  return hipGetLastError();
}
}  // namespace

hipError_t rmsnorm_bwd_launch(int dtype, int rows, int cols, const void* dout, const void* x, const float* rstd,
                              const void* gamma, const void* resid, void* dx, float* dgamma, float* ws,
                              hipStream_t st) {
  if (rows == 0) return hipSuccess;
  const hipError_t e = rms_bwd_rows(dtype, rows, cols, dout, x, rstd, gamma, resid, dx, st);
  if (e != hipSuccess || dgamma == nullptr) return e;
  if (dtype == TPS_BF16)
    return colsum_typed<bf16>(rows, cols, dout, cols, x, nullptr, rstd, dgamma, nullptr, ws, 2, st);
  return colsum_typed<float>(rows, cols, dout, cols, x, nullptr, rstd, dgamma, nullptr, ws, 2, st);
}

hipError_t rmsnorm_bwd_acc_launch(int dtype, int rows, int cols, const void* dout, const void* x, const float* rstd,
                                  const void* gamma, const void* resid, void* dx, float* part_dgamma,
                                  int64_t seg_stride, hipStream_t st) {
  if (rows == 0) return hipSuccess;
  const hipError_t e = rms_bwd_rows(dtype, rows, cols, dout, x, rstd, gamma, resid, dx, st);
  if (e != hipSuccess) return e;
  if (dtype == TPS_BF16)
    return colsum_acc_typed<bf16>(rows, cols, dout, cols, x, nullptr, rstd, part_dgamma, 0, seg_stride, 2, st);
  return colsum_acc_typed<float>(rows, cols, dout, cols, x, nullptr, rstd, part_dgamma, 0, seg_stride, 2, st);
}

hipError_t fill_bytes_launch(void* p, uint64_t bytes, uint8_t value, hipStream_t st) {
  if (bytes == 0) return hipSuccess;
  const uint64_t n16 = bytes / 16;
  const uint32_t ntail = (uint32_t)(bytes % 16);
  uint64_t blocks = (n16 + 255) / 256;
  if (blocks < 1) blocks = 1;
  if (blocks > 4096) blocks = 4096;
  hipLaunchKernelGGL(fill_bytes_kernel, dim3((unsigned)blocks), dim3(256), 0, st, (u32x4*)p, n16,
                     (uint8_t*)p + n16 * 16, ntail, 0x01010101u * value);
  return hipGetLastError();
}

hipError_t fill_zero_launch(void* p, uint64_t bytes, hipStream_t st) { return fill_bytes_launch(p, bytes, 0, st); }

}  // namespace tps
