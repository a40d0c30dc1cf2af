// Fused causal attention on gfx950 (exact softmax attention; the s x s score
// matrix never leaves registers).
//
// Layout: qkv [b*s, 3*H] with q | k | v column blocks, head n at columns
// n*D .. n*D+D-1 of each block; o and do are [b*s, H]; lse [b, heads, s] f32.
//
// Register layout trick: every product is issued so that the 32 queries (or
// keys) a wave owns are the MFMA's N (lane) dimension.  Softmax statistics
// of a query then live in one lane pair (l, l ^ 32), and a probability tile
// held in accumulators is fed straight back as the B operand of the next
// product: accumulator register j of lane l holds row acc_row(j, l), so the
// k-slots a lane supplies are the rows it already holds, and the A operand
// reads its LDS tile in that same row order (two 4-row runs per fragment).
//
// Backward is deterministic: one kernel owns a key block and sums dK, dV over
// all query tiles; a second kernel owns a query block and sums dQ over all key
// tiles.  No atomics, fixed loop orders.
#include "kernels.h"
#include "tps_device.h"

namespace tps {

namespace {

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

// Copy rows [row0, row0 + R) x [0, D) of a row-major global matrix (leading
// dimension ld, rows >= nrows read as zero) into LDS, natural layout
// [R][D + pad].
template <typename T, int R, int D, int LDN>
__device__ __forceinline__ void tile_natural(T* lds, const T* g, int64_t ld, int row0, int nrows) {
  constexpr int VEC = 16 / sizeof(T), CPR = D / VEC, NCH = R * CPR;
  for (int c = threadIdx.x; c < NCH; c += 256) {
    const int r = c / CPR, col = (c % CPR) * VEC;
    Vec16<T> v = (row0 + r < nrows) ? load16(g + (int64_t)(row0 + r) * ld + col) : zero16<T>();
    store16(lds + r * LDN + col, v);
  }
}

// Same rows, stored transposed in LDS: [D][R + pad].
template <typename T, int R, int D, int LDT>
__device__ __forceinline__ void tile_transposed(T* lds, const T* g, int64_t ld, int row0, int nrows) {
  constexpr int VEC = 16 / sizeof(T), RB = R / VEC, DB = D / VEC, NB = RB * DB;
  for (int b = threadIdx.x; b < NB; b += 256) {
    const int rb = b % RB, db = b / RB;
    Vec16<T> v[VEC];
#pragma unroll
    for (int t = 0; t < VEC; ++t) {
      const int r = row0 + rb * VEC + t;
      v[t] = (r < nrows) ? load16(g + (int64_t)r * ld + db * VEC) : zero16<T>();
    }
#pragma unroll
    for (int j = 0; j < VEC; ++j) {
      Vec16<T> w;
      if constexpr (sizeof(T) == 2) {
#pragma unroll
        for (int p = 0; p < 4; ++p) {
          const uint32_t lo = v[2 * p].raw[j >> 1], hi = v[2 * p + 1].raw[j >> 1];
          w.raw[p] = (j & 1) ? ((lo >> 16) | (hi & 0xFFFF0000u)) : ((lo & 0xFFFFu) | (hi << 16));
        }
      } else {
#pragma unroll
        for (int t = 0; t < VEC; ++t) w.set(t, v[t].get(j));
      }
      store16(lds + (db * VEC + j) * LDT + rb * VEC, w);
    }
  }
}

// A-operand fragment from a transposed LDS tile: lane (row m = l % 32 of the
// 32-row block at `base`, half hh) supplies columns rowset(r*KPL + i) of the
// 32-column block starting at col0, where rowset(j) = acc_row(j, lane).
template <typename T>
__device__ __forceinline__ typename Mma<T>::Frag frag_permuted(const T* lds_row, int col0, int r, int lane) {
  typedef typename Mma<T>::Frag F;
  F f;
  constexpr int KPL = Mma<T>::KPL;
  const int hh = lane >> 5;
  if constexpr (KPL == 8) {
    // j = 8r .. 8r+7 -> rows 16r + 4hh + {0..3} and 16r + 8 + 4hh + {0..3}
    const T* p0 = lds_row + col0 + 16 * r + 4 * hh;
    const u32x2 a = *reinterpret_cast<const u32x2*>(p0);
    const u32x2 b = *reinterpret_cast<const u32x2*>(p0 + 8);
    u32x4 w = {a[0], a[1], b[0], b[1]};
    f = *reinterpret_cast<F*>(&w);
  } else {
    f = lds_row[col0 + acc_row(r, lane)];
  }
  return f;
}

// B-operand fragment r from accumulator values (already scaled), rounded to T.
template <typename T>
__device__ __forceinline__ typename Mma<T>::Frag frag_from_acc(const float* v, int r) {
  typename Mma<T>::Frag f;
  constexpr int KPL = Mma<T>::KPL;
#pragma unroll
  for (int i = 0; i < KPL; ++i) frag_at(f, i) = from_f32<T>(v[r * KPL + i]);
  return f;
}

template <typename T>
__device__ __forceinline__ typename Mma<T>::Frag frag_global(const T* p) {
  if constexpr (sizeof(T) == 2) {
    u32x4 w = *reinterpret_cast<const u32x4*>(p);
    return *reinterpret_cast<typename Mma<T>::Frag*>(&w);
  } else {
    return *p;
  }
}

}  // namespace

// ---------------------------------------------------------------------------
// Forward: one workgroup = 128 queries of one (sequence, head); each of the 4
// waves owns 32 queries.  Key tiles of 64 stream through LDS (K natural, V
// transposed).  Online softmax in the exp2 domain.
// ---------------------------------------------------------------------------
template <typename T, int D>
__global__ __attribute__((amdgpu_flat_work_group_size(256, 256)))
void attn_fwd_kernel(const T* __restrict__ qkv, T* __restrict__ o, float* __restrict__ lse,
                     int b, int s, int nh, float scale) {
  typedef Mma<T> MM;
  constexpr int KPL = MM::KPL, KSTEP = 2 * KPL, NKS = D / KSTEP;
  constexpr int VEC = 16 / sizeof(T);
  constexpr int BQ = 128, BKV = 64;
  constexpr int LDK = D + VEC, LDV = BKV + VEC;
  __shared__ __attribute__((aligned(16))) T Ks[BKV * LDK];
  __shared__ __attribute__((aligned(16))) T Vt[D * LDV];

  const int H = nh * D;
  const int64_t ld = 3 * (int64_t)H;
  const int nqb = (s + BQ - 1) / BQ;
  const int idx = blockIdx.x;
  const int qb = nqb - 1 - idx / (nh * b);   // longest rows first
  const int n = (idx % (nh * b)) % nh;
  const int ib = (idx % (nh * b)) / nh;

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int qw0 = qb * BQ + wave * 32;
  const int q = qw0 + (lane & 31);
  const int hh = lane >> 5;
  const T* base = qkv + (int64_t)ib * s * ld;
  const T* Kg = base + H + n * D;
  const T* Vg = base + 2 * H + n * D;

  typename MM::Frag qf[NKS];
#pragma unroll
  for (int ks = 0; ks < NKS; ++ks) {
    if (q < s) {
      qf[ks] = frag_global<T>(base + (int64_t)q * ld + n * D + ks * KSTEP + hh * KPL);
    } else {
#pragma unroll
      for (int i = 0; i < KPL; ++i) frag_at(qf[ks], i) = from_f32<T>(0.f);
    }
  }

  f32x16 oacc[D / 32];
#pragma unroll
  for (int t = 0; t < D / 32; ++t)
#pragma unroll
    for (int r = 0; r < 16; ++r) oacc[t][r] = 0.f;
  float m_run = -INFINITY, l_run = 0.f;
  const float sl2 = scale * kLog2e;

  const int kend = min(s, qb * BQ + BQ);
  const int nkb = (kend + BKV - 1) / BKV;
  for (int kb = 0; kb < nkb; ++kb) {
    const int k0 = kb * BKV;
    tile_natural<T, BKV, D, LDK>(Ks, Kg, ld, k0, s);
    tile_transposed<T, BKV, D, LDV>(Vt, Vg, ld, k0, s);
    __syncthreads();
    if (qw0 + 31 >= k0 && qw0 < s) {
      float sv[BKV / 32][16];
#pragma unroll
      for (int kt = 0; kt < BKV / 32; ++kt) {
        f32x16 acc;
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[r] = 0.f;
        const T* krow = Ks + (kt * 32 + (lane & 31)) * LDK + hh * KPL;
#pragma unroll
        for (int ks = 0; ks < NKS; ++ks) {
          const typename MM::Frag a = *reinterpret_cast<const typename MM::Frag*>(krow + ks * KSTEP);
          acc = MM::run(a, qf[ks], acc);
        }
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int key = k0 + kt * 32 + acc_row(r, lane);
          sv[kt][r] = (key <= q && key < s) ? acc[r] * sl2 : -INFINITY;
        }
      }
      float mloc = -INFINITY;
#pragma unroll
      for (int kt = 0; kt < BKV / 32; ++kt)
#pragma unroll
        for (int r = 0; r < 16; ++r) mloc = fmaxf(mloc, sv[kt][r]);
      mloc = fmaxf(mloc, __shfl_xor(mloc, 32, kWave));
      const float m_new = fmaxf(m_run, mloc);
      const float m_use = (m_new == -INFINITY) ? 0.f : m_new;
      const float alpha = exp2f(m_run - m_use);
      l_run *= alpha;
#pragma unroll
      for (int t = 0; t < D / 32; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r) oacc[t][r] *= alpha;
#pragma unroll
      for (int kt = 0; kt < BKV / 32; ++kt)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const float p = exp2f(sv[kt][r] - m_use);
          sv[kt][r] = p;
          l_run += p;
        }
      m_run = m_new;
      // O^T[d, q] += V^T[d, key] P^T[key, q]
#pragma unroll
      for (int kt = 0; kt < BKV / 32; ++kt) {
#pragma unroll
        for (int r = 0; r < 16 / KPL; ++r) {
          const typename MM::Frag pb = frag_from_acc<T>(sv[kt], r);
#pragma unroll
          for (int t = 0; t < D / 32; ++t) {
            const typename MM::Frag va = frag_permuted<T>(Vt + (t * 32 + (lane & 31)) * LDV, kt * 32, r, lane);
            oacc[t] = MM::run(va, pb, oacc[t]);
          }
        }
      }
    }
    __syncthreads();
  }

  const float l_tot = l_run + __shfl_xor(l_run, 32, kWave);
  if (q < s) {
    const float inv = 1.f / l_tot;
    T* orow = o + ((int64_t)ib * s + q) * H + n * D;
#pragma unroll
    for (int t = 0; t < D / 32; ++t)
#pragma unroll
      for (int r = 0; r < 16; ++r) orow[t * 32 + acc_row(r, lane)] = from_f32<T>(oacc[t][r] * inv);
    if (lse != nullptr && hh == 0)
      lse[((int64_t)ib * nh + n) * s + q] = m_run * kLn2 + logf(l_tot);
  }
}

// ---------------------------------------------------------------------------
// Backward preprocessing: Dv[b, n, q] = sum_d do[q, n*D + d] * o[q, n*D + d].
// LPR lanes per (row, head) read 16 contiguous bytes of each operand (a wave
// covers 64 / LPR whole head rows: fully coalesced), multiply-add them in
// element order and sum across the LPR lanes with a fixed xor butterfly (every
// lane of the group ends with the same value).
// ---------------------------------------------------------------------------
template <typename T, int D>
__global__ void attn_bwd_dot_kernel(const T* __restrict__ o, const T* __restrict__ dout,
                                    float* __restrict__ dvec, int b, int s, int nh) {
  constexpr int VEC = 16 / sizeof(T);
  constexpr int LPR = D / VEC;
  static_assert(LPR <= kWave && kWave % LPR == 0 && (LPR & (LPR - 1)) == 0, "lanes per head row");
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t i = t / LPR;                              // (row, head) index
  const int c = (int)(t % LPR) * VEC;
  const int64_t total = (int64_t)b * s * nh;
  const bool ok = i < total;                              // uniform over the lane group
  const int n = ok ? (int)(i % nh) : 0;
  const int64_t row = ok ? i / nh : 0;
  const int64_t off = row * (int64_t)nh * D + (int64_t)n * D + c;
  float acc = 0.f;
  if (ok) {
    const Vec16<T> a = load16(o + off), g = load16(dout + off);
#pragma unroll
    for (int e = 0; e < VEC; ++e) acc += to_f32(a.get(e)) * to_f32(g.get(e));
  }
#pragma unroll
  for (int m = 1; m < LPR; m <<= 1) acc += __shfl_xor(acc, m, kWave);
  if (ok && c == 0) dvec[((row / s) * nh + n) * s + row % s] = acc;
}

template <typename T, int D>
static hipError_t dot_launch(int b, int s, int nh, const void* o, const void* dout, float* dvec, hipStream_t st) {
  constexpr int LPR = D * (int)sizeof(T) / 16;
  const int64_t threads = (int64_t)b * s * nh * LPR;
  hipLaunchKernelGGL((attn_bwd_dot_kernel<T, D>), dim3((unsigned)((threads + 255) / 256)), dim3(256), 0, st,
                     static_cast<const T*>(o), static_cast<const T*>(dout), dvec, b, s, nh);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// dK, dV: one workgroup = 128 keys (4 waves x 32) of one (sequence, head);
// query tiles of 64 stream through LDS (Q and dO, natural and transposed).
// ---------------------------------------------------------------------------
template <typename T, int D>
__global__ __attribute__((amdgpu_flat_work_group_size(256, 256), amdgpu_waves_per_eu(1, 1)))
void attn_bwd_dkdv_kernel(const T* __restrict__ qkv, const T* __restrict__ dout,
                          const float* __restrict__ lse, const float* __restrict__ dvec,
                          T* __restrict__ dqkv, int b, int s, int nh, float scale) {
  typedef Mma<T> MM;
  constexpr int KPL = MM::KPL, KSTEP = 2 * KPL, NKS = D / KSTEP;
  constexpr int VEC = 16 / sizeof(T);
  constexpr int BKB = 128, BQB = 64;
  constexpr int LDN = D + VEC, LDT = BQB + VEC;
  __shared__ __attribute__((aligned(16))) T Qs[BQB * LDN];
  __shared__ __attribute__((aligned(16))) T Qt[D * LDT];
  __shared__ __attribute__((aligned(16))) T dOs[BQB * LDN];
  __shared__ __attribute__((aligned(16))) T dOt[D * LDT];
  __shared__ float lse_s[BQB], dv_s[BQB];

  const int H = nh * D;
  const int64_t ld = 3 * (int64_t)H;
  const int idx = blockIdx.x;
  const int kb = idx / (nh * b);               // smallest key block = most work
  const int n = (idx % (nh * b)) % nh;
  const int ib = (idx % (nh * b)) / nh;

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, hh = lane >> 5;
  const int kw0 = kb * BKB + wave * 32;
  const int key = kw0 + (lane & 31);
  const T* base = qkv + (int64_t)ib * s * ld;
  const T* Qg = base + n * D;
  const T* dOg = dout + (int64_t)ib * s * H + n * D;
  const float* lse_g = lse + ((int64_t)ib * nh + n) * s;
  const float* dv_g = dvec + ((int64_t)ib * nh + n) * s;

  typename MM::Frag kf[NKS], vf[NKS];
#pragma unroll
  for (int ks = 0; ks < NKS; ++ks) {
    if (key < s) {
      kf[ks] = frag_global<T>(base + (int64_t)key * ld + H + n * D + ks * KSTEP + hh * KPL);
      vf[ks] = frag_global<T>(base + (int64_t)key * ld + 2 * H + n * D + ks * KSTEP + hh * KPL);
    } else {
#pragma unroll
      for (int i = 0; i < KPL; ++i) {
        frag_at(kf[ks], i) = from_f32<T>(0.f);
        frag_at(vf[ks], i) = from_f32<T>(0.f);
      }
    }
  }
  f32x16 dk[D / 32], dv[D / 32];
#pragma unroll
  for (int t = 0; t < D / 32; ++t)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      dk[t][r] = 0.f;
      dv[t][r] = 0.f;
    }
  const float sl2 = scale * kLog2e;

  const int nqt = (s + BQB - 1) / BQB;
  for (int qt = (kb * BKB) / BQB; qt < nqt; ++qt) {
    const int q0 = qt * BQB;
    tile_natural<T, BQB, D, LDN>(Qs, Qg, ld, q0, s);
    tile_transposed<T, BQB, D, LDT>(Qt, Qg, ld, q0, s);
    tile_natural<T, BQB, D, LDN>(dOs, dOg, H, q0, s);
    tile_transposed<T, BQB, D, LDT>(dOt, dOg, H, q0, s);
    if (threadIdx.x < BQB) {
      const int qq = q0 + threadIdx.x;
      lse_s[threadIdx.x] = (qq < s) ? lse_g[qq] * kLog2e : INFINITY;
      dv_s[threadIdx.x] = (qq < s) ? dv_g[qq] : 0.f;
    }
    __syncthreads();
    if (kw0 <= q0 + BQB - 1 && kw0 < s) {
#pragma unroll
      for (int qs = 0; qs < BQB / 32; ++qs) {
        f32x16 sa, pa;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          sa[r] = 0.f;
          pa[r] = 0.f;
        }
        const T* qrow = Qs + (qs * 32 + (lane & 31)) * LDN + hh * KPL;
        const T* drow = dOs + (qs * 32 + (lane & 31)) * LDN + hh * KPL;
#pragma unroll
        for (int ks = 0; ks < NKS; ++ks) {
          sa = MM::run(*reinterpret_cast<const typename MM::Frag*>(qrow + ks * KSTEP), kf[ks], sa);
          pa = MM::run(*reinterpret_cast<const typename MM::Frag*>(drow + ks * KSTEP), vf[ks], pa);
        }
        float pv[16], dsv[16];
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int ql = qs * 32 + acc_row(r, lane);
          const int qq = q0 + ql;
          const float p = (key <= qq && qq < s) ? exp2f(sa[r] * sl2 - lse_s[ql]) : 0.f;
          pv[r] = p;
          dsv[r] = p * (pa[r] - dv_s[ql]);
        }
#pragma unroll
        for (int r = 0; r < 16 / KPL; ++r) {
          const typename MM::Frag pb = frag_from_acc<T>(pv, r);
          const typename MM::Frag sb = frag_from_acc<T>(dsv, r);
#pragma unroll
          for (int t = 0; t < D / 32; ++t) {
            const typename MM::Frag da = frag_permuted<T>(dOt + (t * 32 + (lane & 31)) * LDT, qs * 32, r, lane);
            dv[t] = MM::run(da, pb, dv[t]);
            const typename MM::Frag qa = frag_permuted<T>(Qt + (t * 32 + (lane & 31)) * LDT, qs * 32, r, lane);
            dk[t] = MM::run(qa, sb, dk[t]);
          }
        }
      }
    }
    __syncthreads();
  }
  if (key < s) {
    T* row = dqkv + ((int64_t)ib * s + key) * ld + n * D;
#pragma unroll
    for (int t = 0; t < D / 32; ++t)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int d = t * 32 + acc_row(r, lane);
        row[H + d] = from_f32<T>(dk[t][r] * scale);
        row[2 * H + d] = from_f32<T>(dv[t][r]);
      }
  }
}

// ---------------------------------------------------------------------------
// dQ: one workgroup = 128 queries (4 waves x 32) of one (sequence, head); key
// tiles of 64 stream through LDS (K natural and transposed, V natural).
// ---------------------------------------------------------------------------
template <typename T, int D>
__global__ __attribute__((amdgpu_flat_work_group_size(256, 256)))
void attn_bwd_dq_kernel(const T* __restrict__ qkv, const T* __restrict__ dout,
                        const float* __restrict__ lse, const float* __restrict__ dvec,
                        T* __restrict__ dqkv, int b, int s, int nh, float scale) {
  typedef Mma<T> MM;
  constexpr int KPL = MM::KPL, KSTEP = 2 * KPL, NKS = D / KSTEP;
  constexpr int VEC = 16 / sizeof(T);
  constexpr int BQ = 128, BKT = 64;
  constexpr int LDN = D + VEC, LDT = BKT + VEC;
  __shared__ __attribute__((aligned(16))) T Ks[BKT * LDN];
  __shared__ __attribute__((aligned(16))) T Kt[D * LDT];
  __shared__ __attribute__((aligned(16))) T Vs[BKT * LDN];

  const int H = nh * D;
  const int64_t ld = 3 * (int64_t)H;
  const int nqb = (s + BQ - 1) / BQ;
  const int idx = blockIdx.x;
  const int qb = nqb - 1 - idx / (nh * b);
  const int n = (idx % (nh * b)) % nh;
  const int ib = (idx % (nh * b)) / nh;

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, hh = lane >> 5;
  const int qw0 = qb * BQ + wave * 32;
  const int q = qw0 + (lane & 31);
  const T* base = qkv + (int64_t)ib * s * ld;
  const T* Kg = base + H + n * D;
  const T* Vg = base + 2 * H + n * D;
  const T* dOg = dout + (int64_t)ib * s * H + n * D;

  typename MM::Frag qf[NKS], df[NKS];
#pragma unroll
  for (int ks = 0; ks < NKS; ++ks) {
    if (q < s) {
      qf[ks] = frag_global<T>(base + (int64_t)q * ld + n * D + ks * KSTEP + hh * KPL);
      df[ks] = frag_global<T>(dOg + (int64_t)q * H + ks * KSTEP + hh * KPL);
    } else {
#pragma unroll
      for (int i = 0; i < KPL; ++i) {
        frag_at(qf[ks], i) = from_f32<T>(0.f);
        frag_at(df[ks], i) = from_f32<T>(0.f);
      }
    }
  }
  const float sl2 = scale * kLog2e;
  const float lse2 = (q < s) ? lse[((int64_t)ib * nh + n) * s + q] * kLog2e : INFINITY;
  const float dq_dot = (q < s) ? dvec[((int64_t)ib * nh + n) * s + q] : 0.f;

  f32x16 dq[D / 32];
#pragma unroll
  for (int t = 0; t < D / 32; ++t)
#pragma unroll
    for (int r = 0; r < 16; ++r) dq[t][r] = 0.f;

  const int kend = min(s, qb * BQ + BQ);
  const int nkt = (kend + BKT - 1) / BKT;
  for (int kt = 0; kt < nkt; ++kt) {
    const int k0 = kt * BKT;
    tile_natural<T, BKT, D, LDN>(Ks, Kg, ld, k0, s);
    tile_transposed<T, BKT, D, LDT>(Kt, Kg, ld, k0, s);
    tile_natural<T, BKT, D, LDN>(Vs, Vg, ld, k0, s);
    __syncthreads();
    if (qw0 + 31 >= k0 && qw0 < s) {
#pragma unroll
      for (int ksb = 0; ksb < BKT / 32; ++ksb) {
        f32x16 sa, pa;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          sa[r] = 0.f;
          pa[r] = 0.f;
        }
        const T* krow = Ks + (ksb * 32 + (lane & 31)) * LDN + hh * KPL;
        const T* vrow = Vs + (ksb * 32 + (lane & 31)) * LDN + hh * KPL;
#pragma unroll
        for (int ks = 0; ks < NKS; ++ks) {
          sa = MM::run(*reinterpret_cast<const typename MM::Frag*>(krow + ks * KSTEP), qf[ks], sa);
          pa = MM::run(*reinterpret_cast<const typename MM::Frag*>(vrow + ks * KSTEP), df[ks], pa);
        }
        float dsv[16];
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int kk = k0 + ksb * 32 + acc_row(r, lane);
          const float p = (kk <= q && q < s) ? exp2f(sa[r] * sl2 - lse2) : 0.f;
          dsv[r] = p * (pa[r] - dq_dot);
        }
#pragma unroll
        for (int r = 0; r < 16 / KPL; ++r) {
          const typename MM::Frag sb = frag_from_acc<T>(dsv, r);
#pragma unroll
          for (int t = 0; t < D / 32; ++t) {
            const typename MM::Frag ka = frag_permuted<T>(Kt + (t * 32 + (lane & 31)) * LDT, ksb * 32, r, lane);
            dq[t] = MM::run(ka, sb, dq[t]);
          }
        }
      }
    }
    __syncthreads();
  }
  if (q < s) {
    T* row = dqkv + ((int64_t)ib * s + q) * ld + n * D;
#pragma unroll
    for (int t = 0; t < D / 32; ++t)
#pragma unroll
      for (int r = 0; r < 16; ++r) row[t * 32 + acc_row(r, lane)] = from_f32<T>(dq[t][r] * scale);
  }
}

// ---------------------------------------------------------------------------
// Host launchers
// ---------------------------------------------------------------------------
template <typename T, int D>
static hipError_t fwd_launch(int b, int s, int nh, const void* qkv, void* o, float* lse, hipStream_t st) {
  const int nqb = (s + 127) / 128;
  const float scale = 1.0f / sqrtf((float)D);
  hipLaunchKernelGGL((attn_fwd_kernel<T, D>), dim3(nqb * nh * b), dim3(256), 0, st,
                     static_cast<const T*>(qkv), static_cast<T*>(o), lse, b, s, nh, scale);
  return hipGetLastError();
}

template <typename T, int D>
static hipError_t bwd_launch(int b, int s, int nh, const void* qkv, const void* o, const float* lse,
                             const void* dout, void* dqkv, float* dvec, hipStream_t st) {
  const float scale = 1.0f / sqrtf((float)D);
  hipError_t e = dot_launch<T, D>(b, s, nh, o, dout, dvec, st);
  if (e != hipSuccess) return e;
  const int nkb = (s + 127) / 128;
  hipLaunchKernelGGL((attn_bwd_dkdv_kernel<T, D>), dim3(nkb * nh * b), dim3(256), 0, st,
                     static_cast<const T*>(qkv), static_cast<const T*>(dout), lse, dvec,
                     static_cast<T*>(dqkv), b, s, nh, scale);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int nqb = (s + 127) / 128;
  hipLaunchKernelGGL((attn_bwd_dq_kernel<T, D>), dim3(nqb * nh * b), dim3(256), 0, st,
                     static_cast<const T*>(qkv), static_cast<const T*>(dout), lse, dvec,
                     static_cast<T*>(dqkv), b, s, nh, scale);
  return hipGetLastError();
}

hipError_t attention_fwd_launch(int dtype, int b, int s, int nh, int nkv, int d, const void* qkv, void* o,
                                float* lse, hipStream_t st) {
  if (nkv != nh && !(dtype == TPS_BF16 && d == 128)) return hipErrorInvalidValue;
  if (dtype == TPS_BF16) {
    if (d == 128) return attention_fwd_v3_launch(b, s, nh, nkv, d, qkv, o, lse, st);
    return attention_fwd_v2_launch(b, s, nh, d, qkv, o, lse, st);
  }
  return d == 64 ? fwd_launch<float, 64>(b, s, nh, qkv, o, lse, st) : fwd_launch<float, 128>(b, s, nh, qkv, o, lse, st);
}

hipError_t attention_bwd_launch(int dtype, int b, int s, int nh, int nkv, int d, const void* qkv, const void* o,
                                const float* lse, const void* dout, void* dqkv, float* dvec, void* kv_ws,
                                hipStream_t st) {
  if (nkv != nh && !(dtype == TPS_BF16 && d == 128)) return hipErrorInvalidValue;
  if (dtype == TPS_BF16) {
    const hipError_t e = d == 128 ? dot_launch<bf16, 128>(b, s, nh, o, dout, dvec, st)
                                  : dot_launch<bf16, 64>(b, s, nh, o, dout, dvec, st);
    if (e != hipSuccess) return e;
    if (d == 128) return attention_bwd_v3_launch(b, s, nh, nkv, d, qkv, lse, dout, dqkv, dvec, kv_ws, st);
    return attention_bwd_v2_launch(b, s, nh, d, qkv, lse, dout, dqkv, dvec, st);
  }
  return d == 64 ? bwd_launch<float, 64>(b, s, nh, qkv, o, lse, dout, dqkv, dvec, st)
                 : bwd_launch<float, 128>(b, s, nh, qkv, o, lse, dout, dqkv, dvec, st);
}

}  // namespace tps
