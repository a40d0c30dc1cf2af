// Fused causal attention, bf16 path (head dim 64 or 128), on 16x16x32 MFMAs.
//
// Work split.  A wave owns 16 queries (forward, dQ) or 16 keys (dK/dV), so a
// sequence of 2048 tokens and 16 heads gives 2048 waves: two per SIMD.  The
// causal triangle makes query block j cost j+1 key tiles; each 8-wave
// workgroup takes the block pair (j, n-1-j): waves 0-3 work on block j, waves
// 4-7 on block n-1-j.  Waves w and w+4 share a SIMD, so every SIMD carries
// n+1 tiles of work and every workgroup the same amount.
//
// Data movement.  Key/value (or query/output-gradient) tiles of 64 rows are
// staged in LDS in their natural [row][d] layout, double buffered: tile t+1 is
// loaded into registers while tile t is used and written to the other stage
// afterwards, with one barrier per tile.  16-byte
// chunks are XOR-swizzled per row so that both access patterns are free of
// bank conflicts:
//   ds_read_b128 (16 rows, one chunk): an MFMA operand with d contiguous;
//   ds_read_tr16_b64 (4 rows, two chunks, per 16-lane group): an operand with
//   the row index (key or query) contiguous, i.e. the transposed tile.
//
// Accumulators feed the next product directly: a 16x16 result tile gives lane
// l rows 4*(l/16) + j of column l%16, and the k-slots 8*(l/16) + i of the next
// MFMA are mapped onto rows {4*(l/16) + i, 16 + 4*(l/16) + i} of a 32-row
// chunk; the transposed operand is read in that same row order.
//
// Backward is deterministic: dK, dV by key block over query tiles, dQ by
// query block over key tiles, fixed loop orders, no atomics.
#include "kernels.h"
#include "tps_device.h"

namespace tps {

namespace av2 {

typedef __attribute__((ext_vector_type(4))) short s16x4;
typedef __attribute__((ext_vector_type(8))) short s16x8;

constexpr int BT = 64;          // rows per tile (queries or keys)
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

__device__ __forceinline__ f32x4 mma(const bf16x8& a, const bf16x8& b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// Chunk swizzle of a [64][D] bf16 tile (D/8 chunks of 16 bytes per row).
// D = 128 (256-byte rows): f(r) = 4 (r & 3) + ((r >> 2) & 3) is a permutation
// of 0..15 over any 16 aligned rows, and f >> 1 differs within each aligned
// group of 4 rows.  D = 64 (128-byte rows, odd rows in the other bank half):
// f(r) = 2 ((r >> 1) & 3) + ((r >> 3) & 1), distinct over the even (and odd)
// rows of 16 aligned rows, and f >> 1 distinct for the two even (two odd) rows
// of an aligned group of 4.
template <int D>
__device__ __forceinline__ int swz(int r) {
  if constexpr (D == 128) return ((r & 3) << 2) | ((r >> 2) & 3);
  else return (((r >> 1) & 3) << 1) | ((r >> 3) & 1);
}
template <int D>
__device__ __forceinline__ int off(int r, int c) { return r * (D * 2) + ((c ^ swz<D>(r)) << 4); }

// Tile of rows row0..row0+63 (clamped to nrows-1; callers mask the clamped
// rows) of a [rows][ld] bf16 matrix starting at g, D columns, staged through
// registers: load() issues the global loads, store() writes the swizzled LDS
// tile.  Wave w moves 1 KB slots w, w+8, ...; lane l the 16 bytes at l * 16.
template <int D>
struct TileRegs {
  static constexpr int CPR = D / 8, INST = BT * CPR / 64, N = (INST + 7) / 8;
  u32x4 v[N];
  __device__ __forceinline__ void load(const bf16* g, int64_t ld, int row0, int nrows) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
    for (int n = 0; n < N; ++n) {
      const int slot = (wave + 8 * n) * 64 + lane;
      const int r = slot / CPR, p = slot % CPR;
      const int c = p ^ swz<D>(r);
      const int row = min(row0 + r, nrows - 1);
      v[n] = *reinterpret_cast<const u32x4*>(g + (int64_t)row * ld + c * 8);
    }
  }
  __device__ __forceinline__ void store(char* lds) const {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
    for (int n = 0; n < N; ++n) *reinterpret_cast<u32x4*>(lds + (wave + 8 * n) * 1024 + lane * 16) = v[n];
  }
};
static_assert(TileRegs<64>::INST == 8 && TileRegs<128>::INST == 16, "every wave moves whole slots");

// Operand with d contiguous: rows rbase + (l % 16), d = 32 ks + 8 (l / 16) .. +8.
template <int D>
__device__ __forceinline__ bf16x8 frag_rows(const char* lds, int rbase, int ks, int lane) {
  const int r = rbase + (lane & 15), c = 4 * ks + (lane >> 4);
  return *reinterpret_cast<const bf16x8*>(lds + off<D>(r, c));
}

// Transposed operand: lane (column cbase + l % 16, G = l / 16) gets rows
// rbase + 4G + i (i < 4) and rbase + 16 + 4G + (i - 4) (i >= 4).
template <int D>
__device__ __forceinline__ bf16x8 frag_cols(const char* lds, int rbase, int cbase, int lane) {
  const int G = lane >> 4, s = lane & 15;
  const int col = cbase + ((s & 3) << 2);
  const int c = col >> 3, within = (col & 7) * 2;
  const int r0 = rbase + 4 * G + (s >> 2);
  const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (__attribute__((address_space(3))) s16x4*)(lds + off<D>(r0, c) + within));
  const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (__attribute__((address_space(3))) s16x4*)(lds + off<D>(r0 + 16, c) + within));
  s16x8 v = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
  return *reinterpret_cast<bf16x8*>(&v);
}

// B operand from two accumulator tiles (rows 0-15 and 16-31 of a 32-row chunk).
__device__ __forceinline__ bf16x8 frag_acc(const float* lo, const float* hi) {
  bf16x8 f;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    f[i] = (bf16)lo[i];
    f[4 + i] = (bf16)hi[i];
  }
  return f;
}

// Consume a value before the tile loop: the wait for its global load is
// placed here, so no wait inside the loop has to drain the tile loads
// issued after it.
__device__ __forceinline__ void settle(const bf16x8& v) { asm volatile("" ::"v"(v)); }

__device__ __forceinline__ bf16x8 load_row_frag(const bf16* p) {
  u32x4 w = *reinterpret_cast<const u32x4*>(p);
  return *reinterpret_cast<bf16x8*>(&w);
}

// Block pair of a workgroup: waves 0-3 take block jA, waves 4-7 block jB.
struct Pair {
  int jA, jB, n, head, batch;
};
__device__ __forceinline__ Pair pair_of(int nblk, int nh) {
  const int npairs = (nblk + 1) / 2;
  Pair p;
  const int idx = blockIdx.x;
  const int pr = idx % npairs;
  p.head = (idx / npairs) % nh;
  p.batch = idx / (npairs * nh);
  p.jA = pr;
  p.jB = nblk - 1 - pr;
  p.n = nblk;
  return p;
}

}  // namespace av2

// ---------------------------------------------------------------------------
// Forward
// ---------------------------------------------------------------------------
template <int D>
__global__ __attribute__((amdgpu_flat_work_group_size(512, 512), amdgpu_waves_per_eu(2, 2)))
void attn_fwd_v2_kernel(const bf16* __restrict__ qkv, bf16* __restrict__ o, float* __restrict__ lse, int b, int s,
                        int nh, float scale) {
  using namespace av2;
  constexpr int TILE = BT * D * 2, STAGE = 2 * TILE, NKS = D / 32, NDT = D / 16;
  __shared__ __attribute__((aligned(1024))) char smem[2 * STAGE];

  const int H = nh * D;
  const int64_t ld = 3 * (int64_t)H;
  const int nblk = (s + BT - 1) / BT;
  const Pair pr = pair_of(nblk, nh);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, G = lane >> 4;
  const int jblk = (wave < 4) ? pr.jA : pr.jB;
  const bool active = (wave < 4) || (pr.jB != pr.jA);
  const int q0 = jblk * BT + (wave & 3) * 16;
  const int q = q0 + (lane & 15);
  const bf16* base = qkv + (int64_t)pr.batch * s * ld;
  const bf16* Kg = base + H + pr.head * D;
  const bf16* Vg = base + 2 * H + pr.head * D;

  bf16x8 qf[NKS];
#pragma unroll
  for (int ks = 0; ks < NKS; ++ks) {
    const int qq = min(q, s - 1);
    qf[ks] = load_row_frag(base + (int64_t)qq * ld + pr.head * D + ks * 32 + G * 8);
  }
#pragma unroll
  for (int ks = 0; ks < NKS; ++ks) settle(qf[ks]);
  f32x4 oacc[NDT];
#pragma unroll
  for (int t = 0; t < NDT; ++t) oacc[t] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m_run = -INFINITY, l_run = 0.f;
  const float sl2 = scale * kLog2e;

  const int ntile = pr.jB + 1;   // the longer block of the pair sets the loop length
  // tile t+1 is loaded into registers while tile t is used, then written to
  // the other LDS stage (last read in iteration t-1, before its barrier)
  TileRegs<D> kr, vr;
  kr.load(Kg, ld, 0, s);
  vr.load(Vg, ld, 0, s);
  kr.store(smem);
  vr.store(smem + TILE);
  __syncthreads();
  for (int t = 0; t < ntile; ++t) {
    if (t + 1 < ntile) {
      kr.load(Kg, ld, (t + 1) * BT, s);
      vr.load(Vg, ld, (t + 1) * BT, s);
    }
    if (active && t <= jblk) {
      const char* ks_lds = smem + (t & 1) * STAGE;
      const char* vs_lds = ks_lds + TILE;
      float sv[4][4];
#pragma unroll
      for (int st = 0; st < 4; ++st) {
        f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < NKS; ++ks) acc = mma(frag_rows<D>(ks_lds, st * 16, ks, lane), qf[ks], acc);
#pragma unroll
        for (int j = 0; j < 4; ++j) sv[st][j] = acc[j] * sl2;
      }
      if (t == jblk) {   // diagonal tile (also masks keys past the sequence end)
#pragma unroll
        for (int st = 0; st < 4; ++st)
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const int key = t * BT + st * 16 + 4 * G + j;
            if (key > q) sv[st][j] = -INFINITY;
          }
      }
      float mt = sv[0][0];
#pragma unroll
      for (int st = 0; st < 4; ++st)
#pragma unroll
        for (int j = 0; j < 4; ++j) mt = fmaxf(mt, sv[st][j]);
      mt = fmaxf(mt, __shfl_xor(mt, 16, kWave));
      mt = fmaxf(mt, __shfl_xor(mt, 32, kWave));
      const float m_new = fmaxf(m_run, mt);
      const float m_use = (m_new == -INFINITY) ? 0.f : m_new;
      const float alpha = exp2f(m_run - m_use);
      m_run = m_new;
      float ls = 0.f;
#pragma unroll
      for (int st = 0; st < 4; ++st)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          sv[st][j] = exp2f(sv[st][j] - m_use);
          ls += sv[st][j];
        }
      l_run = l_run * alpha + ls;
#pragma unroll
      for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
        for (int j = 0; j < 4; ++j) oacc[dt][j] *= alpha;
#pragma unroll
      for (int kc = 0; kc < 2; ++kc) {
        const bf16x8 pb = frag_acc(sv[2 * kc], sv[2 * kc + 1]);
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt) oacc[dt] = mma(frag_cols<D>(vs_lds, 32 * kc, dt * 16, lane), pb, oacc[dt]);
      }
    }
    if (t + 1 < ntile) {
      kr.store(smem + ((t + 1) & 1) * STAGE);
      vr.store(smem + ((t + 1) & 1) * STAGE + TILE);
    }
    __syncthreads();
  }
  float l_tot = l_run + __shfl_xor(l_run, 16, kWave);
  l_tot += __shfl_xor(l_tot, 32, kWave);
  if (active && q < s) {
    const float inv = 1.f / l_tot;
    bf16* orow = o + ((int64_t)pr.batch * s + q) * H + pr.head * D;
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt) {
      typedef __attribute__((ext_vector_type(4))) __bf16 bf16x4;
      bf16x4 w;
#pragma unroll
      for (int j = 0; j < 4; ++j) w[j] = (bf16)(oacc[dt][j] * inv);
      *reinterpret_cast<bf16x4*>(orow + dt * 16 + 4 * G) = w;
    }
    if (lse != nullptr && G == 0) lse[((int64_t)pr.batch * nh + pr.head) * s + q] = m_run * kLn2 + logf(l_tot);
  }
}

// ---------------------------------------------------------------------------
// dK, dV: waves own 16 keys; the pair is (key block j, key block n-1-j);
// query tiles t >= block stream through LDS (Q and dO).
// ---------------------------------------------------------------------------
template <int D>
__global__ __attribute__((amdgpu_flat_work_group_size(512, 512), amdgpu_waves_per_eu(2, 2)))
void attn_bwd_dkdv_v2_kernel(const bf16* __restrict__ qkv, const bf16* __restrict__ dout,
                             const float* __restrict__ lse, const float* __restrict__ dvec, bf16* __restrict__ dqkv,
                             int b, int s, int nh, float scale) {
  using namespace av2;
  constexpr int TILE = BT * D * 2, STAGE = 2 * TILE + 2 * BT * 4, NKS = D / 32, NDT = D / 16;
  __shared__ __attribute__((aligned(1024))) char smem[2 * STAGE];

  const int H = nh * D;
  const int64_t ld = 3 * (int64_t)H;
  const int nblk = (s + BT - 1) / BT;
  const Pair pr = pair_of(nblk, nh);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, G = lane >> 4;
  const int jblk = (wave < 4) ? pr.jA : pr.jB;
  const bool active = (wave < 4) || (pr.jB != pr.jA);
  const int key = jblk * BT + (wave & 3) * 16 + (lane & 15);
  const bf16* base = qkv + (int64_t)pr.batch * s * ld;
  const bf16* Qg = base + pr.head * D;
  const bf16* dOg = dout + (int64_t)pr.batch * s * H + pr.head * D;
  const float* lse_g = lse + ((int64_t)pr.batch * nh + pr.head) * s;
  const float* dv_g = dvec + ((int64_t)pr.batch * nh + pr.head) * s;

  bf16x8 kf[NKS], vf[NKS];
  {
    const int kk = min(key, s - 1);
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) {
      kf[ks] = load_row_frag(base + (int64_t)kk * ld + H + pr.head * D + ks * 32 + G * 8);
      vf[ks] = load_row_frag(base + (int64_t)kk * ld + 2 * H + pr.head * D + ks * 32 + G * 8);
    }
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) {
      settle(kf[ks]);
      settle(vf[ks]);
    }
  }
  f32x4 dk[NDT], dv[NDT];
#pragma unroll
  for (int t = 0; t < NDT; ++t) dk[t] = dv[t] = f32x4{0.f, 0.f, 0.f, 0.f};
  const float sl2 = scale * kLog2e;

  // query tiles from the earlier block of the pair to the end
  const int t0 = pr.jA;
  // query tile t+1 (Q, dO and its lse / D entries) is loaded into registers
  // while tile t is used, then written to the other LDS stage
  TileRegs<D> qr, dr;
  // (lse and D are read raw and transformed at the store, so the load of
  // tile t+1 is not waited for before tile t's work)
  float lse_r = 0.f, dv_r = 0.f;
  auto load_tile = [&](int t) {
    qr.load(Qg, ld, t * BT, s);
    dr.load(dOg, H, t * BT, s);
    if (threadIdx.x < BT) {
      const int qq = min(t * BT + (int)threadIdx.x, s - 1);
      lse_r = lse_g[qq];
      dv_r = dv_g[qq];
    }
  };
  auto store_tile = [&](int t, char* st) {
    qr.store(st);
    dr.store(st + TILE);
    if (threadIdx.x < BT) {
      const bool in = t * BT + (int)threadIdx.x < s;
      reinterpret_cast<float*>(st + 2 * TILE)[threadIdx.x] = in ? lse_r * kLog2e : INFINITY;
      reinterpret_cast<float*>(st + 2 * TILE)[BT + threadIdx.x] = in ? dv_r : 0.f;
    }
  };
  load_tile(t0);
  store_tile(t0, smem);
  __syncthreads();
  for (int t = t0; t < nblk; ++t) {
    char* cur = smem + ((t - t0) & 1) * STAGE;
    const float* lse_s = reinterpret_cast<const float*>(cur + 2 * TILE);
    const float* dv_s = lse_s + BT;
    if (t + 1 < nblk) load_tile(t + 1);
    if (active && t >= jblk) {
      const char* qs_lds = cur;
      const char* ds_lds = cur + TILE;
      float pv[4][4], dsv[4][4];
#pragma unroll
      for (int qs = 0; qs < 4; ++qs) {
        f32x4 sa = {0.f, 0.f, 0.f, 0.f}, pa = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < NKS; ++ks) {
          sa = mma(frag_rows<D>(qs_lds, qs * 16, ks, lane), kf[ks], sa);
          pa = mma(frag_rows<D>(ds_lds, qs * 16, ks, lane), vf[ks], pa);
        }
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int ql = qs * 16 + 4 * G + j;
          float p = exp2f(sa[j] * sl2 - lse_s[ql]);
          if (t == jblk && key > t * BT + ql) p = 0.f;
          pv[qs][j] = p;
          dsv[qs][j] = p * (pa[j] - dv_s[ql]);
        }
      }
#pragma unroll
      for (int kc = 0; kc < 2; ++kc) {
        const bf16x8 pb = frag_acc(pv[2 * kc], pv[2 * kc + 1]);
        const bf16x8 sb = frag_acc(dsv[2 * kc], dsv[2 * kc + 1]);
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt) {
          dv[dt] = mma(frag_cols<D>(ds_lds, 32 * kc, dt * 16, lane), pb, dv[dt]);
          dk[dt] = mma(frag_cols<D>(qs_lds, 32 * kc, dt * 16, lane), sb, dk[dt]);
        }
      }
    }
    if (t + 1 < nblk) store_tile(t + 1, smem + ((t + 1 - t0) & 1) * STAGE);
    __syncthreads();
  }
  if (active && key < s) {
    bf16* row = dqkv + ((int64_t)pr.batch * s + key) * ld + pr.head * D;
    typedef __attribute__((ext_vector_type(4))) __bf16 bf16x4;
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt) {
      bf16x4 wk, wv;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        wk[j] = (bf16)(dk[dt][j] * scale);
        wv[j] = (bf16)dv[dt][j];
      }
      *reinterpret_cast<bf16x4*>(row + H + dt * 16 + 4 * G) = wk;
      *reinterpret_cast<bf16x4*>(row + 2 * H + dt * 16 + 4 * G) = wv;
    }
  }
}

// ---------------------------------------------------------------------------
// dQ: waves own 16 queries; pair of query blocks as in the forward; key
// tiles 0..block stream through LDS (K and V).
// ---------------------------------------------------------------------------
template <int D>
__global__ __attribute__((amdgpu_flat_work_group_size(512, 512), amdgpu_waves_per_eu(2, 2)))
void attn_bwd_dq_v2_kernel(const bf16* __restrict__ qkv, const bf16* __restrict__ dout,
                           const float* __restrict__ lse, const float* __restrict__ dvec, bf16* __restrict__ dqkv,
                           int b, int s, int nh, float scale) {
  using namespace av2;
  constexpr int TILE = BT * D * 2, STAGE = 2 * TILE, NKS = D / 32, NDT = D / 16;
  __shared__ __attribute__((aligned(1024))) char smem[2 * STAGE];

  const int H = nh * D;
  const int64_t ld = 3 * (int64_t)H;
  const int nblk = (s + BT - 1) / BT;
  const Pair pr = pair_of(nblk, nh);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, G = lane >> 4;
  const int jblk = (wave < 4) ? pr.jA : pr.jB;
  const bool active = (wave < 4) || (pr.jB != pr.jA);
  const int q = jblk * BT + (wave & 3) * 16 + (lane & 15);
  const bf16* base = qkv + (int64_t)pr.batch * s * ld;
  const bf16* Kg = base + H + pr.head * D;
  const bf16* Vg = base + 2 * H + pr.head * D;
  const bf16* dOg = dout + (int64_t)pr.batch * s * H + pr.head * D;

  bf16x8 qf[NKS], df[NKS];
  {
    const int qq = min(q, s - 1);
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) {
      qf[ks] = load_row_frag(base + (int64_t)qq * ld + pr.head * D + ks * 32 + G * 8);
      df[ks] = load_row_frag(dOg + (int64_t)qq * H + ks * 32 + G * 8);
    }
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) {
      settle(qf[ks]);
      settle(df[ks]);
    }
  }
  const float sl2 = scale * kLog2e;
  const float lse2 = (q < s) ? lse[((int64_t)pr.batch * nh + pr.head) * s + q] * kLog2e : INFINITY;
  const float dq_dot = (q < s) ? dvec[((int64_t)pr.batch * nh + pr.head) * s + q] : 0.f;
  f32x4 dq[NDT];
#pragma unroll
  for (int t = 0; t < NDT; ++t) dq[t] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int ntile = pr.jB + 1;
  // tile t+1 is loaded into registers while tile t is used, then written to
  // the other LDS stage (last read in iteration t-1, before its barrier)
  TileRegs<D> kr, vr;
  kr.load(Kg, ld, 0, s);
  vr.load(Vg, ld, 0, s);
  kr.store(smem);
  vr.store(smem + TILE);
  __syncthreads();
  for (int t = 0; t < ntile; ++t) {
    if (t + 1 < ntile) {
      kr.load(Kg, ld, (t + 1) * BT, s);
      vr.load(Vg, ld, (t + 1) * BT, s);
    }
    if (active && t <= jblk) {
      const char* ks_lds = smem + (t & 1) * STAGE;
      const char* vs_lds = ks_lds + TILE;
      float dsv[4][4];
#pragma unroll
      for (int st = 0; st < 4; ++st) {
        f32x4 sa = {0.f, 0.f, 0.f, 0.f}, pa = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < NKS; ++ks) {
          sa = mma(frag_rows<D>(ks_lds, st * 16, ks, lane), qf[ks], sa);
          pa = mma(frag_rows<D>(vs_lds, st * 16, ks, lane), df[ks], pa);
        }
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int kk = t * BT + st * 16 + 4 * G + j;
          float p = exp2f(sa[j] * sl2 - lse2);
          if (t == jblk && kk > q) p = 0.f;
          dsv[st][j] = p * (pa[j] - dq_dot);
        }
      }
#pragma unroll
      for (int kc = 0; kc < 2; ++kc) {
        const bf16x8 sb = frag_acc(dsv[2 * kc], dsv[2 * kc + 1]);
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt) dq[dt] = mma(frag_cols<D>(ks_lds, 32 * kc, dt * 16, lane), sb, dq[dt]);
      }
    }
    if (t + 1 < ntile) {
      kr.store(smem + ((t + 1) & 1) * STAGE);
      vr.store(smem + ((t + 1) & 1) * STAGE + TILE);
    }
    __syncthreads();
  }
  if (active && q < s) {
    bf16* row = dqkv + ((int64_t)pr.batch * s + q) * ld + pr.head * D;
    typedef __attribute__((ext_vector_type(4))) __bf16 bf16x4;
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt) {
      bf16x4 w;
#pragma unroll
      for (int j = 0; j < 4; ++j) w[j] = (bf16)(dq[dt][j] * scale);
      *reinterpret_cast<bf16x4*>(row + dt * 16 + 4 * G) = w;
    }
  }
}

// ---------------------------------------------------------------------------
// Launchers (bf16 only)
// ---------------------------------------------------------------------------
static int pairs_grid(int b, int s, int nh) {
  const int nblk = (s + av2::BT - 1) / av2::BT;
  return ((nblk + 1) / 2) * nh * b;
}

hipError_t attention_fwd_v2_launch(int b, int s, int nh, int d, const void* qkv, void* o, float* lse,
                                   hipStream_t st) {
  const float scale = 1.0f / sqrtf((float)d);
  const dim3 grid(pairs_grid(b, s, nh)), block(512);
  if (d == 128)
    hipLaunchKernelGGL((attn_fwd_v2_kernel<128>), grid, block, 0, st, (const bf16*)qkv, (bf16*)o, lse, b, s, nh,
                       scale);
  else
    hipLaunchKernelGGL((attn_fwd_v2_kernel<64>), grid, block, 0, st, (const bf16*)qkv, (bf16*)o, lse, b, s, nh,
                       scale);
  return hipGetLastError();
}

hipError_t attention_bwd_v2_launch(int b, int s, int nh, int d, const void* qkv, const float* lse, const void* dout,
                                   void* dqkv, const float* dvec, hipStream_t st) {
  const float scale = 1.0f / sqrtf((float)d);
  const dim3 grid(pairs_grid(b, s, nh)), block(512);
  if (d == 128) {
    hipLaunchKernelGGL((attn_bwd_dkdv_v2_kernel<128>), grid, block, 0, st, (const bf16*)qkv, (const bf16*)dout, lse,
                       dvec, (bf16*)dqkv, b, s, nh, scale);
    hipLaunchKernelGGL((attn_bwd_dq_v2_kernel<128>), grid, block, 0, st, (const bf16*)qkv, (const bf16*)dout, lse, dvec,
                       (bf16*)dqkv, b, s, nh, scale);
  } else {
    hipLaunchKernelGGL((attn_bwd_dkdv_v2_kernel<64>), grid, block, 0, st, (const bf16*)qkv, (const bf16*)dout, lse,
                       dvec, (bf16*)dqkv, b, s, nh, scale);
    hipLaunchKernelGGL((attn_bwd_dq_v2_kernel<64>), grid, block, 0, st, (const bf16*)qkv, (const bf16*)dout, lse, dvec,
                       (bf16*)dqkv, b, s, nh, scale);
  }
  return hipGetLastError();
}

}  // namespace tps
