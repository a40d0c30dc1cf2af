// Fused causal attention backward, bf16, head dim 128, on 32x32x16 MFMAs.
//
// With P = softmax_causal(q k^T / sqrt d), D_i = sum_d dO_id O_id (computed by
// attn_bwd_dot_kernel) and lse the forward's log-sum-exp:
//   P_ij  = exp(s q_i.k_j - lse_i),   dP_ij = dO_i . v_j,
//   dS_ij = P_ij (dP_ij - D_i),
//   dV_j  = sum_i P_ij dO_i,  dK_j = s sum_i dS_ij q_i,  dQ_i = s sum_j dS_ij k_j,
// summed over the causal triangle j <= i.  Two kernels, both deterministic
// (every output element is produced by one wave, or summed from two waves'
// partials, in a fixed order; no atomics).  Each runs one wave per SIMD and
// comes in two shapes: 4 slices of 32 rows (128 rows per workgroup) with one
// tile stream, or 2 slices (64 rows) whose tile range is split in two parts,
// each part with its own stream and ring, summed part 0 first through LDS at
// the end; the second halves the longest chain of tiles of small grids.
//
// dK/dV (attn_bwd_dkdv_v3_kernel): a workgroup owns 32 keys per slice, K and
//   V fragments in registers; 64-query tiles of Q, dO, lse and D stream
//   through a two-stage LDS ring.  With keys along the MFMA N
//   dimension (one key per lane):
//     S  = Q K^T, dP = dO V^T        (Q, dO rows from LDS)
//     dV^T += dO^T P, dK^T += Q^T dS (dO^T, Q^T through transposing reads, in
//                                     the accumulators' query order)
//   64 MFMAs per tile; one wave per SIMD (the dK/dV accumulators take AGPRs).
// dQ (attn_bwd_dq_v3_kernel): a workgroup owns 32 queries per slice, Q and
//   dO fragments plus lse and D in registers; 64-key tiles of K and V stream
//   through the ring.  With queries along N:
//     S^T = K Q^T, dP^T = V dO^T, dQ^T += K^T dS^T
//   48 MFMAs per tile; one wave per SIMD (Q, dO fragments and dQ
//   accumulators do not fit the register budget of two).
// Workgroups are launched heaviest first.  Rows past the sequence end load as
// zeros: their Q and dO rows contribute nothing to dK/dV, and keys past the end
// lie beyond every query, so the causal mask removes them from dQ.
#include "attn_tiles.h"

namespace tps {

using namespace at;

// ---------------------------------------------------------------------------
// dK, dV
// ---------------------------------------------------------------------------
template <int KW, int PARTS>
__global__ __attribute__((amdgpu_flat_work_group_size(64 * KW * PARTS, 64 * KW * PARTS), amdgpu_waves_per_eu(1, 1)))
void attn_bwd_dkdv_v3_kernel(const bf16* __restrict__ qkv, const bf16* __restrict__ dout,
                             const float* __restrict__ lse, const float* __restrict__ dvec, bf16* __restrict__ dqkv,
                             int b, int s, int nh, float scale) {
  constexpr int VEC = 1024;                    // LDS bytes per per-row vector (64 f32 + landing pad)
  constexpr int STAGE = 2 * TILE + 2 * VEC;    // Q, dO, lse, D
  constexpr int RING = 2 * STAGE;              // one query part's two stages
  constexpr int BKEY = 32 * KW;                // keys per workgroup
  static_assert(PARTS == 1 || PARTS == 2, "query parts");
  __shared__ __attribute__((aligned(1024))) char smem[PARTS * RING];

  const int H = nh * D;
  const int64_t ld = 3 * (int64_t)H;
  const int idx = blockIdx.x;
  const int head = idx % nh;
  const int batch = (idx / nh) % b;
  const int kb = idx / (nh * b);                // first key blocks carry the most queries
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int g = lane >> 5;
  const int slice = wave % KW, part = wave / KW;
  const int k0 = kb * BKEY + slice * 32;       // first key of this wave
  const int key = k0 + (lane & 31);

  const bf16* base = qkv + (int64_t)batch * s * ld;
  // K^T and V^T fragments (B operands): lane holds key's d = 16 ks + 8 g .. +8
  bf16x8 kf[D / 16], vf[D / 16];
  {
    const bf16* krow = base + (int64_t)min(key, s - 1) * ld + H + head * D + 8 * g;
#pragma unroll
    for (int ks = 0; ks < D / 16; ++ks) {
      kf[ks] = load_frag_settled(krow + 16 * ks);
      vf[ks] = load_frag_settled(krow + H + 16 * ks);
    }
  }
  // query tiles from the one holding this workgroup's first key to the end,
  // and this part's share of them
  const int t0 = (kb * BKEY) / BT;
  const int ntile = (s + BT - 1) / BT;
  const int n = ntile - t0;
  const int n0 = PARTS == 1 ? n : (n + 1) / 2;
  const int tb = part ? t0 + n0 : t0;          // first tile of this part
  const int np = part ? n - n0 : n0;           // tiles of this part
  const int nit = n0;                          // loop trips (both parts, for the barriers)
  const int wave_first = k0 / BT;              // earlier tiles have no query >= any key of the wave

  TileSrcN<KW> qsrc, dsrc;
  qsrc.init(base + head * D, ld, s, slice, lane);
  dsrc.init(dout + (int64_t)batch * s * H + head * D, H, s, slice, lane);
  VecSrc lsrc, vsrc;
  lsrc.init(lse + ((int64_t)batch * nh + head) * s, s);
  vsrc.init(dvec + ((int64_t)batch * nh + head) * s, s);
  char* const ring = smem + part * RING;
  auto load_tile = [&](int t, int st) {
    char* p = ring + st * STAGE;
    qsrc.load(t * BT, p);
    dsrc.load(t * BT, p + TILE);
    if (slice == 0) {
      lsrc.load(t * BT, p + 2 * TILE, lane);
      vsrc.load(t * BT, p + 2 * TILE + VEC, lane);
    }
  };
  // load instructions per tile: the tiles' share, plus the vectors for slice 0
  constexpr int LPT = 2 * TileSrcN<KW>::IPW;
  FragOff fo;
  fo.init(lane);
  const uint32_t lds0 = lds_u32(ring);

  f32x16 dk[D / 32], dv[D / 32];
#pragma unroll
  for (int mt = 0; mt < D / 32; ++mt)
#pragma unroll
    for (int r = 0; r < 16; ++r) dk[mt][r] = dv[mt][r] = 0.f;
  const float sl2 = scale * kLog2e;
  // causal test on a diagonal tile: query 64 t + c < key  <=>  c < key - 4 g - 64 t,
  // c = 32 qb + 8 (j / 4) + j % 4 the query offset of accumulator j of block qb
  const int kthr = key - 4 * g;

  // One 64-query tile, as two 32-query halves each taken through the whole
  // chain (S, dP -> P, dS -> dV, dK): only one half's scores, probabilities
  // and per-row vectors are live at a time, which keeps the K/V fragments and
  // the dK/dV accumulators resident in registers.
  auto tile = [&](int t, int st, auto diag_c) {
    constexpr bool DIAG = decltype(diag_c)::value;
    const uint32_t qs = lds0 + st * STAGE, ds = qs + TILE, ls = ds + TILE, vs = ls + VEC;
    static_for<2>([&](auto qc) {
      constexpr int qb = decltype(qc)::value;
      // ---- S = Q K^T and dP = dO V^T for queries 32 qb .. +32: 8 d-steps each
      f32x16 sacc, pacc;
#pragma unroll
      for (int r = 0; r < 16; ++r) sacc[r] = pacc[r] = 0.f;
      bf16x8 fr[16];
      // issue order i: operand (Q, dO) = i % 2, d-step = i / 2
      auto read_f = [&](auto ic) {
        constexpr int i = decltype(ic)::value, w = i % 2, ks = i / 2;
        fr[i] = ds_b128<qb * 32 * ROWB>((w ? ds : qs) + fo.row[ks]);
      };
      constexpr int WF = 8;   // fragments in flight
      static_for<WF>([&](auto ic) { read_f(ic); });
      static_for<16>([&](auto ic) {
        constexpr int i = decltype(ic)::value, w = i % 2, ks = i / 2;
        constexpr int issued = (i + WF < 16) ? i + WF : 16;
        wait_lgkm<issued - i - 1>();
        pin(fr[i]);
        if constexpr (w == 0) sacc = Mma<bf16>::run(fr[i], kf[ks], sacc);
        else pacc = Mma<bf16>::run(fr[i], vf[ks], pacc);
        if constexpr (i + WF < 16) read_f(std::integral_constant<int, i + WF>{});
      });
      // ---- lse and D of the rows this lane holds: 32 qb + 8 (j / 4) + 4 g + (j % 4)
      f32x4 lv[4], dvv[4];
#pragma unroll
      for (int j4 = 0; j4 < 4; ++j4) {
        const uint32_t o = (uint32_t)((32 * qb + 8 * j4 + 4 * g) * 4);
        asm volatile("ds_read_b128 %0, %1" : "=v"(lv[j4]) : "v"(ls + o));
        asm volatile("ds_read_b128 %0, %1" : "=v"(dvv[j4]) : "v"(vs + o));
      }
      wait_lgkm<0>();
#pragma unroll
      for (int j4 = 0; j4 < 4; ++j4) {
        pin(lv[j4]);
        pin(dvv[j4]);
      }
      // ---- P, dS
      float p[16], d[16];
#pragma unroll
      for (int j = 0; j < 16; ++j) {
        float pv = __builtin_amdgcn_exp2f(__builtin_fmaf(sacc[j], sl2, -lv[j / 4][j % 4] * kLog2e));
        if constexpr (DIAG) {
          if (32 * qb + 8 * (j / 4) + (j % 4) < kthr - t * BT) pv = 0.f;
        }
        p[j] = pv;
        d[j] = pv * (pacc[j] - dvv[j / 4][j % 4]);
      }
      bf16x8 pb[2], sb[2];
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        pb[u] = to_frag(&p[8 * u]);
        sb[u] = to_frag(&d[8 * u]);
      }
      // ---- dV^T += dO^T P, dK^T += Q^T dS: 2 query steps x 4 d tiles each
      s16x4 lo[16], hi[16];
      // issue order i: operand (dO^T, Q^T) = i % 2, d tile = (i / 2) % 4, query step u = i / 8
      auto read_t = [&](auto ic) {
        constexpr int i = decltype(ic)::value, w = i % 2, mt = (i / 2) % 4, u = i / 8;
        constexpr int roff = 16 * (2 * qb + u) * ROWB;
        const uint32_t src = w ? qs : ds;
        lo[i] = ds_tr16<roff>(src + fo.lo[mt]);
        hi[i] = ds_tr16<roff>(src + fo.hi[mt]);
      };
      constexpr int WT = 7;   // transposed fragments in flight
      static_for<WT>([&](auto ic) { read_t(ic); });
      static_for<16>([&](auto ic) {
        constexpr int i = decltype(ic)::value, w = i % 2, mt = (i / 2) % 4, u = i / 8;
        constexpr int issued = (i + WT < 16) ? i + WT : 16;
        wait_lgkm<2 * (issued - i - 1)>();
        s16x8 v8 = {lo[i][0], lo[i][1], lo[i][2], lo[i][3], hi[i][0], hi[i][1], hi[i][2], hi[i][3]};
        bf16x8 f = *reinterpret_cast<bf16x8*>(&v8);
        pin(f);
        if constexpr (w == 0) dv[mt] = Mma<bf16>::run(f, pb[u], dv[mt]);
        else dk[mt] = Mma<bf16>::run(f, sb[u], dk[mt]);
        if constexpr (i + WT < 16) read_t(std::integral_constant<int, i + WT>{});
      });
    });
  };

  // the part's i-th tile lives in stage i & 1
  if (np > 0) load_tile(tb, 0);
  if (np > 1) {
    load_tile(tb + 1, 1);
    if (slice == 0) wait_vm<LPT + 2>();   // the first tile landed
    else wait_vm<LPT>();
  } else {
    wait_vm<0>();
  }
  lds_barrier();
  // hand the stage of trip `it` back: the next tile has landed, every wave
  // is done with this one
  auto trip_end = [&](int it) {
    wait_vm<0>();
    lds_barrier();
    if (it + 2 < np) load_tile(tb + it + 2, it & 1);
  };
  // The wave skips the part's tiles before the one holding its first key,
  // then takes the tiles where some query precedes some key (masked), then
  // the rest; one loop per kind keeps the accumulators in place.
  const int n_skip = min(max(wave_first - tb, 0), np);
  const int n_diag = min(max((k0 + 30) / BT + 1 - tb, n_skip), np);
  int it = 0;
  for (; it < n_skip; ++it) trip_end(it);
  for (; it < n_diag; ++it) {
    tile(tb + it, it & 1, std::true_type{});
    trip_end(it);
  }
  for (; it < np; ++it) {
    tile(tb + it, it & 1, std::false_type{});
    trip_end(it);
  }
  for (; it < nit; ++it) trip_end(it);

  // ---- sum the query parts of each key slice through LDS (ring memory is
  // free after the loop's last barrier; no tile load is in flight): part 1
  // parks its dK^T, dV^T, part 0 adds them to its own
  if constexpr (PARTS == 2) {
    float* park = reinterpret_cast<float*>(smem) + slice * (2 * D / 32 * 16) * 64;
    if (part == 1) {
#pragma unroll
      for (int mt = 0; mt < D / 32; ++mt)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          park[(mt * 16 + r) * 64 + lane] = dk[mt][r];
          park[((D / 32 + mt) * 16 + r) * 64 + lane] = dv[mt][r];
        }
    }
    __syncthreads();
    if (part == 1) return;
#pragma unroll
    for (int mt = 0; mt < D / 32; ++mt)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        dk[mt][r] += park[(mt * 16 + r) * 64 + lane];
        dv[mt][r] += park[((D / 32 + mt) * 16 + r) * 64 + lane];
      }
  }

  // ---- store: lane holds dK^T / dV^T [32 mt + acc_row(j, l)][key]
  if (key < s) {
    bf16* row = dqkv + ((int64_t)batch * s + key) * ld + head * D;
#pragma unroll
    for (int mt = 0; mt < D / 32; ++mt)
#pragma unroll
      for (int j4 = 0; j4 < 4; ++j4) {
        typedef __attribute__((ext_vector_type(4))) __bf16 bf16x4;
        bf16x4 wk, wv;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          wk[j] = (bf16)(dk[mt][4 * j4 + j] * scale);
          wv[j] = (bf16)dv[mt][4 * j4 + j];
        }
        const int c = 32 * mt + acc_row(4 * j4, lane);
        *reinterpret_cast<bf16x4*>(row + H + c) = wk;
        *reinterpret_cast<bf16x4*>(row + 2 * H + c) = wv;
      }
  }
}

// ---------------------------------------------------------------------------
// dQ
// ---------------------------------------------------------------------------
template <int QW, int PARTS>
__global__ __attribute__((amdgpu_flat_work_group_size(64 * QW * PARTS, 64 * QW * PARTS), amdgpu_waves_per_eu(1, 1)))
void attn_bwd_dq_v3_kernel(const bf16* __restrict__ qkv, const bf16* __restrict__ dout,
                           const float* __restrict__ lse, const float* __restrict__ dvec, bf16* __restrict__ dqkv,
                           int b, int s, int nh, float scale) {
  constexpr int STAGE = 2 * TILE;   // K, V
  constexpr int RING = 2 * STAGE;   // one key part's two stages
  constexpr int BQ = 32 * QW;       // queries per workgroup
  static_assert(PARTS == 1 || PARTS == 2, "key parts");
  __shared__ __attribute__((aligned(1024))) char smem[PARTS * RING];

  const int H = nh * D;
  const int64_t ld = 3 * (int64_t)H;
  const int nqb = (s + BQ - 1) / BQ;
  const int idx = blockIdx.x;
  const int head = idx % nh;
  const int batch = (idx / nh) % b;
  const int qb = nqb - 1 - idx / (nh * b);     // heaviest blocks first
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int g = lane >> 5;
  const int slice = wave % QW, part = wave / QW;
  const int q0 = qb * BQ + slice * 32;
  const int q = q0 + (lane & 31);

  const bf16* base = qkv + (int64_t)batch * s * ld;
  const int qc = min(q, s - 1);
  bf16x8 qf[D / 16], df[D / 16];
  {
    const bf16* qrow = base + (int64_t)qc * ld + head * D + 8 * g;
    const bf16* drow = dout + ((int64_t)batch * s + qc) * H + head * D + 8 * g;
#pragma unroll
    for (int ks = 0; ks < D / 16; ++ks) {
      qf[ks] = load_frag_settled(qrow + 16 * ks);
      df[ks] = load_frag_settled(drow + 16 * ks);
    }
  }
  const float lse2 = lse[((int64_t)batch * nh + head) * s + qc] * kLog2e;
  const float dq_dot = dvec[((int64_t)batch * nh + head) * s + qc];
  // key tiles of the workgroup, and this part's share of them
  const int last_q = min(qb * BQ + BQ - 1, s - 1);
  const int nt = last_q / BT + 1;
  const int nt0 = PARTS == 1 ? nt : (nt + 1) / 2;
  const int tb = part ? nt0 : 0;               // first tile of this part
  const int np = part ? nt - nt0 : nt0;        // tiles of this part
  const int nit = nt0;                         // loop trips (both parts, for the barriers)
  const int wave_last = min(q0 + 31, s - 1) / BT;

  TileSrcN<QW> ksrc, vsrc;
  ksrc.init(base + H + head * D, ld, s, slice, lane);
  vsrc.init(base + 2 * H + head * D, ld, s, slice, lane);
  char* const ring = smem + part * RING;
  auto load_tile = [&](int t, int st) {
    ksrc.load(t * BT, ring + st * STAGE);
    vsrc.load(t * BT, ring + st * STAGE + TILE);
  };
  constexpr int LPT = 2 * TileSrcN<QW>::IPW;   // load instructions per wave per tile
  FragOff fo;
  fo.init(lane);
  const uint32_t lds0 = lds_u32(ring);

  f32x16 dq[D / 32];
#pragma unroll
  for (int mt = 0; mt < D / 32; ++mt)
#pragma unroll
    for (int r = 0; r < 16; ++r) dq[mt][r] = 0.f;
  const float sl2 = scale * kLog2e;
  const int qthr = q - 4 * g;

  auto tile = [&](int t, int st, auto diag_c) {
    constexpr bool DIAG = decltype(diag_c)::value;
    const uint32_t ks_ = lds0 + st * STAGE, vs = ks_ + TILE;
    // ---- S^T = K Q^T and dP^T = V dO^T: 2 key blocks x 8 d-steps each
    f32x16 sacc[2], pacc[2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) sacc[kb][r] = pacc[kb][r] = 0.f;
    bf16x8 fr[32];
    auto read_f = [&](auto ic) {
      constexpr int i = decltype(ic)::value, w = i % 2, kb = (i / 2) % 2, ks = i / 4;
      fr[i] = ds_b128<kb * 32 * ROWB>((w ? vs : ks_) + fo.row[ks]);
    };
    constexpr int WF = 10;   // fragments in flight
    static_for<WF>([&](auto ic) { read_f(ic); });
    static_for<32>([&](auto ic) {
      constexpr int i = decltype(ic)::value, w = i % 2, kb = (i / 2) % 2, ks = i / 4;
      constexpr int issued = (i + WF < 32) ? i + WF : 32;
      wait_lgkm<issued - i - 1>();
      pin(fr[i]);
      if constexpr (w == 0) sacc[kb] = Mma<bf16>::run(fr[i], qf[ks], sacc[kb]);
      else pacc[kb] = Mma<bf16>::run(fr[i], df[ks], pacc[kb]);
      if constexpr (i + WF < 32) read_f(std::integral_constant<int, i + WF>{});
    });
    // ---- dS^T = P^T (dP^T - D), P^T = exp2(S^T s log2e - lse log2e)
    float d[2][16];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int j = 0; j < 16; ++j) {
        float pv = __builtin_amdgcn_exp2f(__builtin_fmaf(sacc[kb][j], sl2, -lse2));
        if constexpr (DIAG) {
          if (32 * kb + 8 * (j / 4) + (j % 4) > qthr - t * BT) pv = 0.f;
        }
        d[kb][j] = pv * (pacc[kb][j] - dq_dot);
      }
    bf16x8 sb[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) sb[u] = to_frag(&d[u / 2][8 * (u % 2)]);
    // ---- dQ^T += K^T dS^T: 4 key steps x 4 d tiles
    s16x4 lo[16], hi[16];
    auto read_t = [&](auto ic) {
      constexpr int i = decltype(ic)::value, mt = i % 4, u = i / 4;
      constexpr int roff = 16 * u * ROWB;
      lo[i] = ds_tr16<roff>(ks_ + fo.lo[mt]);
      hi[i] = ds_tr16<roff>(ks_ + fo.hi[mt]);
    };
    constexpr int WT = 7;   // transposed fragments in flight
    static_for<WT>([&](auto ic) { read_t(ic); });
    static_for<16>([&](auto ic) {
      constexpr int i = decltype(ic)::value, mt = i % 4, u = i / 4;
      constexpr int issued = (i + WT < 16) ? i + WT : 16;
      wait_lgkm<2 * (issued - i - 1)>();
      s16x8 v8 = {lo[i][0], lo[i][1], lo[i][2], lo[i][3], hi[i][0], hi[i][1], hi[i][2], hi[i][3]};
      bf16x8 f = *reinterpret_cast<bf16x8*>(&v8);
      pin(f);
      dq[mt] = Mma<bf16>::run(f, sb[u], dq[mt]);
      if constexpr (i + WT < 16) read_t(std::integral_constant<int, i + WT>{});
    });
  };

  if (np > 0) load_tile(tb, 0);
  if (np > 1) {
    load_tile(tb + 1, 1);
    wait_vm<LPT>();   // the first tile landed
  } else {
    wait_vm<0>();
  }
  lds_barrier();
  auto trip_end = [&](int it) {
    wait_vm<0>();
    lds_barrier();
    if (it + 2 < np) load_tile(tb + it + 2, it & 1);
  };
  // a prefix of the part's tiles (up to the one holding the wave's last
  // query), those crossing the diagonal last; one loop per kind
  const int n_comp = max(0, min(np, wave_last + 1 - tb));
  const int n_plain = max(0, min(n_comp, (q0 + 1) / BT - tb));   // tiles whose last key <= q0
  int it = 0;
  for (; it < n_plain; ++it) {
    tile(tb + it, it & 1, std::false_type{});
    trip_end(it);
  }
  for (; it < n_comp; ++it) {
    tile(tb + it, it & 1, std::true_type{});
    trip_end(it);
  }
  for (; it < nit; ++it) trip_end(it);

  // ---- sum the key parts of each query slice through LDS, part 0 first
  if constexpr (PARTS == 2) {
    float* park = reinterpret_cast<float*>(smem) + slice * (D / 32 * 16) * 64;
    if (part == 1) {
#pragma unroll
      for (int mt = 0; mt < D / 32; ++mt)
#pragma unroll
        for (int r = 0; r < 16; ++r) park[(mt * 16 + r) * 64 + lane] = dq[mt][r];
    }
    __syncthreads();
    if (part == 1) return;
#pragma unroll
    for (int mt = 0; mt < D / 32; ++mt)
#pragma unroll
      for (int r = 0; r < 16; ++r) dq[mt][r] += park[(mt * 16 + r) * 64 + lane];
  }

  if (q < s) {
    bf16* row = dqkv + ((int64_t)batch * s + q) * ld + head * D;
#pragma unroll
    for (int mt = 0; mt < D / 32; ++mt)
#pragma unroll
      for (int j4 = 0; j4 < 4; ++j4) {
        typedef __attribute__((ext_vector_type(4))) __bf16 bf16x4;
        bf16x4 w;
#pragma unroll
        for (int j = 0; j < 4; ++j) w[j] = (bf16)(dq[mt][4 * j4 + j] * scale);
        *reinterpret_cast<bf16x4*>(row + 32 * mt + acc_row(4 * j4, lane)) = w;
      }
  }
}

hipError_t attention_bwd_v3_launch(int b, int s, int nh, int d, const void* qkv, const float* lse, const void* dout,
                                   void* dqkv, const float* dvec, hipStream_t st) {
  if (d != D) return hipErrorInvalidValue;
  const float scale = 1.0f / sqrtf((float)d);
  const bf16* x = (const bf16*)qkv;
  const bf16* dy = (const bf16*)dout;
  bf16* dx = (bf16*)dqkv;
  // 128 rows per workgroup once the grid has more blocks than there are CUs,
  // else 64 rows with the other operand's tiles split in two parts inside the
  // workgroup (half the longest chain of tiles, at a higher cost per tile)
  const int n128 = (s + 127) / 128 * nh * b;
  const bool split = n128 <= 256;
  if (!split) {
    hipLaunchKernelGGL((attn_bwd_dkdv_v3_kernel<4, 1>), dim3(n128), dim3(256), 0, st, x, dy, lse, dvec, dx, b, s, nh,
                       scale);
  } else {
    hipLaunchKernelGGL((attn_bwd_dkdv_v3_kernel<2, 2>), dim3((s + 63) / 64 * nh * b), dim3(256), 0, st, x, dy, lse,
                       dvec, dx, b, s, nh, scale);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (!split) {
    hipLaunchKernelGGL((attn_bwd_dq_v3_kernel<4, 1>), dim3(n128), dim3(256), 0, st, x, dy, lse, dvec, dx, b, s, nh,
                       scale);
  } else {
    hipLaunchKernelGGL((attn_bwd_dq_v3_kernel<2, 2>), dim3((s + 63) / 64 * nh * b), dim3(256), 0, st, x, dy, lse,
                       dvec, dx, b, s, nh, scale);
  }
  return hipGetLastError();
}

}  // namespace tps
