// Fused causal attention backward, bf16, head dim 128, on 32x32x16 MFMAs.
//
// With P = softmax_causal(q k^T / sqrt d), D_i = sum_d dO_id O_id (computed by
// attn_bwd_dot_kernel) and lse the forward's log-sum-exp:
//   P_ij  = exp(s q_i.k_j - lse_i),   dP_ij = dO_i . v_j,
//   dS_ij = P_ij (dP_ij - D_i),
//   dV_j  = sum_i P_ij dO_i,  dK_j = s sum_i dS_ij q_i,  dQ_i = s sum_j dS_ij k_j,
// summed over the causal triangle j <= i.  Deterministic: every output element
// is produced by one wave in a fixed order (no atomics).  A block of 128 rows
// is owned by a 4-wave workgroup (one wave per SIMD, 32 rows per wave) that
// streams 64-row tiles of the other operands through a two-stage LDS ring.
// The dK/dV and dQ blocks run as two kernels, or fused: dK/dV of key block j
// followed by dQ of query block j in one workgroup, which gives every
// workgroup the same number of tiles.
//
// dK/dV (dkdv_block): K and V fragments of the wave's 32 keys in registers;
//   64-query tiles of Q, dO, lse and D stream through the ring.  With keys along the MFMA N
//   dimension (one key per lane):
//     S  = Q K^T, dP = dO V^T        (Q, dO rows from LDS)
//     dV^T += dO^T P, dK^T += Q^T dS (dO^T, Q^T through transposing reads, in
//                                     the accumulators' query order)
//   64 MFMAs per tile; one wave per SIMD (the dK/dV accumulators take AGPRs).
// dQ (dq_block): Q and dO fragments of the wave's 32 queries plus their lse
//   and D in registers; 64-key tiles of K and V stream through the ring.  With queries along N:
//     S^T = K Q^T, dP^T = V dO^T, dQ^T += K^T dS^T
//   48 MFMAs per tile; one wave per SIMD (Q, dO fragments and dQ
//   accumulators do not fit the register budget of two).
// Unfused workgroups are launched heaviest first.  Rows past the sequence end load as
// zeros: their Q and dO rows contribute nothing to dK/dV, and keys past the end
// lie beyond every query, so the causal mask removes them from dQ.
#include "attn_tiles.h"

namespace tps {

using namespace at;

// ---------------------------------------------------------------------------
// dK, dV
// ---------------------------------------------------------------------------
constexpr int kVecBytes = 1024;   // LDS bytes per per-row vector (64 f32 + landing pad)
// LDS of a dK/dV block: a ring of two stages of Q, dO, lse, D
constexpr int kDkdvLds = 2 * (2 * TILE + 2 * kVecBytes);
// LDS of a dQ block: a ring of two stages of K, V
constexpr int kDqLds = 2 * (2 * TILE);

// 16-byte LDS read of four f32 at byte address a + OFF.
template <int OFF>
__device__ __forceinline__ f32x4 ds_f32x4(uint32_t a) {
  f32x4 v;
  asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(v) : "v"(a), "i"(OFF));
  return v;
}

// Where dK/dV blocks write: with one key/value head per query head into
// dqkv's k and v blocks; with grouped heads (nkv < nh) into a workspace
// [T][2 nh d] of per-query-head gradients (dK of head n at column n d, dV at
// nh d + n d) that gqa_fold sums per key/value head.
struct KvOut {
  bf16* p;        // rows of dK | dV
  int64_t ld;     // row stride
  int dk0, dv0;   // column of query head 0's dK and dV
};

// dK, dV of key block kb (32 KW keys) of one (batch, query head); smem holds
// kDkdvLds bytes.  qkv rows: q of nh heads | k, v of nkv heads.
template <int KW>
__device__ __forceinline__ void dkdv_block(const bf16* __restrict__ qkv, const bf16* __restrict__ dout,
                                           const float* __restrict__ lse, const float* __restrict__ dvec,
                                           KvOut ko, int b, int s, int nh, int nkv, float scale, int kb,
                                           int head, int batch, char* smem) {
  constexpr int VEC = kVecBytes;
  constexpr int STAGE = 2 * TILE + 2 * VEC;    // Q, dO, lse, D
  constexpr int BKEY = 32 * KW;                // keys per workgroup

  const int H = nh * D, HK = nkv * D;
  const int64_t ld = (int64_t)H + 2 * HK;
  const int kvh = head / (nh / nkv);
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int g = lane >> 5;
  const int slice = wave;
  const int k0 = kb * BKEY + slice * 32;       // first key of this wave
  const int key = k0 + (lane & 31);

  const bf16* base = qkv + (int64_t)batch * s * ld;
  // K^T and V^T fragments (B operands): lane holds key's d = 16 ks + 8 g .. +8
  bf16x8 kf[D / 16], vf[D / 16];
  {
    const bf16* krow = base + (int64_t)min(key, s - 1) * ld + H + kvh * D + 8 * g;
#pragma unroll
    for (int ks = 0; ks < D / 16; ++ks) {
      kf[ks] = load_frag_settled(krow + 16 * ks);
      vf[ks] = load_frag_settled(krow + HK + 16 * ks);
    }
  }
  // query tiles from the one holding this workgroup's first key to the end
  const int tb = (kb * BKEY) / BT;
  const int np = (s + BT - 1) / BT - tb;
  const int wave_first = k0 / BT;              // earlier tiles have no query >= any key of the wave

  TileSrcN<KW> qsrc, dsrc;
  qsrc.init(base + head * D, ld, s, slice, lane);
  dsrc.init(dout + (int64_t)batch * s * H + head * D, H, s, slice, lane);
  VecSrc lsrc, vsrc;
  lsrc.init(lse + ((int64_t)batch * nh + head) * s, s);
  vsrc.init(dvec + ((int64_t)batch * nh + head) * s, s);
  char* const ring = smem;
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
  // Every LDS read below is a loop-invariant base register plus an immediate
  // offset (stage, operand, row block): the ring's address is folded into the
  // per-lane fragment offsets and the stage is a compile-time argument of the
  // tile, so no address arithmetic runs per read.
  FragOff fo;
  fo.init(lane);
  const uint32_t lds0 = lds_u32(ring);
#pragma unroll
  for (int ks = 0; ks < D / 16; ++ks) fo.row[ks] += lds0;
#pragma unroll
  for (int mt = 0; mt < D / 32; ++mt) {
    fo.lo[mt] += lds0;
    fo.hi[mt] += lds0;
  }
  const uint32_t vbase = lds0 + 2 * TILE + 16 * g;   // lse of row 4 g of the stage-0 tile

  f32x16 dk[D / 32], dv[D / 32];
#pragma unroll
  for (int mt = 0; mt < D / 32; ++mt)
#pragma unroll
    for (int r = 0; r < 16; ++r) dk[mt][r] = dv[mt][r] = 0.f;
  const float sl2 = scale * kLog2e;
  // causal test on a diagonal tile: query 64 t + c < key  <=>  c < key - 4 g - 64 t,
  // c = 32 qb + 8 (j / 4) + j % 4 the query offset of accumulator j of block qb
  const int kthr = key - 4 * g;

  // One 64-query tile, as two 32-query halves each taken through the chain
  // S, dP -> P, dS -> dV, dK.  The two chains are staggered so that the
  // elementwise work of one half runs while the MFMAs of the other issue
  // (independent registers: the vector ALU and the MFMA pipe overlap):
  //   S, dP of half 0
  //   S, dP of half 1          beside  P, dS of half 0
  //   dV, dK from half 0       beside  P, dS of half 1
  //   dV, dK from half 1
  // Only one half's row vectors (lse, D) are live at a time.
  // stage ST of the ring: Q at ST * STAGE, dO at + TILE, lse at + 2 TILE, D at + 2 TILE + VEC
  auto tile = [&](auto st_c, int t, auto diag_c) {
    constexpr int ST = decltype(st_c)::value;
    constexpr int QO = ST * STAGE, DO = QO + TILE;   // immediate offsets of Q and dO
    constexpr bool DIAG = decltype(diag_c)::value;
    // lse and D of the rows this lane holds in half qb: 32 qb + 8 (j / 4) + 4 g + (j % 4)
    f32x4 lv[4], dvv[4];
    auto read_vec = [&](auto qc) {
      constexpr int qb = decltype(qc)::value;
      static_for<4>([&](auto jc) {
        constexpr int j4 = decltype(jc)::value, o = ST * STAGE + (32 * qb + 8 * j4) * 4;
        lv[j4] = ds_f32x4<o>(vbase);
        dvv[j4] = ds_f32x4<o + VEC>(vbase);
      });
    };
    auto pin_vec = [&] {
#pragma unroll
      for (int j4 = 0; j4 < 4; ++j4) {
        pin(lv[j4]);
        pin(dvv[j4]);
      }
    };
    // P and dS of accumulator element j of half qb
    auto elem = [&](auto qc, auto jc, const f32x16& sacc, const f32x16& pacc, float* p, float* d) {
      constexpr int qb = decltype(qc)::value, j = decltype(jc)::value;
      float pv = __builtin_amdgcn_exp2f(__builtin_fmaf(sacc[j], sl2, -lv[j / 4][j % 4] * kLog2e));
      if constexpr (DIAG) {
        if (32 * qb + 8 * (j / 4) + (j % 4) < kthr - t * BT) pv = 0.f;
      }
      p[j] = pv;
      d[j] = pv * (pacc[j] - dvv[j / 4][j % 4]);
    };
    // S = Q K^T and dP = dO V^T of half qb: 8 d-steps each; first() runs
    // after the first wait (every LDS read issued before the phase has
    // landed), mid(i) after MFMA i
    auto sdp = [&](auto qc, f32x16& sacc, f32x16& pacc, auto&& first, auto&& mid) {
      constexpr int qb = decltype(qc)::value;
#pragma unroll
      for (int r = 0; r < 16; ++r) sacc[r] = pacc[r] = 0.f;
      bf16x8 fr[16];
      // issue order i: operand (Q, dO) = i % 2, d-step = i / 2
      auto read_f = [&](auto ic) {
        constexpr int i = decltype(ic)::value, w = i % 2, ks = i / 2;
        fr[i] = ds_b128<qb * 32 * ROWB + (w ? DO : QO)>(fo.row[ks]);
      };
      constexpr int WF = 8;   // fragments in flight
      static_for<WF>([&](auto ic) { read_f(ic); });
      static_for<16>([&](auto ic) {
        constexpr int i = decltype(ic)::value, w = i % 2, ks = i / 2;
        constexpr int issued = (i + WF < 16) ? i + WF : 16;
        wait_lgkm<issued - i - 1>();
        if constexpr (i == 0) first();
        pin(fr[i]);
        if constexpr (w == 0) sacc = Mma<bf16>::run(fr[i], kf[ks], sacc);
        else pacc = Mma<bf16>::run(fr[i], vf[ks], pacc);
        if constexpr (i + WF < 16) read_f(std::integral_constant<int, i + WF>{});
        mid(ic);
      });
    };
    // dV^T += dO^T P, dK^T += Q^T dS of half qb: 2 query steps x 4 d tiles
    // each; first() and mid(i) as for sdp
    auto dvdk = [&](auto qc, const bf16x8* pb, const bf16x8* sb, auto&& first, auto&& mid) {
      constexpr int qb = decltype(qc)::value;
      s16x4 lo[16], hi[16];
      // issue order i: operand (dO^T, Q^T) = i % 2, d tile = (i / 2) % 4, query step u = i / 8
      auto read_t = [&](auto ic) {
        constexpr int i = decltype(ic)::value, w = i % 2, mt = (i / 2) % 4, u = i / 8;
        constexpr int roff = 16 * (2 * qb + u) * ROWB + (w ? QO : DO);
        lo[i] = ds_tr16<roff>(fo.lo[mt]);
        hi[i] = ds_tr16<roff>(fo.hi[mt]);
      };
      constexpr int WT = 7;   // transposed fragments in flight
      static_for<WT>([&](auto ic) { read_t(ic); });
      static_for<16>([&](auto ic) {
        constexpr int i = decltype(ic)::value, w = i % 2, mt = (i / 2) % 4, u = i / 8;
        constexpr int issued = (i + WT < 16) ? i + WT : 16;
        wait_lgkm<2 * (issued - i - 1)>();
        if constexpr (i == 0) first();
        s16x8 v8 = {lo[i][0], lo[i][1], lo[i][2], lo[i][3], hi[i][0], hi[i][1], hi[i][2], hi[i][3]};
        bf16x8 f = *reinterpret_cast<bf16x8*>(&v8);
        pin(f);
        if constexpr (w == 0) dv[mt] = Mma<bf16>::run(f, pb[u], dv[mt]);
        else dk[mt] = Mma<bf16>::run(f, sb[u], dk[mt]);
        if constexpr (i + WT < 16) read_t(std::integral_constant<int, i + WT>{});
        mid(ic);
      });
    };
    auto none = [](auto...) {};
    using Q0 = std::integral_constant<int, 0>;
    using Q1 = std::integral_constant<int, 1>;

    f32x16 sacc0, pacc0, sacc1, pacc1;
    read_vec(Q0{});
    sdp(Q0{}, sacc0, pacc0, pin_vec, none);
    float p[16], d[16];
    bf16x8 pb0[2], sb0[2], pb1[2], sb1[2];
    sdp(Q1{}, sacc1, pacc1, none, [&](auto ic) {
      constexpr int i = decltype(ic)::value;
      elem(Q0{}, ic, sacc0, pacc0, p, d);
      if constexpr (i % 8 == 7) {
        pb0[i / 8] = to_frag(&p[i - 7]);
        sb0[i / 8] = to_frag(&d[i - 7]);
      }
    });
    read_vec(Q1{});
    dvdk(Q0{}, pb0, sb0, pin_vec, [&](auto ic) {
      constexpr int i = decltype(ic)::value;
      elem(Q1{}, ic, sacc1, pacc1, p, d);
      if constexpr (i % 8 == 7) {
        pb1[i / 8] = to_frag(&p[i - 7]);
        sb1[i / 8] = to_frag(&d[i - 7]);
      }
    });
    dvdk(Q1{}, pb1, sb1, none, none);
  };

  // the i-th tile lives in stage i & 1
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
  // The wave skips the tiles before the one holding its first key,
  // then takes the tiles where some query precedes some key (masked), then
  // the rest; one loop per kind keeps the accumulators in place.
  const int n_skip = min(max(wave_first - tb, 0), np);
  const int n_diag = min(max((k0 + 30) / BT + 1 - tb, n_skip), np);
  int it = 0;
  for (; it < n_skip; ++it) trip_end(it);
  // tiles it .. end - 1 of one kind, in pairs (stage 0, stage 1) so that the
  // loop body is straight-line code with both stages' offsets as immediates
  auto run = [&](int end, auto diag_c) {
    using S0 = std::integral_constant<int, 0>;
    using S1 = std::integral_constant<int, 1>;
    if ((it & 1) && it < end) {
      tile(S1{}, tb + it, diag_c);
      trip_end(it);
      ++it;
    }
    for (; it + 1 < end; it += 2) {
      tile(S0{}, tb + it, diag_c);
      trip_end(it);
      tile(S1{}, tb + it + 1, diag_c);
      trip_end(it + 1);
    }
    if (it < end) {
      tile(S0{}, tb + it, diag_c);
      trip_end(it);
      ++it;
    }
  };
  run(n_diag, std::true_type{});
  run(np, std::false_type{});

  // ---- store: lane holds dK^T / dV^T [32 mt + acc_row(j, l)][key]
  if (key < s) {
    bf16* row = ko.p + ((int64_t)batch * s + key) * ko.ld + head * D;
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
        *reinterpret_cast<bf16x4*>(row + ko.dk0 + c) = wk;
        *reinterpret_cast<bf16x4*>(row + ko.dv0 + c) = wv;
      }
  }
}

template <int KW>
__global__ __attribute__((amdgpu_flat_work_group_size(64 * KW, 64 * KW), amdgpu_waves_per_eu(1, 1)))
void attn_bwd_dkdv_v3_kernel(const bf16* __restrict__ qkv, const bf16* __restrict__ dout,
                             const float* __restrict__ lse, const float* __restrict__ dvec, KvOut ko,
                             int b, int s, int nh, int nkv, float scale) {
  __shared__ __attribute__((aligned(1024))) char smem[kDkdvLds];
  const int idx = blockIdx.x;
  // first key blocks carry the most queries
  dkdv_block<KW>(qkv, dout, lse, dvec, ko, b, s, nh, nkv, scale, idx / (nh * b), idx % nh, (idx / nh) % b, smem);
}

// ---------------------------------------------------------------------------
// dQ
// ---------------------------------------------------------------------------
// dQ of query block qb (32 QW queries) of one (batch, head); smem holds
// kDqLds bytes.
template <int QW>
__device__ __forceinline__ void dq_block(const bf16* __restrict__ qkv, const bf16* __restrict__ dout,
                                         const float* __restrict__ lse, const float* __restrict__ dvec,
                                         bf16* __restrict__ dqkv, int b, int s, int nh, int nkv, float scale, int qb,
                                         int head, int batch, char* smem) {
  constexpr int STAGE = 2 * TILE;   // K, V
  constexpr int BQ = 32 * QW;       // queries per workgroup

  const int H = nh * D, HK = nkv * D;
  const int64_t ld = (int64_t)H + 2 * HK;
  const int kvh = head / (nh / nkv);
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int g = lane >> 5;
  const int slice = wave;
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
  // key tiles up to the workgroup's last query
  const int last_q = min(qb * BQ + BQ - 1, s - 1);
  const int tb = 0;
  const int np = last_q / BT + 1;
  const int wave_last = min(q0 + 31, s - 1) / BT;

  TileSrcN<QW> ksrc, vsrc;
  ksrc.init(base + H + kvh * D, ld, s, slice, lane);
  vsrc.init(base + H + HK + kvh * D, ld, s, slice, lane);
  char* const ring = smem;
  auto load_tile = [&](int t, int st) {
    ksrc.load(t * BT, ring + st * STAGE);
    vsrc.load(t * BT, ring + st * STAGE + TILE);
  };
  constexpr int LPT = 2 * TileSrcN<QW>::IPW;   // load instructions per wave per tile
  // LDS reads as base register + immediate, as in dkdv_block
  FragOff fo;
  fo.init(lane);
  const uint32_t lds0 = lds_u32(ring);
#pragma unroll
  for (int ks = 0; ks < D / 16; ++ks) fo.row[ks] += lds0;
#pragma unroll
  for (int mt = 0; mt < D / 32; ++mt) {
    fo.lo[mt] += lds0;
    fo.hi[mt] += lds0;
  }

  f32x16 dq[D / 32];
#pragma unroll
  for (int mt = 0; mt < D / 32; ++mt)
#pragma unroll
    for (int r = 0; r < 16; ++r) dq[mt][r] = 0.f;
  const float sl2 = scale * kLog2e;
  const int qthr = q - 4 * g;

  // One 64-key tile as two 32-key blocks.  The elementwise work of block 0
  // runs while the S^T, dP^T MFMAs of block 1 issue, and that of block 1
  // while the first half of the dQ MFMAs (block 0's key steps) issue.
  // stage ST of the ring: K at ST * STAGE, V at + TILE
  auto tile = [&](auto st_c, int t, auto diag_c) {
    constexpr int ST = decltype(st_c)::value;
    constexpr int KO = ST * STAGE, VO = KO + TILE;   // immediate offsets of K and V
    constexpr bool DIAG = decltype(diag_c)::value;
    // dS^T of accumulator element j of key block kb:
    // dS^T = P^T (dP^T - D), P^T = exp2(S^T s log2e - lse log2e)
    auto elem = [&](auto kc, auto jc, const f32x16& sacc, const f32x16& pacc, float* d) {
      constexpr int kb = decltype(kc)::value, j = decltype(jc)::value;
      float pv = __builtin_amdgcn_exp2f(__builtin_fmaf(sacc[j], sl2, -lse2));
      if constexpr (DIAG) {
        if (32 * kb + 8 * (j / 4) + (j % 4) > qthr - t * BT) pv = 0.f;
      }
      d[j] = pv * (pacc[j] - dq_dot);
    };
    // S^T = K Q^T and dP^T = V dO^T of key block kb: 8 d-steps each; mid(i)
    // runs after MFMA i
    auto sdp = [&](auto kc, f32x16& sacc, f32x16& pacc, auto&& mid) {
      constexpr int kb = decltype(kc)::value;
#pragma unroll
      for (int r = 0; r < 16; ++r) sacc[r] = pacc[r] = 0.f;
      bf16x8 fr[16];
      // issue order i: operand (K, V) = i % 2, d-step = i / 2
      auto read_f = [&](auto ic) {
        constexpr int i = decltype(ic)::value, w = i % 2, ks = i / 2;
        fr[i] = ds_b128<kb * 32 * ROWB + (w ? VO : KO)>(fo.row[ks]);
      };
      constexpr int WF = 8;   // fragments in flight
      static_for<WF>([&](auto ic) { read_f(ic); });
      static_for<16>([&](auto ic) {
        constexpr int i = decltype(ic)::value, w = i % 2, ks = i / 2;
        constexpr int issued = (i + WF < 16) ? i + WF : 16;
        wait_lgkm<issued - i - 1>();
        pin(fr[i]);
        if constexpr (w == 0) sacc = Mma<bf16>::run(fr[i], qf[ks], sacc);
        else pacc = Mma<bf16>::run(fr[i], df[ks], pacc);
        if constexpr (i + WF < 16) read_f(std::integral_constant<int, i + WF>{});
        mid(ic);
      });
    };
    auto none = [](auto...) {};
    using K0 = std::integral_constant<int, 0>;
    using K1 = std::integral_constant<int, 1>;

    f32x16 sacc0, pacc0, sacc1, pacc1;
    sdp(K0{}, sacc0, pacc0, none);
    float d[16];
    bf16x8 sb[4];
    sdp(K1{}, sacc1, pacc1, [&](auto ic) {
      constexpr int i = decltype(ic)::value;
      elem(K0{}, ic, sacc0, pacc0, d);
      if constexpr (i % 8 == 7) sb[i / 8] = to_frag(&d[i - 7]);
    });
    // ---- dQ^T += K^T dS^T: 4 key steps x 4 d tiles; key steps 0, 1 come
    // from block 0, whose MFMAs carry block 1's elementwise work
    s16x4 lo[16], hi[16];
    auto read_t = [&](auto ic) {
      constexpr int i = decltype(ic)::value, mt = i % 4, u = i / 4;
      constexpr int roff = 16 * u * ROWB + KO;
      lo[i] = ds_tr16<roff>(fo.lo[mt]);
      hi[i] = ds_tr16<roff>(fo.hi[mt]);
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
      if constexpr (i < 8) {
        elem(K1{}, std::integral_constant<int, 2 * i>{}, sacc1, pacc1, d);
        elem(K1{}, std::integral_constant<int, 2 * i + 1>{}, sacc1, pacc1, d);
        if constexpr (i % 4 == 3) sb[2 + i / 4] = to_frag(&d[2 * i - 6]);
      }
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
  // a prefix of the tiles (up to the one holding the wave's last query),
  // those crossing the diagonal last; one loop per kind, then barrier-only
  // trips while the other waves finish
  const int n_comp = max(0, min(np, wave_last + 1 - tb));
  const int n_plain = max(0, min(n_comp, (q0 + 1) / BT - tb));   // tiles whose last key <= q0
  int it = 0;
  // tiles it .. end - 1 of one kind in (stage 0, stage 1) pairs, as for dK/dV
  auto run = [&](int end, auto diag_c) {
    using S0 = std::integral_constant<int, 0>;
    using S1 = std::integral_constant<int, 1>;
    if ((it & 1) && it < end) {
      tile(S1{}, tb + it, diag_c);
      trip_end(it);
      ++it;
    }
    for (; it + 1 < end; it += 2) {
      tile(S0{}, tb + it, diag_c);
      trip_end(it);
      tile(S1{}, tb + it + 1, diag_c);
      trip_end(it + 1);
    }
    if (it < end) {
      tile(S0{}, tb + it, diag_c);
      trip_end(it);
      ++it;
    }
  };
  run(n_plain, std::false_type{});
  run(n_comp, std::true_type{});
  for (; it < np; ++it) trip_end(it);

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

template <int QW>
__global__ __attribute__((amdgpu_flat_work_group_size(64 * QW, 64 * QW), amdgpu_waves_per_eu(1, 1)))
void attn_bwd_dq_v3_kernel(const bf16* __restrict__ qkv, const bf16* __restrict__ dout,
                           const float* __restrict__ lse, const float* __restrict__ dvec, bf16* __restrict__ dqkv,
                           int b, int s, int nh, int nkv, float scale) {
  __shared__ __attribute__((aligned(1024))) char smem[kDqLds];
  const int idx = blockIdx.x;
  const int nqb = (s + 32 * QW - 1) / (32 * QW);
  // heaviest blocks first
  dq_block<QW>(qkv, dout, lse, dvec, dqkv, b, s, nh, nkv, scale, nqb - 1 - idx / (nh * b), idx % nh,
               (idx / nh) % b, smem);
}

// dK, dV of key block j and then dQ of query block j (128 rows each): with n
// tiles of 64 rows in the sequence, the first streams the n - 2 j query tiles
// from the one holding key 128 j on, the second the 2 j + 2 key tiles up to
// its last query, so every workgroup streams n + 2 tiles whatever j (the
// causal triangle is balanced without splitting any block).
__global__ __attribute__((amdgpu_flat_work_group_size(256, 256), amdgpu_waves_per_eu(1, 1)))
void attn_bwd_fused_kernel(const bf16* __restrict__ qkv, const bf16* __restrict__ dout, const float* __restrict__ lse,
                           const float* __restrict__ dvec, bf16* __restrict__ dqkv, KvOut ko, int b, int s, int nh,
                           int nkv, float scale) {
  __shared__ __attribute__((aligned(1024))) char smem[kDkdvLds > kDqLds ? kDkdvLds : kDqLds];
  const int idx = blockIdx.x;
  const int j = idx / (nh * b), head = idx % nh, batch = (idx / nh) % b;
  dkdv_block<4>(qkv, dout, lse, dvec, ko, b, s, nh, nkv, scale, j, head, batch, smem);
  __syncthreads();   // the LDS ring is reused
  dq_block<4>(qkv, dout, lse, dvec, dqkv, b, s, nh, nkv, scale, j, head, batch, smem);
}

hipError_t attention_bwd_v3_launch(int b, int s, int nh, int nkv, int d, const void* qkv, const float* lse,
                                   const void* dout, void* dqkv, const float* dvec, void* kv_ws, hipStream_t st) {
  if (d != D || nkv <= 0 || nh % nkv != 0) return hipErrorInvalidValue;
  if (nkv != nh && kv_ws == nullptr) return hipErrorInvalidValue;
  const float scale = 1.0f / sqrtf((float)d);
  const bf16* x = (const bf16*)qkv;
  const bf16* dy = (const bf16*)dout;
  bf16* dx = (bf16*)dqkv;
  const int H = nh * D;
  const KvOut ko = nkv == nh ? KvOut{dx, 3 * (int64_t)H, H, 2 * H} : KvOut{(bf16*)kv_ws, 2 * (int64_t)H, 0, H};
  // Fused workgroups all take the same time, so they pack the CUs well when
  // there is at most one per CU or many per CU; in between, the two kernels
  // (heaviest blocks first) fill the last round better.
  const int n128 = (s + 127) / 128 * nh * b;
  if (n128 <= 256 || n128 >= 1024) {
    hipLaunchKernelGGL(attn_bwd_fused_kernel, dim3(n128), dim3(256), 0, st, x, dy, lse, dvec, dx, ko, b, s, nh, nkv,
                       scale);
  } else {
    hipLaunchKernelGGL((attn_bwd_dkdv_v3_kernel<4>), dim3(n128), dim3(256), 0, st, x, dy, lse, dvec, ko, b, s, nh,
                       nkv, scale);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((attn_bwd_dq_v3_kernel<4>), dim3(n128), dim3(256), 0, st, x, dy, lse, dvec, dx, b, s, nh, nkv,
                       scale);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || nkv == nh) return e;
  return gqa_fold_launch(kv_ws, dqkv, b * s, nh, nkv, d, st);
}

}  // namespace tps
