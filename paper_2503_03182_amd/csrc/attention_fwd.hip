// Fused causal attention forward, bf16, head dim 128, on 32x32x16 MFMAs.
//
// Work split.  A workgroup of 2 QW waves owns 32 QW consecutive queries of one
// (batch, head) and splits both ways: wave w takes the 32 queries of slice
// w % QW against the key tiles of part w / QW (part 0: the first ceil(n/2) of
// the block's n key tiles, part 1: the rest, which hold the diagonal).  The
// causal triangle's longest chain of key tiles per wave is thus halved, which
// balances the grid when there are few (batch, head) pairs, and each K/V
// fragment a wave reads from LDS still feeds 32 queries.  At the end the two
// parts of each query slice are merged in a fixed order (part 0, then part 1)
// through LDS: m = max(m0, m1), O = O0 2^(m0-m) + O1 2^(m1-m), same for the
// row sums.  Workgroups are launched heaviest first.
//
// Per 64-key tile and wave (transposed formulation, queries along MFMA N):
//   S^T[key, q]  = K Q^T          16 MFMAs; K from LDS (ds_read_b128),
//                                 Q^T fragments held in registers;
//   online softmax over keys for each query: a lane holds one query and 16
//                                 keys of each 32-key block, its partner lane
//                                 (l ^ 32) the other 16;
//   O^T[d, q]   += V^T P^T        16 MFMAs; P^T straight from the S^T
//                                 accumulators, V^T from LDS through
//                                 transposing reads in the accumulators' key
//                                 order (attn_tiles.h).
//
// Data movement.  Each key part streams its K and V tiles (64 x 128 bf16 each)
// global -> LDS by buffer loads that write LDS directly, into its own
// two-stage ring; LDS reads are inline assembly with explicit lgkmcnt waits
// (the compiler would otherwise drain all tile loads before each LDS read);
// one barrier per tile hands the stage of tile t back for tile t+2.
//
// Numerics: scores are scaled into the log2 domain (scale * log2 e), the
// softmax uses exp2; lse is returned in natural log.  Causal masking runs only
// on tiles that cross the diagonal; O is rescaled only when some lane's
// running max grew (the multiplier is exactly 1 otherwise).  Every reduction
// runs in a fixed order, so results are bitwise reproducible.
#include "attn_tiles.h"

namespace tps {

using namespace at;

template <int QW, int PARTS>
__global__ __attribute__((amdgpu_flat_work_group_size(64 * QW * PARTS, 64 * QW * PARTS),
                          amdgpu_waves_per_eu(QW / 2, QW / 2)))
void attn_fwd_sk_kernel(const bf16* __restrict__ qkv, bf16* __restrict__ o, float* __restrict__ lse, int b, int s,
                        int nh, float scale, int nkv) {
  constexpr int BQ = 32 * QW;        // queries per workgroup
  constexpr int STAGE = 2 * TILE;    // K and V
  constexpr int RING = 2 * STAGE;    // one key part's two stages
  static_assert(PARTS == 1 || PARTS == 2, "key parts");
  __shared__ __attribute__((aligned(1024))) char smem[PARTS * RING];

  // qkv rows: q of nh heads | k, v of nkv heads; query head n reads
  // key/value head n / (nh / nkv) (nkv == nh: plain multi-head)
  const int H = nh * D, HK = nkv * D;
  const int64_t ld = (int64_t)H + 2 * HK;
  const int nqb = (s + BQ - 1) / BQ;
  const int idx = blockIdx.x;
  const int head = idx % nh;
  const int kvh = head / (nh / nkv);
  const int batch = (idx / nh) % b;
  const int qb = nqb - 1 - idx / (nh * b);   // heaviest blocks first
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int slice = wave % QW, part = wave / QW;
  const int q0 = qb * BQ + slice * 32;   // first query of this wave
  const int q = q0 + (lane & 31);            // this lane's query
  const int g = lane >> 5;

  const bf16* base = qkv + (int64_t)batch * s * ld;
  // key tiles of the block, and this part's share of them
  const int nt = (min(qb * BQ + BQ, s) - 1) / BT + 1;
  const int nt0 = PARTS == 1 ? nt : (nt + 1) / 2;
  const int tb = part ? nt0 : 0;             // first tile of this part
  const int np = part ? nt - nt0 : nt0;      // tiles of this part
  const int nit = nt0;                       // loop trips (both parts, for the barriers)
  const int wave_last = min(q0 + 31, s - 1) / BT;

  // Q^T fragments (B operand): lane holds q's d = 16 ks + 8 g .. +8
  bf16x8 qf[D / 16];
  {
    const bf16* qrow = base + (int64_t)min(q, s - 1) * ld + head * D + 8 * g;
#pragma unroll
    for (int ks = 0; ks < D / 16; ++ks) qf[ks] = load_frag_settled(qrow + 16 * ks);
  }

  TileSrcN<QW> ksrc, vsrc;
  ksrc.init(base + H + kvh * D, ld, s, slice, lane);
  vsrc.init(base + H + HK + kvh * D, ld, s, slice, lane);
  char* const ring = smem + part * RING;
  auto load_tile = [&](int t, int st) {
    ksrc.load(t * BT, ring + st * STAGE);
    vsrc.load(t * BT, ring + st * STAGE + TILE);
  };
  constexpr int LPT = 2 * TileSrcN<QW>::IPW;   // load instructions per wave per tile
  FragOff fo;
  fo.init(lane);
  const uint32_t ring0 = lds_u32(ring);

  f32x16 oacc[D / 32];
#pragma unroll
  for (int mt = 0; mt < D / 32; ++mt)
#pragma unroll
    for (int r = 0; r < 16; ++r) oacc[mt][r] = 0.f;
  float m_run = -INFINITY, l_run = 0.f;
  const float sl2 = scale * kLog2e;
  // causal test on a diagonal tile: key 64 t + c > q  <=>  c > q - 4 g - 64 t,
  // c = 32 kb + 8 (j / 4) + j % 4 the key offset of accumulator j of block kb
  const int qthr = q - 4 * g;
  // one 64-key tile; DIAG: some key of the tile lies past some query of the wave
  auto tile = [&](int t, int st, auto diag_c) {
    constexpr bool DIAG = decltype(diag_c)::value;
    const uint32_t ks_lds = ring0 + st * STAGE, vs_lds = ks_lds + TILE;
    // ---- S^T = K Q^T: 2 key blocks x 8 d-steps, K fragments 8 ahead
    f32x16 sacc[2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) sacc[kb][r] = 0.f;
    bf16x8 kf[16];
    auto read_k = [&](auto ic) {
      constexpr int i = decltype(ic)::value, kb = i % 2, ks = i / 2;
      kf[i] = ds_b128<kb * 32 * ROWB>(ks_lds + fo.row[ks]);
    };
    static_for<8>([&](auto ic) { read_k(ic); });
    static_for<16>([&](auto ic) {
      constexpr int i = decltype(ic)::value, kb = i % 2, ks = i / 2;
      constexpr int issued = (i + 8 < 16) ? i + 8 : 16;
      wait_lgkm<issued - i - 1>();
      pin(kf[i]);
      sacc[kb] = Mma<bf16>::run(kf[i], qf[ks], sacc[kb]);
      if constexpr (i + 8 < 16) read_k(std::integral_constant<int, i + 8>{});
    });

    // ---- online softmax on raw scores (the scale is positive, so the max
    // commutes with it; it enters the exponent's FMA)
    if constexpr (DIAG) {
      const int thr = qthr - t * BT;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int j = 0; j < 16; ++j)
          if (32 * kb + 8 * (j / 4) + (j % 4) > thr) sacc[kb][j] = -INFINITY;
    }
    float mx = sacc[0][0];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int j = 0; j < 16; ++j) mx = fmaxf(mx, sacc[kb][j]);
    mx = fmaxf(mx, __shfl_xor(mx, 32, kWave));
    const float m_new = fmaxf(m_run, mx * sl2);
    const float m_use = (m_new == -INFINITY) ? 0.f : m_new;
    // rescale only when some lane's running max grew (alpha is 1 otherwise)
    const bool grew = m_new > m_run;
    const float alpha = grew ? __builtin_amdgcn_exp2f(m_run - m_use) : 1.f;
    m_run = m_new;
    float ls = 0.f;
    float x[2][16];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int j = 0; j < 16; ++j) {
        x[kb][j] = __builtin_amdgcn_exp2f(__builtin_fmaf(sacc[kb][j], sl2, -m_use));
        ls += x[kb][j];
      }
    l_run = l_run * alpha + ls;
    if (__builtin_amdgcn_ballot_w64(grew) != 0) {
#pragma unroll
      for (int m2 = 0; m2 < D / 32; ++m2)
#pragma unroll
        for (int r = 0; r < 16; ++r) oacc[m2][r] *= alpha;
    }

    // ---- O^T += V^T P^T: 2 key blocks x 2 16-key steps x 4 d tiles
    bf16x8 pb[4];
#pragma unroll
    for (int u = 0; u < 4; ++u)
#pragma unroll
      for (int i = 0; i < 8; ++i) pb[u][i] = (bf16)x[u / 2][8 * (u % 2) + i];
    s16x4 vlo[16], vhi[16];
    auto read_v = [&](auto ic) {
      constexpr int i = decltype(ic)::value, u = i / 4, m2 = i % 4;   // u: 16-key step of the tile
      constexpr int roff = 16 * u * ROWB;
      vlo[i] = ds_tr16<roff>(vs_lds + fo.lo[m2]);
      vhi[i] = ds_tr16<roff>(vs_lds + fo.hi[m2]);
    };
    static_for<7>([&](auto ic) { read_v(ic); });
    static_for<16>([&](auto ic) {
      constexpr int i = decltype(ic)::value, u = i / 4, m2 = i % 4;
      constexpr int issued = (i + 7 < 16) ? i + 7 : 16;
      wait_lgkm<2 * (issued - i - 1)>();
      s16x8 w = {vlo[i][0], vlo[i][1], vlo[i][2], vlo[i][3], vhi[i][0], vhi[i][1], vhi[i][2], vhi[i][3]};
      bf16x8 vf = *reinterpret_cast<bf16x8*>(&w);
      pin(vf);
      oacc[m2] = Mma<bf16>::run(vf, pb[u], oacc[m2]);
      if constexpr (i + 7 < 16) read_v(std::integral_constant<int, i + 7>{});
    });
  };

  // prologue: the first two tiles of each part
  if (np > 0) load_tile(tb, 0);
  if (np > 1) {
    load_tile(tb + 1, 1);
    wait_vm<LPT>();   // the first tile landed
  } else {
    wait_vm<0>();
  }
  lds_barrier();
  // hand the stage of trip `it` back: the next tile (the only loads in
  // flight) has landed and every wave is done with this one
  auto trip_end = [&](int it) {
    wait_vm<0>();
    lds_barrier();
    if (it + 2 < np) load_tile(tb + it + 2, it & 1);
  };
  // The wave computes a prefix of the part's tiles (up to the one holding its
  // last query), the tiles that cross the diagonal last; one loop per kind
  // and a barrier-only loop for the remaining trips keep the accumulators in
  // place (a join of paths inside one loop makes the compiler copy them).
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

  // ---- merge the key parts of each query slice through LDS (ring memory is
  // free after the loop's last barrier): part 1 parks m, l and O^T
  if constexpr (PARTS == 2) {
    float* park = reinterpret_cast<float*>(smem) + slice * (D / 32 * 16 + 2) * 64;
    if (part == 1) {
#pragma unroll
      for (int m2 = 0; m2 < D / 32; ++m2)
#pragma unroll
        for (int r = 0; r < 16; ++r) park[(m2 * 16 + r) * 64 + lane] = oacc[m2][r];
      park[(D / 32 * 16) * 64 + lane] = m_run;
      park[(D / 32 * 16 + 1) * 64 + lane] = l_run;
    }
    __syncthreads();
    if (part == 1) return;
    {
      const float m1 = park[(D / 32 * 16) * 64 + lane], l1 = park[(D / 32 * 16 + 1) * 64 + lane];
      const float m = fmaxf(m_run, m1);   // part 0 always holds key 0 <= q: m is finite
      const float a0 = __builtin_amdgcn_exp2f(m_run - m), a1 = __builtin_amdgcn_exp2f(m1 - m);
#pragma unroll
      for (int m2 = 0; m2 < D / 32; ++m2)
#pragma unroll
        for (int r = 0; r < 16; ++r) oacc[m2][r] = oacc[m2][r] * a0 + park[(m2 * 16 + r) * 64 + lane] * a1;
      l_run = l_run * a0 + l1 * a1;
      m_run = m;
    }
  }

  // ---- normalise and store: lane holds O^T[32 mt + acc_row(j, l)][q]
  float l_tot = l_run + __shfl_xor(l_run, 32, kWave);
  if (q < s) {
    const float inv = 1.f / l_tot;
    bf16* orow = o + ((int64_t)batch * s + q) * H + head * D;
#pragma unroll
    for (int m2 = 0; m2 < D / 32; ++m2)
#pragma unroll
      for (int j4 = 0; j4 < 4; ++j4) {
        typedef __attribute__((ext_vector_type(4))) __bf16 bf16x4;
        bf16x4 w;
#pragma unroll
        for (int j = 0; j < 4; ++j) w[j] = (bf16)(oacc[m2][4 * j4 + j] * inv);
        *reinterpret_cast<bf16x4*>(orow + 32 * m2 + acc_row(4 * j4, lane)) = w;
      }
    if (lse != nullptr && g == 0) lse[((int64_t)batch * nh + head) * s + q] = m_run * kLn2 + logf(l_tot);
  }
}

// grid thresholds (blocks of 128 queries) of the three forward shapes
constexpr int kFwdNoSplit = 512, kFwdWide = 256;

const char* attention_fwd_v3_name(int b, int s, int nh) {
  const int n128 = (s + 127) / 128 * nh * b;
  return n128 >= kFwdNoSplit ? "tps::attn_fwd_sk_kernel<4, 1>"
         : n128 >= kFwdWide  ? "tps::attn_fwd_sk_kernel<4, 2>"
                             : "tps::attn_fwd_sk_kernel<2, 2>";
}

hipError_t attention_fwd_v3_launch(int b, int s, int nh, int nkv, int d, const void* qkv, void* o, float* lse,
                                   hipStream_t st) {
  if (d != D || nkv <= 0 || nh % nkv != 0) return hipErrorInvalidValue;
  const float scale = 1.0f / sqrtf((float)d);
  // 128 queries per workgroup: with two resident workgroups per CU when the
  // grid fills the chip twice over, else with the key tiles split in two
  // parts inside the workgroup; 64 queries in two parts below one workgroup
  // per CU
  const int n128 = (s + 127) / 128 * nh * b;
  const bf16* x = (const bf16*)qkv;
  if (n128 >= kFwdNoSplit) {
    hipLaunchKernelGGL((attn_fwd_sk_kernel<4, 1>), dim3(n128), dim3(256), 0, st, x, (bf16*)o, lse, b, s, nh, scale, nkv);
  } else if (n128 >= kFwdWide) {
    hipLaunchKernelGGL((attn_fwd_sk_kernel<4, 2>), dim3(n128), dim3(512), 0, st, x, (bf16*)o, lse, b, s, nh, scale, nkv);
  } else {
    hipLaunchKernelGGL((attn_fwd_sk_kernel<2, 2>), dim3((s + 63) / 64 * nh * b), dim3(256), 0, st, x, (bf16*)o, lse,
                       b, s, nh, scale, nkv);
  }
  return hipGetLastError();
}

}  // namespace tps
