// Fused causal attention forward, bf16, head dim 128, on 32x32x16 MFMAs.
//
// Work split.  A workgroup of 4 waves owns 128 consecutive queries of one
// (batch, head); each wave owns 32 of them, so every K/V fragment it reads
// from LDS feeds 32 queries (LDS traffic per MFMA flop is half that of a
// 16-query wave).  Workgroups are launched heaviest first (last query block
// first), so the causal triangle's short blocks fill in behind the long ones.
//
// Per 64-key tile and wave (transposed formulation, queries along MFMA N):
//   S^T[key, q]  = K Q^T          16 MFMAs; K from LDS (ds_read_b128),
//                                 Q^T fragments held in registers;
//   online softmax over keys for each query: a lane holds one query and 16
//                                 keys of each 32-key block, its partner lane
//                                 (l ^ 32) the other 16;
//   O^T[d, q]   += V^T P^T        16 MFMAs; P^T straight from the S^T
//                                 accumulators, V^T from LDS through
//                                 transposing reads.  The contraction index k
//                                 of a 16-key step maps to key
//                                 8 (i / 4) + 4 (k / 8) + i % 4 (i = k % 8), the
//                                 order in which the S^T accumulators hold
//                                 keys; V rows are read in that order.
//
// Data movement.  K and V tiles (64 x 128 bf16 each) are copied global -> LDS
// by buffer loads that write LDS directly, into a two-stage ring; chunks of
// 16 bytes are XOR-swizzled per row (f(r) = 4 (r & 3) + ((r >> 2) & 3)) so
// that both the 16-row ds_read_b128 and the 4-row transposing reads are free
// of bank conflicts.  LDS reads are inline assembly with explicit lgkmcnt
// waits (the compiler would otherwise drain all tile loads before each LDS
// read); one barrier per tile hands the stage of tile t back for tile t+2.
//
// Numerics: scores are scaled into the log2 domain (scale * log2 e), the
// softmax uses exp2; lse is returned in natural log.  Every reduction runs in
// a fixed order, so results are bitwise reproducible.
#include "gemm_lds.h"
#include "kernels.h"
#include "tps_device.h"

namespace tps {

namespace af {

using gl::ds_b128;
using gl::ds_tr16;
using gl::lds_barrier;
using gl::lds_u32;
using gl::pin;
using gl::static_for;
using gl::wait_lgkm;

typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((ext_vector_type(4))) short s16x4;
typedef __attribute__((ext_vector_type(8))) short s16x8;

constexpr int D = 128;          // head dim
constexpr int BQ = 128;         // queries per workgroup
constexpr int BK = 64;          // keys per tile
constexpr int ROWB = D * 2;     // bytes per LDS row
constexpr int TILE = BK * ROWB; // one K or V tile (16 KB)
constexpr int STAGE = 2 * TILE; // K and V
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

__device__ __forceinline__ int swz(int r) { return ((r & 3) << 2) | ((r >> 2) & 3); }
// byte offset of 16-byte chunk c of row r in a tile
__device__ __forceinline__ int off(int r, int c) { return r * ROWB + ((c ^ swz(r)) << 4); }

template <int N>
__device__ __forceinline__ void wait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt");
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

}  // namespace af

__global__ __attribute__((amdgpu_flat_work_group_size(256, 256), amdgpu_waves_per_eu(2, 2)))
void attn_fwd_v3_kernel(const bf16* __restrict__ qkv, bf16* __restrict__ o, float* __restrict__ lse, int b, int s,
                        int nh, float scale) {
  using namespace af;
  __shared__ __attribute__((aligned(1024))) char smem[2 * STAGE];

  const int H = nh * D;
  const int64_t ld = 3 * (int64_t)H;
  const int nqb = (s + BQ - 1) / BQ;
  const int idx = blockIdx.x;
  const int head = idx % nh;
  const int batch = (idx / nh) % b;
  const int qb = nqb - 1 - idx / (nh * b);   // heaviest blocks first
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int q0 = qb * BQ + wave * 32;        // first query of this wave
  const int q = q0 + (lane & 31);            // this lane's query
  const int g = lane >> 5;                   // half of the 64 lanes

  const bf16* base = qkv + (int64_t)batch * s * ld;
  // tiles the workgroup streams, and the last one this wave needs
  const int last_q = min(qb * BQ + BQ, s) - 1;
  const int ntile = last_q / BK + 1;
  const int wave_last = min(q0 + 31, s - 1) / BK;

  // Q^T fragments (B operand): lane holds q's d = 16 ks + 8 g .. +8
  bf16x8 qf[D / 16];
  {
    const bf16* qrow = base + (int64_t)min(q, s - 1) * ld + head * D + 8 * g;
#pragma unroll
    for (int ks = 0; ks < D / 16; ++ks) {
      const u32x4 w = *reinterpret_cast<const u32x4*>(qrow + 16 * ks);
      qf[ks] = *reinterpret_cast<const bf16x8*>(&w);
    }
#pragma unroll
    for (int ks = 0; ks < D / 16; ++ks) asm volatile("" ::"v"(qf[ks]));   // wait for them here
  }

  // Tile loads: 16 one-KB instructions for K and 16 for V; wave w issues
  // instructions 4w .. 4w+3 of each.  Instruction i covers rows 4i .. 4i+3;
  // lane l writes LDS slot (row 4i + l / 16, chunk l % 16), which holds
  // logical chunk (l % 16) ^ swz(row); swz depends on i only through i % 4.
  // buffer ranges end at this sequence's last row: rows past s read as zeros
  const int64_t kbytes = ((int64_t)(s - 1) * ld + D) * 2;
  const int nrec = kbytes < 0x7FFFFFFF ? (int)kbytes : 0x7FFFFFFF;
  const __amdgpu_buffer_rsrc_t rk =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<bf16*>(base + H + head * D), (short)0, nrec, 0x00020000);
  const __amdgpu_buffer_rsrc_t rv =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<bf16*>(base + 2 * H + head * D), (short)0, nrec, 0x00020000);
  uint32_t voff[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int i = wave * 4 + j;
    const int r = 4 * i + (lane >> 4);
    const int c = (lane & 15) ^ swz(r);
    voff[j] = (uint32_t)(((int64_t)(lane >> 4) * ld + c * 8) * 2);
  }
  // The row offset goes into the per-lane offset, which the buffer range
  // check covers (rows at or past s then load zeros).
  auto load_tile = [&](int t, int st) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int i = wave * 4 + j;
      const uint32_t vo = voff[j] + (uint32_t)(((int64_t)t * BK + 4 * i) * ld * 2);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rk, (lds_void*)(smem + st * STAGE + i * 1024), 16, vo, 0, 0, 0);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rv, (lds_void*)(smem + st * STAGE + TILE + i * 1024), 16, vo, 0, 0, 0);
    }
  };

  // per-lane LDS offsets
  //  K fragment (key block kb, d-step ks): row 32 kb + l % 32, chunk 2 ks + g
  uint32_t koff[D / 16];
#pragma unroll
  for (int ks = 0; ks < D / 16; ++ks) koff[ks] = off(lane & 31, 2 * ks + g);
  //  V^T fragment (d tile mt, 16-key step u of the tile): two 4-row
  //  transposing reads at rows 16 u + 4 g + (s >> 2) (lo) and 8 further (hi),
  //  columns 32 mt + 16 (G & 1) + 4 (s & 3) (G = l / 16, s = l % 16).  The row
  //  swizzle repeats every 16 rows, so u enters as an immediate; lo and hi
  //  differ in it.
  uint32_t voffl[D / 32], voffh[D / 32];
  {
    const int G = lane >> 4, sl = lane & 15;
    const int r = 4 * (G >> 1) + (sl >> 2);
#pragma unroll
    for (int mt = 0; mt < D / 32; ++mt) {
      const int col = 32 * mt + 16 * (G & 1) + 4 * (sl & 3);
      voffl[mt] = off(r, col >> 3) + (col & 7) * 2;
      voffh[mt] = off(r + 8, col >> 3) + (col & 7) * 2;
    }
  }
  const uint32_t lds0 = lds_u32(smem);

  f32x16 oacc[D / 32];
#pragma unroll
  for (int mt = 0; mt < D / 32; ++mt)
#pragma unroll
    for (int r = 0; r < 16; ++r) oacc[mt][r] = 0.f;
  float m_run = -INFINITY, l_run = 0.f;
  const float sl2 = scale * kLog2e;

  load_tile(0, 0);
  if (ntile > 1) {
    load_tile(1, 1);
    wait_vm<8>();   // tile 0 landed (8 load instructions per wave per tile)
  } else {
    wait_vm<0>();
  }
  lds_barrier();

  // per-lane constant of the causal test: key 64 t + c > q  <=>  c > q - 4 g - 64 t,
  // c = 32 kb + 8 (j / 4) + j % 4 the key offset of accumulator j of block kb
  const int qthr = q - 4 * g;
  // one 64-key tile; DIAG: some key of the tile lies past some query of the wave
  auto tile = [&](int t, auto diag_c) {
    constexpr bool DIAG = decltype(diag_c)::value;
    const uint32_t ks_lds = lds0 + (t & 1) * STAGE, vs_lds = ks_lds + TILE;
    // ---- S^T = K Q^T: 2 key blocks x 8 d-steps, K fragments 8 ahead
    f32x16 sacc[2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) sacc[kb][r] = 0.f;
    bf16x8 kf[16];
    auto read_k = [&](auto ic) {
      constexpr int i = decltype(ic)::value, kb = i % 2, ks = i / 2;
      kf[i] = ds_b128<kb * 32 * ROWB>(ks_lds + koff[ks]);
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
      const int thr = qthr - t * BK;
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
      vlo[i] = ds_tr16<roff>(vs_lds + voffl[m2]);
      vhi[i] = ds_tr16<roff>(vs_lds + voffh[m2]);
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

  for (int t = 0; t < ntile; ++t) {
    if (t <= wave_last) {
      if ((t + 1) * BK - 1 > q0) tile(t, std::true_type{});
      else tile(t, std::false_type{});
    }
    // hand stage t back: tile t+1 (the only loads in flight) has landed and
    // every wave is done with tile t
    wait_vm<0>();
    lds_barrier();
    if (t + 2 < ntile) load_tile(t + 2, t & 1);
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

hipError_t attention_fwd_v3_launch(int b, int s, int nh, int d, const void* qkv, void* o, float* lse, hipStream_t st) {
  if (d != af::D) return hipErrorInvalidValue;
  const float scale = 1.0f / sqrtf((float)d);
  const int nqb = (s + af::BQ - 1) / af::BQ;
  hipLaunchKernelGGL(attn_fwd_v3_kernel, dim3(nqb * nh * b), dim3(256), 0, st, (const bf16*)qkv, (bf16*)o, lse, b, s,
                     nh, scale);
  return hipGetLastError();
}

}  // namespace tps
