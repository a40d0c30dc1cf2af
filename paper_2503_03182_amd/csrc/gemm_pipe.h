// bf16 GEMM, tile-aligned shapes (M % BM, N % BN, K % BK == 0), with the
// K loop software-pipelined so that the MFMA pipe never waits on a barrier:
//
//  * operand tiles go global -> LDS with buffer loads that write LDS directly
//    (the K offset of a tile is a scalar, the per-lane offsets are fixed), in
//    the swizzled layouts of gemm_lds.h;
//  * an LDS ring of STAGES tiles: tiles kt+1 .. kt+STAGES-1 are in flight
//    while tile kt is multiplied;
//  * the one barrier per tile sits before the last k-step's MFMAs: after it
//    the stage of tile kt (whose fragments are all in registers by then) is
//    refilled with tile kt+STAGES and the first fragments of tile kt+1 are
//    read, both overlapping the last MFMAs of tile kt;
//  * inside a tile the fragments of k-step ks+1 are read between the MFMAs of
//    k-step ks (a few reads after each of its first MFMAs).
// Waves own a (BM/WGM) x (BN/WGN) block of 32x32x16 MFMA tiles; the K loop of
// every wave is sequential in steps of 16, so every output element sums its
// products in the same order whatever the tile shape.
#pragma once
#include "gemm_lds.h"

namespace tps {

namespace gp {

using gl::FragAddr;
using gl::lds_barrier;
using gl::lds_u32;
using gl::pin;
using gl::read_frags;
using gl::static_for;
using gl::wait_lgkm;

typedef __attribute__((address_space(3))) void lds_void;

template <int N>
__device__ __forceinline__ void wait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt");
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// Wait until at most `ahead` tiles of LPT loads each are outstanding
// (ahead <= MAXA; the count is an immediate, hence the dispatch).
template <int MAXA, int LPT>
__device__ __forceinline__ void wait_tiles(int ahead) {
  static_assert(MAXA * LPT < 64, "vmcnt range");
  if constexpr (MAXA >= 4) {
    if (ahead >= 4) { wait_vm<4 * LPT>(); return; }
  }
  if constexpr (MAXA >= 3) {
    if (ahead == 3) { wait_vm<3 * LPT>(); return; }
  }
  if constexpr (MAXA >= 2) {
    if (ahead == 2) { wait_vm<2 * LPT>(); return; }
  }
  if constexpr (MAXA >= 1) {
    if (ahead == 1) { wait_vm<LPT>(); return; }
  }
  wait_vm<0>();
}

// Per-lane part of the buffer offsets of one operand's tile loads.  The tile
// is moved in 1 KB wave instructions (lane l: 16 bytes at LDS +16 l); the
// instruction index i enters the global offset only through a uniform term
// and, where the swizzle depends on it, through its parity.
//   K-contiguous [ROWS][BK] from [rows][ld]: chunk p of row r comes from
//     column chunk p ^ swz(r); instruction i covers rows i*RPI .. +RPI.
//   M/N-contiguous [BK][ROWS] from [k][ld]: chunk p of k-row r comes from
//     chunk p ^ 4 (r & 3); instruction i covers k-rows i*RPI .. +RPI.
template <int ROWS, bool KC, int BK>
struct LoadPlan {
  static constexpr int CPR = KC ? BK / 8 : ROWS / 8;   // 16-byte chunks per stored row
  static constexpr int RPI = 64 / CPR;                  // stored rows per instruction
  static constexpr int INST = ROWS * BK * 2 / 1024;     // instructions per tile
  // does the swizzle of a lane depend on the instruction's parity?
  static constexpr bool PARITY = KC ? (BK == 64) : (ROWS == 256);
  uint32_t voff[2];
  uint32_t ustep;   // uniform byte offset between consecutive instructions
  uint32_t kstep;   // uniform byte offset between consecutive K tiles
  __device__ __forceinline__ void init(int64_t ld, int lane) {
    static_assert(CPR * RPI == 64, "instruction covers whole rows");
#pragma unroll
    for (int par = 0; par < 2; ++par) {
      const int r = par * RPI + lane / CPR, p = lane % CPR;
      int c;
      if constexpr (KC) c = (BK == 64) ? (p ^ ((r >> 1) & 7)) : (p ^ ((r >> 2) & 3));
      else c = p ^ ((r & 3) << 2);
      const int r0 = lane / CPR;   // row within the instruction
      voff[par] = (uint32_t)(((int64_t)r0 * ld + c * 8) * 2);
    }
    ustep = (uint32_t)((int64_t)RPI * ld * 2);
    kstep = KC ? (uint32_t)(BK * 2) : (uint32_t)((int64_t)BK * ld * 2);
  }
};

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint64_t bytes) {
  const int n = bytes >= 0xFFFFFFFFull ? (int)0xFFFFFFFF : (int)bytes;
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, n, 0x00020000);
}

}  // namespace gp

template <int LAYOUT, int BM, int BN, int WGM, int WGN, int BK, int STAGES, int EPI>
__global__ __attribute__((amdgpu_flat_work_group_size(64 * WGM * WGN, 64 * WGM * WGN),
                          amdgpu_waves_per_eu(WGM * WGN >= 8 ? 2 : 1, WGM * WGN >= 8 ? 2 : 1)))
void gemm_bf16_kernel(GemmArgs g) {
  using namespace gp;
  constexpr int NW = WGM * WGN, NT = 64 * NW;
  constexpr int WM = BM / WGM, WN = BN / WGN, TM = WM / 32, TN = WN / 32;
  constexpr int KS = BK / 16;
  constexpr bool TWO_AHEAD = NW == 4 && KS == 4;
  constexpr bool A_KC = (LAYOUT != TPS_GEMM_TN);
  constexpr bool B_KC = (LAYOUT == TPS_GEMM_NT);
  constexpr int A_BYTES = BM * BK * 2, B_BYTES = BN * BK * 2, STAGE = A_BYTES + B_BYTES;
  typedef LoadPlan<BM, A_KC, BK> PA;
  typedef LoadPlan<BN, B_KC, BK> PB;
  constexpr int A_IPW = PA::INST / NW, B_IPW = PB::INST / NW;   // load instructions per wave per tile
  constexpr int LPT = A_IPW + B_IPW;
  static_assert(PA::INST % NW == 0 && PB::INST % NW == 0, "tile loads split evenly over waves");
  static_assert((A_IPW % 2 == 0 || !PA::PARITY) && (B_IPW % 2 == 0 || !PB::PARITY), "parity per instruction");
  static_assert(KS >= 2 && STAGES >= 2 && STAGES <= 5 && (STAGES - 1) * LPT < 64, "pipeline shape");
  static_assert(STAGES * STAGE <= 160 * 1024, "LDS");
  __shared__ __attribute__((aligned(1024))) char smem[STAGES * STAGE];

  const int nblk = g.tiles_m * g.tiles_n;
  int pid = blockIdx.x;
  if ((nblk & 7) == 0) pid = (pid & 7) * (nblk >> 3) + (pid >> 3);
  constexpr int GROUP = 8;
  const int group = pid / (GROUP * g.tiles_n);
  const int first_m = group * GROUP;
  const int gm = min(GROUP, g.tiles_m - first_m);
  const int tile_m = first_m + (pid % (GROUP * g.tiles_n)) % gm;
  const int tile_n = (pid % (GROUP * g.tiles_n)) / gm;
  const int m0 = tile_m * BM, n0 = tile_n * BN;

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wm = wave / WGN, wn = wave % WGN;

  // buffer resources over the operand panels this tile reads
  const bf16* A = static_cast<const bf16*>(g.A);
  const bf16* B = static_cast<const bf16*>(g.B);
  const bf16* a_base = A_KC ? A + (int64_t)m0 * g.lda : A + m0;
  const bf16* b_base = B_KC ? B + (int64_t)n0 * g.ldb : B + n0;
  const uint64_t a_bytes = A_KC ? (uint64_t)BM * g.lda * 2 : ((uint64_t)(g.K - 1) * g.lda + BM) * 2;
  const uint64_t b_bytes = B_KC ? (uint64_t)BN * g.ldb * 2 : ((uint64_t)(g.K - 1) * g.ldb + BN) * 2;
  const __amdgpu_buffer_rsrc_t ra = make_rsrc(a_base, a_bytes);
  const __amdgpu_buffer_rsrc_t rb = make_rsrc(b_base, b_bytes);
  PA pa;
  PB pb;
  pa.init(g.lda, lane);
  pb.init(g.ldb, lane);
  char* const lds_gen = smem;

  // issue load instruction j (of this wave's share) of tile kt into stage st
  auto load_a = [&](int j, int kt, int st) {
    const int i = wave * A_IPW + j;
    const uint32_t voff = PA::PARITY ? pa.voff[j & 1] : pa.voff[0];
    const uint32_t soff = (uint32_t)kt * pa.kstep + (uint32_t)i * pa.ustep;
    __builtin_amdgcn_raw_ptr_buffer_load_lds(ra, (lds_void*)(lds_gen + st * STAGE + i * 1024), 16, voff, soff, 0, 0);
  };
  auto load_b = [&](int j, int kt, int st) {
    const int i = wave * B_IPW + j;
    const uint32_t voff = PB::PARITY ? pb.voff[j & 1] : pb.voff[0];
    const uint32_t soff = (uint32_t)kt * pb.kstep + (uint32_t)i * pb.ustep;
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rb, (lds_void*)(lds_gen + st * STAGE + A_BYTES + i * 1024), 16, voff,
                                             soff, 0, 0);
  };
  auto load_tile = [&](int kt, int st) {
#pragma unroll
    for (int j = 0; j < A_IPW; ++j) load_a(j, kt, st);
#pragma unroll
    for (int j = 0; j < B_IPW; ++j) load_b(j, kt, st);
  };

  f32x16 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  FragAddr<BM, A_KC, BK, TM, KS> fra;
  FragAddr<BN, B_KC, BK, TN, KS> frb;
  fra.init(wm * WM, 0, lane);
  frb.init(wn * WN, 0, lane);
  const uint32_t lds0 = lds_u32(smem);
  // the fragment buffers alternate per k-step, so the next tile's first
  // k-step reads into the buffer k-step 0 uses
  static_assert(KS % 2 == 0, "k-steps per tile must be even");

  const int nk = g.K / BK;
  // prologue: fill the ring
#pragma unroll
  for (int t = 0; t < STAGES; ++t)
    if (t < nk) load_tile(t, t);
  // tile 0 has landed once at most min(STAGES, nk) - 1 tiles of loads remain
  wait_tiles<STAGES - 1, LPT>(min(STAGES, nk) - 1);
  lds_barrier();

  constexpr int NFR = TM + TN, NM = TM * TN;
  constexpr int RPM = (NFR + NM / 2 - 1) / (NM / 2);   // fragment reads per MFMA
  int kt = 0;
  if constexpr (TWO_AHEAD) {
    // One wave per SIMD: the fragments of k-step kk + 2 are read during k-step
    // kk (one buffer per k-step of the tile), so a read has two k-steps of
    // MFMAs to land.  The tile barrier moves to k-step KS - 2, whose reads are
    // the first of tile kt + 1: there the wave waits until every fragment of
    // tile kt is in registers, so after the barrier the stage of tile kt is
    // refilled while the last two k-steps run from registers.
    constexpr int R = gl::frag_reads<A_KC, TM>() + gl::frag_reads<B_KC, TN>();   // LDS reads per k-step
    static_assert(R <= 15, "lgkmcnt range");
    bf16x8 fa[KS][TM], fb[KS][TN];
    read_frags<BM, A_KC, BK, TM, KS, 0>(fa[0], fra, lds0);
    read_frags<BN, B_KC, BK, TN, KS, 0>(fb[0], frb, lds0 + A_BYTES);
    read_frags<BM, A_KC, BK, TM, KS, 1>(fa[1], fra, lds0);
    read_frags<BN, B_KC, BK, TN, KS, 1>(fb[1], frb, lds0 + A_BYTES);
    auto k_tile2 = [&](int kt, auto refill_c) {
      constexpr bool REFILL = decltype(refill_c)::value;
      const int cur = kt % STAGES;
      const uint32_t as = lds0 + cur * STAGE;
      const uint32_t nst = lds0 + ((kt + 1) % STAGES) * STAGE;
      static_for<KS>([&](auto kc) {
        constexpr int kk = decltype(kc)::value;
        constexpr int NK = (kk + 2) % KS;     // k-step the reads are for
        constexpr bool NEXT = kk + 2 >= KS;   // ... of tile kt + 1
        constexpr bool BAR = kk + 2 == KS;
        if constexpr (BAR) {
          wait_lgkm<0>();
          if constexpr (REFILL) wait_vm<(STAGES - 2) * LPT>();
          else wait_tiles<STAGES - 2, LPT>(max(0, min(STAGES - 2, nk - 2 - kt)));
          lds_barrier();
        } else {
          wait_lgkm<R>();   // the reads of k-step kk + 1 may still be in flight
        }
#pragma unroll
        for (int i = 0; i < TM; ++i) pin(fa[kk][i]);
#pragma unroll
        for (int j = 0; j < TN; ++j) pin(fb[kk][j]);
        const uint32_t ra = NEXT ? nst : as;
        static_for<NM>([&](auto mc) {
          constexpr int m = decltype(mc)::value, i = m / TN, j = m % TN;
          acc[i][j] = Mma<bf16>::run(fa[kk][i], fb[kk][j], acc[i][j]);
          static_for<RPM>([&](auto rc) {
            constexpr int r = m * RPM + decltype(rc)::value;
            if constexpr (r < TM) gl::read_frag<BM, A_KC, BK, TM, KS, NK, r>(fa[NK], fra, ra);
            else if constexpr (r < NFR) gl::read_frag<BN, B_KC, BK, TN, KS, NK, r - TM>(fb[NK], frb, ra + A_BYTES);
          });
          if constexpr (BAR && REFILL) {
            if constexpr (m < A_IPW) load_a(m, kt + STAGES, cur);
            else if constexpr (m < LPT) load_b(m - A_IPW, kt + STAGES, cur);
          }
          __builtin_amdgcn_sched_barrier(0);
        });
        if constexpr (BAR && REFILL) {
          static_for<(LPT > NM ? LPT - NM : 0)>([&](auto lc) {
            constexpr int m = NM + decltype(lc)::value;
            if constexpr (m < A_IPW) load_a(m, kt + STAGES, cur);
            else load_b(m - A_IPW, kt + STAGES, cur);
          });
        }
        __builtin_amdgcn_sched_barrier(0);
      });
    };
    for (; kt < nk - STAGES; ++kt) k_tile2(kt, std::true_type{});
    for (; kt < nk; ++kt) k_tile2(kt, std::false_type{});
  } else {
  bf16x8 fa[2][TM], fb[2][TN];
  read_frags<BM, A_KC, BK, TM, KS, 0>(fa[0], fra, lds0);
  read_frags<BN, B_KC, BK, TN, KS, 0>(fb[0], frb, lds0 + A_BYTES);

  // One K tile; REFILL: the stage is refilled with tile kt+STAGES (every tile
  // but the last STAGES), which also fixes the number of tiles in flight.
  // The fragments of k-step kk+1 (of the next tile's first k-step in the
  // last one) are read between the MFMAs of k-step kk, all within its first
  // half, so LDS traffic spreads over the MFMA stream.
  auto k_tile = [&](int kt, auto refill_c) {
    constexpr bool REFILL = decltype(refill_c)::value;
    const int cur = kt % STAGES;
    const uint32_t as = lds0 + cur * STAGE;
    const uint32_t nst = lds0 + ((kt + 1) % STAGES) * STAGE;
    static_for<KS>([&](auto kc) {
      constexpr int kk = decltype(kc)::value, fc = kk & 1;
      constexpr bool LAST = kk + 1 == KS;
      constexpr int NK = LAST ? 0 : kk + 1;   // k-step the reads are for
      // the fragments of k-step kk were read during the previous k-step
      wait_lgkm<0>();
#pragma unroll
      for (int i = 0; i < TM; ++i) pin(fa[fc][i]);
#pragma unroll
      for (int j = 0; j < TN; ++j) pin(fb[fc][j]);
      if constexpr (LAST) {
        // tile kt+1 landed (all waves), tile kt's stage no longer read
        if constexpr (REFILL) wait_vm<(STAGES - 2) * LPT>();
        else wait_tiles<STAGES - 2, LPT>(max(0, min(STAGES - 2, nk - 2 - kt)));
        lds_barrier();
      }
      const uint32_t ra = LAST ? nst : as;
      static_for<NM>([&](auto mc) {
        constexpr int m = decltype(mc)::value, i = m / TN, j = m % TN;
        acc[i][j] = Mma<bf16>::run(fa[fc][i], fb[fc][j], acc[i][j]);
        static_for<RPM>([&](auto rc) {
          constexpr int r = m * RPM + decltype(rc)::value;
          if constexpr (r < TM) gl::read_frag<BM, A_KC, BK, TM, KS, NK, r>(fa[fc ^ 1], fra, ra);
          else if constexpr (r < NFR) gl::read_frag<BN, B_KC, BK, TN, KS, NK, r - TM>(fb[fc ^ 1], frb, ra + A_BYTES);
        });
        if constexpr (LAST && REFILL) {
          if constexpr (m < A_IPW) load_a(m, kt + STAGES, cur);
          else if constexpr (m < LPT) load_b(m - A_IPW, kt + STAGES, cur);
        }
        __builtin_amdgcn_sched_barrier(0);
      });
      if constexpr (LAST && REFILL) {
        static_for<(LPT > NM ? LPT - NM : 0)>([&](auto lc) {
          constexpr int m = NM + decltype(lc)::value;
          if constexpr (m < A_IPW) load_a(m, kt + STAGES, cur);
          else load_b(m - A_IPW, kt + STAGES, cur);
        });
      }
      __builtin_amdgcn_sched_barrier(0);
    });
  };
  for (; kt < nk - STAGES; ++kt) k_tile(kt, std::true_type{});
  for (; kt < nk; ++kt) k_tile(kt, std::false_type{});
  }
  wait_vm<0>();
  wait_lgkm<0>();
  __syncthreads();   // LDS is reused below

  gemm_epilogue<EPI, BM, BN, WGM, WGN, TM, TN, STAGES * STAGE>(g, acc, smem, m0, n0, wm, wn, lane, wave);
}

template <int LAYOUT, int BM, int BN, int EPI, bool LONG_K>
static hipError_t launch_pipe_cfg(GemmArgs g, hipStream_t stream) {
  constexpr V3Config c = v3_config(LAYOUT, BM == 256, LONG_K);
  g.tiles_m = g.M / BM;
  g.tiles_n = g.N / BN;
  hipLaunchKernelGGL((gemm_bf16_kernel<LAYOUT, BM, BN, c.wgm, c.wgn, c.bk, c.stages, EPI>), dim3(g.tiles_m * g.tiles_n),
                     dim3(64 * c.wgm * c.wgn), 0, stream, g);
  return hipGetLastError();
}

template <int LAYOUT, int BM, int BN, int EPI>
static hipError_t launch_pipe_epi(GemmArgs g, hipStream_t stream) {
  if constexpr (LAYOUT == TPS_GEMM_TN && BM == 256) {
    if (g.K >= TN_LONG_K) return launch_pipe_cfg<LAYOUT, BM, BN, EPI, true>(g, stream);
  }
  return launch_pipe_cfg<LAYOUT, BM, BN, EPI, false>(g, stream);
}

// Epilogues each layout uses in the stage (others take the generic path).
template <int LAYOUT, int BM, int BN>
static hipError_t launch_pipe(GemmArgs g, hipStream_t stream) {
  if constexpr (LAYOUT == TPS_GEMM_NT) {
    switch (g.epi) {
      case TPS_EPI_BIAS: return launch_pipe_epi<LAYOUT, BM, BN, TPS_EPI_BIAS>(g, stream);
      case TPS_EPI_BIAS_RESID: return launch_pipe_epi<LAYOUT, BM, BN, TPS_EPI_BIAS_RESID>(g, stream);
      case TPS_EPI_BIAS_GELU: return launch_pipe_epi<LAYOUT, BM, BN, TPS_EPI_BIAS_GELU>(g, stream);
      case TPS_EPI_GELU_GRAD: return launch_pipe_epi<LAYOUT, BM, BN, TPS_EPI_GELU_GRAD>(g, stream);
      default: return launch_pipe_epi<LAYOUT, BM, BN, TPS_EPI_STORE>(g, stream);
    }
  } else if constexpr (LAYOUT == TPS_GEMM_NN) {
    if (g.epi == TPS_EPI_GELU_GRAD) return launch_pipe_epi<LAYOUT, BM, BN, TPS_EPI_GELU_GRAD>(g, stream);
    if (g.epi == TPS_EPI_BIAS_RESID) return launch_pipe_epi<LAYOUT, BM, BN, TPS_EPI_BIAS_RESID>(g, stream);
    return launch_pipe_epi<LAYOUT, BM, BN, TPS_EPI_STORE>(g, stream);
  } else {
    if (g.epi == TPS_EPI_ACC_F32) return launch_pipe_epi<LAYOUT, BM, BN, TPS_EPI_ACC_F32>(g, stream);
    return launch_pipe_epi<LAYOUT, BM, BN, TPS_EPI_STORE>(g, stream);
  }
}

}  // namespace tps
