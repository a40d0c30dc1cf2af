// bf16 GEMM main path for tile-aligned shapes (M % BM, N % BN, K % 64 == 0).
//
// Operand tiles are copied global -> LDS with direct-to-LDS loads (each lane's
// 16 bytes land at LDS base + 16 * lane), in their natural memory layout:
//   K-contiguous operand (A of NT/NN, B of NT): [rows][64] bf16, 128-byte rows;
//   M/N-contiguous operand (A of TN, B of NN/TN): [64][rows] bf16.
// 16-byte chunks are XOR-swizzled within a row (the global address of each
// lane is permuted so the chunk lands at its swizzled slot), which keeps the
// fragment reads free of LDS bank conflicts:
//   K-contiguous: ds_read_b128 gives a lane 8 consecutive k of one row;
//   M/N-contiguous: two ds_read_tr16_b64 give a lane 8 consecutive k of one
//   column (the read transposes 4 x 4 blocks of 16-bit values across lanes).
// STAGES LDS stages hold consecutive K tiles: STAGES-1 tiles are in flight
// while one is multiplied, with one barrier per tile.  Waves own a
// (BM/WGM) x (BN/WGN) block of 32x32x16 MFMA tiles; with KSPLIT = 2 a second
// group of waves takes the upper half of every K tile and the two partial
// sums are added in a fixed order at the end (two waves per SIMD on small
// grids).  Within each wave the K loop is sequential in steps of 16.
#pragma once
#include <utility>

#include "kernels.h"
#include "tps_device.h"

namespace tps {

namespace v2 {

typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((ext_vector_type(4))) short s16x4;

// Byte offset of chunk c (16 bytes) of row r in a K-contiguous tile with BK
// columns.  ds_read_b128 serves 16 lanes = 16 consecutive rows at one chunk
// per pass; the swizzle spreads them over all 64 banks:
//   BK = 64 (128-byte rows, odd rows in the other bank half): c ^ ((r >> 1) & 7);
//   BK = 32 (64-byte rows, four rows per 256 bytes): c ^ ((r >> 2) & 3).
template <int BK>
__device__ __forceinline__ int kc_off(int r, int c) {
  if constexpr (BK == 64) return r * 128 + ((c ^ ((r >> 1) & 7)) << 4);
  else return r * 64 + ((c ^ ((r >> 2) & 3)) << 4);
}
// Byte offset of chunk c of row r in an M/N-contiguous tile with ROWB-byte rows
// (ROWB >= 256).  A pass of ds_read_tr16_b64 serves 32 lanes reading 4 rows x
// 4 chunks; XOR-ing chunk bits 2-3 with the row puts the 16 chunks on 16
// different bank groups.
template <int ROWB>
__device__ __forceinline__ int mc_off(int r, int c) { return r * ROWB + ((c ^ ((r & 3) << 2)) << 4); }

template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt");
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// Issue the direct-to-LDS loads of one operand tile.  ROWS = tile extent along
// M or N.  KC: operand is K-contiguous (global [rows][ld], tile rows x 64);
// otherwise M/N-contiguous (global [k][ld], tile 64 x rows).
template <int ROWS, bool KC, int NTHREADS, int BK>
__device__ __forceinline__ void issue_tile(const bf16* g, int64_t ld, int row0, int k0, char* lds) {
  constexpr int TILE_BYTES = ROWS * BK * 2;
  constexpr int PER_WAVE = TILE_BYTES / 1024 / (NTHREADS / 64);   // 1 KB per wave instruction
  static_assert(TILE_BYTES % (1024 * (NTHREADS / 64)) == 0, "tile must split evenly over waves");
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
  for (int i = 0; i < PER_WAVE; ++i) {
    const int inst = wave * PER_WAVE + i;
    const int slot = inst * 64 + lane;       // 16-byte slot in the tile
    const bf16* src;
    if constexpr (KC) {
      constexpr int CPR = BK / 8;
      const int r = slot / CPR, p = slot % CPR;
      const int c = (BK == 64) ? (p ^ ((r >> 1) & 7)) : (p ^ ((r >> 2) & 3));
      src = g + (int64_t)(row0 + r) * ld + k0 + c * 8;
    } else {
      constexpr int CPR = ROWS / 8;           // chunks per row
      const int r = slot / CPR, p = slot % CPR;
      const int c = p ^ ((r & 3) << 2);
      src = g + (int64_t)(k0 + r) * ld + row0 + c * 8;
    }
    __builtin_amdgcn_global_load_lds((const void*)src, (lds_void*)(lds + inst * 1024), 16, 0, 0);
  }
}

// LDS fragment reads are issued as inline assembly.  The compiler orders
// every LDS read it can see after all outstanding direct-to-LDS loads
// (s_waitcnt vmcnt(0)), which would drain the load pipeline once per K tile;
// reads it cannot see are ordered by the explicit lgkmcnt / vmcnt waits and
// barriers below instead.
__device__ __forceinline__ uint32_t lds_u32(const void* p) {
  return (uint32_t)(uintptr_t)((const __attribute__((address_space(3))) char*)p);
}
template <int OFF>
__device__ __forceinline__ bf16x8 ds_b128(uint32_t a) {
  bf16x8 v;
  asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(v) : "v"(a), "i"(OFF));
  return v;
}
template <int OFF>
__device__ __forceinline__ s16x4 ds_tr16(uint32_t a) {
  s16x4 v;
  asm volatile("ds_read_b64_tr_b16 %0, %1 offset:%2" : "=v"(v) : "v"(a), "i"(OFF));
  return v;
}
// Wait until at most N LDS reads are outstanding (LDS reads complete in
// issue order; no scalar loads are in flight inside the K loop).
template <int N>
__device__ __forceinline__ void wait_lgkm() {
  static_assert(N >= 0 && N < 16, "lgkmcnt");
  asm volatile("s_waitcnt lgkmcnt(%0)" ::"n"(N) : "memory");
}
// The value is not consumed before this point (pins uses after a wait).
__device__ __forceinline__ void pin(bf16x8& v) { asm volatile("" : "+v"(v)); }
__device__ __forceinline__ void lds_barrier() { asm volatile("s_barrier" ::: "memory"); }

// Per-lane LDS byte offsets of the fragments a wave reads from one stage,
// for the KSW k-steps of 16 starting at k-step ks0 of the tile.
//   K-contiguous: fragment i (row block i) of k-step ks sits at
//     row (row_base + 32 i + lane % 32), chunk 2 ks + lane / 32; the row swizzle
//     repeats every 32 rows, so only the chunk term depends on ks:
//     off(i, ks) = base[ks] + 4096 i (BK = 64) or 2048 i (BK = 32).
//   M/N-contiguous: fragment j of k-step ks is two transposing reads at
//     k rows (16 ks + 8 (g / 2) + s / 4) and 4 further; the column swizzle
//     depends on k mod 4 only, so off(j, ks) = base[j] + 16 (ks - ks0) ROWB.
template <int ROWS, bool KC, int BK, int NF, int KSW>
struct FragAddr {
  uint32_t base[KC ? KSW : NF];
  __device__ __forceinline__ void init(int row_base, int ks0, int lane) {
    if constexpr (KC) {
      const int r = row_base + (lane & 31);
#pragma unroll
      for (int kk = 0; kk < KSW; ++kk) base[kk] = kc_off<BK>(r, (ks0 + kk) * 2 + (lane >> 5));
    } else {
      constexpr int ROWB = ROWS * 2;
      const int g = lane >> 4, s = lane & 15;
      const int k = 16 * ks0 + ((g >> 1) << 3) + (s >> 2);
#pragma unroll
      for (int j = 0; j < NF; ++j) {
        const int col = row_base + 32 * j + ((g & 1) << 4) + ((s & 3) << 2);
        base[j] = mc_off<ROWB>(k, col >> 3) + (col & 7) * 2;
      }
    }
  }
};

template <typename F, int... I>
__device__ __forceinline__ void static_for_impl(F& f, std::integer_sequence<int, I...>) {
  (f(std::integral_constant<int, I>{}), ...);
}
// f(integral_constant<int, i>) for i = 0 .. N-1, unrolled at compile time.
template <int N, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  static_for_impl(f, std::make_integer_sequence<int, N>{});
}

// LDS reads per fragment set (each transposed fragment takes two reads).
template <bool KC, int NF>
constexpr int frag_reads() { return KC ? NF : 2 * NF; }

// Issue the LDS reads of the NF fragments of the wave's k-step KK from the
// stage at LDS byte address `stage`.
template <int ROWS, bool KC, int BK, int NF, int KSW, int KK>
__device__ __forceinline__ void read_frags(bf16x8 (&f)[NF], const FragAddr<ROWS, KC, BK, NF, KSW>& a,
                                           uint32_t stage) {
  if constexpr (KC) {
    constexpr int RS = BK * 64;   // bytes between row blocks of 32
    const uint32_t p = stage + a.base[KK];
    if constexpr (NF > 0) f[0] = ds_b128<0>(p);
    if constexpr (NF > 1) f[1] = ds_b128<RS>(p);
    if constexpr (NF > 2) f[2] = ds_b128<2 * RS>(p);
    if constexpr (NF > 3) f[3] = ds_b128<3 * RS>(p);
    static_assert(NF <= 4, "fragments per k-step");
  } else {
    constexpr int ROWB = ROWS * 2;
    typedef __attribute__((ext_vector_type(8))) short s16x8;
#pragma unroll
    for (int j = 0; j < NF; ++j) {
      const uint32_t p = stage + a.base[j];
      const s16x4 lo = ds_tr16<16 * KK * ROWB>(p);
      const s16x4 hi = ds_tr16<16 * KK * ROWB + 4 * ROWB>(p);
      s16x8 v = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
      f[j] = *reinterpret_cast<bf16x8*>(&v);
    }
  }
}

}  // namespace v2

template <int LAYOUT, int BM, int BN, int WGM, int WGN, int KSPLIT, int BK, int STAGES, int EPI>
__global__ __attribute__((amdgpu_flat_work_group_size(64 * WGM * WGN * KSPLIT, 64 * WGM * WGN * KSPLIT),
                          amdgpu_waves_per_eu(WGM * WGN * KSPLIT >= 8 ? 2 : 1, WGM * WGN * KSPLIT >= 8 ? 2 : 1)))
void gemm_v2_kernel(GemmArgs g) {
  using namespace v2;
  constexpr int NT = 64 * WGM * WGN * KSPLIT;
  constexpr int WM = BM / WGM, WN = BN / WGN, TM = WM / 32, TN = WN / 32;
  constexpr int KS = BK / 16 / KSPLIT;   // k-steps of 16 per wave per tile
  constexpr bool A_KC = (LAYOUT != TPS_GEMM_TN);
  constexpr bool B_KC = (LAYOUT == TPS_GEMM_NT);
  constexpr int A_BYTES = BM * BK * 2, B_BYTES = BN * BK * 2, STAGE = A_BYTES + B_BYTES;
  constexpr int LOADS = (A_BYTES + B_BYTES) / 1024 / (NT / 64);   // per thread per tile
  static_assert(KS >= 1 && STAGES >= 2, "pipeline shape");
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

  const bf16* A = static_cast<const bf16*>(g.A);
  const bf16* B = static_cast<const bf16*>(g.B);
  const int lane = threadIdx.x & 63, wave_all = threadIdx.x >> 6;
  const int wk = wave_all / (WGM * WGN), wave = wave_all % (WGM * WGN);
  const int wm = wave / WGN, wn = wave % WGN;

  f32x16 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  const int nk = g.K / BK;
  FragAddr<BM, A_KC, BK, TM, KS> fra;
  FragAddr<BN, B_KC, BK, TN, KS> frb;
  fra.init(wm * WM, wk * KS, lane);
  frb.init(wn * WN, wk * KS, lane);
  const uint32_t lds0 = lds_u32(smem);
  // fragments of k-step kk+1 are read while the MFMAs of k-step kk run
  auto mma_tile = [&](uint32_t as) {
    constexpr int RA = frag_reads<A_KC, TM>(), RB = frag_reads<B_KC, TN>();
    static_assert(RA <= 15 && RB <= 15, "lgkmcnt range");
    const uint32_t bs = as + A_BYTES;
    bf16x8 fa[2][TM], fb[2][TN];
    read_frags<BM, A_KC, BK, TM, KS, 0>(fa[0], fra, as);
    read_frags<BN, B_KC, BK, TN, KS, 0>(fb[0], frb, bs);
    static_for<KS>([&](auto kc) {
      constexpr int kk = decltype(kc)::value, cur = kk & 1;
      if constexpr (kk + 1 < KS) {
        read_frags<BM, A_KC, BK, TM, KS, kk + 1>(fa[cur ^ 1], fra, as);
        if constexpr (RA + RB <= 15) {
          read_frags<BN, B_KC, BK, TN, KS, kk + 1>(fb[cur ^ 1], frb, bs);
          wait_lgkm<RA + RB>();
        } else {
          wait_lgkm<RA>();
          read_frags<BN, B_KC, BK, TN, KS, kk + 1>(fb[cur ^ 1], frb, bs);
        }
      } else {
        wait_lgkm<0>();
      }
#pragma unroll
      for (int i = 0; i < TM; ++i) pin(fa[cur][i]);
#pragma unroll
      for (int j = 0; j < TN; ++j) pin(fb[cur][j]);
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = Mma<bf16>::run(fa[cur][i], fb[cur][j], acc[i][j]);
      // keep the k-steps in program order (reads of kk+1 ahead of MFMAs of kk)
      __builtin_amdgcn_sched_barrier(0);
    });
  };
  if constexpr (STAGES == 2) {
    // tile k+1 in flight while tile k is multiplied; a second barrier keeps
    // the stage being refilled out of use
    issue_tile<BM, A_KC, NT, BK>(A, g.lda, m0, 0, smem);
    issue_tile<BN, B_KC, NT, BK>(B, g.ldb, n0, 0, smem + A_BYTES);
    for (int kt = 0; kt < nk; ++kt) {
      if (kt + 1 < nk) {
        char* nxt = smem + ((kt + 1) & 1) * STAGE;
        issue_tile<BM, A_KC, NT, BK>(A, g.lda, m0, (kt + 1) * BK, nxt);
        issue_tile<BN, B_KC, NT, BK>(B, g.ldb, n0, (kt + 1) * BK, nxt + A_BYTES);
        wait_vmcnt<LOADS>();
      } else {
        wait_vmcnt<0>();
      }
      lds_barrier();
      mma_tile(lds0 + (kt & 1) * STAGE);
      lds_barrier();
    }
  } else {
    // prologue: tiles 0 .. STAGES-2 in flight
#pragma unroll
    for (int t = 0; t < STAGES - 1; ++t) {
      if (t < nk) {
        issue_tile<BM, A_KC, NT, BK>(A, g.lda, m0, t * BK, smem + t * STAGE);
        issue_tile<BN, B_KC, NT, BK>(B, g.ldb, n0, t * BK, smem + t * STAGE + A_BYTES);
      }
    }
    for (int kt = 0; kt < nk; ++kt) {
      // tile kt has landed once at most (tiles in flight after it) loads remain
      const int ahead = min(STAGES - 2, nk - 1 - kt);
      if constexpr (STAGES == 4) {
        if (ahead >= 2) wait_vmcnt<2 * LOADS>();
        else if (ahead == 1) wait_vmcnt<LOADS>();
        else wait_vmcnt<0>();
      } else {
        if (ahead >= 1) wait_vmcnt<LOADS>();
        else wait_vmcnt<0>();
      }
      // every wave's share of tile kt is in LDS, and every wave has finished
      // reading the stage refilled below (tile kt - 1, read in iteration kt - 1)
      lds_barrier();
      if (kt + STAGES - 1 < nk) {
        char* nxt = smem + ((kt + STAGES - 1) % STAGES) * STAGE;
        issue_tile<BM, A_KC, NT, BK>(A, g.lda, m0, (kt + STAGES - 1) * BK, nxt);
        issue_tile<BN, B_KC, NT, BK>(B, g.ldb, n0, (kt + STAGES - 1) * BK, nxt + A_BYTES);
      }
      mma_tile(lds0 + (kt % STAGES) * STAGE);
    }
  }
  __syncthreads();   // LDS is reused below

  if constexpr (KSPLIT == 2) {
    // fixed-order combine: the lower-K group adds the upper-K group's sums
    float* park = reinterpret_cast<float*>(smem) + wave * (TM * TN * 16 * 64);
    static_assert(WGM * WGN * TM * TN * 16 * 64 * 4 <= STAGES * STAGE, "combine must fit in LDS");
    if (wk == 1) {
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
          for (int r = 0; r < 16; ++r) park[((i * TN + j) * 16 + r) * 64 + lane] = acc[i][j][r];
    }
    __syncthreads();
    if (wk == 0) {
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
          for (int r = 0; r < 16; ++r) acc[i][j][r] += park[((i * TN + j) * 16 + r) * 64 + lane];
    }
    __syncthreads();
    if (wk != 0) return;
  }

  // Epilogue through LDS: per 32-row strip, each wave parks its accumulators
  // ([32][WN] f32) in its own LDS region, reads them back row-contiguous and
  // applies the epilogue on 8 consecutive columns with 16-byte accesses.
  constexpr int LDE = WN + 8;   // f32 row pitch (keeps the parking writes conflict-free)
  static_assert(WGM * WGN * 32 * LDE * 4 <= STAGES * STAGE, "epilogue staging must fit in LDS");
  float* strip = reinterpret_cast<float*>(smem) + wave * 32 * LDE;
  constexpr int CPR = WN / 8;             // 8-column chunks per row
  constexpr int RPP = 64 / CPR;           // rows per pass
#pragma unroll
  for (int i = 0; i < TM; ++i) {
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) strip[acc_row(r, lane) * LDE + j * 32 + (lane & 31)] = acc[i][j][r];
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
#pragma unroll
    for (int q = 0; q < 32 / RPP; ++q) {
      const int rl = q * RPP + lane / CPR, cl = (lane % CPR) * 8;
      const f32x4 v0 = *reinterpret_cast<const f32x4*>(strip + rl * LDE + cl);
      const f32x4 v1 = *reinterpret_cast<const f32x4*>(strip + rl * LDE + cl + 4);
      const float v[8] = {v0[0], v0[1], v0[2], v0[3], v1[0], v1[1], v1[2], v1[3]};
      const int row = m0 + wm * WM + i * 32 + rl, col = n0 + wn * WN + cl;
      if constexpr (EPI == TPS_EPI_ACC_F32) {
        f32x4* c = reinterpret_cast<f32x4*>(static_cast<float*>(g.C) + (int64_t)row * g.ldc + col);
        f32x4 c0 = c[0], c1 = c[1];
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          c0[t] += v[t];
          c1[t] += v[4 + t];
        }
        c[0] = c0;
        c[1] = c1;
      } else {
        float out[8];
        Vec16<bf16> bias, res, aux;
        if constexpr (EPI == TPS_EPI_BIAS || EPI == TPS_EPI_BIAS_RESID || EPI == TPS_EPI_BIAS_GELU)
          bias = load16(static_cast<const bf16*>(g.bias) + col);
        if constexpr (EPI == TPS_EPI_BIAS_RESID)
          res = load16(static_cast<const bf16*>(g.resid) + (int64_t)row * g.ldr + col);
        if constexpr (EPI == TPS_EPI_GELU_GRAD)
          aux = load16(static_cast<const bf16*>(g.aux) + (int64_t)row * g.ldaux + col);
#pragma unroll
        for (int t = 0; t < 8; ++t) {
          if constexpr (EPI == TPS_EPI_STORE) {
            out[t] = v[t];
          } else if constexpr (EPI == TPS_EPI_BIAS) {
            out[t] = v[t] + to_f32(bias.get(t));
          } else if constexpr (EPI == TPS_EPI_BIAS_RESID) {
            out[t] = v[t] + to_f32(bias.get(t)) + to_f32(res.get(t));
          } else if constexpr (EPI == TPS_EPI_BIAS_GELU) {
            const bf16 u = from_f32<bf16>(v[t] + to_f32(bias.get(t)));
            aux.set(t, u);
            out[t] = gelu_f(to_f32(u));
          } else {
            out[t] = v[t] * gelu_grad_f(to_f32(aux.get(t)));
          }
        }
        if constexpr (EPI == TPS_EPI_BIAS_GELU)
          if (g.aux) store16(static_cast<bf16*>(g.aux) + (int64_t)row * g.ldaux + col, aux);
        Vec16<bf16> o;
#pragma unroll
        for (int t = 0; t < 8; ++t) o.set(t, from_f32<bf16>(out[t]));
        store16(static_cast<bf16*>(g.C) + (int64_t)row * g.ldc + col, o);
      }
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  }
}

template <int LAYOUT, int BM, int BN, int EPI>
static hipError_t launch_v2_epi(GemmArgs g, hipStream_t stream) {
  constexpr V2Config c = v2_config(LAYOUT, BM == 256);
  g.tiles_m = g.M / BM;
  g.tiles_n = g.N / BN;
  hipLaunchKernelGGL((gemm_v2_kernel<LAYOUT, BM, BN, c.wgm, c.wgn, c.ksplit, c.bk, c.stages, EPI>),
                     dim3(g.tiles_m * g.tiles_n), dim3(64 * c.wgm * c.wgn * c.ksplit), 0, stream, g);
  return hipGetLastError();
}

// Epilogues each layout uses in the stage (others fall back to the generic path).
template <int LAYOUT>
constexpr bool v2_has_epi(int epi) {
  return LAYOUT == TPS_GEMM_NT ? (epi == TPS_EPI_STORE || epi == TPS_EPI_BIAS || epi == TPS_EPI_BIAS_RESID ||
                                  epi == TPS_EPI_BIAS_GELU || epi == TPS_EPI_GELU_GRAD)
       : LAYOUT == TPS_GEMM_NN ? (epi == TPS_EPI_STORE || epi == TPS_EPI_GELU_GRAD)
                               : (epi == TPS_EPI_STORE || epi == TPS_EPI_ACC_F32);
}

template <int LAYOUT, int BM, int BN>
static hipError_t launch_v2(GemmArgs g, hipStream_t stream) {
  if constexpr (LAYOUT == TPS_GEMM_NT) {
    switch (g.epi) {
      case TPS_EPI_BIAS: return launch_v2_epi<LAYOUT, BM, BN, TPS_EPI_BIAS>(g, stream);
      case TPS_EPI_BIAS_RESID: return launch_v2_epi<LAYOUT, BM, BN, TPS_EPI_BIAS_RESID>(g, stream);
      case TPS_EPI_BIAS_GELU: return launch_v2_epi<LAYOUT, BM, BN, TPS_EPI_BIAS_GELU>(g, stream);
      case TPS_EPI_GELU_GRAD: return launch_v2_epi<LAYOUT, BM, BN, TPS_EPI_GELU_GRAD>(g, stream);
      default: return launch_v2_epi<LAYOUT, BM, BN, TPS_EPI_STORE>(g, stream);
    }
  } else if constexpr (LAYOUT == TPS_GEMM_NN) {
    if (g.epi == TPS_EPI_GELU_GRAD) return launch_v2_epi<LAYOUT, BM, BN, TPS_EPI_GELU_GRAD>(g, stream);
    return launch_v2_epi<LAYOUT, BM, BN, TPS_EPI_STORE>(g, stream);
  } else {
    if (g.epi == TPS_EPI_ACC_F32) return launch_v2_epi<LAYOUT, BM, BN, TPS_EPI_ACC_F32>(g, stream);
    return launch_v2_epi<LAYOUT, BM, BN, TPS_EPI_STORE>(g, stream);
  }
}

}  // namespace tps
