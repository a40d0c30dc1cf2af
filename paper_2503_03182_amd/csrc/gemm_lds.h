// Building blocks of the bf16 GEMMs on gfx950 (gemm_pipe.h):
//
// LDS tile layouts.  Operand tiles are stored in their natural memory layout:
//   K-contiguous operand (A of NT/NN, B of NT): [rows][BK] bf16;
//   M/N-contiguous operand (A of TN, B of NN/TN): [BK][rows] bf16.
// 16-byte chunks are XOR-swizzled within a row (the global address of each
// lane is permuted so the chunk lands at its swizzled slot), which keeps the
// fragment reads free of LDS bank conflicts:
//   K-contiguous: ds_read_b128 gives a lane 8 consecutive k of one row;
//   M/N-contiguous: two ds_read_b64_tr_b16 give a lane 8 consecutive k of one
//   column (the read transposes 4 x 4 blocks of 16-bit values across lanes).
//
// Fragment reads are issued as inline assembly with explicit waits (see
// below), and the epilogue parks accumulators in LDS to apply bias /
// residual / GeLU / GeLU' / f32 accumulation with 16-byte accesses.
#pragma once
#include <utility>

#include "kernels.h"
#include "tps_device.h"

namespace tps {

namespace gl {

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
__device__ __forceinline__ void pin(f32x4& v) { asm volatile("" : "+v"(v)); }
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

// Issue the LDS read(s) of fragment N alone of the wave's k-step KK.
template <int ROWS, bool KC, int BK, int NF, int KSW, int KK, int N>
__device__ __forceinline__ void read_frag(bf16x8 (&f)[NF], const FragAddr<ROWS, KC, BK, NF, KSW>& a,
                                          uint32_t stage) {
  static_assert(N < NF, "fragment index");
  if constexpr (KC) {
    constexpr int RS = BK * 64;   // bytes between row blocks of 32
    f[N] = ds_b128<N * RS>(stage + a.base[KK]);
  } else {
    constexpr int ROWB = ROWS * 2;
    typedef __attribute__((ext_vector_type(8))) short s16x8;
    const uint32_t p = stage + a.base[N];
    const s16x4 lo = ds_tr16<16 * KK * ROWB>(p);
    const s16x4 hi = ds_tr16<16 * KK * ROWB + 4 * ROWB>(p);
    s16x8 v = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
    f[N] = *reinterpret_cast<bf16x8*>(&v);
  }
}

}  // namespace gl

// Epilogue through LDS: per 32-row strip, each wave parks its accumulators
// ([32][WN] f32) in its own LDS region, reads them back row-contiguous and
// applies the epilogue on 8 consecutive columns with 16-byte accesses.  The
// global inputs of a strip (old f32 sums, residual, kept pre-activation) are
// loaded one strip ahead, before the stores of the current strip: the
// compiler cannot move loads of one pass above the (possibly aliasing)
// stores of the previous one, so issuing them in program order first keeps
// them all in flight together.
// LDS_BYTES: LDS the kernel owns (all of it is free when this runs).
template <int EPI, int P>
struct EpiIn {
  // per pass: f32 sums (ACC_F32) or one 16-byte bf16 vector (residual / aux)
  f32x4 c0[EPI == TPS_EPI_ACC_F32 ? P : 1], c1[EPI == TPS_EPI_ACC_F32 ? P : 1];
  Vec16<bf16> v[(EPI == TPS_EPI_BIAS_RESID || EPI == TPS_EPI_GELU_GRAD) ? P : 1];
};

template <int EPI, int BM, int BN, int WGM, int WGN, int TM, int TN, int LDS_BYTES>
__device__ __forceinline__ void gemm_epilogue(const GemmArgs& g, f32x16 (&acc)[TM][TN], char* smem, int m0, int n0,
                                              int wm, int wn, int lane, int wave) {
  constexpr int WM = BM / WGM, WN = BN / WGN;
  constexpr int LDE = WN + 8;   // f32 row pitch (keeps the parking writes conflict-free)
  static_assert(WGM * WGN * 32 * LDE * 4 <= LDS_BYTES, "epilogue staging must fit in LDS");
  float* strip = reinterpret_cast<float*>(smem) + wave * 32 * LDE;
  constexpr int CPR = WN / 8;             // 8-column chunks per row
  constexpr int RPP = 64 / CPR;           // rows per pass
  constexpr int P = 32 / RPP;             // passes per strip
  const int rl0 = lane / CPR, cl = (lane % CPR) * 8;
  const int col = n0 + wn * WN + cl;
  const int row0 = m0 + wm * WM + rl0;    // row of pass 0 of strip 0
  Vec16<bf16> bias;
  if constexpr (EPI == TPS_EPI_BIAS || EPI == TPS_EPI_BIAS_RESID || EPI == TPS_EPI_BIAS_GELU)
    bias = load16(static_cast<const bf16*>(g.bias) + col);

  auto load_strip = [&](int i, EpiIn<EPI, P>& in) {
#pragma unroll
    for (int q = 0; q < P; ++q) {
      const int64_t row = row0 + i * 32 + q * RPP;
      if constexpr (EPI == TPS_EPI_ACC_F32) {
        if (g.overwrite) {
          in.c0[q] = f32x4{0.f, 0.f, 0.f, 0.f};
          in.c1[q] = f32x4{0.f, 0.f, 0.f, 0.f};
        } else {
          const f32x4* c = reinterpret_cast<const f32x4*>(static_cast<const float*>(g.C) + row * g.ldc + col);
          in.c0[q] = c[0];
          in.c1[q] = c[1];
        }
      } else if constexpr (EPI == TPS_EPI_BIAS_RESID) {
        in.v[q] = load16(static_cast<const bf16*>(g.resid) + row * g.ldr + col);
      } else if constexpr (EPI == TPS_EPI_GELU_GRAD) {
        in.v[q] = load16(static_cast<const bf16*>(g.aux) + row * g.ldaux + col);
      }
    }
  };
  EpiIn<EPI, P> in[2];
  load_strip(0, in[0]);
#pragma unroll
  for (int i = 0; i < TM; ++i) {
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) strip[acc_row(r, lane) * LDE + j * 32 + (lane & 31)] = acc[i][j][r];
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    if (i + 1 < TM) load_strip(i + 1, in[(i + 1) & 1]);
    const EpiIn<EPI, P>& cur = in[i & 1];
#pragma unroll
    for (int q = 0; q < P; ++q) {
      const int rl = q * RPP + rl0;
      const f32x4 v0 = *reinterpret_cast<const f32x4*>(strip + rl * LDE + cl);
      const f32x4 v1 = *reinterpret_cast<const f32x4*>(strip + rl * LDE + cl + 4);
      const float v[8] = {v0[0], v0[1], v0[2], v0[3], v1[0], v1[1], v1[2], v1[3]};
      const int64_t row = row0 + i * 32 + q * RPP;
      if constexpr (EPI == TPS_EPI_ACC_F32) {
        f32x4* c = reinterpret_cast<f32x4*>(static_cast<float*>(g.C) + row * g.ldc + col);
        f32x4 c0 = cur.c0[q], c1 = cur.c1[q];
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          c0[t] += v[t];
          c1[t] += v[4 + t];
        }
        c[0] = c0;
        c[1] = c1;
      } else {
        float out[8];
        Vec16<bf16> aux;
        if constexpr (EPI == TPS_EPI_GELU_GRAD) aux = cur.v[q];
#pragma unroll
        for (int t = 0; t < 8; ++t) {
          if constexpr (EPI == TPS_EPI_STORE) {
            out[t] = v[t];
          } else if constexpr (EPI == TPS_EPI_BIAS) {
            out[t] = v[t] + to_f32(bias.get(t));
          } else if constexpr (EPI == TPS_EPI_BIAS_RESID) {
            out[t] = v[t] + to_f32(bias.get(t)) + to_f32(cur.v[q].get(t));
          } else if constexpr (EPI == TPS_EPI_BIAS_GELU) {
            const bf16 u = from_f32<bf16>(v[t] + to_f32(bias.get(t)));
            aux.set(t, u);
            out[t] = gelu_f(to_f32(u));
          } else {
            out[t] = v[t] * gelu_grad_f(to_f32(aux.get(t)));
          }
        }
        if constexpr (EPI == TPS_EPI_BIAS_GELU)
          if (g.aux) store16(static_cast<bf16*>(g.aux) + row * g.ldaux + col, aux);
        Vec16<bf16> o;
#pragma unroll
        for (int t = 0; t < 8; ++t) o.set(t, from_f32<bf16>(out[t]));
        store16(static_cast<bf16*>(g.C) + row * g.ldc + col, o);
      }
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  }
}

}  // namespace tps
