// GEMM family for the stage's linears on gfx950: C = op(A) op(B) on 32x32
// MFMA tiles, LDS double buffering and fused epilogues.
//
//   NT  C[M,N] = A[M,K] B[N,K]^T   forward linears y = x W^T (+bias, +residual,
//                                  +GeLU with the pre-activation kept)
//   NN  C[M,N] = A[M,K] B[K,N]     input gradients dy W (optionally * GeLU'(u))
//   TN  C[M,N] = A[K,M]^T B[K,N]   weight gradients dy^T x over K = tokens,
//                                  accumulated into f32 (+=)
//
// Both operands are staged in LDS K-contiguous ([rows][BK + pad]) so that
// every lane reads its MFMA fragment with one 16-byte LDS read.  Operands
// that are contiguous along M or N in memory are transposed on the way in:
// each thread loads a VEC x VEC block with VEC 16-byte loads and writes it
// back as VEC 16-byte LDS rows.  The K loop is sequential, so every output
// element sums its products in the same order whatever the tile shape:
// results depend only on (M, N, K) and the data.
#pragma once
#include <type_traits>
#include "gemm_pipe.h"
#include "kernels.h"
#include "tps_device.h"

namespace tps {


// Loader for an operand tile of ROWS (M or N) x BK, K-contiguous in memory.
template <typename T, int ROWS, int BK, int LDSK>
struct LoadKC {
  static constexpr int VEC = 16 / sizeof(T);
  static constexpr int CPR = BK / VEC;                 // 16-byte chunks per row
  static constexpr int NCH = (ROWS * CPR + 255) / 256; // chunks per thread
  Vec16<T> r[NCH];
  __device__ __forceinline__ void load(const T* base, int64_t ld, int row0, int rows, int k0, int K) {
    const int tid = threadIdx.x;
#pragma unroll
    for (int i = 0; i < NCH; ++i) {
      const int c = tid + i * 256;
      const int row = c / CPR, kc = (c % CPR) * VEC;
      const int gr = row0 + row, gk = k0 + kc;
      if (c < ROWS * CPR && gr < rows && gk < K)
        r[i] = load16(base + (int64_t)gr * ld + gk);
      else
        r[i] = zero16<T>();
    }
  }
  __device__ __forceinline__ void store(T* lds) const {
    const int tid = threadIdx.x;
#pragma unroll
    for (int i = 0; i < NCH; ++i) {
      const int c = tid + i * 256;
      if (c < ROWS * CPR) {
        const int row = c / CPR, kc = (c % CPR) * VEC;
        store16(lds + row * LDSK + kc, r[i]);
      }
    }
  }
};

// Loader for an operand tile stored [K][rows] (contiguous along M or N):
// transposed into the K-contiguous LDS layout through VEC x VEC blocks.
template <typename T, int ROWS, int BK, int LDSK>
struct LoadMC {
  static constexpr int VEC = 16 / sizeof(T);
  static constexpr int RB = ROWS / VEC, KB = BK / VEC;
  static constexpr int NBLK = (RB * KB + 255) / 256;
  Vec16<T> r[NBLK][VEC];
  __device__ __forceinline__ void load(const T* base, int64_t ld, int row0, int rows, int k0, int K) {
    const int tid = threadIdx.x;
#pragma unroll
    for (int i = 0; i < NBLK; ++i) {
      const int b = tid + i * 256;
      const int rb = b % RB, kb = b / RB;
      const int gr = row0 + rb * VEC;
#pragma unroll
      for (int t = 0; t < VEC; ++t) {
        const int gk = k0 + kb * VEC + t;
        if (b < RB * KB && gr < rows && gk < K)
          r[i][t] = load16(base + (int64_t)gk * ld + gr);
        else
          r[i][t] = zero16<T>();
      }
    }
  }
  __device__ __forceinline__ void store(T* lds) const {
    const int tid = threadIdx.x;
#pragma unroll
    for (int i = 0; i < NBLK; ++i) {
      const int b = tid + i * 256;
      if (b >= RB * KB) continue;
      const int rb = b % RB, kb = b / RB;
#pragma unroll
      for (int j = 0; j < VEC; ++j) {
        Vec16<T> w;
        transpose_row(r[i], j, w);
        store16(lds + (rb * VEC + j) * LDSK + kb * VEC, w);
      }
    }
  }
  // w[t] = rows[t][j]
  static __device__ __forceinline__ void transpose_row(const Vec16<T> (&rows)[VEC], int j, Vec16<T>& w) {
    if constexpr (sizeof(T) == 2) {
#pragma unroll
      for (int p = 0; p < 4; ++p) {
        const uint32_t lo = rows[2 * p].raw[j >> 1];
        const uint32_t hi = rows[2 * p + 1].raw[j >> 1];
        w.raw[p] = (j & 1) ? ((lo >> 16) | (hi & 0xFFFF0000u)) : ((lo & 0xFFFFu) | (hi << 16));
      }
    } else {
#pragma unroll
      for (int t = 0; t < VEC; ++t) w.set(t, rows[t].get(j));
    }
  }
};

template <typename T, int BM, int BN, int BK, int LAYOUT>
__global__ __attribute__((amdgpu_flat_work_group_size(256, 256), amdgpu_waves_per_eu(BM * BN >= 256 * 128 ? 1 : 2, 2)))
void gemm_kernel(GemmArgs g) {
  typedef Mma<T> MM;
  constexpr int KPL = MM::KPL, KSTEP = 2 * KPL;
  constexpr int PAD = 16 / sizeof(T);
  constexpr int LDSK = BK + PAD;
  constexpr int WM = BM / 2, WN = BN / 2, TM = WM / 32, TN = WN / 32;
  constexpr bool A_KC = (LAYOUT != TPS_GEMM_TN);
  constexpr bool B_KC = (LAYOUT == TPS_GEMM_NT);

  __shared__ __attribute__((aligned(16))) T smem[2 * (BM + BN) * LDSK];
  // buffer i: A tile at smem + i * (BM + BN) * LDSK, B tile right after it
  constexpr int BUF = (BM + BN) * LDSK;

  // tile order: XCD-aware when the grid divides evenly over the 8 XCDs
  // (workgroup i runs on XCD i % 8), then grouped rows for L2 reuse.
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

  const T* A = static_cast<const T*>(g.A);
  const T* B = static_cast<const T*>(g.B);

  typename std::conditional<A_KC, LoadKC<T, BM, BK, LDSK>, LoadMC<T, BM, BK, LDSK>>::type la;
  typename std::conditional<B_KC, LoadKC<T, BN, BK, LDSK>, LoadMC<T, BN, BK, LDSK>>::type lb;

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave >> 1, wn = wave & 1;

  f32x16 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  const int nk = (g.K + BK - 1) / BK;
  la.load(A, g.lda, m0, g.M, 0, g.K);
  lb.load(B, g.ldb, n0, g.N, 0, g.K);
  la.store(smem);
  lb.store(smem + BM * LDSK);
  __syncthreads();

  const int frag_row = lane & 31, frag_k = (lane >> 5) * KPL;
  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    if (kt + 1 < nk) {
      la.load(A, g.lda, m0, g.M, (kt + 1) * BK, g.K);
      lb.load(B, g.ldb, n0, g.N, (kt + 1) * BK, g.K);
    }
    const T* as = smem + cur * BUF + (wm * WM + frag_row) * LDSK + frag_k;
    const T* bs = smem + cur * BUF + BM * LDSK + (wn * WN + frag_row) * LDSK + frag_k;
#pragma unroll
    for (int ks = 0; ks < BK / KSTEP; ++ks) {
      typename MM::Frag fa[TM], fb[TN];
#pragma unroll
      for (int i = 0; i < TM; ++i)
        fa[i] = *reinterpret_cast<const typename MM::Frag*>(as + i * 32 * LDSK + ks * KSTEP);
#pragma unroll
      for (int j = 0; j < TN; ++j)
        fb[j] = *reinterpret_cast<const typename MM::Frag*>(bs + j * 32 * LDSK + ks * KSTEP);
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = MM::run(fa[i], fb[j], acc[i][j]);
    }
    if (kt + 1 < nk) {
      la.store(smem + (cur ^ 1) * BUF);
      lb.store(smem + (cur ^ 1) * BUF + BM * LDSK);
    }
    __syncthreads();
  }

  // epilogue: lane holds column n, 16 rows per 32x32 tile
  const int epi = g.epi;
#pragma unroll
  for (int j = 0; j < TN; ++j) {
    const int col = n0 + wn * WN + j * 32 + (lane & 31);
    if (col >= g.N) continue;
    float bias = 0.f;
    if (epi == TPS_EPI_BIAS || epi == TPS_EPI_BIAS_RESID || epi == TPS_EPI_BIAS_GELU)
      bias = to_f32(static_cast<const T*>(g.bias)[col]);
#pragma unroll
    for (int i = 0; i < TM; ++i) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = m0 + wm * WM + i * 32 + acc_row(r, lane);
        if (row >= g.M) continue;
        const float v = acc[i][j][r];
        if (epi == TPS_EPI_ACC_F32) {
          float* c = static_cast<float*>(g.C) + (int64_t)row * g.ldc + col;
          *c = (g.overwrite ? 0.f : *c) + v;
        } else {
          T* c = static_cast<T*>(g.C) + (int64_t)row * g.ldc + col;
          float out;
          if (epi == TPS_EPI_STORE) {
            out = v;
          } else if (epi == TPS_EPI_BIAS) {
            out = v + bias;
          } else if (epi == TPS_EPI_BIAS_RESID) {
            out = v + bias + to_f32(static_cast<const T*>(g.resid)[(int64_t)row * g.ldr + col]);
          } else if (epi == TPS_EPI_BIAS_GELU) {
            const T u = from_f32<T>(v + bias);
            if (g.aux) static_cast<T*>(g.aux)[(int64_t)row * g.ldaux + col] = u;
            out = gelu_f(to_f32(u));
          } else {  // TPS_EPI_GELU_GRAD
            const float u = to_f32(static_cast<const T*>(g.aux)[(int64_t)row * g.ldaux + col]);
            out = v * gelu_grad_f(u);
          }
          *c = from_f32<T>(out);
        }
      }
    }
  }
}

template <typename T, int BM, int BN, int BK, int LAYOUT>
static hipError_t launch_tile(GemmArgs g, hipStream_t stream) {
  g.tiles_m = (g.M + BM - 1) / BM;
  g.tiles_n = (g.N + BN - 1) / BN;
  const int nblk = g.tiles_m * g.tiles_n;
  hipLaunchKernelGGL((gemm_kernel<T, BM, BN, BK, LAYOUT>), dim3(nblk), dim3(256), 0, stream, g);
  return hipGetLastError();
}

template <int LAYOUT>
static hipError_t launch_layout(int dtype, GemmArgs g, hipStream_t stream) {
  const GemmTile t = gemm_select_tile(dtype, LAYOUT, g);
  if (t.aligned) {
    if (t.bm == 256) return launch_pipe<LAYOUT, 256, 256>(g, stream);
    return launch_pipe<LAYOUT, 128, 128>(g, stream);
  }
  if (dtype == TPS_BF16) {
    if (t.bm == 256) return launch_tile<bf16, 256, 128, 64, LAYOUT>(g, stream);
    return launch_tile<bf16, 128, 128, 64, LAYOUT>(g, stream);
  }
  return launch_tile<float, 128, 128, 32, LAYOUT>(g, stream);
}

}  // namespace tps
