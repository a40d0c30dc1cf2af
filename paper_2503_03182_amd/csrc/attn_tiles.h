// Shared pieces of the bf16, head-dim-128 attention kernels (attention_fwd.hip,
// attention_bwd.hip): the LDS layout of a 64-row tile of one head, its
// buffer-to-LDS loads, and the per-lane LDS offsets of the two fragment
// kinds the kernels read from such a tile.
//
// Tile layout: 64 rows (keys or queries) x 128 bf16 (256 bytes per row);
// 16-byte chunks XOR-swizzled per row with f(r) = 4 (r & 3) + ((r >> 2) & 3),
// a permutation of the 16 chunks over any 16 aligned rows whose top bits
// (f >> 1) also differ within each aligned group of 4 rows, so that
//   - ds_read_b128 by 16 lanes at 16 consecutive rows, one chunk, and
//   - ds_read_b64_tr_b16 by 16 lanes at 4 aligned rows x 2 chunks
// are both free of bank conflicts.
#pragma once
#include "gemm_lds.h"
#include "kernels.h"
#include "tps_device.h"

namespace tps {
namespace at {

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

constexpr int D = 128;            // head dim
constexpr int BT = 64;            // rows per tile
constexpr int ROWB = D * 2;       // bytes per LDS row
constexpr int TILE = BT * ROWB;   // 16 KB
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

__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc(const void* base, int64_t bytes) {
  const int n = bytes < 0x7FFFFFFF ? (int)bytes : 0x7FFFFFFF;
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, n, 0x00020000);
}

// Rows of one head's 128 columns in a [rows][ld] bf16 matrix, copied into
// LDS tiles by 16 one-KB buffer-to-LDS instructions shared by NW waves (16 /
// NW each).  Instruction i covers rows 4i .. 4i+3; lane l writes LDS slot
// (row 4i + l / 16, chunk l % 16), which holds logical chunk (l % 16) ^
// swz(row); swz depends on i only through i % 4.  The row offset is part of
// the per-lane (range-checked) offset: rows at or past `rows` read as zeros.
template <int NW>
struct TileSrcN {
  static constexpr int IPW = 16 / NW;   // instructions per wave per tile
  static_assert(IPW % 4 == 0, "instruction parity pattern");
  __amdgpu_buffer_rsrc_t r;
  uint32_t voff[4];
  int64_t ld;
  int w;   // this wave's index among the NW
  __device__ __forceinline__ void init(const bf16* base, int64_t ld_, int rows, int wave, int lane) {
    ld = ld_;
    w = wave;
    r = rsrc(base, ((int64_t)(rows - 1) * ld + D) * 2);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int row = 4 * j + (lane >> 4);   // i % 4 == j
      const int c = (lane & 15) ^ swz(row);
      voff[j] = (uint32_t)(((int64_t)(lane >> 4) * ld + c * 8) * 2);
    }
  }
  __device__ __forceinline__ void load(int row0, char* tile) const {
#pragma unroll
    for (int j = 0; j < IPW; ++j) {
      const int i = w * IPW + j;
      const uint32_t vo = voff[j % 4] + (uint32_t)(((int64_t)row0 + 4 * i) * ld * 2);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_void*)(tile + i * 1024), 16, vo, 0, 0, 0);
    }
  }
};

// 64 consecutive f32 of a per-row vector (lse, D), one buffer-to-LDS
// instruction (lanes 0-15 carry the 64 values; the other lanes' 16 bytes land
// in the 768 bytes after them).  Entries at or past `rows` read as zeros.
struct VecSrc {
  __amdgpu_buffer_rsrc_t r;
  __device__ __forceinline__ void init(const float* base, int rows) { r = rsrc(base, (int64_t)rows * 4); }
  __device__ __forceinline__ void load(int row0, char* dst, int lane) const {
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_void*)dst, 16, (uint32_t)(row0 * 4 + lane * 16), 0, 0, 0);
  }
};

// Per-lane LDS offsets inside a tile.
//  Row fragment (MFMA operand with d contiguous) for 32-row block rb and
//  d-step ks: row 32 rb + l % 32, chunk 2 ks + l / 32.  The swizzle repeats
//  every 16 rows, so rb enters as an immediate offset of rb * 32 * ROWB.
//  Transposed fragment (operand with the row index contiguous) for d tile mt
//  and 16-row step u: two transposing reads at rows 16 u + 4 g + (s >> 2) (lo)
//  and 8 further (hi), columns 32 mt + 16 (G & 1) + 4 (s & 3)
//  (G = l / 16, s = l % 16, g = l / 32); u enters as an immediate offset of
//  16 u * ROWB.  Lane l then holds column 32 mt + l % 32 at rows
//  {16 u + 4 g + i, 16 u + 8 + 4 g + i} (i < 4): for a 32x32x16 MFMA step this
//  is contraction index k = 8 g + i -> row 16 u + 8 (i / 4) + 4 g + i % 4, the
//  order in which a 32x32 accumulator holds rows (acc_row).
struct FragOff {
  uint32_t row[D / 16];
  uint32_t lo[D / 32], hi[D / 32];
  __device__ __forceinline__ void init(int lane) {
    const int g = lane >> 5, G = lane >> 4, sl = lane & 15;
#pragma unroll
    for (int ks = 0; ks < D / 16; ++ks) row[ks] = off(lane & 31, 2 * ks + g);
    const int r = 4 * (G >> 1) + (sl >> 2);
#pragma unroll
    for (int mt = 0; mt < D / 32; ++mt) {
      const int col = 32 * mt + 16 * (G & 1) + 4 * (sl & 3);
      lo[mt] = off(r, col >> 3) + (col & 7) * 2;
      hi[mt] = off(r + 8, col >> 3) + (col & 7) * 2;
    }
  }
};

// 8 bf16 of one lane, read from global memory and consumed before the tile
// loop (the wait for the load is placed here, so no wait inside the loop has
// to drain the tile loads issued after it).
__device__ __forceinline__ bf16x8 load_frag_settled(const bf16* p) {
  const u32x4 w = *reinterpret_cast<const u32x4*>(p);
  bf16x8 f = *reinterpret_cast<const bf16x8*>(&w);
  asm volatile("" ::"v"(f));
  return f;
}

// B operand of a 32x32x16 MFMA step from accumulator values v[0..7] (the
// rows acc_row(8 t + i) of a 32x32 accumulator), rounded to bf16.
__device__ __forceinline__ bf16x8 to_frag(const float* v) {
  bf16x8 f;
#pragma unroll
  for (int i = 0; i < 8; ++i) f[i] = (bf16)v[i];
  return f;
}

}  // namespace at
}  // namespace tps
