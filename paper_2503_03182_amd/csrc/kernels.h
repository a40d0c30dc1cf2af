// Internal launchers of the gfx950 kernels (host side).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/tpstage_ops.h"

namespace tps {

struct GemmArgs {
  int M, N, K;
  const void* A; int64_t lda;
  const void* B; int64_t ldb;
  void* C; int64_t ldc;
  const void* bias;
  const void* resid; int64_t ldr;
  void* aux; int64_t ldaux;
  int epi;
  int tiles_m, tiles_n;
  int overwrite;   // TPS_EPI_ACC_F32 only: C = A^T B instead of C += A^T B
};

// Tile shape of a GEMM launch.  Depends on the shape only (never on timing)
// and changes no result bit: every tile shape sums K in the same order.
struct GemmTile {
  int bm, bn, bk;
  int aligned;   // 1: tile-aligned bf16 path (gemm_pipe.h)
};
GemmTile gemm_select_tile(int dtype, int layout, const GemmArgs& g);

// Shape of the tile-aligned bf16 kernel per layout and tile size, chosen by
// measurement on MI355X: waves along M and N, K tile and LDS ring depth.
// 256 x 256 tiles run two waves per SIMD (128 x 64 per wave, K tiles of 64,
// a ring of 2), except the weight-gradient (TN) product with a contraction of
// TN_LONG_K or more: both of its operands are read with 8-byte transposing LDS
// reads, so it takes one wave per SIMD of 128 x 128 (one LDS read per MFMA
// instead of 1.5) with K tiles of 32 in a ring of 4 (3-7% faster at
// K = 32768, 1% at 4096; at 2048, where the product runs beside the input-
// gradient chain, the stage lost 0.5%).  128 x 128 tiles, used when 256 x 256
// would leave most CUs idle: one wave per SIMD (64 x 64), K tiles of 64, a
// ring of 4.
struct V3Config {
  int wgm, wgn, bk, stages;
};
constexpr int TN_LONG_K = 4096;
constexpr V3Config v3_config(int layout, bool big, bool long_k) {
  return !big ? V3Config{2, 2, 64, 4}
              : (layout == TPS_GEMM_TN && long_k) ? V3Config{2, 2, 32, 4} : V3Config{2, 4, 64, 2};
}
// Demangled name of the kernel instantiation a launch uses (as profilers
// print it), e.g. "tps::gemm_bf16_kernel<0, 256, 256, 2, 4, 64, 2, 1>".
const char* gemm_kernel_name(int dtype, int layout, const GemmArgs& g);

hipError_t gemm_launch_nt(int dtype, GemmArgs g, hipStream_t stream);
hipError_t gemm_launch_nn(int dtype, GemmArgs g, hipStream_t stream);
hipError_t gemm_launch_tn(int dtype, GemmArgs g, hipStream_t stream);


hipError_t gemm_launch(int dtype, int layout, int epi, int M, int N, int K, const void* A,
                       int64_t lda, const void* B, int64_t ldb, void* C, int64_t ldc,
                       const void* bias, const void* resid, int64_t ldr, void* aux, int64_t ldaux,
                       hipStream_t stream, int overwrite = 0);

// qkv rows: q of nh heads | k, v of nkv heads (nkv == nh: plain multi-head;
// nkv < nh, grouped query heads, bf16 with head dim 128 only)
hipError_t attention_fwd_launch(int dtype, int b, int s, int nh, int nkv, int d, const void* qkv, void* o,
                                float* lse, hipStream_t st);
// dvec: [b, nh, s] f32 scratch; kv_ws: [b s, 2 nh d] scratch of the
// per-query-head dK, dV when nkv < nh (else unused, may be null)
hipError_t attention_bwd_launch(int dtype, int b, int s, int nh, int nkv, int d, const void* qkv, const void* o,
                                const float* lse, const void* dout, void* dqkv, float* dvec, void* kv_ws,
                                hipStream_t st);

// bf16 kernels on 16x16x32 MFMAs with paired causal blocks (attention_v2.hip)
hipError_t attention_fwd_v2_launch(int b, int s, int nh, int d, const void* qkv, void* o, float* lse,
                                   hipStream_t st);
// bf16, head dim 128: 32 queries per wave on 32x32x16 MFMAs, key tiles split
// in two parts per workgroup on small grids (attention_fwd.hip); the name of
// the kernel instance a shape launches
hipError_t attention_fwd_v3_launch(int b, int s, int nh, int nkv, int d, const void* qkv, void* o, float* lse,
                                   hipStream_t st);
const char* attention_fwd_v3_name(int b, int s, int nh);
// bf16, head dim 128: dK/dV by 32-key waves, dQ by 32-query waves (attention_bwd.hip)
hipError_t attention_bwd_v3_launch(int b, int s, int nh, int nkv, int d, const void* qkv, const float* lse,
                                   const void* dout, void* dqkv, const float* dvec, void* kv_ws, hipStream_t st);
hipError_t attention_bwd_v2_launch(int b, int s, int nh, int d, const void* qkv, const float* lse, const void* dout,
                                   void* dqkv, const float* dvec, hipStream_t st);

hipError_t layernorm_fwd_launch(int dtype, int rows, int cols, const void* x, const void* gamma,
                                const void* beta, float eps, void* out, float* mean, float* rstd,
                                hipStream_t st);
// dx = resid + LN^T(dout); when dgamma/dbeta are set, partial column sums go
// to ws ([2 * cols * parts] f32) and are added to dgamma/dbeta in fixed order.
hipError_t layernorm_bwd_launch(int dtype, int rows, int cols, const void* dout, const void* x,
                                const float* mean, const float* rstd, const void* gamma,
                                const void* resid, void* dx, float* dgamma, float* dbeta,
                                float* ws, hipStream_t st);
// out[c] += sum_r x[r, c]  (two passes through ws, fixed order)
hipError_t colsum_launch(int dtype, int rows, int cols, const void* x, int64_t ldx, float* out,
                         float* ws, hipStream_t st);
uint64_t colsum_ws_bytes(int64_t rows, int64_t cols);
// Column sums accumulated over calls: pass 1 of colsum_launch adding each
// row segment's sums into part[segment * seg_stride + c] (colsum_segments(rows)
// segments), and the LayerNorm backward with its dbeta / dgamma sums added the
// same way (dbeta at part_dbeta, dgamma k_stride floats after it).  The
// finalize call sums the segments of every column of a partial block (ranges
// of columns each owned by an f32 vector inside `grads`), adds the sums there
// and clears the partials.
struct ColMap {
  int n;              // ranges (<= 8)
  int c0[9];          // range r covers columns c0[r] .. c0[r+1]
  int64_t goff[8];    // float offset of range r's vector in grads
};
hipError_t colsum_acc_launch(int dtype, int rows, int cols, const void* x, int64_t ldx, float* part,
                             int64_t seg_stride, hipStream_t st);
hipError_t layernorm_bwd_acc_launch(int dtype, int rows, int cols, const void* dout, const void* x,
                                    const float* mean, const float* rstd, const void* gamma, const void* resid,
                                    void* dx, float* part_dbeta, int64_t k_stride, int64_t seg_stride,
                                    hipStream_t st);
// grads (+)= the sum of the segments' partials (overwrite: =), partials cleared
hipError_t colsum_finalize_launch(const ColMap& m, float* part, int segs, int64_t seg_stride, float* grads,
                                  hipStream_t st, int overwrite = 0);
hipError_t gelu_launch(int dtype, int64_t n, const void* u, void* g, hipStream_t st);
hipError_t fill_zero_launch(void* p, uint64_t bytes, hipStream_t st);
// RMSNorm (no centring, no shift): out = x * rstd * gamma, rstd per row
hipError_t rmsnorm_fwd_launch(int dtype, int rows, int cols, const void* x, const void* gamma, float eps, void* out,
                              float* rstd, hipStream_t st);
// dx = resid + RMSNorm^T(dout); dgamma (optional, added to) via ws as in
// layernorm_bwd_launch
hipError_t rmsnorm_bwd_launch(int dtype, int rows, int cols, const void* dout, const void* x, const float* rstd,
                              const void* gamma, const void* resid, void* dx, float* dgamma, float* ws,
                              hipStream_t st);
// same, with the per-segment dgamma sums added into a partial block
hipError_t rmsnorm_bwd_acc_launch(int dtype, int rows, int cols, const void* dout, const void* x, const float* rstd,
                                  const void* gamma, const void* resid, void* dx, float* part_dgamma,
                                  int64_t seg_stride, hipStream_t st);
// LLAMA-style element-wise kernels (llama.hip), bf16
// table [2][s][d/2] f32: cos, then sin, of pos * base^(-2i/d)
hipError_t rope_table_launch(int s, int d, float base, float* table, hipStream_t st);
// in place: columns [0, n_rot d) of each of rows rows (position row % s),
// pairs (i, i + d/2) of every head turned by +angle (inverse: -angle)
hipError_t rope_launch(void* x, int64_t ld, int rows, int s, int n_rot, int d, const float* table, int inverse,
                       hipStream_t st);
// g [rows, f] = SiLU(u[:, :f]) * u[:, f:] for u [rows, 2f]
hipError_t swiglu_launch(int rows, int f, const void* u, void* g, hipStream_t st);
// du [rows, 2f] from dg [rows, f] and u [rows, 2f]
hipError_t swiglu_bwd_launch(int rows, int f, const void* dg, const void* u, void* du, hipStream_t st);
// dqkv's k and v blocks = per key/value head sums of ws [rows, 2 nh d]
hipError_t gqa_fold_launch(const void* ws, void* dqkv, int rows, int nh, int nkv, int d, hipStream_t st);
// every byte of p[0, bytes) set to value
hipError_t fill_bytes_launch(void* p, uint64_t bytes, uint8_t value, hipStream_t st);
// out (bf16) [rows][cols] = bf16(decode_e4m3(q[r][c]) * scale[r]); cols % 8 == 0,
// q 8-byte and out 16-byte aligned
// One AdamW step of n contiguous parameters on the device (f32 master w and
// moments m, v updated in place from the f32 gradient g; out receives w in the
// storage dtype, round to nearest even): the host update's f32 operations in
// its order, so both give the same bits.  c: b1, b2, eps, lr_c, inv_bc2_sqrt,
// wd_c as in AdamwCoef (planner.h).
hipError_t adamw_launch(int dtype, int64_t n, float* w, float* m, float* v, const float* g, void* out,
                        const float c[6], hipStream_t st);

hipError_t dequant_fp8_rows_launch(const void* q, const float* scale, int64_t rows, int64_t cols, void* out,
                                   hipStream_t st);
// out[c][r] = in[r][c] for in [rows, cols]; rows and cols multiples of 8
hipError_t transpose_launch(int dtype, int rows, int cols, const void* in, int64_t ldi, void* out, int64_t ldo,
                            hipStream_t st);

}  // namespace tps
