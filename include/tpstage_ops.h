/*
 * tpstage_ops.h -- op-level C ABI: the individual gfx950 kernels the stage
 * runs, exposed for per-kernel parity tests and microbenchmarks.
 *
 * All pointers are device pointers; `stream` is a hipStream_t (NULL = the
 * null stream).  Storage dtype is TPS_F32 or TPS_BF16 (tpstage.h); every
 * kernel computes in f32 and rounds once to the storage dtype on store
 * (round to nearest even).  All reductions run in a fixed order: results are
 * bitwise reproducible for a given shape.  Calls are asynchronous; argument
 * errors return TPS_EINVAL before anything is launched.
 */
#ifndef TPSTAGE_OPS_H
#define TPSTAGE_OPS_H

#include <stddef.h>
#include <stdint.h>

#include "tpstage.h"

#ifdef __cplusplus
extern "C" {
#endif

/* GEMM operand layouts (row-major storage):
 *   NT: C[M,N] = A[M,K] * B[N,K]^T   (forward linears: x W^T)
 *   NN: C[M,N] = A[M,K] * B[K,N]     (input gradients: dy W)
 *   TN: C[M,N] = A[K,M]^T * B[K,N]   (weight gradients: dy^T x, K = tokens)
 * The contiguous extent of each operand and every leading dimension must be
 * a multiple of 8 elements (bf16) or 4 elements (f32); the other extents are
 * free (ragged tiles are masked). */
enum { TPS_GEMM_NT = 0, TPS_GEMM_NN = 1, TPS_GEMM_TN = 2 };

/* Epilogues (acc = the f32 product, m = row, n = column):
 *   STORE       C = acc
 *   BIAS        C = acc + bias[n]
 *   BIAS_RESID  C = acc + bias[n] + resid[m, n]
 *   BIAS_GELU   u = round(acc + bias[n]); aux[m, n] = u (if aux != NULL);
 *               C = round(GeLU(u)), GeLU(u) = u/2 (1 + erf(u / sqrt 2))
 *   GELU_GRAD   C = acc * GeLU'(aux[m, n]),  GeLU'(u) = Phi(u) + u phi(u)
 *   ACC_F32     C (f32) += acc  (C is float*, read-modify-write) */
enum {
  TPS_EPI_STORE = 0, TPS_EPI_BIAS = 1, TPS_EPI_BIAS_RESID = 2,
  TPS_EPI_BIAS_GELU = 3, TPS_EPI_GELU_GRAD = 4, TPS_EPI_ACC_F32 = 5
};

int tps_op_gemm(int dtype, int layout, int epilogue, int M, int N, int K,
                const void* A, int64_t lda, const void* B, int64_t ldb,
                void* C, int64_t ldc, const void* bias, const void* resid,
                int64_t ldr, void* aux, int64_t ldaux, void* stream);

/* LayerNorm over rows of x[rows, cols]: out = (x - mean) * rstd * gamma + beta
 * with mean, biased variance and rstd = 1/sqrt(var + eps) in f32.  mean and
 * rstd ([rows] f32) are written when non-NULL.  cols <= 16384. */
int tps_op_layernorm_fwd(int dtype, int rows, int cols, const void* x,
                         const void* gamma, const void* beta, float eps,
                         void* out, float* mean, float* rstd, void* stream);

/* LayerNorm backward: with zhat = (x - mean) rstd and g = dout * gamma,
 *   dx = resid_grad + rstd (g - mean(g) - zhat mean(g zhat))
 * (resid_grad may be NULL), and, when dgamma / dbeta are non-NULL,
 *   dgamma += sum_rows dout * zhat,  dbeta += sum_rows dout  (f32, fixed order).
 * workspace: tps_op_workspace_bytes(TPS_WS_COLSUM, rows, 2 * cols) bytes. */
int tps_op_layernorm_bwd(int dtype, int rows, int cols, const void* dout,
                         const void* x, const float* mean, const float* rstd,
                         const void* gamma, const void* resid_grad, void* dx,
                         float* dgamma, float* dbeta, float* workspace,
                         void* stream);

/* Causal attention forward over packed qkv[b*s, 3*heads*d]:
 *   o = softmax(q k^T / sqrt(d), keys j <= query i of the same sequence) v,
 *   lse[b, heads, s] = log sum_{j <= i} exp(q_i . k_j / sqrt(d)) (may be NULL).
 * d = 64 or 128.  o is [b*s, heads*d]. */
int tps_op_attention_fwd(int dtype, int b, int s, int n_heads, int head_dim,
                         const void* qkv, void* o, float* lse, void* stream);

/* Causal attention backward: dqkv[b*s, 3*heads*d] from qkv, o, lse and do.
 * Deterministic (no atomics).  workspace: tps_op_workspace_bytes(
 * TPS_WS_ATTN_BWD, b * s, n_heads) bytes. */
int tps_op_attention_bwd(int dtype, int b, int s, int n_heads, int head_dim,
                         const void* qkv, const void* o, const float* lse,
                         const void* d_o, void* dqkv, float* workspace,
                         void* stream);

/* Allocation-free variant of tps_op_attention_bwd, for callers that cannot
 * allocate device memory (code under stream capture, tight serving loops,
 * harnesses that forbid allocation): same arguments without the workspace
 * and bitwise the same result.  Its row-dot workspace is a fixed device
 * array of the library (4 MiB per GPU, held until the process ends), so
 * b * s * n_heads must not exceed tps_op_attention_bwd_noalloc_max_rows()
 * (TPS_EINVAL otherwise, before anything is launched).  Calls allocate
 * nothing (the first call on a device only looks up the array's address).
 * All calls on one GPU share that GPU's array: calls that overlap in time on
 * one GPU (different streams without ordering between them, or host threads)
 * race; calls ordered on one stream do not. */
int tps_op_attention_bwd_noalloc(int dtype, int b, int s, int n_heads, int head_dim,
                                 const void* qkv, const void* o, const float* lse,
                                 const void* d_o, void* dqkv, void* stream);
int64_t tps_op_attention_bwd_noalloc_max_rows(void);

/* out[c] += sum_r x[r, c] over x[rows, cols] (leading dimension ldx), f32,
 * fixed order.  workspace: tps_op_workspace_bytes(TPS_WS_COLSUM, rows, cols). */
int tps_op_colsum(int dtype, int rows, int cols, const void* x, int64_t ldx,
                  float* out, float* workspace, void* stream);

/* Expansion of an FP8 E4M3 weight matrix with one f32 scale per row (the
 * quantized weight reload of streamed layers, tpstage.h TPS_Q_FP8_ROW):
 * out[r][c] = bf16(decode(q[r][c]) * scale[r]), f32 product rounded to
 * nearest even.  q: rows * cols bytes (8-byte aligned), out: bf16 (16-byte
 * aligned), cols a multiple of 8. */
int tps_op_dequant_fp8_rows(int64_t rows, int64_t cols, const void* q, const float* scale, void* out, void* stream);

/* g[i] = round(GeLU(u[i])) for n elements. */
int tps_op_gelu(int dtype, int64_t n, const void* u, void* g, void* stream);

/* LLAMA-style layer kernels (the layer the paper's evaluation runs as
 * LLAMA2-70B, Section 6.1 "Workloads"; architecture from the public LLAMA-2
 * description).
 *
 * RMSNorm over rows of x[rows, cols]: out = x * rstd * gamma with
 * rstd = 1/sqrt(mean(x^2) + eps) in f32 ([rows] f32, written when non-NULL).
 * cols <= 16384. */
int tps_op_rmsnorm_fwd(int dtype, int rows, int cols, const void* x, const void* gamma, float eps, void* out,
                       float* rstd, void* stream);

/* RMSNorm backward: with zhat = x rstd and g = dout * gamma,
 *   dx = resid_grad + rstd (g - zhat mean(g zhat))   (resid_grad may be NULL)
 * and, when dgamma is non-NULL, dgamma += sum_rows dout * zhat (f32, fixed
 * order).  workspace: tps_op_workspace_bytes(TPS_WS_COLSUM, rows, cols). */
int tps_op_rmsnorm_bwd(int dtype, int rows, int cols, const void* dout, const void* x, const float* rstd,
                       const void* gamma, const void* resid_grad, void* dx, float* dgamma, float* workspace,
                       void* stream);

/* Rotary position embedding, in place, bf16: for each of `rows` rows
 * (position row % s) and each of the first n_rot heads of d columns (d a
 * multiple of 16, ld a multiple of 8), the pair (x_i, x_{i+d/2}), i < d/2,
 * turns by +angle (inverse != 0: -angle, the gradient's transposed rotation),
 * angle = pos * base^(-2i/d).  table: caller's [2 s d/2] f32 workspace,
 * filled with cos and sin (evaluated in double, rounded once) before use. */
int tps_op_rope(void* x, int64_t ld, int rows, int s, int n_rot, int d, float base, int inverse, float* table,
                void* stream);

/* SwiGLU, bf16: g[r, j] = SiLU(u[r, j]) * u[r, f + j] for u [rows, 2f]
 * (gate | up), SiLU(z) = z / (1 + exp(-z)); f a multiple of 8. */
int tps_op_swiglu_fwd(int rows, int f, const void* u, void* g, void* stream);

/* SwiGLU backward: du[r, j] = dg * up * sigma(gate) (1 + gate (1 - sigma(gate))),
 * du[r, f + j] = dg * SiLU(gate), from dg [rows, f] and u [rows, 2f]. */
int tps_op_swiglu_bwd(int rows, int f, const void* dg, const void* u, void* du, void* stream);

/* Causal grouped-query attention, bf16, head dim 128: qkv [b*s, (n_heads +
 * 2 n_kv) 128] holds q of n_heads heads, then k and v of n_kv heads
 * (n_heads a multiple of n_kv); query head n attends with key/value head
 * n / (n_heads / n_kv).  o [b*s, n_heads 128], lse [b, n_heads, s] f32. */
int tps_op_attention_gqa_fwd(int b, int s, int n_heads, int n_kv, const void* qkv, void* o, float* lse,
                             void* stream);

/* Its backward: dqkv (layout of qkv) from qkv, o, lse and do; the key/value
 * gradient of a head is the sum over its query heads in ascending order.
 * workspace: tps_op_workspace_bytes(TPS_WS_ATTN_BWD, b*s, n_heads) bytes;
 * kv_workspace: b*s * 2 * n_heads * 128 bf16 when n_kv < n_heads (may be NULL
 * when n_kv == n_heads). */
int tps_op_attention_gqa_bwd(int b, int s, int n_heads, int n_kv, const void* qkv, const void* o, const float* lse,
                             const void* d_o, void* dqkv, float* workspace, void* kv_workspace, void* stream);

enum { TPS_WS_COLSUM = 0, TPS_WS_ATTN_BWD = 1 };
uint64_t tps_op_workspace_bytes(int kind, int64_t rows, int64_t cols);

#ifdef __cplusplus
}
#endif
#endif /* TPSTAGE_OPS_H */
