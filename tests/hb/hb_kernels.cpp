// Kernel launchers of the stage library (csrc/kernels.h) for the
// happens-before checker build: each records the byte ranges its kernels
// read and write, from the operand shapes and layouts documented in
// csrc/kernels.h and include/tpstage_ops.h, and computes nothing.
#include <cstdint>
#include <string>

#include "hb.h"
#include "kernels.h"
#include "ws.h"

namespace {

uint64_t U(const void* p) { return reinterpret_cast<uint64_t>(p); }

// rows x row_bytes at stride `stride` bytes
void add2d(HbRanges& v, const void* p, int64_t rows, int64_t row_bytes, int64_t stride) {
  if (!p || rows <= 0 || row_bytes <= 0) return;
  if (stride == row_bytes) {
    v.push_back({U(p), U(p) + (uint64_t)(rows * row_bytes)});
    return;
  }
  for (int64_t r = 0; r < rows; ++r) v.push_back({U(p) + (uint64_t)(r * stride), U(p) + (uint64_t)(r * stride + row_bytes)});
}

void add1d(HbRanges& v, const void* p, int64_t bytes) {
  if (p && bytes > 0) v.push_back({U(p), U(p) + (uint64_t)bytes});
}

int64_t esz(int dtype) { return dtype == TPS_BF16 ? 2 : 4; }

}  // namespace

namespace tps {

GemmTile gemm_select_tile(int, int, const GemmArgs&) { return {128, 128, 32, 0}; }
const char* gemm_kernel_name(int, int, const GemmArgs&) { return "gemm"; }
const char* attention_fwd_v3_name(int, int, int) { return "attention forward"; }

hipError_t gemm_launch(int dtype, int layout, int epi, int M, int N, int K, const void* A, int64_t lda, const void* B,
                       int64_t ldb, void* C, int64_t ldc, const void* bias, const void* resid, int64_t ldr, void* aux,
                       int64_t ldaux, hipStream_t stream, int overwrite) {
  const int64_t e = esz(dtype);
  HbRanges rd, wr;
  if (layout == TPS_GEMM_TN) add2d(rd, A, K, M * e, lda * e);
  else add2d(rd, A, M, K * e, lda * e);
  if (layout == TPS_GEMM_NT) add2d(rd, B, N, K * e, ldb * e);
  else add2d(rd, B, K, N * e, ldb * e);
  const int64_t ce = epi == TPS_EPI_ACC_F32 ? 4 : e;
  if (epi == TPS_EPI_ACC_F32 && !overwrite) add2d(rd, C, M, N * ce, ldc * ce);
  add2d(wr, C, M, N * ce, ldc * ce);
  if (epi == TPS_EPI_BIAS || epi == TPS_EPI_BIAS_RESID || epi == TPS_EPI_BIAS_GELU) add1d(rd, bias, N * e);
  if (epi == TPS_EPI_BIAS_RESID) add2d(rd, resid, M, N * e, ldr * e);
  if (epi == TPS_EPI_BIAS_GELU) add2d(wr, aux, M, N * e, ldaux * e);
  if (epi == TPS_EPI_GELU_GRAD) add2d(rd, aux, M, N * e, ldaux * e);
  hb_op(stream, ("gemm layout " + std::to_string(layout) + " epilogue " + std::to_string(epi)).c_str(), rd, wr);
  return hipSuccess;
}

hipError_t attention_fwd_launch(int dtype, int b, int s, int nh, int nkv, int d, const void* qkv, void* o, float* lse,
                                hipStream_t st) {
  const int64_t e = esz(dtype), T = (int64_t)b * s, h = (int64_t)nh * d, qw = (int64_t)(nh + 2 * nkv) * d;
  HbRanges rd, wr;
  add1d(rd, qkv, T * qw * e);
  add1d(wr, o, T * h * e);
  add1d(wr, lse, T * nh * 4);
  hb_op(st, "attention forward", rd, wr);
  return hipSuccess;
}

hipError_t attention_bwd_launch(int dtype, int b, int s, int nh, int nkv, int d, const void* qkv, const void* o,
                                const float* lse, const void* dout, void* dqkv, float* dvec, void* kv_ws,
                                hipStream_t st) {
  const int64_t e = esz(dtype), T = (int64_t)b * s, h = (int64_t)nh * d, qw = (int64_t)(nh + 2 * nkv) * d;
  HbRanges rd, wr, rd2;
  add1d(rd, o, T * h * e);
  add1d(rd, dout, T * h * e);
  add1d(wr, dvec, T * nh * 4);
  hb_op(st, "attention backward row dots", rd, wr);
  add1d(rd2, qkv, T * qw * e);
  add1d(rd2, lse, T * nh * 4);
  add1d(rd2, dout, T * h * e);
  add1d(rd2, dvec, T * nh * 4);
  HbRanges wr2;
  if (nkv == nh) {
    add1d(wr2, dqkv, T * qw * e);
    hb_op(st, "attention backward", rd2, wr2);
    return hipSuccess;
  }
  // dQ into dqkv, per-query-head dK, dV into the workspace, then the fold
  add2d(wr2, dqkv, T, h * e, qw * e);
  add1d(wr2, kv_ws, T * 2 * h * e);
  hb_op(st, "attention backward", rd2, wr2);
  HbRanges rd3, wr3;
  add1d(rd3, kv_ws, T * 2 * h * e);
  add2d(wr3, static_cast<const char*>(dqkv) + h * e, T, (qw - h) * e, qw * e);
  hb_op(st, "grouped key/value gradient fold", rd3, wr3);
  return hipSuccess;
}

hipError_t layernorm_fwd_launch(int dtype, int rows, int cols, const void* x, const void* gamma, const void* beta,
                                float, void* out, float* mean, float* rstd, hipStream_t st) {
  const int64_t e = esz(dtype);
  HbRanges rd, wr;
  add1d(rd, x, (int64_t)rows * cols * e);
  add1d(rd, gamma, cols * e);
  add1d(rd, beta, cols * e);
  add1d(wr, out, (int64_t)rows * cols * e);
  add1d(wr, mean, rows * 4);
  add1d(wr, rstd, rows * 4);
  hb_op(st, "layernorm forward", rd, wr);
  return hipSuccess;
}

hipError_t layernorm_bwd_acc_launch(int dtype, int rows, int cols, const void* dout, const void* x, const float* mean,
                                    const float* rstd, const void* gamma, const void* resid, void* dx,
                                    float* part_dbeta, int64_t k_stride, int64_t seg_stride, hipStream_t st) {
  const int64_t e = esz(dtype);
  HbRanges rd, wr;
  add1d(rd, dout, (int64_t)rows * cols * e);
  add1d(rd, x, (int64_t)rows * cols * e);
  add1d(rd, mean, rows * 4);
  add1d(rd, rstd, rows * 4);
  add1d(rd, gamma, cols * e);
  add1d(rd, resid, (int64_t)rows * cols * e);
  add1d(wr, dx, (int64_t)rows * cols * e);
  const int64_t segs = colsum_segments(rows);
  for (int64_t sgi = 0; sgi < segs; ++sgi) {
    for (int64_t off : {(int64_t)0, k_stride}) {
      const float* p = part_dbeta + sgi * seg_stride + off;
      add1d(rd, p, cols * 4);
      add1d(wr, p, cols * 4);
    }
  }
  hb_op(st, "layernorm backward", rd, wr);
  return hipSuccess;
}

hipError_t colsum_acc_launch(int dtype, int rows, int cols, const void* x, int64_t ldx, float* part, int64_t seg_stride,
                             hipStream_t st) {
  const int64_t e = esz(dtype);
  HbRanges rd, wr;
  add2d(rd, x, rows, cols * e, ldx * e);
  const int64_t segs = colsum_segments(rows);
  for (int64_t sgi = 0; sgi < segs; ++sgi) {
    add1d(rd, part + sgi * seg_stride, cols * 4);
    add1d(wr, part + sgi * seg_stride, cols * 4);
  }
  hb_op(st, "column sums", rd, wr);
  return hipSuccess;
}

hipError_t colsum_finalize_launch(const ColMap& m, float* part, int segs, int64_t seg_stride, float* grads,
                                  hipStream_t st, int overwrite) {
  HbRanges rd, wr;
  for (int sgi = 0; sgi < segs; ++sgi) {
    add1d(rd, part + sgi * seg_stride + m.c0[0], (int64_t)(m.c0[m.n] - m.c0[0]) * 4);
    add1d(wr, part + sgi * seg_stride + m.c0[0], (int64_t)(m.c0[m.n] - m.c0[0]) * 4);
  }
  for (int r = 0; r < m.n; ++r) {
    float* g = grads + m.goff[r];
    const int64_t n = m.c0[r + 1] - m.c0[r];
    if (!overwrite) add1d(rd, g, n * 4);
    add1d(wr, g, n * 4);
  }
  hb_op(st, "bias gradient finalize", rd, wr);
  return hipSuccess;
}

hipError_t rmsnorm_fwd_launch(int dtype, int rows, int cols, const void* x, const void* gamma, float, void* out,
                              float* rstd, hipStream_t st) {
  const int64_t e = esz(dtype);
  HbRanges rd, wr;
  add1d(rd, x, (int64_t)rows * cols * e);
  add1d(rd, gamma, cols * e);
  add1d(wr, out, (int64_t)rows * cols * e);
  add1d(wr, rstd, rows * 4);
  hb_op(st, "rmsnorm forward", rd, wr);
  return hipSuccess;
}

hipError_t rmsnorm_bwd_acc_launch(int dtype, int rows, int cols, const void* dout, const void* x, const float* rstd,
                                  const void* gamma, const void* resid, void* dx, float* part_dgamma,
                                  int64_t seg_stride, hipStream_t st) {
  const int64_t e = esz(dtype);
  HbRanges rd, wr;
  add1d(rd, dout, (int64_t)rows * cols * e);
  add1d(rd, x, (int64_t)rows * cols * e);
  add1d(rd, rstd, rows * 4);
  add1d(rd, gamma, cols * e);
  add1d(rd, resid, (int64_t)rows * cols * e);
  add1d(wr, dx, (int64_t)rows * cols * e);
  const int64_t segs = colsum_segments(rows);
  for (int64_t sgi = 0; sgi < segs; ++sgi) {
    add1d(rd, part_dgamma + sgi * seg_stride, cols * 4);
    add1d(wr, part_dgamma + sgi * seg_stride, cols * 4);
  }
  hb_op(st, "rmsnorm backward", rd, wr);
  return hipSuccess;
}

hipError_t rope_table_launch(int s, int d, float, float* table, hipStream_t st) {
  HbRanges none, wr;
  add1d(wr, table, (int64_t)s * d * 4);
  hb_op(st, "rotation table", none, wr);
  return hipSuccess;
}

hipError_t rope_launch(void* x, int64_t ld, int rows, int s, int n_rot, int d, const float* table, int,
                       hipStream_t st) {
  HbRanges rd, wr;
  add2d(rd, x, rows, (int64_t)n_rot * d * 2, ld * 2);
  add2d(wr, x, rows, (int64_t)n_rot * d * 2, ld * 2);
  add1d(rd, table, (int64_t)s * d * 4);
  hb_op(st, "rope", rd, wr);
  return hipSuccess;
}

hipError_t swiglu_launch(int rows, int f, const void* u, void* g, hipStream_t st) {
  HbRanges rd, wr;
  add1d(rd, u, (int64_t)rows * 2 * f * 2);
  add1d(wr, g, (int64_t)rows * f * 2);
  hb_op(st, "swiglu", rd, wr);
  return hipSuccess;
}

hipError_t swiglu_bwd_launch(int rows, int f, const void* dg, const void* u, void* du, hipStream_t st) {
  HbRanges rd, wr;
  add1d(rd, dg, (int64_t)rows * f * 2);
  add1d(rd, u, (int64_t)rows * 2 * f * 2);
  add1d(wr, du, (int64_t)rows * 2 * f * 2);
  hb_op(st, "swiglu backward", rd, wr);
  return hipSuccess;
}

hipError_t gelu_launch(int dtype, int64_t n, const void* u, void* g, hipStream_t st) {
  HbRanges rd, wr;
  add1d(rd, u, n * esz(dtype));
  add1d(wr, g, n * esz(dtype));
  hb_op(st, "gelu", rd, wr);
  return hipSuccess;
}

hipError_t fill_bytes_launch(void* p, uint64_t bytes, uint8_t value, hipStream_t st) {
  HbRanges none, wr;
  add1d(wr, p, (int64_t)bytes);
  hb_op(st, value ? "fill" : "fill zero", none, wr);
  return hipSuccess;
}

hipError_t fill_zero_launch(void* p, uint64_t bytes, hipStream_t st) { return fill_bytes_launch(p, bytes, 0, st); }

hipError_t adamw_launch(int dtype, int64_t n, float* w, float* m, float* v, const float* g, void* out,
                        const float* /*c*/, hipStream_t st) {
  HbRanges rd, wr;
  for (const float* p : {(const float*)w, (const float*)m, (const float*)v, g}) add1d(rd, p, n * 4);
  for (float* p : {w, m, v}) add1d(wr, p, n * 4);
  add1d(wr, out, n * esz(dtype));
  hb_op(st, "adamw", rd, wr);
  return hipSuccess;
}

hipError_t dequant_fp8_rows_launch(const void* q, const float* scale, int64_t rows, int64_t cols, void* out,
                                   hipStream_t st) {
  HbRanges rd, wr;
  add1d(rd, q, rows * cols);
  add1d(rd, scale, rows * 4);
  add1d(wr, out, rows * cols * 2);
  hb_op(st, "dequantize weights", rd, wr);
  return hipSuccess;
}

hipError_t transpose_launch(int dtype, int rows, int cols, const void* in, int64_t ldi, void* out, int64_t ldo,
                            hipStream_t st) {
  const int64_t e = esz(dtype);
  HbRanges rd, wr;
  add2d(rd, in, rows, cols * e, ldi * e);
  add2d(wr, out, cols, rows * e, ldo * e);
  hb_op(st, "transpose", rd, wr);
  return hipSuccess;
}

}  // namespace tps
