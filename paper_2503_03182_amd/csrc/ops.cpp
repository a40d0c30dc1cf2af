// Op-level C ABI (tpstage_ops.h): argument checks, then one kernel launch
// sequence on the caller's stream.
#include <cstdio>
#include <string>

#include "errors.h"
#include "kernels.h"

using namespace tps;

namespace {

int vec_of(int dtype) { return dtype == TPS_BF16 ? 8 : 4; }
bool dtype_ok(int dtype) { return dtype == TPS_F32 || dtype == TPS_BF16; }
bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

int bad(const std::string& m) { return set_error(TPS_EINVAL, m); }

}  // namespace

extern "C" int tps_op_gemm(int dtype, int layout, int epilogue, int M, int N, int K, const void* A,
                           int64_t lda, const void* B, int64_t ldb, void* C, int64_t ldc,
                           const void* bias, const void* resid, int64_t ldr, void* aux,
                           int64_t ldaux, void* stream) {
  clear_error();
  if (!dtype_ok(dtype)) return bad("gemm: dtype");
  if (layout < TPS_GEMM_NT || layout > TPS_GEMM_TN) return bad("gemm: layout");
  if (epilogue < TPS_EPI_STORE || epilogue > TPS_EPI_ACC_F32) return bad("gemm: epilogue");
  if (M < 0 || N < 0 || K < 0) return bad("gemm: negative extent");
  if (M == 0 || N == 0) return TPS_OK;
  if (!A || !B || !C) return bad("gemm: null operand");
  const int v = vec_of(dtype);
  // contiguous extent of each operand, and leading dimensions
  const int64_t a_contig = (layout == TPS_GEMM_TN) ? M : K;
  const int64_t b_contig = (layout == TPS_GEMM_NT) ? K : N;
  if (a_contig % v || b_contig % v || lda % v || ldb % v)
    return bad("gemm: contiguous extents and lda/ldb must be multiples of 8 (bf16) / 4 (f32)");
  if (lda < a_contig || ldb < b_contig || ldc < N) return bad("gemm: leading dimension too small");
  if (!aligned16(A) || !aligned16(B)) return bad("gemm: A and B must be 16-byte aligned");
  const bool needs_bias = epilogue == TPS_EPI_BIAS || epilogue == TPS_EPI_BIAS_RESID || epilogue == TPS_EPI_BIAS_GELU;
  if (needs_bias && !bias) return bad("gemm: epilogue needs bias");
  if (epilogue == TPS_EPI_BIAS_RESID && (!resid || ldr < N)) return bad("gemm: epilogue needs resid");
  if (epilogue == TPS_EPI_GELU_GRAD && (!aux || ldaux < N)) return bad("gemm: GELU_GRAD needs aux (u)");
  if (epilogue == TPS_EPI_BIAS_GELU && aux && ldaux < N) return bad("gemm: ldaux too small");
  return check_hip(gemm_launch(dtype, layout, epilogue, M, N, K, A, lda, B, ldb, C, ldc, bias, resid, ldr,
                               aux, ldaux, (hipStream_t)stream),
                   "gemm launch");
}

extern "C" int tps_op_layernorm_fwd(int dtype, int rows, int cols, const void* x, const void* gamma,
                                    const void* beta, float eps, void* out, float* mean, float* rstd,
                                    void* stream) {
  clear_error();
  if (!dtype_ok(dtype)) return bad("layernorm: dtype");
  if (rows < 0 || cols <= 0 || cols > 16384 || cols % vec_of(dtype)) return bad("layernorm: cols");
  if (!x || !gamma || !beta || !out) return bad("layernorm: null pointer");
  return check_hip(layernorm_fwd_launch(dtype, rows, cols, x, gamma, beta, eps, out, mean, rstd,
                                        (hipStream_t)stream),
                   "layernorm_fwd launch");
}

extern "C" int tps_op_layernorm_bwd(int dtype, int rows, int cols, const void* dout, const void* x,
                                    const float* mean, const float* rstd, const void* gamma,
                                    const void* resid_grad, void* dx, float* dgamma, float* dbeta,
                                    float* workspace, void* stream) {
  clear_error();
  if (!dtype_ok(dtype)) return bad("layernorm_bwd: dtype");
  if (rows < 0 || cols <= 0 || cols > 16384 || cols % vec_of(dtype)) return bad("layernorm_bwd: cols");
  if (!dout || !x || !mean || !rstd || !gamma || !dx) return bad("layernorm_bwd: null pointer");
  if ((dgamma || dbeta) && !workspace) return bad("layernorm_bwd: workspace needed for dgamma/dbeta");
  return check_hip(layernorm_bwd_launch(dtype, rows, cols, dout, x, mean, rstd, gamma, resid_grad, dx,
                                        dgamma, dbeta, workspace, (hipStream_t)stream),
                   "layernorm_bwd launch");
}

extern "C" int tps_op_attention_fwd(int dtype, int b, int s, int n_heads, int head_dim, const void* qkv,
                                    void* o, float* lse, void* stream) {
  clear_error();
  if (!dtype_ok(dtype)) return bad("attention: dtype");
  if (head_dim != 64 && head_dim != 128) return bad("attention: head_dim must be 64 or 128");
  if (b < 0 || s < 0 || n_heads <= 0) return bad("attention: shape");
  if (b == 0 || s == 0) return TPS_OK;
  if (!qkv || !o || !aligned16(qkv)) return bad("attention: qkv/o");
  return check_hip(attention_fwd_launch(dtype, b, s, n_heads, n_heads, head_dim, qkv, o, lse, (hipStream_t)stream),
                   "attention_fwd launch");
}

extern "C" int tps_op_attention_bwd(int dtype, int b, int s, int n_heads, int head_dim, const void* qkv,
                                    const void* o, const float* lse, const void* d_o, void* dqkv,
                                    float* workspace, void* stream) {
  clear_error();
  if (!dtype_ok(dtype)) return bad("attention_bwd: dtype");
  if (head_dim != 64 && head_dim != 128) return bad("attention_bwd: head_dim must be 64 or 128");
  if (b < 0 || s < 0 || n_heads <= 0) return bad("attention_bwd: shape");
  if (b == 0 || s == 0) return TPS_OK;
  if (!qkv || !o || !lse || !d_o || !dqkv || !workspace) return bad("attention_bwd: null pointer");
  if (!aligned16(qkv) || !aligned16(o) || !aligned16(d_o)) return bad("attention_bwd: alignment");
  return check_hip(attention_bwd_launch(dtype, b, s, n_heads, n_heads, head_dim, qkv, o, lse, d_o, dqkv, workspace,
                                        nullptr, (hipStream_t)stream),
                   "attention_bwd launch");
}

extern "C" int tps_op_rmsnorm_fwd(int dtype, int rows, int cols, const void* x, const void* gamma, float eps,
                                  void* out, float* rstd, void* stream) {
  clear_error();
  if (!dtype_ok(dtype)) return bad("rmsnorm: dtype");
  if (rows < 0 || cols <= 0 || cols > 16384 || cols % vec_of(dtype)) return bad("rmsnorm: shape");
  if (!(eps >= 0.f)) return bad("rmsnorm: eps");
  if (rows == 0) return TPS_OK;
  if (!x || !gamma || !out) return bad("rmsnorm: null pointer");
  return check_hip(rmsnorm_fwd_launch(dtype, rows, cols, x, gamma, eps, out, rstd, (hipStream_t)stream),
                   "rmsnorm_fwd launch");
}

extern "C" int tps_op_rmsnorm_bwd(int dtype, int rows, int cols, const void* dout, const void* x, const float* rstd,
                                  const void* gamma, const void* resid_grad, void* dx, float* dgamma,
                                  float* workspace, void* stream) {
  clear_error();
  if (!dtype_ok(dtype)) return bad("rmsnorm_bwd: dtype");
  if (rows < 0 || cols <= 0 || cols > 16384 || cols % vec_of(dtype)) return bad("rmsnorm_bwd: shape");
  if (rows == 0) return TPS_OK;
  if (!dout || !x || !rstd || !gamma || !dx) return bad("rmsnorm_bwd: null pointer");
  if (dgamma && !workspace) return bad("rmsnorm_bwd: workspace needed for dgamma");
  return check_hip(rmsnorm_bwd_launch(dtype, rows, cols, dout, x, rstd, gamma, resid_grad, dx, dgamma, workspace,
                                      (hipStream_t)stream),
                   "rmsnorm_bwd launch");
}

extern "C" int tps_op_rope(void* x, int64_t ld, int rows, int s, int n_rot, int d, float base, int inverse,
                           float* table, void* stream) {
  clear_error();
  if (rows < 0 || s <= 0 || n_rot < 0 || d <= 0 || d % 16 || ld % 8 || ld < (int64_t)n_rot * d)
    return bad("rope: shape");
  if (!(base > 1.f)) return bad("rope: base must be > 1");
  if (rows == 0 || n_rot == 0) return TPS_OK;
  if (!x || !table || !aligned16(x) || !aligned16(table)) return bad("rope: pointers");
  hipError_t e = rope_table_launch(s, d, base, table, (hipStream_t)stream);
  if (e == hipSuccess) e = rope_launch(x, ld, rows, s, n_rot, d, table, inverse, (hipStream_t)stream);
  return check_hip(e, "rope launch");
}

extern "C" int tps_op_swiglu_fwd(int rows, int f, const void* u, void* g, void* stream) {
  clear_error();
  if (rows < 0 || f <= 0 || f % 8) return bad("swiglu: shape");
  if (rows == 0) return TPS_OK;
  if (!u || !g || !aligned16(u) || !aligned16(g)) return bad("swiglu: pointers");
  return check_hip(swiglu_launch(rows, f, u, g, (hipStream_t)stream), "swiglu launch");
}

extern "C" int tps_op_swiglu_bwd(int rows, int f, const void* dg, const void* u, void* du, void* stream) {
  clear_error();
  if (rows < 0 || f <= 0 || f % 8) return bad("swiglu_bwd: shape");
  if (rows == 0) return TPS_OK;
  if (!dg || !u || !du || !aligned16(dg) || !aligned16(u) || !aligned16(du)) return bad("swiglu_bwd: pointers");
  return check_hip(swiglu_bwd_launch(rows, f, dg, u, du, (hipStream_t)stream), "swiglu_bwd launch");
}

extern "C" int tps_op_attention_gqa_fwd(int b, int s, int n_heads, int n_kv, const void* qkv, void* o, float* lse,
                                        void* stream) {
  clear_error();
  if (b < 0 || s < 0 || n_heads <= 0 || n_kv <= 0 || n_heads % n_kv) return bad("attention_gqa: heads");
  if (b == 0 || s == 0) return TPS_OK;
  if (!qkv || !o || !aligned16(qkv) || !aligned16(o)) return bad("attention_gqa: qkv/o");
  return check_hip(attention_fwd_launch(TPS_BF16, b, s, n_heads, n_kv, 128, qkv, o, lse, (hipStream_t)stream),
                   "attention_gqa_fwd launch");
}

extern "C" int tps_op_attention_gqa_bwd(int b, int s, int n_heads, int n_kv, const void* qkv, const void* o,
                                        const float* lse, const void* d_o, void* dqkv, float* workspace,
                                        void* kv_workspace, void* stream) {
  clear_error();
  if (b < 0 || s < 0 || n_heads <= 0 || n_kv <= 0 || n_heads % n_kv) return bad("attention_gqa_bwd: heads");
  if (b == 0 || s == 0) return TPS_OK;
  if (!qkv || !o || !lse || !d_o || !dqkv || !workspace) return bad("attention_gqa_bwd: null pointer");
  if (n_kv != n_heads && (!kv_workspace || !aligned16(kv_workspace)))
    return bad("attention_gqa_bwd: kv_workspace needed for grouped heads");
  if (!aligned16(qkv) || !aligned16(o) || !aligned16(d_o) || !aligned16(dqkv)) return bad("attention_gqa_bwd: alignment");
  return check_hip(attention_bwd_launch(TPS_BF16, b, s, n_heads, n_kv, 128, qkv, o, lse, d_o, dqkv, workspace,
                                        kv_workspace, (hipStream_t)stream),
                   "attention_gqa_bwd launch");
}

extern "C" int tps_op_colsum(int dtype, int rows, int cols, const void* x, int64_t ldx, float* out,
                             float* workspace, void* stream) {
  clear_error();
  if (!dtype_ok(dtype)) return bad("colsum: dtype");
  if (rows < 0 || cols <= 0 || cols % vec_of(dtype) || ldx % vec_of(dtype) || ldx < cols)
    return bad("colsum: shape");
  if (!x || !out || !workspace) return bad("colsum: null pointer");
  return check_hip(colsum_launch(dtype, rows, cols, x, ldx, out, workspace, (hipStream_t)stream),
                   "colsum launch");
}

extern "C" int tps_op_gelu(int dtype, int64_t n, const void* u, void* g, void* stream) {
  clear_error();
  if (!dtype_ok(dtype) || n < 0) return bad("gelu: args");
  if (n == 0) return TPS_OK;
  if (!u || !g || !aligned16(u) || !aligned16(g)) return bad("gelu: pointers");
  return check_hip(gelu_launch(dtype, n, u, g, (hipStream_t)stream), "gelu launch");
}

extern "C" int tps_op_dequant_fp8_rows(int64_t rows, int64_t cols, const void* q, const float* scale, void* out,
                                       void* stream) {
  clear_error();
  if (rows < 0 || cols <= 0 || cols % 8) return bad("dequant: cols must be a positive multiple of 8");
  if (rows == 0) return TPS_OK;
  if (!q || !scale || !out) return bad("dequant: null pointer");
  if ((reinterpret_cast<uintptr_t>(q) & 7u) || !aligned16(out)) return bad("dequant: alignment");
  return check_hip(dequant_fp8_rows_launch(q, scale, rows, cols, out, (hipStream_t)stream), "dequant launch");
}

extern "C" uint64_t tps_op_workspace_bytes(int kind, int64_t rows, int64_t cols) {
  if (kind == TPS_WS_COLSUM) return colsum_ws_bytes(rows, cols);
  if (kind == TPS_WS_ATTN_BWD) return (uint64_t)(rows * cols * 4);  // rows = b*s, cols = heads
  return 0;
}

namespace tps {

static bool v2_epilogue(int layout, int epi) {
  if (layout == TPS_GEMM_NT)
    return epi == TPS_EPI_STORE || epi == TPS_EPI_BIAS || epi == TPS_EPI_BIAS_RESID || epi == TPS_EPI_BIAS_GELU ||
           epi == TPS_EPI_GELU_GRAD;
  if (layout == TPS_GEMM_NN) return epi == TPS_EPI_STORE || epi == TPS_EPI_GELU_GRAD || epi == TPS_EPI_BIAS_RESID;
  return epi == TPS_EPI_STORE || epi == TPS_EPI_ACC_F32;
}

static bool al16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

GemmTile gemm_select_tile(int dtype, int layout, const GemmArgs& g) {
  const int M = g.M, N = g.N, K = g.K;
  if (dtype == TPS_BF16) {
    // tile-aligned path: every operand 16-byte aligned with leading dimensions
    // in whole 16-byte chunks, and an epilogue it instantiates
    bool ok = K % 64 == 0 && K > 0 && g.lda % 8 == 0 && g.ldb % 8 == 0 && v2_epilogue(layout, g.epi) &&
              al16(g.A) && al16(g.B) && al16(g.C) && g.ldc % 8 == 0;
    if (g.epi == TPS_EPI_BIAS || g.epi == TPS_EPI_BIAS_RESID || g.epi == TPS_EPI_BIAS_GELU) ok = ok && al16(g.bias);
    if (g.epi == TPS_EPI_BIAS_RESID) ok = ok && al16(g.resid) && g.ldr % 8 == 0;
    if (g.epi == TPS_EPI_BIAS_GELU || g.epi == TPS_EPI_GELU_GRAD) ok = ok && al16(g.aux) && g.ldaux % 8 == 0;
    if (ok && M % 256 == 0 && N % 256 == 0 && (int64_t)(M / 256) * (N / 256) >= 160) return {256, 256, 32, 1};
    if (ok && M % 128 == 0 && N % 128 == 0) return {128, 128, 32, 1};
    const int64_t t256 = (int64_t)((M + 255) / 256) * ((N + 127) / 128);
    if (t256 >= 256) return {256, 128, 64, 0};
    return {128, 128, 64, 0};
  }
  return {128, 128, 32, 0};
}

const char* gemm_kernel_name(int dtype, int layout, const GemmArgs& g) {
  static const char* v1[2][2][3] = {
      {{"tps::gemm_kernel<float, 128, 128, 32, 0>", "tps::gemm_kernel<float, 128, 128, 32, 1>",
        "tps::gemm_kernel<float, 128, 128, 32, 2>"},
       {"tps::gemm_kernel<float, 128, 128, 32, 0>", "tps::gemm_kernel<float, 128, 128, 32, 1>",
        "tps::gemm_kernel<float, 128, 128, 32, 2>"}},
      {{"tps::gemm_kernel<__bf16, 128, 128, 64, 0>", "tps::gemm_kernel<__bf16, 128, 128, 64, 1>",
        "tps::gemm_kernel<__bf16, 128, 128, 64, 2>"},
       {"tps::gemm_kernel<__bf16, 256, 128, 64, 0>", "tps::gemm_kernel<__bf16, 256, 128, 64, 1>",
        "tps::gemm_kernel<__bf16, 256, 128, 64, 2>"}}};
  // [long K][tile][layout][epilogue]
  static char v3[2][2][3][6][64];
  static bool init = false;
  if (!init) {
    for (int k = 0; k < 2; ++k)
      for (int t = 0; t < 2; ++t)
        for (int l = 0; l < 3; ++l)
          for (int e = 0; e < 6; ++e) {
            const V3Config c = v3_config(l, t == 1, k == 1);
            const int tile = t ? 256 : 128;
            snprintf(v3[k][t][l][e], sizeof(v3[k][t][l][e]), "tps::gemm_bf16_kernel<%d, %d, %d, %d, %d, %d, %d, %d>",
                     l, tile, tile, c.wgm, c.wgn, c.bk, c.stages, e);
          }
    init = true;
  }
  const GemmTile t = gemm_select_tile(dtype, layout, g);
  if (t.aligned) return v3[g.K >= TN_LONG_K][t.bm == 256][layout][g.epi];
  return v1[dtype == TPS_BF16][t.bm == 256][layout];
}

hipError_t gemm_launch(int dtype, int layout, int epi, int M, int N, int K, const void* A, int64_t lda,
                       const void* B, int64_t ldb, void* C, int64_t ldc, const void* bias, const void* resid,
                       int64_t ldr, void* aux, int64_t ldaux, hipStream_t stream, int overwrite) {
  if (M == 0 || N == 0) return hipSuccess;
  GemmArgs g{M, N, K, A, lda, B, ldb, C, ldc, bias, resid, ldr, aux, ldaux, epi, 0, 0, overwrite};
  if (layout == TPS_GEMM_NT) return gemm_launch_nt(dtype, g, stream);
  if (layout == TPS_GEMM_NN) return gemm_launch_nn(dtype, g, stream);
  return gemm_launch_tn(dtype, g, stream);
}

}  // namespace tps
