"""Per-kernel parity of the gfx950 kernels (through the op-level C ABI) against
the CPU oracle's functions or plain float64 numpy of the same op, at shapes
that span several tiles and leave ragged tails, in f32 and bf16."""

import numpy as np
import pytest

from oracle import decoder_stage as ora
from paper_2503_03182_amd import synth
from paper_2503_03182_amd import tpstage as T

from stage_harness import assert_close, rel_l2, to_dev, to_np

pytestmark = pytest.mark.gpu

# f32 kernels accumulate in f32; bf16 kernels round their output once
TOL = {"f32": 2e-5, "bf16": 8e-3}
DT = {"f32": T.TPS_F32, "bf16": T.TPS_BF16}


def _t(seed, shape, dtype, scale=1.0):
    return synth.uniform_tensor(seed, shape, scale, dtype)


def _round(a, dtype):
    return synth.round_to_storage(np.asarray(a, dtype=np.float32), dtype).astype(np.float64)


# ragged shapes take the generic path; tile-aligned ones (M, N multiples of
# 128 or 256, K of 64) take the direct-to-LDS path at both tile sizes: 256 x
# 256 tiles (2-stage ring) at 1 and 2 K tiles, 128 x 128 tiles (4-stage ring,
# fragments read two k-steps ahead) at 1, 2, 3, 4, 5 and 8 K tiles, so the
# ring's fill, refill and drain each meet short and long loops
GEMM_SHAPES = [(200, 264, 136), (1000, 520, 72), (64, 64, 8), (2072, 4104, 264),
               (256, 384, 192), (4096, 2560, 128), (384, 256, 512), (128, 128, 64), (256, 128, 128),
               (128, 256, 256), (384, 128, 320), (4096, 2560, 64)]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("layout", [T.GEMM_NT, T.GEMM_NN, T.GEMM_TN])
@pytest.mark.parametrize("shape", GEMM_SHAPES)
def test_gemm_store(dtype, layout, shape):
    import torch
    M, N, K = shape
    a_shape = (K, M) if layout == T.GEMM_TN else (M, K)
    b_shape = (N, K) if layout == T.GEMM_NT else (K, N)
    A = _t(11, a_shape, dtype)
    B = _t(12, b_shape, dtype)
    Am = A.astype(np.float64).T if layout == T.GEMM_TN else A.astype(np.float64)
    Bm = B.astype(np.float64).T if layout == T.GEMM_NT else B.astype(np.float64)
    ref = Am @ Bm
    dA, dB = to_dev(A, dtype), to_dev(B, dtype)
    dC = torch.full((M, N), float("nan"), device="cuda").to(dA.dtype)
    T.op_gemm(DT[dtype], layout, T.EPI_STORE, M, N, K, dA, a_shape[1], dB, b_shape[1], dC, N)
    torch.cuda.synchronize()
    assert_close(to_np(dC), ref, TOL[dtype])


@pytest.mark.parametrize("dtype,shape", [("f32", (296, 392, 200)), ("bf16", (296, 392, 200)),
                                         ("bf16", (512, 768, 256)), ("bf16", (4096, 2560, 128))])
def test_gemm_epilogues(dtype, shape):
    import torch
    M, N, K = shape
    A = _t(21, (M, K), dtype)
    B = _t(22, (N, K), dtype, 0.1)
    bias = _t(23, (N,), dtype)
    R = _t(24, (M, N), dtype)
    acc = A.astype(np.float64) @ B.astype(np.float64).T
    dA, dB, dbias, dR = (to_dev(v, dtype) for v in (A, B, bias, R))
    out = torch.empty((M, N), device="cuda", dtype=dA.dtype)
    # BIAS
    T.op_gemm(DT[dtype], T.GEMM_NT, T.EPI_BIAS, M, N, K, dA, K, dB, K, out, N, bias=dbias)
    torch.cuda.synchronize()
    assert_close(to_np(out), acc + bias, TOL[dtype])
    # BIAS_RESID
    T.op_gemm(DT[dtype], T.GEMM_NT, T.EPI_BIAS_RESID, M, N, K, dA, K, dB, K, out, N, bias=dbias, resid=dR, ldr=N)
    torch.cuda.synchronize()
    assert_close(to_np(out), acc + bias + R, TOL[dtype])
    # BIAS_GELU: u = round(acc + b) kept, g = round(GeLU(u))
    u = torch.empty_like(out)
    T.op_gemm(DT[dtype], T.GEMM_NT, T.EPI_BIAS_GELU, M, N, K, dA, K, dB, K, out, N, bias=dbias, aux=u, ldaux=N)
    torch.cuda.synchronize()
    assert_close(to_np(u), acc + bias, TOL[dtype])
    assert_close(to_np(out), ora.gelu(to_np(u)), TOL[dtype])
    # and without keeping u the GeLU output is bitwise the same
    out2 = torch.empty_like(out)
    T.op_gemm(DT[dtype], T.GEMM_NT, T.EPI_BIAS_GELU, M, N, K, dA, K, dB, K, out2, N, bias=dbias)
    torch.cuda.synchronize()
    assert torch.equal(out, out2)
    # GELU_GRAD (NN): C = (A B) * GeLU'(aux)
    B2 = _t(25, (K, N), dtype, 0.1)
    U = _t(26, (M, N), dtype)
    T.op_gemm(DT[dtype], T.GEMM_NN, T.EPI_GELU_GRAD, M, N, K, dA, K, to_dev(B2, dtype), N, out, N,
              aux=to_dev(U, dtype), ldaux=N)
    torch.cuda.synchronize()
    ref = (A.astype(np.float64) @ B2.astype(np.float64)) * ora.gelu_grad(U.astype(np.float64))
    assert_close(to_np(out), ref, TOL[dtype])
    # BIAS_RESID (NN): C = A B + bias + R
    T.op_gemm(DT[dtype], T.GEMM_NN, T.EPI_BIAS_RESID, M, N, K, dA, K, to_dev(B2, dtype), N, out, N, bias=dbias,
              resid=dR, ldr=N)
    torch.cuda.synchronize()
    assert_close(to_np(out), A.astype(np.float64) @ B2.astype(np.float64) + bias + R, TOL[dtype])
    # ACC_F32 (TN): C32 += A^T B over K rows
    A3 = _t(27, (K, M), dtype)
    B3 = _t(28, (K, N), dtype)
    C0 = synth.uniform_tensor(29, (M, N), 1.0, "f32")
    C32 = torch.from_numpy(C0.copy()).cuda()
    T.op_gemm(DT[dtype], T.GEMM_TN, T.EPI_ACC_F32, M, N, K, to_dev(A3, dtype), M, to_dev(B3, dtype), N, C32, N)
    torch.cuda.synchronize()
    ref = C0.astype(np.float64) + A3.astype(np.float64).T @ B3.astype(np.float64)
    assert_close(C32.cpu().numpy(), ref, 2e-6)


def test_gemm_leading_dimensions_and_deterministic():
    """Sub-matrix views (ld > extent) and bitwise repeatability."""
    import torch
    M, N, K = 256, 192, 128
    big_a = _t(31, (M, 3 * K), "bf16")
    big_b = _t(32, (N, 2 * K), "bf16")
    A = big_a[:, K:2 * K]
    B = big_b[:, :K]
    dA, dB = to_dev(big_a, "bf16"), to_dev(big_b, "bf16")
    outs = []
    for _ in range(2):
        C = torch.empty((M, N), device="cuda", dtype=torch.bfloat16)
        T.op_gemm(T.TPS_BF16, T.GEMM_NT, T.EPI_STORE, M, N, K, dA[:, K:], 3 * K, dB, 2 * K, C, N)
        outs.append(C)
    torch.cuda.synchronize()
    assert torch.equal(outs[0], outs[1])
    assert_close(to_np(outs[0]), A.astype(np.float64) @ B.astype(np.float64).T, TOL["bf16"])


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("rows,cols", [(300, 256), (77, 2048), (64, 5120), (33, 8192)])
def test_layernorm_fwd_bwd(dtype, rows, cols):
    import torch
    x = _t(41, (rows, cols), dtype, 2.0) + _round(np.full((rows, cols), 0.5), dtype).astype(np.float32)
    x = synth.round_to_storage(x, dtype)
    gamma = synth.round_to_storage(1.0 + _t(42, (cols,), "f32", 0.1), dtype)
    beta = _t(43, (cols,), dtype, 0.1)
    dout = _t(44, (rows, cols), dtype)
    resid = _t(45, (rows, cols), dtype)
    eps = 1e-5
    ref, mu, rs = ora.layer_norm(x.astype(np.float64), gamma.astype(np.float64), beta.astype(np.float64), eps)
    dx_ref, dg_ref, db_ref = ora.layer_norm_backward(dout.astype(np.float64), x.astype(np.float64), mu, rs,
                                                     gamma.astype(np.float64))
    dx_ref = dx_ref + resid
    dX, dG, dBt, dD, dR = (to_dev(v, dtype) for v in (x, gamma, beta, dout, resid))
    out = torch.empty_like(dX)
    mean = torch.empty(rows, device="cuda")
    rstd = torch.empty(rows, device="cuda")
    T.op_layernorm_fwd(DT[dtype], rows, cols, dX, dG, dBt, eps, out, mean, rstd)
    dxo = torch.empty_like(dX)
    dg = torch.full((cols,), 0.25, device="cuda")
    dbb = torch.full((cols,), -0.5, device="cuda")
    ws = torch.empty(T.op_workspace_bytes(T.WS_COLSUM, rows, 2 * cols) // 4, device="cuda")
    T.op_layernorm_bwd(DT[dtype], rows, cols, dD, dX, mean, rstd, dG, dR, dxo, dg, dbb, ws)
    torch.cuda.synchronize()
    assert_close(to_np(out), ref, TOL[dtype])
    assert np.allclose(mean.cpu().numpy(), mu, rtol=1e-5, atol=1e-5)
    assert np.allclose(rstd.cpu().numpy(), rs, rtol=1e-4)
    assert_close(to_np(dxo), dx_ref, TOL[dtype])
    assert_close(dg.cpu().numpy() - 0.25, dg_ref, 1e-5)
    assert_close(dbb.cpu().numpy() + 0.5, db_ref, 1e-5)


ATTN_CASES = [  # (dtype, b, s, heads, d)
    ("f32", 2, 128, 4, 64),
    ("f32", 1, 70, 2, 128),
    ("bf16", 2, 200, 3, 64),
    ("bf16", 1, 300, 2, 128),
    ("bf16", 1, 1, 2, 128),
    ("bf16", 3, 33, 1, 64),
]


# head dim 128: grids of 256 to 511 blocks of 128 rows take the forward with
# the key tiles split in two parts per workgroup, smaller grids the same with
# 64 rows per workgroup, at least 512 blocks the forward without splits; the
# backward fuses dK/dV and dQ below 257 and above 1023 blocks; ragged lengths
# throughout
ATTN_BIG_CASES = [("bf16", 2, 130, 128, 128), ("bf16", 2, 520, 52, 128), ("bf16", 1, 1000, 40, 128),
                  ("bf16", 1, 1500, 4, 128), ("bf16", 1, 2048, 4, 128), ("bf16", 3, 700, 2, 128),
                  ("bf16", 1, 2048, 16, 128), ("bf16", 1, 1100, 30, 128), ("bf16", 1, 1950, 16, 128),
                  ("bf16", 2, 1024, 16, 128)]


@pytest.mark.parametrize("dtype,b,s,nh,d", ATTN_CASES + ATTN_BIG_CASES)
def test_attention_fwd(dtype, b, s, nh, d):
    import torch
    h = nh * d
    qkv = _t(51, (b * s, 3 * h), dtype)
    o_ref, lse_ref = ora.causal_attention(qkv.astype(np.float64), b, s, nh)
    dq = to_dev(qkv, dtype)
    o = torch.full((b * s, h), float("nan"), device="cuda").to(dq.dtype)
    lse = torch.full((b, nh, s), float("nan"), device="cuda")
    T.op_attention_fwd(DT[dtype], b, s, nh, d, dq, o, lse)
    torch.cuda.synchronize()
    assert_close(to_np(o), o_ref, (2e-5 if dtype == "f32" else 1e-2))
    assert np.abs(lse.cpu().numpy() - lse_ref).max() < (1e-4 if dtype == "f32" else 2e-2)


@pytest.mark.parametrize("dtype,b,s,nh,d", ATTN_CASES + ATTN_BIG_CASES)
def test_attention_bwd(dtype, b, s, nh, d):
    import torch
    h = nh * d
    qkv = _t(61, (b * s, 3 * h), dtype)
    do = _t(62, (b * s, h), dtype)
    o_ref, lse_ref = ora.causal_attention(qkv.astype(np.float64), b, s, nh)
    o_st = _round(o_ref, dtype)
    dqkv_ref = ora.causal_attention_backward(qkv.astype(np.float64), o_st, lse_ref, do.astype(np.float64), b, s, nh)
    dq = to_dev(qkv, dtype)
    dO = to_dev(do, dtype)
    dOut = to_dev(o_st, dtype)
    dlse = torch.from_numpy(lse_ref.astype(np.float32)).cuda()
    dqkv = torch.full((b * s, 3 * h), float("nan"), device="cuda").to(dq.dtype)
    ws = torch.empty(T.op_workspace_bytes(T.WS_ATTN_BWD, b * s, nh) // 4, device="cuda")
    T.op_attention_bwd(DT[dtype], b, s, nh, d, dq, dOut, dlse, dO, dqkv, ws)
    torch.cuda.synchronize()
    got = to_np(dqkv)
    tol = 2e-5 if dtype == "f32" else 2e-2
    for name, sl in (("dq", slice(0, h)), ("dk", slice(h, 2 * h)), ("dv", slice(2 * h, 3 * h))):
        if np.linalg.norm(dqkv_ref[:, sl]) < 1e-12:
            # degenerate case (one key: dS = P (dP - D) vanishes exactly)
            assert np.abs(got[:, sl]).max() < 1e-5, name
        else:
            assert_close(got[:, sl], dqkv_ref[:, sl], tol, name)


def test_attention_deterministic_and_causal_bitwise():
    """Two runs agree bitwise; perturbing query/key/value at position t leaves
    every output row before t bitwise unchanged."""
    import torch
    b, s, nh, d = 1, 257, 2, 128
    h = nh * d
    qkv = _t(71, (b * s, 3 * h), "bf16")
    dq = to_dev(qkv, "bf16")
    outs = []
    for _ in range(2):
        o = torch.empty((b * s, h), device="cuda", dtype=torch.bfloat16)
        T.op_attention_fwd(T.TPS_BF16, b, s, nh, d, dq, o, None)
        outs.append(o)
    q2 = qkv.copy()
    t = 150
    q2[t] = _t(72, (3 * h,), "bf16")
    o2 = torch.empty((b * s, h), device="cuda", dtype=torch.bfloat16)
    T.op_attention_fwd(T.TPS_BF16, b, s, nh, d, to_dev(q2, "bf16"), o2, None)
    torch.cuda.synchronize()
    assert torch.equal(outs[0], outs[1])
    assert torch.equal(outs[0][:t], o2[:t])
    assert not torch.equal(outs[0][t], o2[t])


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_colsum_and_gelu(dtype):
    import torch
    rows, cols = 1000, 776
    x = _t(81, (rows, 2 * cols), dtype)
    out = torch.full((cols,), 1.5, device="cuda")
    ws = torch.empty(T.op_workspace_bytes(T.WS_COLSUM, rows, cols) // 4, device="cuda")
    dx = to_dev(x, dtype)
    T.op_colsum(DT[dtype], rows, cols, dx[:, cols:], 2 * cols, out, ws)
    u = _t(82, (rows * 3 + 5,), dtype, 3.0)
    g = torch.empty(u.size, device="cuda").to(dx.dtype)
    T.op_gelu(DT[dtype], u.size, to_dev(u, dtype), g)
    torch.cuda.synchronize()
    ref = x[:, cols:].astype(np.float64).sum(axis=0) + 1.5
    assert_close(out.cpu().numpy(), ref, 1e-6)
    assert_close(to_np(g), ora.gelu(u.astype(np.float64)), TOL[dtype])
