"""LLAMA-style layers on the GPU through the C ABI, against the float64
oracle (oracle/llama_stage.py): each new kernel (RMSNorm forward and
backward, rotary embedding and its inverse, SwiGLU forward and backward,
grouped-query attention forward and backward) at ragged multi-tile sizes;
whole stages at small sizes under every policy kind and both call styles,
with resident and streamed weights; one full-width layer at the LLAMA2-70B
widths in the launch configuration bench.py times.  The bar: rel-L2 <= 2e-2
(bf16) or 1e-4 (f32) per tensor plus the per-tile bound of
stage_harness.tile_excess; bit-exact between arrangements that make the
same decisions."""
import dataclasses

import numpy as np
import pytest

from oracle import llama_stage as ora
from paper_2503_03182_amd import configs as W
from paper_2503_03182_amd import synth
from paper_2503_03182_amd import tpstage as T
from stage_harness import assert_close, bit_equal, compare, run_gpu, run_oracle, to_dev, to_np

pytestmark = pytest.mark.gpu
BF16_TOL = 2e-2


def _dev(a, dtype="bf16"):
    return to_dev(a, dtype)


def _ws(kind, rows, cols):
    import torch
    return torch.empty(T.op_workspace_bytes(kind, rows, cols) // 4 + 64, dtype=torch.float32, device="cuda")


# ------------------------------------------------------------------ kernels
@pytest.mark.parametrize("dtype,rows,cols", [("bf16", 300, 512), ("bf16", 257, 2056), ("bf16", 64, 8192),
                                             ("f32", 130, 1000)])
def test_rmsnorm_matches_oracle(dtype, rows, cols):
    import torch
    tol = BF16_TOL if dtype == "bf16" else 1e-4
    x = synth.uniform_tensor(101, (rows, cols), 1.5, dtype)
    gmm = synth.round_to_storage(1.0 + synth.uniform_tensor(102, (cols,), 0.1, "f32"), dtype)
    dout = synth.uniform_tensor(103, (rows, cols), 1.0, dtype)
    res = synth.uniform_tensor(104, (rows, cols), 1.0, dtype)
    X, G, DO, R = _dev(x, dtype), _dev(gmm, dtype), _dev(dout, dtype), _dev(res, dtype)
    out = torch.empty_like(X)
    rstd = torch.empty(rows, dtype=torch.float32, device="cuda")
    tc = T.TPS_BF16 if dtype == "bf16" else T.TPS_F32
    T.op_rmsnorm_fwd(tc, rows, cols, X, G, 1e-5, out, rstd)
    dx = torch.empty_like(X)
    dg = torch.zeros(cols, dtype=torch.float32, device="cuda")
    T.op_rmsnorm_bwd(tc, rows, cols, DO, X, rstd, G, R, dx, dg, _ws(T.WS_COLSUM, rows, cols))
    torch.cuda.synchronize()
    ref, rs = ora.rms_norm(x.astype(np.float64), gmm.astype(np.float64), 1e-5)
    rdx, rdg = ora.rms_norm_backward(dout.astype(np.float64), x.astype(np.float64), rs, gmm.astype(np.float64))
    assert_close(to_np(out), ref, tol, "out")
    assert_close(rstd.cpu().numpy(), rs, 1e-5, "rstd")
    assert_close(to_np(dx), rdx + res.astype(np.float64), tol, "dx")
    assert_close(dg.cpu().numpy(), rdg, tol if dtype == "bf16" else 1e-4, "dgamma")


@pytest.mark.parametrize("s,n_rot,extra", [(300, 12, 4), (4096, 2, 2), (17, 1, 0)])
def test_rope_matches_oracle(s, n_rot, extra):
    import torch
    b, d, base = 2, 128, 10000.0
    ld = (n_rot + extra) * d
    x = synth.uniform_tensor(111, (b * s, ld), 1.0, "bf16")
    X = _dev(x)
    table = torch.empty(s * d, dtype=torch.float32, device="cuda")
    T.op_rope(X, ld, b * s, s, n_rot, d, base, False, table)
    torch.cuda.synchronize()
    got = to_np(X)
    ref = ora.rope(x[:, :n_rot * d].astype(np.float64), b, s, n_rot, d, base)
    assert_close(got[:, :n_rot * d], ref, 1e-2, "rotated")
    assert np.array_equal(got[:, n_rot * d:], x[:, n_rot * d:])      # other columns untouched
    # the inverse turns it back (up to bf16 rounding of both passes)
    T.op_rope(X, ld, b * s, s, n_rot, d, base, True, table)
    torch.cuda.synchronize()
    assert_close(to_np(X)[:, :n_rot * d], x[:, :n_rot * d], 1e-2, "round trip")
    inv = ora.rope(got[:, :n_rot * d], b, s, n_rot, d, base, inverse=True)
    assert_close(to_np(X)[:, :n_rot * d], inv, 1e-2, "inverse")


@pytest.mark.parametrize("rows,f", [(300, 1024), (33, 2056)])
def test_swiglu_matches_oracle(rows, f):
    import torch
    u = synth.uniform_tensor(121, (rows, 2 * f), 2.0, "bf16")
    dg = synth.uniform_tensor(122, (rows, f), 1.0, "bf16")
    U, DG = _dev(u), _dev(dg)
    g = torch.empty(rows, f, dtype=torch.bfloat16, device="cuda")
    du = torch.empty(rows, 2 * f, dtype=torch.bfloat16, device="cuda")
    T.op_swiglu_fwd(rows, f, U, g)
    T.op_swiglu_bwd(rows, f, DG, U, du)
    torch.cuda.synchronize()
    assert_close(to_np(g), ora.swiglu(u.astype(np.float64)), 1e-2, "g")
    assert_close(to_np(du), ora.swiglu_backward(dg.astype(np.float64), u.astype(np.float64)), 1e-2, "du")


@pytest.mark.parametrize("b,s,nh,nkv", [(2, 300, 8, 2), (1, 1000, 8, 1), (2, 129, 4, 4), (1, 2048, 16, 8),
                                        (1, 2048, 32, 4)])
def test_gqa_attention_matches_oracle(b, s, nh, nkv):
    import torch
    d = 128
    qw = (nh + 2 * nkv) * d
    qkv = synth.uniform_tensor(131, (b * s, qw), 1.0, "bf16")
    do = synth.uniform_tensor(132, (b * s, nh * d), 1.0, "bf16")
    Q, DO = _dev(qkv), _dev(do)
    o = torch.empty(b * s, nh * d, dtype=torch.bfloat16, device="cuda")
    lse = torch.empty(b * nh * s, dtype=torch.float32, device="cuda")
    T.op_attention_gqa_fwd(b, s, nh, nkv, Q, o, lse)
    dq = torch.empty_like(Q)
    kvws = torch.empty(b * s, 2 * nh * d, dtype=torch.bfloat16, device="cuda") if nkv < nh else None
    T.op_attention_gqa_bwd(b, s, nh, nkv, Q, o, lse, DO, dq, _ws(T.WS_ATTN_BWD, b * s, nh), kvws)
    torch.cuda.synchronize()
    q64 = qkv.astype(np.float64)
    ro, rl = ora.gqa_attention(q64, b, s, nh, nkv)
    assert_close(to_np(o), ro, BF16_TOL, "o")
    assert_close(lse.cpu().numpy().reshape(b, nh, s), rl, 1e-3, "lse")
    # the backward from the device's own (rounded) o, as the stage runs it
    rd = ora.gqa_attention_backward(q64, to_np(o), rl, do.astype(np.float64), b, s, nh, nkv)
    H, HK = nh * d, nkv * d
    got = to_np(dq)
    assert_close(got[:, :H], rd[:, :H], BF16_TOL, "dq")
    assert_close(got[:, H:H + HK], rd[:, H:H + HK], BF16_TOL, "dk")
    assert_close(got[:, H + HK:], rd[:, H + HK:], BF16_TOL, "dv")


# ------------------------------------------------------------------- stages
def _mid(**kw):
    base = dict(n_layers=3, hidden=512, n_heads=4, mlp=1024, seq=200, micro_batch=2, n_micro=3, dtype="bf16",
                arch=T.ARCH_LLAMA, n_kv_heads=2)
    base.update(kw)
    return T.StageConfig(**base)


def test_llama_stage_matches_oracle():
    for cfg in (_mid(policy=W.policy_selective(3)), _mid(n_kv_heads=1, seq=130), _mid(n_kv_heads=4)):
        gpu = run_gpu(cfg)
        ref = run_oracle(cfg)
        worst, bad = compare(gpu, ref, BF16_TOL)
        assert not bad, (cfg.n_kv_heads, bad)


def test_llama_bitexact_across_policies_orders_and_groups():
    L = 3
    order = [("F", 0), ("F", 1), ("B", 0), ("F", 2), ("B", 1), ("B", 2)]
    keep = run_gpu(_mid(ops=order))
    mixed = [{t: [T.KEEP, T.RECOMPUTE, T.OFFLOAD][(l + i) % 3] for i, t in enumerate(T.TENSORS)} for l in range(L)]
    mixed[0]["x"] = T.KEEP
    variants = {
        "selective": _mid(ops=order, policy=W.policy_selective(L)),
        "layer_inputs_segment": _mid(ops=order, policy=W.policy_layer_inputs(L), granularity=T.GRAN_SEGMENT),
        "layer_inputs_layer": _mid(ops=order, policy=W.policy_layer_inputs(L), granularity=T.GRAN_LAYER),
        "recompute_all": _mid(ops=order, policy=W.policy_all(L, T.RECOMPUTE)),
        "offload_all": _mid(ops=order, policy=W.policy_all(L, T.OFFLOAD), offload_mb_mask=0b111),
        "mixed": _mid(ops=order, policy=mixed, offload_mb_mask=0b101),
        "inline_wgrad": _mid(ops=order, wgrad_stream=T.WGRAD_INLINE),
    }
    for name, cfg in variants.items():
        assert bit_equal(keep, run_gpu(cfg)) == [], name
    grp = run_gpu(_mid(policy=W.policy_layer_inputs(L), granularity=T.GRAN_LAYER), group=True)
    assert bit_equal(keep, grp) == []


def test_llama_streamed_weights_match_oracle_and_resident():
    L = 4
    resident = run_gpu(_mid(n_layers=L, policy=W.policy_layer_inputs(L), granularity=T.GRAN_LAYER))
    cfg = _mid(n_layers=L, policy=W.policy_layer_inputs(L), granularity=T.GRAN_LAYER, weights=T.W_STREAM, window=2)
    ref = run_oracle(cfg)
    for group in (False, True):
        out = run_gpu(cfg, group=group)
        assert bit_equal(resident, out) == [], group
        worst, bad = compare(out, ref, BF16_TOL)
        assert not bad, (group, bad)


def test_llama_batched_group_weight_gradients():
    L = 4
    cfg = _mid(n_layers=L, policy=W.policy_layer_inputs(L), granularity=T.GRAN_LAYER, weights=T.W_STREAM, window=2)
    per_mb = run_gpu(cfg, group=True)
    bat = run_gpu(dataclasses.replace(cfg, group_wgrad=1), group=True)
    from stage_harness import rel_l2
    for mb in range(cfg.n_micro):
        assert np.array_equal(per_mb["ys"][mb], bat["ys"][mb]) and np.array_equal(per_mb["dxs"][mb], bat["dxs"][mb])
    for l in range(L):
        for k, v in per_mb["grads"][l].items():
            assert rel_l2(bat["grads"][l][k], v) <= 1e-5, (l, k)
    worst, bad = compare(bat, run_oracle(cfg), BF16_TOL)
    assert not bad, bad


def _device_params(cfg, seed):
    """Seeded device parameters and inputs (for self-comparisons at full
    widths, where drawing ~10^9 values on the host would dominate)."""
    import torch
    from stage_harness import param_shapes
    po, pb, go, gb = T.param_layout(cfg)
    shapes = param_shapes(cfg)
    gen = torch.Generator(device="cuda").manual_seed(seed)
    blocks = []
    for _ in range(cfg.n_layers):
        blk = torch.zeros(pb, dtype=torch.uint8, device="cuda")
        for i, name in enumerate(T.PARAMS):
            if name not in shapes:
                continue
            n = int(np.prod(shapes[name]))
            v = torch.randn(n, generator=gen, device="cuda") * 0.02
            if name in ("g1", "g2"):
                v += 1.0
            blk[po[i]:po[i] + 2 * n].view(torch.bfloat16).copy_(v.to(torch.bfloat16))
        blocks.append(blk)
    xs = [torch.randn(cfg.tokens, cfg.hidden, generator=gen, device="cuda").to(torch.bfloat16)
          for _ in range(cfg.n_micro)]
    dys = [torch.randn(cfg.tokens, cfg.hidden, generator=gen, device="cuda").to(torch.bfloat16)
           for _ in range(cfg.n_micro)]
    return blocks, xs, dys


def _run_dev(cfg, blocks, xs, dys, group):
    import torch
    from stage_harness import drive_iteration
    po, pb, go, gb = T.param_layout(cfg)
    if cfg.weights == T.W_STREAM:
        host = []
        for blk in blocks:
            hb = torch.empty(pb, dtype=torch.uint8, pin_memory=True)
            hb.copy_(blk)
            host.append(hb)
        blocks = host
        grads = [torch.zeros(gb, dtype=torch.uint8, pin_memory=True) for _ in range(cfg.n_layers)]
    else:
        grads = [torch.zeros(gb, dtype=torch.uint8, device="cuda") for _ in range(cfg.n_layers)]
    st = T.Stage(cfg, blocks, grads)
    Y = [torch.empty_like(x) for x in xs]
    DX = [torch.empty_like(x) for x in xs]
    torch.cuda.synchronize()
    drive_iteration(st, cfg, xs, dys, Y, DX, group=group)
    st.sync()
    out = dict(ys=[y.cpu() for y in Y], dxs=[d.cpu() for d in DX], grads=[g.cpu() for g in grads])
    st.close()
    return out


@pytest.mark.timeout(900)
def test_llama70b_width_streamed_bitexact_to_resident():
    """4 layers at the LLAMA2-70B widths (seq 4096, 2 micro-batches): weights
    and f32 gradients streamed through a window of 3 layers, as bench.py runs
    them, against the same stage with resident weights."""
    import torch
    cfg = dataclasses.replace(W.llama12_h8192_stream(), n_layers=4, n_micro=2)
    cfg.policy = cfg.policy[:4]
    print("LLAMA2-70B widths, 4 layers, 2 micro-batches: streamed", flush=True)
    blocks, xs, dys = _device_params(cfg, 7)
    a = _run_dev(cfg, blocks, xs, dys, group=True)
    print("resident", flush=True)
    b = _run_dev(dataclasses.replace(cfg, weights=T.W_RESIDENT), blocks, xs, dys, group=True)
    for k in ("ys", "dxs", "grads"):
        for u, v in zip(a[k], b[k]):
            assert torch.equal(u, v), k
    # per-micro-batch weight-gradient products: same outputs, gradients up to
    # the f32 summation order
    print("per-micro-batch weight gradients", flush=True)
    c = _run_dev(dataclasses.replace(cfg, group_wgrad=0), blocks, xs, dys, group=True)
    for k in ("ys", "dxs"):
        for u, v in zip(a[k], c[k]):
            assert torch.equal(u, v), k
    for l, (u, v) in enumerate(zip(a["grads"], c["grads"])):
        u32, v32 = u.view(torch.float32).double(), v.view(torch.float32).double()
        r = ((u32 - v32).norm() / v32.norm()).item()
        assert r <= 1e-5, (l, r)


@pytest.mark.timeout(1500)
def test_llama70b_one_streamed_layer_matches_oracle():
    """One full-width LLAMA2-70B layer (hidden 8192, 64 query and 8 key/value
    heads, SwiGLU MLP 28672, seq 4096) in the launch configuration of the
    LLAMA workload (weights streamed in, f32 gradients streamed out,
    layer-input recompute, group calls), one micro-batch, against the float64
    oracle."""
    cfg = dataclasses.replace(W.llama12_h8192_stream(), n_layers=1, n_micro=1, window=2)
    cfg.policy = cfg.policy[:1]
    print("LLAMA2-70B widths, one streamed layer: GPU run", flush=True)
    gpu = run_gpu(cfg, group=True)
    assert gpu["stats"]["h2d_bytes"] > 0 and gpu["stats"]["d2h_bytes"] > 0
    print("oracle run", flush=True)
    ref = run_oracle(cfg)
    worst, bad = compare(gpu, ref, BF16_TOL)
    print("worst rel-L2", max(worst.values()), flush=True)
    assert not bad, bad
