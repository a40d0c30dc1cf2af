"""Pins of the LLAMA-style layer oracle against facts that do not come from
the oracle itself:

* brute force: central finite differences of a whole two-layer stage, every
  parameter and stage-input coordinate, at a tiny shape with grouped
  key/value heads; the rotation written out as explicit 2 x 2 matrices in
  pure-Python loops;
* independent library routines: torch float64 ``rms_norm``, ``silu``,
  ``scaled_dot_product_attention(is_causal=True, enable_gqa=True)`` and
  ``linear`` with autograd, over a layer assembled in the test;
* reductions to other code: grouped attention with one query head per
  key/value head is the GPT oracle's multi-head attention, and with groups it
  equals multi-head attention over repeated keys and values (whose key/value
  gradients sum over the group);
* invariants: RMSNorm scale invariance and the null space of its backward,
  the rotation's norm preservation, relative-position property and inverse,
  causality, and keep / recompute / offload invariance;
* planted mistakes: each plausible slip, planted into a copy of the oracle on
  the CPU, breaks at least one of these pins.
"""
import math

import numpy as np
import pytest

from oracle import decoder_stage as gpt
from oracle import llama_stage as ora
from paper_2503_03182_amd import synth

TINY = dict(L=2, h=16, nh=4, nkv=2, f=24, s=6, b=2, M=2, eps=1e-5, base=10000.0)


def _params(L, h, nh, nkv, f, dtype="f32"):
    return [{k: v.astype(np.float64) for k, v in synth.llama_layer_params(l, h, nh, nkv, f, dtype).items()}
            for l in range(L)]


def _inputs(M, T, h):
    xs = [synth.stage_input(mb, T, h, "f32").astype(np.float64) for mb in range(M)]
    dys = [synth.output_grad(mb, T, h, "f32").astype(np.float64) for mb in range(M)]
    return xs, dys


def _stage(mod, c, params, xs, dys, **kw):
    return mod.run_stage(params, xs, dys, c["nh"], c["nkv"], c["b"], c["s"], eps=c["eps"], rope_base=c["base"], **kw)


# ---------------------------------------------------------------- brute force
def _fd_check(mod, c=TINY, tol=1e-6):
    L, h, nh, nkv, f, s, b, M, eps, base = (c[k] for k in ("L", "h", "nh", "nkv", "f", "s", "b", "M", "eps", "base"))
    T = b * s
    params = _params(L, h, nh, nkv, f)
    xs, G = _inputs(M, T, h)
    ref = _stage(mod, c, params, xs, G)

    def loss():
        total = 0.0
        for mb in range(M):
            hc = xs[mb]
            for l in range(L):
                hc, _ = mod.layer_forward(params[l], hc, b, s, nh, nkv, eps, base)
            total += float((hc * G[mb]).sum())
        return total

    step, worst = 1e-5, 0.0
    targets = [(params[l][n], ref["grads"][l][n]) for l in range(L) for n in ora.PARAM_NAMES]
    targets += [(xs[mb], ref["dxs"][mb]) for mb in range(M)]
    for arr, an in targets:
        flat = arr.reshape(-1)
        fd = np.zeros(flat.size)
        for i in range(flat.size):
            old = flat[i]
            flat[i] = old + step
            lp = loss()
            flat[i] = old - step
            lm = loss()
            flat[i] = old
            fd[i] = (lp - lm) / (2 * step)
        worst = max(worst, np.abs(fd - an.reshape(-1)).max() / max(np.abs(an).max(), 1e-3))
    return worst <= tol, worst


def test_finite_differences_every_coordinate():
    ok, worst = _fd_check(ora)
    assert ok, worst


def test_rope_against_explicit_rotations():
    b, s, nh, d, base = 2, 5, 3, 8, 500.0
    x = synth.uniform_tensor(11, (b * s, nh * d), 1.0, "f32").astype(np.float64)
    got = ora.rope(x, b, s, nh, d, base)
    for r in range(b * s):
        pos = r % s
        for n in range(nh):
            for i in range(d // 2):
                th = pos * base ** (-2.0 * i / d)
                R = [[math.cos(th), -math.sin(th)], [math.sin(th), math.cos(th)]]
                lo, hi = x[r, n * d + i], x[r, n * d + i + d // 2]
                assert abs(got[r, n * d + i] - (R[0][0] * lo + R[0][1] * hi)) < 1e-12
                assert abs(got[r, n * d + i + d // 2] - (R[1][0] * lo + R[1][1] * hi)) < 1e-12


def test_rope_invariants():
    b, s, nh, d, base = 1, 9, 2, 16, 10000.0
    x = synth.uniform_tensor(12, (b * s, nh * d), 1.0, "f32").astype(np.float64)
    y = ora.rope(x, b, s, nh, d, base)
    # each pair keeps its length; position 0 is the identity; inverse undoes it
    lo, hi = x.reshape(s, nh, 2, d // 2), y.reshape(s, nh, 2, d // 2)
    assert np.allclose((lo ** 2).sum(axis=2), (hi ** 2).sum(axis=2), atol=1e-12)
    assert np.array_equal(y[0], x[0])
    assert np.allclose(ora.rope(y, b, s, nh, d, base, inverse=True), x, atol=1e-12)
    # relative position: q at m and k at n interact through m - n only
    q = np.tile(x[:1, :d], (s, 1))
    k = np.tile(x[1:2, :d], (s, 1))
    rq, rk = ora.rope(q, 1, s, 1, d, base), ora.rope(k, 1, s, 1, d, base)
    for delta in range(0, 4):
        dots = [rq[m] @ rk[m - delta] for m in range(delta, s)]
        assert np.allclose(dots, dots[0], atol=1e-12), delta


# ------------------------------------------------------ independent libraries
def _torch_layer(p, x, c):
    import torch
    import torch.nn.functional as F
    b, s, nh, nkv, eps, base = c["b"], c["s"], c["nh"], c["nkv"], c["eps"], c["base"]
    h = x.shape[1]
    d = h // nh
    a = F.rms_norm(x, (h,), p["g1"], eps)
    qkv = F.linear(a, p["w_qkv"])
    q, k, v = qkv.split([nh * d, nkv * d, nkv * d], dim=1)

    def rot(t, heads):
        t = t.view(b, s, heads, d)
        pos = torch.arange(s, dtype=torch.float64)[:, None]
        inv = base ** (-2.0 * torch.arange(d // 2, dtype=torch.float64) / d)
        ang = (pos * inv)[None, :, None, :]
        lo, hi = t[..., :d // 2], t[..., d // 2:]
        return torch.cat([lo * ang.cos() - hi * ang.sin(), hi * ang.cos() + lo * ang.sin()], -1)

    qh = rot(q, nh).transpose(1, 2)
    kh = rot(k, nkv).transpose(1, 2)
    vh = v.reshape(b, s, nkv, d).transpose(1, 2)
    o = F.scaled_dot_product_attention(qh, kh, vh, is_causal=True, enable_gqa=True)
    o = o.transpose(1, 2).reshape(b * s, h)
    x1 = x + F.linear(o, p["w_o"])
    cc = F.rms_norm(x1, (h,), p["g2"], eps)
    u = F.linear(cc, p["w_1"])
    f = u.shape[1] // 2
    g = F.silu(u[:, :f]) * u[:, f:]
    return x1 + F.linear(g, p["w_2"])


def test_layer_against_torch_autograd():
    import torch
    c = dict(TINY, h=64, nh=4, nkv=2, f=96, s=7)
    h, nh, nkv, f, b, s = c["h"], c["nh"], c["nkv"], c["f"], c["b"], c["s"]
    p = _params(1, h, nh, nkv, f)[0]
    x = synth.stage_input(0, b * s, h, "f32").astype(np.float64)
    dy = synth.output_grad(0, b * s, h, "f32").astype(np.float64)
    y, sv = ora.layer_forward(p, x, b, s, nh, nkv, c["eps"], c["base"])
    dx, gr = ora.layer_backward(p, sv, dy, b, s, nh, nkv, c["base"])
    tp = {k: torch.tensor(v, requires_grad=True) for k, v in p.items()}
    tx = torch.tensor(x, requires_grad=True)
    ty = _torch_layer(tp, tx, c)
    ty.backward(torch.tensor(dy))
    assert np.allclose(y, ty.detach().numpy(), rtol=1e-11, atol=1e-11)
    assert np.allclose(dx, tx.grad.numpy(), rtol=1e-10, atol=1e-11)
    for k in ora.PARAM_NAMES:
        assert np.allclose(gr[k], tp[k].grad.numpy(), rtol=1e-10, atol=1e-11), k


def test_rms_norm_against_torch():
    import torch
    import torch.nn.functional as F
    z = synth.uniform_tensor(21, (9, 40), 2.0, "f32").astype(np.float64)
    gmm = 1.0 + synth.uniform_tensor(22, (40,), 0.1, "f32").astype(np.float64)
    dout = synth.uniform_tensor(23, (9, 40), 1.0, "f32").astype(np.float64)
    out, rstd = ora.rms_norm(z, gmm, 1e-5)
    dz, dg = ora.rms_norm_backward(dout, z, rstd, gmm)
    tz, tg = torch.tensor(z, requires_grad=True), torch.tensor(gmm, requires_grad=True)
    to = F.rms_norm(tz, (40,), tg, 1e-5)
    to.backward(torch.tensor(dout))
    assert np.allclose(out, to.detach().numpy(), rtol=1e-12)
    assert np.allclose(dz, tz.grad.numpy(), rtol=1e-10, atol=1e-12)
    assert np.allclose(dg, tg.grad.numpy(), rtol=1e-10, atol=1e-12)


def test_swiglu_against_torch():
    import torch
    import torch.nn.functional as F
    u = synth.uniform_tensor(31, (5, 2 * 12), 3.0, "f32").astype(np.float64)
    dg = synth.uniform_tensor(32, (5, 12), 1.0, "f32").astype(np.float64)
    tu = torch.tensor(u, requires_grad=True)
    tg = F.silu(tu[:, :12]) * tu[:, 12:]
    tg.backward(torch.tensor(dg))
    assert np.allclose(ora.swiglu(u), tg.detach().numpy(), rtol=1e-12)
    assert np.allclose(ora.swiglu_backward(dg, u), tu.grad.numpy(), rtol=1e-11, atol=1e-13)


# ------------------------------------------------------------------ reductions
def test_gqa_reduces_to_multi_head():
    b, s, nh, d = 2, 7, 4, 8
    qkv = synth.uniform_tensor(41, (b * s, 3 * nh * d), 1.0, "f32").astype(np.float64)
    do = synth.uniform_tensor(42, (b * s, nh * d), 1.0, "f32").astype(np.float64)
    o, lse = ora.gqa_attention(qkv, b, s, nh, nh)
    o2, lse2 = gpt.causal_attention(qkv, b, s, nh)
    assert np.allclose(o, o2, atol=1e-13) and np.allclose(lse, lse2, atol=1e-13)
    d1 = ora.gqa_attention_backward(qkv, o, lse, do, b, s, nh, nh)
    d2 = gpt.causal_attention_backward(qkv, o2, lse2, do, b, s, nh)
    assert np.allclose(d1, d2, atol=1e-12)


def test_grouped_heads_equal_repeated_keys_and_values():
    b, s, nh, nkv, d = 2, 6, 6, 2, 8
    grp = nh // nkv
    H, HK = nh * d, nkv * d
    qkv = synth.uniform_tensor(43, (b * s, H + 2 * HK), 1.0, "f32").astype(np.float64)
    do = synth.uniform_tensor(44, (b * s, H), 1.0, "f32").astype(np.float64)
    k, v = qkv[:, H:H + HK], qkv[:, H + HK:]
    rep = lambda t: np.concatenate([t[:, (n // grp) * d:(n // grp + 1) * d] for n in range(nh)], axis=1)
    full = np.concatenate([qkv[:, :H], rep(k), rep(v)], axis=1)
    o, lse = ora.gqa_attention(qkv, b, s, nh, nkv)
    o2, lse2 = gpt.causal_attention(full, b, s, nh)
    assert np.allclose(o, o2, atol=1e-13) and np.allclose(lse, lse2, atol=1e-13)
    dg = ora.gqa_attention_backward(qkv, o, lse, do, b, s, nh, nkv)
    df = gpt.causal_attention_backward(full, o2, lse2, do, b, s, nh)
    assert np.allclose(dg[:, :H], df[:, :H], atol=1e-12)
    def fold(t):
        return np.concatenate([sum(t[:, (kv * grp + j) * d:(kv * grp + j + 1) * d] for j in range(grp))
                               for kv in range(nkv)], axis=1)
    assert np.allclose(dg[:, H:H + HK], fold(df[:, H:2 * H]), atol=1e-12)
    assert np.allclose(dg[:, H + HK:], fold(df[:, 2 * H:]), atol=1e-12)


def test_gqa_against_torch_sdpa():
    import torch
    import torch.nn.functional as F
    b, s, nh, nkv, d = 2, 9, 8, 2, 16
    H, HK = nh * d, nkv * d
    qkv = synth.uniform_tensor(45, (b * s, H + 2 * HK), 1.0, "f32").astype(np.float64)
    o, _ = ora.gqa_attention(qkv, b, s, nh, nkv)
    t = torch.tensor(qkv)
    q = t[:, :H].view(b, s, nh, d).transpose(1, 2)
    k = t[:, H:H + HK].reshape(b, s, nkv, d).transpose(1, 2)
    v = t[:, H + HK:].reshape(b, s, nkv, d).transpose(1, 2)
    ref = F.scaled_dot_product_attention(q, k, v, is_causal=True, enable_gqa=True).transpose(1, 2).reshape(b * s, H)
    assert np.allclose(o, ref.numpy(), atol=1e-13)


# ------------------------------------------------------------------ invariants
def test_rms_norm_scale_invariance_and_null_space():
    z = synth.uniform_tensor(51, (6, 32), 1.5, "f32").astype(np.float64)
    gmm = 1.0 + synth.uniform_tensor(52, (32,), 0.1, "f32").astype(np.float64)
    dout = synth.uniform_tensor(53, (6, 32), 1.0, "f32").astype(np.float64)
    out, rstd = ora.rms_norm(z, gmm, 0.0)
    assert np.allclose(ora.rms_norm(3.7 * z, gmm, 0.0)[0], out, atol=1e-13)
    assert np.allclose(((out / gmm) ** 2).mean(axis=1), 1.0, atol=1e-13)
    dz, _ = ora.rms_norm_backward(dout, z, rstd, gmm)
    # the output does not change along z itself, so the gradient is orthogonal to it
    assert np.allclose((dz * z).sum(axis=1), 0.0, atol=1e-12)


def test_causality_bitwise():
    c = TINY
    p = _params(1, c["h"], c["nh"], c["nkv"], c["f"])[0]
    x = synth.stage_input(0, c["b"] * c["s"], c["h"], "f32").astype(np.float64)
    y, _ = ora.layer_forward(p, x, c["b"], c["s"], c["nh"], c["nkv"], c["eps"], c["base"])
    x2 = x.copy()
    x2[c["s"] - 1] += 1.0                    # last position of sequence 0
    y2, _ = ora.layer_forward(p, x2, c["b"], c["s"], c["nh"], c["nkv"], c["eps"], c["base"])
    assert np.array_equal(y[:c["s"] - 1], y2[:c["s"] - 1])
    assert np.array_equal(y[c["s"]:], y2[c["s"]:])
    assert not np.array_equal(y[c["s"] - 1], y2[c["s"] - 1])


@pytest.mark.parametrize("which", ["recompute_all", "layer_inputs", "offload_all"])
def test_policy_invariance_bitwise(which):
    c = TINY
    L, M = c["L"], c["M"]
    params = _params(L, c["h"], c["nh"], c["nkv"], c["f"])
    xs, dys = _inputs(M, c["b"] * c["s"], c["h"])
    keep = _stage(ora, c, params, xs, dys)
    if which == "recompute_all":
        pol = [{t: (0 if (l == 0 and t == "x") else 1) for t in ora.TENSORS} for l in range(L)]
        out = _stage(ora, c, params, xs, dys, policy=pol)
    elif which == "layer_inputs":
        pol = [{t: (0 if t == "x" else 1) for t in ora.TENSORS} for l in range(L)]
        out = _stage(ora, c, params, xs, dys, policy=pol)
    else:
        pol = [{t: 2 for t in ora.TENSORS} for l in range(L)]
        out = _stage(ora, c, params, xs, dys, policy=pol, offload_mbs=range(M))
    for a, b_ in zip(keep["ys"] + keep["dxs"], out["ys"] + out["dxs"]):
        assert np.array_equal(a, b_)
    for gk, go in zip(keep["grads"], out["grads"]):
        for n in ora.PARAM_NAMES:
            assert np.array_equal(gk[n], go[n])


def test_unit_flops_by_enumeration():
    T, h, nh, nkv, f, b, s = 12, 64, 8, 2, 96, 2, 6
    d = h // nh
    mats = [((nh + 2 * nkv) * d, h), (h, h), (2 * f, h), (h, f)]
    gemm = sum(2 * T * m * n for m, n in mats)
    attn = sum(2 * 2 * d * (i + 1) for _ in range(b) for _ in range(nh) for i in range(s))
    got = ora.unit_flops(T, h, nh, nkv, f, b, s)
    assert got["fwd_gemm"] == gemm and got["fwd_attn"] == attn and got["bwd"] == 2 * (gemm + attn)


# ------------------------------------------------------------ planted mistakes
MUTATIONS = {
    # the gradient turned back the wrong way
    "rope_backward_same_direction": ("inverse=True)", "inverse=False)"),
    # key/value head n % n_kv instead of n // (n_heads / n_kv), in both passes
    "kv_head_modulo": ("kv = n // grp", "kv = n % n_kv"),
    # SiLU' without the gate (1 - sigma) term
    "swiglu_dropped_term": ("sg * (1.0 + gate * (1.0 - sg))", "sg"),
    # RMSNorm backward without the projection onto zhat
    "rms_missing_projection": ("(dzhat - zhat * m[:, None])", "dzhat"),
    # frequencies base^(-i/d) instead of base^(-2i/d), in both passes
    "rope_frequency": ("-2.0 * np.arange(d // 2", "-1.0 * np.arange(d // 2"),
    # a key/value head keeps only its last query head's gradient
    "gqa_dk_overwritten": ("dqkv[rows, kc] += ", "dqkv[rows, kc] = "),
    # eps outside the square root
    "rms_eps_outside": ("np.sqrt((z * z).mean(axis=1) + eps)", "(np.sqrt((z * z).mean(axis=1)) + eps)"),
    # interleaved pairs (2i, 2i + 1) instead of (i, i + d/2), in both passes
    "rope_interleaved": ("lo = x[rows, n * d:n * d + half]\n            hi = x[rows, n * d + half:(n + 1) * d]",
                         "lo = x[rows, n * d:(n + 1) * d:2]\n            hi = x[rows, n * d + 1:(n + 1) * d:2]"),
}


def _mutant(name):
    """A copy of the oracle module with one plausible slip in its source."""
    import types
    old, new = MUTATIONS[name]
    src = open(ora.__file__).read()
    assert src.count(old) >= 1, name
    src = src.replace(old, new)
    if name == "rope_interleaved":
        src = src.replace("out[rows, n * d:n * d + half] = lo * cos - hi * sin",
                          "out[rows, n * d:(n + 1) * d:2] = lo * cos - hi * sin")
        src = src.replace("out[rows, n * d + half:(n + 1) * d] = hi * cos + lo * sin",
                          "out[rows, n * d + 1:(n + 1) * d:2] = hi * cos + lo * sin")
    m = types.ModuleType("llama_mutant_" + name)
    m.__dict__["__package__"] = "oracle"
    exec(compile(src, ora.__file__, "exec"), m.__dict__)
    return m


def _torch_pin(m):
    c = dict(TINY, h=64, nh=4, nkv=2, f=96, s=7)
    h, nh, nkv, f, b, s = c["h"], c["nh"], c["nkv"], c["f"], c["b"], c["s"]
    import torch
    p = _params(1, h, nh, nkv, f)[0]
    x = synth.stage_input(0, b * s, h, "f32").astype(np.float64)
    dy = synth.output_grad(0, b * s, h, "f32").astype(np.float64)
    y, sv = m.layer_forward(p, x, b, s, nh, nkv, c["eps"], c["base"])
    dx, gr = m.layer_backward(p, sv, dy, b, s, nh, nkv, c["base"])
    tp = {k: torch.tensor(v, requires_grad=True) for k, v in p.items()}
    tx = torch.tensor(x, requires_grad=True)
    _torch_layer(tp, tx, c).backward(torch.tensor(dy))
    ty = _torch_layer({k: v.detach() for k, v in tp.items()}, tx.detach(), c).numpy()
    ok = np.allclose(y, ty, rtol=1e-11, atol=1e-11) and np.allclose(dx, tx.grad.numpy(), rtol=1e-10, atol=1e-11)
    return ok and all(np.allclose(gr[k], tp[k].grad.numpy(), rtol=1e-10, atol=1e-11) for k in ora.PARAM_NAMES)


def test_unmutated_copy_passes_the_pins():
    import types
    src = open(ora.__file__).read()
    m = types.ModuleType("llama_copy")
    m.__dict__["__package__"] = "oracle"
    exec(compile(src, ora.__file__, "exec"), m.__dict__)
    assert _fd_check(m, dict(TINY, L=1, M=1))[0]
    assert _torch_pin(m)


@pytest.mark.parametrize("name", list(MUTATIONS))
def test_planted_mistakes_are_caught(name):
    m = _mutant(name)
    caught = not _torch_pin(m) or not _fd_check(m, dict(TINY, L=1, M=1))[0]
    assert caught, name
