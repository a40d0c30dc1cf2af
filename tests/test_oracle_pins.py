"""Pins of the CPU oracle against facts that do not come from the oracle itself.

Each pin is chosen so that a plausible slip in the oracle (a dropped term, a
wrong sign or index, a transposed operand, a wrong scale or variance) breaks at
least one of them:

* brute force: central finite differences of the whole stage, every
  coordinate of every parameter and of the stage input, at a tiny shape;
* independent library routines: torch float64 ``layer_norm``, ``gelu`` (erf),
  ``scaled_dot_product_attention(is_causal=True)`` and ``linear`` with
  autograd, and ``math.erf``;
* closed forms: all-zero weight matrices, attention at s = 1 and with q = 0;
* invariants: LayerNorm moments and the null space of its backward,
  causality, batch separation, linearity in dy, micro-batch additivity and
  invariance under keep / recompute / offload.
"""

import math

import numpy as np
import pytest

from oracle import decoder_stage as ora
from paper_2503_03182_amd import synth

pytestmark = pytest.mark.filterwarnings("ignore::DeprecationWarning")


def _params(L, h, f, dtype="f32"):
    return [{k: v.astype(np.float64) for k, v in synth.layer_params(l, h, f, dtype).items()}
            for l in range(L)]


def _stage_inputs(M, T, h):
    xs = [synth.stage_input(mb, T, h, "f32").astype(np.float64) for mb in range(M)]
    dys = [synth.output_grad(mb, T, h, "f32").astype(np.float64) for mb in range(M)]
    return xs, dys


# ---------------------------------------------------------------- brute force
def test_finite_differences_every_coordinate():
    """Central differences of L = sum_mb sum(y_mb * G_mb) for every parameter
    coordinate and every stage-input coordinate (L=2, h=16, nh=2, f=64, s=8,
    b=2, M=2)."""
    L, h, nh, f, s, b, M, eps = 2, 16, 2, 64, 8, 2, 2, 1e-5
    T = b * s
    params = _params(L, h, f)
    xs, G = _stage_inputs(M, T, h)
    ref = ora.run_stage(params, xs, G, nh, b, s, eps)

    def loss(ps, xin):
        total = 0.0
        for mb in range(M):
            hcur = xin[mb]
            for l in range(L):
                hcur, _ = ora.layer_forward(ps[l], hcur, b, s, nh, eps)
            total += float((hcur * G[mb]).sum())
        return total

    step = 1e-5
    for l in range(L):
        for name in ora.PARAM_NAMES:
            p = params[l][name]
            fd = np.zeros_like(p)
            flat = p.reshape(-1)
            for i in range(flat.size):
                old = flat[i]
                flat[i] = old + step
                lp = loss(params, xs)
                flat[i] = old - step
                lm = loss(params, xs)
                flat[i] = old
                fd.reshape(-1)[i] = (lp - lm) / (2 * step)
            an = ref["grads"][l][name]
            err = np.abs(fd - an).max() / max(np.abs(an).max(), 1e-3)
            assert err < 1e-6, (l, name, err)
    for mb in range(M):
        x = xs[mb]
        fd = np.zeros_like(x)
        for i in range(x.size):
            old = x.reshape(-1)[i]
            x.reshape(-1)[i] = old + step
            lp = loss(params, xs)
            x.reshape(-1)[i] = old - step
            lm = loss(params, xs)
            x.reshape(-1)[i] = old
            fd.reshape(-1)[i] = (lp - lm) / (2 * step)
        an = ref["dxs"][mb]
        err = np.abs(fd - an).max() / np.abs(an).max()
        assert err < 1e-6, (mb, err)


def test_attention_brute_force_loops():
    """Pure-Python loops over (i, j) against the vectorised attention."""
    b, s, nh, d = 2, 5, 2, 3
    h = nh * d
    rng = np.random.default_rng(7)
    qkv = rng.standard_normal((b * s, 3 * h))
    o, lse = ora.causal_attention(qkv, b, s, nh)
    for ib in range(b):
        for n in range(nh):
            for i in range(s):
                r = ib * s + i
                q = qkv[r, n * d:(n + 1) * d]
                scores = []
                for j in range(i + 1):
                    k = qkv[ib * s + j, h + n * d:h + (n + 1) * d]
                    scores.append(sum(q[t] * k[t] for t in range(d)) / math.sqrt(d))
                mx = max(scores)
                z = sum(math.exp(v - mx) for v in scores)
                assert abs(lse[ib, n, i] - (mx + math.log(z))) < 1e-12
                for t in range(d):
                    acc = 0.0
                    for j in range(i + 1):
                        acc += math.exp(scores[j] - mx) / z * qkv[ib * s + j, 2 * h + n * d + t]
                    assert abs(o[r, n * d + t] - acc) < 1e-12


# ------------------------------------------------- independent library routine
def test_against_torch_library_autograd():
    torch = pytest.importorskip("torch")
    F = torch.nn.functional
    L, h, nh, f, s, b, M, eps = 2, 64, 4, 256, 32, 2, 2, 1e-5
    T = b * s
    params = _params(L, h, f)
    xs, dys = _stage_inputs(M, T, h)
    ref = ora.run_stage(params, xs, dys, nh, b, s, eps)

    tp = [{k: torch.tensor(v, dtype=torch.float64, requires_grad=True) for k, v in p.items()}
          for p in params]
    d = h // nh
    for mb in range(M):
        x = torch.tensor(xs[mb], requires_grad=True)
        hcur = x
        for l in range(L):
            p = tp[l]
            a = F.layer_norm(hcur, (h,), p["g1"], p["be1"], eps)
            qkv = F.linear(a, p["w_qkv"], p["b_qkv"])
            q, k, v = qkv.split(h, dim=1)

            def heads(t):
                return t.reshape(b, s, nh, d).permute(0, 2, 1, 3)
            o = F.scaled_dot_product_attention(heads(q), heads(k), heads(v), is_causal=True)
            o = o.permute(0, 2, 1, 3).reshape(T, h)
            x1 = hcur + F.linear(o, p["w_o"], p["b_o"])
            c = F.layer_norm(x1, (h,), p["g2"], p["be2"], eps)
            g = F.gelu(F.linear(c, p["w_1"], p["b_1"]))
            hcur = x1 + F.linear(g, p["w_2"], p["b_2"])
        rel = np.linalg.norm(hcur.detach().numpy() - ref["ys"][mb]) / np.linalg.norm(ref["ys"][mb])
        assert rel < 1e-12, rel
        (hcur * torch.tensor(dys[mb])).sum().backward()
        rel = np.linalg.norm(x.grad.numpy() - ref["dxs"][mb]) / np.linalg.norm(ref["dxs"][mb])
        assert rel < 1e-12, rel
    for l in range(L):
        for name in ora.PARAM_NAMES:
            tg = tp[l][name].grad.numpy()
            og = ref["grads"][l][name]
            rel = np.linalg.norm(tg - og) / np.linalg.norm(og)
            assert rel < 1e-12, (l, name, rel)


def test_gelu_against_math_erf():
    us = np.array([-6.0, -3.0, -1.5, -1.0, -0.25, 0.0, 1e-3, 0.5, 1.0, 2.0, 4.0, 8.0])
    want = np.array([0.5 * u * (1.0 + math.erf(u / math.sqrt(2.0))) for u in us])
    assert np.allclose(ora.gelu(us), want, rtol=1e-15, atol=1e-300)
    assert ora.gelu(np.array([0.0]))[0] == 0.0
    assert ora.gelu_grad(np.array([0.0]))[0] == 0.5
    assert abs(ora.gelu(np.array([10.0]))[0] - 10.0) < 1e-12
    step = 1e-6
    fd = (ora.gelu(us + step) - ora.gelu(us - step)) / (2 * step)
    assert np.allclose(ora.gelu_grad(us), fd, atol=1e-8)


# ------------------------------------------------------------- closed forms
def test_zero_weight_matrices_closed_form():
    L, h, nh, f, s, b, M, eps = 2, 32, 4, 128, 8, 2, 3, 1e-5
    T = b * s
    params = _params(L, h, f)
    for p in params:
        for name in ("w_qkv", "w_o", "w_1", "w_2"):
            p[name][:] = 0.0
    xs, dys = _stage_inputs(M, T, h)
    out = ora.run_stage(params, xs, dys, nh, b, s, eps)
    shift = sum(p["b_o"] + p["b_2"] for p in params)
    colsum = sum(dy.sum(axis=0) for dy in dys)
    for mb in range(M):
        assert np.allclose(out["ys"][mb], xs[mb] + shift[None, :], rtol=0, atol=1e-13)
        assert np.allclose(out["dxs"][mb], dys[mb], rtol=0, atol=1e-13)
    for l, p in enumerate(params):
        gr = out["grads"][l]
        b_v = p["b_qkv"][2 * h:]
        assert np.allclose(gr["w_o"], np.outer(colsum, b_v), atol=1e-12)
        assert np.allclose(gr["w_2"], np.outer(colsum, ora.gelu(p["b_1"])), atol=1e-12)
        assert np.allclose(gr["b_o"], colsum, atol=1e-12)
        assert np.allclose(gr["b_2"], colsum, atol=1e-12)
        for name in ("w_qkv", "b_qkv", "w_1", "b_1", "g1", "be1", "g2", "be2"):
            assert np.abs(gr[name]).max() == 0.0, name


def test_attention_single_position():
    b, s, nh, d = 3, 1, 2, 4
    h = nh * d
    qkv = np.random.default_rng(1).standard_normal((b * s, 3 * h))
    o, lse = ora.causal_attention(qkv, b, s, nh)
    assert np.array_equal(o, qkv[:, 2 * h:])
    for ib in range(b):
        for n in range(nh):
            q = qkv[ib, n * d:(n + 1) * d]
            k = qkv[ib, h + n * d:h + (n + 1) * d]
            assert abs(lse[ib, n, 0] - q @ k / math.sqrt(d)) < 1e-14


def test_attention_zero_queries_is_causal_mean():
    b, s, nh, d = 2, 7, 3, 4
    h = nh * d
    qkv = np.random.default_rng(2).standard_normal((b * s, 3 * h))
    qkv[:, :h] = 0.0
    o, lse = ora.causal_attention(qkv, b, s, nh)
    for ib in range(b):
        v = qkv[ib * s:(ib + 1) * s, 2 * h:]
        want = np.cumsum(v, axis=0) / np.arange(1, s + 1)[:, None]
        assert np.allclose(o[ib * s:(ib + 1) * s], want, atol=1e-14)
        assert np.allclose(lse[ib], np.log(np.arange(1, s + 1))[None, :], atol=1e-14)


# --------------------------------------------------------------- invariants
def test_layer_norm_moments_and_backward_null_space():
    rng = np.random.default_rng(3)
    z = rng.standard_normal((9, 40)) * 3.0 + 1.5
    gamma = 1.0 + 0.1 * rng.standard_normal(40)
    beta = 0.1 * rng.standard_normal(40)
    eps = 1e-5
    out, mean, rstd = ora.layer_norm(z, gamma, beta, eps)
    zhat = (out - beta) / gamma
    var = z.var(axis=1)
    assert np.allclose(zhat.mean(axis=1), 0.0, atol=1e-13)
    assert np.allclose((zhat ** 2).mean(axis=1), var / (var + eps), rtol=1e-12)
    assert np.allclose(mean, z.mean(axis=1), rtol=1e-14)
    # with eps = 0 the input gradient is orthogonal to 1 and to zhat
    out0, mean0, rstd0 = ora.layer_norm(z, gamma, beta, 0.0)
    dz, dg, db = ora.layer_norm_backward(rng.standard_normal(z.shape), z, mean0, rstd0, gamma)
    zhat0 = (z - mean0[:, None]) * rstd0[:, None]
    assert np.allclose(dz.sum(axis=1), 0.0, atol=1e-12)
    assert np.allclose((dz * zhat0).sum(axis=1), 0.0, atol=1e-12)


def test_causality_bitwise():
    L, h, nh, f, s, b, eps = 2, 32, 4, 128, 12, 2, 1e-5
    T = b * s
    params = _params(L, h, f)
    x = synth.stage_input(0, T, h, "f32").astype(np.float64)
    t = 7

    def fwd(xin):
        hc = xin
        for l in range(L):
            hc, _ = ora.layer_forward(params[l], hc, b, s, nh, eps)
        return hc
    y0 = fwd(x)
    x2 = x.copy()
    x2[t] += 0.5           # token t of sequence 0
    y2 = fwd(x2)
    assert np.array_equal(y0[:t], y2[:t])
    assert not np.array_equal(y0[t], y2[t])
    assert np.array_equal(y0[s:], y2[s:])     # the other sequence is untouched


def test_batch_separation_swap():
    L, h, nh, f, s, b, eps = 2, 32, 4, 128, 6, 2, 1e-5
    params = _params(L, h, f)
    x = synth.stage_input(1, b * s, h, "f32").astype(np.float64)
    dy = synth.output_grad(1, b * s, h, "f32").astype(np.float64)
    swap = np.concatenate([np.arange(s, 2 * s), np.arange(0, s)])
    r1 = ora.run_stage(params, [x], [dy], nh, b, s, eps)
    r2 = ora.run_stage(params, [x[swap]], [dy[swap]], nh, b, s, eps)
    assert np.allclose(r1["ys"][0][swap], r2["ys"][0], rtol=0, atol=1e-13)
    assert np.allclose(r1["dxs"][0][swap], r2["dxs"][0], rtol=0, atol=1e-13)


def test_linearity_in_dy_bitwise():
    L, h, nh, f, s, b, M, eps = 2, 32, 4, 128, 8, 2, 2, 1e-5
    params = _params(L, h, f)
    xs, dys = _stage_inputs(M, b * s, h)
    r1 = ora.run_stage(params, xs, dys, nh, b, s, eps)
    r2 = ora.run_stage(params, xs, [2.0 * d for d in dys], nh, b, s, eps)
    for mb in range(M):
        assert np.array_equal(2.0 * r1["dxs"][mb], r2["dxs"][mb])
    for l in range(L):
        for name in ora.PARAM_NAMES:
            assert np.array_equal(2.0 * r1["grads"][l][name], r2["grads"][l][name]), name


def test_micro_batch_additivity():
    L, h, nh, f, s, b, M, eps = 2, 32, 4, 128, 8, 1, 3, 1e-5
    params = _params(L, h, f)
    xs, dys = _stage_inputs(M, b * s, h)
    acc = ora.run_stage(params, xs, dys, nh, b, s, eps)
    singles = [ora.run_stage(params, [xs[i]], [dys[i]], nh, b, s, eps) for i in range(M)]
    for l in range(L):
        for name in ora.PARAM_NAMES:
            tot = sum(r["grads"][l][name] for r in singles)
            assert np.allclose(tot, acc["grads"][l][name], rtol=1e-13, atol=1e-15)


@pytest.mark.parametrize("which", ["recompute_all", "selective", "layer_inputs", "offload_all",
                                   "mixed"])
def test_policy_invariance_bitwise(which):
    L, h, nh, f, s, b, M, eps = 3, 32, 4, 128, 8, 2, 3, 1e-5
    params = _params(L, h, f)
    xs, dys = _stage_inputs(M, b * s, h)
    keep = ora.run_stage(params, xs, dys, nh, b, s, eps)
    K, R, O = ora.KEEP, ora.RECOMPUTE, ora.OFFLOAD
    if which == "recompute_all":
        pol = [{t: (K if (t == "x" and l == 0) else R) for t in ora.TENSORS} for l in range(L)]
        mbs = ()
    elif which == "selective":
        pol = [{t: (R if t in ("o", "g") else K) for t in ora.TENSORS} for l in range(L)]
        mbs = ()
    elif which == "layer_inputs":
        pol = [{t: (K if t == "x" else R) for t in ora.TENSORS} for l in range(L)]
        mbs = ()
    elif which == "offload_all":
        pol = [{t: O for t in ora.TENSORS} for l in range(L)]
        mbs = range(M)
    else:
        pol = [{t: [K, R, O][(l + i) % 3] for i, t in enumerate(ora.TENSORS)} for l in range(L)]
        pol[0]["x"] = K
        mbs = (0, 2)
    order = [("F", 0), ("F", 1), ("B", 0), ("F", 2), ("B", 1), ("B", 2)]
    other = ora.run_stage(params, xs, dys, nh, b, s, eps, policy=pol, offload_mbs=mbs, order=order)
    for mb in range(M):
        assert np.array_equal(keep["ys"][mb], other["ys"][mb])
        assert np.array_equal(keep["dxs"][mb], other["dxs"][mb])
    for l in range(L):
        for name in ora.PARAM_NAMES:
            assert np.array_equal(keep["grads"][l][name], other["grads"][l][name]), (l, name)


def test_unit_flop_count_by_enumeration():
    """The algorithmic flop count equals 2 x the multiply-adds enumerated
    over the four linears and the causal lower triangle."""
    b, s, h, nh, f = 2, 5, 8, 2, 32
    T = b * s
    d = h // nh
    macs = T * h * 3 * h + T * h * h + T * h * f + T * f * h
    for _ in range(b):
        for _n in range(nh):
            for i in range(s):
                macs += 2 * d * (i + 1)      # q.k over j <= i, then P v
    got = ora.unit_flops(T, h, f, b, s)
    assert got["fwd"] == 2 * macs
    assert got["bwd"] == 4 * macs
