"""Plain fp64 CPU oracle for one pipeline stage of GPT-style pre-LN decoder layers.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import or run this module.  The product
path (the HIP library and its Python binding) never imports it, and this module
imports nothing from the product path: the two share no code.

What it computes
----------------
A pipeline stage is a block of consecutive transformer layers; the activation
memory m_a of the paper counts the layers only, without the input embedding and
the language-model head (paper, Section 2, symbol list), so the stage holds no
embedding, no final norm and no head.  Forward computation runs through the
stage micro-batch by micro-batch and one activation tensor leaves it; in the
backward pass the gradient of that tensor comes back (Section 2.1).  The
evaluated workloads include GPT-3 (Section 6.1, "Workloads"), with exact fused
attention (FlashAttention) enabled (Section 6.1), so every layer is the GPT
pre-LN decoder block with exact causal softmax attention:

    a   = LN(x; g1, be1)
    qkv = a W_qkv^T + b_qkv                      (q | k | v column blocks)
    o   = causal softmax(q k^T / sqrt(d)) v      (per sequence, per head)
    x1  = x + o W_o^T + b_o
    c   = LN(x1; g2, be2)
    u   = c W_1^T + b_1,   g = GeLU(u) = u/2 (1 + erf(u / sqrt 2))
    y   = x1 + g W_2^T + b_2

Weights follow the nn.Linear convention [out, in]; activations are token-major
[T, width] with T = b * s and row r = batch_index * s + position.

Recomputation keeps a subset of forward activations (checkpoints) and
regenerates the others in the backward pass (Section 2.2); offloading moves
tensors to host DRAM and back (Section 2.2; Section 5).  Neither changes the
mathematical result, so :func:`run_stage` implements both literally (drop and
re-run the forward; copy out and copy back) to let tests check that invariance
on the oracle itself.

Everything is float64 numpy; matrix products use ``@`` (a library matmul used
as one step), everything else is written out.  Gradients of parameters are
summed over micro-batches in ascending micro-batch order.
"""

from __future__ import annotations

import math

import numpy as np
from scipy.special import erf as _erf

# Names of the per-(layer, micro-batch) tensors a backward pass reads.  The
# same vocabulary is used by the policy tables of the stage library.
TENSORS = ("x", "a", "qkv", "o", "lse", "x1", "c", "u", "g", "ln1", "ln2")

PARAM_NAMES = ("w_qkv", "b_qkv", "w_o", "b_o", "w_1", "b_1", "w_2", "b_2",
               "g1", "be1", "g2", "be2")


# --------------------------------------------------------------------------
# Layer normalisation (biased variance, eps inside the square root).
# --------------------------------------------------------------------------
def layer_norm(z, gamma, beta, eps):
    """LN over the last axis: (z - mean) / sqrt(var + eps) * gamma + beta.

    Returns (out, mean, rstd) with mean and rstd of shape [rows]."""
    z = np.asarray(z, dtype=np.float64)
    mean = z.mean(axis=1)
    centred = z - mean[:, None]
    var = (centred * centred).mean(axis=1)
    rstd = 1.0 / np.sqrt(var + eps)
    zhat = centred * rstd[:, None]
    return zhat * gamma[None, :] + beta[None, :], mean, rstd


def layer_norm_backward(dout, z, mean, rstd, gamma):
    """Gradient of :func:`layer_norm` w.r.t. its input, gamma and beta.

    With zhat = (z - mean) * rstd and dzhat = dout * gamma, the input gradient
    is rstd * (dzhat - mean_j(dzhat) - zhat * mean_j(dzhat * zhat))."""
    zhat = (z - mean[:, None]) * rstd[:, None]
    dgamma = (dout * zhat).sum(axis=0)
    dbeta = dout.sum(axis=0)
    dzhat = dout * gamma[None, :]
    m1 = dzhat.mean(axis=1)
    m2 = (dzhat * zhat).mean(axis=1)
    dz = rstd[:, None] * (dzhat - m1[:, None] - zhat * m2[:, None])
    return dz, dgamma, dbeta


# --------------------------------------------------------------------------
# GeLU, exact (erf) form.
# --------------------------------------------------------------------------
def gelu(u):
    return 0.5 * u * (1.0 + _erf(u / math.sqrt(2.0)))


def gelu_grad(u):
    """d/du GeLU(u) = Phi(u) + u * phi(u)."""
    cdf = 0.5 * (1.0 + _erf(u / math.sqrt(2.0)))
    pdf = np.exp(-0.5 * u * u) / math.sqrt(2.0 * math.pi)
    return cdf + u * pdf


# --------------------------------------------------------------------------
# Causal multi-head attention over packed q | k | v (exact; no s x s tensor is
# kept between calls, but inside one call the plain definition is used).
# --------------------------------------------------------------------------
def _split(qkv, h):
    return qkv[:, 0:h], qkv[:, h:2 * h], qkv[:, 2 * h:3 * h]


def causal_attention(qkv, b, s, n_heads):
    """Per sequence and head: S = q k^T / sqrt(d) for key j <= query i,
    P = softmax_j(S), o = P v, lse_i = log sum_{j<=i} exp(S_ij).

    qkv: [b*s, 3h].  Returns o [b*s, h] and lse [b, n_heads, s]."""
    h = qkv.shape[1] // 3
    d = h // n_heads
    q, k, v = _split(qkv, h)
    o = np.zeros((b * s, h))
    lse = np.zeros((b, n_heads, s))
    mask = np.triu(np.ones((s, s), dtype=bool), k=1)   # True where j > i
    scale = 1.0 / math.sqrt(d)
    for ib in range(b):
        rows = slice(ib * s, (ib + 1) * s)
        for n in range(n_heads):
            cols = slice(n * d, (n + 1) * d)
            S = (q[rows, cols] @ k[rows, cols].T) * scale
            S[mask] = -np.inf
            m = S.max(axis=1)
            e = np.exp(S - m[:, None])
            denom = e.sum(axis=1)
            P = e / denom[:, None]
            o[rows, cols] = P @ v[rows, cols]
            lse[ib, n] = m + np.log(denom)
    return o, lse


def causal_attention_backward(qkv, o, lse, do, b, s, n_heads):
    """Gradient of :func:`causal_attention`: with P rebuilt from lse,
    dv = P^T do, dP = do v^T, D_i = do_i . o_i, dS = P * (dP - D),
    dq = dS k / sqrt(d), dk = dS^T q / sqrt(d).  Returns dqkv [b*s, 3h]."""
    h = qkv.shape[1] // 3
    d = h // n_heads
    q, k, v = _split(qkv, h)
    dqkv = np.zeros_like(qkv, dtype=np.float64)
    mask = np.triu(np.ones((s, s), dtype=bool), k=1)
    scale = 1.0 / math.sqrt(d)
    for ib in range(b):
        rows = slice(ib * s, (ib + 1) * s)
        for n in range(n_heads):
            cols = slice(n * d, (n + 1) * d)
            qh, kh, vh = q[rows, cols], k[rows, cols], v[rows, cols]
            S = (qh @ kh.T) * scale
            S[mask] = -np.inf
            P = np.exp(S - lse[ib, n][:, None])
            doh = do[rows, cols]
            dv = P.T @ doh
            dP = doh @ vh.T
            D = (doh * o[rows, cols]).sum(axis=1)
            dS = P * (dP - D[:, None])
            dqkv[rows, cols] = (dS @ kh) * scale
            dqkv[rows, h + n * d:h + (n + 1) * d] = (dS.T @ qh) * scale
            dqkv[rows, 2 * h + n * d:2 * h + (n + 1) * d] = dv
    return dqkv


# --------------------------------------------------------------------------
# One decoder layer.
# --------------------------------------------------------------------------
def layer_forward(p, x, b, s, n_heads, eps):
    """Forward of one pre-LN decoder layer.  Returns (y, saved) where saved
    holds every tensor the backward pass reads (names in TENSORS)."""
    x = np.asarray(x, dtype=np.float64)
    a, mu1, rstd1 = layer_norm(x, p["g1"], p["be1"], eps)
    qkv = a @ p["w_qkv"].T + p["b_qkv"][None, :]
    o, lse = causal_attention(qkv, b, s, n_heads)
    x1 = x + o @ p["w_o"].T + p["b_o"][None, :]
    c, mu2, rstd2 = layer_norm(x1, p["g2"], p["be2"], eps)
    u = c @ p["w_1"].T + p["b_1"][None, :]
    g = gelu(u)
    y = x1 + g @ p["w_2"].T + p["b_2"][None, :]
    saved = dict(x=x, a=a, qkv=qkv, o=o, lse=lse, x1=x1, c=c, u=u, g=g,
                 ln1=(mu1, rstd1), ln2=(mu2, rstd2))
    return y, saved


def layer_backward(p, sv, dy, b, s, n_heads):
    """Backward of one decoder layer from its saved tensors.

    Returns (dx, grads) with grads keyed like the parameters."""
    gr = {}
    # MLP: y = x1 + g W_2^T + b_2, g = GeLU(u), u = c W_1^T + b_1
    gr["w_2"] = dy.T @ sv["g"]
    gr["b_2"] = dy.sum(axis=0)
    dg = dy @ p["w_2"]
    du = dg * gelu_grad(sv["u"])
    gr["w_1"] = du.T @ sv["c"]
    gr["b_1"] = du.sum(axis=0)
    dc = du @ p["w_1"]
    dx1_ln, gr["g2"], gr["be2"] = layer_norm_backward(
        dc, sv["x1"], sv["ln2"][0], sv["ln2"][1], p["g2"])
    dx1 = dy + dx1_ln
    # attention block: x1 = x + o W_o^T + b_o
    gr["w_o"] = dx1.T @ sv["o"]
    gr["b_o"] = dx1.sum(axis=0)
    do = dx1 @ p["w_o"]
    dqkv = causal_attention_backward(sv["qkv"], sv["o"], sv["lse"], do,
                                     b, s, n_heads)
    gr["w_qkv"] = dqkv.T @ sv["a"]
    gr["b_qkv"] = dqkv.sum(axis=0)
    da = dqkv @ p["w_qkv"]
    dx_ln, gr["g1"], gr["be1"] = layer_norm_backward(
        da, sv["x"], sv["ln1"][0], sv["ln1"][1], p["g1"])
    dx = dx1 + dx_ln
    return dx, gr


# --------------------------------------------------------------------------
# The stage: L layers, M micro-batches, keep / recompute / offload policies.
# --------------------------------------------------------------------------
KEEP, RECOMPUTE, OFFLOAD = 0, 1, 2


class _HostStore:
    """Stand-in for pinned host DRAM: tensors are copied out and back."""

    def __init__(self):
        self.data = {}

    def put(self, key, value):
        self.data[key] = _deep_copy(value)

    def take(self, key):
        return self.data.pop(key)


def _deep_copy(v):
    if isinstance(v, tuple):
        return tuple(np.array(t, copy=True) for t in v)
    return np.array(v, copy=True)


def run_stage(params, xs, dys, n_heads, b, s, eps=1e-5, policy=None,
              offload_mbs=(), order=None, layer=None):
    """Forward and backward of the whole stage for every micro-batch.

    params : list (one per layer) of dicts keyed by PARAM_NAMES (float64)
    xs, dys: lists (one per micro-batch) of [b*s, h] arrays
    policy : None (keep everything) or [L][name] -> KEEP/RECOMPUTE/OFFLOAD.
             RECOMPUTE drops the tensor after the forward and regenerates it
             by re-running the forward from the layer input before the
             backward (Section 2.2).  OFFLOAD copies the tensor to a host
             store after the forward and back before the backward, for the
             micro-batches listed in ``offload_mbs``; for the others it acts
             as KEEP.
    order  : op list of ("F", mb) / ("B", mb); default: all forwards, then
             all backwards in ascending micro-batch order.

    layer  : None (the GPT layer of this module) or dict(forward=, backward=,
             output=) with the signatures of layer_forward, layer_backward
             and _layer_output, for another layer kind run by the same
             stage logic.

    Returns dict(ys=[...], dxs=[...], grads=[per-layer dicts]) where grads
    are summed over micro-batches in the order the backwards run.
    """
    fwd = layer["forward"] if layer else layer_forward
    bwd = layer["backward"] if layer else layer_backward
    out = layer["output"] if layer else _layer_output
    L = len(params)
    M = len(xs)
    if order is None:
        order = [("F", i) for i in range(M)] + [("B", i) for i in range(M)]
    pol = policy if policy is not None else [
        {t: KEEP for t in TENSORS} for _ in range(L)]
    offload_mbs = set(offload_mbs)
    grads = [{k: np.zeros_like(np.asarray(v, dtype=np.float64))
              for k, v in p.items()} for p in params]
    ys, dxs = [None] * M, [None] * M
    device = {}            # (mb, layer) -> dict of resident saved tensors
    host = _HostStore()
    stage_inputs = {}

    def mode(layer, name, mb):
        m = pol[layer][name]
        if m == OFFLOAD and mb not in offload_mbs:
            return KEEP
        return m

    for op, mb in order:
        if op == "F":
            h = np.asarray(xs[mb], dtype=np.float64)
            stage_inputs[mb] = h
            for l in range(L):
                h_next, sv = fwd(params[l], h, b, s, n_heads, eps)
                kept = {}
                for name in TENSORS:
                    m = mode(l, name, mb)
                    if m == KEEP:
                        kept[name] = sv[name]
                    elif m == OFFLOAD:
                        host.put((mb, l, name), sv[name])
                    # RECOMPUTE: dropped here
                device[(mb, l)] = kept
                h = h_next
            ys[mb] = h
        else:
            # bring back offloaded tensors and regenerate dropped ones
            full = {}
            for l in range(L):
                kept = device.pop((mb, l))
                for name in TENSORS:
                    if mode(l, name, mb) == OFFLOAD:
                        kept[name] = host.take((mb, l, name))
                full[l] = kept
            for l in range(L):
                missing = [n for n in TENSORS if n not in full[l]]
                if not missing:
                    continue
                # the layer input is either kept or is the previous layer's
                # (regenerated) output
                if "x" in full[l]:
                    x_in = full[l]["x"]
                elif l == 0:
                    x_in = stage_inputs[mb]
                else:
                    x_in = out(params[l - 1], full[l - 1], b, s, n_heads, eps)
                _, sv = fwd(params[l], x_in, b, s, n_heads, eps)
                for n in missing:
                    full[l][n] = sv[n]
            g = np.asarray(dys[mb], dtype=np.float64)
            for l in reversed(range(L)):
                g, gr = bwd(params[l], full[l], g, b, s, n_heads)
                for k in gr:
                    grads[l][k] += gr[k]
            dxs[mb] = g
            stage_inputs.pop(mb, None)
    return dict(ys=ys, dxs=dxs, grads=grads)


def _layer_output(p, sv, b, s, n_heads, eps):
    """Output y of a layer from a complete saved set (x1 and g suffice)."""
    return sv["x1"] + sv["g"] @ p["w_2"].T + p["b_2"][None, :]


# --------------------------------------------------------------------------
# Work counts used by the measurement (algorithmic flops, Section 6 metric).
# --------------------------------------------------------------------------
def unit_flops(T, h, f, b, s):
    """Algorithmic flops of one layer x one micro-batch.

    Forward GEMMs 2T(4h^2 + 2hf); causal attention forward 2 b h s (s+1)
    (two products over the lower triangle including the diagonal); the
    backward is twice the forward."""
    gemm = 2.0 * T * (4.0 * h * h + 2.0 * h * f)
    attn = 2.0 * b * h * s * (s + 1)
    return dict(fwd_gemm=gemm, fwd_attn=attn, fwd=gemm + attn,
                bwd=2.0 * (gemm + attn))
