"""Plain fp64 CPU oracle for one pipeline stage of LLAMA-style decoder layers.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import or run this module.  The product
path never imports it, and it imports nothing from the product path.

What it computes
----------------
LLAMA is the paper's main evaluated model family (Section 6.1, "Workloads":
LLAMA2-70B and GPT3-175B; the end-to-end results of Figure 8 train LLAMA-based
models of 48 and 96 layers), but the paper does not restate the
architecture.  The layer here is the publicly described LLAMA-2 decoder block
(the LLAMA2 reference the paper cites):

    a   = RMSNorm(x; g1)                = x / sqrt(mean(x^2) + eps) * g1
    qkv = a W_qkv^T                      (q: n_heads heads | k, v: n_kv heads)
    q, k rotated by RoPE                 (pairs (i, i + d/2) of every head,
                                          angle pos * base^(-2i/d))
    o   = causal softmax(q k^T / sqrt d) v,  query head n reading key/value
                                          head n // (n_heads / n_kv)  (GQA)
    x1  = x + o W_o^T
    c   = RMSNorm(x1; g2)
    u   = c W_1^T                        (gate | up column blocks, f each)
    g   = SiLU(gate) * up,  SiLU(z) = z / (1 + exp(-z))
    y   = x1 + g W_2^T

No biases.  The tensor vocabulary of the stage (what a backward pass reads) is
that of the GPT stage: ``qkv`` is stored after the rotation (it is what the
attention reads), ``ln1``/``ln2`` hold the per-row reciprocal RMS, ``u`` holds
gate and up.  Everything is float64 numpy; matrix products use ``@``.
Recompute and offload are implemented literally by :mod:`decoder_stage`'s
stage runner, to which this module hands its layer.
"""

from __future__ import annotations

import math

import numpy as np

from . import decoder_stage as _gpt

TENSORS = _gpt.TENSORS
PARAM_NAMES = ("w_qkv", "w_o", "w_1", "w_2", "g1", "g2")


# --------------------------------------------------------------------------
# RMS normalisation (eps inside the square root, no centring, no shift).
# --------------------------------------------------------------------------
def rms_norm(z, gamma, eps):
    """z / sqrt(mean_j z^2 + eps) * gamma.  Returns (out, rstd[rows])."""
    z = np.asarray(z, dtype=np.float64)
    rstd = 1.0 / np.sqrt((z * z).mean(axis=1) + eps)
    return z * rstd[:, None] * gamma[None, :], rstd


def rms_norm_backward(dout, z, rstd, gamma):
    """Gradient of :func:`rms_norm`: with zhat = z * rstd and dzhat =
    dout * gamma, dz = rstd * (dzhat - zhat * mean_j(dzhat * zhat)) and
    dgamma = sum over rows of dout * zhat."""
    zhat = z * rstd[:, None]
    dzhat = dout * gamma[None, :]
    m = (dzhat * zhat).mean(axis=1)
    return rstd[:, None] * (dzhat - zhat * m[:, None]), (dout * zhat).sum(axis=0)


# --------------------------------------------------------------------------
# Rotary position embedding.
# --------------------------------------------------------------------------
def rope_angles(s, d, base):
    """angle[pos, i] = pos * base^(-2 i / d) for i < d/2."""
    inv = base ** (-2.0 * np.arange(d // 2, dtype=np.float64) / d)
    return np.arange(s, dtype=np.float64)[:, None] * inv[None, :]


def rope(x, b, s, n_heads, d, base, inverse=False):
    """Rotates every head of x [b*s, n_heads*d]: for i < d/2 the pair
    (x_i, x_{i+d/2}) at position pos turns by +angle (inverse: -angle)."""
    ang = rope_angles(s, d, base)
    cos, sin = np.cos(ang), np.sin(ang)
    if inverse:
        sin = -sin
    out = np.empty_like(np.asarray(x, dtype=np.float64))
    half = d // 2
    for ib in range(b):
        rows = slice(ib * s, (ib + 1) * s)
        for n in range(n_heads):
            lo = x[rows, n * d:n * d + half]
            hi = x[rows, n * d + half:(n + 1) * d]
            out[rows, n * d:n * d + half] = lo * cos - hi * sin
            out[rows, n * d + half:(n + 1) * d] = hi * cos + lo * sin
    return out


# --------------------------------------------------------------------------
# Causal grouped-query attention over packed q | k | v.
# --------------------------------------------------------------------------
def _blocks(n_heads, n_kv, d):
    H, HK = n_heads * d, n_kv * d
    return H, HK, n_heads // n_kv


def gqa_attention(qkv, b, s, n_heads, n_kv):
    """Query head n attends with key/value head n // (n_heads / n_kv):
    S = q_n k^T / sqrt(d) for key j <= query i, P = softmax_j(S), o_n = P v,
    lse_i = log sum_{j<=i} exp(S_ij).  qkv: [b*s, (n_heads + 2 n_kv) d].
    Returns o [b*s, n_heads d] and lse [b, n_heads, s]."""
    d = qkv.shape[1] // (n_heads + 2 * n_kv)
    H, HK, grp = _blocks(n_heads, n_kv, d)
    o = np.zeros((b * s, H))
    lse = np.zeros((b, n_heads, s))
    mask = np.triu(np.ones((s, s), dtype=bool), k=1)
    scale = 1.0 / math.sqrt(d)
    for ib in range(b):
        rows = slice(ib * s, (ib + 1) * s)
        for n in range(n_heads):
            kv = n // grp
            q = qkv[rows, n * d:(n + 1) * d]
            k = qkv[rows, H + kv * d:H + (kv + 1) * d]
            v = qkv[rows, H + HK + kv * d:H + HK + (kv + 1) * d]
            S = (q @ k.T) * scale
            S[mask] = -np.inf
            m = S.max(axis=1)
            e = np.exp(S - m[:, None])
            den = e.sum(axis=1)
            o[rows, n * d:(n + 1) * d] = (e / den[:, None]) @ v
            lse[ib, n] = m + np.log(den)
    return o, lse


def gqa_attention_backward(qkv, o, lse, do, b, s, n_heads, n_kv):
    """Gradient of :func:`gqa_attention`.  Per query head, with P rebuilt
    from lse: dv += P^T do, dP = do v^T, D_i = do_i . o_i, dS = P (dP - D),
    dq = dS k / sqrt(d), dk += dS^T q / sqrt(d); a key/value head sums the
    contributions of its query heads in ascending head order."""
    d = qkv.shape[1] // (n_heads + 2 * n_kv)
    H, HK, grp = _blocks(n_heads, n_kv, d)
    dqkv = np.zeros_like(qkv, dtype=np.float64)
    mask = np.triu(np.ones((s, s), dtype=bool), k=1)
    scale = 1.0 / math.sqrt(d)
    for ib in range(b):
        rows = slice(ib * s, (ib + 1) * s)
        for n in range(n_heads):
            kv = n // grp
            kc = slice(H + kv * d, H + (kv + 1) * d)
            vc = slice(H + HK + kv * d, H + HK + (kv + 1) * d)
            q, k, v = qkv[rows, n * d:(n + 1) * d], qkv[rows, kc], qkv[rows, vc]
            S = (q @ k.T) * scale
            S[mask] = -np.inf
            P = np.exp(S - lse[ib, n][:, None])
            don = do[rows, n * d:(n + 1) * d]
            dP = don @ v.T
            D = (don * o[rows, n * d:(n + 1) * d]).sum(axis=1)
            dS = P * (dP - D[:, None])
            dqkv[rows, n * d:(n + 1) * d] = (dS @ k) * scale
            dqkv[rows, kc] += (dS.T @ q) * scale
            dqkv[rows, vc] += P.T @ don
    return dqkv


# --------------------------------------------------------------------------
# SwiGLU.
# --------------------------------------------------------------------------
def _sigmoid(z):
    return 1.0 / (1.0 + np.exp(-z))


def swiglu(u):
    """u = [gate | up] (f columns each) -> SiLU(gate) * up."""
    f = u.shape[1] // 2
    gate, up = u[:, :f], u[:, f:]
    return gate * _sigmoid(gate) * up


def swiglu_backward(dg, u):
    """d gate = dg * up * sigma (1 + gate (1 - sigma)), d up = dg * SiLU(gate)."""
    f = u.shape[1] // 2
    gate, up = u[:, :f], u[:, f:]
    sg = _sigmoid(gate)
    return np.concatenate([dg * up * sg * (1.0 + gate * (1.0 - sg)), dg * gate * sg], axis=1)


# --------------------------------------------------------------------------
# One layer.
# --------------------------------------------------------------------------
def layer_forward(p, x, b, s, n_heads, n_kv, eps, rope_base):
    x = np.asarray(x, dtype=np.float64)
    d = p["w_o"].shape[1] // n_heads
    H, HK, _ = _blocks(n_heads, n_kv, d)
    a, r1 = rms_norm(x, p["g1"], eps)
    qkv = a @ p["w_qkv"].T
    qkv[:, :H] = rope(qkv[:, :H], b, s, n_heads, d, rope_base)
    qkv[:, H:H + HK] = rope(qkv[:, H:H + HK], b, s, n_kv, d, rope_base)
    o, lse = gqa_attention(qkv, b, s, n_heads, n_kv)
    x1 = x + o @ p["w_o"].T
    c, r2 = rms_norm(x1, p["g2"], eps)
    u = c @ p["w_1"].T
    g = swiglu(u)
    y = x1 + g @ p["w_2"].T
    saved = dict(x=x, a=a, qkv=qkv, o=o, lse=lse, x1=x1, c=c, u=u, g=g, ln1=r1, ln2=r2)
    return y, saved


def layer_backward(p, sv, dy, b, s, n_heads, n_kv, rope_base):
    gr = {}
    d = p["w_o"].shape[1] // n_heads
    H, HK, _ = _blocks(n_heads, n_kv, d)
    gr["w_2"] = dy.T @ sv["g"]
    dg = dy @ p["w_2"]
    du = swiglu_backward(dg, sv["u"])
    gr["w_1"] = du.T @ sv["c"]
    dc = du @ p["w_1"]
    dx1_n, gr["g2"] = rms_norm_backward(dc, sv["x1"], sv["ln2"], p["g2"])
    dx1 = dy + dx1_n
    gr["w_o"] = dx1.T @ sv["o"]
    do = dx1 @ p["w_o"]
    dqkv = gqa_attention_backward(sv["qkv"], sv["o"], sv["lse"], do, b, s, n_heads, n_kv)
    # the rotation is orthogonal: its gradient turns back by the same angle
    dqkv[:, :H] = rope(dqkv[:, :H], b, s, n_heads, d, rope_base, inverse=True)
    dqkv[:, H:H + HK] = rope(dqkv[:, H:H + HK], b, s, n_kv, d, rope_base, inverse=True)
    gr["w_qkv"] = dqkv.T @ sv["a"]
    da = dqkv @ p["w_qkv"]
    dx_n, gr["g1"] = rms_norm_backward(da, sv["x"], sv["ln1"], p["g1"])
    return dx1 + dx_n, gr


def layer_output(p, sv):
    return sv["x1"] + sv["g"] @ p["w_2"].T


def run_stage(params, xs, dys, n_heads, n_kv, b, s, eps=1e-5, rope_base=10000.0, policy=None, offload_mbs=(),
              order=None):
    """Forward and backward of a stage of LLAMA-style layers for every
    micro-batch, with the keep / recompute / offload semantics of
    :func:`decoder_stage.run_stage` (same arguments, plus n_kv and
    rope_base)."""
    layer = dict(
        forward=lambda p, x, b_, s_, nh, e: layer_forward(p, x, b_, s_, nh, n_kv, e, rope_base),
        backward=lambda p, sv, dy, b_, s_, nh: layer_backward(p, sv, dy, b_, s_, nh, n_kv, rope_base),
        output=lambda p, sv, b_, s_, nh, e: layer_output(p, sv))
    return _gpt.run_stage(params, xs, dys, n_heads, b, s, eps=eps, policy=policy, offload_mbs=offload_mbs,
                          order=order, layer=layer)


def unit_flops(T, h, n_heads, n_kv, f, b, s):
    """Algorithmic flops of one layer x one micro-batch: forward GEMMs
    2T h ((n_heads + 2 n_kv) d + h + 3 f), causal attention 2 b h s (s + 1)
    (h = n_heads d), backward twice the forward."""
    d = h // n_heads
    gemm = 2.0 * T * h * ((n_heads + 2 * n_kv) * d + h + 3.0 * f)
    attn = 2.0 * b * h * s * (s + 1)
    return dict(fwd_gemm=gemm, fwd_attn=attn, fwd=gemm + attn, bwd=2.0 * (gemm + attn))
