"""Seeded synthetic inputs for the stage: parameters, stage inputs, output grads.

This module holds generators only (no arithmetic of the method) and is the one
piece shared by the GPU path's callers and by the oracle's tests.

Recipe (fixed so that every test, the bench and the oracle see the same bits):

* generator ``numpy.random.Generator(PCG64(seed))``;
* parameter seeds ``1000 + 16 * layer + tensor_id`` (tensor ids in PARAM_ORDER);
* stage input x of micro-batch mb: seed ``2000 + mb``, N(0, 1);
* output gradient dy of micro-batch mb: seed ``3000 + mb``, N(0, 1);
* matrices and biases N(0, 0.02); LayerNorm gains 1 + N(0, 0.02); LayerNorm
  shifts N(0, 0.02) (nonzero, so that a dropped bias or shift is visible);
* values are drawn in float32; for bf16 storage they are rounded once to
  bf16 with round-to-nearest-even, and consumers that work in higher precision
  take the rounded values.
"""

from __future__ import annotations

import numpy as np

PARAM_ORDER = ("w_qkv", "b_qkv", "w_o", "b_o", "w_1", "b_1", "w_2", "b_2",
               "g1", "be1", "g2", "be2")


def param_shapes(h: int, f: int) -> dict:
    return {
        "w_qkv": (3 * h, h), "b_qkv": (3 * h,),
        "w_o": (h, h), "b_o": (h,),
        "w_1": (f, h), "b_1": (f,),
        "w_2": (h, f), "b_2": (h,),
        "g1": (h,), "be1": (h,), "g2": (h,), "be2": (h,),
    }


def llama_param_shapes(h: int, n_heads: int, n_kv: int, f: int) -> dict:
    """LLAMA-style layer: packed q | k | v projection with n_kv key/value
    heads, packed gate | up projection, no biases, RMSNorm gains only."""
    d = h // n_heads
    return {"w_qkv": ((n_heads + 2 * n_kv) * d, h), "w_o": (h, h), "w_1": (2 * f, h), "w_2": (h, f),
            "g1": (h,), "g2": (h,)}


def _rng(seed: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(seed))


def to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """float32 -> bf16 bit patterns (uint16), round to nearest even."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32).astype(np.uint64)
    rounded = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    return rounded.astype(np.uint16)


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def round_to_storage(a: np.ndarray, dtype: str) -> np.ndarray:
    """Values of ``a`` as stored in ``dtype`` ("f32" or "bf16"), as float32."""
    a = np.asarray(a, dtype=np.float32)
    if dtype == "f32":
        return a
    if dtype == "bf16":
        return bf16_bits_to_f32(to_bf16_bits(a))
    raise ValueError(dtype)


def layer_params(layer: int, h: int, f: int, dtype: str) -> dict:
    """Parameters of one layer as float32 arrays holding storage-dtype values."""
    out = {}
    for tid, (name, shape) in enumerate(param_shapes(h, f).items()):
        r = _rng(1000 + 16 * layer + tid)
        v = r.standard_normal(shape, dtype=np.float32) * np.float32(0.02)
        if name in ("g1", "g2"):
            v = v + np.float32(1.0)
        out[name] = round_to_storage(v, dtype)
    return out


def llama_layer_params(layer: int, h: int, n_heads: int, n_kv: int, f: int, dtype: str) -> dict:
    """LLAMA-style layer parameters, same recipe (a tensor's seed uses its
    GPT-layer id: w_qkv 0, w_o 2, w_1 4, w_2 6, g1 8, g2 10)."""
    out = {}
    for name, shape in llama_param_shapes(h, n_heads, n_kv, f).items():
        r = _rng(1000 + 16 * layer + PARAM_ORDER.index(name))
        v = r.standard_normal(shape, dtype=np.float32) * np.float32(0.02)
        if name in ("g1", "g2"):
            v = v + np.float32(1.0)
        out[name] = round_to_storage(v, dtype)
    return out


def stage_input(mb: int, tokens: int, h: int, dtype: str) -> np.ndarray:
    r = _rng(2000 + mb)
    return round_to_storage(r.standard_normal((tokens, h), dtype=np.float32), dtype)


def output_grad(mb: int, tokens: int, h: int, dtype: str) -> np.ndarray:
    r = _rng(3000 + mb)
    return round_to_storage(r.standard_normal((tokens, h), dtype=np.float32), dtype)


def uniform_tensor(seed: int, shape, scale: float, dtype: str) -> np.ndarray:
    """Generic seeded N(0, scale^2) tensor for per-kernel tests."""
    r = _rng(seed)
    return round_to_storage(r.standard_normal(shape, dtype=np.float32) * np.float32(scale), dtype)
