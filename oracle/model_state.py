"""Plain float64 CPU oracle of the model-state half of T-Offload.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import or run this module; it
imports nothing from the product path.

What it computes
----------------
T-Offload moves the model state of layers with poor temporal locality out of
HBM: after a layer's last backward of the mini-batch its gradients go to host
DRAM, the optimizer update of that layer runs on the CPU, and the updated
weights come back to the device before the layer's next forward, in a
quantized form (paper, Section 5, "Hardware-agnostic T-Offload Solution by
Co-design with T-Pipe").  The paper names neither the optimizer nor the
quantization, so this oracle fixes both (readings stated in the design notes):

* the optimizer is AdamW: first and second moment estimates with bias
  correction, and weight decay decoupled from the gradient step;
* the reloaded weights are either the storage dtype (bf16, round to nearest
  even) or FP8 E4M3 (1 sign, 4 exponent bits with bias 7, 3 mantissa bits, no
  infinities, largest finite value 448) with one float32 scale per matrix row,
  scale = max|row| / 448, rounding to the nearest representable value with
  ties to even mantissa and saturating at +-448; the device then computes
  with bf16(decode(q) * scale).
"""

from __future__ import annotations

import numpy as np

E4M3_MAX = 448.0


def adamw_step(w, m, v, g, step, lr, beta1, beta2, eps, weight_decay):
    """One AdamW update of parameter w with gradient g (step counts from 1).

    m <- beta1 m + (1 - beta1) g
    v <- beta2 v + (1 - beta2) g^2
    w <- w - lr (m / (1 - beta1^step)) / (sqrt(v / (1 - beta2^step)) + eps)
           - lr weight_decay w
    Returns new (w, m, v); inputs are not modified."""
    w = np.asarray(w, dtype=np.float64)
    g = np.asarray(g, dtype=np.float64)
    m = beta1 * np.asarray(m, dtype=np.float64) + (1.0 - beta1) * g
    v = beta2 * np.asarray(v, dtype=np.float64) + (1.0 - beta2) * g * g
    mhat = m / (1.0 - beta1 ** step)
    vhat = v / (1.0 - beta2 ** step)
    w_new = w - lr * mhat / (np.sqrt(vhat) + eps) - lr * weight_decay * w
    return w_new, m, v


def e4m3_values() -> np.ndarray:
    """The 256 codes of FP8 E4M3 decoded from the format's definition (code
    order; the two NaN codes 0x7F and 0xFF decode to NaN)."""
    out = np.empty(256, dtype=np.float64)
    for code in range(256):
        s = -1.0 if code & 0x80 else 1.0
        e = (code >> 3) & 0xF
        f = code & 0x7
        if e == 0xF and f == 0x7:
            out[code] = np.nan
        elif e == 0:
            out[code] = s * (f / 8.0) * 2.0 ** (1 - 7)          # subnormal
        else:
            out[code] = s * (1.0 + f / 8.0) * 2.0 ** (e - 7)
    return out


def e4m3_encode(x) -> np.ndarray:
    """Nearest E4M3 code of each value (ties to the even mantissa, i.e. the
    code with an even low bit), saturating to +-448; NaN is not expected.
    Works by search over the finite codes, the plain definition."""
    x = np.asarray(x, dtype=np.float64)
    vals = e4m3_values()
    finite = [c for c in range(128) if not np.isnan(vals[c])]   # non-negative codes
    pos = np.array([vals[c] for c in finite])
    codes = np.array(finite, dtype=np.int64)
    order = np.argsort(pos)
    pos, codes = pos[order], codes[order]
    a = np.minimum(np.abs(x), E4M3_MAX)
    idx = np.searchsorted(pos, a)               # pos[idx-1] < a <= pos[idx]
    idx = np.clip(idx, 1, len(pos) - 1)
    lo, hi = pos[idx - 1], pos[idx]
    pick_hi = (a - lo > hi - a) | ((a - lo == hi - a) & ((codes[idx] & 1) == 0))
    c = np.where(pick_hi, codes[idx], codes[idx - 1])
    c = np.where(a == 0.0, 0, c)
    sign = (x < 0) & (c != 0)
    return (c | np.where(sign, 0x80, 0)).astype(np.uint8)


def quantize_rows(wmat):
    """Per-row FP8 E4M3 quantization of a matrix: (codes uint8 [rows, cols],
    scales float32 [rows]) with scale = max|row| / 448 in float32 (1 for an
    all-zero row); the codes encode w / scale, computed in float32."""
    w32 = np.asarray(wmat, dtype=np.float32)
    amax = np.abs(w32).max(axis=1)
    scale = np.where(amax > 0, amax / np.float32(E4M3_MAX), np.float32(1.0)).astype(np.float32)
    q = e4m3_encode((w32 / scale[:, None]).astype(np.float32).astype(np.float64))
    return q, scale


def dequantize_rows(q, scale):
    """The weights the device computes with: decode(q) * scale in float32,
    as float64 values (before the bf16 rounding of storage)."""
    vals = e4m3_values()
    return (vals[np.asarray(q, dtype=np.int64)].astype(np.float32) * np.asarray(scale, np.float32)[:, None]).astype(np.float64)
