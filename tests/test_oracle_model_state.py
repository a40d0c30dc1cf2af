"""Pins of the model-state oracle (oracle/model_state.py): AdamW against
torch's AdamW in float64 and against its step-1 closed form, and FP8 E4M3
against the properties the format's definition fixes (largest finite 448,
smallest normal 2^-6, smallest subnormal 2^-9, one NaN pattern per sign),
exhaustive round trips and brute-force nearest-value search."""
import numpy as np
import pytest

from oracle import model_state as ms


def test_adamw_matches_torch_float64_over_steps():
    import torch
    rng = np.random.default_rng(0)
    w0 = rng.standard_normal(257)
    grads = [rng.standard_normal(257) for _ in range(4)]
    hp = dict(lr=1e-3, beta1=0.9, beta2=0.95, eps=1e-8, weight_decay=0.1)
    p = torch.tensor(w0, dtype=torch.float64, requires_grad=True)
    opt = torch.optim.AdamW([p], lr=hp["lr"], betas=(hp["beta1"], hp["beta2"]), eps=hp["eps"],
                            weight_decay=hp["weight_decay"])
    w, m, v = w0, np.zeros_like(w0), np.zeros_like(w0)
    for t, g in enumerate(grads, start=1):
        p.grad = torch.tensor(g, dtype=torch.float64)
        opt.step()
        w, m, v = ms.adamw_step(w, m, v, g, t, **hp)
        assert np.allclose(w, p.detach().numpy(), rtol=1e-13, atol=1e-15), t


def test_adamw_first_step_closed_form():
    """At step 1 the bias-corrected moments are g and g^2: with eps = 0 the
    update is lr * sign(g) plus the decoupled decay lr * wd * w."""
    w = np.array([1.0, -2.0, 0.5, 3.0])
    g = np.array([0.3, -4.0, 1e-3, -0.2])
    w1, m1, v1 = ms.adamw_step(w, 0 * w, 0 * w, g, 1, lr=0.01, beta1=0.9, beta2=0.999, eps=0.0, weight_decay=0.5)
    assert np.allclose(w1, w - 0.01 * np.sign(g) - 0.01 * 0.5 * w, rtol=0, atol=1e-15)
    assert np.allclose(m1, 0.1 * g) and np.allclose(v1, 0.001 * g * g)


def test_e4m3_table_properties():
    vals = ms.e4m3_values()
    assert np.isnan(vals[0x7F]) and np.isnan(vals[0xFF])
    assert np.isfinite(vals).sum() == 254
    assert vals[0x00] == 0.0 and vals[0x80] == 0.0
    assert vals[0x01] == 2.0 ** -9            # smallest subnormal
    assert vals[0x07] == 7 * 2.0 ** -9        # largest subnormal
    assert vals[0x08] == 2.0 ** -6            # smallest normal
    assert vals[0x38] == 1.0 and vals[0xB8] == -1.0
    assert vals[0x7E] == 448.0 and vals[0xFE] == -448.0
    pos = vals[:0x7F]
    assert np.all(np.diff(pos) > 0)           # codes 0..126 increase
    assert np.array_equal(vals[0x80:0xFF], -vals[:0x7F])


def test_e4m3_encode_round_trip_and_nearest():
    vals = ms.e4m3_values()
    for c in range(256):
        if np.isnan(vals[c]) or c == 0x80:
            continue
        assert ms.e4m3_encode(np.array([vals[c]]))[0] == c
    rng = np.random.default_rng(1)
    x = np.concatenate([rng.standard_normal(4000) * 10 ** rng.uniform(-3, 2.5, 4000), [0.0, -0.0, 500.0, -1e6]])
    q = ms.e4m3_encode(x)
    dec = vals[q.astype(int)]
    finite = vals[np.isfinite(vals)]
    for xi, di in zip(x, dec):
        t = np.clip(xi, -448, 448)
        best = np.min(np.abs(finite - t))
        assert abs(t - di) == best


def test_e4m3_ties_to_even_and_saturation():
    # 1.0625 lies halfway between 1.0 (mantissa 000) and 1.125 (001): even -> 1.0
    # 1.1875 lies halfway between 1.125 (001) and 1.25 (010): even -> 1.25
    q = ms.e4m3_encode(np.array([1.0625, 1.1875, -1.0625, 464.0, 1000.0, -1000.0, 2.0 ** -10, 3 * 2.0 ** -10]))
    vals = ms.e4m3_values()
    assert list(vals[q.astype(int)]) == [1.0, 1.25, -1.0, 448.0, 448.0, -448.0, 0.0, 2 * 2.0 ** -9]


def test_quantize_rows_error_bound():
    rng = np.random.default_rng(2)
    w = rng.standard_normal((33, 70)) * 0.02
    w[5] = 0.0
    q, s = ms.quantize_rows(w)
    assert s.dtype == np.float32 and q.dtype == np.uint8
    assert s[5] == 1.0 and np.all(q[5] == 0)
    d = ms.dequantize_rows(q, s)
    # the row maximum maps to 448 exactly; every element is within half a
    # step of the E4M3 grid (relative 2^-4 for normals) of its scaled value
    amax = np.abs(w).max(axis=1)
    for r in range(33):
        if r == 5:
            continue
        assert np.isclose(np.abs(d[r]).max(), amax[r], rtol=1e-6)
        err = np.abs(d[r] - w[r])
        assert np.all(err <= np.maximum(np.abs(w[r]) * 2.0 ** -4, s[r] * 2.0 ** -10) * 1.0001)
