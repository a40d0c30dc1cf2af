"""Host side of T-Offload's model-state path (tps_host_adamw_layer, host
only): the f32 AdamW update against the float64 oracle, and the parameter
block it writes for the device (bf16 rounding, or FP8 E4M3 codes with row
scales) bit-exact against the oracle's encoding of the same f32 values."""
import numpy as np
import pytest

from oracle import model_state as ms
from paper_2503_03182_amd import synth
from paper_2503_03182_amd import tpstage as T


def _cfg():
    return T.StageConfig(n_layers=1, hidden=256, n_heads=2, mlp=512, seq=16, micro_batch=1, n_micro=1,
                         dtype="bf16", weights=T.W_STREAM, window=2)


def _block(cfg, vals, offsets, nbytes, dtype=np.float32):
    out = np.zeros(nbytes // 4, dtype=np.float32)
    for i, name in enumerate(T.PARAMS):
        v = vals[name].reshape(-1).astype(np.float32)
        out[offsets[i] // 4: offsets[i] // 4 + v.size] = v
    return out


def _unpack(cfg, block, offsets):
    shapes = synth.param_shapes(cfg.hidden, cfg.mlp)
    return {n: block[offsets[i] // 4: offsets[i] // 4 + int(np.prod(shapes[n]))].reshape(shapes[n]).astype(np.float64)
            for i, n in enumerate(T.PARAMS)}


def bf16_bits_rne(x32):
    b = np.asarray(x32, dtype=np.float32).view(np.uint32).astype(np.uint64)
    return ((b + 0x7FFF + ((b >> 16) & 1)) >> 16).astype(np.uint16)


HP = dict(lr=2e-3, beta1=0.9, beta2=0.95, eps=1e-8, weight_decay=0.05)


@pytest.mark.parametrize("quant", [T.Q_NONE, T.Q_FP8_ROW])
def test_host_adamw_matches_oracle_and_writes_the_device_block(quant):
    cfg = _cfg()
    po, pb, go, gb = T.param_layout(cfg)
    qo, so, qb = T.param_layout_q(cfg)
    shapes = synth.param_shapes(cfg.hidden, cfg.mlp)
    rng = np.random.default_rng(5)
    w0 = {n: (rng.standard_normal(shapes[n]) * 0.05).astype(np.float32) for n in T.PARAMS}
    master = _block(cfg, w0, go, gb)
    m = np.zeros_like(master)
    v = np.zeros_like(master)
    ora_w = {n: w0[n].astype(np.float64) for n in T.PARAMS}
    ora_m = {n: np.zeros(shapes[n]) for n in T.PARAMS}
    ora_v = {n: np.zeros(shapes[n]) for n in T.PARAMS}
    out = np.zeros(qb if quant == T.Q_FP8_ROW else pb, dtype=np.uint8)
    for step in (1, 2, 3):
        g = {n: (rng.standard_normal(shapes[n]) * 0.01).astype(np.float32) for n in T.PARAMS}
        grad = _block(cfg, g, go, gb)
        T.host_adamw_layer(cfg, step, master, m, v, grad, out, quant=quant, n_threads=4, **HP)
        for n in T.PARAMS:
            ora_w[n], ora_m[n], ora_v[n] = ms.adamw_step(ora_w[n], ora_m[n], ora_v[n], g[n], step, **HP)
        got = _unpack(cfg, master, go)
        for n in T.PARAMS:
            err = np.abs(got[n] - ora_w[n]).max()
            assert err <= 1e-6 * (1 + np.abs(ora_w[n]).max()), (step, n, err)
        gm, gv = _unpack(cfg, m, go), _unpack(cfg, v, go)
        for n in T.PARAMS:
            assert np.allclose(gm[n], ora_m[n], rtol=1e-5, atol=1e-9)
            assert np.allclose(gv[n], ora_v[n], rtol=1e-5, atol=1e-12)
    # the block for the device, from the library's own f32 master weights
    w32 = {n: _unpack(cfg, master, go)[n].astype(np.float32) for n in T.PARAMS}
    mats = ("w_qkv", "w_o", "w_1", "w_2")
    for i, n in enumerate(T.PARAMS):
        size = int(np.prod(shapes[n]))
        if quant == T.Q_FP8_ROW and n in mats:
            k = mats.index(n)
            codes = out[qo[i]: qo[i] + size].reshape(shapes[n])
            scales = out[so[k]: so[k] + 4 * shapes[n][0]].view(np.float32)
            q_ref, s_ref = ms.quantize_rows(w32[n])
            assert np.array_equal(scales, s_ref), n
            assert np.array_equal(codes, q_ref), n
        else:
            off = qo[i] if quant == T.Q_FP8_ROW else po[i]
            bits = out[off: off + 2 * size].view(np.uint16)
            assert np.array_equal(bits, bf16_bits_rne(w32[n].reshape(-1))), n


def test_step_zero_only_writes_the_block():
    cfg = _cfg()
    po, pb, go, gb = T.param_layout(cfg)
    rng = np.random.default_rng(6)
    shapes = synth.param_shapes(cfg.hidden, cfg.mlp)
    w0 = {n: (rng.standard_normal(shapes[n]) * 0.05).astype(np.float32) for n in T.PARAMS}
    master = _block(cfg, w0, go, gb)
    before = master.copy()
    out = np.zeros(pb, dtype=np.uint8)
    T.host_adamw_layer(cfg, 0, master, None, None, None, out)
    assert np.array_equal(master, before)
    for i, n in enumerate(T.PARAMS):
        size = int(np.prod(shapes[n]))
        assert np.array_equal(out[po[i]: po[i] + 2 * size].view(np.uint16), bf16_bits_rne(w0[n].reshape(-1)))


def test_host_adamw_argument_errors():
    cfg = _cfg()
    po, pb, go, gb = T.param_layout(cfg)
    buf = np.zeros(gb // 4, dtype=np.float32)
    out = np.zeros(pb, dtype=np.uint8)
    with pytest.raises(T.TpsError):
        T.host_adamw_layer(cfg, -1, buf, buf, buf, buf, out)
    with pytest.raises(T.TpsError):
        T.host_adamw_layer(cfg, 1, buf, None, buf, buf, out)
    with pytest.raises(T.TpsError):
        T.host_adamw_layer(cfg, 1, buf, buf.copy(), buf.copy(), buf, out, beta1=1.5)
    f32 = T.StageConfig(**{**_cfg().__dict__, "dtype": "f32", "_keep": []})
    with pytest.raises(T.TpsError):
        T.host_adamw_layer(f32, 0, buf, None, None, None, out, quant=T.Q_FP8_ROW)


def test_fp8_encoding_at_every_code_midpoint_and_boundary():
    """The library's E4M3 encoder (branch-free, in the quantized block) against
    the oracle's nearest-code search on every code value, every midpoint
    between neighbouring codes (ties), one f32 step either side of each
    midpoint, the subnormal/normal boundary and values beyond 448.  A row
    whose largest magnitude is 448 has scale 1, so the encoder sees the
    values themselves."""
    cfg = _cfg()
    po, pb, go, gb = T.param_layout(cfg)
    qo, so, qb = T.param_layout_q(cfg)
    shapes = synth.param_shapes(cfg.hidden, cfg.mlp)
    vals = ms.e4m3_values()
    pos = np.sort(np.array([v for v in vals[:128] if not np.isnan(v)]))
    mids = (pos[:-1] + pos[1:]) / 2
    f32 = lambda a: np.asarray(a, dtype=np.float32)
    probes = np.concatenate([pos, mids, np.nextafter(f32(mids), f32(0)), np.nextafter(f32(mids), f32(1e9)),
                             [2.0 ** -6, np.nextafter(np.float32(2.0 ** -6), np.float32(0)), 2.0 ** -9 / 2,
                              2.0 ** -10, 1e-30, 0.0, 447.99, 464.0, 500.0, 1e6]]).astype(np.float32)
    probes = np.concatenate([probes, -probes])
    rows, cols = shapes["w_1"]
    w = np.zeros((rows, cols), dtype=np.float32)
    flat = np.concatenate([probes, np.zeros((-probes.size) % (cols - 1), dtype=np.float32)])
    chunks = flat.reshape(-1, cols - 1)
    assert chunks.shape[0] <= rows
    w[:chunks.shape[0], :cols - 1] = chunks
    w[:chunks.shape[0], cols - 1] = 448.0          # scale 1 for these rows (values above 448 saturate)
    vals_in = {n: np.zeros(shapes[n], dtype=np.float32) for n in T.PARAMS}
    vals_in["w_1"] = w
    master = _block(cfg, vals_in, go, gb)
    out = np.zeros(qb, dtype=np.uint8)
    T.host_adamw_layer(cfg, 0, master, None, None, None, out, quant=T.Q_FP8_ROW, n_threads=2)
    i = T.PARAMS.index("w_1")
    codes = out[qo[i]: qo[i] + rows * cols].reshape(rows, cols)
    scales = out[so[2]: so[2] + 4 * rows].view(np.float32)
    n = chunks.shape[0]
    # rows holding a value above 448 have a larger scale; compare through the oracle's own quantization
    q_ref, s_ref = ms.quantize_rows(w[:n])
    assert np.array_equal(scales[:n], s_ref)
    assert np.array_equal(codes[:n], q_ref)
    assert (scales[:n] == 1.0).sum() >= n - 2
