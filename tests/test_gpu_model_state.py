"""T-Offload of model state on the GPU, through the C ABI: quantized weight
reload (FP8 E4M3 codes with row scales expanded on the device) and the host
AdamW update of every streamed layer between iterations, against the
oracle: the oracle runs the same iterations with its own float64 AdamW and
the weights the device computes with (bf16 of the f32 master, or
bf16(decode(q) * scale) of the oracle's quantization of it)."""
import numpy as np
import pytest

from oracle import model_state as ms
from paper_2503_03182_amd import configs as W
from paper_2503_03182_amd import synth
from paper_2503_03182_amd import tpstage as T
from stage_harness import compare, drive_iteration, inputs, read_grads, results, run_oracle, to_dev, to_np

pytestmark = pytest.mark.gpu
BF16_TOL = 2e-2
MATS = ("w_qkv", "w_o", "w_1", "w_2")
# eps large against the gradients keeps the update linear in them, so the
# bf16-level gradient differences of the two sides stay small in the update
HP = dict(lr=0.05, beta1=0.9, beta2=0.95, eps=1.0, weight_decay=0.1)


def test_dequant_kernel_bitexact():
    import torch
    rng = np.random.default_rng(3)
    rows, cols = 300, 520
    codes = rng.integers(0, 256, size=(rows, cols)).astype(np.uint8)
    codes[(codes & 0x7F) == 0x7F] = 0x12          # no NaN codes
    scale = (rng.random(rows).astype(np.float32) * 0.01 + 1e-4).astype(np.float32)
    q = torch.from_numpy(codes).cuda()
    s = torch.from_numpy(scale).cuda()
    out = torch.empty(rows, cols, dtype=torch.bfloat16, device="cuda")
    T.op_dequant_fp8_rows(rows, cols, q, s, out)
    torch.cuda.synchronize()
    ref = synth.round_to_storage(ms.dequantize_rows(codes, scale).astype(np.float32), "bf16")
    got = out.float().cpu().numpy()
    assert np.array_equal(got, ref)


def _cfg(quant, **kw):
    L = 3
    base = dict(n_layers=L, hidden=512, n_heads=4, mlp=2048, seq=200, micro_batch=2, n_micro=3, dtype="bf16",
                policy=W.policy_layer_inputs(L), granularity=T.GRAN_LAYER, weights=T.W_STREAM, window=2,
                weights_quant=quant)
    base.update(kw)
    return T.StageConfig(**base)


def _master_blocks(cfg):
    """Per-layer f32 master blocks in the gradient layout from the synthetic
    parameters."""
    po, pb, go, gb = T.param_layout(cfg)
    out = []
    for l in range(cfg.n_layers):
        vals = synth.layer_params(l, cfg.hidden, cfg.mlp, "f32")
        blk = np.zeros(gb // 4, dtype=np.float32)
        for i, n in enumerate(T.PARAMS):
            v = vals[n].reshape(-1).astype(np.float32)
            blk[go[i] // 4: go[i] // 4 + v.size] = v
        out.append(blk)
    return out


def _unpack(cfg, blk):
    po, pb, go, gb = T.param_layout(cfg)
    shapes = synth.param_shapes(cfg.hidden, cfg.mlp)
    return {n: blk[go[i] // 4: go[i] // 4 + int(np.prod(shapes[n]))].reshape(shapes[n]).astype(np.float64)
            for i, n in enumerate(T.PARAMS)}


def _device_weights(cfg, master32: dict) -> dict:
    """The weights the device computes with, from f32 master values."""
    out = {}
    for n, w in master32.items():
        w32 = np.asarray(w, dtype=np.float32)
        if cfg.weights_quant == T.Q_FP8_ROW and n in MATS:
            q, s = ms.quantize_rows(w32)
            w32 = ms.dequantize_rows(q, s).astype(np.float32)
        out[n] = synth.round_to_storage(w32, "bf16").astype(np.float64)
    return out


def _host_param_blocks(cfg, masters):
    import torch
    nbytes = T.param_layout_q(cfg)[2] if cfg.weights_quant == T.Q_FP8_ROW else T.param_layout(cfg)[1]
    blocks = []
    for mblk in masters:
        hb = torch.zeros(nbytes, dtype=torch.uint8, pin_memory=True)
        T.host_adamw_layer(cfg, 0, mblk, None, None, None, hb, quant=cfg.weights_quant)
        blocks.append(hb)
    return blocks


@pytest.mark.parametrize("quant", [T.Q_NONE, T.Q_FP8_ROW])
def test_reloaded_weights_match_oracle(quant):
    import torch
    for group in (False, True):
        cfg = _cfg(quant)
        masters = _master_blocks(cfg)
        blocks = _host_param_blocks(cfg, masters)
        gb = T.param_layout(cfg)[3]
        grads = [torch.zeros(gb, dtype=torch.uint8, pin_memory=True) for _ in range(cfg.n_layers)]
        xs, dys = inputs(cfg)
        st = T.Stage(cfg, blocks, grads)
        X = [to_dev(x, cfg.dtype) for x in xs]
        DY = [to_dev(d, cfg.dtype) for d in dys]
        Y = [torch.empty_like(x) for x in X]
        DX = [torch.empty_like(x) for x in X]
        drive_iteration(st, cfg, X, DY, Y, DX, group=group)
        out = results(cfg, st, Y, DX, grads)
        st.close()
        ora_params = [_device_weights(cfg, {n: v.astype(np.float32) for n, v in _unpack(cfg, m).items()})
                      for m in masters]
        ref = run_oracle(cfg, xs, dys, ora_params=ora_params)
        worst, bad = compare(out, ref, BF16_TOL)
        assert not bad, (quant, group, bad)


def _check_steps(cfg, xs, dys, outs, states, weights_cfg=None, tol=5e-2):
    """Each iteration i against the oracle's iteration on the weights the
    device computed with (from its master weights before the iteration,
    states[i]), and each update: the device's master weights after the
    iteration (states[i + 1]) against the oracle's float64 AdamW step from the
    device's state before it with the oracle's gradients.  Starting every step
    from the device's own state keeps FP8 codes of weights at a rounding
    boundary from flipping between two diverging trajectories.
    weights_cfg(l): the config whose storage rules layer l's weights follow."""
    L = cfg.n_layers
    wcfg = weights_cfg or (lambda l: cfg)
    for it, got in enumerate(outs):
        mst = [_unpack(cfg, b) for b in states[it][0]]
        ora_params = [_device_weights(wcfg(l), {n: v.astype(np.float32) for n, v in mst[l].items()})
                      for l in range(L)]
        ref = run_oracle(cfg, xs, dys, ora_params=ora_params)
        got = dict(got)
        got["grads"] = [ref["grads"][l] if got["grads"][l] is None else got["grads"][l] for l in range(L)]
        worst, bad = compare(got, ref, BF16_TOL)
        assert not bad, (it, bad)
        mo = [_unpack(cfg, b) for b in states[it][1]]
        vo = [_unpack(cfg, b) for b in states[it][2]]
        after = [_unpack(cfg, b) for b in states[it + 1][0]]
        for l in range(L):
            for n in T.PARAMS:
                exp, _, _ = ms.adamw_step(mst[l][n], mo[l][n], vo[l][n], ref["grads"][l][n], it + 1, **HP)
                du, dr = after[l][n] - mst[l][n], exp - mst[l][n]
                rel = np.linalg.norm(du - dr) / max(np.linalg.norm(dr), 1e-30)
                # bf16-level gradient differences carry into the update
                # linearly (the k part of the qkv bias has an exactly zero
                # true gradient, so its rounding noise is all relative error)
                assert rel < tol, (it, l, n, rel)


@pytest.mark.parametrize("quant", [T.Q_NONE, T.Q_FP8_ROW])
@pytest.mark.parametrize("group", [False, True])
def test_host_optimizer_iterations_match_oracle(quant, group):
    """Two iterations with the stage's host AdamW between them: the second
    iteration runs on the updated (and reloaded) weights and matches the
    oracle's second iteration; the master weights after both updates match
    the oracle's."""
    import torch
    cfg = _cfg(quant)
    L = cfg.n_layers
    masters = _master_blocks(cfg)
    m0 = [np.zeros_like(b) for b in masters]
    v0 = [np.zeros_like(b) for b in masters]
    blocks = _host_param_blocks(cfg, masters)
    gb = T.param_layout(cfg)[3]
    grads = [torch.zeros(gb, dtype=torch.uint8, pin_memory=True) for _ in range(L)]
    xs, dys = inputs(cfg)
    st = T.Stage(cfg, blocks, grads)
    st.set_optimizer(masters, m0, v0, first_step=1, n_threads=4, **HP)
    X = [to_dev(x, cfg.dtype) for x in xs]
    DY = [to_dev(d, cfg.dtype) for d in dys]
    Y = [torch.empty_like(x) for x in X]
    DX = [torch.empty_like(x) for x in X]
    snap = lambda: tuple([b.copy() for b in arr] for arr in (masters, m0, v0))
    states = [snap()]
    outs = []
    for _ in range(2):
        drive_iteration(st, cfg, X, DY, Y, DX, group=group)
        outs.append(results(cfg, st, Y, DX, grads))   # waits for the host updates
        states.append(snap())
    st.close()
    # the update reached the device: the second iteration's output moved
    assert any(np.linalg.norm(outs[1]["ys"][mb] - outs[0]["ys"][mb]) > 1e-2 * np.linalg.norm(outs[0]["ys"][mb])
               for mb in range(cfg.n_micro))
    _check_steps(cfg, xs, dys, outs, states)


def _run_split(cfg, n_dev, group, iterations=3, hp=HP):
    """`iterations` iterations with the AdamW of layers < n_dev on the GPU
    (device master, moments and parameter blocks) and of the others on the
    host; returns the per-iteration outputs, input gradients and host
    gradient blocks (None for the device-updated layers, whose blocks stay on
    the device) and the master weights and moments of every layer (numpy)
    before the first and after every iteration."""
    import torch
    L = cfg.n_layers
    masters = _master_blocks(cfg)
    m0 = [np.zeros_like(b) for b in masters]
    v0 = [np.zeros_like(b) for b in masters]
    blocks = _host_param_blocks(cfg, masters)
    gb = T.param_layout(cfg)[3]
    grads = [torch.zeros(gb, dtype=torch.uint8, pin_memory=True) for _ in range(L)]
    xs, dys = inputs(cfg)
    st = T.Stage(cfg, blocks, grads)
    dev = [[torch.from_numpy(b[l]).cuda() for l in range(n_dev)] for b in (masters, m0, v0)]
    # the device parameter blocks start as the host blocks (storage dtype)
    pb = T.param_layout(cfg)[1]
    dpar = [_host_param_blocks(dataclasses_replace_quant(cfg), [masters[l]])[0][:pb].cuda() for l in range(n_dev)]
    pick = lambda d, h: [d[l] if l < n_dev else h[l] for l in range(L)]
    st.set_optimizer(pick(dev[0], masters), pick(dev[1], m0), pick(dev[2], v0), first_step=1, n_threads=4,
                     dparams=dpar, **hp)
    X = [to_dev(x, cfg.dtype) for x in xs]
    DY = [to_dev(d, cfg.dtype) for d in dys]
    Y = [torch.empty_like(x) for x in X]
    DX = [torch.empty_like(x) for x in X]
    snap = lambda: tuple([(d[l].cpu().numpy() if l < n_dev else h[l].copy()) for l in range(L)]
                         for d, h in zip(dev, (masters, m0, v0)))
    states = [snap()]
    outs = []
    for _ in range(iterations):
        drive_iteration(st, cfg, X, DY, Y, DX, group=group)
        out = results(cfg, st, Y, DX, grads)   # waits for the updates
        out["grads"] = [None if l < n_dev else g for l, g in enumerate(out["grads"])]
        outs.append(out)
        states.append(snap())
    st.close()
    return outs, states


def dataclasses_replace_quant(cfg):
    import dataclasses
    return dataclasses.replace(cfg, weights_quant=T.Q_NONE)


@pytest.mark.parametrize("group", [False, True])
def test_device_updated_layers_bitexact_to_host_updates(group):
    """The AdamW of the shallowest layers on the GPU
    (tps_stage_set_optimizer_split) gives the bits of the host update: over
    three iterations with layer 0, then layers 0 and 1, updated on the
    device, the outputs and input gradients of every iteration, the host
    layers' gradient blocks and every layer's master weights and moments
    equal those of the run with every layer updated on the host."""
    cfg = _cfg(T.Q_NONE)
    ref_outs, ref_state = _run_split(cfg, 0, group)
    for n_dev in (1, 2):
        outs, state = _run_split(cfg, n_dev, group)
        for it, (a, b) in enumerate(zip(outs, ref_outs)):
            for mb in range(cfg.n_micro):
                assert np.array_equal(a["ys"][mb], b["ys"][mb]), (n_dev, it, mb)
                assert np.array_equal(a["dxs"][mb], b["dxs"][mb]), (n_dev, it, mb)
        for l in range(n_dev, cfg.n_layers):
            for n in outs[-1]["grads"][l]:
                assert np.array_equal(outs[-1]["grads"][l][n], ref_outs[-1]["grads"][l][n]), (n_dev, l, n)
        for it, (got_s, ref_s) in enumerate(zip(state, ref_state)):
            for k, (got, ref) in enumerate(zip(got_s, ref_s)):
                for l in range(cfg.n_layers):
                    assert np.array_equal(got[l], ref[l]), (n_dev, it, k, l)
        # the updates reached the device
        assert not np.array_equal(outs[1]["ys"][0], outs[0]["ys"][0])


def test_device_updated_layer_with_quantized_reload_matches_oracle():
    """FP8 reload of the host-updated layers with layer 0 updated on the GPU:
    layer 0 computes with bf16 of its master weights, the others with the
    decoded FP8 codes of theirs; both iterations and both updates match the
    oracle's."""
    cfg = _cfg(T.Q_FP8_ROW)
    outs, states = _run_split(cfg, 1, True, iterations=2)
    xs, dys = inputs(cfg)
    bf16_cfg = dataclasses_replace_quant(cfg)
    _check_steps(cfg, xs, dys, outs, states, weights_cfg=lambda l: bf16_cfg if l == 0 else cfg)


def test_device_optimizer_argument_errors():
    import torch
    cfg = _cfg(T.Q_NONE)
    L = cfg.n_layers
    masters = _master_blocks(cfg)
    blocks = _host_param_blocks(cfg, masters)
    gb = T.param_layout(cfg)[3]
    grads = [torch.zeros(gb, dtype=torch.uint8, pin_memory=True) for _ in range(L)]
    st = T.Stage(cfg, blocks, grads)
    zeros = [np.zeros_like(b) for b in masters]
    try:
        with pytest.raises(T.TpsError):   # more device layers than layers
            st.set_optimizer(masters, zeros, zeros, dparams=[blocks[0].cuda()] * (L + 1))
        dm = torch.from_numpy(masters[0]).cuda()
        dz = torch.zeros_like(dm)
        st.set_optimizer([dm] + masters[1:], [dz] + zeros[1:], [dz.clone()] + zeros[1:],
                         dparams=[blocks[0][:T.param_layout(cfg)[1]].cuda()])
        with pytest.raises(T.TpsError) as e:   # device layers need zero_grads
            st.begin_iteration(zero_grads=False)
        assert e.value.code == T.TPS_EINVAL
    finally:
        st.close()
