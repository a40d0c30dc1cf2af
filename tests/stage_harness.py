"""Helpers shared by the GPU tests: marshal synthetic inputs to the device,
run the stage through the C ABI in its planned order, read results back, and
run the CPU oracle on the same (storage-rounded) inputs."""

from __future__ import annotations

import numpy as np

from paper_2503_03182_amd import synth
from paper_2503_03182_amd import tpstage as T


def torch_dtype(dtype: str):
    import torch
    return torch.bfloat16 if dtype == "bf16" else torch.float32


def to_dev(a: np.ndarray, dtype: str):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to("cuda").to(torch_dtype(dtype))


def to_np(t) -> np.ndarray:
    return t.detach().float().cpu().numpy().astype(np.float64)


def rel_l2(a, b) -> float:
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    return float(np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-30))


def is_llama(cfg) -> bool:
    return cfg.arch == T.ARCH_LLAMA


def n_kv(cfg) -> int:
    return cfg.n_kv_heads or cfg.n_heads


def layer_vals(cfg, l):
    """Synthetic parameters of layer l (float32 arrays of storage values)."""
    if is_llama(cfg):
        return synth.llama_layer_params(l, cfg.hidden, cfg.n_heads, n_kv(cfg), cfg.mlp, cfg.dtype)
    return synth.layer_params(l, cfg.hidden, cfg.mlp, cfg.dtype)


def param_shapes(cfg) -> dict:
    if is_llama(cfg):
        return synth.llama_param_shapes(cfg.hidden, cfg.n_heads, n_kv(cfg), cfg.mlp)
    return synth.param_shapes(cfg.hidden, cfg.mlp)


def make_params(cfg):
    """Per-layer packed parameter blocks (device) and zeroed f32 gradient
    blocks, plus the float64 parameter dicts for the oracle."""
    import torch
    po, pb, go, gb = T.param_layout(cfg)
    es = 2 if cfg.dtype == "bf16" else 4
    blocks, grads, ora = [], [], []
    stream_host = cfg.weights == T.W_STREAM
    for l in range(cfg.n_layers):
        vals = layer_vals(cfg, l)
        blk = torch.zeros(pb, dtype=torch.uint8, device="cuda")
        for i, name in enumerate(T.PARAMS):
            if name not in vals:
                continue
            v = to_dev(vals[name].reshape(-1), cfg.dtype)
            n = v.numel()
            blk[po[i]:po[i] + n * es].view(torch_dtype(cfg.dtype)).copy_(v)
        if stream_host:
            hb = torch.empty(pb, dtype=torch.uint8, pin_memory=True)
            hb.copy_(blk)
            blk = hb
            g = torch.zeros(gb, dtype=torch.uint8, pin_memory=True)
        else:
            g = torch.zeros(gb, dtype=torch.uint8, device="cuda")
        blocks.append(blk)
        grads.append(g)
        ora.append({k: v.astype(np.float64) for k, v in vals.items()})
    return blocks, grads, ora


def read_grads(cfg, grads):
    import torch
    po, pb, go, gb = T.param_layout(cfg)
    shapes = param_shapes(cfg)
    out = []
    for g in grads:
        d = {}
        for i, name in enumerate(T.PARAMS):
            if name not in shapes:
                continue
            n = int(np.prod(shapes[name]))
            d[name] = g[go[i]:go[i] + 4 * n].view(torch.float32).cpu().numpy().astype(np.float64).reshape(shapes[name])
        out.append(d)
    return out


def inputs(cfg):
    xs = [synth.stage_input(mb, cfg.tokens, cfg.hidden, cfg.dtype) for mb in range(cfg.n_micro)]
    dys = [synth.output_grad(mb, cfg.tokens, cfg.hidden, cfg.dtype) for mb in range(cfg.n_micro)]
    return xs, dys


def drive_iteration(st, cfg, X, DY, Y, DX, group=False, calls=None):
    """One iteration of the planned order through the C ABI.  group: each run
    of consecutive micro-batches with the same task kind is one group call.
    calls: explicit [(kind, [mbs], as_group)] (kind "F" or "B"), for mixing
    per-micro-batch and group calls."""
    st.begin_iteration(zero_grads=True)
    if calls is None:
        calls = []
        if group:
            for k, mb0, n in cfg.groups():
                calls.append((k, list(range(mb0, mb0 + n)), True))
        else:
            calls = [(k, [mb], False) for k, mb in cfg.order()]
    for k, mbs, as_group in calls:
        if as_group:
            if k == "F":
                st.forward_group(mbs[0], [X[m] for m in mbs], [Y[m] for m in mbs])
            else:
                st.backward_group(mbs[0], [DY[m] for m in mbs], [DX[m] for m in mbs])
        else:
            for mb in mbs:
                if k == "F":
                    st.forward(mb, X[mb], Y[mb])
                else:
                    st.backward(mb, DY[mb], DX[mb])


def results(cfg, st, Y, DX, grads):
    """numpy copies of the outputs and gradient blocks (waits for the stage)."""
    st.sync()
    return dict(ys=[to_np(y) for y in Y], dxs=[to_np(d) for d in DX], grads=read_grads(cfg, grads),
                stats=st.stats(), plan=st.info)


def run_gpu(cfg, xs=None, dys=None, iterations=1, group=False, params=None, one_copy_stream=False, calls=None):
    """Runs `iterations` iterations of the planned order; returns numpy results
    of the last one: dict(ys, dxs, grads, stats, plan).  one_copy_stream: both
    host-link directions on one stream (no prefetch stream of their own)."""
    import torch
    if xs is None:
        xs, dys = inputs(cfg)
    blocks, grads, _ = params if params is not None else make_params(cfg)
    if one_copy_stream:
        xs_ = torch.cuda.Stream()
        st = T.Stage(cfg, blocks, grads, copy_stream=xs_, prefetch_stream=xs_)
    else:
        st = T.Stage(cfg, blocks, grads)
    X = [to_dev(x, cfg.dtype) for x in xs]
    DY = [to_dev(d, cfg.dtype) for d in dys]
    Y = [torch.empty_like(x) for x in X]
    DX = [torch.empty_like(x) for x in X]
    torch.cuda.synchronize()
    for _ in range(iterations):
        drive_iteration(st, cfg, X, DY, Y, DX, group=group, calls=calls)
        st.sync()
    out = dict(ys=[to_np(y) for y in Y], dxs=[to_np(d) for d in DX], grads=read_grads(cfg, grads),
               stats=st.stats(), plan=st.info)
    st.close()
    return out


def run_oracle(cfg, xs=None, dys=None, ora_params=None):
    from oracle import decoder_stage as ora
    from oracle import llama_stage as lla
    if xs is None:
        xs, dys = inputs(cfg)
    if ora_params is None:
        ora_params = [{k: v.astype(np.float64) for k, v in layer_vals(cfg, l).items()} for l in range(cfg.n_layers)]
    xs = [x.astype(np.float64) for x in xs]
    dys = [d.astype(np.float64) for d in dys]
    if is_llama(cfg):
        return lla.run_stage(ora_params, xs, dys, cfg.n_heads, n_kv(cfg), cfg.micro_batch, cfg.seq, cfg.ln_eps,
                             cfg.rope_base)
    return ora.run_stage(ora_params, xs, dys, cfg.n_heads, cfg.micro_batch, cfg.seq, cfg.ln_eps)


def tile_excess(a, b, tol, tile=256) -> float:
    """Per-tile bound beside the per-tensor rel-L2: for every tile (256 x 256
    of a matrix, 256 elements of a vector) the error norm must stay within
    tol times the larger of the tile's own reference norm and its fair share
    of the tensor's reference norm (||ref|| * sqrt(tile size / size)).
    Returns the worst ratio error / bound (<= 1 passes): a single tile
    carrying a large error fails even when the whole tensor's rel-L2 passes."""
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    if a.ndim == 1:
        a, b = a[None, :], b[None, :]
    a = a.reshape(-1, a.shape[-1])
    b = b.reshape(-1, b.shape[-1])
    rows, cols = b.shape
    tr = tile if rows > 1 else 1
    total = float(np.linalg.norm(b))
    n = b.size
    worst = 0.0
    for r0 in range(0, rows, tr):
        for c0 in range(0, cols, tile):
            rb = b[r0:r0 + tr, c0:c0 + tile]
            ra = a[r0:r0 + tr, c0:c0 + tile]
            err = float(np.linalg.norm(ra - rb))
            bound = tol * max(float(np.linalg.norm(rb)), total * np.sqrt(rb.size / n), 1e-30)
            worst = max(worst, err / bound)
    return worst


def assert_close(got, ref, tol, what=""):
    """Parity bar of one tensor: rel-L2 below tol and every tile within the
    per-tile bound of tile_excess."""
    r = rel_l2(got, ref)
    assert r < tol, f"{what} rel-L2 {r:.3g} >= {tol:g}"
    t = tile_excess(got, ref, tol)
    assert t <= 1.0, f"{what} worst tile at {t:.3g} x its bound (tol {tol:g})"


def compare(gpu, ref, tol, tiles=True):
    """Worst rel-L2 over y, dx of every micro-batch and every parameter grad;
    with tiles, also the per-tile bound of tile_excess (reported as
    "<name>@tile", failing above 1)."""
    worst, tile_worst = {}, {}
    pairs = []
    for mb in range(len(ref["ys"])):
        pairs.append((f"y{mb}", gpu["ys"][mb], ref["ys"][mb]))
        pairs.append((f"dx{mb}", gpu["dxs"][mb], ref["dxs"][mb]))
    for l, g in enumerate(ref["grads"]):
        for k, v in g.items():
            pairs.append((f"L{l}.{k}", gpu["grads"][l][k], v))
    for name, a, b in pairs:
        worst[name] = rel_l2(a, b)
        if tiles:
            tile_worst[name] = tile_excess(a, b, tol)
    bad = {k: v for k, v in worst.items() if not v <= tol}
    bad.update({f"{k}@tile": v for k, v in tile_worst.items() if not v <= 1.0})
    return worst, bad


def bit_equal(a, b) -> list:
    """Names of outputs that differ bitwise between two GPU runs."""
    diff = []
    for mb in range(len(a["ys"])):
        if not np.array_equal(a["ys"][mb], b["ys"][mb]):
            diff.append(f"y{mb}")
        if not np.array_equal(a["dxs"][mb], b["dxs"][mb]):
            diff.append(f"dx{mb}")
    for l in range(len(a["grads"])):
        for k in a["grads"][l]:
            if not np.array_equal(a["grads"][l][k], b["grads"][l][k]):
                diff.append(f"L{l}.{k}")
    return diff
