"""Whole-stage parity through the C ABI: the HIP path against the CPU oracle
(f32: rel-L2 <= 1e-4, bf16: rel-L2 <= 2e-2 on y, dx and every parameter
gradient), and bit-exactness of the HIP path across keep / recompute /
offload policies, op orders, group calls and streamed weights."""

import dataclasses

import numpy as np
import pytest

from paper_2503_03182_amd import configs as W
from paper_2503_03182_amd import tpstage as T

from stage_harness import bit_equal, compare, inputs, read_grads, run_gpu, run_oracle, to_np

pytestmark = pytest.mark.gpu

F32_TOL = 1e-4
BF16_TOL = 2e-2


def test_tiny_f32_three_policies_match_oracle_and_each_other():
    ref = run_oracle(W.tiny())
    outs = {}
    for pol in ("keep", "recompute", "offload"):
        cfg = W.tiny(pol)
        outs[pol] = run_gpu(cfg)
        worst, bad = compare(outs[pol], ref, F32_TOL)
        assert not bad, (pol, bad)
    assert outs["recompute"]["stats"]["replays"] > 0
    assert outs["offload"]["stats"]["d2h_bytes"] > 0 and outs["offload"]["stats"]["h2d_bytes"] > 0
    assert bit_equal(outs["keep"], outs["recompute"]) == []
    assert bit_equal(outs["keep"], outs["offload"]) == []


def _mid(**kw):
    base = dict(n_layers=3, hidden=512, n_heads=4, mlp=2048, seq=200, micro_batch=2, n_micro=3, dtype="bf16")
    base.update(kw)
    return T.StageConfig(**base)


def test_bf16_stage_matches_oracle():
    cfg = _mid(policy=W.policy_selective(3))
    gpu = run_gpu(cfg)
    ref = run_oracle(cfg)
    worst, bad = compare(gpu, ref, BF16_TOL)
    assert not bad, bad


def test_bf16_bitexact_across_policies_orders_and_groups():
    L, M = 3, 3
    order = [("F", 0), ("F", 1), ("B", 0), ("F", 2), ("B", 1), ("B", 2)]
    keep = run_gpu(_mid(ops=order))
    mixed = [{t: [T.KEEP, T.RECOMPUTE, T.OFFLOAD][(l + i) % 3] for i, t in enumerate(T.TENSORS)} for l in range(L)]
    mixed[0]["x"] = T.KEEP
    variants = {
        "selective": _mid(ops=order, policy=W.policy_selective(L)),
        "layer_inputs_segment": _mid(ops=order, policy=W.policy_layer_inputs(L), granularity=T.GRAN_SEGMENT),
        "layer_inputs_layer": _mid(ops=order, policy=W.policy_layer_inputs(L), granularity=T.GRAN_LAYER),
        "recompute_all": _mid(ops=order, policy=W.policy_all(L, T.RECOMPUTE)),
        "offload_all": _mid(ops=order, policy=W.policy_all(L, T.OFFLOAD), offload_mb_mask=0b111),
        "offload_one_lookahead2": _mid(ops=order, policy=W.policy_all(L, T.OFFLOAD), offload_mb_mask=0b100,
                                       lookahead=2),
        "mixed": _mid(ops=order, policy=mixed, offload_mb_mask=0b101),
    }
    for name, cfg in variants.items():
        out = run_gpu(cfg)
        assert bit_equal(keep, out) == [], name
    # offloads and prefetches sharing one copy stream
    out = run_gpu(variants["offload_all"], one_copy_stream=True)
    assert bit_equal(keep, out) == []
    # same stage, all forwards first: per-mb results do not depend on the order
    assert bit_equal(keep, run_gpu(_mid())) == []
    # layer-major group calls
    grp = run_gpu(_mid(policy=W.policy_layer_inputs(L), granularity=T.GRAN_LAYER), group=True)
    assert bit_equal(keep, grp) == []


def test_streamed_weights_bitexact_to_resident():
    L = 4
    resident = run_gpu(_mid(n_layers=L, policy=W.policy_layer_inputs(L), granularity=T.GRAN_LAYER))
    for window in (2, 3):
        cfg = _mid(n_layers=L, policy=W.policy_layer_inputs(L), granularity=T.GRAN_LAYER, weights=T.W_STREAM,
                   window=window)
        for group in (False, True):
            out = run_gpu(cfg, group=group)
            assert bit_equal(resident, out) == [], (window, group)
            assert out["stats"]["h2d_bytes"] > 0 and out["stats"]["d2h_bytes"] > 0
        assert bit_equal(resident, run_gpu(cfg, one_copy_stream=True)) == [], (window, "one copy stream")


def test_wgrad_inline_bitexact_to_side_stream():
    """Parameter-gradient kernels inline on the compute stream give the same
    bits as on their own stream (same kernels, same accumulation order)."""
    L = 4
    order = [("F", 0), ("F", 1), ("B", 0), ("F", 2), ("B", 1), ("B", 2)]
    cases = {
        "keep": (_mid(n_layers=L, ops=order), False),
        "selective": (_mid(n_layers=L, policy=W.policy_selective(L)), False),
        "offload": (_mid(n_layers=L, ops=order, policy=W.policy_all(L, T.OFFLOAD), offload_mb_mask=0b101), False),
        "streamed_groups": (_mid(n_layers=L, policy=W.policy_layer_inputs(L), granularity=T.GRAN_LAYER,
                                 weights=T.W_STREAM, window=2), True),
    }
    for name, (cfg, group) in cases.items():
        side = run_gpu(dataclasses.replace(cfg, wgrad_stream=T.WGRAD_SIDE), group=group)
        inline = run_gpu(dataclasses.replace(cfg, wgrad_stream=T.WGRAD_INLINE), group=group)
        assert bit_equal(side, inline) == [], name


def test_poison_leaves_results_unchanged(monkeypatch):
    """TPS_POISON fills dead slots, replay buffers and evicted transposes with
    NaN as they are handed back; no read escapes the protocol, so the results
    stay bit-identical."""
    L = 4
    order = [("F", 0), ("F", 1), ("B", 0), ("F", 2), ("B", 1), ("B", 2)]
    cases = {
        "selective": (_mid(n_layers=L, ops=order, policy=W.policy_selective(L)), False),
        "offload": (_mid(n_layers=L, ops=order, policy=W.policy_all(L, T.OFFLOAD), offload_mb_mask=0b101,
                         lookahead=2), False),
        "segment": (_mid(n_layers=L, policy=W.policy_layer_inputs(L), granularity=T.GRAN_SEGMENT), False),
        "streamed_groups": (_mid(n_layers=L, policy=W.policy_layer_inputs(L), granularity=T.GRAN_LAYER,
                                 weights=T.W_STREAM, window=2), True),
    }
    plain = {name: run_gpu(cfg, group=group, iterations=2) for name, (cfg, group) in cases.items()}
    monkeypatch.setenv("TPS_POISON", "1")
    for name, (cfg, group) in cases.items():
        for mode in (T.WGRAD_SIDE, T.WGRAD_INLINE):
            out = run_gpu(dataclasses.replace(cfg, wgrad_stream=mode), group=group, iterations=2)
            assert bit_equal(plain[name], out) == [], (name, mode)


def _same_outputs_close_grads(a, b, tol=1e-5):
    """ys and dxs bitwise equal; weight and vector gradients within tol
    (rel-L2): only the f32 summation order of the weight gradients differs."""
    from stage_harness import rel_l2
    for mb in range(len(a["ys"])):
        assert np.array_equal(a["ys"][mb], b["ys"][mb]), f"y{mb}"
        assert np.array_equal(a["dxs"][mb], b["dxs"][mb]), f"dx{mb}"
    for l in range(len(a["grads"])):
        for k, v in a["grads"][l].items():
            r = rel_l2(b["grads"][l][k], v)
            assert r <= tol, (l, k, r)


def test_batched_group_weight_gradients():
    """Backward groups that issue each weight-gradient product once per layer
    over the group's micro-batches: outputs bit-identical to per-micro-batch
    products, weight gradients equal up to f32 summation order, and within
    the bf16 bar of the oracle; a layer that keeps one of its operands (not
    batchable) next to batchable ones; groups of some of the micro-batches."""
    L = 4
    pol = W.policy_layer_inputs(L)
    mixed = [dict(q) for q in pol]
    mixed[1]["c"] = T.KEEP
    cases = {
        "resident": _mid(n_layers=L, policy=pol, granularity=T.GRAN_LAYER),
        "mixed": _mid(n_layers=L, policy=mixed, granularity=T.GRAN_LAYER),
        "streamed": _mid(n_layers=L, policy=pol, granularity=T.GRAN_LAYER, weights=T.W_STREAM, window=2),
    }
    for name, cfg in cases.items():
        per_mb = run_gpu(cfg, group=True)
        for mode in (T.WGRAD_SIDE, T.WGRAD_INLINE):
            bcfg = dataclasses.replace(cfg, group_wgrad=1, wgrad_stream=mode)
            assert T.plan(bcfg)["group_wgrad_slots"] == cfg.n_micro
            bat = run_gpu(bcfg, group=True)
            _same_outputs_close_grads(per_mb, bat)
        worst, bad = compare(bat, run_oracle(cfg), BF16_TOL)
        assert not bad, (name, bad)
    cfg = dataclasses.replace(cases["resident"], n_micro=4)
    calls = [("F", [0, 1, 2, 3], True), ("B", [0, 1], True), ("B", [2], False), ("B", [3], True)]
    per_mb = run_gpu(cfg, calls=calls)
    bat = run_gpu(dataclasses.replace(cfg, group_wgrad=1), calls=calls, iterations=2)
    _same_outputs_close_grads(per_mb, bat)


def test_repeat_iterations_reproduce():
    cfg = _mid(policy=W.policy_all(3, T.OFFLOAD), offload_mb_mask=0b011, inflight=2)
    one = run_gpu(cfg, iterations=1)
    three = run_gpu(cfg, iterations=3)
    assert bit_equal(one, three) == []
    # host slots reused across iterations by offloads (copy stream) and
    # prefetches (prefetch stream) in both orders
    assert bit_equal(one, run_gpu(cfg, iterations=3, one_copy_stream=True)) == []


def test_gradient_accumulation_across_iterations():
    """zero_grads=False adds the iteration's gradients to the blocks; a later
    zero_grads=True restarts them (bit-identical to a fresh first iteration)."""
    import torch
    from stage_harness import make_params, read_grads, to_dev
    for weights in (T.W_RESIDENT, T.W_STREAM):
        cfg = _mid(weights=weights, window=2) if weights == T.W_STREAM else _mid()
        xs, dys = inputs(cfg)
        blocks, grads, _ = make_params(cfg)
        st = T.Stage(cfg, blocks, grads)
        X = [to_dev(x, cfg.dtype) for x in xs]
        DY = [to_dev(d, cfg.dtype) for d in dys]
        Y = [torch.empty_like(x) for x in X]
        DX = [torch.empty_like(x) for x in X]
        snaps = []
        for zero in (True, False, True):
            st.begin_iteration(zero_grads=zero)
            for k, mb in cfg.order():
                if k == "F":
                    st.forward(mb, X[mb], Y[mb])
                else:
                    st.backward(mb, DY[mb], DX[mb])
            st.sync()
            snaps.append(read_grads(cfg, grads))
        st.close()
        for l in range(cfg.n_layers):
            for name, g1 in snaps[0][l].items():
                g2 = snaps[1][l][name]
                assert np.linalg.norm(g2 - 2 * g1) <= 1e-5 * np.linalg.norm(g1), (weights, l, name)
                assert np.array_equal(snaps[2][l][name], g1), (weights, l, name)


def test_linearity_in_dy_bitwise():
    cfg = _mid(policy=W.policy_selective(3))
    xs, dys = inputs(cfg)
    a = run_gpu(cfg, xs, dys)
    b = run_gpu(cfg, xs, [2.0 * d for d in dys])
    for mb in range(cfg.n_micro):
        assert np.array_equal(2.0 * a["dxs"][mb], b["dxs"][mb])
    for l in range(cfg.n_layers):
        for k in T.PARAMS:
            assert np.array_equal(2.0 * a["grads"][l][k], b["grads"][l][k]), (l, k)


def test_causality_bitwise():
    cfg = _mid(n_micro=1, policy=W.policy_selective(3))
    xs, dys = inputs(cfg)
    a = run_gpu(cfg, xs, dys)
    x2 = [xs[0].copy()]
    t = 123
    x2[0][t] = -x2[0][t]
    b = run_gpu(cfg, x2, dys)
    assert np.array_equal(a["ys"][0][:t], b["ys"][0][:t])
    assert not np.array_equal(a["ys"][0][t], b["ys"][0][t])
    s = cfg.seq
    assert np.array_equal(a["ys"][0][s:], b["ys"][0][s:])     # other sequence untouched


def test_order_errors():
    import torch
    from stage_harness import make_params, to_dev
    cfg = W.tiny()
    blocks, grads, _ = make_params(cfg)
    st = T.Stage(cfg, blocks, grads)
    xs, dys = inputs(cfg)
    X = to_dev(xs[0], cfg.dtype)
    Y = torch.empty_like(X)
    with pytest.raises(T.TpsError) as e:
        st.forward(0, X, Y)
    assert e.value.code == T.TPS_ESTATE
    st.begin_iteration()
    with pytest.raises(T.TpsError) as e:
        st.backward(0, X, Y)
    assert e.value.code == T.TPS_EORDER
    with pytest.raises(T.TpsError) as e:
        st.forward(1, X, Y)
    assert e.value.code == T.TPS_EORDER and "expected F(0)" in str(e.value)
    with pytest.raises(T.TpsError) as e:
        st.forward(7, X, Y)
    assert e.value.code == T.TPS_EORDER
    st.forward(0, X, Y)
    with pytest.raises(T.TpsError) as e:
        st.forward(0, X, Y)
    assert e.value.code == T.TPS_EORDER
    st.sync()
    st.close()


def test_arena_too_small_is_enomem():
    import ctypes as C
    import torch
    from stage_harness import make_params
    cfg = W.tiny()
    blocks, grads, _ = make_params(cfg)
    info = T.plan(cfg)
    arena = torch.empty(info["device_arena_bytes"] // 2, dtype=torch.uint8, device="cuda")
    L = cfg.n_layers
    pp = (C.c_void_p * L)(*[t.data_ptr() for t in blocks])
    gp = (C.c_void_p * L)(*[t.data_ptr() for t in grads])
    prm = T.Params(C.cast(pp, C.POINTER(C.c_void_p)), C.cast(gp, C.POINTER(C.c_void_p)))
    s = torch.cuda.Stream()
    mem = T.Memory(arena.data_ptr(), arena.numel(), None, 0, s.cuda_stream, s.cuda_stream)
    c = cfg.to_c()
    h = C.c_void_p()
    rc = T.lib().tps_stage_init(C.byref(c), C.byref(prm), C.byref(mem), C.byref(h))
    assert rc == T.TPS_ENOMEM
    assert b"plan needs" in T.lib().tps_last_error()


def test_full_shape_stage4_h2048_two_microbatches_matches_oracle():
    """The bench workload's shapes and launch configuration (hidden 2048, 16
    heads, MLP 8192, seq 2048, selective recompute), two micro-batches so the
    float64 oracle finishes in seconds."""
    cfg = dataclasses.replace(W.stage4_h2048(), n_micro=2)
    print("full-shape stage4_h2048, n_micro=2: GPU run", flush=True)
    gpu = run_gpu(cfg)
    print("oracle run", flush=True)
    ref = run_oracle(cfg)
    worst, bad = compare(gpu, ref, BF16_TOL)
    print("worst rel-L2", max(worst.values()), flush=True)
    assert not bad, bad


def _streamed(window, granularity, policy=None, **kw):
    L = 4
    return _mid(n_layers=L, policy=policy or W.policy_layer_inputs(L), granularity=granularity,
                weights=T.W_STREAM, window=window, **kw)


def test_streamed_weights_match_oracle():
    """Weights streamed in and f32 gradients streamed out (window < layers)
    against the oracle, through per-micro-batch calls and group calls, at
    both recompute granularities (segment granularity in groups of one
    micro-batch: inflight 1 makes the order F0 B0 F1 B1 F2 B2)."""
    L = 4
    ref = run_oracle(_mid(n_layers=L))
    cases = [
        ("per-mb, segment, window 2", _streamed(2, T.GRAN_SEGMENT), False),
        ("per-mb, layer, window 3", _streamed(3, T.GRAN_LAYER), False),
        ("group, layer, window 2", _streamed(2, T.GRAN_LAYER), True),
        ("groups of one, segment, window 2", _streamed(2, T.GRAN_SEGMENT, inflight=1), True),
        ("groups of one, selective segment, window 3",
         _streamed(3, T.GRAN_SEGMENT, policy=W.policy_selective(L), inflight=1), True),
    ]
    for name, cfg, group in cases:
        print(name, flush=True)
        out = run_gpu(cfg, group=group)
        worst, bad = compare(out, ref, BF16_TOL)
        assert not bad, (name, bad)
        assert out["stats"]["h2d_bytes"] > 0 and out["stats"]["d2h_bytes"] > 0, name


def _permuted_blocks(blocks):
    """New parameters for every layer: layer l takes the values of layer L-1-l."""
    return [b.clone() for b in reversed(blocks)]


def test_parameters_changed_between_iterations():
    """An optimizer step between iterations (here: the layers' parameter
    blocks permuted in place) must reach every layer of the next iteration:
    the second iteration of one stage equals, bitwise, a fresh stage built on
    the new parameters, for resident weights and for a streamed window whose
    entries survive the iteration boundary."""
    import torch
    from stage_harness import drive_iteration, make_params, results, to_dev
    variants = [("resident", _mid(n_layers=4, policy=W.policy_selective(4)), False),
                ("streamed, layer, window 2", _streamed(2, T.GRAN_LAYER), True),
                ("streamed, segment, window 3", _streamed(3, T.GRAN_SEGMENT), False)]
    for name, cfg, group in variants:
        print(name, flush=True)
        xs, dys = inputs(cfg)
        blocks, grads, _ = make_params(cfg)
        new_blocks = _permuted_blocks(blocks)
        X = [to_dev(x, cfg.dtype) for x in xs]
        DY = [to_dev(d, cfg.dtype) for d in dys]
        Y = [torch.empty_like(x) for x in X]
        DX = [torch.empty_like(x) for x in X]
        torch.cuda.synchronize()
        st = T.Stage(cfg, blocks, grads)
        drive_iteration(st, cfg, X, DY, Y, DX, group=group)
        st.sync()
        for b, nb in zip(blocks, new_blocks):
            b.copy_(nb)
        torch.cuda.synchronize()
        drive_iteration(st, cfg, X, DY, Y, DX, group=group)
        second = results(cfg, st, Y, DX, grads)
        st.close()
        fb, fg, _ = make_params(cfg)
        for b, nb in zip(fb, new_blocks):
            b.copy_(nb)
        torch.cuda.synchronize()
        fresh = run_gpu(cfg, xs, dys, group=group, params=(fb, fg, None))
        assert bit_equal(second, fresh) == [], name


def test_group_calls_after_per_microbatch_calls_bitexact():
    """Group calls that follow per-micro-batch calls in one iteration (the
    per-micro-batch backward leaves its last parameter-gradient kernels
    running): bit-exact to the same iteration made of per-micro-batch calls
    only."""
    keep_order = [("F", 0), ("F", 1), ("F", 2), ("B", 0), ("B", 1), ("B", 2)]
    ref = run_gpu(_mid(ops=keep_order))
    mixed = run_gpu(_mid(ops=keep_order), calls=[("F", [0, 1, 2], False), ("B", [0], False), ("B", [1, 2], True)])
    assert bit_equal(ref, mixed) == []
    order2 = [("F", 0), ("B", 0), ("F", 1), ("F", 2), ("B", 1), ("B", 2)]
    mixed2 = run_gpu(_mid(ops=order2), calls=[("F", [0], False), ("B", [0], False), ("F", [1, 2], True),
                                              ("B", [1, 2], False)])
    assert bit_equal(ref, mixed2) == []
    # the same with the selective policy (segment replays; groups of one)
    sel = _mid(ops=keep_order, policy=W.policy_selective(3))
    ref_sel = run_gpu(sel)
    mixed_sel = run_gpu(sel, calls=[("F", [0, 1], False), ("F", [2], True), ("B", [0], False), ("B", [1], True),
                                    ("B", [2], False)])
    assert bit_equal(ref_sel, mixed_sel) == []


def test_stream_ordering_without_explicit_synchronize():
    """The binding orders the stage after the caller's current stream and the
    caller after the stage: inputs written by a late kernel on the caller's
    stream just before each call are the ones the stage reads, and outputs
    read on the caller's stream are complete, with no torch.cuda.synchronize().
    Both with the caller on a stream of its own (the stage then runs on it)
    and on the default stream (the stage on a private stream)."""
    import torch
    from stage_harness import drive_iteration, make_params, results, to_dev
    cfg = _mid(policy=W.policy_selective(3))
    ref = run_gpu(cfg)
    xs, dys = inputs(cfg)
    torch.cuda.synchronize()
    for own_stream in (True, False):
        s = torch.cuda.Stream() if own_stream else torch.cuda.default_stream()
        with torch.cuda.stream(s):
            blocks, grads, _ = make_params(cfg)
            st = T.Stage(cfg, blocks, grads)
            assert (st.cs.cuda_stream == s.cuda_stream) == own_stream
            X = [torch.zeros(cfg.tokens, cfg.hidden, device="cuda", dtype=torch.bfloat16) for _ in xs]
            DY = [torch.zeros_like(x) for x in X]
            Y = [torch.empty_like(x) for x in X]
            DX = [torch.empty_like(x) for x in X]
            srcX = [to_dev(x, cfg.dtype) for x in xs]
            srcDY = [to_dev(d, cfg.dtype) for d in dys]
            # a spin kernel delays the input writes on the caller's stream
            torch.cuda._sleep(50_000_000)
            for a, b in zip(X + DY, srcX + srcDY):
                a.copy_(b)
            drive_iteration(st, cfg, X, DY, Y, DX)
            out = dict(ys=[to_np(y) for y in Y], dxs=[to_np(d) for d in DX], grads=read_grads(cfg, grads))
        st.close()
        assert bit_equal(ref, out) == [], own_stream


def test_sync_for_times_out_and_recovers():
    """tps_stage_sync_for returns TPS_ETIMEOUT while the compute stream is
    still busy (a bounded spin kernel holds it), and TPS_OK once the work is
    done; the stage stays usable."""
    import torch
    from stage_harness import make_params
    cfg = W.tiny()
    blocks, grads, _ = make_params(cfg)
    st = T.Stage(cfg, blocks, grads)
    torch.cuda.synchronize()
    assert st.sync_for(0) == T.TPS_OK
    with torch.cuda.stream(st.cs):
        torch.cuda._sleep(200_000_000)
    assert st.sync_for(1.0) == T.TPS_ETIMEOUT
    assert "compute stream still has work" in T.lib().tps_last_error().decode()
    assert st.sync_for(120_000.0) == T.TPS_OK
    with pytest.raises(T.TpsError) as e:
        st.sync_for(-1.0)
    assert e.value.code == T.TPS_EINVAL
    st.close()


def test_tpipe_stage_orders_bitexact_to_default():
    """One stage of a 4-stage T-Pipe with T-Recomp over 8 micro-batches, as
    the simulator orders it: chunk 1 (full recompute from the chunk input,
    replayed as one block before each backward) and chunk 2 (every tensor
    kept) are two stage objects on one stream, called in the stage's
    interleaved order.  Each is bit-exact to the same chunk run alone in the
    default order (all forwards first), and the planner holds fewer
    checkpoint slots for chunk 2 under the T-Pipe order."""
    import torch
    from stage_harness import make_params, results, to_dev
    _, tasks = T.tpipe_schedule(4, 8, stage=1, t_recomp=True)
    o1, o2, calls = T.chunk_orders(tasks)
    c1 = _mid(n_layers=2, n_micro=8, policy=W.policy_all(2, T.RECOMPUTE), granularity=T.GRAN_SEGMENT, ops=o1)
    c2 = _mid(n_layers=2, n_micro=8, ops=o2)
    ref1 = run_gpu(dataclasses.replace(c1, ops=None))
    ref2 = run_gpu(dataclasses.replace(c2, ops=None))
    assert T.plan(c2)["n_slots"] < T.plan(dataclasses.replace(c2, ops=None))["n_slots"]
    xs, dys = inputs(c1)
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        stages, io = {}, {}
        for ch, cfg in ((1, c1), (2, c2)):
            blocks, grads, _ = make_params(cfg)
            st = T.Stage(cfg, blocks, grads)
            X = [to_dev(x, cfg.dtype) for x in xs]
            DY = [to_dev(d, cfg.dtype) for d in dys]
            io[ch] = (X, DY, [torch.empty_like(x) for x in X], [torch.empty_like(x) for x in X], grads, cfg)
            stages[ch] = st
            st.begin_iteration(zero_grads=True)
        for ch, kind, mb in calls:
            X, DY, Y, DX, _, _ = io[ch]
            if kind == "F":
                stages[ch].forward(mb, X[mb], Y[mb])
            else:
                stages[ch].backward(mb, DY[mb], DX[mb])
        outs = {}
        for ch in (1, 2):
            X, DY, Y, DX, grads, cfg = io[ch]
            outs[ch] = results(cfg, stages[ch], Y, DX, grads)
            stages[ch].close()
    assert bit_equal(ref1, outs[1]) == []
    assert bit_equal(ref2, outs[2]) == []
