"""Happens-before checks of the stage executor's stream and event protocol,
on the CPU.  The executor's host code is built against a stand-in HIP
runtime (tests/hb) that models streams and events with vector clocks and
records the bytes every kernel and copy reads and writes; the checker flags
any access that is not ordered after a conflicting earlier one (a read
before its producer has finished, a buffer overwritten while a kernel on
another stream may still read it, a host-to-device copy still in flight at
its consumer, host access to pinned blocks without a synchronisation).
The same op sequences the GPU tests and bench.py issue are checked here at
the full workload shapes, in every order and call style the GPU tests use.
The checker itself is checked by leaving out each stream wait in turn."""
import dataclasses

import pytest

from paper_2503_03182_amd import configs as W
from paper_2503_03182_amd import tpstage as T

from hb import driver as D


def _run(cfg, iterations=2, group=None, calls=None, **kw):
    D.reset()
    st = D.FakeStage(cfg, **kw)
    st.write_inputs()
    for _ in range(iterations):
        st.iteration(group=cfg.layer_major if group is None else group, calls=calls)
    st.read_results()
    st.close()
    return D.races()


def _mid(**kw):
    base = dict(n_layers=3, hidden=512, n_heads=4, mlp=2048, seq=200, micro_batch=2, n_micro=3, dtype="bf16")
    base.update(kw)
    return T.StageConfig(**base)


WORKLOADS = ["tiny", "stage4_h2048", "stage5_h5120_offload", "stage5_h5120_resident", "stage4_seq8192_recompute",
             "stage12_h8192_stream", "stage12_h8192_stream_m20", "llama4_h4096", "llama12_h8192_stream"]


@pytest.mark.parametrize("name", WORKLOADS)
def test_workloads_race_free(name):
    cfg = W.WORKLOADS[name]()
    assert _run(cfg) == 0, D.report()


@pytest.mark.parametrize("policy", ["recompute", "offload"])
def test_tiny_policies_race_free(policy):
    assert _run(W.tiny(policy)) == 0, D.report()


def test_orders_groups_and_copy_streams_race_free():
    L = 3
    order = [("F", 0), ("F", 1), ("B", 0), ("F", 2), ("B", 1), ("B", 2)]
    mixed = [{t: [T.KEEP, T.RECOMPUTE, T.OFFLOAD][(l + i) % 3] for i, t in enumerate(T.TENSORS)} for l in range(L)]
    mixed[0]["x"] = T.KEEP
    cfgs = [
        _mid(ops=order), _mid(ops=order, policy=W.policy_selective(L)),
        _mid(ops=order, policy=W.policy_layer_inputs(L), granularity=T.GRAN_SEGMENT),
        _mid(ops=order, policy=W.policy_layer_inputs(L), granularity=T.GRAN_LAYER),
        _mid(ops=order, policy=W.policy_all(L, T.RECOMPUTE)),
        _mid(ops=order, policy=W.policy_all(L, T.OFFLOAD), offload_mb_mask=0b111),
        _mid(ops=order, policy=W.policy_all(L, T.OFFLOAD), offload_mb_mask=0b100, lookahead=2),
        _mid(ops=order, policy=mixed, offload_mb_mask=0b101),
        _mid(policy=W.policy_all(3, T.OFFLOAD), offload_mb_mask=0b011, inflight=2),
    ]
    for i, cfg in enumerate(cfgs):
        assert _run(cfg, iterations=3) == 0, (i, D.report())
    assert _run(cfgs[5], iterations=3, one_copy_stream=True) == 0, D.report()
    assert _run(cfgs[5], iterations=2, own_copy_streams=False) == 0, D.report()
    assert _run(_mid(policy=W.policy_layer_inputs(L), granularity=T.GRAN_LAYER), group=True) == 0, D.report()


def test_streamed_weights_race_free():
    for window in (2, 3):
        for gran in (T.GRAN_LAYER, T.GRAN_SEGMENT):
            for inflight in (0, 1):
                cfg = _mid(n_layers=4, policy=W.policy_layer_inputs(4), granularity=gran, weights=T.W_STREAM,
                           window=window, inflight=inflight)
                for group in (False, True):
                    if group and gran == T.GRAN_SEGMENT and inflight == 0:
                        continue   # groups of several micro-batches need layer granularity
                    assert _run(cfg, iterations=3, group=group) == 0, (window, gran, inflight, group, D.report())


def test_quantized_weight_reload_race_free():
    """Streamed weights reloaded as FP8 codes with row scales: the staging area
    of a window entry and its expansion into the entry's parameter block."""
    for window in (2, 3):
        cfg = _mid(n_layers=4, policy=W.policy_layer_inputs(4), granularity=T.GRAN_LAYER, weights=T.W_STREAM,
                   window=window, weights_quant=T.Q_FP8_ROW)
        for group in (False, True):
            assert _run(cfg, iterations=3, group=group) == 0, (window, group, D.report())


def test_wgrad_arrangements_race_free():
    """Parameter-gradient kernels on their own stream and inline on the
    compute stream, for both call styles and the replay-stream and streamed
    configurations."""
    L = 4
    cfgs = [_mid(n_layers=L), _mid(n_layers=L, policy=W.policy_selective(L)),
            _mid(n_layers=L, policy=W.policy_all(L, T.OFFLOAD), offload_mb_mask=0b101),
            _mid(n_layers=L, policy=W.policy_layer_inputs(L), granularity=T.GRAN_LAYER, weights=T.W_STREAM, window=2)]
    for i, base in enumerate(cfgs):
        for mode in (T.WGRAD_SIDE, T.WGRAD_INLINE):
            cfg = dataclasses.replace(base, wgrad_stream=mode)
            for group in ((False, True) if base.granularity == T.GRAN_LAYER else (False,)):
                assert _run(cfg, iterations=2, group=group) == 0, (i, mode, group, D.report())


def test_poison_fills_race_free(monkeypatch):
    """With TPS_POISON the dead memory is filled as it is handed back; every
    fill is ordered after the last reader of that memory and before its next
    writer (a fill that raced would itself be reported)."""
    monkeypatch.setenv("TPS_POISON", "1")
    L = 4
    cfgs = [(_mid(n_layers=L, policy=W.policy_selective(L)), False),
            (_mid(n_layers=L, policy=W.policy_all(L, T.OFFLOAD), offload_mb_mask=0b101, lookahead=2), False),
            (_mid(n_layers=L, policy=W.policy_layer_inputs(L), granularity=T.GRAN_SEGMENT), False),
            (_mid(n_layers=L, policy=W.policy_layer_inputs(L), granularity=T.GRAN_LAYER, weights=T.W_STREAM,
                  window=2), True),
            (_mid(n_layers=L, policy=W.policy_layer_inputs(L), granularity=T.GRAN_LAYER, weights=T.W_STREAM,
                  window=3, weights_quant=T.Q_FP8_ROW), False)]
    for i, (base, group) in enumerate(cfgs):
        for mode in (T.WGRAD_SIDE, T.WGRAD_INLINE):
            before = D.count_ops("fill")
            assert _run(dataclasses.replace(base, wgrad_stream=mode), iterations=2, group=group) == 0, \
                (i, mode, D.report())
            assert D.count_ops("fill") > before, (i, mode)
    monkeypatch.delenv("TPS_POISON")
    before = D.count_ops("fill")
    assert _run(cfgs[1][0]) == 0
    assert D.count_ops("fill") == before


def test_batched_group_weight_gradients_race_free():
    """Backward groups that issue each weight-gradient product once per layer
    over their micro-batches: resident and streamed weights, GPT and LLAMA
    layers, both parameter-gradient arrangements, groups of all and of some
    micro-batches, layers that cannot batch (kept activations) beside ones
    that can."""
    L = 4
    pol = W.policy_layer_inputs(L)
    mixed = [dict(p) for p in pol]
    mixed[1]["c"] = T.KEEP            # layer 1 keeps c: its products stay per micro-batch
    cfgs = [_mid(n_layers=L, policy=pol, granularity=T.GRAN_LAYER, group_wgrad=1),
            _mid(n_layers=L, policy=mixed, granularity=T.GRAN_LAYER, group_wgrad=1),
            _mid(n_layers=L, policy=pol, granularity=T.GRAN_LAYER, weights=T.W_STREAM, window=2, group_wgrad=1),
            _mid(n_layers=L, policy=pol, granularity=T.GRAN_LAYER, weights=T.W_STREAM, window=3, group_wgrad=1,
                 arch=T.ARCH_LLAMA, n_kv_heads=2)]
    for i, cfg in enumerate(cfgs):
        for mode in (T.WGRAD_SIDE, T.WGRAD_INLINE):
            assert _run(dataclasses.replace(cfg, wgrad_stream=mode), iterations=2, group=True) == 0, \
                (i, mode, D.report())
    # groups of some of the micro-batches, with per-micro-batch calls between
    cfg = _mid(n_layers=L, policy=pol, granularity=T.GRAN_LAYER, group_wgrad=1, n_micro=4)
    calls = [("F", [0, 1, 2, 3], True), ("B", [0, 1], True), ("B", [2], False), ("B", [3], True)]
    assert _run(cfg, iterations=2, calls=calls) == 0, D.report()


def test_llama_layers_race_free():
    """LLAMA-style layers (rotation, grouped attention with its key/value
    workspace, SwiGLU) under every policy kind, both call styles, streamed
    weights and both parameter-gradient arrangements."""
    L = 4
    order = [("F", 0), ("F", 1), ("B", 0), ("F", 2), ("B", 1), ("B", 2)]
    base = dict(n_layers=L, hidden=512, n_heads=4, mlp=1024, seq=200, micro_batch=2, n_micro=3, dtype="bf16",
                arch=T.ARCH_LLAMA, n_kv_heads=2)
    mixed = [{t: [T.KEEP, T.RECOMPUTE, T.OFFLOAD][(l + i) % 3] for i, t in enumerate(T.TENSORS)} for l in range(L)]
    mixed[0]["x"] = T.KEEP
    cfgs = [(T.StageConfig(**base, ops=order), False),
            (T.StageConfig(**base, policy=W.policy_selective(L)), False),
            (T.StageConfig(**base, ops=order, policy=mixed, offload_mb_mask=0b101), False),
            (T.StageConfig(**base, policy=W.policy_layer_inputs(L), granularity=T.GRAN_SEGMENT), False),
            (T.StageConfig(**base, policy=W.policy_layer_inputs(L), granularity=T.GRAN_LAYER, weights=T.W_STREAM,
                           window=2), True),
            (T.StageConfig(**dict(base, n_kv_heads=4), policy=W.policy_all(L, T.RECOMPUTE)), False)]
    for i, (cfg, group) in enumerate(cfgs):
        for mode in (T.WGRAD_SIDE, T.WGRAD_INLINE):
            assert _run(dataclasses.replace(cfg, wgrad_stream=mode), iterations=2, group=group) == 0, \
                (i, mode, D.report())


def test_mixed_per_microbatch_and_group_calls_race_free():
    keep_order = [("F", 0), ("F", 1), ("F", 2), ("B", 0), ("B", 1), ("B", 2)]
    assert _run(_mid(ops=keep_order), calls=[("F", [0, 1, 2], False), ("B", [0], False), ("B", [1, 2], True)]) == 0, \
        D.report()
    order2 = [("F", 0), ("B", 0), ("F", 1), ("F", 2), ("B", 1), ("B", 2)]
    assert _run(_mid(ops=order2), calls=[("F", [0], False), ("B", [0], False), ("F", [1, 2], True),
                                         ("B", [1, 2], False)]) == 0, D.report()
    sel = _mid(ops=keep_order, policy=W.policy_selective(3))
    assert _run(sel, calls=[("F", [0, 1], False), ("F", [2], True), ("B", [0], False), ("B", [1], True),
                            ("B", [2], False)]) == 0, D.report()


def test_tpipe_two_chunks_on_one_stream_race_free():
    _, tasks = T.tpipe_schedule(4, 8, stage=1, t_recomp=True)
    o1, o2, calls = T.chunk_orders(tasks)
    c1 = _mid(n_layers=2, n_micro=8, policy=W.policy_all(2, T.RECOMPUTE), granularity=T.GRAN_SEGMENT, ops=o1)
    c2 = _mid(n_layers=2, n_micro=8, ops=o2)
    D.reset()
    cs = D.lib().tps_hb_new_stream(b"compute")
    s1 = D.FakeStage(c1, tag=1, cs=cs)
    s2 = D.FakeStage(c2, tag=2, cs=cs)
    for it in range(2):
        for s in (s1, s2):
            if it == 0:
                s.write_inputs()
            s.begin()
        for ch, kind, mb in calls:
            (s1 if ch == 1 else s2).call(kind, [mb], False)
    s1.read_results()
    s2.read_results()
    s1.close()
    s2.close()
    assert D.races() == 0, D.report()


def _dropped_wait_detection(cfg, group=False):
    """For each stream wait the executor issues (two iterations), rerun with
    that wait left out: (waits, number whose removal the checker reports)."""
    L = D.lib()
    D.reset()
    w0 = L.tps_hb_waits()
    assert _run(cfg, group=group) == 0, D.report()
    n = L.tps_hb_waits() - w0
    detected = 0
    for k in range(n):
        L.tps_hb_drop_wait(L.tps_hb_waits() + k)
        try:
            if _run(cfg, group=group) > 0:
                detected += 1
        finally:
            L.tps_hb_drop_wait(-1)
    return n, detected


def test_checker_reports_left_out_waits():
    """Nearly every wait is load-bearing: leaving one out makes the checker
    report a race (the few that do not are implied by other edges)."""
    c2 = dataclasses.replace(W.stage4_h2048(), n_micro=4)
    n, det = _dropped_wait_detection(c2)
    assert n > 100 and det >= 0.95 * n, (n, det)
    # (the side-stream arrangement: inline, the parameter-gradient waits are
    # on the compute stream itself and leave nothing to detect)
    c5 = dataclasses.replace(W.stage12_h8192_stream(), n_layers=4, n_micro=4, wgrad_stream=T.WGRAD_SIDE,
                             group_wgrad=0)
    c5.policy = c5.policy[:4]
    n, det = _dropped_wait_detection(c5, group=True)
    assert n > 100 and det >= 0.9 * n, (n, det)
    # batched weight gradients: every micro-batch of a group has its own
    # operand slots, so some per-micro-batch joins guard nothing there
    n, det = _dropped_wait_detection(dataclasses.replace(c5, group_wgrad=1), group=True)
    assert n > 100 and det >= 0.75 * n, (n, det)
    off = _mid(policy=W.policy_all(3, T.OFFLOAD), offload_mb_mask=0b111)
    n, det = _dropped_wait_detection(off)
    # (per-layer ready events of one prefetch are recorded in order on one
    # stream, so waiting on a later one implies the earlier ones)
    assert n > 50 and det >= 0.65 * n, (n, det)


def test_host_access_needs_sync():
    """Pinned host gradient blocks of streamed weights may be read only after
    tps_stage_sync: without it the checker reports the host read racing with
    the device-to-host copies; and changing the host parameter blocks for the
    next iteration needs the same synchronisation."""
    cfg = _mid(n_layers=4, policy=W.policy_layer_inputs(4), granularity=T.GRAN_LAYER, weights=T.W_STREAM, window=2)
    D.reset()
    st = D.FakeStage(cfg)
    st.write_inputs()
    st.iteration()
    st.read_results(sync=False)
    assert D.races() > 0 and "host read" in D.report()
    st.close()
    D.reset()
    st = D.FakeStage(cfg)
    st.write_inputs()
    st.iteration()
    st.read_results(sync=True)
    for p in st.params:      # an optimizer step on the host blocks, after the sync
        D.lib().tps_hb_host_access(p, st.pbytes, 1)
    st.iteration()
    st.read_results(sync=True)
    assert D.races() == 0, D.report()
    st.close()


def test_device_optimizer_race_free():
    """Every layer's AdamW on the device: the update reads the gradients the
    layer's last backward wrote and rewrites the device parameter block that
    the next iteration's loads copy into the window; per-micro-batch and
    group calls, bf16 and quantized reload configs, windows of 2 and 3."""
    for window in (2, 3):
        for quant in (T.Q_NONE, T.Q_FP8_ROW):
            cfg = _mid(n_layers=4, policy=W.policy_layer_inputs(4), granularity=T.GRAN_LAYER, weights=T.W_STREAM,
                       window=window, weights_quant=quant)
            for group in (False, True):
                D.reset()
                st = D.FakeStage(cfg)
                st.write_inputs()
                st.set_device_optimizer()
                for _ in range(3):
                    st.iteration(group=group)
                st.read_results()
                st.close()
                assert D.races() == 0, (window, quant, group, D.report())
    # one update per parameter tensor of every layer per iteration, and the
    # host link carries no gradient block of a device-updated layer
    cfg = _mid(n_layers=4, policy=W.policy_layer_inputs(4), granularity=T.GRAN_LAYER, weights=T.W_STREAM, window=4)
    D.reset()
    st = D.FakeStage(cfg)
    st.write_inputs()
    st.set_device_optimizer()
    updates0 = D.count_ops("adamw")
    d2h0 = D.count_ops("copy device->host") + D.count_ops("pitched copy device->host")
    for it in range(2):
        st.iteration(group=True)
        assert D.count_ops("adamw") - updates0 == (it + 1) * 4 * len(T.PARAMS)
    st.read_results()
    st.close()
    assert D.races() == 0, D.report()
    assert D.count_ops("copy device->host") + D.count_ops("pitched copy device->host") == d2h0
