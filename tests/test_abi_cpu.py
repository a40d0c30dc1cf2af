"""Host-side checks of the C ABI (no GPU): the library loads, exports every
symbol the headers declare, and the planner's layout, accounting and error
conventions match closed forms computed here from the shapes."""

import ctypes as C
import os
import re

import pytest

from paper_2503_03182_amd import configs as W
from paper_2503_03182_amd import tpstage as T

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
pytestmark = pytest.mark.skipif(not os.path.exists(T.lib_path()), reason="libtpstage.so not built")


def _declared():
    names = set()
    for h in ("tpstage.h", "tpstage_ops.h"):
        src = open(os.path.join(ROOT, "include", h)).read()
        src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
        names |= set(re.findall(r"\b(tps_[a-z_0-9]+)\s*\(", src))
    return names


def test_library_exports_every_declared_symbol():
    lib = C.CDLL(T.lib_path())
    declared = _declared()
    assert len(declared) >= 19
    for name in sorted(declared):
        assert hasattr(lib, name), name
    assert declared == set(T.EXPORTED)


def _align(x):
    return (x + 255) // 256 * 256


def _widths(cfg):
    """(qkv width, u width, LN statistics per row) of the layer kind."""
    h, f = cfg.hidden, cfg.mlp
    if cfg.arch == T.ARCH_LLAMA:
        d, nkv = h // cfg.n_heads, cfg.n_kv_heads or cfg.n_heads
        return (cfg.n_heads + 2 * nkv) * d, 2 * f, 1
    return 3 * h, f, 2


def _tensor_bytes(cfg):
    es = 2 if cfg.dtype == "bf16" else 4
    Tk, h, f = cfg.tokens, cfg.hidden, cfg.mlp
    qw, uw, ns = _widths(cfg)
    b = {n: Tk * h * es for n in ("x", "a", "o", "x1", "c")}
    b.update(qkv=Tk * qw * es, u=Tk * uw * es, g=Tk * f * es,
             lse=cfg.micro_batch * cfg.n_heads * cfg.seq * 4, ln1=ns * Tk * 4, ln2=ns * Tk * 4)
    return b


@pytest.mark.parametrize("name", list(W.WORKLOADS))
def test_plan_accounting_closed_forms(name):
    cfg = W.WORKLOADS[name]()
    p = T.plan(cfg)
    tb = _tensor_bytes(cfg)
    L, M = cfg.n_layers, cfg.n_micro
    pol = cfg.policy or [{t: T.KEEP for t in T.TENSORS} for _ in range(L)]
    keep = sum(_align(tb[t]) for l in range(L) for t in T.TENSORS if pol[l][t] == T.KEEP)
    off = sum(_align(tb[t]) for l in range(L) for t in T.TENSORS if pol[l][t] == T.OFFLOAD)
    assert p["slot_bytes"] == keep
    assert p["offload_slot_bytes"] == off
    # all forwards first (W = M): every micro-batch is in flight at the peak
    assert p["max_inflight"] == M
    if keep:
        assert p["n_slots"] == M
    assert p["keep_all_bytes"] == M * L * sum(_align(v) for v in tb.values())
    Tk, h, f, s, b = cfg.tokens, cfg.hidden, cfg.mlp, cfg.seq, cfg.micro_batch
    qw, uw, _ = _widths(cfg)
    unit = 2 * Tk * (h * qw + h * h + h * uw + f * h) + 2 * b * h * s * (s + 1)
    assert p["fwd_flops"] == pytest.approx(unit * L * M, rel=1e-12)
    assert p["bwd_flops"] == pytest.approx(2 * unit * L * M, rel=1e-12)
    n_off = bin(p["offload_mb_mask"]).count("1")
    assert p["n_offload_mbs"] == n_off
    if cfg.weights == T.W_RESIDENT:
        assert p["h2d_bytes"] == n_off * off
        assert p["predicted_peak_bytes"] == p["device_arena_bytes"] + L * (p["param_bytes"] + p["grad_bytes"])


def test_replay_programs_and_recompute_flops():
    # selective: attention and GeLU outputs -> replay attention and GeLU only
    cfg = W.stage4_h2048()
    p = T.plan(cfg)
    Tk, h, s, b = cfg.tokens, cfg.hidden, cfg.seq, cfg.micro_batch
    attn = 2 * b * h * s * (s + 1)
    assert p["recompute_flops"] == pytest.approx(attn * cfg.n_layers * cfg.n_micro)
    assert p["n_replay_layers"] == cfg.n_layers
    # layer inputs kept: every operator but FC2 is replayed (its output, the
    # next layer's input, is kept)
    cfg = W.stage4_seq8192_recompute()
    p = T.plan(cfg)
    Tk, h, f, s, b = cfg.tokens, cfg.hidden, cfg.mlp, cfg.seq, cfg.micro_batch
    per = 2 * Tk * (4 * h * h + h * f) + 2 * b * h * s * (s + 1)
    assert p["recompute_flops"] == pytest.approx(per * cfg.n_layers * cfg.n_micro)
    # only the stage input kept: the top layers also replay FC2 of the layer
    # below to regenerate their inputs
    cfg = W.tiny("recompute")
    p = T.plan(cfg)
    Tk, h, f, s, b = cfg.tokens, cfg.hidden, cfg.mlp, cfg.seq, cfg.micro_batch
    full = 2 * Tk * (4 * h * h + 2 * h * f) + 2 * b * h * s * (s + 1)
    # layer 1 needs its input: layer 0 replays fully (with FC2); layer 1 replays all but FC2
    assert p["recompute_flops"] == pytest.approx((full + full - 2 * Tk * f * h) * cfg.n_micro)


def test_llama_layout_and_validation():
    """LLAMA-style layers: parameter blocks with the packed q | k | v and gate
    | up matrices, the two RMSNorm gains and empty bias / shift slots; bf16
    and head dim 128 only; n_kv_heads must divide n_heads."""
    import dataclasses
    cfg = W.llama4_h4096()
    h, f, nh, nkv = cfg.hidden, cfg.mlp, cfg.n_heads, cfg.n_kv_heads
    qw = (nh + 2 * nkv) * 128
    po, pb, go, gb = T.param_layout(cfg)
    elems = dict(w_qkv=qw * h, b_qkv=0, w_o=h * h, b_o=0, w_1=2 * f * h, b_1=0, w_2=h * f, b_2=0, g1=h, be1=0, g2=h,
                 be2=0)
    o, g = 0, 0
    for i, n in enumerate(T.PARAMS):
        assert po[i] == o and go[i] == g, n
        o, g = _align(o + 2 * elems[n]), _align(g + 4 * elems[n])
    assert pb == o and gb == g
    with pytest.raises(T.TpsError):
        T.plan(dataclasses.replace(cfg, n_kv_heads=5))
    with pytest.raises(T.TpsError):
        T.plan(dataclasses.replace(cfg, dtype="f32"))
    with pytest.raises(T.TpsError):
        T.plan(dataclasses.replace(cfg, n_heads=64))     # head dim 64
    with pytest.raises(T.TpsError):
        T.plan(dataclasses.replace(W.stage4_h2048(), n_kv_heads=4))   # GPT layers: multi-head only
    # grouped attention needs the per-query-head key/value workspace
    es = 2
    Tk = cfg.tokens
    p = T.plan(cfg)
    p1 = T.plan(dataclasses.replace(cfg, n_kv_heads=nh))
    assert p["work_bytes"] - p1["work_bytes"] == _align(Tk * 2 * h * es) - 2 * (
        _align(Tk * (nh + 2 * nh) * 128 * es) - _align(Tk * qw * es))


def test_backward_work_buffers():
    # resident weights with a segment replay (or none): the parameter-gradient
    # kernels lag, so the running input gradient rotates over three buffers and
    # the intermediate gradients (dX1, dU, dQKV) have a set per layer parity;
    # otherwise two gradient buffers and one set.  Plus t1 and the attention
    # backward's row dot products.
    def expect(cfg, lag):
        es = 2 if cfg.dtype == "bf16" else 4
        Tk, h, f = cfg.tokens, cfg.hidden, cfg.mlp
        hb, fb, qb = _align(Tk * h * es), _align(Tk * f * es), _align(Tk * 3 * h * es)
        dvec = _align(cfg.micro_batch * cfg.n_heads * cfg.seq * 4)
        base = (3 if lag else 2) * hb + (2 if lag else 1) * (hb + fb + qb) + hb + dvec
        if cfg.group_wgrad:
            # batched weight gradients: n slots of a, o, c, g, du, dx1, dqkv
            # and of two running-gradient buffers
            base += cfg.n_micro * (3 * hb + fb + fb + hb + qb + 2 * hb)
        return base

    for name, lag in [("stage4_h2048", True), ("stage5_h5120_offload", True),
                      ("stage4_seq8192_recompute", True), ("stage12_h8192_stream", False)]:
        cfg = W.WORKLOADS[name]()
        assert T.plan(cfg)["work_bytes"] == expect(cfg, lag), name
    cfg = W.tiny("recompute")
    cfg.granularity = T.GRAN_LAYER   # replays between layer backwards: no lag
    cfg.policy = W.policy_layer_inputs(cfg.n_layers)
    assert T.plan(cfg)["work_bytes"] == expect(cfg, False)
    cfg.granularity = T.GRAN_SEGMENT
    assert T.plan(cfg)["work_bytes"] == expect(cfg, True)


def test_slots_follow_the_order():
    cfg = W.tiny("keep")
    cfg.inflight = 2
    p = T.plan(cfg)
    assert p["max_inflight"] == 2 and p["n_slots"] == 2
    assert p["device_arena_bytes"] < T.plan(W.tiny("keep"))["device_arena_bytes"]


def test_offload_slots_and_auto_victims():
    cfg = W.tiny("offload")
    p = T.plan(cfg)
    assert p["n_offload_mbs"] == cfg.n_micro
    # a staging slot is held until its micro-batch's copy to host is done (a
    # forward never waits for one): with a link far faster than compute,
    # every micro-batch offloaded needs the slot being filled, the one still
    # draining to host and the prefetched one; slower links keep more slots
    # taken, never more than keeping everything
    slots = []
    for gbps in (1e9, 1000.0, 50.0, 1.0):
        c2 = W.tiny("offload")
        c2.link_gbps_hint = gbps
        slots.append(T.plan(c2)["n_offload_slots"])
    assert slots[0] <= 3 and slots == sorted(slots) and slots[-1] <= cfg.n_micro, slots
    assert p["n_offload_slots"] == slots[2]
    assert p["host_arena_bytes"] == p["n_host_slots"] * p["offload_slot_bytes"]
    # victims (taken in slack order while the round keeps its time and the
    # staging peak drops) are a pure function of the config
    big = W.stage5_h5120_offload()
    a, b2 = T.plan(big), T.plan(big)
    assert a["offload_mb_mask"] == b2["offload_mb_mask"] != 0
    assert a["predicted_peak_bytes"] < T.plan(W.stage5_h5120_resident())["predicted_peak_bytes"]
    # all forwards first: the staging peak comes at the last forwards, so a
    # victim helps only if its copy to host is done by then and its prefetch
    # comes after; faster links drain more of them in time (more victims, a
    # lower peak), and no victim is one whose prefetch precedes the last
    # forward (the first `lookahead` micro-batches) or the last forward itself
    prev = a
    for gbps in (100.0, 500.0, 50000.0):
        big.link_gbps_hint = gbps
        q = T.plan(big)
        assert q["n_offload_mbs"] >= prev["n_offload_mbs"], gbps
        assert q["predicted_peak_bytes"] <= prev["predicted_peak_bytes"], gbps
        prev = q
    assert prev["n_offload_mbs"] > a["n_offload_mbs"]
    assert prev["predicted_peak_bytes"] < 0.7 * a["predicted_peak_bytes"]
    assert prev["offload_mb_mask"] & ((1 << big.lookahead) - 1) == 0
    assert not prev["offload_mb_mask"] >> (big.n_micro - 1)
    # a tiny link hides none
    big.link_gbps_hint = 0.01
    assert T.plan(big)["n_offload_mbs"] == 0


def _expect(cfg, code, pattern):
    with pytest.raises(T.TpsError) as e:
        T.plan(cfg)
    assert e.value.code == code
    assert re.search(pattern, str(e.value)), str(e.value)


def test_config_errors():
    cfg = W.tiny()
    cfg.n_heads = 8      # head dim 32
    _expect(cfg, T.TPS_EINVAL, "head dim")
    cfg = W.tiny()
    cfg.hidden, cfg.n_heads = 260, 2
    _expect(cfg, T.TPS_EINVAL, "head dim|multiple")
    cfg = W.tiny("recompute")
    cfg.policy[0]["x"] = T.RECOMPUTE
    _expect(cfg, T.TPS_EINVAL, "stage input")
    cfg = W.tiny("recompute")
    cfg.granularity = T.GRAN_LAYER
    _expect(cfg, T.TPS_EINVAL, "layer granularity")
    cfg = W.tiny()
    cfg.ops = [("F", 0), ("F", 0), ("B", 1), ("B", 2), ("F", 3), ("B", 3), ("F", 1), ("B", 0)]
    _expect(cfg, T.TPS_EINVAL, "twice")
    cfg = W.tiny()
    cfg.ops = [("B", 0), ("F", 0), ("F", 1), ("B", 1), ("F", 2), ("B", 2), ("F", 3), ("B", 3)]
    _expect(cfg, T.TPS_EINVAL, "follow")
    cfg = W.tiny("offload")
    cfg.offload_mb_mask = 1 << 5
    _expect(cfg, T.TPS_EINVAL, "beyond n_micro")
    cfg = W.tiny()
    cfg.n_micro = 65
    _expect(cfg, T.TPS_EINVAL, "n_micro")
    c = W.tiny().to_c()
    c.abi_version = 99
    info = T.PlanInfo()
    assert T.lib().tps_plan(C.byref(c), C.byref(info)) == T.TPS_EINVAL
    assert b"abi_version" in T.lib().tps_last_error()


def test_op_argument_errors_without_gpu():
    # argument checks run before any launch, so they work without a device
    with pytest.raises(T.TpsError) as e:
        T.op_gemm(T.TPS_BF16, T.GEMM_NT, T.EPI_STORE, 64, 64, 60, None, 60, None, 60, None, 64)
    assert e.value.code == T.TPS_EINVAL
    with pytest.raises(T.TpsError):
        T.op_attention_fwd(T.TPS_BF16, 1, 16, 2, 96, None, None, None)
    with pytest.raises(T.TpsError):
        T.op_layernorm_fwd(T.TPS_F32, 4, 20000, None, None, None, 1e-5, None)
    # 100 rows: segments of 64 rows (multiple of 32, at least 64) -> 2 partials per column
    assert T.op_workspace_bytes(T.WS_COLSUM, 100, 64) == 2 * 64 * 4
    assert T.op_workspace_bytes(T.WS_COLSUM, 8192, 64) == 16 * 64 * 4
    assert T.op_workspace_bytes(T.WS_ATTN_BWD, 256, 4) == 256 * 4 * 4


def test_stage_init_argument_errors_without_gpu():
    # the memory checks run before any device call: fake (never dereferenced)
    # device addresses are enough to reach each of them
    cfg = W.tiny("offload")
    p = T.plan(cfg)
    L = cfg.n_layers
    blk = (C.c_void_p * L)(*([0x10000] * L))
    gblk = (C.c_void_p * L)(*([0x20000] * L))
    prm = T.Params(C.cast(blk, C.POINTER(C.c_void_p)), C.cast(gblk, C.POINTER(C.c_void_p)))
    c = cfg.to_c()

    def init(arena, nbytes, host, hbytes, cs, xs, ps):
        h = C.c_void_p()
        mem = T.Memory(arena, nbytes, host, hbytes, cs, xs, ps)
        rc = T.lib().tps_stage_init(C.byref(c), C.byref(prm), C.byref(mem), C.byref(h))
        assert not h.value
        return rc, T.lib().tps_last_error().decode()

    A, HB = p["device_arena_bytes"], p["host_arena_bytes"]
    assert HB > 0
    rc, msg = init(0x100000, A - 1, 0x200000, HB, 0x1, None, None)
    assert rc == T.TPS_ENOMEM and "device arena" in msg
    rc, msg = init(0x100080, A, 0x200000, HB, 0x1, None, None)
    assert rc == T.TPS_EINVAL and "aligned" in msg
    rc, msg = init(0x100000, A, 0x200000, HB - 1, 0x1, None, None)
    assert rc == T.TPS_ENOMEM and "host arena" in msg
    rc, msg = init(0x100000, A, 0x200000, HB, 0x1, 0x1, None)
    assert rc == T.TPS_EINVAL and "distinct" in msg
    rc, msg = init(0x100000, A, 0x200000, HB, 0x1, 0x2, 0x1)
    assert rc == T.TPS_EINVAL and "distinct" in msg


def test_param_layout_offsets():
    cfg = W.tiny()
    po, pb, go, gb = T.param_layout(cfg)
    h, f = cfg.hidden, cfg.mlp
    sizes = [3 * h * h, 3 * h, h * h, h, f * h, f, h * f, h, h, h, h, h]
    off = 0
    for i, n in enumerate(sizes):
        assert po[i] == off and po[i] % 256 == 0
        off = _align(off + 4 * n)
    assert pb == off
    assert gb == pb   # f32 storage: same layout as the gradients


def test_oversubscribed_stage_exceeds_hbm_only_when_kept():
    """The hidden-8192 streamed stage with 20 micro-batches in flight: keeping
    every tensor (activations at the in-flight peak, bf16 weights and f32
    gradients of all 12 layers) would need more than the 288 GB of HBM of one
    MI355X, while the planned peak with layer-input recompute and streamed
    weights and gradients stays far below it."""
    from paper_2503_03182_amd import configs as W
    cfg = W.stage12_h8192_stream_m20()
    info = T.plan(cfg)
    L = cfg.n_layers
    keep_all = info["keep_all_bytes"] + L * (info["param_bytes"] + info["grad_bytes"])
    assert keep_all > 288e9
    assert info["predicted_peak_bytes"] < 0.25 * 288e9
    # the same stage at 8 micro-batches fits either way (the workload's
    # premise needs the larger in-flight count)
    info8 = T.plan(W.stage12_h8192_stream())
    assert info8["keep_all_bytes"] + L * (info8["param_bytes"] + info8["grad_bytes"]) < 288e9


def test_wgrad_stream_choice():
    """AUTO issues the parameter-gradient kernels inline from 4096 tokens per
    micro-batch on; SIDE and INLINE force either arrangement; other values are
    rejected."""
    import dataclasses
    small, large = W.stage4_h2048(), W.stage12_h8192_stream()
    assert small.tokens < 4096 <= large.tokens
    assert T.plan(small)["wgrad_inline"] == 0
    assert T.plan(large)["wgrad_inline"] == 1
    assert T.plan(W.stage4_seq8192_recompute())["wgrad_inline"] == 1
    assert T.plan(dataclasses.replace(small, wgrad_stream=T.WGRAD_INLINE))["wgrad_inline"] == 1
    assert T.plan(dataclasses.replace(large, wgrad_stream=T.WGRAD_SIDE))["wgrad_inline"] == 0
    with pytest.raises(T.TpsError):
        T.plan(dataclasses.replace(small, wgrad_stream=3))
