"""ctypes binding of libtpstage.so (include/tpstage.h, include/tpstage_ops.h).

Argument marshalling only: every step of the stage runs in the library's HIP
kernels.  PyTorch supplies device memory, pinned host memory and streams.  If
the library has not been built, importing the binding raises at first use;
there is no fallback path.
"""
from __future__ import annotations

import ctypes as C
import os
from dataclasses import dataclass, field
from typing import Optional, Sequence

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libtpstage.so")

# --- constants (mirror tpstage.h) ------------------------------------------
TPS_ABI_VERSION = 7
TPS_OK, TPS_EINVAL, TPS_ENOMEM, TPS_EORDER, TPS_EHIP, TPS_ETIMEOUT, TPS_ESTATE = 0, -1, -2, -3, -4, -5, -6
TPS_F32, TPS_BF16 = 0, 1
KEEP, RECOMPUTE, OFFLOAD = 0, 1, 2
TENSORS = ("x", "a", "qkv", "o", "lse", "x1", "c", "u", "g", "ln1", "ln2")
T_INDEX = {n: i for i, n in enumerate(TENSORS)}
W_RESIDENT, W_STREAM = 0, 1
Q_NONE, Q_FP8_ROW = 0, 1
WGRAD_AUTO, WGRAD_SIDE, WGRAD_INLINE = 0, 1, 2
ARCH_GPT, ARCH_LLAMA = 0, 1
GRAN_LAYER, GRAN_SEGMENT = 0, 1
OP_F, OP_B, OP_R = 0, 1, 2
PARAMS = ("w_qkv", "b_qkv", "w_o", "b_o", "w_1", "b_1", "w_2", "b_2", "g1", "be1", "g2", "be2")
GEMM_NT, GEMM_NN, GEMM_TN = 0, 1, 2
EPI_STORE, EPI_BIAS, EPI_BIAS_RESID, EPI_BIAS_GELU, EPI_GELU_GRAD, EPI_ACC_F32 = range(6)
WS_COLSUM, WS_ATTN_BWD = 0, 1

_ERRNAMES = {TPS_EINVAL: "TPS_EINVAL", TPS_ENOMEM: "TPS_ENOMEM", TPS_EORDER: "TPS_EORDER",
             TPS_EHIP: "TPS_EHIP", TPS_ETIMEOUT: "TPS_ETIMEOUT", TPS_ESTATE: "TPS_ESTATE"}


class TpsError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"{_ERRNAMES.get(code, code)}: {msg}")
        self.code = code


# --- structures --------------------------------------------------------------
class Config(C.Structure):
    _fields_ = [
        ("abi_version", C.c_int32), ("n_layers", C.c_int32), ("hidden", C.c_int32),
        ("n_heads", C.c_int32), ("mlp", C.c_int32), ("seq", C.c_int32),
        ("micro_batch", C.c_int32), ("n_micro", C.c_int32), ("dtype", C.c_int32),
        ("ln_eps", C.c_float), ("policy", C.POINTER(C.c_uint8)), ("offload_mb_mask", C.c_uint64),
        ("offload_auto", C.c_int32), ("weights", C.c_int32), ("window", C.c_int32),
        ("recompute_granularity", C.c_int32), ("n_ops", C.c_int32), ("ops", C.POINTER(C.c_int32)),
        ("inflight", C.c_int32), ("link_gbps_hint", C.c_float), ("tflops_hint", C.c_float),
        ("lookahead", C.c_int32), ("weights_quant", C.c_int32), ("wgrad_stream", C.c_int32),
        ("arch", C.c_int32), ("n_kv_heads", C.c_int32), ("rope_base", C.c_float), ("group_wgrad", C.c_int32),
    ]


class PlanInfo(C.Structure):
    _fields_ = [
        ("device_arena_bytes", C.c_uint64), ("host_arena_bytes", C.c_uint64),
        ("slot_bytes", C.c_uint64), ("n_slots", C.c_int32),
        ("offload_slot_bytes", C.c_uint64), ("n_offload_slots", C.c_int32),
        ("n_host_slots", C.c_int32), ("max_inflight", C.c_int32),
        ("replay_bytes", C.c_uint64), ("work_bytes", C.c_uint64),
        ("weight_window_bytes", C.c_uint64), ("param_bytes", C.c_uint64),
        ("grad_bytes", C.c_uint64), ("keep_all_bytes", C.c_uint64),
        ("predicted_peak_bytes", C.c_uint64), ("offload_mb_mask", C.c_uint64),
        ("n_offload_mbs", C.c_int32), ("n_replay_layers", C.c_int32),
        ("fwd_flops", C.c_double), ("bwd_flops", C.c_double), ("recompute_flops", C.c_double),
        ("h2d_bytes", C.c_uint64), ("d2h_bytes", C.c_uint64), ("wgrad_inline", C.c_int32),
        ("group_wgrad_slots", C.c_int32),
    ]

    def as_dict(self) -> dict:
        return {k: getattr(self, k) for k, _ in self._fields_}


class Params(C.Structure):
    _fields_ = [("layer_params", C.POINTER(C.c_void_p)), ("layer_grads", C.POINTER(C.c_void_p))]


class Memory(C.Structure):
    _fields_ = [("device_arena", C.c_void_p), ("device_bytes", C.c_uint64),
                ("host_arena", C.c_void_p), ("host_bytes", C.c_uint64),
                ("compute_stream", C.c_void_p), ("copy_stream", C.c_void_p), ("prefetch_stream", C.c_void_p)]


class KernelTime(C.Structure):
    _fields_ = [("name", C.c_char * 120), ("launches", C.c_uint64), ("ms", C.c_double),
                ("flops", C.c_double), ("bytes", C.c_double)]


class TPipeConfig(C.Structure):
    _fields_ = [("stages", C.c_int32), ("micro", C.c_int32), ("t_recomp", C.c_int32), ("delay", C.c_int32)]


class TPipeTask(C.Structure):
    _fields_ = [("kind", C.c_int32), ("chunk", C.c_int32), ("mb", C.c_int32), ("start", C.c_int32),
                ("end", C.c_int32)]


class TPipeResult(C.Structure):
    _fields_ = [("delay", C.c_int32), ("makespan", C.c_int32), ("busy", C.c_int32), ("bubble_ratio", C.c_double),
                ("peak_blocks_chunk1", C.c_int32), ("peak_blocks_chunk2", C.c_int32),
                ("peak_buffer_blocks", C.c_int32), ("peak_blocks", C.c_int32),
                ("max_stage_peak_blocks", C.c_int32), ("life_chunk1", C.c_int32), ("life_chunk2", C.c_int32),
                ("offload_window", C.c_int32), ("upload_window", C.c_int32)]


class AdamW(C.Structure):
    _fields_ = [("lr", C.c_float), ("beta1", C.c_float), ("beta2", C.c_float), ("eps", C.c_float),
                ("weight_decay", C.c_float)]


class Stats(C.Structure):
    _fields_ = [("h2d_bytes", C.c_uint64), ("d2h_bytes", C.c_uint64), ("kernels", C.c_uint64),
                ("replays", C.c_uint64), ("ops_done", C.c_int32), ("host_update_ms", C.c_double),
                ("host_wait_ms", C.c_double), ("host_updates", C.c_int32)]


# --- library -----------------------------------------------------------------
_lib = None

EXPORTED = (
    "tps_param_layout", "tps_plan", "tps_stage_init", "tps_stage_begin_iteration",
    "tps_stage_forward", "tps_stage_backward", "tps_stage_forward_group",
    "tps_stage_backward_group", "tps_stage_sync", "tps_stage_sync_for", "tps_stage_stats", "tps_stage_destroy",
    "tps_last_error", "tps_op_gemm", "tps_op_layernorm_fwd", "tps_op_layernorm_bwd",
    "tps_op_attention_fwd", "tps_op_attention_bwd", "tps_op_colsum", "tps_op_gelu",
    "tps_op_workspace_bytes", "tps_stage_time_kernels", "tps_stage_kernel_times",
    "tps_host_alloc", "tps_host_free", "tps_tpipe_schedule", "tps_op_attention_bwd_noalloc",
    "tps_op_attention_bwd_noalloc_max_rows", "tps_param_layout_q", "tps_host_adamw_layer",
    "tps_stage_set_optimizer", "tps_stage_set_optimizer_split", "tps_op_dequant_fp8_rows", "tps_op_rmsnorm_fwd",
    "tps_op_rmsnorm_bwd", "tps_op_rope",
    "tps_op_swiglu_fwd", "tps_op_swiglu_bwd", "tps_op_attention_gqa_fwd", "tps_op_attention_gqa_bwd",
)


def lib_path() -> str:
    return _LIB_PATH


def lib() -> C.CDLL:
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            raise RuntimeError(f"{_LIB_PATH} is missing: build it with "
                               "`python -m paper_2503_03182_amd.build` (no fallback exists)")
        L = C.CDLL(_LIB_PATH)
        vp, i32, i64, u64 = C.c_void_p, C.c_int, C.c_int64, C.c_uint64
        L.tps_last_error.restype = C.c_char_p
        L.tps_param_layout.argtypes = [C.POINTER(Config), C.POINTER(C.c_uint64), C.POINTER(C.c_uint64),
                                       C.POINTER(C.c_uint64), C.POINTER(C.c_uint64)]
        L.tps_plan.argtypes = [C.POINTER(Config), C.POINTER(PlanInfo)]
        L.tps_stage_init.argtypes = [C.POINTER(Config), C.POINTER(Params), C.POINTER(Memory), C.POINTER(vp)]
        L.tps_stage_begin_iteration.argtypes = [vp, i32]
        L.tps_stage_forward.argtypes = [vp, i32, vp, vp]
        L.tps_stage_backward.argtypes = [vp, i32, vp, vp]
        L.tps_stage_forward_group.argtypes = [vp, i32, i32, C.POINTER(vp), C.POINTER(vp)]
        L.tps_stage_backward_group.argtypes = [vp, i32, i32, C.POINTER(vp), C.POINTER(vp)]
        L.tps_stage_sync.argtypes = [vp]
        L.tps_stage_sync_for.argtypes = [vp, C.c_double]
        L.tps_stage_stats.argtypes = [vp, C.POINTER(Stats)]
        L.tps_stage_destroy.argtypes = [vp]
        L.tps_stage_time_kernels.argtypes = [vp, C.c_char_p]
        L.tps_stage_kernel_times.argtypes = [vp, C.POINTER(KernelTime), i32, C.POINTER(C.c_int)]
        L.tps_op_gemm.argtypes = [i32, i32, i32, i32, i32, i32, vp, i64, vp, i64, vp, i64, vp, vp, i64, vp, i64, vp]
        L.tps_op_layernorm_fwd.argtypes = [i32, i32, i32, vp, vp, vp, C.c_float, vp, vp, vp, vp]
        L.tps_op_layernorm_bwd.argtypes = [i32, i32, i32, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp]
        L.tps_op_attention_fwd.argtypes = [i32, i32, i32, i32, i32, vp, vp, vp, vp]
        L.tps_op_attention_bwd.argtypes = [i32, i32, i32, i32, i32, vp, vp, vp, vp, vp, vp, vp]
        L.tps_op_attention_bwd_noalloc.argtypes = [i32, i32, i32, i32, i32, vp, vp, vp, vp, vp, vp]
        L.tps_op_attention_bwd_noalloc_max_rows.argtypes = []
        L.tps_op_attention_bwd_noalloc_max_rows.restype = i64
        L.tps_op_dequant_fp8_rows.argtypes = [i64, i64, vp, vp, vp, vp]
        L.tps_op_colsum.argtypes = [i32, i32, i32, vp, i64, vp, vp, vp]
        L.tps_op_rmsnorm_fwd.argtypes = [i32, i32, i32, vp, vp, C.c_float, vp, vp, vp]
        L.tps_op_rmsnorm_bwd.argtypes = [i32, i32, i32, vp, vp, vp, vp, vp, vp, vp, vp, vp]
        L.tps_op_rope.argtypes = [vp, i64, i32, i32, i32, i32, C.c_float, i32, vp, vp]
        L.tps_op_swiglu_fwd.argtypes = [i32, i32, vp, vp, vp]
        L.tps_op_swiglu_bwd.argtypes = [i32, i32, vp, vp, vp, vp]
        L.tps_op_attention_gqa_fwd.argtypes = [i32, i32, i32, i32, vp, vp, vp, vp]
        L.tps_op_attention_gqa_bwd.argtypes = [i32, i32, i32, i32, vp, vp, vp, vp, vp, vp, vp, vp]
        L.tps_op_gelu.argtypes = [i32, i64, vp, vp, vp]
        L.tps_op_workspace_bytes.argtypes = [i32, i64, i64]
        L.tps_op_workspace_bytes.restype = u64
        L.tps_host_alloc.argtypes = [u64, C.POINTER(vp)]
        L.tps_host_free.argtypes = [vp]
        L.tps_param_layout_q.argtypes = [C.POINTER(Config), C.POINTER(C.c_uint64), C.POINTER(C.c_uint64),
                                         C.POINTER(C.c_uint64)]
        L.tps_host_adamw_layer.argtypes = [C.POINTER(Config), C.POINTER(AdamW), i32, vp, vp, vp, vp, vp, i32, i32]
        L.tps_stage_set_optimizer.argtypes = [vp, C.POINTER(AdamW), C.POINTER(vp), C.POINTER(vp), C.POINTER(vp),
                                              i32, i32]
        L.tps_stage_set_optimizer_split.argtypes = [vp, C.POINTER(AdamW), C.POINTER(vp), C.POINTER(vp), C.POINTER(vp),
                                                   C.POINTER(vp), i32, i32, i32]
        L.tps_tpipe_schedule.argtypes = [C.POINTER(TPipeConfig), i32, C.POINTER(TPipeTask), i32,
                                         C.POINTER(C.c_int32), C.POINTER(TPipeResult)]
        _lib = L
    return _lib


def check(rc: int) -> None:
    if rc != TPS_OK:
        raise TpsError(rc, lib().tps_last_error().decode())


class HostBuffer:
    """Exactly `nbytes` of pinned host memory from tps_host_alloc (the
    caching pinned allocator of the framework rounds requests up to powers of
    two, which the host side of a large streamed stage cannot afford).
    `data_ptr()` gives the address, `numpy()` a uint8 view."""

    def __init__(self, nbytes: int):
        self.nbytes = int(nbytes)
        p = C.c_void_p()
        check(lib().tps_host_alloc(self.nbytes, C.byref(p)))
        self._p = p.value

    def data_ptr(self) -> int:
        return self._p or 0

    def numpy(self):
        import numpy as np
        if not self._p:
            return np.zeros(0, dtype=np.uint8)
        return np.ctypeslib.as_array((C.c_uint8 * self.nbytes).from_address(self._p))

    def free(self) -> None:
        if self._p:
            check(lib().tps_host_free(self._p))
            self._p = None

    def __del__(self):
        try:
            self.free()
        except Exception:
            pass


# --- configuration -----------------------------------------------------------
@dataclass
class StageConfig:
    n_layers: int
    hidden: int
    n_heads: int
    mlp: int
    seq: int
    micro_batch: int
    n_micro: int
    dtype: str = "bf16"                      # "bf16" or "f32"
    ln_eps: float = 1e-5
    policy: Optional[list] = None            # [L] dicts name -> KEEP/RECOMPUTE/OFFLOAD
    offload_mb_mask: int = 0
    offload_auto: bool = False
    weights: int = W_RESIDENT
    window: int = 2
    granularity: int = GRAN_SEGMENT
    ops: Optional[Sequence] = None           # [("F"|"B", mb)]
    inflight: int = 0
    link_gbps_hint: float = 50.0
    tflops_hint: float = 1000.0
    lookahead: int = 1
    weights_quant: int = Q_NONE
    wgrad_stream: int = WGRAD_AUTO
    arch: int = ARCH_GPT
    n_kv_heads: int = 0                      # LLAMA: key/value heads (0: n_heads)
    rope_base: float = 10000.0
    group_wgrad: int = 0                     # 1: batch a backward group's weight gradients per layer
    # drive the planned order with layer-major group calls (each run of
    # consecutive F (or B) tasks is one tps_stage_forward_group / _backward_group)
    layer_major: bool = False
    _keep: list = field(default_factory=list, repr=False)

    def groups(self) -> list:
        """The planned order as runs of consecutive micro-batches with the same
        task kind: [("F"|"B", first_mb, count)]."""
        out = []
        for k, mb in self.order():
            if out and out[-1][0] == k and out[-1][1] + out[-1][2] == mb:
                out[-1] = (k, out[-1][1], out[-1][2] + 1)
            else:
                out.append((k, mb, 1))
        return out

    @property
    def tokens(self) -> int:
        return self.micro_batch * self.seq

    @property
    def dtype_code(self) -> int:
        return TPS_BF16 if self.dtype == "bf16" else TPS_F32

    def to_c(self) -> Config:
        c = Config()
        c.abi_version = TPS_ABI_VERSION
        c.n_layers, c.hidden, c.n_heads, c.mlp = self.n_layers, self.hidden, self.n_heads, self.mlp
        c.seq, c.micro_batch, c.n_micro = self.seq, self.micro_batch, self.n_micro
        c.dtype = self.dtype_code
        c.ln_eps = self.ln_eps
        self._keep = []
        if self.policy is not None:
            flat = (C.c_uint8 * (self.n_layers * len(TENSORS)))()
            for l in range(self.n_layers):
                for name, mode in self.policy[l].items():
                    flat[l * len(TENSORS) + T_INDEX[name]] = mode
            self._keep.append(flat)
            c.policy = C.cast(flat, C.POINTER(C.c_uint8))
        c.offload_mb_mask = self.offload_mb_mask
        c.offload_auto = int(self.offload_auto)
        c.weights, c.window, c.recompute_granularity = self.weights, self.window, self.granularity
        if self.ops is not None:
            arr = (C.c_int32 * (2 * len(self.ops)))()
            for i, (k, mb) in enumerate(self.ops):
                arr[2 * i] = OP_F if k == "F" else OP_B
                arr[2 * i + 1] = mb
            self._keep.append(arr)
            c.n_ops = len(self.ops)
            c.ops = C.cast(arr, C.POINTER(C.c_int32))
        c.inflight = self.inflight
        c.link_gbps_hint, c.tflops_hint = self.link_gbps_hint, self.tflops_hint
        c.lookahead = self.lookahead
        c.weights_quant = self.weights_quant
        c.wgrad_stream = self.wgrad_stream
        c.arch, c.n_kv_heads, c.rope_base = self.arch, self.n_kv_heads, self.rope_base
        c.group_wgrad = int(self.group_wgrad)
        return c

    def order(self) -> list:
        """The planned op order (the library's default when ops is None)."""
        if self.ops is not None:
            return list(self.ops)
        M = self.n_micro
        W = M if self.inflight <= 0 or self.inflight > M else self.inflight
        out = [("F", i) for i in range(W)]
        nxt = W
        for i in range(M):
            out.append(("B", i))
            if nxt < M:
                out.append(("F", nxt))
                nxt += 1
        return out


def plan(cfg: StageConfig) -> dict:
    info = PlanInfo()
    c = cfg.to_c()
    check(lib().tps_plan(C.byref(c), C.byref(info)))
    return info.as_dict()


def param_layout(cfg: StageConfig):
    po = (C.c_uint64 * len(PARAMS))()
    go = (C.c_uint64 * len(PARAMS))()
    pb, gb = C.c_uint64(), C.c_uint64()
    c = cfg.to_c()
    check(lib().tps_param_layout(C.byref(c), po, C.byref(pb), go, C.byref(gb)))
    return list(po), pb.value, list(go), gb.value


def param_layout_q(cfg: StageConfig):
    """(offsets of the 12 tensors, offsets of the 4 matrices' row scales, bytes)
    of one layer's quantized host parameter block."""
    qo = (C.c_uint64 * len(PARAMS))()
    so = (C.c_uint64 * 4)()
    nb = C.c_uint64()
    c = cfg.to_c()
    check(lib().tps_param_layout_q(C.byref(c), qo, so, C.byref(nb)))
    return list(qo), list(so), nb.value


def host_adamw_layer(cfg: StageConfig, step: int, master, m, v, grad, params_out, quant: int = Q_NONE,
                     lr=1e-3, beta1=0.9, beta2=0.95, eps=1e-8, weight_decay=0.0, n_threads: int = 0) -> None:
    """tps_host_adamw_layer on host buffers (anything with data_ptr(), or
    numpy arrays): one AdamW step of a layer (step >= 1; 0 = only write
    params_out) and its parameter block for the device."""
    def ptr(a):
        if a is None:
            return None
        if hasattr(a, "data_ptr"):
            return a.data_ptr()
        return a.ctypes.data
    opt = AdamW(lr, beta1, beta2, eps, weight_decay)
    c = cfg.to_c()
    check(lib().tps_host_adamw_layer(C.byref(c), C.byref(opt), step, ptr(master), ptr(m), ptr(v), ptr(grad),
                                     ptr(params_out), quant, n_threads))


# --- T-Pipe schedule -------------------------------------------------------------
def tpipe_schedule(stages: int, micro: int, stage: int = 0, t_recomp: bool = False, delay: int = -1):
    """The T-Pipe two-chunk schedule of `stages` pipeline stages over `micro`
    micro-batches, simulated in T_unit (tps_tpipe_schedule).  Returns
    (summary dict, tasks of `stage` in execution order as
    (kind "F"|"B"|"R", chunk 1|2, mb, start, end))."""
    cfg = TPipeConfig(stages, micro, int(t_recomp), delay)
    res = TPipeResult()
    n = C.c_int32()
    check(lib().tps_tpipe_schedule(C.byref(cfg), stage, None, 0, C.byref(n), C.byref(res)))
    arr = (TPipeTask * max(n.value, 1))()
    check(lib().tps_tpipe_schedule(C.byref(cfg), stage, arr, n.value, C.byref(n), C.byref(res)))
    names = {OP_F: "F", OP_B: "B", OP_R: "R"}
    tasks = [(names[t.kind], t.chunk, t.mb, t.start, t.end) for t in arr[:n.value]]
    return {k: getattr(res, k) for k, _ in TPipeResult._fields_}, tasks


def chunk_orders(tasks):
    """Splits a stage's T-Pipe task list into the F/B order of each chunk's
    layers (StageConfig.ops form: [("F"|"B", mb)]); a recompute task is run by
    the chunk's backward that follows it.  Also returns the interleaved call
    sequence [(chunk, "F"|"B", mb)]."""
    orders = {1: [], 2: []}
    calls = []
    for kind, chunk, mb, _, _ in tasks:
        if kind == "R":
            continue
        orders[chunk].append((kind, mb))
        calls.append((chunk, kind, mb))
    return orders[1], orders[2], calls


def tpipe_t_offload_stages(t_offload, t_upload, t_unit, micro=None, max_stages=256):
    """Smallest pipeline depths p at which T-Offload's host transfers of one
    chunk fit T-Pipe's bubbles (appendix "Scalability of T-Offload"): the
    gradient offload plus host optimizer step of a chunk (`t_offload`) within
    the cool-down window of the simulated schedule, and the reload of a
    chunk's weights (`t_upload`) within its warm-up window.  `t_unit` is the
    forward of one chunk for one micro-batch (a backward takes two), all three
    in the same unit; the windows are those of stage 0 of the plain schedule
    (no T-Recomp, no delay) with max(micro, 2p) micro-batches, where every
    stage has the same windows.  Returns (p for the offload, p for the
    upload), None where no p up to max_stages suffices."""
    if not (t_unit > 0) or t_offload < 0 or t_upload < 0:
        raise ValueError("t_unit must be positive, t_offload and t_upload non-negative")
    p_off = p_up = None
    for p in range(1, max_stages + 1):
        r, _ = tpipe_schedule(p, max(micro or 0, 2 * p), delay=0)
        if p_off is None and t_offload <= r["offload_window"] * t_unit:
            p_off = p
        if p_up is None and t_upload <= r["upload_window"] * t_unit:
            p_up = p
        if p_off is not None and p_up is not None:
            break
    return p_off, p_up


# --- stage ---------------------------------------------------------------------
class Stage:
    """One pipeline stage on one GPU.  The device arena is a torch allocation
    and the pinned host arena a HostBuffer, both sized by the plan; parameter
    and f32 gradient blocks are byte buffers (torch tensors or HostBuffers)
    laid out by param_layout().

    Stream order: the stage's kernels run on its compute stream `cs`: the
    given one, else the stream current at construction unless that is the
    device's default (null) stream, else a private stream.  Every call that
    enqueues work first makes `cs` wait for the caller's current stream (so
    inputs and parameters written there are complete) and afterwards makes
    the caller's current stream wait for `cs` (so outputs are complete, and
    buffers freed there are not reused while the stage still reads them).
    When the two are the same stream no event is needed.  Work on the
    default stream synchronizes with the copy and side streams the library
    creates, so callers that want calls to overlap the library's copies run
    under a `torch.cuda.stream(...)` of their own."""

    def __init__(self, cfg: StageConfig, layer_params, layer_grads, device="cuda",
                 compute_stream=None, copy_stream=None, prefetch_stream=None):
        import torch
        self.cfg = cfg
        self.info = plan(cfg)
        self.device = torch.device(device)
        self.arena = torch.empty(max(self.info["device_arena_bytes"], 256), dtype=torch.uint8, device=self.device)
        hb = self.info["host_arena_bytes"]
        self.host = HostBuffer(hb) if hb else None
        # compute on a torch stream; copy streams default to the stage's own
        if compute_stream is None:
            cur = torch.cuda.current_stream(self.device)
            compute_stream = cur if cur.cuda_stream != 0 else torch.cuda.Stream(device=self.device)
        self.cs = compute_stream
        self.xs, self.ps = copy_stream, prefetch_stream
        self.layer_params, self.layer_grads = list(layer_params), list(layer_grads)
        L = cfg.n_layers
        self._pp = (C.c_void_p * L)(*[t.data_ptr() for t in self.layer_params])
        self._gp = (C.c_void_p * L)(*[t.data_ptr() for t in self.layer_grads])
        prm = Params(C.cast(self._pp, C.POINTER(C.c_void_p)), C.cast(self._gp, C.POINTER(C.c_void_p)))
        mem = Memory(self.arena.data_ptr(), self.arena.numel(),
                     self.host.data_ptr() if self.host is not None else None, hb,
                     self.cs.cuda_stream, _stream(self.xs), _stream(self.ps))
        self._c = cfg.to_c()
        h = C.c_void_p()
        check(lib().tps_stage_init(C.byref(self._c), C.byref(prm), C.byref(mem), C.byref(h)))
        self.handle = h

    def _ordered(self, fn, *args) -> None:
        """Runs one enqueuing call between the two stream waits described in
        the class docstring."""
        import torch
        cur = torch.cuda.current_stream(self.device)
        same = cur.cuda_stream == self.cs.cuda_stream
        if not same:
            self.cs.wait_stream(cur)
        try:
            check(fn(*args))
        finally:
            if not same:
                cur.wait_stream(self.cs)

    def begin_iteration(self, zero_grads: bool = True) -> None:
        self._ordered(lib().tps_stage_begin_iteration, self.handle, int(zero_grads))

    def forward(self, mb: int, x, y) -> None:
        self._ordered(lib().tps_stage_forward, self.handle, mb, x.data_ptr(), y.data_ptr())

    def backward(self, mb: int, dy, dx) -> None:
        self._ordered(lib().tps_stage_backward, self.handle, mb, dy.data_ptr(), dx.data_ptr())

    def forward_group(self, mb0: int, xs, ys) -> None:
        n = len(xs)
        a = (C.c_void_p * n)(*[t.data_ptr() for t in xs])
        b = (C.c_void_p * n)(*[t.data_ptr() for t in ys])
        self._ordered(lib().tps_stage_forward_group, self.handle, mb0, n, a, b)

    def backward_group(self, mb0: int, dys, dxs) -> None:
        n = len(dys)
        a = (C.c_void_p * n)(*[t.data_ptr() for t in dys])
        b = (C.c_void_p * n)(*[t.data_ptr() for t in dxs])
        self._ordered(lib().tps_stage_backward_group, self.handle, mb0, n, a, b)

    def sync(self) -> None:
        check(lib().tps_stage_sync(self.handle))

    def set_optimizer(self, master, m, v, first_step: int = 1, lr=1e-3, beta1=0.9, beta2=0.95, eps=1e-8,
                      weight_decay=0.0, n_threads: int = 0, dparams=None) -> None:
        """tps_stage_set_optimizer(_split): AdamW of every streamed layer once
        its gradients of the iteration are final (master, m, v: per-layer f32
        blocks in the gradient layout, each with data_ptr() or a numpy array).
        With dparams (device parameter blocks of the first len(dparams)
        layers), those layers' master, m and v are device tensors and their
        update runs on the GPU; the other layers' blocks are host memory."""
        def ptrs(blocks):
            return (C.c_void_p * len(blocks))(*[b.data_ptr() if hasattr(b, "data_ptr") else b.ctypes.data
                                                for b in blocks])
        dparams = list(dparams or [])
        self._opt_keep = (ptrs(master), ptrs(m), ptrs(v), ptrs(dparams) if dparams else None, master, m, v, dparams)
        opt = AdamW(lr, beta1, beta2, eps, weight_decay)
        cast = lambda a: C.cast(a, C.POINTER(C.c_void_p)) if a is not None else None
        check(lib().tps_stage_set_optimizer_split(self.handle, C.byref(opt), cast(self._opt_keep[0]),
                                                  cast(self._opt_keep[1]), cast(self._opt_keep[2]),
                                                  cast(self._opt_keep[3]), len(dparams), first_step, n_threads))

    def sync_for(self, timeout_ms: float) -> int:
        """Bounded wait: TPS_OK when every stream of the stage is idle,
        TPS_ETIMEOUT if work is still pending after timeout_ms (the work keeps
        running); raises on other errors."""
        rc = lib().tps_stage_sync_for(self.handle, float(timeout_ms))
        if rc not in (TPS_OK, TPS_ETIMEOUT):
            check(rc)
        return rc

    def stats(self) -> dict:
        s = Stats()
        check(lib().tps_stage_stats(self.handle, C.byref(s)))
        return {k: getattr(s, k) for k, _ in Stats._fields_}

    def time_kernels(self, prefix: Optional[str]) -> None:
        """Bracket launches whose kernel name starts with prefix with HIP
        events ("" = all, None = off); clears accumulated times."""
        check(lib().tps_stage_time_kernels(self.handle, None if prefix is None else prefix.encode()))

    def kernel_times(self) -> list:
        n = C.c_int()
        check(lib().tps_stage_kernel_times(self.handle, None, 0, C.byref(n)))
        arr = (KernelTime * max(n.value, 1))()
        check(lib().tps_stage_kernel_times(self.handle, arr, n.value, C.byref(n)))
        return [dict(name=a.name.decode(), launches=a.launches, ms=a.ms, flops=a.flops, bytes=a.bytes)
                for a in arr[:n.value]]

    def close(self) -> None:
        if getattr(self, "handle", None):
            lib().tps_stage_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


# --- op-level calls (torch tensors in, kernels run on `stream`) ----------------
def _ptr(t):
    return None if t is None else t.data_ptr()


def _stream(stream):
    return None if stream is None else stream.cuda_stream


def op_gemm(dtype, layout, epi, M, N, K, A, lda, B, ldb, Cm, ldc, bias=None, resid=None, ldr=0,
            aux=None, ldaux=0, stream=None):
    check(lib().tps_op_gemm(dtype, layout, epi, M, N, K, _ptr(A), lda, _ptr(B), ldb, _ptr(Cm), ldc,
                            _ptr(bias), _ptr(resid), ldr, _ptr(aux), ldaux, _stream(stream)))


def op_layernorm_fwd(dtype, rows, cols, x, gamma, beta, eps, out, mean=None, rstd=None, stream=None):
    check(lib().tps_op_layernorm_fwd(dtype, rows, cols, _ptr(x), _ptr(gamma), _ptr(beta), eps, _ptr(out),
                                     _ptr(mean), _ptr(rstd), _stream(stream)))


def op_layernorm_bwd(dtype, rows, cols, dout, x, mean, rstd, gamma, resid, dx, dgamma, dbeta, ws, stream=None):
    check(lib().tps_op_layernorm_bwd(dtype, rows, cols, _ptr(dout), _ptr(x), _ptr(mean), _ptr(rstd),
                                     _ptr(gamma), _ptr(resid), _ptr(dx), _ptr(dgamma), _ptr(dbeta), _ptr(ws),
                                     _stream(stream)))


def op_attention_fwd(dtype, b, s, nh, d, qkv, o, lse, stream=None):
    check(lib().tps_op_attention_fwd(dtype, b, s, nh, d, _ptr(qkv), _ptr(o), _ptr(lse), _stream(stream)))


def op_attention_bwd(dtype, b, s, nh, d, qkv, o, lse, do, dqkv, ws, stream=None):
    check(lib().tps_op_attention_bwd(dtype, b, s, nh, d, _ptr(qkv), _ptr(o), _ptr(lse), _ptr(do), _ptr(dqkv),
                                     _ptr(ws), _stream(stream)))


def op_attention_bwd_noalloc(dtype, b, s, nh, d, qkv, o, lse, do, dqkv, stream=None):
    check(lib().tps_op_attention_bwd_noalloc(dtype, b, s, nh, d, _ptr(qkv), _ptr(o), _ptr(lse), _ptr(do),
                                             _ptr(dqkv), _stream(stream)))


def op_dequant_fp8_rows(rows, cols, q, scale, out, stream=None):
    check(lib().tps_op_dequant_fp8_rows(rows, cols, _ptr(q), _ptr(scale), _ptr(out), _stream(stream)))


def op_colsum(dtype, rows, cols, x, ldx, out, ws, stream=None):
    check(lib().tps_op_colsum(dtype, rows, cols, _ptr(x), ldx, _ptr(out), _ptr(ws), _stream(stream)))


def op_rmsnorm_fwd(dtype, rows, cols, x, gamma, eps, out, rstd=None, stream=None):
    check(lib().tps_op_rmsnorm_fwd(dtype, rows, cols, _ptr(x), _ptr(gamma), eps, _ptr(out), _ptr(rstd),
                                   _stream(stream)))


def op_rmsnorm_bwd(dtype, rows, cols, dout, x, rstd, gamma, resid, dx, dgamma, ws, stream=None):
    check(lib().tps_op_rmsnorm_bwd(dtype, rows, cols, _ptr(dout), _ptr(x), _ptr(rstd), _ptr(gamma), _ptr(resid),
                                   _ptr(dx), _ptr(dgamma), _ptr(ws), _stream(stream)))


def op_rope(x, ld, rows, s, n_rot, d, base, inverse, table, stream=None):
    check(lib().tps_op_rope(_ptr(x), ld, rows, s, n_rot, d, base, int(inverse), _ptr(table), _stream(stream)))


def op_swiglu_fwd(rows, f, u, g, stream=None):
    check(lib().tps_op_swiglu_fwd(rows, f, _ptr(u), _ptr(g), _stream(stream)))


def op_swiglu_bwd(rows, f, dg, u, du, stream=None):
    check(lib().tps_op_swiglu_bwd(rows, f, _ptr(dg), _ptr(u), _ptr(du), _stream(stream)))


def op_attention_gqa_fwd(b, s, nh, nkv, qkv, o, lse, stream=None):
    check(lib().tps_op_attention_gqa_fwd(b, s, nh, nkv, _ptr(qkv), _ptr(o), _ptr(lse), _stream(stream)))


def op_attention_gqa_bwd(b, s, nh, nkv, qkv, o, lse, do, dqkv, ws, kv_ws, stream=None):
    check(lib().tps_op_attention_gqa_bwd(b, s, nh, nkv, _ptr(qkv), _ptr(o), _ptr(lse), _ptr(do), _ptr(dqkv),
                                         _ptr(ws), _ptr(kv_ws), _stream(stream)))


def op_gelu(dtype, n, u, g, stream=None):
    check(lib().tps_op_gelu(dtype, n, _ptr(u), _ptr(g), _stream(stream)))


def op_workspace_bytes(kind, rows, cols) -> int:
    return int(lib().tps_op_workspace_bytes(kind, rows, cols))
