"""Builds and drives the happens-before checker build of the stage library
(host code of csrc/stage.cpp, planner.cpp, errors.cpp compiled for the CPU
against the stand-in HIP runtime of tests/hb; kernels record the memory they
touch, nothing is computed).  Device and host buffers are fake addresses;
the checker reports every access that is not ordered after a conflicting
one."""
from __future__ import annotations

import ctypes as C
import os
import subprocess

from paper_2503_03182_amd import tpstage as T

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
CSRC = os.path.join(ROOT, "paper_2503_03182_amd", "csrc")
OUT = os.path.join(HERE, "_build", "libtpstage_hb.so")

_lib = None


def build() -> str:
    os.makedirs(os.path.dirname(OUT), exist_ok=True)
    tmp = f"{OUT}.{os.getpid()}.tmp"   # parallel test workers build side by side
    srcs = [os.path.join(CSRC, n) for n in ("stage.cpp", "planner.cpp", "errors.cpp", "host_optim.cpp")]
    srcs += [os.path.join(HERE, n) for n in ("hb_runtime.cpp", "hb_kernels.cpp")]
    cmd = ["g++", "-std=c++17", "-O1", "-fPIC", "-shared", "-pthread", "-I", os.path.join(HERE, "fakeinc"), "-I", HERE,
           "-I", os.path.join(ROOT, "include"), "-I", CSRC, *srcs, "-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode:
        raise RuntimeError("checker build failed:\n" + r.stderr)
    os.replace(tmp, OUT)
    return OUT


def lib() -> C.CDLL:
    global _lib
    if _lib is None:
        build()
        L = C.CDLL(OUT)
        vp, i32 = C.c_void_p, C.c_int
        L.tps_last_error.restype = C.c_char_p
        L.tps_plan.argtypes = [C.POINTER(T.Config), C.POINTER(T.PlanInfo)]
        L.tps_param_layout.argtypes = [C.POINTER(T.Config), C.POINTER(C.c_uint64), C.POINTER(C.c_uint64),
                                       C.POINTER(C.c_uint64), C.POINTER(C.c_uint64)]
        L.tps_stage_init.argtypes = [C.POINTER(T.Config), C.POINTER(T.Params), C.POINTER(T.Memory), C.POINTER(vp)]
        L.tps_stage_begin_iteration.argtypes = [vp, i32]
        L.tps_stage_forward.argtypes = [vp, i32, vp, vp]
        L.tps_stage_backward.argtypes = [vp, i32, vp, vp]
        L.tps_stage_forward_group.argtypes = [vp, i32, i32, C.POINTER(vp), C.POINTER(vp)]
        L.tps_stage_backward_group.argtypes = [vp, i32, i32, C.POINTER(vp), C.POINTER(vp)]
        L.tps_stage_sync.argtypes = [vp]
        L.tps_stage_destroy.argtypes = [vp]
        L.tps_hb_new_stream.argtypes = [C.c_char_p]
        L.tps_hb_new_stream.restype = vp
        L.tps_hb_name_region.argtypes = [C.c_uint64, C.c_uint64, C.c_char_p]
        L.tps_hb_host_access.argtypes = [C.c_uint64, C.c_uint64, i32]
        L.tps_hb_stream_access.argtypes = [vp, C.c_uint64, C.c_uint64, i32]
        L.tps_hb_report.restype = C.c_char_p
        L.tps_hb_waits.restype = C.c_int64
        L.tps_hb_drop_wait.argtypes = [C.c_int64]
        L.tps_hb_ops.restype = C.c_uint64
        _lib = L
    return _lib


def check(rc):
    if rc != T.TPS_OK:
        raise T.TpsError(rc, lib().tps_last_error().decode())


GiB = 1 << 30
TiB = 1 << 40


class FakeStage:
    """One stage object of the checker build with fake buffers: the arena,
    host arena, parameter and gradient blocks and the caller's x / y / dy / dx
    each in an address range of its own."""

    def __init__(self, cfg: T.StageConfig, tag: int = 0, own_copy_streams: bool = True, cs=None,
                 one_copy_stream: bool = False):
        L = lib()
        self.cfg = cfg
        c = cfg.to_c()
        self._c = c
        info = T.PlanInfo()
        check(L.tps_plan(C.byref(c), C.byref(info)))
        self.info = info.as_dict()
        po = (C.c_uint64 * 12)()
        go = (C.c_uint64 * 12)()
        pb, gb = C.c_uint64(), C.c_uint64()
        check(L.tps_param_layout(C.byref(c), po, C.byref(pb), go, C.byref(gb)))
        self.pbytes, self.gbytes = pb.value, gb.value
        base = (tag + 1) * 64 * TiB
        self.arena = base + 1 * TiB
        self.host = base + 2 * TiB
        self.params = [base + 3 * TiB + l * 16 * GiB for l in range(cfg.n_layers)]
        self.grads = [base + 4 * TiB + l * 16 * GiB for l in range(cfg.n_layers)]
        es = 2 if cfg.dtype == "bf16" else 4
        self.tbytes = cfg.tokens * cfg.hidden * es
        self.x = [base + 5 * TiB + mb * 4 * GiB for mb in range(cfg.n_micro)]
        self.y = [base + 6 * TiB + mb * 4 * GiB for mb in range(cfg.n_micro)]
        self.dy = [base + 7 * TiB + mb * 4 * GiB for mb in range(cfg.n_micro)]
        self.dx = [base + 8 * TiB + mb * 4 * GiB for mb in range(cfg.n_micro)]
        for name, a, n in [("arena", self.arena, self.info["device_arena_bytes"]),
                           ("host arena", self.host, self.info["host_arena_bytes"])]:
            L.tps_hb_name_region(a, max(n, 1), f"{name}[{tag}]".encode())
        for l in range(cfg.n_layers):
            L.tps_hb_name_region(self.params[l], self.pbytes, f"params[{tag}][{l}]".encode())
            L.tps_hb_name_region(self.grads[l], self.gbytes, f"grads[{tag}][{l}]".encode())
        for nm, arr in (("x", self.x), ("y", self.y), ("dy", self.dy), ("dx", self.dx)):
            for mb, a in enumerate(arr):
                L.tps_hb_name_region(a, self.tbytes, f"{nm}[{tag}][{mb}]".encode())
        self.cs = cs if cs is not None else L.tps_hb_new_stream(f"compute[{tag}]".encode())
        xs = None if own_copy_streams else L.tps_hb_new_stream(f"copy[{tag}]".encode())
        ps = None if own_copy_streams else L.tps_hb_new_stream(f"prefetch[{tag}]".encode())
        if one_copy_stream:
            xs = ps = L.tps_hb_new_stream(f"copy[{tag}]".encode())
        L_ = cfg.n_layers
        self._pp = (C.c_void_p * L_)(*self.params)
        self._gp = (C.c_void_p * L_)(*self.grads)
        prm = T.Params(C.cast(self._pp, C.POINTER(C.c_void_p)), C.cast(self._gp, C.POINTER(C.c_void_p)))
        mem = T.Memory(self.arena, max(self.info["device_arena_bytes"], 256), self.host if self.info["host_arena_bytes"] else None,
                       self.info["host_arena_bytes"], self.cs, xs, ps)
        h = C.c_void_p()
        # the caller fills parameters (and host blocks) before the stage exists
        for l in range(L_):
            if cfg.weights == T.W_STREAM:
                L.tps_hb_host_access(self.params[l], self.pbytes, 1)
                L.tps_hb_host_access(self.grads[l], self.gbytes, 1)
            else:
                L.tps_hb_stream_access(self.cs, self.params[l], self.pbytes, 1)
                L.tps_hb_stream_access(self.cs, self.grads[l], self.gbytes, 1)
        check(L.tps_stage_init(C.byref(c), C.byref(prm), C.byref(mem), C.byref(h)))
        self.h = h

    def write_inputs(self):
        """The caller writes x and dy on its stream (the stage's compute stream)."""
        L = lib()
        for mb in range(self.cfg.n_micro):
            L.tps_hb_stream_access(self.cs, self.x[mb], self.tbytes, 1)
            L.tps_hb_stream_access(self.cs, self.dy[mb], self.tbytes, 1)

    def begin(self):
        check(lib().tps_stage_begin_iteration(self.h, 1))

    def call(self, kind, mbs, as_group):
        L = lib()
        if as_group:
            n = len(mbs)
            if kind == "F":
                a = (C.c_void_p * n)(*[self.x[m] for m in mbs])
                b = (C.c_void_p * n)(*[self.y[m] for m in mbs])
                check(L.tps_stage_forward_group(self.h, mbs[0], n, a, b))
            else:
                a = (C.c_void_p * n)(*[self.dy[m] for m in mbs])
                b = (C.c_void_p * n)(*[self.dx[m] for m in mbs])
                check(L.tps_stage_backward_group(self.h, mbs[0], n, a, b))
        else:
            for mb in mbs:
                if kind == "F":
                    check(L.tps_stage_forward(self.h, mb, self.x[mb], self.y[mb]))
                else:
                    check(L.tps_stage_backward(self.h, mb, self.dy[mb], self.dx[mb]))

    def calls_for(self, group):
        if group:
            return [(k, list(range(mb0, mb0 + n)), True) for k, mb0, n in self.cfg.groups()]
        return [(k, [mb], False) for k, mb in self.cfg.order()]

    def iteration(self, group=False, calls=None):
        self.begin()
        for k, mbs, g in (calls if calls is not None else self.calls_for(group)):
            self.call(k, mbs, g)

    def read_results(self, sync=True):
        """The caller reads y, dx (and host gradient blocks) after a sync."""
        L = lib()
        if sync:
            check(L.tps_stage_sync(self.h))
        for mb in range(self.cfg.n_micro):
            L.tps_hb_host_access(self.y[mb], self.tbytes, 0)
            L.tps_hb_host_access(self.dx[mb], self.tbytes, 0)
        for l in range(self.cfg.n_layers):
            L.tps_hb_host_access(self.grads[l], self.gbytes, 0)

    def set_device_optimizer(self, tag: int = 0):
        """Every layer's AdamW on the device (tps_stage_set_optimizer_split
        with n_device = n_layers): fake device master, moment and parameter
        blocks, written by the caller on the compute stream beforehand."""
        L = lib()
        n = self.cfg.n_layers
        base = (tag + 1) * 64 * TiB + 9 * TiB
        blocks = {k: [base + i * TiB + l * 16 * GiB for l in range(n)] for i, k in enumerate(("m", "mo", "v", "p"))}
        for k, arr in blocks.items():
            for l, a in enumerate(arr):
                nb = self.pbytes if k == "p" else self.gbytes
                L.tps_hb_name_region(a, nb, f"opt-{k}[{tag}][{l}]".encode())
                L.tps_hb_stream_access(self.cs, a, nb, 1)
        self.opt_blocks = blocks
        arr = {k: (C.c_void_p * n)(*v) for k, v in blocks.items()}
        self._opt_keep = arr
        opt = T.AdamW(1e-3, 0.9, 0.95, 1e-8, 0.0)
        cast = lambda a: C.cast(a, C.POINTER(C.c_void_p))
        check(L.tps_stage_set_optimizer_split(C.c_void_p(self.h.value), C.byref(opt), cast(arr["m"]), cast(arr["mo"]),
                                              cast(arr["v"]), cast(arr["p"]), n, 1, 1))

    def close(self):
        if self.h:
            lib().tps_stage_destroy(self.h)
            self.h = None


def reset():
    lib().tps_hb_reset()


def races() -> int:
    return lib().tps_hb_races()


def report() -> str:
    return lib().tps_hb_report().decode()


def count_ops(name: str) -> int:
    """Operations recorded so far (since the library was loaded) with this name."""
    f = lib().tps_hb_count_ops
    f.restype = C.c_int64
    f.argtypes = [C.c_char_p]
    return f(name.encode())
