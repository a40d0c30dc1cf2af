#!/usr/bin/env python3
"""Stage throughput on one MI355X.

One step = one training iteration of the pipeline stage: F(mb) and B(mb) of
every micro-batch in the planned order (forward, the policy's recompute and
backward, with f32 gradient accumulation), all through the C ABI.  Inputs,
parameters and output gradients are resident in HBM before the timed region.

Prints one JSON line: stage TFLOP/s over the algorithmic flops the policy
requires, % of the dense bf16 MFMA peak, peak HBM, the dominant kernel's
roofline from HIP events around its launches inside the timed region, and the
CPU oracle timed on a bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import dataclasses
import json
import os
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "stage TFLOP/s (fwd+recompute+bwd, % bf16 MFMA peak); peak HBM GB"
PEAK_BF16_TFLOPS = 2500.0      # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0          # MI355X HBM3E


def log(*a):
    print(*a, file=sys.stderr, flush=True)


# Sources each kernel family is compiled from (device code and the headers it
# includes); counters recorded for a kernel stay valid while these are unchanged.
KERNEL_SOURCES = {
    "tps::gemm_bf16_kernel": ("gemm_pipe.h", "gemm_lds.h", "gemm_impl.h", "gemm_nt.hip", "gemm_nn.hip",
                              "gemm_tn.hip", "tps_device.h", "kernels.h"),
    "tps::attn": ("attention.hip", "attention_fwd.hip", "attention_bwd.hip", "attn_tiles.h", "tps_device.h",
                  "kernels.h"),
}


def kernel_source_hash(kernel: str) -> str:
    """sha256 over the sources `kernel` is built from (every library source
    for a kernel outside the known families)."""
    import hashlib
    csrc = os.path.join(ROOT, "paper_2503_03182_amd", "csrc")
    names = next((v for k, v in KERNEL_SOURCES.items() if kernel.startswith(k)), None)
    if names is None:
        names = [n for n in os.listdir(csrc) if n.endswith((".hip", ".h", ".cpp"))]
    h = hashlib.sha256()
    for name in sorted(names):
        h.update(name.encode())
        h.update(open(os.path.join(csrc, name), "rb").read())
    return h.hexdigest()


def measured_traffic(workload: str, kernel: str):
    """HBM bytes per launch of `kernel` from the counter runs recorded in
    profiles/, or None when they were taken on other kernel sources."""
    path = os.path.join(ROOT, "profiles", f"{workload}_dominant_traffic.txt")
    if not os.path.exists(path):
        return None
    rec = dict(line.rstrip("\n").split("\t", 1) for line in open(path) if "\t" in line)
    if rec.get("kernel") != kernel or rec.get("source_sha256") != kernel_source_hash(kernel):
        return None
    return float(rec["bytes_per_launch"])


def build_stage(cfg):
    import torch
    from paper_2503_03182_amd import synth
    from paper_2503_03182_amd import tpstage as T
    po, pb, go, gb = T.param_layout(cfg)
    td = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32
    es = 2 if cfg.dtype == "bf16" else 4
    blocks, grads = [], []
    llama = cfg.arch == T.ARCH_LLAMA
    nkv = cfg.n_kv_heads or cfg.n_heads
    shapes = (synth.llama_param_shapes(cfg.hidden, cfg.n_heads, nkv, cfg.mlp) if llama
              else synth.param_shapes(cfg.hidden, cfg.mlp))
    for l in range(cfg.n_layers):
        blk = torch.zeros(pb, dtype=torch.uint8, device="cuda")
        if cfg.weights == T.W_STREAM:
            # streamed weights live in pinned host memory (exact-size blocks);
            # the values come from a seeded device generator with the same
            # distributions as the synthetic parameters (throughput does not
            # depend on them, and it avoids drawing ~10^10 values on the CPU)
            gen = torch.Generator(device="cuda").manual_seed(1000 + 16 * l)
            for i, name in enumerate(T.PARAMS):
                if name not in shapes:
                    continue
                n = 1
                for d in shapes[name]:
                    n *= d
                v = torch.randn(n, generator=gen, device="cuda") * 0.02
                if name in ("g1", "g2"):
                    v += 1.0
                blk[po[i]:po[i] + n * es].view(td).copy_(v.to(td))
            hb = T.HostBuffer(pb)
            torch.cuda.synchronize()
            hb.numpy()[:] = blk.cpu().numpy()
            del blk
            blk = hb
            g = T.HostBuffer(gb)
            g.numpy()[:] = 0
        else:
            vals = (synth.llama_layer_params(l, cfg.hidden, cfg.n_heads, nkv, cfg.mlp, cfg.dtype) if llama
                    else synth.layer_params(l, cfg.hidden, cfg.mlp, cfg.dtype))
            for i, name in enumerate(T.PARAMS):
                if name not in vals:
                    continue
                v = torch.from_numpy(vals[name].reshape(-1)).to("cuda").to(td)
                blk[po[i]:po[i] + v.numel() * es].view(td).copy_(v)
            g = torch.zeros(gb, dtype=torch.uint8, device="cuda")
        blocks.append(blk)
        grads.append(g)
    xs, dys = [], []
    for mb in range(cfg.n_micro):
        xs.append(torch.from_numpy(synth.stage_input(mb, cfg.tokens, cfg.hidden, cfg.dtype)).to("cuda").to(td))
        dys.append(torch.from_numpy(synth.output_grad(mb, cfg.tokens, cfg.hidden, cfg.dtype)).to("cuda").to(td))
    ys = [torch.empty_like(x) for x in xs]
    dxs = [torch.empty_like(x) for x in xs]
    return blocks, grads, xs, dys, ys, dxs


def t_offload_state(cfg, blocks, n_device=0):
    """Model state of T-Offload: f32 master weights (from the streamed bf16
    parameter blocks), zero AdamW moments, all in the gradient layout; with
    the FP8 reload the host parameter blocks are rewritten in the quantized
    layout from the masters.  The first n_device layers keep their state on
    the GPU: device master, moments and a device copy of their bf16
    parameter block.  Returns (parameter blocks, (master, m, v), device
    parameter blocks)."""
    import numpy as np
    from paper_2503_03182_amd import tpstage as T
    from paper_2503_03182_amd import synth
    po, pb, go, gb = T.param_layout(cfg)
    shapes = (synth.llama_param_shapes(cfg.hidden, cfg.n_heads, cfg.n_kv_heads or cfg.n_heads, cfg.mlp)
              if cfg.arch == T.ARCH_LLAMA else synth.param_shapes(cfg.hidden, cfg.mlp))
    masters, ms, vs = [], [], []
    for blk in blocks:
        src = blk.numpy()
        mst = np.zeros(gb // 4, dtype=np.float32)
        for i, name in enumerate(T.PARAMS):
            if name not in shapes:
                continue
            n = int(np.prod(shapes[name]))
            bits = src[po[i]:po[i] + 2 * n].view(np.uint16)
            mst[go[i] // 4:go[i] // 4 + n] = (bits.astype(np.uint32) << 16).view(np.float32)
        masters.append(mst)
        ms.append(np.zeros_like(mst))
        vs.append(np.zeros_like(mst))
    import torch
    dparams = [torch.from_numpy(blocks[l].numpy()).cuda() for l in range(n_device)]
    if cfg.weights_quant == T.Q_FP8_ROW:
        qbytes = T.param_layout_q(cfg)[2]
        qblocks = []
        for mst in masters:
            hb = T.HostBuffer(qbytes)
            T.host_adamw_layer(cfg, 0, mst, None, None, None, hb, quant=T.Q_FP8_ROW,
                               n_threads=len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else 0)
            qblocks.append(hb)
        blocks = qblocks
    for l in range(n_device):
        masters[l], ms[l], vs[l] = (torch.from_numpy(a).cuda() for a in (masters[l], ms[l], vs[l]))
    return blocks, (masters, ms, vs), dparams


def host_link_rates(stream, gib: float = 1.0, reps: int = 3):
    """Copy-engine rates (GB/s) between pinned host memory and HBM, host to
    device and device to host, timed with events on `stream`."""
    import torch
    n = int(gib * (1 << 30))
    host = torch.empty(n, dtype=torch.uint8, pin_memory=True)
    dev = torch.empty(n, dtype=torch.uint8, device="cuda")
    rates = []
    for h2d in (True, False):
        with torch.cuda.stream(stream):
            (dev.copy_(host, non_blocking=True) if h2d else host.copy_(dev, non_blocking=True))
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            for _ in range(reps):
                (dev.copy_(host, non_blocking=True) if h2d else host.copy_(dev, non_blocking=True))
            e1.record(stream)
        e1.synchronize()
        rates.append(reps * n / (e0.elapsed_time(e1) * 1e-3) / 1e9)
    del host, dev
    return rates[0], rates[1]


def t_offload_stages(cfg, info, link, gpu_ms_per_step, h2d_gbs, d2h_gbs, n_device=0):
    """The appendix "Scalability of T-Offload" applied to this stage taken as
    one chunk: the smallest pipeline depths at which the measured host work
    would fit T-Pipe's bubbles (tpipe_t_offload_stages).  T_unit is the
    chunk's forward for one micro-batch, a third of its GPU time per
    micro-batch (backward = two forwards, as in the schedule's unit-time
    model); the chunk's offload time is the gradients of its host-updated
    layers over the measured device-to-host rate plus their measured host
    updates; its upload time is one load of their host parameter blocks over
    the host-to-device rate."""
    from paper_2503_03182_amd import tpstage as T
    t_unit = gpu_ms_per_step / (3 * cfg.n_micro)
    n_host = cfg.n_layers - n_device
    grad_gb = n_host * info["grad_bytes"] / 1e9
    blk = T.param_layout_q(cfg)[2] if cfg.weights_quant == T.Q_FP8_ROW else T.param_layout(cfg)[1]
    up_gb = n_host * blk / 1e9
    # the update thread lags the GPU: a step's window also sees updates of
    # the step before, so the chunk's time is the mean per layer times the layers
    t_off = grad_gb / d2h_gbs * 1e3 + n_host * link["host_update_ms"] / max(link["host_updates"], 1)
    t_up = up_gb / h2d_gbs * 1e3
    p_off, p_up = T.tpipe_t_offload_stages(t_off, t_up, t_unit)
    return {"t_unit_ms": round(t_unit, 2), "link_gbs": {"h2d": round(h2d_gbs, 1), "d2h": round(d2h_gbs, 1)},
            "chunk_offload_ms": round(t_off, 1), "chunk_upload_ms": round(t_up, 1),
            "min_stages_offload": p_off, "min_stages_upload": p_up}


def cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(cfg, budget_s):
    """The oracle as it stands, on one (layer, micro-batch) unit of the
    workload (forward, the policy's recompute, backward) at the workload's
    widths, repeated while the budget lasts.  Where one unit at the full
    sequence length would take far longer than the budget, the sample keeps
    the widths and shortens the sequence by powers of two; TFLOP/s is taken
    over the sample's own algorithmic flops (same formulas as the GPU
    number)."""
    import dataclasses

    import numpy as np
    from oracle import decoder_stage as ora
    from paper_2503_03182_amd import synth
    from paper_2503_03182_amd import tpstage as T
    try:
        from threadpoolctl import threadpool_info
        threads = max((p.get("num_threads", 1) for p in threadpool_info()), default=1)
    except Exception:  # pragma: no cover
        threads = os.cpu_count() or 1
    pol1 = None if cfg.policy is None else [cfg.policy[0]]
    unit_cfg = dataclasses.replace(cfg, n_layers=1, n_micro=1, policy=pol1, weights=T.W_RESIDENT,
                                   offload_auto=False, offload_mb_mask=0, ops=None, inflight=0)
    # a sample of at most ~4 TFLOP (~15 s at the 0.28 TFLOP/s measured on the machine's host)
    while unit_cfg.seq > 128:
        info = T.plan(unit_cfg)
        if info["fwd_flops"] + info["bwd_flops"] + info["recompute_flops"] <= 4e12:
            break
        unit_cfg = dataclasses.replace(unit_cfg, seq=unit_cfg.seq // 2)
    info = T.plan(unit_cfg)
    unit_flops = info["fwd_flops"] + info["bwd_flops"] + info["recompute_flops"]
    llama = cfg.arch == T.ARCH_LLAMA
    nkv = cfg.n_kv_heads or cfg.n_heads
    vals = (synth.llama_layer_params(0, cfg.hidden, cfg.n_heads, nkv, cfg.mlp, cfg.dtype) if llama
            else synth.layer_params(0, cfg.hidden, cfg.mlp, cfg.dtype))
    params = [{k: v.astype(np.float64) for k, v in vals.items()}]
    x = [synth.stage_input(0, unit_cfg.tokens, cfg.hidden, cfg.dtype).astype(np.float64)]
    dy = [synth.output_grad(0, unit_cfg.tokens, cfg.hidden, cfg.dtype).astype(np.float64)]
    policy = None if pol1 is None else [{k: (v if v != T.OFFLOAD else T.KEEP) for k, v in pol1[0].items()}]
    times = []
    t_end = time.perf_counter() + budget_s
    while len(times) < 3 and (not times or time.perf_counter() < t_end):
        t0 = time.perf_counter()
        if llama:
            from oracle import llama_stage
            llama_stage.run_stage(params, x, dy, cfg.n_heads, nkv, unit_cfg.micro_batch, unit_cfg.seq, cfg.ln_eps,
                                  cfg.rope_base, policy=policy)
        else:
            ora.run_stage(params, x, dy, cfg.n_heads, unit_cfg.micro_batch, unit_cfg.seq, cfg.ln_eps, policy=policy)
        times.append(time.perf_counter() - t0)
    med = statistics.median(times)
    ncpu = len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else (os.cpu_count() or 1)
    return {"value": round(unit_flops / med / 1e12, 6), "unit": "TFLOP/s", "cores": int(threads),
            "kind": "oracle", "nproc": ncpu, "cpu_model": cpu_model(),
            "sample": f"one layer x one micro-batch at the workload's widths and policy, seq "
                      f"{unit_cfg.seq} (workload {cfg.seq}), {unit_flops / 1e12:.3f} TFLOP of forward, "
                      f"recompute and backward, in float64 numpy on {int(threads)} BLAS threads; median of "
                      f"{len(times)} run(s), {med:.2f} s each; TFLOP/s over the sample's own algorithmic flops"}


def standalone_gemms(cfg, reps: int = 10) -> list:
    """Every GEMM of one (layer, micro-batch) unit of the workload launched
    alone through the op-level C ABI (same kernels, layouts, epilogues and
    tile choices as in the stage), each timed with HIP events over `reps`
    launches on an otherwise idle GPU: the kernels' stand-alone rates beside
    their in-stage rates."""
    import torch
    from paper_2503_03182_amd import tpstage as T
    Tk, h, f = cfg.tokens, cfg.hidden, cfg.mlp
    nn = lambda K: K >= 12288   # the stage's layout choice for long contractions
    td = torch.bfloat16
    dev = "cuda"

    def t(r, c):
        return (torch.randn(r, c, device=dev) * 0.05).to(td)

    shapes = [
        ("QKV forward", T.GEMM_NT, T.EPI_BIAS, Tk, 3 * h, h),
        ("out-proj forward", T.GEMM_NT, T.EPI_BIAS_RESID, Tk, h, h),
        ("FC1 forward (GeLU)", T.GEMM_NT, T.EPI_BIAS_GELU, Tk, f, h),
        ("FC2 forward", T.GEMM_NN if (nn(f) and cfg.weights == T.W_RESIDENT) else T.GEMM_NT, T.EPI_BIAS_RESID,
         Tk, h, f),
        ("dgelu input grad (FC2)", T.GEMM_NN if nn(h) else T.GEMM_NT, T.EPI_GELU_GRAD, Tk, f, h),
        ("FC1 input grad", T.GEMM_NN if nn(f) else T.GEMM_NT, T.EPI_STORE, Tk, h, f),
        ("out-proj input grad", T.GEMM_NN if nn(h) else T.GEMM_NT, T.EPI_STORE, Tk, h, h),
        ("QKV input grad", T.GEMM_NN if nn(3 * h) else T.GEMM_NT, T.EPI_STORE, Tk, h, 3 * h),
        ("W2 weight grad", T.GEMM_TN, T.EPI_ACC_F32, h, f, Tk),
        ("W1 weight grad", T.GEMM_TN, T.EPI_ACC_F32, f, h, Tk),
        ("Wo weight grad", T.GEMM_TN, T.EPI_ACC_F32, h, h, Tk),
        ("Wqkv weight grad", T.GEMM_TN, T.EPI_ACC_F32, 3 * h, h, Tk),
    ]
    out = []
    for name, layout, epi, M, N, K in shapes:
        a = t(K, M) if layout == T.GEMM_TN else t(M, K)
        b = t(N, K) if layout == T.GEMM_NT else t(K, N)
        lda = M if layout == T.GEMM_TN else K
        ldb = K if layout == T.GEMM_NT else N
        c = torch.zeros(M, N, device=dev, dtype=torch.float32 if epi == T.EPI_ACC_F32 else td)
        bias = t(1, N).reshape(-1) if epi in (T.EPI_BIAS, T.EPI_BIAS_RESID, T.EPI_BIAS_GELU) else None
        resid = t(M, N) if epi == T.EPI_BIAS_RESID else None
        aux = t(M, N) if epi in (T.EPI_BIAS_GELU, T.EPI_GELU_GRAD) else None
        s = torch.cuda.current_stream()

        def launch():
            T.op_gemm(T.TPS_BF16, layout, epi, M, N, K, a, lda, b, ldb, c, N, bias=bias, resid=resid,
                      ldr=N if resid is not None else 0, aux=aux, ldaux=N if aux is not None else 0, stream=s)
        launch()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(s)
        for _ in range(reps):
            launch()
        e1.record(s)
        torch.cuda.synchronize()
        us = e0.elapsed_time(e1) * 1e3 / reps
        fl = 2.0 * M * N * K
        out.append({"gemm": name, "layout": ["NT", "NN", "TN"][layout], "M": M, "N": N, "K": K,
                    "us": round(us, 1), "tflops": round(fl / (us * 1e-6) / 1e12, 1),
                    "frac_bf16_peak": round(fl / (us * 1e-6) / 1e12 / PEAK_BF16_TFLOPS, 4)})
        del a, b, c, bias, resid, aux
    return out


def main():
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=None, help="timed steps (default: 5 for the hidden-8192 "
                    "streamed workload, 20 otherwise)")
    ap.add_argument("--warmup", type=int, default=None, help="untimed steps (default: 2, resp. 3)")
    ap.add_argument("--workload", default="stage12_h8192_stream")
    ap.add_argument("--cpu-seconds", type=float, default=20.0, help="budget of the oracle sample")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="run only a plain 512 MiB device-to-device copy (reference for HBM byte counters)")
    ap.add_argument("--standalone-gemms", action="store_true",
                    help="time every GEMM of one (layer, micro-batch) unit of the workload alone and exit")
    ap.add_argument("--t-offload", choices=("bf16", "fp8"), default=None,
                    help="streamed workloads: attach the host AdamW update of every layer (T-Offload of model "
                         "state) and reload the updated weights as bf16 or as FP8 codes with row scales")
    ap.add_argument("--device-layers", type=int, default=None,
                    help="with --t-offload: the shallowest layers whose model state and AdamW step stay on the GPU "
                         "(default: 2, at most the layer count)")
    ap.add_argument("--layers", type=int, default=None, help="override the workload's layer count")
    ap.add_argument("--wgrad", choices=("auto", "side", "inline"), default="auto",
                    help="where the parameter-gradient kernels run: the plan's choice (auto), a stream "
                         "of their own beside the input-gradient chain (side) or the compute stream (inline)")
    args = ap.parse_args()
    if args.standalone_gemms:
        import torch
        from paper_2503_03182_amd import configs
        cfg = configs.WORKLOADS[args.workload]()
        print(json.dumps({"workload": args.workload, "standalone_gemms": standalone_gemms(cfg)}), flush=True)
        return
    if args.copy_calibration:
        import torch
        n = 512 << 20
        src = torch.ones(n, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes_read": n, "copy_bytes_written": n, "launches": 3}))
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU's share of the stage; --gpus {args.gpus} is not supported "
              f"(the library runs one GPU per process and has no multi-GPU path)", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2503_03182_amd import configs
    from paper_2503_03182_amd import tpstage as T

    cfg = configs.WORKLOADS[args.workload]()
    if args.layers is not None:
        cfg = dataclasses.replace(cfg, n_layers=args.layers,
                                  policy=None if cfg.policy is None else cfg.policy[:args.layers])
    if args.wgrad != "auto":
        cfg = dataclasses.replace(cfg, wgrad_stream=T.WGRAD_SIDE if args.wgrad == "side" else T.WGRAD_INLINE)
    if args.t_offload is not None:
        if cfg.weights != T.W_STREAM:
            print("--t-offload needs a workload with streamed weights", file=sys.stderr)
            sys.exit(2)
        if args.t_offload == "fp8":
            cfg = dataclasses.replace(cfg, weights_quant=T.Q_FP8_ROW)
        if args.device_layers is None:
            args.device_layers = min(2, cfg.n_layers)
        if not 0 <= args.device_layers <= cfg.n_layers:
            print("--device-layers must be in 0..layers", file=sys.stderr)
            sys.exit(2)
    long_step = cfg.hidden >= 8192
    if args.steps is None:
        args.steps = 5 if long_step else 20
    if args.warmup is None:
        args.warmup = 2 if long_step else 3
    info = T.plan(cfg)
    # the whole run on a stream of its own: the stage computes on it, and
    # nothing synchronizes implicitly with the library's copy streams
    run_stream = torch.cuda.Stream()
    torch.cuda.set_stream(run_stream)
    free0, total = torch.cuda.mem_get_info()
    torch.cuda.reset_peak_memory_stats()
    log(f"[bench] workload {args.workload}: building parameters and inputs")
    blocks, grads, xs, dys, ys, dxs = build_stage(cfg)
    torch.cuda.synchronize()
    opt_state = None
    dparams = []
    if args.t_offload is not None:
        blocks, opt_state, dparams = t_offload_state(cfg, blocks, args.device_layers)
    stage = T.Stage(cfg, blocks, grads)
    link_rates = None
    if opt_state is not None:
        link_rates = host_link_rates(run_stream)
        log(f"[bench] host link {link_rates[0]:.1f} GB/s to the device, {link_rates[1]:.1f} GB/s back")
        n_threads = len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else (os.cpu_count() or 1)
        stage.set_optimizer(*opt_state, first_step=1, lr=1e-5, n_threads=n_threads, dparams=dparams)
        log(f"[bench] AdamW of layers 0..{args.device_layers - 1} on the GPU, of the others on {n_threads} host "
            f"threads, reload as {args.t_offload}")
    assert stage.cs.cuda_stream == run_stream.cuda_stream
    order = cfg.order()
    step_flops = info["fwd_flops"] + info["bwd_flops"] + info["recompute_flops"]

    groups = cfg.groups()

    def step():
        stage.begin_iteration(zero_grads=True)
        if cfg.layer_major:
            for k, mb0, n in groups:
                if k == "F":
                    stage.forward_group(mb0, xs[mb0:mb0 + n], ys[mb0:mb0 + n])
                else:
                    stage.backward_group(mb0, dys[mb0:mb0 + n], dxs[mb0:mb0 + n])
            return
        for k, mb in order:
            if k == "F":
                stage.forward(mb, xs[mb], ys[mb])
            else:
                stage.backward(mb, dys[mb], dxs[mb])

    for _ in range(args.warmup):
        step()
    stage.sync()
    torch.cuda.synchronize()
    log("[bench] warmup done")

    # one instrumented step: per-kernel breakdown, picks the dominant kernel
    stage.time_kernels("")
    step()
    stage.sync()
    breakdown = sorted(stage.kernel_times(), key=lambda r: -r["ms"])
    singles = [r for r in breakdown if r["name"].startswith("tps::")]
    dominant = singles[0]["name"]
    log(f"[bench] dominant kernel {dominant}")

    # timed region: only the dominant kernel is bracketed with events
    stage.time_kernels(dominant)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    stage.sync()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    link = stage.stats()   # bytes the last timed iteration moved over the host link
    dom = [r for r in stage.kernel_times() if r["name"] == dominant][0]
    stage.time_kernels(None)
    free1, _ = torch.cuda.mem_get_info()
    log(f"[bench] timed {args.steps} steps in {t1 - t0:.3f} s")

    ms_per_step = (t1 - t0) * 1e3 / args.steps
    value = step_flops * args.steps / (t1 - t0) / 1e12
    t_offload = None
    if opt_state is not None:
        t_offload = {"reload": args.t_offload, "optimizer": "AdamW (f32 master weights)",
                     "device_layers": args.device_layers,
                     "host_update_ms_per_layer": round(link["host_update_ms"] / max(link["host_updates"], 1), 1),
                     "host_updates_finished_during_last_step": link["host_updates"],
                     "reload_wait_ms_last_step": round(link["host_wait_ms"], 1),
                     "host_state_gb": round(3 * (cfg.n_layers - args.device_layers) * info["grad_bytes"] / 1e9, 2),
                     "device_state_gb": round(args.device_layers * (3 * info["grad_bytes"] + info["param_bytes"]) / 1e9,
                                              2),
                     "tpipe_bubbles": t_offload_stages(cfg, info, link, sum(r["ms"] for r in breakdown),
                                                       *link_rates, n_device=args.device_layers)}
    achieved = dom["flops"] / (dom["ms"] * 1e-3) / 1e12
    step_ms_breakdown = sum(r["ms"] for r in breakdown)
    out = {
        "metric": METRIC,
        "value": round(value, 3),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": cfg.dtype,
        "data": "synthetic: seeded N(0,0.02) weights, N(0,1) stage inputs and output gradients",
        "config": {
            "workload": args.workload,
            "layer": "LLAMA-style (RMSNorm, rotary, grouped-query attention, SwiGLU)" if cfg.arch == T.ARCH_LLAMA
                     else "GPT pre-LN (LayerNorm, biases, GeLU)",
            "layers": cfg.n_layers, "hidden": cfg.hidden, "heads": cfg.n_heads,
            "kv_heads": cfg.n_kv_heads or cfg.n_heads, "mlp": cfg.mlp,
            "seq": cfg.seq, "micro_batch": cfg.micro_batch, "micro_batches": cfg.n_micro,
            "policy": configs.WORKLOADS[args.workload].__doc__.split(";")[-1].strip().rstrip("."),
            "order": ("layer-major: one forward group and one backward group over all micro-batches"
                      if cfg.layer_major else "all forwards, then all backwards (in-flight = micro-batches)"),
            "parameter_gradients": ("inline on the compute stream" if info["wgrad_inline"]
                                    else "on a stream of their own beside the input-gradient chain"),
            "parallelism": "one GPU",
        },
        "pct_bf16_peak": round(100.0 * value / PEAK_BF16_TFLOPS, 2),
        "flops_per_step": step_flops,
        "mfu_pct": round(100.0 * 3 * info["fwd_flops"] * args.steps / (t1 - t0) / 1e12 / PEAK_BF16_TFLOPS, 2),
        "peak_hbm_gb": {
            "planned": round(info["predicted_peak_bytes"] / 1e9, 3),
            "torch_max_allocated": round(torch.cuda.max_memory_allocated() / 1e9, 3),
            "device_used_delta": round((free0 - min(free0, free1)) / 1e9, 3),
            "keep_all_activations": round(info["keep_all_bytes"] / 1e9, 3),
        },
        "roofline": {
            "bound": "mfma",
            "kernel": dominant,
            "achieved": round(achieved, 2),
            "peak": PEAK_BF16_TFLOPS,
            "unit": "TFLOP/s",
            "frac": round(achieved / PEAK_BF16_TFLOPS, 4),
            "traffic": measured_traffic(args.workload, dominant),
            "launches": dom["launches"],
            "avg_launch_us": round(dom["ms"] * 1e3 / max(dom["launches"], 1), 2),
        },
        "t_offload": t_offload,
        "host_link": {
            "h2d_gb_per_step": round(link["h2d_bytes"] / 1e9, 3),
            "d2h_gb_per_step": round(link["d2h_bytes"] / 1e9, 3),
            "h2d_gbs_over_step": round(link["h2d_bytes"] / (ms_per_step * 1e-3) / 1e9, 2),
            "d2h_gbs_over_step": round(link["d2h_bytes"] / (ms_per_step * 1e-3) / 1e9, 2),
        },
        "kernels_per_step": [
            {"name": r["name"], "launches": r["launches"], "ms": round(r["ms"], 3),
             "tflops": round(r["flops"] / (r["ms"] * 1e-3) / 1e12, 1) if r["flops"] else None,
             "gbs": round(r["bytes"] / (r["ms"] * 1e-3) / 1e9, 1) if not r["flops"] else None}
            for r in breakdown[:12]
        ],
        "instrumented_step_ms": round(step_ms_breakdown, 3),
    }
    stage.close()
    if not args.no_cpu_baseline:
        log("[bench] timing the CPU oracle sample")
        out["cpu_baseline"] = cpu_baseline(cfg, args.cpu_seconds)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
