"""The stage workloads (shapes and policies) used by tests and the bench.

Every workload is one pipeline stage of decoder layers (GPT pre-LN, or
LLAMA-style for the llama* workloads) run micro-batch by micro-batch; names
say what the workload is.
"""
from __future__ import annotations

from .tpstage import (ARCH_LLAMA, GRAN_LAYER, GRAN_SEGMENT, KEEP, OFFLOAD, RECOMPUTE, TENSORS, W_RESIDENT,
                      W_STREAM, StageConfig)


def policy_all(L: int, mode: int, keep_inputs: bool = False) -> list:
    pol = [{t: mode for t in TENSORS} for _ in range(L)]
    if keep_inputs or mode == RECOMPUTE:
        for l in range(L):
            if keep_inputs or l == 0:
                pol[l]["x"] = KEEP
    return pol


def policy_selective(L: int) -> list:
    """Operator-level recompute: attention output and GeLU output dropped."""
    return [{t: (RECOMPUTE if t in ("o", "g") else KEEP) for t in TENSORS} for _ in range(L)]


def policy_layer_inputs(L: int) -> list:
    """Full-layer recompute: only each layer's input stays resident."""
    return [{t: (KEEP if t == "x" else RECOMPUTE) for t in TENSORS} for _ in range(L)]


def tiny(policy: str = "keep") -> StageConfig:
    """2 layers, hidden 256, 4 heads, MLP 1024, causal seq 128, micro-batch 2,
    4 micro-batches, f32.  policy: keep | recompute | offload."""
    L, M = 2, 4
    cfg = StageConfig(n_layers=L, hidden=256, n_heads=4, mlp=1024, seq=128, micro_batch=2, n_micro=M,
                      dtype="f32")
    if policy == "recompute":
        cfg.policy = policy_all(L, RECOMPUTE)
    elif policy == "offload":
        cfg.policy = policy_all(L, OFFLOAD)
        cfg.offload_mb_mask = (1 << M) - 1
    return cfg


def stage4_h2048() -> StageConfig:
    """4 layers, hidden 2048, 16 heads, MLP 8192, causal seq 2048, micro-batch 1,
    8 micro-batches, bf16; selective recompute of attention and GeLU outputs."""
    return StageConfig(n_layers=4, hidden=2048, n_heads=16, mlp=8192, seq=2048, micro_batch=1, n_micro=8,
                       dtype="bf16", policy=policy_selective(4), granularity=GRAN_SEGMENT)


def stage5_h5120_offload() -> StageConfig:
    """5 layers, hidden 5120, 40 heads, MLP 20480, causal seq 2048, micro-batch 1,
    16 micro-batches in flight, bf16; every activation offloadable: the planner
    offloads the micro-batches (by slack) whose copies over the host link (55
    GB/s, measured per direction on MI355X) lower the device peak without
    lengthening the round, and prefetches each three ops before its backward
    (late enough that it returns after the peak has passed)."""
    return StageConfig(n_layers=5, hidden=5120, n_heads=40, mlp=20480, seq=2048, micro_batch=1, n_micro=16,
                       dtype="bf16", policy=policy_all(5, OFFLOAD), offload_auto=True, lookahead=3,
                       link_gbps_hint=55.0, tflops_hint=1000.0)


def stage5_h5120_resident() -> StageConfig:
    """The activation-offload workload's shapes with every activation kept in
    HBM (no offload): the reference point for how much of the offload the
    copy engines hide."""
    return StageConfig(n_layers=5, hidden=5120, n_heads=40, mlp=20480, seq=2048, micro_batch=1, n_micro=16,
                       dtype="bf16", policy=policy_all(5, KEEP))


def stage4_seq8192_recompute() -> StageConfig:
    """4 layers, hidden 4096, 32 heads, MLP 16384, causal seq 8192, micro-batch 1,
    8 micro-batches, bf16; full-layer recompute keeping only layer inputs."""
    return StageConfig(n_layers=4, hidden=4096, n_heads=32, mlp=16384, seq=8192, micro_batch=1, n_micro=8,
                       dtype="bf16", policy=policy_layer_inputs(4), granularity=GRAN_SEGMENT)


def stage12_h8192_stream(n_micro: int = 8) -> StageConfig:
    """12 layers, hidden 8192, 64 heads, MLP 32768, causal seq 4096, micro-batch 1,
    8 micro-batches, bf16 weights and f32 grads streamed from pinned host per
    layer, run as layer-major groups (each streamed layer serves every
    micro-batch before the next one comes in, and its weight gradients are
    one product per layer over the group); activations recomputed from
    layer inputs."""
    return StageConfig(n_layers=12, hidden=8192, n_heads=64, mlp=32768, seq=4096, micro_batch=1,
                       n_micro=n_micro, dtype="bf16", policy=policy_layer_inputs(12), granularity=GRAN_LAYER,
                       weights=W_STREAM, window=3, layer_major=True, group_wgrad=1)


def stage12_h8192_stream_m20() -> StageConfig:
    """The hidden-8192 streamed workload with 20 micro-batches in flight
    (same layers, shapes and policy): every tensor kept would need more than
    the 288 GB of one MI355X (activations of 20 x 12 layer-micro-batch units
    plus bf16 weights and f32 gradients), while layer-input recompute and
    streamed weights and gradients keep the stage's peak a small fraction of
    it."""
    return stage12_h8192_stream(n_micro=20)


def llama12_h8192_stream() -> StageConfig:
    """12 LLAMA-style layers at the LLAMA2-70B widths: hidden 8192, 64 query
    heads and 8 key/value heads of 128, SwiGLU MLP 28672 (gate and up
    packed), causal seq 4096, micro-batch 1, 8 micro-batches, bf16; weights
    and f32 grads streamed from pinned host per layer, run as layer-major
    groups; activations recomputed from layer inputs."""
    return StageConfig(n_layers=12, hidden=8192, n_heads=64, mlp=28672, seq=4096, micro_batch=1, n_micro=8,
                       dtype="bf16", policy=policy_layer_inputs(12), granularity=GRAN_LAYER, weights=W_STREAM,
                       window=3, layer_major=True, arch=ARCH_LLAMA, n_kv_heads=8, group_wgrad=1)


def llama4_h4096() -> StageConfig:
    """4 LLAMA-style layers, hidden 4096, 32 query heads and 8 key/value heads
    of 128, SwiGLU MLP 14336, causal seq 4096, micro-batch 1, 8
    micro-batches, bf16, resident weights; selective recompute of the
    attention and SwiGLU outputs."""
    return StageConfig(n_layers=4, hidden=4096, n_heads=32, mlp=14336, seq=4096, micro_batch=1, n_micro=8,
                       dtype="bf16", policy=policy_selective(4), granularity=GRAN_SEGMENT, arch=ARCH_LLAMA,
                       n_kv_heads=8)


WORKLOADS = {
    "tiny": tiny,
    "stage4_h2048": stage4_h2048,
    "stage5_h5120_offload": stage5_h5120_offload,
    "stage5_h5120_resident": stage5_h5120_resident,
    "stage4_seq8192_recompute": stage4_seq8192_recompute,
    "stage12_h8192_stream": stage12_h8192_stream,
    "stage12_h8192_stream_m20": stage12_h8192_stream_m20,
    "llama4_h4096": llama4_h4096,
    "llama12_h8192_stream": llama12_h8192_stream,
}
