"""The allocation-free attention backward (tps_op_attention_bwd_noalloc)
against the workspace version (tps_op_attention_bwd), through the C ABI:
bitwise equal results on two calls in a row (the second smaller, so the
fixed workspace keeps stale rows from the first), in both storage dtypes
and head dims; sizes beyond the fixed workspace are rejected before any
launch; and the call allocates no device memory."""
import ctypes as C

import numpy as np
import pytest

from paper_2503_03182_amd import synth
from paper_2503_03182_amd import tpstage as T

pytestmark = pytest.mark.gpu


def _inputs(seed, b, s, nh, d, dtype):
    import torch
    td = torch.bfloat16 if dtype == T.TPS_BF16 else torch.float32
    sd = "bf16" if dtype == T.TPS_BF16 else "f32"
    h = nh * d
    qkv = torch.from_numpy(synth.uniform_tensor(seed, (b * s, 3 * h), 1.0, sd)).cuda().to(td)
    do = torch.from_numpy(synth.uniform_tensor(seed + 1, (b * s, h), 1.0, sd)).cuda().to(td)
    o = torch.empty((b * s, h), device="cuda", dtype=td)
    lse = torch.empty((b, nh, s), device="cuda", dtype=torch.float32)
    T.op_attention_fwd(dtype, b, s, nh, d, qkv, o, lse)
    return qkv, o, lse, do


@pytest.mark.parametrize("dtype,d", [(T.TPS_BF16, 128), (T.TPS_BF16, 64), (T.TPS_F32, 64)])
def test_noalloc_matches_workspace_version_two_calls(dtype, d):
    import torch
    shapes = [(2, 1000, 8), (1, 333, 3)]          # second call smaller
    for i, (b, s, nh) in enumerate(shapes):
        print("noalloc attention backward", dtype, d, (b, s, nh), flush=True)
        qkv, o, lse, do = _inputs(100 + 7 * i, b, s, nh, d, dtype)
        ws = torch.empty(T.op_workspace_bytes(T.WS_ATTN_BWD, b * s, nh) // 4, device="cuda")
        ref = torch.full_like(qkv, float("nan"))
        T.op_attention_bwd(dtype, b, s, nh, d, qkv, o, lse, do, ref, ws)
        got = torch.full_like(qkv, float("nan"))
        stream = torch.cuda.Stream()
        stream.wait_stream(torch.cuda.current_stream())
        T.op_attention_bwd_noalloc(dtype, b, s, nh, d, qkv, o, lse, do, got, stream=stream)
        torch.cuda.current_stream().wait_stream(stream)
        torch.cuda.synchronize()
        assert not torch.isnan(got.float()).any()
        assert torch.equal(got, ref), (dtype, d, (b, s, nh))


def test_noalloc_rejects_oversize_and_allocates_nothing():
    import torch
    max_rows = T.lib().tps_op_attention_bwd_noalloc_max_rows()
    assert max_rows == 1 << 20
    b, s, nh, d = 1, 512, 4, 128
    qkv, o, lse, do = _inputs(5, b, s, nh, d, T.TPS_BF16)
    out = torch.empty_like(qkv)
    # first call on the device: looks up the fixed array (and the runtime
    # loads the kernels); the calls after it are the ones measured
    T.op_attention_bwd_noalloc(T.TPS_BF16, b, s, nh, d, qkv, o, lse, do, out)
    torch.cuda.synchronize()
    free0 = torch.cuda.mem_get_info()[0]
    # too many rows for the fixed workspace: refused before any launch
    rc = T.lib().tps_op_attention_bwd_noalloc(T.TPS_BF16, 1, max_rows // 16 + 1, 16, d, qkv.data_ptr(),
                                              o.data_ptr(), lse.data_ptr(), do.data_ptr(), out.data_ptr(), None)
    assert rc == T.TPS_EINVAL
    assert b"exceeds the fixed workspace" in T.lib().tps_last_error()
    for _ in range(3):
        T.op_attention_bwd_noalloc(T.TPS_BF16, b, s, nh, d, qkv, o, lse, do, out)
    torch.cuda.synchronize()
    assert torch.cuda.mem_get_info()[0] == free0
