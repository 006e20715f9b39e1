"""kata_fwd_chunked_noalloc (workspace in the library's per-device scratch
array, no allocation) against kata_fwd_chunked (stream-ordered workspace),
through the C ABI: the same kernels at the same span, so the outputs agree
bit for bit.  Two calls in a row, the second with a smaller input, so the
second call runs on what the first left in the array.  Every case prints its
name and shape before it launches."""
from __future__ import annotations

import numpy as np
import pytest

import workloads
from gpu_helpers import assert_bf16_close, assert_f32_close, log, to_device

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def kata():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2607_17419_amd as k
    k.lib()  # raises if libkata.so is missing: no fallback
    return k


def _dev3(inp, dtype):
    return tuple(to_device(inp[n], dtype) for n in ("q_dev", "k_dev", "v_dev"))


def test_noalloc_matches_allocating_entry_point(kata, orc):
    import torch
    cases = [("mid_bf16", dict(B=2, H=3, T=5000), "bf16", 64),
             ("mid_bf16", dict(B=1, H=2, T=777), "bf16", 64)]
    for name, shape, dtype, C in cases:
        log(f"case noalloc vs kata_fwd_chunked {name} {shape} C{C}")
        inp = workloads.make_inputs(name, **shape)
        q, k, v = _dev3(inp, dtype)
        a = kata.fwd_chunked_noalloc(q, k, v, C)
        b = kata.fwd_chunked_alloc(q, k, v, C)
        torch.cuda.synchronize()
        assert torch.equal(a, b), f"{name} {shape}"
        ref = orc.fwd(inp["q"], inp["k"], inp["v"])
        assert_bf16_close(a.cpu().numpy(), ref, f"noalloc {shape}")


def test_noalloc_fp32_path_twice(kata, orc):
    import torch
    for T in (300, 65):
        log(f"case noalloc fp32 path tiny_f32 B1 H2 T{T} d16 C32")
        inp = workloads.make_inputs("tiny_f32", T=T)
        q, k, v = _dev3(inp, "f32")
        a = kata.fwd_chunked_noalloc(q, k, v, 32)
        b = kata.fwd_chunked_alloc(q, k, v, 32)
        torch.cuda.synchronize()
        assert torch.equal(a, b)
        assert_f32_close(a.cpu().numpy(), orc.fwd(inp["q"], inp["k"], inp["v"]), f"T{T}")


def test_noalloc_rejects_beyond_scratch(kata):
    import torch
    # the long workload's workspace (about 0.84 GB) exceeds the 256 MiB array;
    # the call is rejected on the host before any launch
    log("case noalloc rejects B1 H16 T131072 d64 (workspace above the scratch size)")
    need = kata.workspace_bytes(1, 16, 131072, 64, 64, 64, kata.KATA_BF16)
    assert need > kata.noalloc_scratch_bytes()
    x = torch.zeros((1, 16, 131072, 64), dtype=torch.bfloat16, device="cuda:0")
    with pytest.raises(kata.KataError) as ei:
        kata.fwd_chunked_noalloc(x, x, x, 64)
    assert ei.value.status == kata.KATA_ERR_UNSUPPORTED
    # a fitting call right after still works
    inp = workloads.make_inputs("mid_bf16", B=1, H=1, T=100)
    q, k, v = _dev3(inp, "bf16")
    a = kata.fwd_chunked_noalloc(q, k, v, 64)
    b = kata.fwd_chunked_alloc(q, k, v, 64)
    torch.cuda.synchronize()
    assert torch.equal(a, b)
