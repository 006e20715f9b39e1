"""GPU parity of the quadratic (flash-style) form, kata_fwd_quadratic_ws,
against the CPU oracle's O(T^2) definition.  Every case prints its name and
shape before it launches anything."""
from __future__ import annotations

import numpy as np
import pytest

import workloads
from gpu_helpers import assert_bf16_close, log, sample_rows, to_device

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def kata():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2607_17419_amd as k
    k.lib()  # raises if libkata.so is missing: no fallback
    return k


def _run(kata, inp, alloc=False):
    import torch
    q = to_device(inp["q_dev"], "bf16")
    k = to_device(inp["k_dev"], "bf16")
    v = to_device(inp["v_dev"], "bf16")
    out = kata.fwd_quadratic_alloc(q, k, v) if alloc else kata.fwd_quadratic(q, k, v)
    torch.cuda.synchronize()
    return out.cpu().numpy()


@pytest.mark.parametrize("T", [1, 2, 31, 33, 255, 256, 257, 1000, 1025])
def test_quadratic_ragged(kata, orc, T):
    log(f"case quadratic ragged T={T} B1 H2 d64")
    inp = workloads.make_inputs("mid_bf16", B=1, H=2, T=T)
    got = _run(kata, inp)
    ref = orc.fwd(inp["q"], inp["k"], inp["v"])
    assert_bf16_close(got, ref, f"quadratic T {T}")


def test_quadratic_d32_recall(kata, orc):
    log("case quadratic recall d32 B2 H2 T3000")
    inp = workloads.make_inputs("recall_bf16", B=2, H=2, T=3000)
    got = _run(kata, inp, alloc=True)
    ref = orc.fwd(inp["q"], inp["k"], inp["v"])
    assert_bf16_close(got, ref, "quadratic recall d32")


def test_quadratic_zero_query_rows(kata, orc):
    log("case quadratic zero query rows (D_t = 0 -> 0)")
    inp = workloads.make_inputs("mid_bf16", B=1, H=1, T=700)
    for key in ("q_dev", "q"):
        inp[key] = inp[key].copy()
        inp[key][0, 0, [0, 5, 64, 640]] = 0
    got = _run(kata, inp)
    assert np.all(got[0, 0, [0, 5, 64, 640]] == 0.0)
    ref = orc.fwd(inp["q"], inp["k"], inp["v"])
    assert_bf16_close(got, ref, "quadratic zero rows")


def test_quadratic_matches_chunked(kata):
    import torch
    log("case quadratic vs chunked B2 H4 T4096 d64")
    inp = workloads.make_inputs("mid_bf16", B=2, H=4, T=4096)
    q = to_device(inp["q_dev"], "bf16")
    k = to_device(inp["k_dev"], "bf16")
    v = to_device(inp["v_dev"], "bf16")
    a = kata.fwd_quadratic(q, k, v)
    b = kata.fwd_chunked(q, k, v, 64)
    torch.cuda.synchronize()
    a, b = a.cpu().numpy(), b.cpu().numpy()
    rel = np.linalg.norm(a - b, axis=-1) / np.linalg.norm(b, axis=-1)
    log(f"  quadratic vs chunked: max row rel diff {rel.max():.3e}")
    assert rel.max() <= 2e-2


def test_quadratic_long_sampled(kata, orc):
    T = 32768
    log(f"case quadratic sampled B1 H4 T{T} d64")
    inp = workloads.make_inputs("long_bf16", B=1, H=4, T=T)
    got = _run(kata, inp)
    assert np.all(np.isfinite(got))
    bh, tt = sample_rows(1, 4, T, 7, n_random=256, head_rows=128, tail_rows=4)
    ref = orc.fwd_rows(inp["q"], inp["k"], inp["v"], bh, tt)
    assert_bf16_close(got.reshape(4, T, 64)[bh, tt], ref, "quadratic T32768 sampled")
