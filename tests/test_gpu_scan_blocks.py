"""GPU parity of the record scans at every record-block shape.

The bf16 span-record scan splits a head's records into blocks of 1, 2, 4 or 8
row groups of 16 records (chosen by the record count), keeps a block in
registers and carries an fp32 running sum from one block to the next; the
fp32 path's chunk-record scan does the same with 128-record blocks.  The
row-group cases sit on both sides of each row-group boundary; every other
case gives a head more than 128 records, so the carry runs (section
"Tree-scan inter-chunk reduction": the associative scan over chunk states).
Each compares the output with the CPU oracle's definition and prints its
name and shape before it launches anything.
"""
from __future__ import annotations

import numpy as np
import pytest

import workloads
from gpu_helpers import assert_bf16_close, assert_f32_close, log, sample_rows, to_device

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def kata():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2607_17419_amd as k
    k.lib()  # raises if libkata.so is missing: no fallback
    return k


def _run(kata, inp, dtype, C, span=0, g=1):
    import torch
    q = to_device(inp["q_dev"], dtype)
    k = to_device(inp["k_dev"], dtype)
    v = to_device(inp["v_dev"], dtype)
    if g == 1:
        out = kata.fwd_chunked(q, k, v, C, span_chunks=span)
    else:
        out = kata.mg_fwd_chunked(q, k, v, C, g, span_chunks=span)
    torch.cuda.synchronize()
    res = out.cpu().numpy()
    del q, k, v, out
    torch.cuda.empty_cache()
    return res


@pytest.mark.parametrize("n_rec", [1, 2, 5, 16, 17, 32, 33, 64, 65])
def test_span1_row_group_boundaries(kata, orc, n_rec):
    # the scan takes 1, 2, 4 or 8 row groups of 16 records by the record
    # count; these counts sit on both sides of each boundary
    T = 64 * n_rec - 13
    log(f"case span_chunks=1 B1 H2 T{T} d64 C64 ({n_rec} records per head), all rows")
    inp = workloads.make_inputs("mid_bf16", B=1, H=2, T=T)
    got = _run(kata, inp, "bf16", 64, span=1)
    ref = orc.fwd(inp["q"], inp["k"], inp["v"])
    assert_bf16_close(got, ref, f"span 1, {n_rec} records")


def test_span1_129_records_all_rows(kata, orc):
    # one chunk per record: T = 8192 + 37 at C = 64 gives 129 records per head
    T = 8192 + 37
    log(f"case span_chunks=1 B1 H2 T{T} d64 C64 (129 records per head), all rows")
    inp = workloads.make_inputs("mid_bf16", B=1, H=2, T=T)
    got = _run(kata, inp, "bf16", 64, span=1)
    ref = orc.fwd(inp["q"], inp["k"], inp["v"])
    assert_bf16_close(got, ref, "span 1, 129 records")


def test_span1_d32_past_128_records(kata, orc):
    T = 128 * 129 + 5
    log(f"case recall d32 span_chunks=1 B1 H2 T{T} C128 (130 records per head), sampled")
    inp = workloads.make_inputs("recall_bf16", B=1, H=2, T=T)
    got = _run(kata, inp, "bf16", 128, span=1)
    bh, tt = sample_rows(1, 2, T, 3, n_random=2048, head_rows=512, tail_rows=512)
    ref = orc.fwd_rows(inp["q"], inp["k"], inp["v"], bh, tt)
    assert_bf16_close(got.reshape(2, T, 64)[bh, tt], ref, "d32 span 1, 130 records")


def test_default_span_past_128_records(kata, orc):
    # the default 1024-token span: T = 131072 + 1000 gives 129 records per head
    T = 131072 + 1000
    log(f"case default span B1 H2 T{T} d64 C64 (129 records per head), sampled")
    inp = workloads.make_inputs("long_bf16", B=1, H=2, T=T)
    got = _run(kata, inp, "bf16", 64)
    bh, tt = sample_rows(1, 2, T, 2, n_random=2048, head_rows=1024, tail_rows=1024)
    ref = orc.fwd_rows(inp["q"], inp["k"], inp["v"], bh, tt)
    assert_bf16_close(got.reshape(2, T, 64)[bh, tt], ref, "default span, 129 records")


def test_m2_span1_past_128_records(kata, orc):
    T = 8192 + 100
    log(f"case M2 span_chunks=1 B1 H2 T{T} d64 g2 C64 (130 records per head), all rows")
    inp = workloads.make_inputs("mid_bf16", B=1, H=2, T=T)
    got = _run(kata, inp, "bf16", 64, span=1, g=2)
    ref = orc.fwd_mg(inp["q"], inp["k"], inp["v"], 2)
    assert_bf16_close(got, ref, "M2 span 1, 130 records")


@pytest.mark.parametrize("T,C", [(300, 2), (1000, 3), (600, 1)])
def test_fp32_path_past_128_chunks(kata, orc, T, C):
    log(f"case fp32 path d16 dv16 B1 H2 T{T} C{C} ({-(-T // C)} chunks per head)")
    rng = np.random.default_rng(T + C)
    q, k, v = workloads.gaussian_qkv(rng, 1, 2, T, 16, 16)
    got = _run(kata, dict(q_dev=q, k_dev=k, v_dev=v), "f32", C)
    assert_f32_close(got, orc.fwd(q, k, v), f"fp32 path T {T} C {C}")


# ---------------------------------------------------------------------------
# the long workload (B1 H16 T131072 d64 C64) on the measurement row set:
# every head's rows 0..4095 and its last 1024 rows, plus 4096 uniform rows
# ---------------------------------------------------------------------------

@pytest.fixture(scope="module")
def long_rows(orc):
    w = workloads.WORKLOADS["long_bf16"]
    inp = workloads.make_inputs(w)
    bh, tt = sample_rows(w.B, w.H, w.T, w.seed, n_random=4096, head_rows=4096, tail_rows=1024)
    log(f"  oracle on {bh.size} rows of the long workload")
    ref = orc.fwd_rows(inp["q"], inp["k"], inp["v"], bh, tt)
    return w, inp, bh, tt, ref


@pytest.mark.parametrize("span", [0, 1])
def test_long_workload_measurement_rows(kata, long_rows, span):
    # span 0: the library default (1024 tokens, 128 records per head);
    # span 1: the per-chunk form, 2048 records per head (16 scan blocks)
    w, inp, bh, tt, ref = long_rows
    log(f"case long workload span_chunks={span}: {w.note}, {bh.size} rows")
    got = _run(kata, inp, "bf16", w.C, span=span)
    assert np.all(np.isfinite(got))
    assert_bf16_close(got.reshape(w.B * w.H, w.T, w.dv)[bh, tt], ref,
                      f"long workload span {span}")
