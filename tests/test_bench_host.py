"""Host-side accounting of the benchmark: algorithmic work of the chunked
forward (packed features n = d(d+1)/2; a chunk's state is needed only by later
chunks and a chunk's readout only where earlier chunks exist)."""
import os
import sys
from types import SimpleNamespace

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
import bench  # noqa: E402


def _count_by_chunks(B, H, T, d, dv, C):
    n = d * (d + 1) // 2
    state = readout = intra = 0
    for c0 in range(0, T, C):
        rows = min(C, T - c0)
        if c0 + C < T:
            state += rows * (2 * n * dv + n)
        if c0 > 0:
            readout += rows * (2 * n * dv + 2 * n)
        intra += rows * (C + 1) * (d + dv)
    return B * H * state, B * H * (readout + intra)


def test_algorithmic_matches_a_per_chunk_count():
    for T in (1, 63, 64, 65, 200, 4096):
        w = SimpleNamespace(B=2, H=3, T=T, d=8, dv=4, C=64)
        a = bench.algorithmic(w, 1024)
        st, out = _count_by_chunks(2, 3, T, 8, 4, 64)
        assert (a["state_flop"], a["output_flop"]) == (st, out), T
        assert a["total_flop"] == st + out


def test_one_chunk_needs_no_state_and_no_readout():
    w = SimpleNamespace(B=1, H=1, T=64, d=16, dv=16, C=64)
    a = bench.algorithmic(w, 1024)
    assert a["state_flop"] == 0
    assert a["output_flop"] == 64 * 65 * 32


def test_scan_bytes_skip_the_last_span_record():
    w = SimpleNamespace(B=1, H=2, T=4096, d=64, dv=64, C=64)
    n = 64 * 65 // 2
    rec = n * 65 * 2
    # four spans of 1024 tokens: three records read, four prefixes written
    assert bench.algorithmic(w, 1024)["scan_bytes"] == 2 * (3 + 4) * rec
