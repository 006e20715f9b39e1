"""Helpers for the GPU tests: move seeded workload inputs to the device and
compare results with the CPU oracle at the stated tolerances."""
from __future__ import annotations

import sys

import numpy as np

# Tolerances.  fp32 inputs: max-abs error <= 1e-5.  bf16 inputs with fp32
# accumulation: per-row relative l2 error ||o - o_ref|| / ||o_ref|| <= 2e-2.
F32_MAX_ABS = 1e-5
BF16_ROW_REL = 2e-2


def log(msg: str):
    print(msg, flush=True)
    sys.stdout.flush()


def to_device(payload: np.ndarray, dtype: str, device="cuda:0"):
    import torch
    if dtype == "bf16":
        t = torch.from_numpy(np.ascontiguousarray(payload).view(np.int16))
        return t.to(device).view(torch.bfloat16)
    return torch.from_numpy(np.ascontiguousarray(payload, dtype=np.float32)).to(device)


def row_rel_err(got: np.ndarray, ref: np.ndarray) -> np.ndarray:
    """Per-row relative l2 error over the last axis."""
    got = np.asarray(got, dtype=np.float64).reshape(-1, ref.shape[-1])
    ref = np.asarray(ref, dtype=np.float64).reshape(-1, ref.shape[-1])
    num = np.linalg.norm(got - ref, axis=1)
    den = np.linalg.norm(ref, axis=1)
    both_zero = (den == 0) & (num == 0)
    rel = np.where(den > 0, num / np.where(den > 0, den, 1.0), np.inf)
    rel[both_zero] = 0.0
    return rel


def assert_bf16_close(got, ref, what=""):
    rel = row_rel_err(got, ref)
    worst = float(rel.max()) if rel.size else 0.0
    log(f"  {what}: rows={rel.size} max row rel err={worst:.3e} "
        f"median={float(np.median(rel)) if rel.size else 0.0:.3e}")
    assert np.all(np.isfinite(np.asarray(got))), f"{what}: non-finite output"
    assert worst <= BF16_ROW_REL, f"{what}: max row rel err {worst:.3e} > {BF16_ROW_REL}"


def assert_f32_close(got, ref, what=""):
    err = float(np.max(np.abs(np.asarray(got, dtype=np.float64) - ref))) if ref.size else 0.0
    log(f"  {what}: max abs err={err:.3e}")
    assert err <= F32_MAX_ABS, f"{what}: max abs err {err:.3e} > {F32_MAX_ABS}"


def sample_rows(B: int, H: int, T: int, seed: int, n_random: int, head_rows: int,
                tail_rows: int):
    """Deterministic row sample: the first `head_rows` and last `tail_rows`
    rows of every head, plus `n_random` uniform (head, row) pairs."""
    rng = np.random.default_rng(seed + 1000)
    bh, tt = [], []
    for h in range(B * H):
        r = list(range(min(head_rows, T))) + list(range(max(0, T - tail_rows), T))
        bh += [h] * len(r)
        tt += r
    bh += list(rng.integers(0, B * H, size=n_random))
    tt += list(rng.integers(0, T, size=n_random))
    pairs = sorted(set(zip(bh, tt)))
    return np.array([p[0] for p in pairs]), np.array([p[1] for p in pairs])
