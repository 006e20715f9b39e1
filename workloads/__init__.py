"""Seeded synthetic inputs for the causal KATA-M1 forward and decode step.

This module holds the workload table and the input generators only; it holds
none of the method's arithmetic.  Both the CPU oracle's tests and the GPU path's
tests and bench draw their inputs from here, so they see identical values.

Recipe (every config):
  * ``numpy.random.default_rng(seed)`` (PCG64), draws in float32;
  * q and k rows are L2-normalised in float32 (the paper's workloads use
    normalised query/key directions), v ~ N(0, 1);
  * bf16 configs then round every float32 value to bf16 with round-to-nearest-
    even and do not renormalise; the oracle consumes the rounded values.
Draw order: q, k, v.  The recall-shaped config draws its key pool, key indices,
query sources, query noise and values in that order.  The decode config draws the
prefix (q, k, v) and then the steps (q, k, v).
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np


@dataclass(frozen=True)
class Workload:
    name: str
    B: int
    H: int
    T: int
    d: int
    dv: int
    C: int
    dtype: str          # "f32" or "bf16": dtype of q, k, v
    seed: int
    kind: str = "gaussian"   # "gaussian", "recall" or "decode"
    steps: int = 0           # decode steps (decode kind only)
    pool: int = 0            # key pool size (recall kind only)
    noise_var: float = 0.0   # query noise variance (recall kind only)
    note: str = field(default="", compare=False)


# The five workloads.  Names say what they are; sizes are the paper-derived
# shapes: the mid config is the paper's B=8, H=16, d=64 latency-table shape at
# T=4096; the long one is its single-sequence 131072-token case.
WORKLOADS = {
    "tiny_f32": Workload("tiny_f32", 1, 2, 256, 16, 16, 32, "f32", 0,
                         note="B1 H2 T256 d16 dv16 C32, fp32"),
    "mid_bf16": Workload("mid_bf16", 8, 16, 4096, 64, 64, 64, "bf16", 1,
                         note="B8 H16 T4096 d64 dv64 C64, bf16"),
    "long_bf16": Workload("long_bf16", 1, 16, 131072, 64, 64, 64, "bf16", 2,
                          note="B1 H16 T131072 d64 dv64 C64, bf16 (2048 chunks)"),
    "recall_bf16": Workload("recall_bf16", 4, 8, 16384, 32, 64, 128, "bf16", 3,
                            kind="recall", pool=512, noise_var=0.01,
                            note="B4 H8 T16384 d32 dv64 C128, keys from a 512-key pool"),
    "decode_bf16": Workload("decode_bf16", 256, 16, 1024, 64, 64, 64, "bf16", 4,
                            kind="decode", steps=128,
                            note="B256 H16 d64 dv64, 1024-token prefix then 128 steps"),
    # linear (n_psi = d) features: the shape of the paper's small-batch
    # associative-scan table (B = 1, H = 16, d_head = 64, C = 128, bf16)
    "scan_long_bf16": Workload("scan_long_bf16", 1, 16, 131072, 64, 64, 128, "bf16", 5,
                               note="B1 H16 T131072 d64 dv64 C128, bf16, linear features"),
}


def round_bf16(x: np.ndarray) -> np.ndarray:
    """float32 -> bf16 bit patterns (uint16), round-to-nearest-even."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32).astype(np.uint64)
    rounded = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    out = rounded.astype(np.uint16)
    nan = np.isnan(x)
    if nan.any():
        out[nan] = 0x7FC0
    return out


def bf16_to_f32(bits: np.ndarray) -> np.ndarray:
    """bf16 bit patterns (uint16) -> float32, exact."""
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def _unit_rows(x: np.ndarray) -> np.ndarray:
    nrm = np.sqrt(np.sum(x.astype(np.float32) ** 2, axis=-1, keepdims=True, dtype=np.float32))
    return (x / np.maximum(nrm, np.float32(1e-30))).astype(np.float32)


def _finish(arrs, dtype: str):
    """Return (values as float32 exactly as the device sees them, device payloads).

    For bf16 the payload is the uint16 bit pattern array; for f32 it is float32.
    """
    vals, payload = [], []
    for a in arrs:
        if dtype == "bf16":
            bits = round_bf16(a)
            payload.append(bits)
            vals.append(bf16_to_f32(bits))
        else:
            a = np.ascontiguousarray(a, dtype=np.float32)
            payload.append(a)
            vals.append(a)
    return vals, payload


def gaussian_qkv(rng, B, H, T, d, dv):
    q = _unit_rows(rng.standard_normal((B, H, T, d), dtype=np.float32))
    k = _unit_rows(rng.standard_normal((B, H, T, d), dtype=np.float32))
    v = rng.standard_normal((B, H, T, dv), dtype=np.float32)
    return q, k, v


def recall_qkv(rng, B, H, T, d, dv, pool, noise_var):
    """Keys drawn i.i.d. from a per-head pool of unit keys; query t re-presents
    the key at a uniform earlier position j < t (j = 0 at t = 0) plus
    N(0, noise_var) noise per coordinate, then is renormalised."""
    keys = _unit_rows(rng.standard_normal((B, H, pool, d), dtype=np.float32))
    idx = rng.integers(0, pool, size=(B, H, T))
    bb = np.arange(B)[:, None, None]
    hh = np.arange(H)[None, :, None]
    k = keys[bb, hh, idx]
    t = np.arange(T)[None, None, :]
    j = np.floor(rng.random((B, H, T)) * t).astype(np.int64)
    src = k[bb, hh, j]
    noise = rng.standard_normal((B, H, T, d), dtype=np.float32) * np.float32(np.sqrt(noise_var))
    q = _unit_rows(src + noise)
    v = rng.standard_normal((B, H, T, dv), dtype=np.float32)
    return q, k.astype(np.float32), v


def make_inputs(w: Workload | str, B: int | None = None, H: int | None = None,
                T: int | None = None):
    """Seeded inputs of a workload (optionally with a smaller B, H or T, drawn
    with the same recipe and seed).

    Returns a dict with ``q, k, v`` (float32 values exactly as the device sees
    them), ``q_dev, k_dev, v_dev`` (float32 or bf16 bit patterns) and, for the
    decode kind, ``steps_q, steps_k, steps_v`` (+ ``*_dev``) of shape
    [B, H, steps, .].
    """
    if isinstance(w, str):
        w = WORKLOADS[w]
    B = w.B if B is None else B
    H = w.H if H is None else H
    T = w.T if T is None else T
    rng = np.random.default_rng(w.seed)
    if w.kind == "recall":
        q, k, v = recall_qkv(rng, B, H, T, w.d, w.dv, w.pool, w.noise_var)
    else:
        q, k, v = gaussian_qkv(rng, B, H, T, w.d, w.dv)
    (qv, kv, vv), (qd, kd, vd) = _finish([q, k, v], w.dtype)
    out = dict(q=qv, k=kv, v=vv, q_dev=qd, k_dev=kd, v_dev=vd)
    if w.kind == "decode":
        sq, sk, sv = gaussian_qkv(rng, B, H, w.steps, w.d, w.dv)
        (sqv, skv, svv), (sqd, skd, svd) = _finish([sq, sk, sv], w.dtype)
        out.update(steps_q=sqv, steps_k=skv, steps_v=svv,
                   steps_q_dev=sqd, steps_k_dev=skd, steps_v_dev=svd)
    return out
