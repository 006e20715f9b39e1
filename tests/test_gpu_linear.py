"""GPU parity of causal linear attention with the linear feature maps
(identity, ReLU + eps, ELU + 1, the Lorentz lift and its n_psi = d variant)
through the kata_lin_* C ABI, against the CPU oracle's definition.  Every case
prints its name and shape before it launches."""
from __future__ import annotations

import ctypes

import numpy as np
import pytest

import workloads
from gpu_helpers import (assert_bf16_close, log, row_rel_err, sample_rows, to_device)

pytestmark = pytest.mark.gpu

IDENT, RELU, ELU, LOR, LOR_S = 0, 1, 2, 3, 4
NAMES = {IDENT: "identity", RELU: "relu", ELU: "elu", LOR: "lorentz", LOR_S: "lorentz_s"}
EPS = 1e-3
# fp32 inputs: max-abs error <= 1e-5, relative to the output scale for the
# unnormalised readout (its outputs are not bounded by the values)
F32_TOL = 1e-5


@pytest.fixture(scope="module")
def kata():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2607_17419_amd as k
    k.lib()  # raises if libkata.so is missing: no fallback
    return k


def _norm_of(feature):
    return feature != IDENT


def _dev3(inp, dtype):
    return (to_device(inp["q_dev"], dtype), to_device(inp["k_dev"], dtype),
            to_device(inp["v_dev"], dtype))


def _run(kata, inp, dtype, C, feature, normalize, span=0, eps=EPS):
    import torch
    q, k, v = _dev3(inp, dtype)
    out = kata.lin_fwd_chunked(q, k, v, C, feature, eps, normalize, span_chunks=span)
    torch.cuda.synchronize()
    return out.cpu().numpy()


@pytest.mark.parametrize("feature", [IDENT, RELU, ELU, LOR, LOR_S])
@pytest.mark.parametrize("T", [1, 63, 64, 65, 300, 1025, 2100])
def test_fast_path_ragged(kata, orc, feature, T):
    norm = _norm_of(feature)
    log(f"case linear {NAMES[feature]} (bf16 MFMA) T={T} B1 H2 d64 C128 normalize={norm}")
    inp = workloads.make_inputs("scan_long_bf16", B=1, H=2, T=T)
    got = _run(kata, inp, "bf16", 128, feature, norm)
    ref = orc.lin_fwd(inp["q"], inp["k"], inp["v"], feature, EPS, norm)
    assert_bf16_close(got, ref, f"{NAMES[feature]} T {T}")


def test_fast_path_lorentz_unnormalised_and_scaled(kata, orc):
    # the lift's extra term in the plain readout (no denominator to hide an
    # error in it), and keys whose norms vary over the span, so that the
    # rank-one term's share of every weight differs from token to token
    T = 1500
    log(f"case linear lorentz plain readout, key scales 0.25..4, B1 H2 T{T} C64 span 2")
    inp = dict(workloads.make_inputs("scan_long_bf16", B=1, H=2, T=T))
    rng = np.random.default_rng(77)
    scale = (2.0 ** rng.integers(-2, 3, size=(1, 2, T, 1))).astype(np.float32)
    inp["k"] = inp["k"] * scale  # powers of two: the bf16 copy stays exact
    inp["k_dev"] = workloads.round_bf16(inp["k"])
    got = _run(kata, inp, "bf16", 64, LOR, False, span=2)
    ref = orc.lin_fwd(inp["q"], inp["k"], inp["v"], LOR, EPS, False)
    assert_bf16_close(got, ref, "lorentz plain readout")


@pytest.mark.parametrize("C,span", [(64, 1), (64, 3), (128, 2), (256, 1), (1024, 1), (64, 0)])
def test_fast_path_spans(kata, orc, C, span):
    T = 2500
    for feature in (IDENT, ELU, LOR):
        norm = _norm_of(feature)
        log(f"case linear {NAMES[feature]} C={C} span={span} B2 H2 T{T}")
        inp = workloads.make_inputs("scan_long_bf16", B=2, H=2, T=T)
        got = _run(kata, inp, "bf16", C, feature, norm, span)
        ref = orc.lin_fwd(inp["q"], inp["k"], inp["v"], feature, EPS, norm)
        assert_bf16_close(got, ref, f"{NAMES[feature]} C {C} span {span}")


def test_fast_path_normalised_identity_positive_inputs(kata, orc):
    # psi(x) = x with the normalised readout is well posed where every weight
    # is positive: entrywise non-negative q and k
    T = 700
    log(f"case linear identity normalised, non-negative q,k, B1 H2 T{T}")
    inp = workloads.make_inputs("scan_long_bf16", B=1, H=2, T=T)
    inp = dict(inp)
    for name in ("q", "k"):
        inp[name + "_dev"] = inp[name + "_dev"] & np.uint16(0x7FFF)  # clear the sign bit
        inp[name] = np.abs(inp[name])
    got = _run(kata, inp, "bf16", 128, IDENT, True)
    ref = orc.lin_fwd(inp["q"], inp["k"], inp["v"], IDENT, 0.0, True)
    assert_bf16_close(got, ref, "identity normalised")


def test_fast_path_zero_denominator(kata):
    # ReLU with eps = 0 and queries with no positive coordinate: psi(q) = 0,
    # the denominator is 0 and the readout is defined as 0
    import torch
    T = 200
    log(f"case linear relu eps=0, non-positive queries, B1 H2 T{T}")
    inp = dict(workloads.make_inputs("scan_long_bf16", B=1, H=2, T=T))
    inp["q_dev"] = inp["q_dev"] | np.uint16(0x8000)
    got = _run(kata, inp, "bf16", 128, RELU, True, eps=0.0)
    assert np.array_equal(got, np.zeros_like(got))
    torch.cuda.synchronize()


@pytest.mark.parametrize("feature", [IDENT, RELU, ELU, LOR, LOR_S])
@pytest.mark.parametrize("d,dv,C", [(16, 16, 32), (64, 64, 128), (32, 40, 100)])
def test_fp32_path(kata, orc, feature, d, dv, C):
    norm = _norm_of(feature)
    T = 300
    log(f"case linear {NAMES[feature]} fp32 inputs d={d} dv={dv} C={C} B1 H2 T{T}")
    rng = np.random.default_rng(11 + d + dv + feature)
    q = rng.standard_normal((1, 2, T, d)).astype(np.float32)
    k = rng.standard_normal((1, 2, T, d)).astype(np.float32)
    q /= np.linalg.norm(q, axis=-1, keepdims=True)
    k /= np.linalg.norm(k, axis=-1, keepdims=True)
    v = rng.standard_normal((1, 2, T, dv)).astype(np.float32)
    inp = dict(q_dev=q, k_dev=k, v_dev=v)
    got = _run(kata, inp, "f32", C, feature, norm)
    ref = orc.lin_fwd(q, k, v, feature, EPS, norm)
    err = float(np.max(np.abs(got.astype(np.float64) - ref)))
    tol = F32_TOL * max(1.0, float(np.max(np.abs(ref)))) if not norm else F32_TOL
    log(f"  {NAMES[feature]} fp32: max abs err={err:.3e} (tol {tol:.1e})")
    assert err <= tol


@pytest.mark.parametrize("feature", [LOR, RELU])
def test_bf16_inputs_fp32_path(kata, orc, feature):
    # chunk sizes that are not multiples of 64 run on the fp32 path with
    # bf16 inputs (the Lorentz lift, n_psi = d + 1, with its d + 1 features)
    T = 777
    log(f"case linear {NAMES[feature]} bf16 inputs on the fp32 path C=96 B1 H2 T{T}")
    inp = workloads.make_inputs("scan_long_bf16", B=1, H=2, T=T)
    got = _run(kata, inp, "bf16", 96, feature, True)
    ref = orc.lin_fwd(inp["q"], inp["k"], inp["v"], feature, EPS, True)
    assert_bf16_close(got, ref, f"{NAMES[feature]} fp32 path")


def test_timed_and_alloc_entry_points_match(kata):
    import torch
    T = 3000
    log(f"case linear elu: ws vs timed vs alloc entry points, B1 H4 T{T}")
    inp = workloads.make_inputs("scan_long_bf16", B=1, H=4, T=T)
    q, k, v = _dev3(inp, "bf16")
    a = kata.lin_fwd_chunked(q, k, v, 128, ELU, EPS, True)
    hip = ctypes.CDLL("libamdhip64.so")
    vp = ctypes.c_void_p
    hip.hipEventCreate.argtypes = [ctypes.POINTER(vp)]
    hip.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), vp, vp]
    hip.hipEventDestroy.argtypes = [vp]
    evs = (vp * 4)()
    for i in range(4):
        h = vp()
        assert hip.hipEventCreate(ctypes.byref(h)) == 0
        evs[i] = h
    b = kata.lin_fwd_chunked(q, k, v, 128, ELU, EPS, True, events=evs)
    c = kata.lin_fwd_chunked_alloc(q, k, v, 128, ELU, EPS, True)
    torch.cuda.synchronize()
    assert torch.equal(a, b) and torch.equal(a, c)
    for i in range(3):
        ms = ctypes.c_float()
        assert hip.hipEventElapsedTime(ctypes.byref(ms), evs[i], evs[i + 1]) == 0
        assert ms.value >= 0.0
    for i in range(4):
        hip.hipEventDestroy(evs[i])


@pytest.mark.parametrize("feature", [IDENT, ELU, LOR, LOR_S])
def test_full_size_sampled_rows(kata, orc, feature):
    # the bench workload (B1 H16 T131072 d64 C128) in the bench's launch
    # configuration (default span), checked on sampled rows
    import torch
    w = workloads.WORKLOADS["scan_long_bf16"]
    norm = _norm_of(feature)
    log(f"case linear {NAMES[feature]} full size B1 H16 T{w.T} C{w.C} normalize={norm}")
    inp = workloads.make_inputs(w)
    q, k, v = _dev3(inp, "bf16")
    out = kata.lin_fwd_chunked(q, k, v, w.C, feature, EPS, norm)
    torch.cuda.synchronize()
    bh, tt = sample_rows(w.B, w.H, w.T, 31, n_random=96, head_rows=2, tail_rows=2)
    got = out.reshape(w.B * w.H, w.T, w.dv)[torch.as_tensor(bh), torch.as_tensor(tt)].cpu().numpy()
    ref = orc.lin_fwd_rows(inp["q"], inp["k"], inp["v"], feature, EPS, norm, bh, tt)
    assert_bf16_close(got, ref, f"{NAMES[feature]} sampled rows")
    assert bool(torch.isfinite(out).all())
