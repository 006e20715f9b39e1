"""GPU parity of KATA-Mg (block-diagonal PSD feature, g blocks of d/g
coordinates) through the kata_mg_* C ABI against the CPU oracle's KATA-Mg
definition.  Every case prints its name and shape before it launches."""
from __future__ import annotations

import numpy as np
import pytest

import workloads
from gpu_helpers import (assert_bf16_close, assert_f32_close, log, sample_rows, to_device)

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
    return (to_device(inp["q_dev"], dtype), to_device(inp["k_dev"], dtype),
            to_device(inp["v_dev"], dtype))


def _run(kata, inp, dtype, C, g, span=0):
    import torch
    q, k, v = _dev3(inp, dtype)
    out = kata.mg_fwd_chunked(q, k, v, C, g, span_chunks=span)
    torch.cuda.synchronize()
    return out.cpu().numpy()


@pytest.mark.parametrize("T", [1, 2, 33, 257, 1025, 2100])
def test_m2_ragged(kata, orc, T):
    log(f"case M2 (bf16 MFMA) ragged T={T} B1 H2 d64 g2 C64")
    inp = workloads.make_inputs("mid_bf16", B=1, H=2, T=T)
    got = _run(kata, inp, "bf16", 64, 2)
    ref = orc.fwd_mg(inp["q"], inp["k"], inp["v"], 2)
    assert_bf16_close(got, ref, f"M2 T {T}")


@pytest.mark.parametrize("C,span", [(64, 1), (64, 4), (32, 16), (128, 8), (256, 0)])
def test_m2_spans_and_chunks(kata, orc, C, span):
    T = 2500
    log(f"case M2 C={C} span={span} B1 H2 T{T}")
    inp = workloads.make_inputs("mid_bf16", B=1, H=2, T=T)
    got = _run(kata, inp, "bf16", C, 2, span)
    ref = orc.fwd_mg(inp["q"], inp["k"], inp["v"], 2)
    assert_bf16_close(got, ref, f"M2 C {C} span {span}")


@pytest.mark.parametrize("T", [1, 31, 300, 1025])
def test_m2_quadratic(kata, orc, T):
    import torch
    log(f"case M2 quadratic T={T} B1 H2 d64")
    inp = workloads.make_inputs("mid_bf16", B=1, H=2, T=T)
    q, k, v = _dev3(inp, "bf16")
    out = kata.mg_fwd_quadratic(q, k, v, 2)
    torch.cuda.synchronize()
    ref = orc.fwd_mg(inp["q"], inp["k"], inp["v"], 2)
    assert_bf16_close(out.cpu().numpy(), ref, f"M2 quadratic T {T}")


@pytest.mark.parametrize("d,g,C", [(16, 2, 32), (16, 4, 16), (8, 8, 32), (64, 4, 64)])
def test_mg_fp32_path(kata, orc, d, g, C):
    log(f"case Mg fp32 inputs d={d} g={g} C={C} B1 H2 T300")
    rng = np.random.default_rng(5 + d + g)
    q = rng.standard_normal((1, 2, 300, d)).astype(np.float32)
    k = rng.standard_normal((1, 2, 300, d)).astype(np.float32)
    q /= np.linalg.norm(q, axis=-1, keepdims=True)
    k /= np.linalg.norm(k, axis=-1, keepdims=True)
    v = rng.standard_normal((1, 2, 300, 16)).astype(np.float32)
    inp = dict(q_dev=q, k_dev=k, v_dev=v)
    got = _run(kata, inp, "f32", C, g)
    ref = orc.fwd_mg(q, k, v, g)
    assert_f32_close(got, ref, f"Mg fp32 d {d} g {g}")


def test_mg_bf16_on_fp32_path(kata, orc):
    log("case M4 bf16 inputs on the fp32 path, d64 g4 C64 B1 H2 T700")
    inp = workloads.make_inputs("mid_bf16", B=1, H=2, T=700)
    got = _run(kata, inp, "bf16", 64, 4)
    ref = orc.fwd_mg(inp["q"], inp["k"], inp["v"], 4)
    assert_bf16_close(got, ref, "M4 on the fp32 path")


def test_mg_g1_is_m1(kata):
    import torch
    log("case Mg API with g=1 equals the M1 API (bf16 MFMA, fp32 path)")
    inp = workloads.make_inputs("mid_bf16", B=1, H=2, T=1500)
    q, k, v = _dev3(inp, "bf16")
    a = kata.mg_fwd_chunked(q, k, v, 64, 1)
    b = kata.fwd_chunked(q, k, v, 64)
    torch.cuda.synchronize()
    assert torch.equal(a, b)
    inp = workloads.make_inputs("tiny_f32")
    q, k, v = _dev3(inp, "f32")
    a = kata.mg_fwd_chunked(q, k, v, 32, 1)
    b = kata.fwd_chunked(q, k, v, 32)
    torch.cuda.synchronize()
    assert torch.equal(a, b)


def test_m2_zero_query_rows(kata, orc):
    log("case M2 zero query rows (D_t = 0 -> 0)")
    inp = workloads.make_inputs("mid_bf16", B=1, H=1, T=700)
    for key in ("q_dev", "q"):
        inp[key] = inp[key].copy()
        inp[key][0, 0, [0, 5, 64, 640]] = 0
    got = _run(kata, inp, "bf16", 64, 2)
    assert np.all(got[0, 0, [0, 5, 64, 640]] == 0.0)
    ref = orc.fwd_mg(inp["q"], inp["k"], inp["v"], 2)
    assert_bf16_close(got, ref, "M2 zero rows")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_m2_prefill_decode(kata, orc, dtype):
    import torch
    B, H, P, steps, d, dv = 2, 3, 200, 8, 64, 64
    log(f"case M2 prefill + {steps} decode steps {dtype} B{B} H{H} prefix {P} d64 dv64")
    rng = np.random.default_rng(17)
    q, k, v = workloads.gaussian_qkv(rng, B, H, P + steps, d, dv)
    (qv, kv, vv), (qd, kd, vd) = workloads._finish([q, k, v], dtype)
    S, z = kata.mg_prefill_state(to_device(kd[:, :, :P].copy(), dtype),
                                 to_device(vd[:, :, :P].copy(), dtype), 2)
    torch.cuda.synchronize()
    S_ref, z_ref = orc.state_mg(kv[:, :, :P], vv[:, :, :P], 2)
    errS = np.max(np.abs(S.cpu().numpy() - S_ref)) / max(1.0, np.max(np.abs(S_ref)))
    errz = np.max(np.abs(z.cpu().numpy() - z_ref)) / max(1.0, np.max(np.abs(z_ref)))
    log(f"  prefill rel err S={errS:.2e} z={errz:.2e}")
    assert errS < 1e-5 and errz < 1e-5
    ref = orc.fwd_mg(qv, kv, vv, 2)
    for s in range(steps):
        t = P + s
        o = kata.mg_decode_step(S, z, to_device(qd[:, :, t].copy(), dtype),
                                to_device(kd[:, :, t].copy(), dtype),
                                to_device(vd[:, :, t].copy(), dtype), 2)
        torch.cuda.synchronize()
        assert_f32_close(o.cpu().numpy(), ref[:, :, t], f"M2 decode step {s}")


def test_m2_long_sampled(kata, orc):
    w = workloads.WORKLOADS["long_bf16"]
    log(f"case M2 full-size long workload, sampled rows: {w.note}, g=2")
    inp = workloads.make_inputs(w)
    got = _run(kata, inp, "bf16", w.C, 2)
    assert np.all(np.isfinite(got))
    bh, tt = sample_rows(w.B, w.H, w.T, w.seed, n_random=512, head_rows=256, tail_rows=4)
    ref = orc.fwd_mg_rows(inp["q"], inp["k"], inp["v"], 2, bh, tt)
    assert_bf16_close(got.reshape(w.B * w.H, w.T, w.dv)[bh, tt], ref, "M2 long sampled")
