"""GPU parity: libkata (through its C ABI) against the CPU oracle.

Every case prints its name and shape before it launches anything, so a run
that dies on the GPU still says which case was running.
"""
from __future__ import annotations

import numpy as np
import pytest

import workloads
from gpu_helpers import (assert_bf16_close, assert_f32_close, log, row_rel_err, sample_rows,
                         to_device)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def kata():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2607_17419_amd as k
    k.lib()  # raises if libkata.so is missing: no fallback
    return k


def _inputs(name, **kw):
    return workloads.make_inputs(name, **kw)


def _run_fwd(kata, inp, dtype, C, span=0):
    import torch
    q = to_device(inp["q_dev"], dtype)
    k = to_device(inp["k_dev"], dtype)
    v = to_device(inp["v_dev"], dtype)
    out = kata.fwd_chunked(q, k, v, C, span_chunks=span)
    torch.cuda.synchronize()
    return out.cpu().numpy()


# ---------------------------------------------------------------------------
# fp32 workload (tiny): full output, max-abs <= 1e-5
# ---------------------------------------------------------------------------

def test_tiny_f32_full(kata, orc):
    w = workloads.WORKLOADS["tiny_f32"]
    log(f"case tiny_f32 {w.note}")
    inp = _inputs("tiny_f32")
    got = _run_fwd(kata, inp, "f32", w.C)
    ref = orc.fwd(inp["q"], inp["k"], inp["v"])
    assert_f32_close(got, ref, "tiny_f32")


@pytest.mark.parametrize("shape", [
    (1, 1, 1, 16, 16, 32), (1, 2, 77, 16, 16, 32), (2, 1, 130, 8, 5, 7),
    (1, 1, 200, 32, 64, 64), (1, 1, 129, 64, 64, 128), (1, 2, 64, 3, 1, 1),
])
def test_fp32_path_shapes(kata, orc, shape):
    B, H, T, d, dv, C = shape
    log(f"case fp32 path B{B} H{H} T{T} d{d} dv{dv} C{C}")
    rng = np.random.default_rng(sum(shape))
    q = rng.standard_normal((B, H, T, d)).astype(np.float32)
    k = rng.standard_normal((B, H, T, d)).astype(np.float32)
    q /= np.linalg.norm(q, axis=-1, keepdims=True)
    k /= np.linalg.norm(k, axis=-1, keepdims=True)
    v = rng.standard_normal((B, H, T, dv)).astype(np.float32)
    got = _run_fwd(kata, dict(q_dev=q, k_dev=k, v_dev=v), "f32", C)
    assert_f32_close(got, orc.fwd(q, k, v), f"fp32 {shape}")


def test_bf16_on_fp32_path(kata, orc):
    # d = 16 is not an MFMA shape: bf16 inputs run through the fp32 kernels
    log("case bf16 d16 on the fp32 path")
    rng = np.random.default_rng(5)
    B, H, T, d, dv, C = 1, 2, 300, 16, 16, 32
    q, k, v = workloads.gaussian_qkv(rng, B, H, T, d, dv)
    (qv, kv, vv), (qd, kd, vd) = workloads._finish([q, k, v], "bf16")
    got = _run_fwd(kata, dict(q_dev=qd, k_dev=kd, v_dev=vd), "bf16", C)
    assert_f32_close(got, orc.fwd(qv, kv, vv), "bf16 d16 (exact products, fp32 sums)")


# ---------------------------------------------------------------------------
# bf16 MFMA path
# ---------------------------------------------------------------------------

def test_mid_bf16_two_heads_full(kata, orc):
    log("case mid_bf16 B1 H2 T4096 (all rows)")
    inp = _inputs("mid_bf16", B=1, H=2)
    got = _run_fwd(kata, inp, "bf16", 64)
    ref = orc.fwd(inp["q"], inp["k"], inp["v"])
    assert_bf16_close(got, ref, "mid_bf16 B1 H2")


@pytest.mark.parametrize("span", [1, 2, 3, 4, 8, 16, 32, 64])
def test_span_modes_agree(kata, orc, span):
    # span_chunks = 1 is the per-chunk form; larger spans fold chunks on chip
    # (8: one 512-query output workgroup per span; 32 and 64: several per
    # span, some of them wholly past T)
    T = 2 * 1024 + 37
    log(f"case span={span} B1 H2 T{T} d64 C64")
    inp = _inputs("mid_bf16", B=1, H=2, T=T)
    got = _run_fwd(kata, inp, "bf16", 64, span)
    ref = orc.fwd(inp["q"], inp["k"], inp["v"])
    assert_bf16_close(got, ref, f"span {span}")


@pytest.mark.parametrize("C", [32, 64, 128, 256])
def test_chunk_size_independent(kata, orc, C):
    T = 1500
    log(f"case C={C} B1 H1 T{T} d64")
    inp = _inputs("mid_bf16", B=1, H=1, T=T)
    got = _run_fwd(kata, inp, "bf16", C)
    ref = orc.fwd(inp["q"], inp["k"], inp["v"])
    assert_bf16_close(got, ref, f"C {C}")


@pytest.mark.parametrize("T", [1, 2, 31, 33, 63, 64, 65, 257, 1023, 1025])
def test_ragged_lengths(kata, orc, T):
    log(f"case ragged T={T} d64 C64")
    inp = _inputs("mid_bf16", B=1, H=2, T=T)
    got = _run_fwd(kata, inp, "bf16", 64)
    ref = orc.fwd(inp["q"], inp["k"], inp["v"])
    assert_bf16_close(got, ref, f"T {T}")


@pytest.mark.parametrize("span", [1, 4, 8])
def test_recall_d32(kata, orc, span):
    T = 3000
    log(f"case recall d32 B2 H2 T{T} C128 span {span}")
    inp = _inputs("recall_bf16", B=2, H=2, T=T)
    got = _run_fwd(kata, inp, "bf16", 128, span)
    ref = orc.fwd(inp["q"], inp["k"], inp["v"])
    assert_bf16_close(got, ref, f"recall d32 span {span}")


def test_zero_query_row(kata, orc):
    log("case zero query rows (D_t = 0 -> 0)")
    inp = _inputs("mid_bf16", B=1, H=1, T=700)
    for key in ("q_dev", "q"):
        inp[key] = inp[key].copy()
        inp[key][0, 0, [0, 5, 64, 640]] = 0
    got = _run_fwd(kata, inp, "bf16", 64)
    assert np.all(got[0, 0, [0, 5, 64, 640]] == 0.0)
    ref = orc.fwd(inp["q"], inp["k"], inp["v"])
    assert_bf16_close(got, ref, "zero rows")


def test_deterministic_and_metamorphic(kata):
    # No atomics: bitwise run-to-run identical.  q -> 2q scales every product
    # and sum by a power of two, so the output is bitwise unchanged.  k -> -k
    # leaves phi(k) and the squared scores unchanged in exact arithmetic, but
    # the matrix cores need not round a negated sum to the negated result, so
    # that one is held to a tight tolerance instead.
    import torch
    log("case determinism + sign/scale invariance, B1 H2 T2100")
    inp = _inputs("mid_bf16", B=1, H=2, T=2100)
    q = to_device(inp["q_dev"], "bf16")
    k = to_device(inp["k_dev"], "bf16")
    v = to_device(inp["v_dev"], "bf16")
    a = kata.fwd_chunked(q, k, v, 64)
    b = kata.fwd_chunked(q, k, v, 64)
    c = kata.fwd_chunked(q, -k, v, 64)
    e = kata.fwd_chunked(q * 2, k, v, 64)
    torch.cuda.synchronize()
    assert torch.equal(a, b)
    assert torch.equal(a, e)
    diff = float((a - c).abs().max() / a.abs().max())
    log(f"  k -> -k max rel diff {diff:.3e}")
    assert diff < 1e-4


def test_library_allocated_workspace(kata):
    import torch
    log("case kata_fwd_chunked (stream-ordered workspace) vs caller workspace")
    inp = _inputs("mid_bf16", B=1, H=2, T=1200)
    q = to_device(inp["q_dev"], "bf16")
    k = to_device(inp["k_dev"], "bf16")
    v = to_device(inp["v_dev"], "bf16")
    a = kata.fwd_chunked(q, k, v, 64)
    b = kata.fwd_chunked_alloc(q, k, v, 64)
    torch.cuda.synchronize()
    assert torch.equal(a, b)


def test_error_codes_live(kata):
    import torch
    log("case error codes with a live device")
    x = torch.zeros((1, 1, 8, 65), dtype=torch.bfloat16, device="cuda:0")
    with pytest.raises(kata.KataError) as ei:
        kata.fwd_chunked(x, x, x, 64)
    assert ei.value.status == kata.KATA_ERR_UNSUPPORTED
    q = torch.zeros((1, 1, 64, 64), dtype=torch.bfloat16, device="cuda:0")
    ws = torch.empty(16, dtype=torch.uint8, device="cuda:0")
    with pytest.raises(kata.KataError) as ei:
        kata.lib()  # noqa
        import ctypes
        st = kata.lib().kata_fwd_chunked_ws(
            ctypes.c_void_p(q.data_ptr()), ctypes.c_void_p(q.data_ptr()),
            ctypes.c_void_p(q.data_ptr()), ctypes.c_void_p(ws.data_ptr()), 1, 1, 64, 64, 64, 64,
            kata.KATA_BF16, 0, ctypes.c_void_p(ws.data_ptr()), 16, None)
        kata._check(st, "kata_fwd_chunked_ws")
    assert ei.value.status == kata.KATA_ERR_INVALID_ARG


def test_allocation_failure_then_success(kata):
    # a workspace of terabytes: the allocation fails, KATA_ERR_HIP comes back
    # before any launch, and the failure does not leak into the next call
    import torch
    from test_abi_cpu import FAKE, huge_alloc_calls
    log("case allocation failure (terabyte workspaces) then a normal call")
    L = kata.lib()
    for name, call in huge_alloc_calls(L, FAKE):
        assert call() == kata.KATA_ERR_HIP, name
        inp = _inputs("mid_bf16", B=1, H=1, T=300)
        q, k, v = (to_device(inp[n], "bf16") for n in ("q_dev", "k_dev", "v_dev"))
        a = kata.fwd_chunked_alloc(q, k, v, 64)
        b = kata.fwd_chunked(q, k, v, 64)
        torch.cuda.synchronize()
        assert torch.equal(a, b), name


# ---------------------------------------------------------------------------
# full-size workloads in the bench's launch configuration, sampled rows
# ---------------------------------------------------------------------------

# (the long workload's measurement row set is in test_gpu_scan_blocks.py)
@pytest.mark.parametrize("name", ["mid_bf16", "recall_bf16"])
def test_full_size_sampled(kata, orc, name):
    w = workloads.WORKLOADS[name]
    log(f"case full-size {name}: {w.note}")
    inp = _inputs(name)
    got = _run_fwd(kata, inp, "bf16", w.C)
    assert np.all(np.isfinite(got))
    bh, tt = sample_rows(w.B, w.H, w.T, w.seed, n_random=4096, head_rows=1024, tail_rows=256)
    ref = orc.fwd_rows(inp["q"], inp["k"], inp["v"], bh, tt)
    got_rows = got.reshape(w.B * w.H, w.T, w.dv)[bh, tt]
    assert_bf16_close(got_rows, ref, f"{name} sampled")


# ---------------------------------------------------------------------------
# prefill + decode
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_prefill_state(kata, orc, dtype):
    import torch
    log(f"case prefill state {dtype} B2 H3 T300 d64 dv64")
    rng = np.random.default_rng(11)
    q, k, v = workloads.gaussian_qkv(rng, 2, 3, 300, 64, 64)
    (qv, kv, vv), (qd, kd, vd) = workloads._finish([q, k, v], dtype)
    S, z = kata.prefill_state(to_device(kd, dtype), to_device(vd, dtype))
    torch.cuda.synchronize()
    S_ref, z_ref = orc.state(kv, vv)
    errS = np.max(np.abs(S.cpu().numpy() - S_ref)) / max(1.0, np.max(np.abs(S_ref)))
    errz = np.max(np.abs(z.cpu().numpy() - z_ref)) / max(1.0, np.max(np.abs(z_ref)))
    log(f"  prefill rel err S={errS:.2e} z={errz:.2e}")
    assert errS < 1e-5 and errz < 1e-5


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_decode_small(kata, orc, dtype):
    import torch
    B, H, P, steps, d, dv = 2, 3, 100, 12, 64, 64
    log(f"case decode {dtype} B{B} H{H} prefix {P} steps {steps}")
    rng = np.random.default_rng(13)
    q, k, v = workloads.gaussian_qkv(rng, B, H, P + steps, d, dv)
    (qv, kv, vv), (qd, kd, vd) = workloads._finish([q, k, v], dtype)
    ref = orc.fwd(qv, kv, vv)
    S, z = kata.prefill_state(to_device(kd[:, :, :P].copy(), dtype),
                              to_device(vd[:, :, :P].copy(), dtype))
    for s in range(steps):
        t = P + s
        o = kata.decode_step(S, z, to_device(qd[:, :, t].copy(), dtype),
                             to_device(kd[:, :, t].copy(), dtype),
                             to_device(vd[:, :, t].copy(), dtype))
        torch.cuda.synchronize()
        assert_f32_close(o.cpu().numpy(), ref[:, :, t], f"decode step {s}")


def test_decode_full_size_sampled(kata, orc):
    import torch
    w = workloads.WORKLOADS["decode_bf16"]
    log(f"case decode full size {w.note}")
    inp = _inputs("decode_bf16")
    S, z = kata.prefill_state(to_device(inp["k_dev"], "bf16"), to_device(inp["v_dev"], "bf16"))
    sq = to_device(inp["steps_q_dev"], "bf16")
    sk = to_device(inp["steps_k_dev"], "bf16")
    sv = to_device(inp["steps_v_dev"], "bf16")
    outs = []
    for s in range(w.steps):
        outs.append(kata.decode_step(S, z, sq[:, :, s].contiguous(), sk[:, :, s].contiguous(),
                                     sv[:, :, s].contiguous()))
    torch.cuda.synchronize()
    got = torch.stack(outs, dim=2).cpu().numpy()  # [B,H,steps,dv]
    # oracle on 64 heads of the concatenated sequence: the first and last
    # eight plus 48 drawn uniformly
    rng = np.random.default_rng(w.seed + 2000)
    heads = sorted(set(list(range(8)) + list(range(w.B * w.H - 8, w.B * w.H)) +
                       list(rng.choice(np.arange(8, w.B * w.H - 8), 48, replace=False))))
    for bh in heads:
        b, h = divmod(bh, w.H)
        qc = np.concatenate([inp["q"][b, h], inp["steps_q"][b, h]])[None, None]
        kc = np.concatenate([inp["k"][b, h], inp["steps_k"][b, h]])[None, None]
        vc = np.concatenate([inp["v"][b, h], inp["steps_v"][b, h]])[None, None]
        rows = np.arange(w.T, w.T + w.steps)
        ref = orc.fwd_rows(qc, kc, vc, np.zeros_like(rows), rows)
        assert_bf16_close(got[b, h], ref, f"decode head {bh}")
        assert float(np.max(row_rel_err(got[b, h], ref))) < 1e-4


# ---------------------------------------------------------------------------
# input magnitudes: the MFMA path's state products are fp16 with per-span
# power-of-two scales; every case must match the oracle at the same bar
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("ks,vs", [(300.0, 1.0), (2.0 ** -10, 1.0), (1.0, 3.0e4), (1.0, 1e-6),
                                   (2.0 ** -40, 2.0 ** 20), (50.0, 200.0), (4.0, 50.0)])
def test_input_magnitudes(kata, orc, ks, vs):
    log(f"case magnitudes k x {ks:g}, v x {vs:g}: B1 H2 T2500 d64 C64")
    rng = np.random.default_rng(71)
    q, k, v = workloads.gaussian_qkv(rng, 1, 2, 2500, 64, 64)
    (qv, kv, vv), (qd, kd, vd) = workloads._finish([q, k * np.float32(ks), v * np.float32(vs)],
                                                   "bf16")
    got = _run_fwd(kata, dict(q_dev=qd, k_dev=kd, v_dev=vd), "bf16", 64)
    assert_bf16_close(got, orc.fwd(qv, kv, vv), f"k x {ks:g}, v x {vs:g}")


def test_later_block_outgrows_first(kata, orc):
    # the first 128 keys of every span are unit vectors, later keys are 2000x
    # larger (their fp16 feature products overflow without a scale): the
    # span is redone with its exact scales
    log("case later keys 2000x the first block's: B1 H2 T3000 d64 C64")
    rng = np.random.default_rng(72)
    q, k, v = workloads.gaussian_qkv(rng, 1, 2, 3000, 64, 64)
    big = (np.arange(3000) % 1024) >= 128
    k = k * np.where(big, np.float32(2000.0), np.float32(1.0))[None, None, :, None]
    (qv, kv, vv), (qd, kd, vd) = workloads._finish([q, k, v], "bf16")
    got = _run_fwd(kata, dict(q_dev=qd, k_dev=kd, v_dev=vd), "bf16", 64)
    assert_bf16_close(got, orc.fwd(qv, kv, vv), "later keys 2000x")
