"""GPU parity of the O(T) chunked backward (kata_bwd_chunked*) against the CPU
oracle's backward by the definition.  Gradients are of sum_t <dout_t, o_t>.
Every case prints its name and shape before it launches.

Tolerances: fp32 inputs, max-abs error <= 1e-5 relative to the gradient's
scale (max |ref|, at least 1); bf16 inputs, the relative l2 error of each
gradient tensor per head <= 2e-2.  Rows with a small denominator D_t have
large gradients (a_t = dout_t / D_t), hence the scale-relative forms.

Two gradient kernels serve bf16 inputs.  For d = dv = C = 64 and one feature
block the products run on the bf16 matrix cores: the prefix and suffix states
and the in-chunk score products are rounded to bf16 once (8 significant bits,
unit roundoff u = 2^-8), and every product of the gradients carries at most
two rounded factors, so each term is off by at most 2u = 2^-7 relative.  Fed
the exact forward output, that path is held to the bf16 bound 2e-2 (2.5 x
2^-7, room for cancellation between terms of either sign; measured about
2e-3).  Every other shape runs in fp32 arithmetic and is held to 1e-4."""
from __future__ import annotations

import ctypes

import numpy as np
import pytest

import workloads
from gpu_helpers import log, to_device

pytestmark = pytest.mark.gpu

F32_TOL = 1e-5
BF16_REL = 2e-2
BF16_GRAD_REL = 2e-2  # bf16 matrix-core gradients, exact forward output given
F32_GRAD_REL = 1e-4   # fp32 gradients kernels, exact forward output given
U2 = 2.0 ** -7        # relative error bound of a product of two bf16-rounded factors


def _bf_path(d, dv, C, g):
    """True when bf16 inputs of this shape take the bf16 matrix-core gradients."""
    return d == 64 and dv == 64 and C == 64 and g == 1


@pytest.fixture(scope="module")
def kata():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2607_17419_amd as k
    k.lib()  # raises if libkata.so is missing: no fallback
    return k


def _dout(shape, seed):
    return np.random.default_rng(seed).standard_normal(shape).astype(np.float32)


def _gpu_bwd(kata, inp, dtype, dout, C, g, out=None, fwd_C=None):
    """o from the library forward (unless given), then the library backward."""
    import torch
    q, k, v = (to_device(inp[n], dtype) for n in ("q_dev", "k_dev", "v_dev"))
    if out is None:
        out = kata.mg_fwd_chunked(q, k, v, fwd_C or C, g)
    else:
        out = torch.from_numpy(np.ascontiguousarray(out, dtype=np.float32)).to(q.device)
    d_out = torch.from_numpy(dout).to(q.device)
    dq, dk, dv = kata.bwd_chunked(q, k, v, out, d_out, C, g)
    torch.cuda.synchronize()
    return dq.cpu().numpy(), dk.cpu().numpy(), dv.cpu().numpy()


def _check_f32(got, ref, what):
    for name, a, b in zip(("dq", "dk", "dv"), got, ref):
        err = float(np.max(np.abs(a.astype(np.float64) - b)))
        tol = F32_TOL * max(1.0, float(np.max(np.abs(b))))
        log(f"  {what} {name}: max abs err {err:.3e} (tol {tol:.2e})")
        assert np.all(np.isfinite(a)) and err <= tol, (what, name)


def _check_rel(got, ref, what, tol=BF16_REL, per_row=True):
    """Per-head relative l2 error of each gradient tensor, and per row: the
    error of row t against max(|ref_t|, the rms row norm of its head), so an
    error confined to one chunk or slab of a long head cannot hide under the
    head's norm, while rows with tiny gradients are held to the head's scale.

    The per-row bound applies to the backward fed the exact forward output.
    Given the library's own forward output instead, dq_t carries b_t =
    -<dout_t, o_t> / D_t times dD_t/dq_t, a term that cancels exactly against
    the rest of dq_t only for the exact o_t: the forward's bf16 rounding of
    o_t (a few 1e-3) then shows up in rows where that cancellation is deep,
    which is conditioning of the composition, not an error of the backward;
    those runs keep the per-head bound only."""
    for name, a, b in zip(("dq", "dk", "dv"), got, ref):
        T, w = b.shape[2], b.shape[3]
        a = a.astype(np.float64).reshape(-1, T, w)
        b = b.reshape(-1, T, w)
        rel = (np.linalg.norm((a - b).reshape(-1, T * w), axis=1) /
               np.maximum(np.linalg.norm(b.reshape(-1, T * w), axis=1), 1e-30))
        row_err = np.linalg.norm(a - b, axis=2)
        row_ref = np.linalg.norm(b, axis=2)
        rms = np.sqrt(np.mean(row_ref ** 2, axis=1, keepdims=True))
        row_rel = row_err / np.maximum(np.maximum(row_ref, rms), 1e-30)
        log(f"  {what} {name}: max per-head rel l2 err {float(rel.max()):.3e}, "
            f"max per-row {float(row_rel.max()):.3e} (tol {tol:.0e})")
        assert np.all(np.isfinite(a)) and float(rel.max()) <= tol, (what, name)
        if per_row:
            assert float(row_rel.max()) <= tol, (what, name, "per row")


@pytest.mark.parametrize("g", [1, 2, 4])
def test_bwd_fp32_inputs(kata, orc, g):
    log(f"case bwd fp32 tiny B1 H2 T256 d16 dv16 C32 g={g}")
    inp = workloads.make_inputs("tiny_f32")
    dout = _dout(inp["v"].shape, 7 + g)
    ref = orc.bwd_mg(inp["q"], inp["k"], inp["v"], dout, g)
    # the backward alone (o from the oracle), then forward + backward on the GPU
    o_ref = orc.fwd_mg(inp["q"], inp["k"], inp["v"], g)
    _check_f32(_gpu_bwd(kata, inp, "f32", dout, 32, g, out=o_ref), ref, f"g{g} bwd")
    _check_f32(_gpu_bwd(kata, inp, "f32", dout, 32, g), ref, f"g{g} fwd+bwd")


def test_bwd_one_token(kata, orc):
    # T = 1: o_0 = v_0, so dv_0 = dout_0 and dq_0 = dk_0 = 0 exactly; the GPU
    # values are rounding residues of <dout, v_0 - o_0> / D_0 with D_0 = (q.k)^2
    log("case bwd one token B1 H2 T1 d64 C64 bf16")
    inp = workloads.make_inputs("mid_bf16", B=1, H=2, T=1)
    dout = _dout(inp["v"].shape, 41)
    o_ref = orc.fwd(inp["q"], inp["k"], inp["v"])
    dq, dk, dv = _gpu_bwd(kata, inp, "bf16", dout, 64, 1, out=o_ref)
    # dv_0 = w_00 a_0 with w_00 and a_0 each rounded to bf16 once
    assert np.allclose(dv, dout, rtol=1.25 * U2, atol=1e-6)
    D = np.einsum("bhtd,bhtd->bht", inp["q"], inp["k"]) ** 2
    # a_0 and b_0 enter <a_0, v_0> + b_0 as bf16 pairs hi + lo (within 2^-16
    # relative), so the cancelling sum leaves about 2 x 2^-16 of |a| |v|
    scale = 4e-5 * np.abs(dout).sum(-1) * np.abs(inp["v"]).sum(-1) / D
    for g_ in (dq, dk):
        assert np.all(np.linalg.norm(g_, axis=-1) <= scale * 2 * np.sqrt(D) + 1e-6)


@pytest.mark.parametrize("T", [2, 63, 64, 65, 300, 1025, 2100])
def test_bwd_ragged_m1(kata, orc, T):
    log(f"case bwd M1 bf16 inputs B1 H2 T{T} d64 dv64 C64")
    inp = workloads.make_inputs("mid_bf16", B=1, H=2, T=T)
    dout = _dout(inp["v"].shape, 11)
    ref = orc.bwd_mg(inp["q"], inp["k"], inp["v"], dout, 1)
    o_ref = orc.fwd(inp["q"], inp["k"], inp["v"])
    _check_rel(_gpu_bwd(kata, inp, "bf16", dout, 64, 1, out=o_ref), ref, f"T{T} bwd",
               tol=BF16_GRAD_REL)
    _check_rel(_gpu_bwd(kata, inp, "bf16", dout, 64, 1), ref, f"T{T} fwd+bwd", per_row=False)


@pytest.mark.parametrize("B,H,T", [(2, 16, 333), (3, 6, 130), (2, 8, 200), (1, 40, 64),
                                   (16, 1, 37)])
def test_bwd_fused_state_scan(kata, orc, B, H, T):
    # From 16 heads on, the bf16 path computes each record stream (prefix of the
    # forward states, suffix of the backward states) in one launch that walks a
    # head's chunks in order; with fewer heads it runs the chunk-parallel state
    # launch and a scan.  B x H = 32, 18 (not a multiple of the 8 heads a
    # workgroup row spans), 16 (the smallest fused count), 40 with a single
    # chunk and 16 batches of one head with one partial chunk; against the
    # oracle, and
    # against the same heads run one at a time (the other path).
    import torch
    log(f"case bwd fused state+scan bf16 B{B} H{H} T{T} d64 dv64 C64")
    inp = workloads.make_inputs("mid_bf16", B=B, H=H, T=T)
    dout = _dout(inp["v"].shape, 41 + H)
    ref = orc.bwd_mg(inp["q"], inp["k"], inp["v"], dout, 1)
    o_ref = orc.fwd(inp["q"], inp["k"], inp["v"])
    got = _gpu_bwd(kata, inp, "bf16", dout, 64, 1, out=o_ref)
    _check_rel(got, ref, f"B{B} H{H} T{T} bwd", tol=BF16_GRAD_REL)
    q, k, v = (to_device(inp[n], "bf16") for n in ("q_dev", "k_dev", "v_dev"))
    out = torch.from_numpy(np.ascontiguousarray(o_ref, dtype=np.float32)).to(q.device)
    d_out = torch.from_numpy(dout).to(q.device)
    for b, h in ((0, 0), (B - 1, H - 1)):
        one = kata.bwd_chunked(*(x[b:b + 1, h:h + 1].contiguous() for x in (q, k, v, out, d_out)),
                               64, 1)
        torch.cuda.synchronize()
        for name, a, g_ in zip(("dq", "dk", "dv"), one, got):
            a = a.cpu().numpy()[0, 0].astype(np.float64)
            g_ = g_[b, h].astype(np.float64)
            rel = np.linalg.norm(a - g_) / max(np.linalg.norm(g_), 1e-30)
            log(f"  head ({b}, {h}) {name}: fused vs per-head rel l2 {rel:.3e}")
            assert rel <= BF16_GRAD_REL, (b, h, name)


def test_bwd_bench_configuration_sampled_heads(kata, orc):
    # the training step's own shape (the mid workload, B8 H16 T4096, 128 heads:
    # the fused state+scan path) against the oracle on three heads; those
    # heads get the exact forward output, so the per-row bound applies
    import torch
    w = workloads.WORKLOADS["mid_bf16"]
    log(f"case bwd bench configuration B{w.B} H{w.H} T{w.T} d64 C64, heads 0, 77, 127")
    assert kata.bwd_fused_scan(w.B, w.H, w.T, 64, 64, 64, 1, kata.KATA_BF16) == 1
    inp = workloads.make_inputs("mid_bf16")
    q, k, v = (to_device(inp[n], "bf16") for n in ("q_dev", "k_dev", "v_dev"))
    out = kata.fwd_chunked(q, k, v, 64)
    dout = _dout(inp["v"].shape, 47)
    heads = [0, 77, w.B * w.H - 1]
    sel = lambda x, bh: x.reshape(w.B * w.H, w.T, x.shape[-1])[bh][None, None]
    o_ex = {bh: orc.fwd(sel(inp["q"], bh), sel(inp["k"], bh), sel(inp["v"], bh)) for bh in heads}
    out_flat = out.view(w.B * w.H, w.T, 64)
    for bh in heads:
        out_flat[bh] = torch.from_numpy(np.ascontiguousarray(o_ex[bh][0, 0], dtype=np.float32)).to(
            out.device)
    d_out = torch.from_numpy(dout).to(q.device)
    got = kata.bwd_chunked(q, k, v, out, d_out, 64, 1)
    torch.cuda.synchronize()
    got = [g_.cpu().numpy() for g_ in got]
    for bh in heads:
        ref = orc.bwd_mg(sel(inp["q"], bh), sel(inp["k"], bh), sel(inp["v"], bh), sel(dout, bh), 1)
        mine = tuple(sel(g_, bh) for g_ in got)
        _check_rel(mine, ref, f"head {bh} bwd", tol=BF16_GRAD_REL)


def test_bwd_fused_long_against_chunk_parallel(kata):
    # 16 heads of 16421 tokens (257 chunks, the last one 37 tokens): the fused
    # state+scan walk over many chunks against the chunk-parallel states and
    # the blocked scan (the same heads run one at a time), on the same forward
    # output; the two differ only in where the chunk states are rounded
    import torch
    B, H, T = 1, 16, 16384 + 37
    log(f"case bwd fused vs chunk-parallel bf16 B{B} H{H} T{T} d64 C64")
    assert kata.bwd_fused_scan(B, H, T, 64, 64, 64, 1, kata.KATA_BF16) == 1
    assert kata.bwd_fused_scan(1, 1, T, 64, 64, 64, 1, kata.KATA_BF16) == 0
    inp = workloads.make_inputs("mid_bf16", B=B, H=H, T=T)
    q, k, v = (to_device(inp[n], "bf16") for n in ("q_dev", "k_dev", "v_dev"))
    out = kata.fwd_chunked(q, k, v, 64)
    d_out = torch.from_numpy(_dout(inp["v"].shape, 43)).to(q.device)
    got = kata.bwd_chunked(q, k, v, out, d_out, 64, 1)
    torch.cuda.synchronize()
    for h in (0, 7, 15):
        one = kata.bwd_chunked(*(x[:, h:h + 1].contiguous() for x in (q, k, v, out, d_out)), 64, 1)
        torch.cuda.synchronize()
        for name, a, g_ in zip(("dq", "dk", "dv"), one, got):
            a = a[0, 0].double()
            b = g_[0, h].double()
            assert torch.isfinite(b).all(), (h, name)
            rel = float((a - b).norm() / max(float(b.norm()), 1e-30))
            log(f"  head {h} {name}: fused vs chunk-parallel rel l2 {rel:.3e}")
            assert rel <= BF16_GRAD_REL, (h, name)


@pytest.mark.parametrize("C,g", [(16, 1), (32, 1), (48, 2), (64, 2), (64, 4)])
def test_bwd_chunks_and_blocks(kata, orc, C, g):
    T = 700
    log(f"case bwd bf16 inputs B2 H1 T{T} d64 dv64 C{C} g={g}")
    inp = workloads.make_inputs("mid_bf16", B=2, H=1, T=T)
    dout = _dout(inp["v"].shape, 13 + C + g)
    ref = orc.bwd_mg(inp["q"], inp["k"], inp["v"], dout, g)
    o_ref = orc.fwd_mg(inp["q"], inp["k"], inp["v"], g)
    _check_rel(_gpu_bwd(kata, inp, "bf16", dout, C, g, out=o_ref), ref, f"C{C} g{g} bwd",
               tol=BF16_GRAD_REL if _bf_path(64, 64, C, g) else F32_GRAD_REL)
    _check_rel(_gpu_bwd(kata, inp, "bf16", dout, C, g, fwd_C=64), ref, f"C{C} g{g} fwd+bwd",
               per_row=False)


def test_bwd_value_width_and_recall(kata, orc):
    # dv != d on the fp32 path, and the recall-shaped inputs (d = 32, C = 64)
    log("case bwd fp32 inputs d24 dv40 C24 B1 H2 T333")
    rng = np.random.default_rng(17)
    q = rng.standard_normal((1, 2, 333, 24)).astype(np.float32)
    k = rng.standard_normal((1, 2, 333, 24)).astype(np.float32)
    v = rng.standard_normal((1, 2, 333, 40)).astype(np.float32)
    dout = _dout(v.shape, 19)
    inp = dict(q_dev=q, k_dev=k, v_dev=v)
    ref = orc.bwd_mg(q, k, v, dout, 3)
    _check_f32(_gpu_bwd(kata, inp, "f32", dout, 24, 3, out=orc.fwd_mg(q, k, v, 3)), ref,
               "d24 dv40 g3 bwd")
    # dv > 64 takes the VALU kernels (the matrix-core variants stage 64 columns)
    log("case bwd fp32 inputs d16 dv96 C40 B1 H2 T301 (VALU kernels)")
    q = rng.standard_normal((1, 2, 301, 16)).astype(np.float32)
    k = rng.standard_normal((1, 2, 301, 16)).astype(np.float32)
    v = rng.standard_normal((1, 2, 301, 96)).astype(np.float32)
    dout = _dout(v.shape, 21)
    inp = dict(q_dev=q, k_dev=k, v_dev=v)
    ref = orc.bwd_mg(q, k, v, dout, 2)
    _check_f32(_gpu_bwd(kata, inp, "f32", dout, 40, 2, out=orc.fwd_mg(q, k, v, 2)), ref,
               "d16 dv96 g2 bwd")
    log("case bwd recall-shaped bf16 B1 H2 T1500 d32 dv64 C64")
    inp = workloads.make_inputs("recall_bf16", B=1, H=2, T=1500)
    dout = _dout(inp["v"].shape, 23)
    ref = orc.bwd_mg(inp["q"], inp["k"], inp["v"], dout, 1)
    _check_rel(_gpu_bwd(kata, inp, "bf16", dout, 64, 1, out=orc.fwd(inp["q"], inp["k"], inp["v"])),
               ref, "recall bwd", tol=F32_GRAD_REL)
    _check_rel(_gpu_bwd(kata, inp, "bf16", dout, 64, 1, fwd_C=128), ref, "recall fwd+bwd",
               per_row=False)


def test_bwd_zero_denominator(kata, orc):
    import torch
    log("case bwd zero query rows B1 H1 T200 d16 dv16 C32 fp32")
    inp = dict(workloads.make_inputs("tiny_f32", B=1, H=1, T=200))
    q = inp["q_dev"].copy()
    q[:, :, [0, 77, 199]] = 0.0
    inp["q_dev"] = q
    dout = _dout(inp["v"].shape, 29)
    got = _gpu_bwd(kata, inp, "f32", dout, 32, 1)
    for t in (0, 77, 199):
        assert np.array_equal(got[0][:, :, t], np.zeros_like(got[0][:, :, t]))
    ref = orc.bwd_mg(q, inp["k"], inp["v"], dout, 1)
    _check_f32(got, ref, "zero rows")
    torch.cuda.synchronize()


def test_bwd_entry_points_match(kata):
    import torch
    log("case bwd ws vs timed vs alloc, bf16 B1 H3 T900 d64 C64")
    inp = workloads.make_inputs("mid_bf16", B=1, H=3, T=900)
    q, k, v = (to_device(inp[n], "bf16") for n in ("q_dev", "k_dev", "v_dev"))
    out = kata.fwd_chunked(q, k, v, 64)
    dout = torch.from_numpy(_dout(inp["v"].shape, 31)).to(q.device)
    a = kata.bwd_chunked(q, k, v, out, dout, 64)
    hip = ctypes.CDLL("libamdhip64.so")
    vp = ctypes.c_void_p
    hip.hipEventCreate.argtypes = [ctypes.POINTER(vp)]
    hip.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), vp, vp]
    hip.hipEventDestroy.argtypes = [vp]
    evs = (vp * 7)()
    for i in range(7):
        h = vp()
        assert hip.hipEventCreate(ctypes.byref(h)) == 0
        evs[i] = h
    b = kata.bwd_chunked(q, k, v, out, dout, 64, events=evs)
    c = kata.bwd_chunked_alloc(q, k, v, out, dout, 64)
    torch.cuda.synchronize()
    for x, y, z in zip(a, b, c):
        assert torch.equal(x, y) and torch.equal(x, z)
    for i in range(6):
        ms = ctypes.c_float()
        assert hip.hipEventElapsedTime(ctypes.byref(ms), evs[i], evs[i + 1]) == 0
        assert ms.value >= 0.0
    for i in range(7):
        hip.hipEventDestroy(evs[i])


def test_bwd_full_length_two_heads(kata, orc):
    # the mid workload's full sequence (T = 4096, d = 64, C = 64) on two of its
    # heads, forward on the MFMA path and backward, against the oracle
    log("case bwd mid workload shape T4096 d64 C64, heads 0..1 (B1 H2)")
    inp = workloads.make_inputs("mid_bf16", B=1, H=2)
    dout = _dout(inp["v"].shape, 37)
    ref = orc.bwd_mg(inp["q"], inp["k"], inp["v"], dout, 1)
    got = _gpu_bwd(kata, inp, "bf16", dout, 64, 1)
    _check_rel(got, ref, "T4096 fwd+bwd", per_row=False)
    # invariants, on the backward fed the exact forward output (q_t . dq_t equals
    # 2 <dout_t, o_t - o_given>, so it vanishes only for the exact o): the value
    # gradients sum to the output cotangents; q_t . dq_t = 0.  C = 32 runs the
    # fp32 gradients kernel (tight bounds), C = 64 the bf16 matrix-core one:
    # there each term w_ti a_t is off by at most 2^-7 and sum_i w_ti = D_t, so
    # |sum dv - sum dout| <= 2^-7 sum |dout| per column; q . dq, an exactly
    # cancelling sum of terms of size up to |q| |dq|, stays within 4 x 2^-7 of
    # |q| rms|dq| (measured 5e-3)
    o_ref = orc.fwd(inp["q"], inp["k"], inp["v"])
    q64 = inp["q"].astype(np.float64)
    for C in (32, 64):
        log(f"  invariants, C = {C}")
        ex = _gpu_bwd(kata, inp, "bf16", dout, C, 1, out=o_ref)
        bf = _bf_path(64, 64, C, 1)
        _check_rel(ex, ref, f"T4096 C{C} bwd", tol=BF16_GRAD_REL if bf else F32_GRAD_REL)
        qd = np.einsum("bhtd,bhtd->bht", q64, ex[0])
        if bf:
            dsum = np.abs(ex[2].sum(axis=2) - dout.sum(axis=2))
            assert np.all(dsum <= U2 * np.abs(dout).sum(axis=2))
            rms = np.sqrt((ex[0].astype(np.float64) ** 2).sum(-1).mean(-1, keepdims=True))
            assert np.all(np.abs(qd) <= 4 * U2 * np.linalg.norm(q64, axis=-1) * rms)
        else:
            assert np.allclose(ex[2].sum(axis=2), dout.sum(axis=2), rtol=1e-4, atol=1e-3)
            scale = np.linalg.norm(ex[0], axis=-1) * np.linalg.norm(inp["q"], axis=-1)
            assert np.all(np.abs(qd) <= 1e-4 * scale + 1e-5)



# ---------------------------------------------------------------------------
# The training pair: a forward that saves the denominators D_t
# (kata_fwd_chunked_train_ws) and the backward that takes them
# (kata_bwd_chunked_ex) instead of forming D_t again from the prefix states.
# The forward's D_t carries the bf16 rounding of the prefix records (Z_pre),
# so it is held to the bf16 bound 2e-2 against the oracle's denominators (rows
# with D_t at least 1e-6 of the head's largest); the gradients, of the
# library's own forward output, to the per-head bound.
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("B,H,T", [(1, 16, 1100), (1, 2, 700), (2, 3, 257), (1, 16, 4096),
                                   (1, 2, 1), (1, 3, 63)])
def test_bwd_with_saved_denominators(kata, orc, B, H, T):
    import torch
    fused = kata.bwd_fused_scan(B, H, T, 64, 64, 64, 1, kata.KATA_BF16)
    log(f"case train forward + backward with saved D_t: B{B} H{H} T{T} d64 C64 "
        f"(state and scan fused: {fused})")
    inp = workloads.make_inputs("mid_bf16", B=B, H=H, T=T)
    q, k, v = (to_device(inp[n], "bf16") for n in ("q_dev", "k_dev", "v_dev"))
    out, den = kata.fwd_chunked_train(q, k, v, 64)
    plain = kata.fwd_chunked(q, k, v, 64)
    torch.cuda.synchronize()
    assert torch.equal(out, plain), "the training forward's output differs from the plain forward"
    got_den = den.cpu().numpy().astype(np.float64)
    ref_den = orc.den(inp["q"], inp["k"])
    scale = np.max(ref_den, axis=2, keepdims=True)
    live = ref_den >= 1e-6 * scale
    rel = np.abs(got_den - ref_den)[live] / ref_den[live]
    log(f"  D_t: max rel err {float(rel.max()):.3e} over {int(live.sum())} rows (tol {BF16_REL:.0e})")
    assert np.all(np.isfinite(got_den)) and float(rel.max()) <= BF16_REL
    dout = _dout(inp["v"].shape, 31 + T)
    d_out = torch.from_numpy(dout).to(q.device)
    got = [t.cpu().numpy() for t in kata.bwd_chunked(q, k, v, out, d_out, 64, den=den)]
    if T == 1:
        # o_0 = v_0, dv_0 = dout_0 (w_00 a_0, each rounded to bf16 once); the
        # exact dq_0 = dk_0 = 0 leave only residues of the forward's rounding
        # of o_0, which no relative bound holds (see _check_rel)
        assert np.allclose(got[2], dout, rtol=1.25 * U2, atol=1e-6)
        return
    if B * H * T <= 20000:
        ref = orc.bwd_mg(inp["q"], inp["k"], inp["v"], dout, 1)
        _check_rel(got, ref, f"saved D_t B{B} H{H} T{T}", per_row=False)
    # against the backward that forms D_t itself (same library forward output)
    own = [t.cpu().numpy() for t in kata.bwd_chunked(q, k, v, out, d_out, 64)]
    _check_rel(got, [o.astype(np.float64) for o in own], f"saved vs recomputed D_t T{T}",
               per_row=False)


@pytest.mark.parametrize("span", [0, 1])
def test_train_forward_d32_denominators(kata, orc, span):
    # d = 32 (recall inputs, C = 128): the training forward's output equals the
    # plain forward's and its denominators match the oracle's
    import torch
    B, H, T = 1, 3, 3000
    log(f"case train forward d32 B{B} H{H} T{T} C128 span_chunks={span}")
    inp = workloads.make_inputs("recall_bf16", B=B, H=H, T=T)
    q, k, v = (to_device(inp[n], "bf16") for n in ("q_dev", "k_dev", "v_dev"))
    out, den = kata.fwd_chunked_train(q, k, v, 128, span_chunks=span)
    plain = kata.fwd_chunked(q, k, v, 128, span_chunks=span)
    torch.cuda.synchronize()
    assert torch.equal(out, plain)
    got = den.cpu().numpy().astype(np.float64)
    ref = orc.den(inp["q"], inp["k"])
    live = ref >= 1e-6 * np.max(ref, axis=2, keepdims=True)
    rel = np.abs(got - ref)[live] / ref[live]
    log(f"  D_t: max rel err {float(rel.max()):.3e} (tol {BF16_REL:.0e})")
    assert np.all(np.isfinite(got)) and float(rel.max()) <= BF16_REL
