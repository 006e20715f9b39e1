"""HIP graph capture of the entry points that take caller-owned memory (the
forward with a workspace, the allocation-free forward, the quadratic form and
the backward): each call is captured once, and every replay, with eager work
and synchronisations between replays, must give the eager call's outputs bit
for bit (the same kernels on the same inputs).  Every case prints its name
and shape before it launches."""
from __future__ import annotations

import numpy as np
import pytest

import workloads
from gpu_helpers import log, to_device

pytestmark = pytest.mark.gpu

REPLAYS = 3


@pytest.fixture(scope="module")
def kata():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2607_17419_amd as k
    k.lib()  # raises if libkata.so is missing: no fallback
    return k


def _dev3(inp, dtype="bf16"):
    return tuple(to_device(inp[n], dtype) for n in ("q_dev", "k_dev", "v_dev"))


def _replay_and_check(graph, outs, refs, what):
    import torch
    for r in range(REPLAYS):
        for o in outs:
            o.fill_(float("nan"))  # eager work between replays
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for o, ref, name in zip(outs, refs, ("0", "1", "2")):
            got = o.cpu().numpy()
            assert np.array_equal(got, ref), f"{what}: replay {r} output {name} differs"


def _capture(fn):
    import torch
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        fn()  # warm-up on the capture stream's side
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        fn()
    torch.cuda.synchronize()
    return g


def test_forward_workspace_graph(kata):
    import torch
    B, H, T, C = 1, 4, 3000, 64
    log(f"case graph: kata_fwd_chunked_ws B{B} H{H} T{T} d64 C{C} (three spans, ragged)")
    q, k, v = _dev3(workloads.make_inputs("mid_bf16", B=B, H=H, T=T))
    ws = torch.empty(kata.workspace_bytes(B, H, T, 64, 64, C, kata.KATA_BF16), dtype=torch.uint8,
                     device="cuda:0")
    ref = kata.fwd_chunked(q, k, v, C, workspace=ws).cpu().numpy()
    out = torch.empty((B, H, T, 64), dtype=torch.float32, device="cuda:0")
    g = _capture(lambda: kata.fwd_chunked(q, k, v, C, out=out, workspace=ws))
    _replay_and_check(g, [out], [ref], "forward (workspace)")


def test_forward_noalloc_graph(kata):
    import torch
    B, H, T, C = 2, 2, 2100, 64
    log(f"case graph: kata_fwd_chunked_noalloc B{B} H{H} T{T} d64 C{C}")
    q, k, v = _dev3(workloads.make_inputs("mid_bf16", B=B, H=H, T=T))
    ref = kata.fwd_chunked_noalloc(q, k, v, C).cpu().numpy()
    out = torch.empty((B, H, T, 64), dtype=torch.float32, device="cuda:0")
    g = _capture(lambda: kata.fwd_chunked_noalloc(q, k, v, C, out=out))
    _replay_and_check(g, [out], [ref], "forward (no allocation)")


def test_quadratic_graph(kata):
    import torch
    B, H, T = 1, 3, 1500
    log(f"case graph: kata_fwd_quadratic_ws B{B} H{H} T{T} d32 (recall inputs)")
    q, k, v = _dev3(workloads.make_inputs("recall_bf16", B=B, H=H, T=T))
    ws = torch.empty(kata.quadratic_workspace_bytes(B, H, T, 32, 64, kata.KATA_BF16),
                     dtype=torch.uint8, device="cuda:0")
    ref = kata.fwd_quadratic(q, k, v, workspace=ws).cpu().numpy()
    out = torch.empty((B, H, T, 64), dtype=torch.float32, device="cuda:0")
    g = _capture(lambda: kata.fwd_quadratic(q, k, v, out=out, workspace=ws))
    _replay_and_check(g, [out], [ref], "quadratic form")


@pytest.mark.parametrize("H,T", [(16, 1100), (2, 700)])
def test_backward_graph(kata, H, T):
    import torch
    B, C = 1, 64
    fused = kata.bwd_fused_scan(B, H, T, 64, 64, C, 1, kata.KATA_BF16)
    log(f"case graph: kata_bwd_chunked_ws B{B} H{H} T{T} d64 C{C} (state and scan fused: {fused})")
    q, k, v = _dev3(workloads.make_inputs("mid_bf16", B=B, H=H, T=T))
    out = kata.fwd_chunked(q, k, v, C)
    gen = torch.Generator(device="cuda:0")
    gen.manual_seed(H * 1000 + T)
    dout = torch.randn(out.shape, device="cuda:0", generator=gen)
    ws = torch.empty(max(256, kata.bwd_workspace_bytes(B, H, T, 64, 64, C, 1, kata.KATA_BF16)),
                     dtype=torch.uint8, device="cuda:0")
    refs = [t.cpu().numpy() for t in kata.bwd_chunked(q, k, v, out, dout, C, workspace=ws)]
    grads = tuple(torch.empty_like(t) for t in (q.float(), k.float(), v.float()))
    g = _capture(lambda: kata.bwd_chunked(q, k, v, out, dout, C, workspace=ws, grads=grads))
    _replay_and_check(g, list(grads), refs, "backward")


def test_decode_step_graph(kata):
    # one decode step captured; each replay advances the state by that step,
    # so replay r must match the r-th of a run of eager steps on a copy
    import torch
    B, H, d, dv, T = 4, 3, 64, 64, 200
    log(f"case graph: kata_decode_step B{B} H{H} d{d} dv{dv} after a {T}-token prefill")
    inp = workloads.make_inputs("mid_bf16", B=B, H=H, T=T + 1)
    q, k, v = _dev3(inp)
    S0, z0 = kata.prefill_state(k[:, :, :T].contiguous(), v[:, :, :T].contiguous())
    qt, kt, vt = (x[:, :, T].contiguous() for x in (q, k, v))
    S_e, z_e = S0.clone(), z0.clone()
    refs = []
    for r in range(REPLAYS + 1):  # one step for the warm-up, then one per replay
        o = kata.decode_step(S_e, z_e, qt, kt, vt)
        refs.append((o.cpu().numpy(), S_e.cpu().numpy(), z_e.cpu().numpy()))
    S_g, z_g = S0.clone(), z0.clone()
    out = torch.empty((B, H, dv), dtype=torch.float32, device="cuda:0")
    g = _capture(lambda: kata.decode_step(S_g, z_g, qt, kt, vt, out=out))  # warm-up: step 0
    for r in range(REPLAYS):
        out.fill_(float("nan"))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        ro, rS, rz = refs[r + 1]
        assert np.array_equal(out.cpu().numpy(), ro), f"decode replay {r}: output differs"
        assert np.array_equal(S_g.cpu().numpy(), rS), f"decode replay {r}: S differs"
        assert np.array_equal(z_g.cpu().numpy(), rz), f"decode replay {r}: z differs"


def test_training_pair_graph(kata):
    # the forward that saves the denominators and the backward that takes
    # them, captured together as one training step
    import torch
    B, H, T, C = 1, 16, 1100, 64
    log(f"case graph: kata_fwd_chunked_train_ws + kata_bwd_chunked_ex B{B} H{H} T{T} d64 C{C}")
    q, k, v = _dev3(workloads.make_inputs("mid_bf16", B=B, H=H, T=T))
    gen = torch.Generator(device="cuda:0")
    gen.manual_seed(5)
    dout = torch.randn((B, H, T, 64), device="cuda:0", generator=gen)
    fws = torch.empty(kata.workspace_bytes(B, H, T, 64, 64, C, kata.KATA_BF16), dtype=torch.uint8,
                      device="cuda:0")
    bws = torch.empty(kata.bwd_workspace_bytes(B, H, T, 64, 64, C, 1, kata.KATA_BF16),
                      dtype=torch.uint8, device="cuda:0")
    out, den = kata.fwd_chunked_train(q, k, v, C, workspace=fws)
    grads = kata.bwd_chunked(q, k, v, out, dout, C, workspace=bws, den=den)
    refs = [t.cpu().numpy() for t in (out, den) + tuple(grads)]
    outs = [torch.empty_like(t) for t in (out, den) + tuple(grads)]

    def step():
        kata.fwd_chunked_train(q, k, v, C, out=outs[0], den=outs[1], workspace=fws)
        kata.bwd_chunked(q, k, v, outs[0], dout, C, workspace=bws, den=outs[1],
                         grads=tuple(outs[2:]))
    g = _capture(step)
    for r in range(REPLAYS):
        for o in outs:
            o.fill_(float("nan"))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for i, (o, ref) in enumerate(zip(outs, refs)):
            assert np.array_equal(o.cpu().numpy(), ref), f"training pair: replay {r} output {i} differs"


@pytest.mark.parametrize("feature", [0, 3])
def test_linear_features_graph(kata, feature):
    # linear features (identity / Lorentz lift) and KATA-M2, caller workspaces
    import torch
    B, H, T, C = 1, 4, 2500, 128
    log(f"case graph: kata_lin_fwd_chunked_ws feature {feature} B{B} H{H} T{T} d64 C{C}")
    q, k, v = _dev3(workloads.make_inputs("mid_bf16", B=B, H=H, T=T))
    ws = torch.empty(max(256, kata.lin_workspace_bytes(B, H, T, 64, 64, C, feature,
                                                       kata.KATA_BF16)),
                     dtype=torch.uint8, device="cuda:0")
    ref = kata.lin_fwd_chunked(q, k, v, C, feature, eps=1e-3, workspace=ws).cpu().numpy()
    out = torch.empty((B, H, T, 64), dtype=torch.float32, device="cuda:0")
    g = _capture(lambda: kata.lin_fwd_chunked(q, k, v, C, feature, eps=1e-3, out=out,
                                              workspace=ws))
    _replay_and_check(g, [out], [ref], f"linear feature {feature}")


def test_mg_graph(kata):
    import torch
    B, H, T, C = 1, 4, 2500, 64
    log(f"case graph: kata_mg_fwd_chunked_ws g2 B{B} H{H} T{T} d64 C{C}")
    q, k, v = _dev3(workloads.make_inputs("mid_bf16", B=B, H=H, T=T))
    ws = torch.empty(max(256, int(kata.lib().kata_mg_fwd_workspace_bytes(B, H, T, 64, 64, C, 2,
                                                                          kata.KATA_BF16, 0))),
                     dtype=torch.uint8, device="cuda:0")
    ref = kata.mg_fwd_chunked(q, k, v, C, 2, workspace=ws).cpu().numpy()
    out = torch.empty((B, H, T, 64), dtype=torch.float32, device="cuda:0")
    g = _capture(lambda: kata.mg_fwd_chunked(q, k, v, C, 2, out=out, workspace=ws))
    _replay_and_check(g, [out], [ref], "KATA-M2")
