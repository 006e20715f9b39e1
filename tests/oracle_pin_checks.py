"""Checks that pin the CPU oracle to facts the paper and the mathematics fix.

Each ``pin_*`` function takes an ``oracle.Oracle`` and raises AssertionError
when the oracle disagrees with the fact it checks.  None of them re-types the
oracle's formula: they compare against closed forms, invariants, a
hand-computed example, brute force in a different feature space (unpacked
d*d features) or library routines.  The same functions run against planted
mutants of the oracle in test_oracle_mutants.py, to show that a plausible
mistake anywhere in the oracle fails at least one of them.
"""
from __future__ import annotations

import json
import math
import os

import numpy as np

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _rng(seed=1234):
    return np.random.default_rng(seed)


def _rand_qkv(rng, B, H, T, d, dv, unit=True):
    q = rng.standard_normal((B, H, T, d))
    k = rng.standard_normal((B, H, T, d))
    if unit:
        q /= np.linalg.norm(q, axis=-1, keepdims=True)
        k /= np.linalg.norm(k, axis=-1, keepdims=True)
    v = rng.standard_normal((B, H, T, dv))
    return q, k, v


def _brute_unpacked(q, k, v):
    """Forward in the unpacked feature space: phi(x) = vec(x x^T) in R^{d^2},
    scores = Phi(Q) Phi(K)^T with a lower-triangular mask (diagonal kept),
    O = (P V) / (P 1).  numpy only; a different route from the oracle's
    (q.k)^2 loop."""
    B, H, T, d = q.shape
    out = np.zeros(v.shape)
    mask = np.tril(np.ones((T, T)))
    for b in range(B):
        for h in range(H):
            PQ = np.einsum("ta,tb->tab", q[b, h], q[b, h]).reshape(T, d * d)
            PK = np.einsum("ta,tb->tab", k[b, h], k[b, h]).reshape(T, d * d)
            P = (PQ @ PK.T) * mask
            D = P.sum(axis=1, keepdims=True)
            N = P @ v[b, h]
            out[b, h] = np.where(D > 0, N / np.where(D > 0, D, 1.0), 0.0)
    return out


# ---------------------------------------------------------------------------
# PIN: packed feature map, sizes
# ---------------------------------------------------------------------------

def pin_packed_sizes(orc):
    # Widths printed in the paper: d=64 gives d^2 = 4096 direct and 2080 packed.
    assert orc.packed_dim(64) == 2080 and 64 * 64 == 4096
    # KATA-M1 state of the MQAR table: 2 layers x n x dv = 266,240 at d = dv = 64.
    assert 2 * orc.packed_dim(64) * 64 == 266240
    # KATA-M2 (two 32-dim blocks): 2 layers x 2 blocks x 528 x 64 = 135,168.
    assert 2 * 2 * orc.packed_dim(32) * 64 == 135168
    for d in (1, 2, 3, 16, 32):
        assert orc.packed_dim(d) == d * (d + 1) // 2


def pin_packed_order(orc):
    # Row-major upper triangle: numpy's triu_indices enumerates exactly that order.
    for d in (1, 2, 5, 16):
        ia, ib = np.triu_indices(d)
        got = [orc.packed_index(int(a), int(b), d) for a, b in zip(ia, ib)]
        assert got == list(range(len(ia)))
        # unordered pair
        assert all(orc.packed_index(int(b), int(a), d) == orc.packed_index(int(a), int(b), d)
                   for a, b in zip(ia, ib))
        # phi lays out x_a x_b in that order
        x = _rng(d).standard_normal(d)
        assert np.array_equal(orc.phi(x), np.outer(x, x)[ia, ib])


def pin_phi_identity(orc):
    # <phi_w(q), phi(k)> = <q q^T, k k^T>_F = (q . k)^2
    rng = _rng(7)
    for d in (1, 2, 3, 8, 16, 64):
        for _ in range(5):
            q = rng.standard_normal(d)
            k = rng.standard_normal(d)
            packed = float(orc.phi(q, weighted=True) @ orc.phi(k))
            unpacked = float(np.outer(q, q).ravel() @ np.outer(k, k).ravel())
            gram = float(q @ np.outer(k, k) @ q)
            ref = float(np.dot(q, k)) ** 2
            scale = max(1.0, abs(ref))
            assert abs(packed - ref) <= 1e-13 * scale
            assert abs(unpacked - ref) <= 1e-13 * scale
            assert abs(gram - ref) <= 1e-13 * scale


# ---------------------------------------------------------------------------
# PIN: hand-computed worked example
# ---------------------------------------------------------------------------

def pin_worked_example(orc):
    with open(os.path.join(GOLDEN, "worked_example_d2.json")) as f:
        g = json.load(f)
    K = np.array(g["keys"])[None, None]
    V = np.array(g["values"])[None, None]
    Q = np.array(g["queries"])[None, None]
    out = orc.fwd(Q, K, V)[0, 0]
    assert np.allclose(out, np.array(g["outputs"]), rtol=0, atol=1e-15)
    S, z = orc.state(K[:, :, :2], V[:, :, :2])
    assert np.allclose(S[0, 0], np.array(g["state_after_2"]["S"]), atol=1e-15)
    assert np.allclose(z[0, 0], np.array(g["state_after_2"]["z"]), atol=1e-15)
    q11 = np.array(g["query_11_at_3"]["q"])
    Q2 = Q.copy()
    Q2[0, 0, 2] = q11
    o = orc.fwd(Q2, K, V)[0, 0, 2, 0]
    assert abs(o - g["query_11_at_3"]["output"]) <= 1e-15
    # the same through the decode recurrence: state after 2 tokens, then step 3
    out3, S3, z3 = orc.decode_step(S, z, q11[None, None], K[:, :, 2], V[:, :, 2])
    assert abs(out3[0, 0, 0] - g["query_11_at_3"]["output"]) <= 1e-15
    assert abs(float(orc.phi(q11, weighted=True) @ S3[0, 0][:, 0]) - g["query_11_at_3"]["N"]) <= 1e-14
    assert abs(float(orc.phi(q11, weighted=True) @ z3[0, 0]) - g["query_11_at_3"]["D"]) <= 1e-14


# ---------------------------------------------------------------------------
# PIN: brute force in unpacked feature space
# ---------------------------------------------------------------------------

def pin_brute_force_unpacked(orc):
    rng = _rng(11)
    for (B, H, T, d, dv, unit) in [(1, 2, 13, 3, 2, True), (2, 1, 9, 8, 5, False),
                                   (1, 1, 1, 4, 3, True), (1, 1, 24, 2, 1, False)]:
        q, k, v = _rand_qkv(rng, B, H, T, d, dv, unit)
        ref = _brute_unpacked(q, k, v)
        got = orc.fwd(q, k, v)
        assert np.allclose(got, ref, rtol=1e-12, atol=1e-12)


# ---------------------------------------------------------------------------
# PIN: output-gate proposition (convex weights, t = 1, gate recursion)
# ---------------------------------------------------------------------------

def pin_convex_hull(orc):
    rng = _rng(3)
    q, k, v = _rand_qkv(rng, 1, 3, 40, 6, 4, unit=False)
    o = orc.fwd(q, k, v)
    lo = np.minimum.accumulate(v, axis=2)
    hi = np.maximum.accumulate(v, axis=2)
    assert (o >= lo - 1e-12).all() and (o <= hi + 1e-12).all()
    # Weights are nonnegative, causal and sum to one: with one-hot values
    # (dv = T, v_i = e_i) each output row is the weight vector itself.
    T = 17
    q, k, _ = _rand_qkv(rng, 1, 1, T, 5, 1)
    w = orc.fwd(q, k, np.eye(T)[None, None])[0, 0]
    assert (w >= 0).all()
    assert np.allclose(w.sum(axis=1), 1.0, atol=1e-14)
    assert np.all(np.triu(w, 1) == 0.0)
    # constant values are reproduced exactly (up to rounding)
    o1 = orc.fwd(q, k, np.full((1, 1, T, 2), 3.25))
    assert np.allclose(o1, 3.25, atol=1e-14)


def pin_first_token(orc):
    # D_0 = 0, so the first output is the first value (alpha, beta) = (0, 1).
    rng = _rng(5)
    q, k, v = _rand_qkv(rng, 2, 2, 6, 4, 3)
    o = orc.fwd(q, k, v)
    assert np.allclose(o[:, :, 0], v[:, :, 0], rtol=0, atol=1e-15)


def pin_gate_recursion(orc):
    # o_t = alpha_t zbar_{t|t-1} + beta_t v_t,  alpha = D_{t-1}/D_t, beta = c_t/D_t,
    # with zbar = phi(q_t)^T S_{t-1} / D_{t-1} read from the state of tokens < t.
    rng = _rng(9)
    q, k, v = _rand_qkv(rng, 1, 1, 12, 5, 3)
    o = orc.fwd(q, k, v)[0, 0]
    for t in range(1, 12):
        S, z = orc.state(k[:, :, :t], v[:, :, :t])
        pq = orc.phi(q[0, 0, t], weighted=True)
        Dprev = float(pq @ z[0, 0])
        c = float(np.dot(q[0, 0, t], k[0, 0, t])) ** 2
        D = Dprev + c
        zbar = (pq @ S[0, 0]) / Dprev
        alpha, beta = Dprev / D, c / D
        assert alpha >= 0 and beta >= 0 and abs(alpha + beta - 1) < 1e-15
        assert np.allclose(o[t], alpha * zbar + beta * v[0, 0, t], rtol=1e-12, atol=1e-13)


def pin_zero_denominator(orc):
    # A zero query makes D_t = 0; the output row is defined as 0.
    rng = _rng(13)
    q, k, v = _rand_qkv(rng, 1, 1, 8, 4, 3)
    q[0, 0, 5] = 0.0
    o = orc.fwd(q, k, v)
    assert np.all(o[0, 0, 5] == 0.0)
    assert np.all(np.isfinite(o))
    oc = orc.fwd_chunked(q, k, v, 3, 1)
    assert np.all(oc[0, 0, 5] == 0.0)
    # the decode readout follows the same convention
    S, z = orc.state(k[:, :, :5], v[:, :, :5])
    out, _, _ = orc.decode_step(S, z, q[:, :, 5], k[:, :, 5], v[:, :, 5])
    assert np.all(out == 0.0)


# ---------------------------------------------------------------------------
# PIN: closed forms
# ---------------------------------------------------------------------------

def pin_identical_keys_running_mean(orc):
    rng = _rng(17)
    T, d, dv = 20, 6, 3
    kk = rng.standard_normal(d)
    k = np.tile(kk, (1, 1, T, 1))
    q = rng.standard_normal((1, 1, T, d))
    v = rng.standard_normal((1, 1, T, dv))
    o = orc.fwd(q, k, v)[0, 0]
    mean = np.cumsum(v[0, 0], axis=0) / np.arange(1, T + 1)[:, None]
    assert np.allclose(o, mean, rtol=1e-13, atol=1e-13)


def pin_orthonormal_keys_exact_recall(orc):
    # k_i = e_i (T <= d) and q_t = e_j with j <= t: only token j has nonzero
    # weight, so o_t = v_j exactly (orthogonal-value identity).
    d = 8
    T = 8
    k = np.eye(d)[None, None, :T]
    rng = _rng(19)
    v = rng.standard_normal((1, 1, T, 4))
    js = [0, 0, 1, 3, 2, 5, 6, 4]
    q = np.stack([np.eye(d)[j] for j in js])[None, None]
    o = orc.fwd(q, k, v)[0, 0]
    for t, j in enumerate(js):
        assert np.array_equal(o[t], v[0, 0, j])


def pin_weight_sample(orc):
    # Unit q and k at an angle of 0.1024 rad: the KATA weight is cos^2 = 0.9896
    # (four places, as printed).  Read back through two tokens: k_0 = q (weight 1),
    # k_1 at the angle, v_0 = 0, v_1 = 1, so o_1 = w / (1 + w).
    th = 0.1024
    q = np.array([1.0, 0.0])
    k0 = q.copy()
    k1 = np.array([math.cos(th), math.sin(th)])
    Q = np.stack([q, q])[None, None]
    K = np.stack([k0, k1])[None, None]
    V = np.array([[0.0], [1.0]])[None, None]
    o = orc.fwd(Q, K, V)[0, 0, 1, 0]
    w = o / (1.0 - o)
    assert round(w, 4) == 0.9896


# ---------------------------------------------------------------------------
# PIN: invariances (isometric invariance, phi(-x) = phi(x), value affinity)
# ---------------------------------------------------------------------------

def pin_invariances(orc):
    rng = _rng(23)
    q, k, v = _rand_qkv(rng, 1, 2, 15, 5, 3, unit=False)
    o = orc.fwd(q, k, v)
    sign = rng.choice([-1.0, 1.0], size=(1, 2, 15, 1))
    assert np.allclose(orc.fwd(q, k * sign, v), o, rtol=1e-12, atol=1e-12)
    alpha = rng.uniform(0.3, 3.0, size=(1, 2, 15, 1)) * sign
    assert np.allclose(orc.fwd(q * alpha, k, v), o, rtol=1e-12, atol=1e-12)
    U, _ = np.linalg.qr(rng.standard_normal((5, 5)))
    assert np.allclose(orc.fwd(q @ U.T, k @ U.T, v), o, rtol=1e-12, atol=1e-12)
    c = rng.standard_normal(3)
    assert np.allclose(orc.fwd(q, k, v + c), o + c, rtol=1e-12, atol=1e-12)
    A = rng.standard_normal((3, 4))
    assert np.allclose(orc.fwd(q, k, v @ A), o @ A, rtol=1e-12, atol=1e-12)


# ---------------------------------------------------------------------------
# PIN: chunked form = definition, tree scan = recurrence
# ---------------------------------------------------------------------------

def pin_chunked_equals_definition(orc):
    rng = _rng(29)
    B, H, T, d, dv = 1, 2, 37, 4, 3
    q, k, v = _rand_qkv(rng, B, H, T, d, dv, unit=False)
    ref = orc.fwd(q, k, v)
    for C in (1, 2, 3, 5, 7, 16, 32, T, T + 3):
        for mode in (0, 1):
            got = orc.fwd_chunked(q, k, v, C, mode)
            assert np.allclose(got, ref, rtol=1e-12, atol=1e-12), (C, mode)


def pin_scan_equals_recurrence(orc):
    rng = _rng(31)
    for N in (1, 2, 3, 5, 8, 13, 64, 2048):
        xi = rng.integers(-50, 50, size=(N, 7)).astype(np.float64)
        seq = orc.scan_exclusive(xi, 0)
        tree = orc.scan_exclusive(xi, 1)
        lib = np.cumsum(xi, axis=0) - xi        # exclusive prefix via numpy
        assert np.array_equal(seq, lib) and np.array_equal(tree, lib)
        assert np.all(seq[0] == 0) and np.all(tree[0] == 0)
        xr = rng.standard_normal((N, 5))
        ref = np.cumsum(xr, axis=0) - xr
        scale = np.maximum(1.0, np.abs(np.cumsum(np.abs(xr), axis=0)))
        assert np.all(np.abs(orc.scan_exclusive(xr, 1) - ref) <= 1e-13 * scale)
        assert np.all(np.abs(orc.scan_exclusive(xr, 0) - ref) <= 1e-13 * scale)


# ---------------------------------------------------------------------------
# PIN: decode recurrence = forward on the concatenated sequence
# ---------------------------------------------------------------------------

def pin_decode_equals_forward(orc):
    rng = _rng(37)
    B, H, P, steps, d, dv = 2, 2, 10, 6, 4, 3
    q, k, v = _rand_qkv(rng, B, H, P + steps, d, dv)
    ref = orc.fwd(q, k, v)
    S, z = orc.state(k[:, :, :P], v[:, :, :P])
    for s in range(steps):
        t = P + s
        out, S, z = orc.decode_step(S, z, q[:, :, t], k[:, :, t], v[:, :, t])
        assert np.allclose(out, ref[:, :, t], rtol=1e-12, atol=1e-13)
    S_all, z_all = orc.state(k, v)
    assert np.allclose(S, S_all, rtol=1e-12, atol=1e-12)
    assert np.allclose(z, z_all, rtol=1e-12, atol=1e-12)


def pin_rows_match_full(orc):
    rng = _rng(41)
    q, k, v = _rand_qkv(rng, 2, 3, 21, 4, 5)
    full = orc.fwd(q, k, v).reshape(6, 21, 5)
    bh = rng.integers(0, 6, size=30)
    tt = rng.integers(0, 21, size=30)
    rows = orc.fwd_rows(q, k, v, bh, tt)
    assert np.array_equal(rows, full[bh, tt])


# ---------------------------------------------------------------------------
# PIN: KATA-Mg, the block-diagonal PSD feature (section "From rank-one rays to
# low-rank PSD packing"): g blocks of m = d/g coordinates, weight
# sum_a (q_a . k_a)^2; g = 1 is KATA-M1
# ---------------------------------------------------------------------------

def _brute_unpacked_mg(q, k, v, g):
    """Forward with unpacked blockwise features, the concatenation over blocks
    of vec(u_a u_a^T) in R^(g m^2); numpy only, a different route from the
    oracle's per-block dot-product loop."""
    B, H, T, d = q.shape
    m = d // g
    out = np.zeros(v.shape)
    mask = np.tril(np.ones((T, T)))

    def feats(x):
        return np.concatenate([np.einsum("ta,tb->tab", x[:, a * m:(a + 1) * m],
                                         x[:, a * m:(a + 1) * m]).reshape(T, m * m)
                               for a in range(g)], axis=1)
    for b in range(B):
        for h in range(H):
            P = (feats(q[b, h]) @ feats(k[b, h]).T) * mask
            D = P.sum(axis=1, keepdims=True)
            N = P @ v[b, h]
            out[b, h] = np.where(D > 0, N / np.where(D > 0, D, 1.0), 0.0)
    return out


def pin_mg_widths(orc):
    # State sizes printed in the MQAR table (tab:mqar) at d_h = 64: KATA-M1
    # 266,240, KATA-M2 135,168, KATA-M4 69,632, each 2 x n_g x d_v (d_v = 64).
    for g, dims in ((1, 266240), (2, 135168), (4, 69632)):
        assert 2 * orc.packed_dim_mg(64, g) * 64 == dims
    # the paper's closed form of the state size: g m(m+1)/2 = d(d/g + 1)/2
    for d in (2, 4, 6, 8, 16, 32, 64):
        for g in range(1, d + 1):
            if d % g == 0:
                assert orc.packed_dim_mg(d, g) == d * (d // g + 1) // 2
    assert orc.packed_dim_mg(64, 1) == orc.packed_dim(64)


def pin_mg_phi(orc):
    rng = _rng(43)
    # layout: block a's packed M1 lift at offset a m(m+1)/2
    x = rng.standard_normal(12)
    for g in (1, 2, 3, 4, 6, 12):
        m = 12 // g
        ref = np.concatenate([orc.phi(x[a * m:(a + 1) * m]) for a in range(g)])
        assert np.array_equal(orc.phi_mg(x, g), ref)
    # <psi_w(q), psi(k)> = sum_a (q_a . k_a)^2, against unpacked block outer products
    for d, g in ((4, 2), (6, 3), (8, 2), (8, 4), (16, 2), (64, 2), (64, 4)):
        m = d // g
        for _ in range(4):
            q = rng.standard_normal(d)
            k = rng.standard_normal(d)
            packed = float(orc.phi_mg(q, g, weighted=True) @ orc.phi_mg(k, g))
            unpacked = sum(float(np.outer(q[a * m:(a + 1) * m], q[a * m:(a + 1) * m]).ravel()
                                 @ np.outer(k[a * m:(a + 1) * m], k[a * m:(a + 1) * m]).ravel())
                           for a in range(g))
            ref = sum(float(q[a * m:(a + 1) * m] @ k[a * m:(a + 1) * m]) ** 2 for a in range(g))
            scale = max(1.0, abs(ref))
            assert abs(packed - ref) <= 1e-13 * scale
            assert abs(unpacked - ref) <= 1e-13 * scale


def pin_mg_brute_force(orc):
    rng = _rng(47)
    q, k, v = _rand_qkv(rng, 2, 2, 19, 8, 3, unit=False)
    for g in (1, 2, 4, 8):
        assert np.allclose(orc.fwd_mg(q, k, v, g), _brute_unpacked_mg(q, k, v, g),
                           rtol=1e-11, atol=1e-12), g
    assert np.array_equal(orc.fwd_mg(q, k, v, 1), orc.fwd(q, k, v))


def pin_mg_special_cases(orc):
    rng = _rng(53)
    q, k, v = _rand_qkv(rng, 1, 2, 23, 8, 4, unit=False)
    # only the first block of the queries non-zero: the weight is (q_1 . k_1)^2,
    # i.e. KATA-M1 on the first block
    q1 = q.copy()
    q1[..., 4:] = 0.0
    assert np.allclose(orc.fwd_mg(q1, k, v, 2), orc.fwd(q[..., :4], k[..., :4], v),
                       rtol=1e-12, atol=1e-12)
    # g = d (m = 1): w = sum_i q_i^2 k_i^2, linear attention with the feature x -> x*x
    w = np.einsum("bhtd,bhsd->bhts", q * q, k * k) * np.tril(np.ones((23, 23)))
    ref = np.einsum("bhts,bhsj->bhtj", w, v) / w.sum(axis=-1, keepdims=True)
    assert np.allclose(orc.fwd_mg(q, k, v, 8), ref, rtol=1e-12, atol=1e-12)
    # permuting the blocks of q and k together, and rotating inside each block
    # (an isometry per block), leaves the output unchanged
    o = orc.fwd_mg(q, k, v, 2)
    perm = np.r_[4:8, 0:4]
    assert np.allclose(orc.fwd_mg(q[..., perm], k[..., perm], v, 2), o, rtol=1e-12, atol=1e-12)
    U1, _ = np.linalg.qr(rng.standard_normal((4, 4)))
    U2, _ = np.linalg.qr(rng.standard_normal((4, 4)))
    U = np.zeros((8, 8))
    U[:4, :4], U[4:, 4:] = U1, U2
    assert np.allclose(orc.fwd_mg(q @ U.T, k @ U.T, v, 2), o, rtol=1e-12, atol=1e-12)
    # a rotation that mixes the blocks does change it (the feature is not M1's)
    R, _ = np.linalg.qr(rng.standard_normal((8, 8)))
    assert not np.allclose(orc.fwd_mg(q @ R.T, k @ R.T, v, 2), o, rtol=1e-6, atol=1e-6)
    # convex combination of the values
    lo = np.minimum.accumulate(v, axis=2)
    hi = np.maximum.accumulate(v, axis=2)
    assert np.all(o >= lo - 1e-12) and np.all(o <= hi + 1e-12)


def pin_mg_chunked_equals_definition(orc):
    rng = _rng(59)
    q, k, v = _rand_qkv(rng, 1, 2, 33, 8, 3, unit=False)
    for g in (1, 2, 4):
        ref = orc.fwd_mg(q, k, v, g)
        for C in (1, 3, 8, 16, 33, 40):
            for mode in (0, 1):
                got = orc.fwd_chunked_mg(q, k, v, C, g, mode)
                assert np.allclose(got, ref, rtol=1e-12, atol=1e-12), (g, C, mode)


def pin_mg_decode_equals_forward(orc):
    rng = _rng(61)
    B, H, P, steps, d, dv = 2, 2, 9, 5, 8, 3
    q, k, v = _rand_qkv(rng, B, H, P + steps, d, dv)
    for g in (2, 4):
        ref = orc.fwd_mg(q, k, v, g)
        S, z = orc.state_mg(k[:, :, :P], v[:, :, :P], g)
        for s in range(steps):
            t = P + s
            out, S, z = orc.decode_step_mg(S, z, q[:, :, t], k[:, :, t], v[:, :, t], g)
            assert np.allclose(out, ref[:, :, t], rtol=1e-12, atol=1e-13)
        S_all, z_all = orc.state_mg(k, v, g)
        assert np.allclose(S, S_all, rtol=1e-12, atol=1e-12)
        assert np.allclose(z, z_all, rtol=1e-12, atol=1e-12)
    # g = 1 state is M1's
    S1, z1 = orc.state_mg(k, v, 1)
    S0, z0 = orc.state(k, v)
    assert np.array_equal(S1, S0) and np.array_equal(z1, z0)


def pin_mg_rows_match_full(orc):
    rng = _rng(67)
    q, k, v = _rand_qkv(rng, 2, 2, 17, 8, 5)
    full = orc.fwd_mg(q, k, v, 2).reshape(4, 17, 5)
    bh = rng.integers(0, 4, size=25)
    tt = rng.integers(0, 17, size=25)
    assert np.array_equal(orc.fwd_mg_rows(q, k, v, 2, bh, tt), full[bh, tt])


# ---------------------------------------------------------------------------
# PIN: linear (n_psi ~ d) features of normalised linear attention
# ---------------------------------------------------------------------------

LIN_IDENTITY, LIN_RELU, LIN_ELU, LIN_LORENTZ, LIN_LORENTZ_S = 0, 1, 2, 3, 4


def _lib_features(x, feature, eps):
    """Feature rows from library routines (torch's relu/elu, numpy's norm),
    independent of the oracle's scalar feature code; x: [T, d]."""
    import torch
    t = torch.from_numpy(np.ascontiguousarray(x))
    if feature == LIN_IDENTITY:
        return x.copy()
    if feature == LIN_RELU:
        return (torch.relu(t) + eps).numpy()
    if feature == LIN_ELU:
        return (torch.nn.functional.elu(t) + 1.0).numpy()
    if feature == LIN_LORENTZ:
        return np.concatenate([x, np.linalg.norm(x, axis=-1, keepdims=True)], axis=-1)
    y, s = x[:, :-1], x[:, -1:]
    return np.concatenate([y, np.linalg.norm(y, axis=-1, keepdims=True) * (1.0 + s * s)],
                          axis=-1)


def _brute_lin(q, k, v, feature, eps, normalize):
    """Matrix form: P = (Psi(Q) Psi(K)^T) .* tril, N = P V, D = P 1."""
    B, H, T, d = q.shape
    out = np.zeros(v.shape)
    mask = np.tril(np.ones((T, T)))
    for b in range(B):
        for h in range(H):
            P = (_lib_features(q[b, h], feature, eps) @ _lib_features(k[b, h], feature, eps).T) * mask
            N = P @ v[b, h]
            if not normalize:
                out[b, h] = N
                continue
            D = P.sum(axis=1, keepdims=True)
            out[b, h] = np.where(D > 0, N / np.where(D > 0, D, 1.0), 0.0)
    return out


def pin_lin_widths(orc):
    # n_psi printed for the orthant and Lorentz rows of the associative-scan
    # throughput table at d = 64 (the appendix Lorentz variant keeps d), and
    # d + 1 for the lift (y, ||y||) of section "Classical feature maps".
    for f in (LIN_IDENTITY, LIN_RELU, LIN_ELU, LIN_LORENTZ_S):
        assert orc.lin_dim(64, f) == 64
    assert orc.lin_dim(64, LIN_LORENTZ) == 65
    for d in (1, 2, 7, 32):
        assert orc.lin_dim(d, LIN_LORENTZ) == d + 1 and orc.lin_dim(d, LIN_RELU) == d


def pin_lin_features(orc):
    rng = _rng(71)
    for d in (1, 3, 8, 64):
        for _ in range(3):
            x = rng.standard_normal(d) * 2.0
            for f in (LIN_IDENTITY, LIN_RELU, LIN_ELU, LIN_LORENTZ, LIN_LORENTZ_S):
                if f == LIN_LORENTZ_S and d < 2:
                    continue
                got = orc.lin_feature(x, f, 1e-3)
                ref = _lib_features(x[None, :], f, 1e-3)[0]
                assert np.allclose(got, ref, rtol=1e-15, atol=1e-15), (d, f)
            # orthant maps land in the open positive orthant
            assert (orc.lin_feature(x, LIN_RELU, 1e-3) >= 1e-3).all()
            assert (orc.lin_feature(x, LIN_ELU) > 0).all()
    # the Lorentz lift: <psi(x), psi(y)> = <x, y> + ||x|| ||y|| >= 0, and for unit
    # vectors the halved kernel is 1/2 + z/2 (z = <x, y>), ||psi(x)||^2 = 2
    for _ in range(20):
        x = rng.standard_normal(9)
        y = rng.standard_normal(9)
        px, py = orc.lin_feature(x, LIN_LORENTZ), orc.lin_feature(y, LIN_LORENTZ)
        ref = x @ y + np.linalg.norm(x) * np.linalg.norm(y)
        assert abs(px @ py - ref) <= 1e-13 * max(1.0, abs(ref)) and px @ py >= -1e-13
        xu, yu = x / np.linalg.norm(x), y / np.linalg.norm(y)
        pxu, pyu = orc.lin_feature(xu, LIN_LORENTZ), orc.lin_feature(yu, LIN_LORENTZ)
        assert abs(0.5 * (pxu @ pyu) - (0.5 + 0.5 * (xu @ yu))) <= 1e-14
        assert abs(pxu @ pxu - 2.0) <= 1e-14
        # appendix variant: inside the closed cone t >= ||y||; s = 0 gives the lift of y
        ps = orc.lin_feature(x, LIN_LORENTZ_S)
        assert ps[-1] >= np.linalg.norm(x[:-1]) and ps @ orc.lin_feature(y, LIN_LORENTZ_S) >= 0
        x0 = x.copy()
        x0[-1] = 0.0
        assert np.array_equal(orc.lin_feature(x0, LIN_LORENTZ_S),
                              orc.lin_feature(x[:-1], LIN_LORENTZ))


def pin_lin_brute_force(orc):
    rng = _rng(73)
    q, k, v = _rand_qkv(rng, 2, 2, 21, 8, 5, unit=False)
    for f in (LIN_IDENTITY, LIN_RELU, LIN_ELU, LIN_LORENTZ, LIN_LORENTZ_S):
        for norm in ((False,) if f == LIN_IDENTITY else (True, False)):
            got = orc.lin_fwd(q, k, v, f, 0.05, norm)
            ref = _brute_lin(q, k, v, f, 0.05, norm)
            assert np.allclose(got, ref, rtol=1e-11, atol=1e-12), (f, norm)


def pin_lin_special_cases(orc):
    rng = _rng(79)
    T = 19
    q, k, v = _rand_qkv(rng, 1, 2, T, 6, 4, unit=True)
    tril = np.tril(np.ones((T, T)))
    # unnormalised identity feature: o = tril(Q K^T) V, bilinear in (q, v)
    ref = np.einsum("bhts,bhsj->bhtj", np.einsum("bhtd,bhsd->bhts", q, k) * tril, v)
    o = orc.lin_fwd(q, k, v, LIN_IDENTITY, 0.0, False)
    assert np.allclose(o, ref, rtol=1e-12, atol=1e-13)
    assert np.allclose(orc.lin_fwd(-2.5 * q, k, v, LIN_IDENTITY, 0.0, False), -2.5 * o,
                       rtol=1e-12, atol=1e-13)
    # Lorentz lift on unit vectors: the weight is 1 + <q, k> (section on the dense
    # associative memory hierarchy gives the halved kernel 1/2 + z/2)
    w = (1.0 + np.einsum("bhtd,bhsd->bhts", q, k)) * tril
    ref = np.einsum("bhts,bhsj->bhtj", w, v) / w.sum(axis=-1, keepdims=True)
    assert np.allclose(orc.lin_fwd(q, k, v, LIN_LORENTZ, 0.0, True), ref, rtol=1e-12, atol=1e-12)
    # positive features: the first output is v_0, every output lies in the
    # running hull of the values, identical keys give the running mean
    for f in (LIN_RELU, LIN_ELU, LIN_LORENTZ, LIN_LORENTZ_S):
        on = orc.lin_fwd(q, k, v, f, 1e-2, True)
        assert np.allclose(on[:, :, 0], v[:, :, 0], rtol=1e-13, atol=1e-14)
        lo = np.minimum.accumulate(v, axis=2)
        hi = np.maximum.accumulate(v, axis=2)
        assert np.all(on >= lo - 1e-12) and np.all(on <= hi + 1e-12)
        ks = np.broadcast_to(k[:, :, :1], k.shape)
        mean = np.cumsum(v, axis=2) / np.arange(1, T + 1)[None, None, :, None]
        assert np.allclose(orc.lin_fwd(q, ks, v, f, 1e-2, True), mean, rtol=1e-12, atol=1e-13)
    # positively homogeneous features (ReLU with eps = 0, the Lorentz lift): a
    # positive scale of q or k leaves the normalised output unchanged; a rotation
    # of both leaves the Lorentz output unchanged
    for f in (LIN_RELU, LIN_LORENTZ):
        base = orc.lin_fwd(q, k, v, f, 0.0, True)
        assert np.allclose(orc.lin_fwd(3.0 * q, 0.25 * k, v, f, 0.0, True), base,
                           rtol=1e-12, atol=1e-12)
    U, _ = np.linalg.qr(rng.standard_normal((6, 6)))
    base = orc.lin_fwd(q, k, v, LIN_LORENTZ, 0.0, True)
    assert np.allclose(orc.lin_fwd(q @ U.T, k @ U.T, v, LIN_LORENTZ, 0.0, True), base,
                       rtol=1e-12, atol=1e-12)
    # a query with no positive coordinate has a zero ReLU feature at eps = 0:
    # the denominator is 0 and the readout is 0
    qn = -np.abs(q)
    assert np.array_equal(orc.lin_fwd(qn, k, v, LIN_RELU, 0.0, True), np.zeros(v.shape))
    # ... while eps > 0 keeps it defined (a uniform-weight mean of the values only
    # when the keys have no positive coordinate either)
    kn = -np.abs(k)
    mean = np.cumsum(v, axis=2) / np.arange(1, T + 1)[None, None, :, None]
    assert np.allclose(orc.lin_fwd(qn, kn, v, LIN_RELU, 1e-3, True), mean, rtol=1e-12, atol=1e-13)


def pin_lin_chunked_equals_definition(orc):
    rng = _rng(83)
    q, k, v = _rand_qkv(rng, 1, 2, 29, 6, 3, unit=False)
    for f in (LIN_IDENTITY, LIN_RELU, LIN_ELU, LIN_LORENTZ, LIN_LORENTZ_S):
        norm = f != LIN_IDENTITY
        ref = orc.lin_fwd(q, k, v, f, 0.01, norm)
        for C in (1, 3, 8, 29, 40):
            for mode in (0, 1):
                got = orc.lin_fwd_chunked(q, k, v, C, f, 0.01, norm, mode)
                assert np.allclose(got, ref, rtol=1e-12, atol=1e-12), (f, C, mode)


def pin_lin_rows_match_full(orc):
    rng = _rng(89)
    q, k, v = _rand_qkv(rng, 2, 2, 15, 8, 5, unit=False)
    bh = rng.integers(0, 4, size=25)
    tt = rng.integers(0, 15, size=25)
    for f, norm in ((LIN_IDENTITY, False), (LIN_ELU, True), (LIN_LORENTZ, True)):
        full = orc.lin_fwd(q, k, v, f, 0.0, norm).reshape(4, 15, 5)
        assert np.array_equal(orc.lin_fwd_rows(q, k, v, f, 0.0, norm, bh, tt), full[bh, tt])


# ---------------------------------------------------------------------------
# PIN: backward (gradients of sum_t <dout_t, o_t>)
# ---------------------------------------------------------------------------

def _torch_grads(q, k, v, dout, g):
    """Gradients by torch autograd of a float64 matrix-form forward (scores
    (Q K^T)^2 summed over blocks, lower-triangular mask, row normalisation):
    a different route from the oracle's loops."""
    import torch
    B, H, T, d = q.shape
    m = d // g
    tq = torch.tensor(q, dtype=torch.float64, requires_grad=True)
    tk = torch.tensor(k, dtype=torch.float64, requires_grad=True)
    tv = torch.tensor(v, dtype=torch.float64, requires_grad=True)
    P = 0
    for a in range(g):
        sl = slice(a * m, (a + 1) * m)
        P = P + torch.matmul(tq[..., sl], tk[..., sl].transpose(-1, -2)) ** 2
    P = P * torch.tril(torch.ones(T, T, dtype=torch.float64))
    o = torch.matmul(P, tv) / P.sum(-1, keepdim=True)
    (o * torch.tensor(dout)).sum().backward()
    return tq.grad.numpy(), tk.grad.numpy(), tv.grad.numpy()


def pin_bwd_finite_differences(orc):
    rng = _rng(97)
    q, k, v = _rand_qkv(rng, 1, 1, 6, 4, 3, unit=False)
    dout = rng.standard_normal(v.shape)
    h = 1e-5
    for g in (1, 2):
        grads = orc.bwd_mg(q, k, v, dout, g)
        for idx, X in enumerate((q, k, v)):
            num = np.zeros_like(X)
            for ii in np.ndindex(X.shape):
                args = [q, k, v]
                Xp, Xm = X.copy(), X.copy()
                Xp[ii] += h
                Xm[ii] -= h
                args[idx] = Xp
                lp = float((orc.fwd_mg(*args, g) * dout).sum())
                args[idx] = Xm
                lm = float((orc.fwd_mg(*args, g) * dout).sum())
                num[ii] = (lp - lm) / (2 * h)
            assert np.allclose(grads[idx], num, rtol=1e-6, atol=1e-8), (g, idx)


def pin_bwd_torch_autograd(orc):
    rng = _rng(101)
    q, k, v = _rand_qkv(rng, 2, 2, 19, 8, 5, unit=False)
    dout = rng.standard_normal(v.shape)
    for g in (1, 2, 4):
        got = orc.bwd_mg(q, k, v, dout, g)
        ref = _torch_grads(q, k, v, dout, g)
        for a, b in zip(got, ref):
            assert np.allclose(a, b, rtol=1e-10, atol=1e-12), g
    # g = 1 through the M1 forward as well
    assert np.array_equal(orc.fwd_mg(q, k, v, 1), orc.fwd(q, k, v))


def pin_bwd_invariants(orc):
    rng = _rng(103)
    T = 17
    q, k, v = _rand_qkv(rng, 1, 2, T, 6, 4, unit=False)
    dout = rng.standard_normal(v.shape)
    for g in (1, 2, 3):
        dq, dk, dv = orc.bwd_mg(q, k, v, dout, g)
        # o(v + c) = o(v) + c: the value gradients sum to the output cotangents
        assert np.allclose(dv.sum(axis=2), dout.sum(axis=2), rtol=1e-12, atol=1e-12)
        # o_t is invariant to scaling q_t, and to scaling every key together
        assert np.allclose(np.einsum("bhtd,bhtd->bht", q, dq), 0.0, atol=1e-12)
        assert np.allclose(np.einsum("bhtd,bhtd->bh", k, dk), 0.0, atol=1e-11)
        # k -> -k leaves the forward unchanged: dk flips, dq and dv stay
        dq2, dk2, dv2 = orc.bwd_mg(q, -k, v, dout, g)
        assert np.allclose(dq2, dq, rtol=1e-12, atol=1e-13)
        assert np.allclose(dk2, -dk, rtol=1e-12, atol=1e-13)
        assert np.allclose(dv2, dv, rtol=1e-12, atol=1e-13)
    # one token: o_0 = v_0, so dv_0 = dout_0 and dq_0 = dk_0 = 0
    dq, dk, dv = orc.bwd_mg(q[:, :, :1], k[:, :, :1], v[:, :, :1], dout[:, :, :1], 1)
    assert np.allclose(dv, dout[:, :, :1], rtol=1e-14, atol=1e-15)
    assert np.allclose(dq, 0.0, atol=1e-14) and np.allclose(dk, 0.0, atol=1e-14)


def pin_bwd_zero_denominator(orc):
    # a zero query row has D_t = 0 and the constant readout 0: it passes no
    # gradient (its own dq is 0, and its dout changes nothing)
    rng = _rng(107)
    q, k, v = _rand_qkv(rng, 1, 1, 9, 4, 3, unit=False)
    q[:, :, 4] = 0.0
    dout = rng.standard_normal(v.shape)
    dq, dk, dv = orc.bwd_mg(q, k, v, dout, 1)
    assert np.array_equal(dq[:, :, 4], np.zeros_like(dq[:, :, 4]))
    dout2 = dout.copy()
    dout2[:, :, 4] += 10.0
    for a, b in zip(orc.bwd_mg(q, k, v, dout2, 1), (dq, dk, dv)):
        assert np.array_equal(a, b)


def pin_bwd_chunked_equals_definition(orc):
    rng = _rng(109)
    q, k, v = _rand_qkv(rng, 1, 2, 27, 8, 3, unit=False)
    dout = rng.standard_normal(v.shape)
    for g in (1, 2, 4):
        ref = orc.bwd_mg(q, k, v, dout, g)
        for C in (1, 3, 8, 27, 32):
            for mode in (0, 1):
                got = orc.bwd_chunked_mg(q, k, v, dout, C, g, mode)
                for a, b in zip(got, ref):
                    assert np.allclose(a, b, rtol=1e-11, atol=1e-12), (g, C, mode)


# ---------------------------------------------------------------------------
# PIN: row denominators (the normaliser of eq. linatt), against the unpacked
# feature space and closed forms
# ---------------------------------------------------------------------------
def pin_den(orc):
    rng = _rng(77)
    q, k, _ = _rand_qkv(rng, 1, 2, 9, 4, 3, unit=False)
    got = orc.den(q, k)
    for h in range(2):
        PQ = np.einsum("ta,tb->tab", q[0, h], q[0, h]).reshape(9, 16)
        PK = np.einsum("ta,tb->tab", k[0, h], k[0, h]).reshape(9, 16)
        P = (PQ @ PK.T) * np.tril(np.ones((9, 9)))
        assert np.allclose(got[0, h], P.sum(axis=1), rtol=1e-13, atol=1e-13)
    # one unit direction for every query and key: D_t = t + 1
    e = np.zeros((1, 1, 6, 5))
    e[..., 2] = 1.0
    assert np.array_equal(orc.den(e, e)[0, 0], np.arange(1.0, 7.0))
    # queries orthogonal to every key: D = 0
    qo = np.zeros((1, 1, 6, 5))
    qo[..., 0] = 1.0
    assert np.array_equal(orc.den(qo, e)[0, 0], np.zeros(6))


ALL_PINS = [
    pin_packed_sizes, pin_packed_order, pin_phi_identity, pin_worked_example,
    pin_brute_force_unpacked, pin_convex_hull, pin_first_token, pin_gate_recursion,
    pin_zero_denominator, pin_identical_keys_running_mean,
    pin_orthonormal_keys_exact_recall, pin_weight_sample, pin_invariances,
    pin_chunked_equals_definition, pin_scan_equals_recurrence,
    pin_decode_equals_forward, pin_rows_match_full, pin_den,
    pin_mg_widths, pin_mg_phi, pin_mg_brute_force, pin_mg_special_cases,
    pin_mg_chunked_equals_definition, pin_mg_decode_equals_forward, pin_mg_rows_match_full,
    pin_lin_widths, pin_lin_features, pin_lin_brute_force, pin_lin_special_cases,
    pin_lin_chunked_equals_definition, pin_lin_rows_match_full,
    pin_bwd_finite_differences, pin_bwd_torch_autograd, pin_bwd_invariants,
    pin_bwd_zero_denominator, pin_bwd_chunked_equals_definition,
]
