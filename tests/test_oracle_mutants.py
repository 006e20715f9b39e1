"""Plant plausible mistakes in a copy of the oracle and check the pins catch each.

The mutants are built on the CPU from a temporary, textually edited copy of
oracle/kata_oracle.c; the committed oracle is never changed.
"""
import os
import tempfile

import pytest

import oracle
from oracle_pin_checks import ALL_PINS

SRC = os.path.join(os.path.dirname(oracle.__file__), "kata_oracle.c")

# (name, exact text in the oracle, replacement[, which occurrence: 0 = the
# first, in the KATA-M1 code; 1 = the second, in the KATA-Mg code after it;
# 2 = the third, in the linear-feature code])
MUTANTS = [
    ("drop_diagonal", "for (long i = 0; i <= t; ++i) {", "for (long i = 0; i < t; ++i) {"),
    ("den_drop_diagonal", "for (long i = 0; i <= t; ++i) {", "for (long i = 0; i < t; ++i) {", 5),
    ("den_not_squared", "        D += s * s;\n      }\n      den[bh * T + t] = D;",
     "        D += s;\n      }\n      den[bh * T + t] = D;"),
    ("abs_not_square", "double w = s * s;", "double w = fabs(s);"),
    ("weight_on_diagonal", "double w = (weighted && a != b) ? 2.0 : 1.0;",
     "double w = (weighted && a == b) ? 2.0 : 1.0;"),
    ("packed_index_off_by_one", "return a * d - a * (a - 1) / 2 + (b - a);",
     "return a * d - a * (a + 1) / 2 + (b - a);"),
    ("no_zero_guard", "if (D > 0.0) {", "if (1) {"),
    ("decode_no_zero_guard", "out[bh * dv + j] = (D > 0.0) ? acc / D : 0.0;",
     "out[bh * dv + j] = acc / D;"),
    ("inclusive_scan", "x[c * E + e] = run[e];\n        run[e] += cur;",
     "run[e] += cur;\n        x[c * E + e] = run[e];"),
    ("tree_no_root_clear", "for (long e = 0; e < E; ++e) a[(P - 1) * E + e] = 0.0;", ""),
    ("transposed_mask", "P[r * C + s] = (s <= r) ? a : 0.0;", "P[r * C + s] = (s >= r) ? a : 0.0;"),
    ("chunk_drops_intra_denominator", "for (long s = 0; s < C; ++s) D += P[r * C + s];", ""),
    ("state_value_index", "Sh[f * dv + j] += phi[f] * vt[j];", "Sh[f * dv + j] += phi[f] * vt[0];"),
    ("decode_readout_before_update",
     "    double D = 0.0;\n    for (long f = 0; f < n; ++f) D += pq[f] * zh[f];",
     "    double D = -pq[0] * pk[0];\n    for (long f = 0; f < n; ++f) D += pq[f] * zh[f];"),
    ("chunk_key_feature_weighted", "kata_oracle_phi(Kc + r * d, d, 0, PhiK + r * n);",
     "kata_oracle_phi(Kc + r * d, d, 1, PhiK + r * n);"),
    # KATA-Mg
    ("mg_full_dot", "for (long c = a * m; c < (a + 1) * m; ++c) s += qt[c] * ki[c];",
     "for (long c = 0; c < d; ++c) s += qt[c] * ki[c];"),
    ("mg_block_offset", "kata_oracle_phi(x + a * m, m, weighted, out + a * nm);",
     "kata_oracle_phi(x, m, weighted, out + a * nm);"),
    ("mg_width", "return g * (m * (m + 1) / 2);", "return g * (m * (m + 1) / 2) + 1;"),
    ("mg_sum_not_squared", "w += s * s;", "w += s * fabs(s);"),
    ("mg_drop_diagonal", "for (long i = 0; i <= t; ++i) {", "for (long i = 0; i < t; ++i) {", 1),
    ("mg_transposed_mask", "P[r * C + s] = (s <= r) ? a : 0.0;",
     "P[r * C + s] = (s >= r) ? a : 0.0;", 1),
    ("mg_chunk_query_unweighted", "kata_oracle_phi_mg(Qc + r * d, d, g, 1, PhiQ + r * n);",
     "kata_oracle_phi_mg(Qc + r * d, d, g, 0, PhiQ + r * n);"),
    ("mg_chunk_drops_intra_denominator", "for (long s = 0; s < C; ++s) D += P[r * C + s];", "", 1),
    ("mg_state_value_index", "Sh[f * dv + j] += phi[f] * vt[j];",
     "Sh[f * dv + j] += phi[f] * vt[0];", 1),
    ("mg_decode_readout_before_update",
     "    double D = 0.0;\n    for (long f = 0; f < n; ++f) D += pq[f] * zh[f];",
     "    double D = -pq[0] * pk[0];\n    for (long f = 0; f < n; ++f) D += pq[f] * zh[f];", 1),
    # linear features
    ("lin_relu_no_eps", "y = (y > 0.0 ? y : 0.0) + eps;", "y = (y > 0.0 ? y : 0.0);"),
    ("lin_elu_no_shift", "exp(y) - 1.0", "exp(y)"),
    ("lin_lorentz_squared_norm", "out[d] = sqrt(s);", "out[d] = s;"),
    ("lin_lorentz_s_factor", "(1.0 + x[d - 1] * x[d - 1])", "(1.0 + x[d - 1])"),
    ("lin_lorentz_width", "return feature == 3 ? d + 1 : d;", "return d;"),
    ("lin_drop_diagonal", "for (long i = 0; i <= t; ++i) {", "for (long i = 0; i < t; ++i) {", 2),
    ("lin_abs_weight", "for (long f = 0; f < n; ++f) w += fq[f] * fk[f];",
     "for (long f = 0; f < n; ++f) w += fabs(fq[f] * fk[f]);"),
    ("lin_normalize_flag_inverted", "if (!normalize) return;", "if (normalize) return;"),
    ("lin_chunk_strict_mask", "for (long s = 0; s <= r; ++s) {", "for (long s = 0; s < r; ++s) {"),
    ("lin_chunk_drops_prefix_denominator",
     "for (long f = 0; f < n; ++f) D += FQ[r * n + f] * St[n * dv + f];", ""),
    ("lin_chunk_z_from_values", "for (long r = 0; r < C; ++r) zs += FK[r * n + f];",
     "for (long r = 0; r < C; ++r) zs += Vc[r * dv];"),
    ("lin_state_transposed", "for (long r = 0; r < C; ++r) s += FK[r * n + f] * Vc[r * dv + j];",
     "for (long r = 0; r < C; ++r) s += FK[r * n + j % n] * Vc[r * dv + f % dv];"),
    ("lin_readout_query_index",
     "for (long f = 0; f < n; ++f) acc += FQ[r * n + f] * St[f * dv + j];",
     "for (long f = 0; f < n; ++f) acc += FQ[f] * St[f * dv + j];"),
    ("lin_chunk_key_feature_from_query",
     "kata_oracle_lin_feature(K + (t0 + r) * d, d, feature, eps, FK + r * n);",
     "kata_oracle_lin_feature(Q + (t0 + r) * d, d, feature, eps, FK + r * n);"),
    # backward
    ("bwd_b_sign", "    bt = -go / D;", "    bt = go / D;"),
    ("bwd_a_not_divided", "        A[t * dv + j] = G[t * dv + j] / D;", "        A[t * dv + j] = G[t * dv + j];"),
    ("bwd_no_factor_two_q", "            dQ[t * d + c] += 2.0 * cw * s[a] * K[i * d + c];",
     "            dQ[t * d + c] += cw * s[a] * K[i * d + c];"),
    ("bwd_dv_unweighted", "          dV[i * dv + j] += w * A[t * dv + j];",
     "          dV[i * dv + j] += A[t * dv + j];"),
    ("bwd_dk_from_k", "            dK[i * d + c] += 2.0 * cw * s[a] * Q[t * d + c];",
     "            dK[i * d + c] += 2.0 * cw * s[a] * K[i * d + c];"),
    ("bwd_chunk_b_sign", "        bv[t] = -go / D;", "        bv[t] = go / D;"),
    ("vjp_one_sided", "          dx[xb] += 2.0 * y * x[xa];", ""),
    ("bwd_chunk_no_reversal", "      double* Bt = bst + (NC - 1 - t / C) * SE;",
     "      double* Bt = bst + (t / C) * SE;"),
    ("bwd_chunk_dz_unweighted", "        Bt[n * dv + f] += bv[t] * ph[f];", "        Bt[n * dv + f] += ph[f];"),
    ("bwd_chunk_dv_query_side_weight", "      kata_oracle_phi_mg(K + t * d, d, g, 1, pw);",
     "      kata_oracle_phi_mg(K + t * d, d, g, 0, pw);"),
    ("bwd_chunk_inter_dq_missing_b", "        double y = bv[t] * St[n * dv + f];", "        double y = 0.0;"),
]


def _pins_that_fail(orc):
    failed = []
    for pin in ALL_PINS:
        try:
            pin(orc)
        except Exception:
            failed.append(pin.__name__)
    return failed


def _replace_nth(text, old, new, nth):
    at = -1
    for _ in range(nth + 1):
        at = text.index(old, at + 1)
    return text[:at] + new + text[at + len(old):]


@pytest.mark.parametrize("mutant", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_mutant_is_caught(mutant, tmp_path):
    name, old, new = mutant[:3]
    nth = mutant[3] if len(mutant) > 3 else 0
    with open(SRC) as f:
        text = f.read()
    # the site must exist (occurrences follow the file: KATA-M1, KATA-Mg, linear)
    assert text.count(old) >= nth + 1, f"mutation site {nth} for {name} not found"
    src = tmp_path / "mutant.c"
    src.write_text(_replace_nth(text, old, new, nth))
    lib_path = str(tmp_path / "libmutant.so")
    oracle.build(str(src), lib_path)
    mut = oracle.Oracle(oracle.load(lib_path))
    failed = _pins_that_fail(mut)
    assert failed, f"mutant {name} passed every pin"
