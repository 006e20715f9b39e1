/*
 * kata_oracle.c -- plain CPU oracle for the causal KATA-M1 attention forward
 * (rank-one PSD feature map phi(x) = vec(x x^T)) and its recurrent decode step,
 * and for the block-diagonal KATA-Mg variant (one rank-one factor per block of
 * d/g coordinates; g = 1 is M1).
 *
 * TEST INFRASTRUCTURE ONLY. Nothing in the product library links, loads,
 * imports or calls this file; only the test suite, the smoke check and the
 * bench's CPU-baseline leg do.  It shares no code, header, table or helper
 * with the GPU path.
 *
 * Everything is evaluated in IEEE double precision from the exact input values
 * (bf16 or fp32 inputs are widened exactly by the caller).  Loops are written
 * for a reader checking them against the paper, not for speed; the only
 * concession is an OpenMP loop over independent (batch, head, row) triples.
 *
 * Layouts (all row-major, contiguous):
 *   q, k : [B][H][T][d]      v : [B][H][T][dv]      out : [B][H][T][dv]
 *   packed feature index of the pair (a, b), a <= b, in a d x d symmetric
 *   matrix, upper triangle in row-major order:
 *       f(a, b) = a*d - a*(a-1)/2 + (b - a),   n = d*(d+1)/2 features.
 *   decode state: S : [B][H][n][dv],  z : [B][H][n]  (unscaled sums of
 *   k_a*k_b*v and k_a*k_b).
 *
 * Parity status: every function here is pinned by the CPU test suite
 * (closed forms, invariants, a hand-computed example, brute force with
 * unpacked d*d features, chunked-versus-definition agreement, scan-versus-
 * recurrence agreement).  None is "parity unpinned".
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define EXPORT __attribute__((visibility("default")))

/* Number of OpenMP threads the oracle's parallel loops use. */
EXPORT int kata_oracle_num_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}

EXPORT long kata_oracle_packed_dim(long d) { return d * (d + 1) / 2; }

/* Packed index of the unordered pair (a, b) (row-major upper triangle). */
EXPORT long kata_oracle_packed_index(long a, long b, long d) {
  if (a > b) { long t = a; a = b; b = t; }
  return a * d - a * (a - 1) / 2 + (b - a);
}

/*
 * Rank-one PSD lift, packed (section "Rank-one packing into the PSD cone" and
 * "From rank-one rays to low-rank PSD packing"): the feature of x is the
 * symmetric matrix x x^T, kept as its n = d(d+1)/2 upper-triangle entries.
 * weighted = 0: out[f(a,b)] = x_a x_b                (state side)
 * weighted = 1: out[f(a,b)] = (a==b ? 1 : 2) x_a x_b  (query side)
 * With these, sum_f phi_w(q)_f phi(k)_f equals the Frobenius inner product
 * <q q^T, k k^T> = (q . k)^2.
 */
EXPORT void kata_oracle_phi(const double* x, long d, int weighted, double* out) {
  for (long a = 0; a < d; ++a)
    for (long b = a; b < d; ++b) {
      double w = (weighted && a != b) ? 2.0 : 1.0;
      out[kata_oracle_packed_index(a, b, d)] = w * x[a] * x[b];
    }
}

/*
 * One output row of the definition: normalised linear attention (eq. linatt)
 * with psi = phi, where <phi(q), phi(k)> = (q . k)^2:
 *     w_i = (q_t . k_i)^2 for i <= t,
 *     o_t = sum_i w_i v_i / sum_i w_i,   o_t = 0 when the sum is 0.
 * Rows are 0-indexed; the sum includes i = t (the current token, which is the
 * c_t term of the output-gate proposition).
 */
static void definition_row(const double* q, const double* k, const double* v,
                           long t, long d, long dv, double* o) {
  double D = 0.0;
  for (long j = 0; j < dv; ++j) o[j] = 0.0;
  const double* qt = q + t * d;
  for (long i = 0; i <= t; ++i) {
    const double* ki = k + i * d;
    double s = 0.0;
    for (long a = 0; a < d; ++a) s += qt[a] * ki[a];
    double w = s * s;
    D += w;
    const double* vi = v + i * dv;
    for (long j = 0; j < dv; ++j) o[j] += w * vi[j];
  }
  if (D > 0.0) {
    for (long j = 0; j < dv; ++j) o[j] /= D;
  } else {
    for (long j = 0; j < dv; ++j) o[j] = 0.0;
  }
}

/* Full causal forward by the definition, O(T^2) per head. */
EXPORT void kata_oracle_fwd(const double* q, const double* k, const double* v,
                            double* out, long B, long H, long T, long d, long dv) {
  long BH = B * H;
#pragma omp parallel for collapse(2) schedule(dynamic, 16)
  for (long bh = 0; bh < BH; ++bh)
    for (long t = 0; t < T; ++t)
      definition_row(q + bh * T * d, k + bh * T * d, v + bh * T * dv, t, d, dv,
                     out + (bh * T + t) * dv);
}

/*
 * The definition evaluated only at listed rows: entry r is head bh_idx[r]
 * (flattened b*H + h) and token t_idx[r]; out is [nrows][dv].
 */
EXPORT void kata_oracle_fwd_rows(const double* q, const double* k, const double* v,
                                 long B, long H, long T, long d, long dv,
                                 const long* bh_idx, const long* t_idx, long nrows,
                                 double* out) {
  (void)B; (void)H;
#pragma omp parallel for schedule(dynamic, 1)
  for (long r = 0; r < nrows; ++r) {
    long bh = bh_idx[r];
    definition_row(q + bh * T * d, k + bh * T * d, v + bh * T * dv, t_idx[r], d, dv,
                   out + r * dv);
  }
}

/*
 * Exclusive prefix sum along the leading axis of x : [N][E], in place:
 * x[c] <- sum_{c' < c} x[c'], x[0] <- 0 (section "Tree-scan inter-chunk
 * reduction": the inter-chunk prefix is exclusive, the first one is zero).
 * mode 0: the sequential recurrence.  mode 1: the work-efficient tree scan
 * (up-sweep building partial sums over power-of-two blocks, then down-sweep
 * distributing them), over N rounded up to a power of two with zero padding;
 * ceil(log2 N) rounds in each sweep.
 */
EXPORT void kata_oracle_scan_exclusive(double* x, long N, long E, int mode) {
  if (N <= 0) return;
  if (mode == 0) {
    double* run = (double*)calloc((size_t)E, sizeof(double));
    for (long c = 0; c < N; ++c)
      for (long e = 0; e < E; ++e) {
        double cur = x[c * E + e];
        x[c * E + e] = run[e];
        run[e] += cur;
      }
    free(run);
    return;
  }
  long P = 1;
  while (P < N) P <<= 1;
  double* a = (double*)calloc((size_t)(P * E), sizeof(double));
  memcpy(a, x, (size_t)(N * E) * sizeof(double));
  /* up-sweep: after round r, a[i] for i = m*2^(r+1) - 1 holds the sum of its block */
  for (long step = 1; step < P; step <<= 1)
    for (long i = 2 * step - 1; i < P; i += 2 * step)
      for (long e = 0; e < E; ++e) a[i * E + e] += a[(i - step) * E + e];
  /* clear the root, then down-sweep: each node passes its prefix to the left
     child and prefix + left-sum to the right child */
  for (long e = 0; e < E; ++e) a[(P - 1) * E + e] = 0.0;
  for (long step = P >> 1; step >= 1; step >>= 1)
    for (long i = 2 * step - 1; i < P; i += 2 * step)
      for (long e = 0; e < E; ++e) {
        double left = a[(i - step) * E + e];
        a[(i - step) * E + e] = a[i * E + e];
        a[i * E + e] += left;
      }
  memcpy(x, a, (size_t)(N * E) * sizeof(double));
  free(a);
}

/*
 * Chunkwise forward (eq. chunk-SZ and eq. chunk-out; the chunkwise algorithm
 * of the appendix), for every head, in packed features:
 *   N_C = ceil(T / C); the last chunk is padded with zero rows; the output is
 *   truncated to T rows.
 *   Local chunk state   S_loc[c] = Psi(K_c)^T V_c,  Z_loc[c] = Psi(K_c)^T 1.
 *   Prefix              S_[c] = sum_{c' < c} S_loc[c'] (exclusive; S_[0] = 0)
 *                       via the sequential recurrence (scan_mode 0) or the
 *                       tree scan (scan_mode 1).
 *   Chunk output        P = (Psi_w(Q_c) Psi(K_c)^T) .* M, M lower-triangular
 *                       including the diagonal,
 *                       N = Psi_w(Q_c) S_[c] + P V_c,  D = Psi_w(Q_c) Z_[c] + P 1,
 *                       O = diag(D)^-1 N  (rows with D = 0 give 0).
 * Psi_w is the query-side weighted packed feature, so that
 * Psi_w(q) . Psi(k) = (q . k)^2.
 */
EXPORT void kata_oracle_fwd_chunked(const double* q, const double* k, const double* v,
                                    double* out, long B, long H, long T, long d,
                                    long dv, long C, int scan_mode) {
  long n = d * (d + 1) / 2;
  long NC = (T + C - 1) / C;
  long BH = B * H;
  long SE = n * dv + n; /* one state record: S (n x dv) then Z (n) */
#pragma omp parallel for schedule(dynamic, 1)
  for (long bh = 0; bh < BH; ++bh) {
    const double* Q = q + bh * T * d;
    const double* K = k + bh * T * d;
    const double* V = v + bh * T * dv;
    double* O = out + bh * T * dv;
    /* padded chunk inputs */
    double* Qc = (double*)calloc((size_t)(C * d), sizeof(double));
    double* Kc = (double*)calloc((size_t)(C * d), sizeof(double));
    double* Vc = (double*)calloc((size_t)(C * dv), sizeof(double));
    double* PhiQ = (double*)malloc((size_t)(C * n) * sizeof(double));
    double* PhiK = (double*)malloc((size_t)(C * n) * sizeof(double));
    double* P = (double*)malloc((size_t)(C * C) * sizeof(double));
    double* Nrow = (double*)malloc((size_t)dv * sizeof(double));
    double* states = (double*)calloc((size_t)(NC * SE), sizeof(double));

    for (long pass = 0; pass < 2; ++pass) {
      /* pass 0: local chunk states; then the prefix; pass 1: chunk outputs */
      for (long c = 0; c < NC; ++c) {
        long t0 = c * C;
        memset(Qc, 0, (size_t)(C * d) * sizeof(double));
        memset(Kc, 0, (size_t)(C * d) * sizeof(double));
        memset(Vc, 0, (size_t)(C * dv) * sizeof(double));
        for (long r = 0; r < C && t0 + r < T; ++r) {
          memcpy(Qc + r * d, Q + (t0 + r) * d, (size_t)d * sizeof(double));
          memcpy(Kc + r * d, K + (t0 + r) * d, (size_t)d * sizeof(double));
          memcpy(Vc + r * dv, V + (t0 + r) * dv, (size_t)dv * sizeof(double));
        }
        for (long r = 0; r < C; ++r) {
          kata_oracle_phi(Kc + r * d, d, 0, PhiK + r * n);
          kata_oracle_phi(Qc + r * d, d, 1, PhiQ + r * n);
        }
        double* St = states + c * SE; /* S then Z of this chunk */
        if (pass == 0) {
          /* S_loc = Psi(K_c)^T V_c ; Z_loc = Psi(K_c)^T 1 */
          for (long f = 0; f < n; ++f) {
            for (long j = 0; j < dv; ++j) {
              double s = 0.0;
              for (long r = 0; r < C; ++r) s += PhiK[r * n + f] * Vc[r * dv + j];
              St[f * dv + j] = s;
            }
            double zs = 0.0;
            for (long r = 0; r < C; ++r) zs += PhiK[r * n + f];
            St[n * dv + f] = zs;
          }
          continue;
        }
        /* pass 1: St now holds the exclusive prefix (S_[c], Z_[c]) */
        for (long r = 0; r < C; ++r)
          for (long s = 0; s < C; ++s) {
            double a = 0.0;
            for (long f = 0; f < n; ++f) a += PhiQ[r * n + f] * PhiK[s * n + f];
            P[r * C + s] = (s <= r) ? a : 0.0;
          }
        for (long r = 0; r < C && t0 + r < T; ++r) {
          double D = 0.0;
          for (long f = 0; f < n; ++f) D += PhiQ[r * n + f] * St[n * dv + f];
          for (long s = 0; s < C; ++s) D += P[r * C + s];
          for (long j = 0; j < dv; ++j) {
            double acc = 0.0;
            for (long f = 0; f < n; ++f) acc += PhiQ[r * n + f] * St[f * dv + j];
            for (long s = 0; s < C; ++s) acc += P[r * C + s] * Vc[s * dv + j];
            Nrow[j] = acc;
          }
          for (long j = 0; j < dv; ++j) O[(t0 + r) * dv + j] = (D > 0.0) ? Nrow[j] / D : 0.0;
        }
      }
      if (pass == 0) kata_oracle_scan_exclusive(states, NC, SE, scan_mode);
    }
    free(Qc); free(Kc); free(Vc); free(PhiQ); free(PhiK); free(P); free(Nrow);
    free(states);
  }
}

/*
 * State after T tokens by the additive recurrence of eq. linatt:
 *   S_t = S_{t-1} + phi(k_t) v_t^T,  Z_t = Z_{t-1} + phi(k_t),  S_0 = 0, Z_0 = 0.
 * Overwrites S : [B][H][n][dv] and z : [B][H][n].
 */
EXPORT void kata_oracle_state(const double* k, const double* v, double* S, double* z,
                              long B, long H, long T, long d, long dv) {
  long n = d * (d + 1) / 2;
  long BH = B * H;
#pragma omp parallel for schedule(dynamic, 1)
  for (long bh = 0; bh < BH; ++bh) {
    double* Sh = S + bh * n * dv;
    double* zh = z + bh * n;
    double* phi = (double*)malloc((size_t)n * sizeof(double));
    memset(Sh, 0, (size_t)(n * dv) * sizeof(double));
    memset(zh, 0, (size_t)n * sizeof(double));
    for (long t = 0; t < T; ++t) {
      kata_oracle_phi(k + (bh * T + t) * d, d, 0, phi);
      const double* vt = v + (bh * T + t) * dv;
      for (long f = 0; f < n; ++f) {
        for (long j = 0; j < dv; ++j) Sh[f * dv + j] += phi[f] * vt[j];
        zh[f] += phi[f];
      }
    }
    free(phi);
  }
}

/*
 * One recurrent decode step for every head (eq. linatt's recurrence, then its
 * normalised readout with the updated state, so the current token is included
 * as in the forward):
 *   S <- S + phi(k) v^T,  z <- z + phi(k),
 *   o = phi_w(q)^T S / phi_w(q)^T z   (o = 0 when the denominator is 0).
 * q, k : [B][H][d]; v, out : [B][H][dv]; S, z updated in place.
 */
EXPORT void kata_oracle_decode_step(double* S, double* z, const double* q,
                                    const double* k, const double* v, double* out,
                                    long B, long H, long d, long dv) {
  long n = d * (d + 1) / 2;
  long BH = B * H;
#pragma omp parallel for schedule(static)
  for (long bh = 0; bh < BH; ++bh) {
    double* Sh = S + bh * n * dv;
    double* zh = z + bh * n;
    double* pk = (double*)malloc((size_t)n * sizeof(double));
    double* pq = (double*)malloc((size_t)n * sizeof(double));
    kata_oracle_phi(k + bh * d, d, 0, pk);
    kata_oracle_phi(q + bh * d, d, 1, pq);
    const double* vt = v + bh * dv;
    for (long f = 0; f < n; ++f) {
      for (long j = 0; j < dv; ++j) Sh[f * dv + j] += pk[f] * vt[j];
      zh[f] += pk[f];
    }
    double D = 0.0;
    for (long f = 0; f < n; ++f) D += pq[f] * zh[f];
    for (long j = 0; j < dv; ++j) {
      double acc = 0.0;
      for (long f = 0; f < n; ++f) acc += pq[f] * Sh[f * dv + j];
      out[bh * dv + j] = (D > 0.0) ? acc / D : 0.0;
    }
    free(pk);
    free(pq);
  }
}

/* ======================================================================
 * KATA-Mg (section "From rank-one rays to low-rank PSD packing"): each
 * projected query or key u in R^d is split into g blocks of m = d/g
 * consecutive coordinates, u = (u_1, ..., u_g), and the feature keeps one
 * rank-one PSD factor per block, psi_Mg(u) = (u_1 u_1^T, ..., u_g u_g^T), so
 *     <psi_Mg(q), psi_Mg(k)> = sum_a (q_a . k_a)^2 .
 * g = 1 is KATA-M1 above.  Packed layout: block a's m(m+1)/2 upper-triangle
 * entries (row-major, as for M1 with d -> m) at offset a*m(m+1)/2; the
 * feature width is n_g = g*m(m+1)/2 = d(d/g + 1)/2.
 * ====================================================================== */

EXPORT long kata_oracle_packed_dim_mg(long d, long g) {
  long m = d / g;
  return g * (m * (m + 1) / 2);
}

/* Blockwise packed lift: kata_oracle_phi applied to each block in turn
 * (weighted = 1: weight 2 off each block's diagonal, the query side). */
EXPORT void kata_oracle_phi_mg(const double* x, long d, long g, int weighted, double* out) {
  long m = d / g, nm = m * (m + 1) / 2;
  for (long a = 0; a < g; ++a) kata_oracle_phi(x + a * m, m, weighted, out + a * nm);
}

/* One output row of the definition with the KATA-Mg weight
 *     w_i = sum_a (q_{t,a} . k_{i,a})^2,  i <= t,
 *     o_t = sum_i w_i v_i / sum_i w_i  (0 when the sum is 0). */
static void definition_row_mg(const double* q, const double* k, const double* v, long t,
                              long d, long dv, long g, double* o) {
  long m = d / g;
  double D = 0.0;
  for (long j = 0; j < dv; ++j) o[j] = 0.0;
  const double* qt = q + t * d;
  for (long i = 0; i <= t; ++i) {
    const double* ki = k + i * d;
    double w = 0.0;
    for (long a = 0; a < g; ++a) {
      double s = 0.0;
      for (long c = a * m; c < (a + 1) * m; ++c) s += qt[c] * ki[c];
      w += s * s;
    }
    D += w;
    const double* vi = v + i * dv;
    for (long j = 0; j < dv; ++j) o[j] += w * vi[j];
  }
  if (D > 0.0) {
    for (long j = 0; j < dv; ++j) o[j] /= D;
  } else {
    for (long j = 0; j < dv; ++j) o[j] = 0.0;
  }
}

EXPORT void kata_oracle_fwd_mg(const double* q, const double* k, const double* v, double* out,
                               long B, long H, long T, long d, long dv, long g) {
  long BH = B * H;
#pragma omp parallel for collapse(2) schedule(dynamic, 16)
  for (long bh = 0; bh < BH; ++bh)
    for (long t = 0; t < T; ++t)
      definition_row_mg(q + bh * T * d, k + bh * T * d, v + bh * T * dv, t, d, dv, g,
                        out + (bh * T + t) * dv);
}

EXPORT void kata_oracle_fwd_mg_rows(const double* q, const double* k, const double* v,
                                    long B, long H, long T, long d, long dv, long g,
                                    const long* bh_idx, const long* t_idx, long nrows,
                                    double* out) {
  (void)B; (void)H;
#pragma omp parallel for schedule(dynamic, 1)
  for (long r = 0; r < nrows; ++r) {
    long bh = bh_idx[r];
    definition_row_mg(q + bh * T * d, k + bh * T * d, v + bh * T * dv, t_idx[r], d, dv, g,
                      out + r * dv);
  }
}

/* Chunkwise KATA-Mg forward: kata_oracle_fwd_chunked with Psi = psi_Mg
 * (same chunk states, exclusive prefix and chunk output; n = n_g). */
EXPORT void kata_oracle_fwd_chunked_mg(const double* q, const double* k, const double* v,
                                       double* out, long B, long H, long T, long d, long dv,
                                       long C, long g, int scan_mode) {
  long n = kata_oracle_packed_dim_mg(d, g);
  long NC = (T + C - 1) / C;
  long BH = B * H;
  long SE = n * dv + n; /* one state record: S (n x dv) then Z (n) */
#pragma omp parallel for schedule(dynamic, 1)
  for (long bh = 0; bh < BH; ++bh) {
    const double* Q = q + bh * T * d;
    const double* K = k + bh * T * d;
    const double* V = v + bh * T * dv;
    double* O = out + bh * T * dv;
    double* Qc = (double*)calloc((size_t)(C * d), sizeof(double));
    double* Kc = (double*)calloc((size_t)(C * d), sizeof(double));
    double* Vc = (double*)calloc((size_t)(C * dv), sizeof(double));
    double* PhiQ = (double*)malloc((size_t)(C * n) * sizeof(double));
    double* PhiK = (double*)malloc((size_t)(C * n) * sizeof(double));
    double* P = (double*)malloc((size_t)(C * C) * sizeof(double));
    double* Nrow = (double*)malloc((size_t)dv * sizeof(double));
    double* states = (double*)calloc((size_t)(NC * SE), sizeof(double));
    for (long pass = 0; pass < 2; ++pass) {
      for (long c = 0; c < NC; ++c) {
        long t0 = c * C;
        memset(Qc, 0, (size_t)(C * d) * sizeof(double));
        memset(Kc, 0, (size_t)(C * d) * sizeof(double));
        memset(Vc, 0, (size_t)(C * dv) * sizeof(double));
        for (long r = 0; r < C && t0 + r < T; ++r) {
          memcpy(Qc + r * d, Q + (t0 + r) * d, (size_t)d * sizeof(double));
          memcpy(Kc + r * d, K + (t0 + r) * d, (size_t)d * sizeof(double));
          memcpy(Vc + r * dv, V + (t0 + r) * dv, (size_t)dv * sizeof(double));
        }
        for (long r = 0; r < C; ++r) {
          kata_oracle_phi_mg(Kc + r * d, d, g, 0, PhiK + r * n);
          kata_oracle_phi_mg(Qc + r * d, d, g, 1, PhiQ + r * n);
        }
        double* St = states + c * SE;
        if (pass == 0) {
          for (long f = 0; f < n; ++f) {
            for (long j = 0; j < dv; ++j) {
              double s = 0.0;
              for (long r = 0; r < C; ++r) s += PhiK[r * n + f] * Vc[r * dv + j];
              St[f * dv + j] = s;
            }
            double zs = 0.0;
            for (long r = 0; r < C; ++r) zs += PhiK[r * n + f];
            St[n * dv + f] = zs;
          }
          continue;
        }
        for (long r = 0; r < C; ++r)
          for (long s = 0; s < C; ++s) {
            double a = 0.0;
            for (long f = 0; f < n; ++f) a += PhiQ[r * n + f] * PhiK[s * n + f];
            P[r * C + s] = (s <= r) ? a : 0.0;
          }
        for (long r = 0; r < C && t0 + r < T; ++r) {
          double D = 0.0;
          for (long f = 0; f < n; ++f) D += PhiQ[r * n + f] * St[n * dv + f];
          for (long s = 0; s < C; ++s) D += P[r * C + s];
          for (long j = 0; j < dv; ++j) {
            double acc = 0.0;
            for (long f = 0; f < n; ++f) acc += PhiQ[r * n + f] * St[f * dv + j];
            for (long s = 0; s < C; ++s) acc += P[r * C + s] * Vc[s * dv + j];
            Nrow[j] = acc;
          }
          for (long j = 0; j < dv; ++j) O[(t0 + r) * dv + j] = (D > 0.0) ? Nrow[j] / D : 0.0;
        }
      }
      if (pass == 0) kata_oracle_scan_exclusive(states, NC, SE, scan_mode);
    }
    free(Qc); free(Kc); free(Vc); free(PhiQ); free(PhiK); free(P); free(Nrow);
    free(states);
  }
}

/* KATA-Mg state after T tokens (the additive recurrence of eq. linatt with
 * psi_Mg): S : [B][H][n_g][dv], z : [B][H][n_g]. */
EXPORT void kata_oracle_state_mg(const double* k, const double* v, double* S, double* z,
                                 long B, long H, long T, long d, long dv, long g) {
  long n = kata_oracle_packed_dim_mg(d, g);
  long BH = B * H;
#pragma omp parallel for schedule(dynamic, 1)
  for (long bh = 0; bh < BH; ++bh) {
    double* Sh = S + bh * n * dv;
    double* zh = z + bh * n;
    double* phi = (double*)malloc((size_t)n * sizeof(double));
    memset(Sh, 0, (size_t)(n * dv) * sizeof(double));
    memset(zh, 0, (size_t)n * sizeof(double));
    for (long t = 0; t < T; ++t) {
      kata_oracle_phi_mg(k + (bh * T + t) * d, d, g, 0, phi);
      const double* vt = v + (bh * T + t) * dv;
      for (long f = 0; f < n; ++f) {
        for (long j = 0; j < dv; ++j) Sh[f * dv + j] += phi[f] * vt[j];
        zh[f] += phi[f];
      }
    }
    free(phi);
  }
}

/* One KATA-Mg decode step (kata_oracle_decode_step with psi_Mg): update the
 * state with the current token, then read out with the updated state. */
EXPORT void kata_oracle_decode_step_mg(double* S, double* z, const double* q,
                                       const double* k, const double* v, double* out,
                                       long B, long H, long d, long dv, long g) {
  long n = kata_oracle_packed_dim_mg(d, g);
  long BH = B * H;
#pragma omp parallel for schedule(static)
  for (long bh = 0; bh < BH; ++bh) {
    double* Sh = S + bh * n * dv;
    double* zh = z + bh * n;
    double* pk = (double*)malloc((size_t)n * sizeof(double));
    double* pq = (double*)malloc((size_t)n * sizeof(double));
    kata_oracle_phi_mg(k + bh * d, d, g, 0, pk);
    kata_oracle_phi_mg(q + bh * d, d, g, 1, pq);
    const double* vt = v + bh * dv;
    for (long f = 0; f < n; ++f) {
      for (long j = 0; j < dv; ++j) Sh[f * dv + j] += pk[f] * vt[j];
      zh[f] += pk[f];
    }
    double D = 0.0;
    for (long f = 0; f < n; ++f) D += pq[f] * zh[f];
    for (long j = 0; j < dv; ++j) {
      double acc = 0.0;
      for (long f = 0; f < n; ++f) acc += pq[f] * Sh[f * dv + j];
      out[bh * dv + j] = (D > 0.0) ? acc / D : 0.0;
    }
    free(pk);
    free(pq);
  }
}

/* ======================================================================
 * Linear (n_psi ~ d) features of normalised linear attention (eq. linatt):
 * the feature maps of section "Classical feature maps", used by the paper's
 * tree-scan measurements.
 *   feature 0  identity     psi(x) = x                       n_psi = d
 *   feature 1  orthant      psi(x) = ReLU(x) + eps           n_psi = d
 *   feature 2  orthant      psi(x) = ELU(x) + 1              n_psi = d
 *   feature 3  Lorentz      psi(y) = (y, ||y||_2)            n_psi = d + 1
 *   feature 4  Lorentz, the appendix variant of the KATA-Lorentz model: with
 *              y = x_1..x_{d-1} and s = x_d, psi(x) = (y, ||y||_2 (1 + s^2))
 *                                                            n_psi = d
 * Output: o_t = N_t / D_t with N_t = sum_{i<=t} w_ti v_i, D_t = sum_{i<=t} w_ti,
 * w_ti = <psi(q_t), psi(k_i)>, and o_t = 0 unless D_t > 0 (normalize = 1; the
 * readout is defined for a positive denominator, eq. linatt); or
 * o_t = N_t (normalize = 0, the unnormalised readout used with psi(x) = x,
 * whose weights have no sign).
 * ====================================================================== */

EXPORT long kata_oracle_lin_dim(long d, int feature) { return feature == 3 ? d + 1 : d; }

EXPORT void kata_oracle_lin_feature(const double* x, long d, int feature, double eps,
                                    double* out) {
  if (feature == 3) {
    double s = 0.0;
    for (long a = 0; a < d; ++a) {
      out[a] = x[a];
      s += x[a] * x[a];
    }
    out[d] = sqrt(s);
    return;
  }
  if (feature == 4) {
    double s = 0.0;
    for (long a = 0; a + 1 < d; ++a) {
      out[a] = x[a];
      s += x[a] * x[a];
    }
    out[d - 1] = sqrt(s) * (1.0 + x[d - 1] * x[d - 1]);
    return;
  }
  for (long a = 0; a < d; ++a) {
    double y = x[a];
    if (feature == 1) y = (y > 0.0 ? y : 0.0) + eps;
    else if (feature == 2) y = (y > 0.0 ? y : exp(y) - 1.0) + 1.0;
    out[a] = y;
  }
}

static void lin_definition_row(const double* q, const double* k, const double* v, long t,
                               long d, long dv, int feature, double eps, int normalize,
                               double* fq, double* fk, double* o) {
  long n = kata_oracle_lin_dim(d, feature);
  double D = 0.0;
  for (long j = 0; j < dv; ++j) o[j] = 0.0;
  kata_oracle_lin_feature(q + t * d, d, feature, eps, fq);
  for (long i = 0; i <= t; ++i) {
    kata_oracle_lin_feature(k + i * d, d, feature, eps, fk);
    double w = 0.0;
    for (long f = 0; f < n; ++f) w += fq[f] * fk[f];
    D += w;
    const double* vi = v + i * dv;
    for (long j = 0; j < dv; ++j) o[j] += w * vi[j];
  }
  if (!normalize) return;
  if (D > 0.0) {
    for (long j = 0; j < dv; ++j) o[j] /= D;
  } else {
    for (long j = 0; j < dv; ++j) o[j] = 0.0;
  }
}

/* Definition forward, O(T^2) per head. */
EXPORT void kata_oracle_lin_fwd(const double* q, const double* k, const double* v, double* out,
                                long B, long H, long T, long d, long dv, int feature, double eps,
                                int normalize) {
  long BH = B * H;
  long n = kata_oracle_lin_dim(d, feature);
#pragma omp parallel
  {
    double* fq = (double*)malloc((size_t)n * sizeof(double));
    double* fk = (double*)malloc((size_t)n * sizeof(double));
#pragma omp for collapse(2) schedule(dynamic, 16)
    for (long bh = 0; bh < BH; ++bh)
      for (long t = 0; t < T; ++t)
        lin_definition_row(q + bh * T * d, k + bh * T * d, v + bh * T * dv, t, d, dv, feature,
                           eps, normalize, fq, fk, out + (bh * T + t) * dv);
    free(fq);
    free(fk);
  }
}

EXPORT void kata_oracle_lin_fwd_rows(const double* q, const double* k, const double* v, long B,
                                     long H, long T, long d, long dv, int feature, double eps,
                                     int normalize, const long* bh_idx, const long* t_idx,
                                     long nrows, double* out) {
  (void)B; (void)H;
  long n = kata_oracle_lin_dim(d, feature);
#pragma omp parallel
  {
    double* fq = (double*)malloc((size_t)n * sizeof(double));
    double* fk = (double*)malloc((size_t)n * sizeof(double));
#pragma omp for schedule(dynamic, 1)
    for (long r = 0; r < nrows; ++r) {
      long bh = bh_idx[r];
      lin_definition_row(q + bh * T * d, k + bh * T * d, v + bh * T * dv, t_idx[r], d, dv,
                         feature, eps, normalize, fq, fk, out + r * dv);
    }
    free(fq);
    free(fk);
  }
}

/* Chunkwise form (eq. chunk-SZ, eq. chunk-out) with a linear feature: local
 * chunk states S_loc = psi(K_c)^T V_c, z_loc = psi(K_c)^T 1, their exclusive
 * prefix (scan_mode 0 sequential, 1 tree), and per chunk
 *   N = psi(Q_c) S_[c] + (psi(Q_c) psi(K_c)^T .* M) V_c,
 *   D = psi(Q_c) z_[c] + (psi(Q_c) psi(K_c)^T .* M) 1, O = N / D (or N). */
EXPORT void kata_oracle_lin_fwd_chunked(const double* q, const double* k, const double* v,
                                        double* out, long B, long H, long T, long d, long dv,
                                        long C, int feature, double eps, int normalize,
                                        int scan_mode) {
  long n = kata_oracle_lin_dim(d, feature);
  long NC = (T + C - 1) / C;
  long BH = B * H;
  long SE = n * dv + n;
#pragma omp parallel for schedule(dynamic, 1)
  for (long bh = 0; bh < BH; ++bh) {
    const double* Q = q + bh * T * d;
    const double* K = k + bh * T * d;
    const double* V = v + bh * T * dv;
    double* O = out + bh * T * dv;
    double* FQ = (double*)calloc((size_t)(C * n), sizeof(double));
    double* FK = (double*)calloc((size_t)(C * n), sizeof(double));
    double* Vc = (double*)calloc((size_t)(C * dv), sizeof(double));
    double* states = (double*)calloc((size_t)(NC * SE), sizeof(double));
    for (long pass = 0; pass < 2; ++pass) {
      for (long c = 0; c < NC; ++c) {
        long t0 = c * C;
        memset(FQ, 0, (size_t)(C * n) * sizeof(double));
        memset(FK, 0, (size_t)(C * n) * sizeof(double));
        memset(Vc, 0, (size_t)(C * dv) * sizeof(double));
        /* rows past T stay zero: a padded key has no feature (weight 0) */
        for (long r = 0; r < C && t0 + r < T; ++r) {
          kata_oracle_lin_feature(Q + (t0 + r) * d, d, feature, eps, FQ + r * n);
          kata_oracle_lin_feature(K + (t0 + r) * d, d, feature, eps, FK + r * n);
          memcpy(Vc + r * dv, V + (t0 + r) * dv, (size_t)dv * sizeof(double));
        }
        double* St = states + c * SE;
        if (pass == 0) {
          for (long f = 0; f < n; ++f) {
            for (long j = 0; j < dv; ++j) {
              double s = 0.0;
              for (long r = 0; r < C; ++r) s += FK[r * n + f] * Vc[r * dv + j];
              St[f * dv + j] = s;
            }
            double zs = 0.0;
            for (long r = 0; r < C; ++r) zs += FK[r * n + f];
            St[n * dv + f] = zs;
          }
          continue;
        }
        for (long r = 0; r < C && t0 + r < T; ++r) {
          double D = 0.0;
          for (long f = 0; f < n; ++f) D += FQ[r * n + f] * St[n * dv + f];
          for (long j = 0; j < dv; ++j) {
            double acc = 0.0;
            for (long f = 0; f < n; ++f) acc += FQ[r * n + f] * St[f * dv + j];
            O[(t0 + r) * dv + j] = acc;
          }
          for (long s = 0; s <= r; ++s) {
            double w = 0.0;
            for (long f = 0; f < n; ++f) w += FQ[r * n + f] * FK[s * n + f];
            D += w;
            for (long j = 0; j < dv; ++j) O[(t0 + r) * dv + j] += w * Vc[s * dv + j];
          }
          if (normalize)
            for (long j = 0; j < dv; ++j)
              O[(t0 + r) * dv + j] = (D > 0.0) ? O[(t0 + r) * dv + j] / D : 0.0;
        }
      }
      if (pass == 0) kata_oracle_scan_exclusive(states, NC, SE, scan_mode);
    }
    free(FQ); free(FK); free(Vc); free(states);
  }
}

/* ======================================================================
 * Backward of the causal KATA-Mg forward (g = 1 is KATA-M1) for a loss with
 * output cotangents dout_t = dL/do_t.  With N_t = sum_{i<=t} w_ti v_i,
 * D_t = sum_{i<=t} w_ti and o_t = N_t / D_t:
 *     dL/dN_t = a_t = dout_t / D_t,   dL/dD_t = b_t = -<dout_t, o_t> / D_t,
 *     dL/dw_ti = <a_t, v_i> + b_t                  (i <= t),
 *     dv_i = sum_{t >= i} w_ti a_t,
 * and with s_ti,blk = q_t,blk . k_i,blk (w_ti = sum_blk s^2):
 *     dq_t,blk = sum_{i <= t} 2 (dL/dw_ti) s_ti,blk k_i,blk,
 *     dk_i,blk = sum_{t >= i} 2 (dL/dw_ti) s_ti,blk q_t,blk.
 * A row with D_t = 0 has the constant readout 0 (the reading of the forward),
 * so it contributes nothing: a_t = 0, b_t = 0.
 * ====================================================================== */

static void head_readout_mg(const double* Q, const double* K, const double* V, long T, long d,
                            long dv, long g, const double* G, double* A, double* bvec) {
  /* per token: o_t, D_t from the definition, then a_t (A, T x dv) and b_t */
  double* o = (double*)malloc((size_t)dv * sizeof(double));
  long m = d / g;
  for (long t = 0; t < T; ++t) {
    double D = 0.0;
    for (long j = 0; j < dv; ++j) o[j] = 0.0;
    for (long i = 0; i <= t; ++i) {
      double w = 0.0;
      for (long a = 0; a < g; ++a) {
        double s = 0.0;
        for (long c = a * m; c < (a + 1) * m; ++c) s += Q[t * d + c] * K[i * d + c];
        w += s * s;
      }
      D += w;
      for (long j = 0; j < dv; ++j) o[j] += w * V[i * dv + j];
    }
    double bt = 0.0;
    if (D > 0.0) {
      double go = 0.0;
      for (long j = 0; j < dv; ++j) {
        o[j] /= D;
        go += G[t * dv + j] * o[j];
        A[t * dv + j] = G[t * dv + j] / D;
      }
      bt = -go / D;
    } else {
      for (long j = 0; j < dv; ++j) A[t * dv + j] = 0.0;
    }
    bvec[t] = bt;
  }
  free(o);
}

EXPORT void kata_oracle_bwd_mg(const double* q, const double* k, const double* v,
                               const double* dout, double* dq, double* dk, double* dvo, long B,
                               long H, long T, long d, long dv, long g) {
  long BH = B * H, m = d / g;
#pragma omp parallel for schedule(dynamic, 1)
  for (long bh = 0; bh < BH; ++bh) {
    const double* Q = q + bh * T * d;
    const double* K = k + bh * T * d;
    const double* V = v + bh * T * dv;
    const double* G = dout + bh * T * dv;
    double* dQ = dq + bh * T * d;
    double* dK = dk + bh * T * d;
    double* dV = dvo + bh * T * dv;
    double* A = (double*)malloc((size_t)(T * dv) * sizeof(double));
    double* bv = (double*)malloc((size_t)T * sizeof(double));
    double* s = (double*)malloc((size_t)g * sizeof(double));
    head_readout_mg(Q, K, V, T, d, dv, g, G, A, bv);
    memset(dQ, 0, (size_t)(T * d) * sizeof(double));
    memset(dK, 0, (size_t)(T * d) * sizeof(double));
    memset(dV, 0, (size_t)(T * dv) * sizeof(double));
    for (long t = 0; t < T; ++t) {
      for (long i = 0; i <= t; ++i) {
        double w = 0.0;
        for (long a = 0; a < g; ++a) {
          s[a] = 0.0;
          for (long c = a * m; c < (a + 1) * m; ++c) s[a] += Q[t * d + c] * K[i * d + c];
          w += s[a] * s[a];
        }
        double cw = bv[t];
        for (long j = 0; j < dv; ++j) {
          cw += A[t * dv + j] * V[i * dv + j];
          dV[i * dv + j] += w * A[t * dv + j];
        }
        for (long a = 0; a < g; ++a)
          for (long c = a * m; c < (a + 1) * m; ++c) {
            dQ[t * d + c] += 2.0 * cw * s[a] * K[i * d + c];
            dK[i * d + c] += 2.0 * cw * s[a] * Q[t * d + c];
          }
      }
    }
    free(A); free(bv); free(s);
  }
}

/* Feature-map VJP of the packed block lift: a cotangent Y over the n packed
 * features (pair (x, y) of a block, x <= y, unscaled) gives
 *     dx += 2 X x,  X the symmetric d x d block-diagonal matrix with
 *     X_xy = X_yx = Y_(x,y),
 * i.e. dx = (dPsi + dPsi^T) x for each block (the chunked backward's closing
 * step for queries and keys). */
static void phi_mg_vjp(const double* Y, const double* x, long d, long g, double* dx) {
  long m = d / g, nm = m * (m + 1) / 2;
  for (long blk = 0; blk < g; ++blk)
    for (long a = 0; a < m; ++a)
      for (long b = a; b < m; ++b) {
        double y = Y[blk * nm + kata_oracle_packed_index(a, b, m)];
        long xa = blk * m + a, xb = blk * m + b;
        if (a == b) {
          dx[xa] += 2.0 * y * x[xa];
        } else {
          dx[xa] += 2.0 * y * x[xb];
          dx[xb] += 2.0 * y * x[xa];
        }
      }
}

/* Chunkwise backward (the chunked backward of the appendix's chunkwise
 * algorithm: a reverse scan over chunks carrying the state cotangent, forward
 * quantities recomputed from the chunk-boundary states, and the feature-map VJP
 * closing the chain), for the KATA-Mg forward:
 *   forward:  S_loc, z_loc per chunk, exclusive prefix S_pre, z_pre; per token
 *             D_t, o_t from the chunk output, then a_t, b_t;
 *   backward: dS_loc = sum_{t in c} psi(q_t) a_t^T, dz_loc = sum_t b_t psi(q_t);
 *             exclusive suffix dS_suf[c] = sum_{c' > c} dS_loc[c'] (the scan of
 *             the reversed sequence of chunks, scan_mode 0 sequential, 1 tree);
 *   per chunk: dq_t = VJP(S_pre a_t + b_t z_pre) at q_t + in-chunk terms,
 *              dk_i = VJP(dS_suf v_i + dz_suf) at k_i + in-chunk terms,
 *              dv_i = dS_suf^T psi_w(k_i) + sum_{t in c, t >= i} w_ti a_t. */
EXPORT void kata_oracle_bwd_chunked_mg(const double* q, const double* k, const double* v,
                                       const double* dout, double* dq, double* dk, double* dvo,
                                       long B, long H, long T, long d, long dv, long C, long g,
                                       int scan_mode) {
  long n = kata_oracle_packed_dim_mg(d, g);
  long NC = (T + C - 1) / C;
  long BH = B * H, m = d / g;
  long SE = n * dv + n;
#pragma omp parallel for schedule(dynamic, 1)
  for (long bh = 0; bh < BH; ++bh) {
    const double* Q = q + bh * T * d;
    const double* K = k + bh * T * d;
    const double* V = v + bh * T * dv;
    const double* G = dout + bh * T * dv;
    double* dQ = dq + bh * T * d;
    double* dK = dk + bh * T * d;
    double* dV = dvo + bh * T * dv;
    double* fst = (double*)calloc((size_t)(NC * SE), sizeof(double));
    double* bst = (double*)calloc((size_t)(NC * SE), sizeof(double));
    double* A = (double*)calloc((size_t)(T * dv), sizeof(double));
    double* bv = (double*)calloc((size_t)T, sizeof(double));
    double* ph = (double*)malloc((size_t)n * sizeof(double));
    double* pw = (double*)malloc((size_t)n * sizeof(double));
    double* Y = (double*)malloc((size_t)n * sizeof(double));
    double* s = (double*)malloc((size_t)g * sizeof(double));
    /* forward chunk states and their exclusive prefix */
    for (long t = 0; t < T; ++t) {
      double* St = fst + (t / C) * SE;
      kata_oracle_phi_mg(K + t * d, d, g, 0, ph);
      for (long f = 0; f < n; ++f) {
        for (long j = 0; j < dv; ++j) St[f * dv + j] += ph[f] * V[t * dv + j];
        St[n * dv + f] += ph[f];
      }
    }
    kata_oracle_scan_exclusive(fst, NC, SE, scan_mode);
    /* forward readout per token: D_t, o_t, then a_t, b_t */
    for (long t = 0; t < T; ++t) {
      long c = t / C, t0 = c * C;
      const double* St = fst + c * SE;
      kata_oracle_phi_mg(Q + t * d, d, g, 1, pw);
      double D = 0.0, go = 0.0;
      /* the A row holds N_t first, then a_t */
      for (long f = 0; f < n; ++f) D += pw[f] * St[n * dv + f];
      for (long j = 0; j < dv; ++j) {
        double acc = 0.0;
        for (long f = 0; f < n; ++f) acc += pw[f] * St[f * dv + j];
        A[t * dv + j] = acc; /* N_t, inter part */
      }
      for (long i = t0; i <= t; ++i) {
        double w = 0.0;
        for (long a = 0; a < g; ++a) {
          double sa = 0.0;
          for (long x = a * m; x < (a + 1) * m; ++x) sa += Q[t * d + x] * K[i * d + x];
          w += sa * sa;
        }
        D += w;
        for (long j = 0; j < dv; ++j) A[t * dv + j] += w * V[i * dv + j];
      }
      if (D > 0.0) {
        for (long j = 0; j < dv; ++j) go += G[t * dv + j] * (A[t * dv + j] / D);
        for (long j = 0; j < dv; ++j) A[t * dv + j] = G[t * dv + j] / D;
        bv[t] = -go / D;
      } else {
        for (long j = 0; j < dv; ++j) A[t * dv + j] = 0.0;
        bv[t] = 0.0;
      }
    }
    /* backward chunk states, reversed in chunk order, and their exclusive
     * prefix = the exclusive suffix in the original order */
    for (long t = 0; t < T; ++t) {
      double* Bt = bst + (NC - 1 - t / C) * SE;
      kata_oracle_phi_mg(Q + t * d, d, g, 0, ph);
      for (long f = 0; f < n; ++f) {
        for (long j = 0; j < dv; ++j) Bt[f * dv + j] += ph[f] * A[t * dv + j];
        Bt[n * dv + f] += bv[t] * ph[f];
      }
    }
    kata_oracle_scan_exclusive(bst, NC, SE, scan_mode);
    memset(dQ, 0, (size_t)(T * d) * sizeof(double));
    memset(dK, 0, (size_t)(T * d) * sizeof(double));
    memset(dV, 0, (size_t)(T * dv) * sizeof(double));
    for (long t = 0; t < T; ++t) {
      long c = t / C, t0 = c * C;
      const double* St = fst + c * SE;                 /* S_pre, z_pre */
      const double* Bs = bst + (NC - 1 - c) * SE;      /* dS_suf, dz_suf */
      /* inter-chunk terms of token t as a query, then as a key */
      for (long f = 0; f < n; ++f) {
        double y = bv[t] * St[n * dv + f];
        for (long j = 0; j < dv; ++j) y += St[f * dv + j] * A[t * dv + j];
        Y[f] = y;
      }
      phi_mg_vjp(Y, Q + t * d, d, g, dQ + t * d);
      for (long f = 0; f < n; ++f) {
        double y = Bs[n * dv + f];
        for (long j = 0; j < dv; ++j) y += Bs[f * dv + j] * V[t * dv + j];
        Y[f] = y;
      }
      phi_mg_vjp(Y, K + t * d, d, g, dK + t * d);
      kata_oracle_phi_mg(K + t * d, d, g, 1, pw);
      for (long j = 0; j < dv; ++j) {
        double acc = 0.0;
        for (long f = 0; f < n; ++f) acc += pw[f] * Bs[f * dv + j];
        dV[t * dv + j] += acc;
      }
      /* in-chunk pairs (t as the query, i <= t in the same chunk) */
      for (long i = t0; i <= t; ++i) {
        double w = 0.0;
        for (long a = 0; a < g; ++a) {
          s[a] = 0.0;
          for (long x = a * m; x < (a + 1) * m; ++x) s[a] += Q[t * d + x] * K[i * d + x];
          w += s[a] * s[a];
        }
        double cw = bv[t];
        for (long j = 0; j < dv; ++j) {
          cw += A[t * dv + j] * V[i * dv + j];
          dV[i * dv + j] += w * A[t * dv + j];
        }
        for (long a = 0; a < g; ++a)
          for (long x = a * m; x < (a + 1) * m; ++x) {
            dQ[t * d + x] += 2.0 * cw * s[a] * K[i * d + x];
            dK[i * d + x] += 2.0 * cw * s[a] * Q[t * d + x];
          }
      }
    }
    free(fst); free(bst); free(A); free(bv); free(ph); free(pw); free(Y); free(s);
  }
}

/*
 * Denominators of the definition: den[bh][t] = sum_{i<=t} (q_t . k_i)^2, the
 * normaliser phi(q_t)^T sum_{i<=t} phi(k_i) of eq. linatt with the rank-one
 * PSD feature (<phi(q), phi(k)> = (q . k)^2); [B][H][T].
 */
EXPORT void kata_oracle_den(const double* q, const double* k, double* den, long B, long H,
                            long T, long d) {
  long BH = B * H;
#pragma omp parallel for collapse(2) schedule(dynamic, 16)
  for (long bh = 0; bh < BH; ++bh)
    for (long t = 0; t < T; ++t) {
      const double* qt = q + (bh * T + t) * d;
      double D = 0.0;
      for (long i = 0; i <= t; ++i) {
        const double* ki = k + (bh * T + i) * d;
        double s = 0.0;
        for (long a = 0; a < d; ++a) s += qt[a] * ki[a];
        D += s * s;
      }
      den[bh * T + t] = D;
    }
}
