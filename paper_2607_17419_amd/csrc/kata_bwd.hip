// kata_bwd.hip -- O(T) chunked backward of the causal KATA-Mg forward (g = 1
// is KATA-M1), fp32 VALU kernels for d <= 64, dv <= 256, C <= 64, fp32 or bf16
// inputs, fp32 gradients.
//
// For the loss with output cotangents dout_t = dL/do_t, with N_t, D_t the
// numerator and denominator of o_t = N_t / D_t:
//   a_t = dout_t / D_t,  b_t = -<dout_t, o_t> / D_t  (0 when D_t = 0, where
//   the readout is the constant 0),  dL/dw_ti = <a_t, v_i> + b_t  (i <= t).
// The pass follows the chunked backward of the appendix's chunkwise algorithm:
// a reverse scan over chunks carries the state cotangent, forward quantities
// are recomputed from the chunk-boundary states, and the feature-map VJP
// dx = (dPsi + dPsi^T) x closes the chain.  Six launches:
//   1. chunk states of the forward (S_loc = psi(K)^T V, z_loc = psi(K)^T 1),
//   2. their exclusive prefix (associative scan),
//   3. per token D_t from the prefix and the in-chunk weights, then (a_t, b_t),
//   4. backward chunk states dS_loc = psi(Q)^T A, dz_loc = psi(Q)^T b,
//   5. their exclusive suffix (the same scan over the chunks in reverse),
//   6. per chunk: dq from S_pre a_t + b_t z_pre and the in-chunk pairs, dk from
//      dS_suf v_i + dz_suf and the in-chunk pairs, dv from dS_suf^T psi_w(k_i)
//      and the in-chunk weights.
// Feature layout and records as on the fp32 forward path: packed pairs (x, y),
// x <= y, of each block of m = d/g coordinates; a record is S[f][j] (n x dv)
// then z[f] (n), fp32.
#include "kata_common.hpp"
#include "kata_internal.hpp"
#include "kata_scan.hpp"

namespace kata {

namespace {

struct BwdUnitWeight {
  __device__ __forceinline__ float operator()(long long) const { return 1.f; }
};

// Pair table of the packed block features: entry f holds (x, y) in the
// low / high byte.  Block-wide.
__device__ __forceinline__ void bwd_pair_table(uint16_t* tab, int d, int g) {
  const int m = d / g, nm = m * (m + 1) / 2;
  for (int x = threadIdx.x; x < d; x += blockDim.x) {
    const int blk = x / m, a = x % m;
    for (int b = a; b < m; ++b)
      tab[blk * nm + packed_index(a, b, m)] =
          static_cast<uint16_t>((blk * m + a) | ((blk * m + b) << 8));
  }
}

__host__ __device__ __forceinline__ int bwd_n(int d, int g) {
  return g * ((d / g) * (d / g + 1) / 2);
}

constexpr int kBFB = 16;  // features per workgroup of the state kernels
constexpr int kBTB = 32;  // tokens staged per pass

// ---------------------------------------------------------------------------
// Chunk states over the tokens of chunk c:
//   S[f][j] = sum_t psi_f(x_t) y_tj  (j < dv),   z[f] = sum_t wt_t psi_f(x_t)
// with psi_f(x) = x_a x_b (unscaled).  Forward: x = k, y = v, wt = 1.
// Backward: x = q, y = a (row stride dv + 1), wt = b (the last column).
// grid (ceil(n / kBFB), NC, BH), block 256.
// ---------------------------------------------------------------------------
template <typename Tx, typename Ty, bool kWeightedZ>
__global__ __launch_bounds__(256) void bwd_chunk_state(const Tx* __restrict__ x,
                                                       const Ty* __restrict__ y, int y_stride,
                                                       float* __restrict__ rec, int T, int d,
                                                       int dv, int C, int g, long long bh_stride,
                                                       long long E) {
  __shared__ float xs[kBTB][65];
  __shared__ float ys[kBTB][258];
  __shared__ uint16_t pairs[kBFB];
  const int n = bwd_n(d, g);
  const int m = d / g, nm = m * (m + 1) / 2;
  const int f0 = blockIdx.x * kBFB;
  const int c = blockIdx.y, bh = blockIdx.z;
  const int tid = threadIdx.x;
  if (tid < kBFB && f0 + tid < n) {
    const int f = f0 + tid, blk = f / nm, fl = f % nm;
    int a = 0;
    while (a + 1 < m && packed_index(a + 1, a + 1, m) <= fl) ++a;
    const int b = a + (fl - packed_index(a, a, m));
    pairs[tid] = static_cast<uint16_t>((blk * m + a) | ((blk * m + b) << 8));
  }
  const int nf = min(kBFB, n - f0);
  const int nout = nf * dv;
  constexpr int R = kBFB;  // at most kBFB * 256 outputs (dv <= 256)
  float acc[R];
#pragma unroll
  for (int r = 0; r < R; ++r) acc[r] = 0.f;
  float zacc = 0.f;
  const long long tb = static_cast<long long>(c) * C;
  const long long te = min(static_cast<long long>(T), tb + C);
  const Tx* xh = x + static_cast<long long>(bh) * T * d;
  const Ty* yh = y + static_cast<long long>(bh) * T * y_stride;
  for (long long t0 = tb; t0 < te; t0 += kBTB) {
    const int nt = static_cast<int>(min(static_cast<long long>(kBTB), te - t0));
    __syncthreads();
    for (int i = tid; i < kBTB * d; i += 256) {
      const int t = i / d, a = i % d;
      xs[t][a] = (t < nt) ? load_f32(xh, (t0 + t) * d + a) : 0.f;
    }
    const int yw = kWeightedZ ? dv + 1 : dv;
    for (int i = tid; i < kBTB * yw; i += 256) {
      const int t = i / yw, j = i % yw;
      ys[t][j] = (t < nt) ? load_f32(yh, (t0 + t) * y_stride + j) : 0.f;
    }
    __syncthreads();
#pragma unroll
    for (int r = 0; r < R; ++r) {
      const int o = tid + 256 * r;
      if (o < nout) {
        const int fl = o / dv, j = o % dv;
        const int a = pairs[fl] & 0xFF, b = pairs[fl] >> 8;
        float s = acc[r];
        for (int t = 0; t < nt; ++t) s += (xs[t][a] * xs[t][b]) * ys[t][j];
        acc[r] = s;
      }
    }
    if (tid < nf) {
      const int a = pairs[tid] & 0xFF, b = pairs[tid] >> 8;
      for (int t = 0; t < nt; ++t) zacc += (kWeightedZ ? ys[t][dv] : 1.f) * xs[t][a] * xs[t][b];
    }
  }
  float* r0 = rec + bh * bh_stride + c * E;
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const int o = tid + 256 * r;
    if (o < nout) r0[static_cast<long long>(f0) * dv + o] = acc[r];
  }
  if (tid < nf) r0[static_cast<long long>(n) * dv + f0 + tid] = zacc;
}

// ---------------------------------------------------------------------------
// Per-token coefficients: D_t = psi_w(q_t) . z_pre + sum_{s <= t in chunk} w_ts,
// ab[t] = (dout_t / D_t, -<dout_t, o_t> / D_t), zeros when D_t = 0.
// grid (NC, BH), block 256, dynamic LDS (2 C d + C) floats + n uint16.
// ---------------------------------------------------------------------------
template <typename Tin>
__global__ __launch_bounds__(256) void bwd_coef(const Tin* __restrict__ q,
                                                const Tin* __restrict__ k,
                                                const float* __restrict__ o,
                                                const float* __restrict__ dout,
                                                const float* __restrict__ frec,
                                                float* __restrict__ ab, int T, int d, int dv, int C,
                                                int g, long long bh_stride, long long E) {
  extern __shared__ float bsm[];
  const int n = bwd_n(d, g), m = d / g;
  float* qs = bsm;            // [C][d]
  float* ks = qs + C * d;     // [C][d]
  float* Dn = ks + C * d;     // [C]
  uint16_t* pairs = reinterpret_cast<uint16_t*>(Dn + C);
  const int c = blockIdx.x, bh = blockIdx.y, tid = threadIdx.x;
  const long long t0 = static_cast<long long>(c) * C;
  const int nt = static_cast<int>(min(static_cast<long long>(C), T - t0));
  const Tin* qh = q + static_cast<long long>(bh) * T * d;
  const Tin* kh = k + static_cast<long long>(bh) * T * d;
  bwd_pair_table(pairs, d, g);
  for (int i = tid; i < C * d; i += 256) {
    const int r = i / d, a = i % d;
    qs[i] = (r < nt) ? load_f32(qh, (t0 + r) * d + a) : 0.f;
    ks[i] = (r < nt) ? load_f32(kh, (t0 + r) * d + a) : 0.f;
  }
  __syncthreads();
  const float* zp = frec + bh * bh_stride + c * E + static_cast<long long>(n) * dv;
  for (int r = tid; r < nt; r += 256) {
    float D = 0.f;
    for (int f = 0; f < n; ++f) {
      const int a = pairs[f] & 0xFF, b = pairs[f] >> 8;
      D += ((a == b) ? 1.f : 2.f) * qs[r * d + a] * qs[r * d + b] * zp[f];
    }
    for (int s = 0; s <= r; ++s)
      for (int blk = 0; blk < g; ++blk) {
        float sc = 0.f;
        for (int x = blk * m; x < blk * m + m; ++x) sc += qs[r * d + x] * ks[s * d + x];
        D += sc * sc;
      }
    Dn[r] = D;
  }
  __syncthreads();
  for (int r = tid; r < nt; r += 256) {
    const long long row = static_cast<long long>(bh) * T + t0 + r;
    const float D = Dn[r];
    float go = 0.f;
    for (int j = 0; j < dv; ++j) go += dout[row * dv + j] * o[row * dv + j];
    float* abr = ab + row * (dv + 1);
    const float inv = D > 0.f ? 1.f / D : 0.f;
    for (int j = 0; j < dv; ++j) abr[j] = dout[row * dv + j] * inv;
    abr[dv] = -go * inv;
  }
}

// ---------------------------------------------------------------------------
// Gradients of chunk c.  grid (NC, BH), block 256, dynamic LDS
// (4 C d + 3 C C + 2 C kYB) floats + n uint16 (C <= 64, d <= 64).
// ---------------------------------------------------------------------------
constexpr int kYB = 32;  // features per pass of the inter-chunk VJP

template <typename Tin>
__global__ __launch_bounds__(256) void bwd_grad(const Tin* __restrict__ q,
                                                const Tin* __restrict__ k,
                                                const Tin* __restrict__ v,
                                                const float* __restrict__ ab,
                                                const float* __restrict__ frec,
                                                const float* __restrict__ brec,
                                                float* __restrict__ dq, float* __restrict__ dk,
                                                float* __restrict__ dvo, int T, int d, int dv,
                                                int C, int g, long long bh_stride, long long E) {
  extern __shared__ float bsm[];
  const int n = bwd_n(d, g), m = d / g;
  float* qs = bsm;             // [C][d]
  float* ks = qs + C * d;      // [C][d]
  float* dqs = ks + C * d;     // [C][d]
  float* dks = dqs + C * d;    // [C][d]
  float* cs = dks + C * d;     // [C][C]  dL/dw_ti (i <= t)
  float* sb = cs + C * C;      // [C][C]  block scores
  float* W = sb + C * C;       // [C][C]  weights w_ti (i <= t)
  float* Yq = W + C * C;       // [C][kYB]
  float* Yk = Yq + C * kYB;    // [C][kYB]
  uint16_t* pairs = reinterpret_cast<uint16_t*>(Yk + C * kYB);
  const int c = blockIdx.x, bh = blockIdx.y, tid = threadIdx.x;
  const long long t0 = static_cast<long long>(c) * C;
  const int nt = static_cast<int>(min(static_cast<long long>(C), T - t0));
  const long long hb = static_cast<long long>(bh) * T;
  const Tin* qh = q + hb * d;
  const Tin* kh = k + hb * d;
  const Tin* vh = v + hb * dv;
  const float* abh = ab + hb * (dv + 1);
  bwd_pair_table(pairs, d, g);
  for (int i = tid; i < C * d; i += 256) {
    const int r = i / d, a = i % d;
    qs[i] = (r < nt) ? load_f32(qh, (t0 + r) * d + a) : 0.f;
    ks[i] = (r < nt) ? load_f32(kh, (t0 + r) * d + a) : 0.f;
    dqs[i] = 0.f;
    dks[i] = 0.f;
  }
  for (int i = tid; i < C * C; i += 256) {
    const int t = i / C, s = i % C;
    float cw = 0.f;
    if (s <= t && t < nt) {
      const float* at = abh + (t0 + t) * (dv + 1);
      cw = at[dv];
      for (int j = 0; j < dv; ++j) cw += at[j] * load_f32(vh, (t0 + s) * dv + j);
    }
    cs[i] = cw;
    W[i] = 0.f;
  }
  __syncthreads();
  // in-chunk pairs, one feature block at a time
  for (int blk = 0; blk < g; ++blk) {
    for (int i = tid; i < C * C; i += 256) {
      const int t = i / C, s = i % C;
      float sc = 0.f;
      if (s <= t)
        for (int x = blk * m; x < blk * m + m; ++x) sc += qs[t * d + x] * ks[s * d + x];
      sb[i] = sc;
      W[i] += sc * sc;
    }
    __syncthreads();
    for (int i = tid; i < C * m; i += 256) {
      const int t = i / m, x = blk * m + i % m;
      float aq = 0.f, ak = 0.f;
      for (int s = 0; s <= t; ++s) aq += cs[t * C + s] * sb[t * C + s] * ks[s * d + x];
      for (int u = t; u < C; ++u) ak += cs[u * C + t] * sb[u * C + t] * qs[u * d + x];
      dqs[t * d + x] += 2.f * aq;  // row t as the query
      dks[t * d + x] += 2.f * ak;  // row t as the key
    }
    __syncthreads();
  }
  // dv: in-chunk weights, then the suffix state read with the key-side lift
  const float* Bs = brec + bh * bh_stride + c * E;  // dS_suf, then dz_suf
  for (int o = tid; o < nt * dv; o += 256) {
    const int i = o / dv, j = o % dv;
    float acc = 0.f;
    for (int t = i; t < nt; ++t) acc += W[t * C + i] * abh[(t0 + t) * (dv + 1) + j];
    for (int f = 0; f < n; ++f) {
      const int a = pairs[f] & 0xFF, b = pairs[f] >> 8;
      acc += ((a == b) ? 1.f : 2.f) * ks[i * d + a] * ks[i * d + b] *
             Bs[static_cast<long long>(f) * dv + j];
    }
    dvo[(hb + t0 + i) * dv + j] = acc;
  }
  // inter-chunk dq, dk: feature cotangents Y (query side from the prefix,
  // key side from the suffix) and their VJP, kYB features per pass
  const float* Sp = frec + bh * bh_stride + c * E;  // S_pre, then z_pre
  for (int f0 = 0; f0 < n; f0 += kYB) {
    const int nf = min(kYB, n - f0);
    __syncthreads();
    for (int i = tid; i < C * kYB; i += 256) {
      const int t = i / kYB, fl = i % kYB, f = f0 + fl;
      float yq = 0.f, yk = 0.f;
      if (fl < nf && t < nt) {
        const float* at = abh + (t0 + t) * (dv + 1);
        yq = at[dv] * Sp[static_cast<long long>(n) * dv + f];
        yk = Bs[static_cast<long long>(n) * dv + f];
        for (int j = 0; j < dv; ++j) {
          yq += Sp[static_cast<long long>(f) * dv + j] * at[j];
          yk += Bs[static_cast<long long>(f) * dv + j] * load_f32(vh, (t0 + t) * dv + j);
        }
      }
      Yq[i] = yq;
      Yk[i] = yk;
    }
    __syncthreads();
    for (int i = tid; i < C * kYB; i += 256) {
      const int t = i / kYB, fl = i % kYB;
      if (fl >= nf || t >= nt) continue;
      const int a = pairs[f0 + fl] & 0xFF, b = pairs[f0 + fl] >> 8;
      const float yq = 2.f * Yq[i], yk = 2.f * Yk[i];
      if (a == b) {
        atomicAdd(&dqs[t * d + a], yq * qs[t * d + a]);
        atomicAdd(&dks[t * d + a], yk * ks[t * d + a]);
      } else {
        atomicAdd(&dqs[t * d + a], yq * qs[t * d + b]);
        atomicAdd(&dqs[t * d + b], yq * qs[t * d + a]);
        atomicAdd(&dks[t * d + a], yk * ks[t * d + b]);
        atomicAdd(&dks[t * d + b], yk * ks[t * d + a]);
      }
    }
  }
  __syncthreads();
  for (int i = tid; i < nt * d; i += 256) {
    dq[(hb + t0) * d + i] = dqs[i];
    dk[(hb + t0) * d + i] = dks[i];
  }
}

size_t bwd_grad_smem(int d, int C, int g) {
  const size_t n = static_cast<size_t>(bwd_n(d, g));
  return (4 * static_cast<size_t>(C) * d + 3 * static_cast<size_t>(C) * C +
          2 * static_cast<size_t>(C) * kYB) * sizeof(float) + n * sizeof(uint16_t);
}

size_t bwd_coef_smem(int d, int C, int g) {
  const size_t n = static_cast<size_t>(bwd_n(d, g));
  return (2 * static_cast<size_t>(C) * d + C) * sizeof(float) + n * sizeof(uint16_t);
}

}  // namespace

size_t bwd_workspace(int BH, int T, int d, int dv, int C, int g) {
  const size_t n = static_cast<size_t>(bwd_n(d, g));
  const size_t NC = (static_cast<size_t>(T) + C - 1) / C;
  const size_t rec = n * dv + n;
  return static_cast<size_t>(BH) * (2 * NC * rec + static_cast<size_t>(T) * (dv + 1)) *
         sizeof(float);
}

bool bwd_supported(int d, int dv, int C, int g) {
  return d >= 1 && d <= 64 && dv >= 1 && dv <= 256 && C >= 1 && C <= 64 && g >= 1 &&
         d % g == 0 && bwd_grad_smem(d, C, g) <= 160 * 1024;
}

template <typename Tin>
hipError_t launch_bwd(const void* q, const void* k, const void* v, const float* out,
                      const float* dout, float* dq, float* dk, float* dv_out, int BH, int T,
                      int d, int dv, int C, int g, void* ws, hipStream_t st, hipEvent_t* ev) {
  const int n = bwd_n(d, g);
  const int NC = (T + C - 1) / C;
  const long long E = static_cast<long long>(n) * dv + n;
  const long long bh_stride = E * NC;
  float* frec = static_cast<float*>(ws);
  float* brec = frec + static_cast<size_t>(BH) * bh_stride;
  float* ab = brec + static_cast<size_t>(BH) * bh_stride;
  const Tin* qi = static_cast<const Tin*>(q);
  const Tin* ki = static_cast<const Tin*>(k);
  const Tin* vi = static_cast<const Tin*>(v);
  const dim3 gs((n + kBFB - 1) / kBFB, NC, BH);
  const dim3 gscan(static_cast<unsigned>((E + kEB - 1) / kEB), BH);
  hipError_t e = record(ev, 0, st);
  if (e != hipSuccess) return e;
  bwd_chunk_state<Tin, Tin, false><<<gs, 256, 0, st>>>(ki, vi, dv, frec, T, d, dv, C, g,
                                                      bh_stride, E);
  if ((e = record(ev, 1, st)) != hipSuccess) return e;
  scan_exclusive<float, BwdUnitWeight, false><<<gscan, 256, 0, st>>>(frec, frec, NC, E, bh_stride,
                                                                    BwdUnitWeight{});
  if ((e = record(ev, 2, st)) != hipSuccess) return e;
  const size_t cshm = bwd_coef_smem(d, C, g);
  bwd_coef<Tin><<<dim3(NC, BH), 256, cshm, st>>>(qi, ki, out, dout, frec, ab, T, d, dv, C, g,
                                                 bh_stride, E);
  if ((e = record(ev, 3, st)) != hipSuccess) return e;
  bwd_chunk_state<Tin, float, true><<<gs, 256, 0, st>>>(qi, ab, dv + 1, brec, T, d, dv, C, g,
                                                       bh_stride, E);
  if ((e = record(ev, 4, st)) != hipSuccess) return e;
  scan_exclusive<float, BwdUnitWeight, true><<<gscan, 256, 0, st>>>(brec, brec, NC, E, bh_stride,
                                                                   BwdUnitWeight{});
  if ((e = record(ev, 5, st)) != hipSuccess) return e;
  const size_t gshm = bwd_grad_smem(d, C, g);
  if (gshm > 65536) {
    e = hipFuncSetAttribute(reinterpret_cast<const void*>(&bwd_grad<Tin>),
                            hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(gshm));
    if (e != hipSuccess) return e;
  }
  bwd_grad<Tin><<<dim3(NC, BH), 256, gshm, st>>>(qi, ki, vi, ab, frec, brec, dq, dk, dv_out, T, d,
                                                 dv, C, g, bh_stride, E);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  return record(ev, 6, st);
}

template hipError_t launch_bwd<float>(const void*, const void*, const void*, const float*,
                                      const float*, float*, float*, float*, int, int, int, int,
                                      int, int, void*, hipStream_t, hipEvent_t*);
template hipError_t launch_bwd<bf16_t>(const void*, const void*, const void*, const float*,
                                       const float*, float*, float*, float*, int, int, int, int,
                                       int, int, void*, hipStream_t, hipEvent_t*);

}  // namespace kata
