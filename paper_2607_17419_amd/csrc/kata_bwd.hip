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
#include <type_traits>

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

typedef float mf32x16 __attribute__((ext_vector_type(16)));

__device__ __forceinline__ mf32x16 mfma_f32(float a, float b, mf32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
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
// Per-token coefficients: D_t = q_t^T Z_pre q_t + sum_{s <= t in chunk} w_ts,
// with Z_pre the prefix z (fp32, chunk c at zsrc + bh z_bh + c z_c, diagonal
// features scaled by zdiag) unpacked into a symmetric d x d matrix (zero across
// feature blocks), then ab[t] = (dout_t / D_t, -<dout_t, o_t> / D_t), zeros
// when D_t = 0.  Both sums are contractions on the fp32 matrix cores
// (v_mfma_f32_32x32x2_f32): wave w takes the coordinate / key tile w >> 1 and
// the token tile w & 1 of  Y = Z_pre Q^T  (then q_t . Y[:, t] over its rows)
// and of the block scores  Sc_b = K_b Q_b^T  (squared, s <= t); the two tiles'
// partial sums meet in LDS.  Four lanes per token then form a_t | b_t.
// grid (NC, BH), block 256 (C <= 64), dynamic LDS bwd_coef_smem.
// ---------------------------------------------------------------------------
constexpr int kCS = 65;  // fp32 row stride of the coefficient kernel's tiles

// Eight consecutive elements as fp32 (p 16-byte aligned).
__device__ __forceinline__ void load8_f32(const bf16_t* p, float* v) {
  const uint4 w = *reinterpret_cast<const uint4*>(p);
  const uint32_t u[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    v[2 * e] = bf16lo_f32(u[e]);
    v[2 * e + 1] = bf16hi_f32(u[e]);
  }
}
__device__ __forceinline__ void load8_f32(const float* p, float* v) {
  const float4 a = reinterpret_cast<const float4*>(p)[0];
  const float4 b = reinterpret_cast<const float4*>(p)[1];
  v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
  v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
}

template <typename Tin>
__global__ __launch_bounds__(256) void bwd_coef(const Tin* __restrict__ q,
                                                const Tin* __restrict__ k,
                                                const float* __restrict__ o,
                                                const float* __restrict__ dout,
                                                const float* __restrict__ zsrc,
                                                float* __restrict__ ab, int T, int d, int dv, int C,
                                                int g, long long z_bh, long long z_c,
                                                float zdiag) {
  extern __shared__ float bsm[];
  const int m = d / g, nm = m * (m + 1) / 2;
  float* Z = bsm;             // [64][kCS] unpacked z_pre
  float* qs = Z + 64 * kCS;   // [64][kCS]
  float* ks = qs + 64 * kCS;  // [64][kCS]
  float* red = ks + 64 * kCS;  // [2][64] partial D of the two coordinate tiles
  const int c = blockIdx.x, bh = blockIdx.y, tid = threadIdx.x;
  const long long t0 = static_cast<long long>(c) * C;
  const int nt = static_cast<int>(min(static_cast<long long>(C), T - t0));
  const Tin* qh = q + (static_cast<long long>(bh) * T + t0) * d;
  const Tin* kh = k + (static_cast<long long>(bh) * T + t0) * d;
  const float* zp = zsrc + bh * z_bh + c * z_c;
  // the output and cotangent rows of the epilogue (4 lanes per token, columns
  // p, p + 4, ...), loaded first so that they arrive under the contractions
  // dv = 64: sixteen lanes per token, four tokens per wave at a time (token
  // 16 w + 4 it + lane / 16, 16-byte piece lane % 16), so that each load reads
  // four whole rows; other dv: four lanes per token, columns p, p + 4, ...
  const int sub = (tid & 63) >> 4, pc = tid & 15, w6 = tid >> 6;
  const bool pre = dv == 64;
  float4 dre4[4], ore4[4];
  if (pre) {
#pragma unroll
    for (int it = 0; it < 4; ++it) {
      const int rt = 16 * w6 + 4 * it + sub;
      dre4[it] = ore4[it] = make_float4(0.f, 0.f, 0.f, 0.f);
      if (rt < nt) {
        const long long rowt = static_cast<long long>(bh) * T + t0 + rt;
        dre4[it] = reinterpret_cast<const float4*>(dout + rowt * 64)[pc];
        ore4[it] = reinterpret_cast<const float4*>(o + rowt * 64)[pc];
      }
    }
  }
  // z_pre (g nm <= 2080 floats) is read once, coalesced, into the k tile's
  // LDS and unpacked from there; q and k rows are read in 8-element pieces
  // (16 bytes of bf16) where d allows it, k held in registers until every
  // read of the staged z_pre is done
  float* zl = ks;
  static_assert(64 * kCS >= 2080, "the packed z_pre fits the k tile");
  for (int i = tid; i < g * nm; i += 256) zl[i] = zp[i];
  __syncthreads();
  for (int i = tid; i < 64 * 64; i += 256) {
    const int x = i >> 6, y = i & 63;
    float zv = 0.f;
    if (g == 1) {  // one block: no block index to divide out
      if (x < d && y < d) zv = zl[packed_index(min(x, y), max(x, y), d)];
    } else if (x < d && y < d && x / m == y / m) {
      zv = zl[(x / m) * nm + packed_index(min(x, y) % m, max(x, y) % m, m)];
    }
    Z[x * kCS + y] = (x == y ? zdiag : 1.f) * zv;
  }
  // 8-element pieces need d % 8 == 0 and 16-byte aligned q, k (row starts are
  // then aligned too: t0 and every row offset are multiples of d)
  const bool vec = d % 8 == 0 && ((reinterpret_cast<uintptr_t>(q) | reinterpret_cast<uintptr_t>(k)) & 15) == 0;
  const int pieces = d / 8;  // 8-element pieces per row (vec)
  float kv[2][8];            // this thread's k pieces (vec: at most 64 x 8 / 256 = 2)
  if (vec) {
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int i = tid + 256 * j;
      if (i >= 64 * pieces) break;
      const int x = i / pieces, y0 = 8 * (i % pieces);
      float qv[8];
      if (x < nt) {
        load8_f32(qh + static_cast<long long>(x) * d + y0, qv);
        load8_f32(kh + static_cast<long long>(x) * d + y0, kv[j]);
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) qv[e] = kv[j][e] = 0.f;
      }
#pragma unroll
      for (int e = 0; e < 8; ++e) qs[x * kCS + y0 + e] = qv[e];
    }
  } else {
    for (int i = tid; i < 64 * 64; i += 256) {
      const int x = i >> 6, y = i & 63;
      const bool in = x < nt && y < d;
      qs[x * kCS + y] = in ? load_f32(qh, static_cast<long long>(x) * d + y) : 0.f;
    }
  }
  __syncthreads();  // every read of the staged z_pre is done: the k tile may be written
  if (vec) {
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int i = tid + 256 * j;
      if (i >= 64 * pieces) break;
      const int x = i / pieces, y0 = 8 * (i % pieces);
#pragma unroll
      for (int e = 0; e < 8; ++e) ks[x * kCS + y0 + e] = kv[j][e];
    }
  } else {
    for (int i = tid; i < 64 * 64; i += 256) {
      const int x = i >> 6, y = i & 63;
      const bool in = x < nt && y < d;
      ks[x * kCS + y] = in ? load_f32(kh, static_cast<long long>(x) * d + y) : 0.f;
    }
  }
  // columns d .. 63 of the q and k tiles are read by the contractions below
  // (K = 64): zero them when d < 64
  if (d < 64) {
    for (int i = tid; i < 64 * (64 - d); i += 256) {
      const int x = i / (64 - d), y = d + i % (64 - d);
      qs[x * kCS + y] = 0.f;
      ks[x * kCS + y] = 0.f;
    }
  }
  __syncthreads();
  {
    const int lane = tid & 63, w = tid >> 6, h = lane >> 5, l32 = lane & 31;
    const int X = w >> 1, t = 32 * (w & 1) + l32;
    const float* qt = qs + t * kCS;
    // prefix: Y[x][t] = sum_y Z[x][y] q_t[y] for the 32 rows x of tile X
    mf32x16 yz = {};
    const float* zr = Z + (32 * X + l32) * kCS;
    for (int s2 = 0; s2 < 32; ++s2) yz = mfma_f32(zr[2 * s2 + h], qt[2 * s2 + h], yz);
    float part = 0.f;
#pragma unroll
    for (int i = 0; i < 16; ++i) part += qt[32 * X + 8 * (i >> 2) + 4 * h + (i & 3)] * yz[i];
    // in-chunk: Sc_b[s][t] = sum_{x in block b} k_s[x] q_t[x] for the keys s of tile X
    const float* kr = ks + (32 * X + l32) * kCS;
    for (int blk = 0; blk < g; ++blk) {
      const int x0 = blk * m, x1 = x0 + m;
      mf32x16 sc = {};
      for (int xs = x0 & ~1; xs < x1; xs += 2) {
        const int x = xs + h;
        const bool inb = x >= x0 && x < x1;
        sc = mfma_f32(inb ? kr[x] : 0.f, inb ? qt[x] : 0.f, sc);
      }
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int s_ = 32 * X + 8 * (i >> 2) + 4 * h + (i & 3);
        if (s_ <= t) part += sc[i] * sc[i];
      }
    }
    part += __shfl_xor(part, 32);
    if (h == 0) red[X * 64 + t] = part;
  }
  __syncthreads();
  if (pre) {
#pragma unroll
    for (int it = 0; it < 4; ++it) {
      const int rt = 16 * w6 + 4 * it + sub;
      const float D = red[rt] + red[64 + rt];
      const float inv = D > 0.f ? 1.f / D : 0.f;
      const float4 x = dre4[it], y = ore4[it];
      float go = x.x * y.x + x.y * y.y + x.z * y.z + x.w * y.w;
#pragma unroll
      for (int m = 8; m > 0; m >>= 1) go += __shfl_xor(go, m);
      if (rt < nt) {  // ab rows are 65 floats apart: four 4-byte stores
        float* abr = ab + (static_cast<long long>(bh) * T + t0 + rt) * 65;
        abr[4 * pc] = x.x * inv;
        abr[4 * pc + 1] = x.y * inv;
        abr[4 * pc + 2] = x.z * inv;
        abr[4 * pc + 3] = x.w * inv;
        if (pc == 0) abr[64] = -go * inv;
      }
    }
    return;
  }
  const int r = tid >> 2, p = tid & 3;
  if (r < nt) {
    const long long row = static_cast<long long>(bh) * T + t0 + r;
    const float D = red[r] + red[64 + r];
    float* abr = ab + row * (dv + 1);
    const float inv = D > 0.f ? 1.f / D : 0.f;
    float go = 0.f;
    const float* dr = dout + row * dv;
    const float* orow = o + row * dv;
    for (int j = p; j < dv; j += 4) go += dr[j] * orow[j];
    for (int j = p; j < dv; j += 4) abr[j] = dr[j] * inv;
    go += __shfl_xor(go, 1);
    go += __shfl_xor(go, 2);
    if (p == 0) abr[dv] = -go * inv;
  }
}

// ---------------------------------------------------------------------------
// Per-token coefficients from denominators the forward pass saved (den[t] =
// D_t): ab[t] = (dout_t / D_t, -<dout_t, o_t> / D_t), zeros when D_t = 0, as
// bwd_coef forms them, without recomputing D_t from the prefix records.
// Sixteen lanes per token, so that each load instruction of a wave reads four
// whole rows (16-byte pieces when dv % 4 == 0; rows are then 16-byte aligned);
// the dot product meets over the 16 lanes.  A workgroup takes 64 tokens, each
// wave 16 of them four at a time.  grid (ceil(T / 64), BH), block 256.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void bwd_coef_den(const float* __restrict__ o,
                                                    const float* __restrict__ dout,
                                                    const float* __restrict__ den,
                                                    float* __restrict__ ab, int T, int dv) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int sub = lane >> 4, pc = lane & 15;
  const bool vec = (dv & 3) == 0;
#pragma unroll
  for (int it = 0; it < 4; ++it) {
    const long long t = static_cast<long long>(blockIdx.x) * 64 + 16 * w + 4 * it + sub;
    const bool ok = t < T;  // lanes past the sequence compute on its last row, store nothing
    const long long row = static_cast<long long>(blockIdx.y) * T + (ok ? t : T - 1);
    const float D = den[row];
    const float inv = D > 0.f ? 1.f / D : 0.f;
    const float* dr = dout + row * dv;
    const float* orow = o + row * dv;
    float* abr = ab + row * (dv + 1);
    float go = 0.f;
    if (vec) {
      for (int j4 = pc; 4 * j4 < dv; j4 += 16) {
        const float4 x = reinterpret_cast<const float4*>(dr)[j4];
        const float4 y = reinterpret_cast<const float4*>(orow)[j4];
        go += x.x * y.x + x.y * y.y + x.z * y.z + x.w * y.w;
        if (ok) {  // ab rows are dv + 1 floats apart: four 4-byte stores
          abr[4 * j4] = x.x * inv;
          abr[4 * j4 + 1] = x.y * inv;
          abr[4 * j4 + 2] = x.z * inv;
          abr[4 * j4 + 3] = x.w * inv;
        }
      }
    } else {
      for (int j = pc; j < dv; j += 16) {
        const float x = dr[j];
        go += x * orow[j];
        if (ok) abr[j] = x * inv;
      }
    }
#pragma unroll
    for (int m = 8; m > 0; m >>= 1) go += __shfl_xor(go, m);
    if (ok && pc == 0) abr[dv] = -go * inv;
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

// ===========================================================================
// fp32 matrix-core variants (v_mfma_f32_32x32x2_f32: lane l holds A[l % 32][l / 32]
// and B[l / 32][l % 32]; result column l % 32, rows 8 (i / 4) + 4 (l / 32) + i % 4),
// for C <= 64, d <= 64, dv <= 64.  Same arithmetic (fp32 products, fp32
// accumulation) as the VALU kernels above, in another summation order.  The
// coefficient kernel above uses the same instruction (mfma_f32).
// ===========================================================================

constexpr int kMS = 65;  // LDS row stride (floats) of the 64-row staging tiles

// Chunk states on the matrix cores: one workgroup per chunk stages the chunk's
// x and y rows once; its waves take the (feature tile fp, value tile vj)
// 32 x 32 tiles of S in turn, two tokens per MFMA; the tiles with vj = 0 also
// sum z.  grid (NC, BH), block 256.
template <typename Tx, typename Ty, bool kWeightedZ>
__global__ __launch_bounds__(256) void bwd_state_mf(const Tx* __restrict__ x,
                                                    const Ty* __restrict__ y, int y_stride,
                                                    float* __restrict__ rec, int T, int d, int dv,
                                                    int C, int g, long long bh_stride,
                                                    long long E) {
  __shared__ float xs[64 * kMS];
  __shared__ float ys[64 * (kMS + 1)];
  __shared__ uint16_t pairs[2080];
  const int n = bwd_n(d, g);
  const int c = blockIdx.x, bh = blockIdx.y, tid = threadIdx.x;
  const int lane = tid & 63, w = tid >> 6, h = lane >> 5, l32 = lane & 31;
  bwd_pair_table(pairs, d, g);
  const long long tb = static_cast<long long>(c) * C;
  const int nt = static_cast<int>(min(static_cast<long long>(C), T - tb));
  const Tx* xh = x + (static_cast<long long>(bh) * T + tb) * d;
  const Ty* yh = y + (static_cast<long long>(bh) * T + tb) * y_stride;
  const int yw = kWeightedZ ? dv + 1 : dv;
  for (int i = tid; i < 64 * d; i += 256) {
    const int t = i / d, a = i % d;
    xs[t * kMS + a] = (t < nt) ? load_f32(xh, static_cast<long long>(t) * d + a) : 0.f;
  }
  for (int i = tid; i < 64 * (kMS + 1); i += 256) {
    const int t = i / (kMS + 1), j = i % (kMS + 1);
    ys[i] = (t < nt && j < yw) ? load_f32(yh, static_cast<long long>(t) * y_stride + j) : 0.f;
  }
  __syncthreads();
  float* r0 = rec + bh * bh_stride + c * E;
  const int nft = (n + 31) / 32, nvt = (dv + 31) / 32;
  for (int tile = w; tile < nft * nvt; tile += 4) {
    const int fp = tile / nvt, vj = tile % nvt;
    const int p = 32 * fp + l32;
    // lanes of a partial last feature tile feed zeros and store nothing
    const uint16_t pr = pairs[p < n ? p : n - 1];
    const int pa = pr & 0xFF, pb = pr >> 8;
    const float pon = p < n ? 1.f : 0.f;
    const int jc = 32 * vj + l32;
    mf32x16 acc = {};
    float zp = 0.f;
    for (int s2 = 0; s2 < 32; ++s2) {
      const int t = 2 * s2 + h;
      const float a = pon * xs[t * kMS + pa] * xs[t * kMS + pb];
      acc = mfma_f32(a, ys[t * (kMS + 1) + jc], acc);  // staged zeros past dv
      if (vj == 0) zp += a * (kWeightedZ ? ys[t * (kMS + 1) + dv] : 1.f);
    }
    zp += __shfl_xor(zp, 32);
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int f = 32 * fp + 8 * (i >> 2) + 4 * h + (i & 3);
      if (f < n && jc < dv) r0[static_cast<long long>(f) * dv + jc] = acc[i];
    }
    if (vj == 0 && h == 0 && p < n) r0[static_cast<long long>(n) * dv + p] = zp;
  }
}

// LDS element type of the staged q, k, v rows: bf16 inputs stay bf16 (exact),
// which halves those tiles; fp32 inputs stay fp32.
template <typename Tin> struct GradLds { using T = float; static constexpr int S = kMS; };
template <> struct GradLds<bf16_t> { using T = uint16_t; static constexpr int S = kMS + 1; };
__device__ __forceinline__ float lds_f32(float x) { return x; }
__device__ __forceinline__ float lds_f32(uint16_t x) {
  return __uint_as_float(static_cast<uint32_t>(x) << 16);
}
__device__ __forceinline__ void lds_put(float* p, float x) { *p = x; }
__device__ __forceinline__ void lds_put(uint16_t* p, float x) {
  *p = static_cast<uint16_t>(__float_as_uint(x) >> 16);  // exact: x is a bf16 value
}
__device__ __forceinline__ float in_f32(const float* p, long long i) { return p[i]; }
__device__ __forceinline__ float in_f32(const bf16_t* p, long long i) { return to_f32(p[i]); }

// Gradients of chunk c with the inter-chunk products on the matrix cores.
// In-chunk terms in VALU with each thread's 16 (token, coordinate) and
// (token, value) entries kept in registers; inter-chunk terms as dense
// products over the symmetric states, one coordinate y at a time:
//   dq_t[x] += 2 sum_y q_t[y] (sum_j S[x,y][j] a_tj + b_t z[x,y])
//   dk_i[x] += 2 sum_y k_i[y] (sum_j dS[x,y][j] v_ij + dz[x,y])
//   dv_i[j] += sum_{x >= y} w_xy k_ix k_iy dS[x,y][j]      (w = 1 on x = y, else 2)
// with S[x,y] = S[y,x] the packed prefix row of the pair (0 across blocks)
// and dS the suffix row.  grid (NC, BH), block 256, dynamic LDS
// bwd_grad_mf_smem(...); two workgroups fit a CU for bf16 inputs.
template <typename Tin>
__global__ __launch_bounds__(256, 2) void bwd_grad_mf(const Tin* __restrict__ q,
                                                   const Tin* __restrict__ k,
                                                   const Tin* __restrict__ v,
                                                   const float* __restrict__ ab,
                                                   const float* __restrict__ frec,
                                                   const float* __restrict__ brec,
                                                   float* __restrict__ dq, float* __restrict__ dk,
                                                   float* __restrict__ dvo, int T, int d, int dv,
                                                   int C, int g, long long bh_stride,
                                                   long long E) {
  using LT = typename GradLds<Tin>::T;
  constexpr int LS = GradLds<Tin>::S;
  extern __shared__ float bsm[];
  const int n = bwd_n(d, g), m = d / g;
  float* as = bsm;                  // [64][kMS + 1]: a_t (dv), b_t at column dv
  float* cs = as + 64 * (kMS + 1);  // [64][kMS] dL/dw_ti; later the suffix slab SB
  float* sb = cs + 64 * kMS;        // [64][kMS] block scores; later the prefix slab SA
  LT* qs = reinterpret_cast<LT*>(sb + 64 * kMS);  // [64][LS]
  LT* ks = qs + 64 * LS;
  LT* vs = ks + 64 * LS;            // column dv holds 1 (the coefficient of dz)
  uint16_t* pairs = reinterpret_cast<uint16_t*>(vs + 64 * LS);
  const int c = blockIdx.x, bh = blockIdx.y, tid = threadIdx.x;
  const int lane = tid & 63, w = tid >> 6, h = lane >> 5, l32 = lane & 31;
  const long long t0 = static_cast<long long>(c) * C;
  const int nt = static_cast<int>(min(static_cast<long long>(C), T - t0));
  const long long hb = static_cast<long long>(bh) * T;
  const Tin* qh = q + (hb + t0) * d;
  const Tin* kh = k + (hb + t0) * d;
  const Tin* vh = v + (hb + t0) * dv;
  const float* abh = ab + (hb + t0) * (dv + 1);
  bwd_pair_table(pairs, d, g);
  for (int i = tid; i < 64 * LS; i += 256) {
    const int t = i / LS, a = i % LS;
    const bool in = t < nt;
    lds_put(&qs[i], (in && a < d) ? in_f32(qh, static_cast<long long>(t) * d + a) : 0.f);
    lds_put(&ks[i], (in && a < d) ? in_f32(kh, static_cast<long long>(t) * d + a) : 0.f);
    lds_put(&vs[i], (in && a < dv) ? in_f32(vh, static_cast<long long>(t) * dv + a)
                                   : (a == dv ? 1.f : 0.f));
  }
  for (int i = tid; i < 64 * (kMS + 1); i += 256) {
    const int t = i / (kMS + 1), j = i % (kMS + 1);
    as[i] = (t < nt && j <= dv) ? abh[static_cast<long long>(t) * (dv + 1) + j] : 0.f;
  }
  __syncthreads();
  // dL/dw_ti = <a_t, v_i> + b_t for i <= t
  for (int i = tid; i < 64 * 64; i += 256) {
    const int t = i >> 6, s2 = i & 63;
    float cw = 0.f;
    if (s2 <= t && t < nt) {
      cw = as[t * (kMS + 1) + dv];
      for (int j = 0; j < dv; ++j) cw += as[t * (kMS + 1) + j] * lds_f32(vs[s2 * LS + j]);
    }
    cs[t * kMS + s2] = cw;
  }
  // this thread's register entries: (token e >> 6, coordinate / value e & 63)
  // for e = tid + 256 r, r = 0..15
  float dqi[16], dki[16], dvi[16];
#pragma unroll
  for (int r = 0; r < 16; ++r) dqi[r] = dki[r] = dvi[r] = 0.f;
  __syncthreads();
  for (int blk = 0; blk < g; ++blk) {
    for (int i = tid; i < 64 * 64; i += 256) {
      const int t = i >> 6, s2 = i & 63;
      float sc = 0.f;
      if (s2 <= t)
        for (int x2 = blk * m; x2 < blk * m + m; ++x2)
          sc += lds_f32(qs[t * LS + x2]) * lds_f32(ks[s2 * LS + x2]);
      sb[t * kMS + s2] = sc;
    }
    __syncthreads();
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int e = tid + 256 * r, t = e >> 6, x2 = e & 63;
      if (x2 >= blk * m && x2 < blk * m + m && x2 < d) {
        float aq = 0.f, ak = 0.f;
        for (int s2 = 0; s2 <= t; ++s2)
          aq += cs[t * kMS + s2] * sb[t * kMS + s2] * lds_f32(ks[s2 * LS + x2]);
        for (int u = t; u < 64; ++u)
          ak += cs[u * kMS + t] * sb[u * kMS + t] * lds_f32(qs[u * LS + x2]);
        dqi[r] += 2.f * aq;  // row t as the query
        dki[r] += 2.f * ak;  // row t as the key
      }
      if (x2 < dv) {  // in-chunk dv of row t: sum_{u >= t} w_ut a_u over this block
        float av = 0.f;
        for (int u = t; u < nt; ++u) av += sb[u * kMS + t] * sb[u * kMS + t] * as[u * (kMS + 1) + x2];
        dvi[r] += av;
      }
    }
    __syncthreads();
  }
  // inter-chunk products: the y-slabs SA (prefix rows, z at column dv) and SB
  // (suffix rows, dz at column dv) over sb and cs; the next y's rows are
  // gathered into registers while this y is consumed
  float* SA = sb;
  float* SB = cs;
  const float* Sp = frec + bh * bh_stride + c * E;
  const float* Bs = brec + bh * bh_stride + c * E;
  const int nm = m * (m + 1) / 2;
  const int mi = w >> 1, nj = w & 1;  // this wave's token tile and value tile (dv)
  const int sx = tid >> 2, sq = tid & 3;  // staging: slab row x, column quarter
  float pA[16], pB[16], pzA = 0.f, pzB = 0.f;
  bool rin = false;
  // rows start 16-byte aligned when the record length and dv are multiples of
  // 4: then each thread fetches its 16 columns as four 16-byte loads
  const bool v4 = (E % 4 == 0) && (dv % 16 == 0);
  auto fetch = [&](int y) {
    rin = sx < d && sx / m == y / m;
    const int a = min(sx, y) % m, b = max(sx, y) % m;
    const long long f = rin ? static_cast<long long>(y / m) * nm + packed_index(a, b, m) : 0;
    if (v4) {
      const int c0 = min(16 * sq, dv - 16);  // clamped address; masked when written
#pragma unroll
      for (int e4 = 0; e4 < 4; ++e4) {
        const float4 ua = *reinterpret_cast<const float4*>(Sp + f * dv + c0 + 4 * e4);
        const float4 ub = *reinterpret_cast<const float4*>(Bs + f * dv + c0 + 4 * e4);
        pA[4 * e4] = ua.x; pA[4 * e4 + 1] = ua.y; pA[4 * e4 + 2] = ua.z; pA[4 * e4 + 3] = ua.w;
        pB[4 * e4] = ub.x; pB[4 * e4 + 1] = ub.y; pB[4 * e4 + 2] = ub.z; pB[4 * e4 + 3] = ub.w;
      }
    } else {
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int j = min(16 * sq + e, dv - 1);  // clamped address; masked when written
        pA[e] = Sp[f * dv + j];
        pB[e] = Bs[f * dv + j];
      }
    }
    pzA = Sp[static_cast<long long>(n) * dv + f];
    pzB = Bs[static_cast<long long>(n) * dv + f];
  };
  mf32x16 accx[2] = {{}, {}};  // waves 0-1: dq tiles, waves 2-3: dk tiles (x tile 0, 1)
  mf32x16 dvacc = {};
  const bool qside = w < 2;
  const int tt = 32 * (w & 1) + l32;  // A row of the dq / dk product: token
  const LT* Xr = (qside ? qs : ks) + tt * LS;
  const int nks = (dv + 2) / 2;       // K-steps over j = 0..dv (column dv: z)
  fetch(0);
  for (int y = 0; y < d; ++y) {
    __syncthreads();  // the previous y's readers are done with the slabs
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const int j = 16 * sq + e;
      const float za = (j == dv) ? pzA : 0.f, zb = (j == dv) ? pzB : 0.f;
      SA[sx * kMS + j] = rin ? (j < dv ? pA[e] : za) : 0.f;
      SB[sx * kMS + j] = rin ? (j < dv ? pB[e] : zb) : 0.f;
    }
    if (sq == 3) {
      SA[sx * kMS + 64] = (rin && dv == 64) ? pzA : 0.f;
      SB[sx * kMS + 64] = (rin && dv == 64) ? pzB : 0.f;
    }
    __syncthreads();
    fetch(y + 1 < d ? y + 1 : y);
    {
      // A: x_t[y] times a_tj (j < dv), b_t (j = dv) on the query side, v_ij
      // (j < dv), 1 (j = dv) on the key side; zero past dv.  Operands of step
      // s + 1 are loaded before the MFMAs of step s.
      const float xy = lds_f32(Xr[y]);
      const float* Bm = qside ? SA : SB;
      auto ldA = [&](int s2) {
        const int j = 2 * s2 + h, jj = j <= dv ? j : dv;
        const float av = qside ? as[tt * (kMS + 1) + jj] : lds_f32(vs[tt * LS + jj]);
        return (j <= dv ? xy : 0.f) * av;
      };
      auto ldB = [&](int s2, int xt) {
        const int j = 2 * s2 + h;
        return Bm[(32 * xt + l32) * kMS + (j <= dv ? j : dv)];
      };
      float a = ldA(0), b0 = ldB(0, 0), b1 = ldB(0, 1);
      for (int s2 = 0; s2 < nks; ++s2) {
        const int sn = s2 + 1 < nks ? s2 + 1 : s2;
        const float an = ldA(sn), b0n = ldB(sn, 0), b1n = ldB(sn, 1);
        accx[0] = mfma_f32(a, b0, accx[0]);
        accx[1] = mfma_f32(a, b1, accx[1]);
        a = an;
        b0 = b0n;
        b1 = b1n;
      }
    }
    {
      const int ti = 32 * mi + l32;
      const float ky = lds_f32(ks[ti * LS + y]);
      const int nx = (64 - y + 1) / 2;
      auto ldK = [&](int s2) {
        const int x2 = y + 2 * s2 + h;
        const int xc = x2 < 64 ? x2 : 63;
        const float wgt = x2 < 64 ? (x2 == y ? 1.f : 2.f) : 0.f;
        return wgt * ky * lds_f32(ks[ti * LS + xc]);
      };
      auto ldS = [&](int s2) {
        const int x2 = y + 2 * s2 + h;
        return SB[(x2 < 64 ? x2 : 63) * kMS + 32 * nj + l32];
      };
      float a = ldK(0), b = ldS(0);
      for (int s2 = 0; s2 < nx; ++s2) {
        const int sn = s2 + 1 < nx ? s2 + 1 : s2;
        const float an = ldK(sn), bn = ldS(sn);
        dvacc = mfma_f32(a, b, dvacc);
        a = an;
        b = bn;
      }
    }
  }
  __syncthreads();
  // the waves' products into LDS (dq over SA, dk over SB, dv over as), then
  // each thread adds its in-chunk register entries and writes them out
  {
    float* dP = qside ? SA : SB;
#pragma unroll
    for (int xt = 0; xt < 2; ++xt)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int t = 32 * (w & 1) + 8 * (i >> 2) + 4 * h + (i & 3);
        dP[t * kMS + 32 * xt + l32] = 2.f * accx[xt][i];
      }
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int r = 32 * mi + 8 * (i >> 2) + 4 * h + (i & 3);
      as[r * (kMS + 1) + 32 * nj + l32] = dvacc[i];
    }
  }
  __syncthreads();
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    const int e = tid + 256 * r, t = e >> 6, x2 = e & 63;
    if (t < nt && x2 < d) {
      dq[(hb + t0 + t) * d + x2] = dqi[r] + SA[t * kMS + x2];
      dk[(hb + t0 + t) * d + x2] = dki[r] + SB[t * kMS + x2];
    }
    if (t < nt && x2 < dv) dvo[(hb + t0 + t) * dv + x2] = dvi[r] + as[t * (kMS + 1) + x2];
  }
}

size_t bwd_grad_mf_smem(int d, int g, bool bf16_lds) {
  const size_t n = static_cast<size_t>(bwd_n(d, g));
  const size_t f32 = (static_cast<size_t>(64) * (kMS + 1) + 2 * 64 * kMS) * sizeof(float);
  const size_t xyz = bf16_lds ? 3 * 64 * (kMS + 1) * sizeof(uint16_t) : 3 * 64 * kMS * sizeof(float);
  return f32 + xyz + n * sizeof(uint16_t);
}

bool bwd_mf_ok(int d, int dv, int C) { return d <= 64 && dv <= 64 && C <= 64; }


size_t bwd_grad_smem(int d, int C, int g) {
  const size_t n = static_cast<size_t>(bwd_n(d, g));
  return (4 * static_cast<size_t>(C) * d + 3 * static_cast<size_t>(C) * C +
          2 * static_cast<size_t>(C) * kYB) * sizeof(float) + n * sizeof(uint16_t);
}

size_t bwd_coef_smem(int, int, int) { return (3 * 64 * kCS + 2 * 64) * sizeof(float); }

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
         d % g == 0 && bwd_grad_smem(d, C, g) <= 160 * 1024 &&
         (!bwd_mf_ok(d, dv, C) || bwd_grad_mf_smem(d, g, false) <= 160 * 1024);
}

template <typename Tin>
hipError_t launch_bwd(const void* q, const void* k, const void* v, const float* out,
                      const float* dout, const float* den, float* dq, float* dk, float* dv_out,
                      int BH, int T, int d, int dv, int C, int g, void* ws, hipStream_t st,
                      hipEvent_t* ev) {
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
  const bool mf = bwd_mf_ok(d, dv, C);
  const dim3 gsm(NC, BH);
  // bf16 inputs at d = dv = C = 64, g = 1: chunk states and gradients on the
  // bf16 matrix cores
  // (the C ABI has checked that every tensor is 16-byte aligned)
  bool bf = false;
  if constexpr (std::is_same<Tin, bf16_t>::value) bf = bwd_bf_ok(d, dv, C, g);
  // bf16 path: from bwd_bf_fused_min_heads() heads on, each state launch also
  // scans (one pass, sequential over a head's chunks); with fewer heads the
  // chunk-parallel state launch and the record scan are faster
  const bool fused = bf && bwd_fused_scan(BH, d, dv, C, g, true);
  hipError_t e = record(ev, 0, st);
  if (e != hipSuccess) return e;
  if (fused) {
    if ((e = launch_bwd_prefix_bf(false, k, v, frec, BH, T, st)) != hipSuccess) return e;
  } else if (bf) {
    if ((e = launch_bwd_state_bf(false, k, v, frec, BH, T, st)) != hipSuccess) return e;
  } else if (mf)
    bwd_state_mf<Tin, Tin, false><<<gsm, 256, 0, st>>>(ki, vi, dv, frec, T, d, dv, C, g,
                                                      bh_stride, E);
  else
    bwd_chunk_state<Tin, Tin, false><<<gs, 256, 0, st>>>(ki, vi, dv, frec, T, d, dv, C, g,
                                                        bh_stride, E);
  if ((e = record(ev, 1, st)) != hipSuccess) return e;
  const bool v4 = E % 4 == 0;
  const dim3 gscan4(static_cast<unsigned>((E + kEB4 - 1) / kEB4), BH);
  if (fused) {
    // scanned by the state launch
  } else if (bf) {
    if ((e = launch_bwd_scan_bf(false, frec, BH, T, st)) != hipSuccess) return e;
  } else if (v4)
    scan_exclusive_f32x4<BwdUnitWeight, false><<<gscan4, 256, 0, st>>>(frec, NC, E, bh_stride,
                                                                      BwdUnitWeight{});
  else
    scan_exclusive<float, BwdUnitWeight, false><<<gscan, 256, 0, st>>>(frec, frec, NC, E,
                                                                      bh_stride, BwdUnitWeight{});
  if ((e = record(ev, 2, st)) != hipSuccess) return e;
  const size_t cshm = bwd_coef_smem(d, C, g);
  // z_pre: fp32 after S in both record layouts; the bf16-state records carry
  // the diagonal features halved
  const long long rq = static_cast<long long>(bwd_bf_record_bytes() / sizeof(float));
  const float* zsrc = bf ? reinterpret_cast<const float*>(reinterpret_cast<const char*>(frec) +
                                                          bwd_bf_record_bytes() - 4 * n)
                         : frec + static_cast<long long>(n) * dv;
  if (den != nullptr)
    bwd_coef_den<<<dim3((T + 63) / 64, BH), 256, 0, st>>>(out, dout, den, ab, T, dv);
  else
    bwd_coef<Tin><<<dim3(NC, BH), 256, cshm, st>>>(qi, ki, out, dout, zsrc, ab, T, d, dv, C, g,
                                                   bf ? NC * rq : bh_stride, bf ? rq : E,
                                                   bf ? 2.f : 1.f);
  if ((e = record(ev, 3, st)) != hipSuccess) return e;
  if (fused) {
    if ((e = launch_bwd_prefix_bf(true, q, ab, brec, BH, T, st)) != hipSuccess) return e;
  } else if (bf) {
    if ((e = launch_bwd_state_bf(true, q, ab, brec, BH, T, st)) != hipSuccess) return e;
  } else if (mf)
    bwd_state_mf<Tin, float, true><<<gsm, 256, 0, st>>>(qi, ab, dv + 1, brec, T, d, dv, C, g,
                                                       bh_stride, E);
  else
    bwd_chunk_state<Tin, float, true><<<gs, 256, 0, st>>>(qi, ab, dv + 1, brec, T, d, dv, C, g,
                                                         bh_stride, E);
  if ((e = record(ev, 4, st)) != hipSuccess) return e;
  if (fused) {
    // scanned by the state launch
  } else if (bf) {
    if ((e = launch_bwd_scan_bf(true, brec, BH, T, st)) != hipSuccess) return e;
  } else if (v4)
    scan_exclusive_f32x4<BwdUnitWeight, true><<<gscan4, 256, 0, st>>>(brec, NC, E, bh_stride,
                                                                     BwdUnitWeight{});
  else
    scan_exclusive<float, BwdUnitWeight, true><<<gscan, 256, 0, st>>>(brec, brec, NC, E,
                                                                     bh_stride, BwdUnitWeight{});
  if ((e = record(ev, 5, st)) != hipSuccess) return e;
  if (bf) {
    e = launch_bwd_grad_bf(q, k, v, ab, frec, brec, dq, dk, dv_out, BH, T, st);
    if (e != hipSuccess) return e;
  } else if (mf) {
    const size_t gshm = bwd_grad_mf_smem(d, g, sizeof(Tin) == 2);
    e = hipFuncSetAttribute(reinterpret_cast<const void*>(&bwd_grad_mf<Tin>),
                            hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(gshm));
    if (e != hipSuccess) return e;
    bwd_grad_mf<Tin><<<dim3(NC, BH), 256, gshm, st>>>(qi, ki, vi, ab, frec, brec, dq, dk, dv_out,
                                                      T, d, dv, C, g, bh_stride, E);
  } else {
    const size_t gshm = bwd_grad_smem(d, C, g);
    if (gshm > 65536) {
      e = hipFuncSetAttribute(reinterpret_cast<const void*>(&bwd_grad<Tin>),
                              hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(gshm));
      if (e != hipSuccess) return e;
    }
    bwd_grad<Tin><<<dim3(NC, BH), 256, gshm, st>>>(qi, ki, vi, ab, frec, brec, dq, dk, dv_out, T,
                                                   d, dv, C, g, bh_stride, E);
  }
  if ((e = hipGetLastError()) != hipSuccess) return e;
  return record(ev, 6, st);
}

template hipError_t launch_bwd<float>(const void*, const void*, const void*, const float*,
                                      const float*, const float*, float*, float*, float*, int,
                                      int, int, int, int, int, void*, hipStream_t, hipEvent_t*);
template hipError_t launch_bwd<bf16_t>(const void*, const void*, const void*, const float*,
                                       const float*, const float*, float*, float*, float*, int,
                                       int, int, int, int, int, void*, hipStream_t, hipEvent_t*);

}  // namespace kata
