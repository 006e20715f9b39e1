// kata_linear.hip -- causal linear attention with the linear (n_psi ~ d)
// feature maps: psi(x) = x, the orthant maps ReLU(x) + eps and ELU(x) + 1
// (section "Classical feature maps"), the Lorentz lift (x, ||x||) of the same
// section and the n_psi = d Lorentz variant of the appendix KATA-Lorentz
// model, (x_1..x_{d-1}, ||x_1..x_{d-1}|| (1 + x_d^2)).  The readout is either
// normalised, o_t = psi(q_t)^T S_t / psi(q_t)^T z_t (eq. linatt; 0 unless the
// denominator is positive), or plain, o_t = psi(q_t)^T S_t (the signed kernel
// of unnormalised linear attention).
//
// Both paths run the three-stage pipeline of the associative-scan appendix
// (paragraph "Three-kernel pipeline"): a state kernel writes each record's
// local S_loc = psi(K)^T V and z_loc = psi(K)^T 1 (fp32, record = S row-major
// [n][dv] then z [n]); the associative (Blelloch) scan of kata_scan.hpp turns
// the records into exclusive prefixes in place; an output kernel combines each
// record's prefix with the causal pattern inside the record.
//  - fp32 path: one record per chunk of C tokens, fp32 arithmetic, any
//    feature, d <= 64, dv <= 256, C <= 128, fp32 or bf16 inputs.
//  - bf16 MFMA path (d = dv = 64; every feature): one record per span of L
//    tokens (a multiple of 64); inside a span the output kernel walks 64-token
//    chunks in order and carries the running state on chip.  Every d x d
//    contraction is a v_mfma_f32_32x32x16_bf16 with fp32 accumulation.  The
//    Lorentz lift's extra coordinate ||x|| is a rank-one addition to the
//    weights, <psi(q), psi(k)> = q . k + ||q|| ||k||: it adds one state row
//    sum ||k|| v^T and one normaliser term sum ||k||, kept in fp32 beside
//    the d x d part, and the term ||q|| ||k|| to each in-chunk score.
#include <cmath>

#include "kata_internal.hpp"
#include "kata_scan.hpp"

namespace kata {

// Unit weight of the prefix scan over linear-feature records (a type of its
// own, so this file's scan instantiation is not shared with another file's).
struct LinUnitWeight {
  __device__ __forceinline__ float operator()(long long) const { return 1.f; }
};

// ===========================================================================
// fp32 path
// ===========================================================================

__device__ __forceinline__ float lin_psi_scalar(float x, int feature, float eps) {
  if (feature == kLinRelu) return fmaxf(x, 0.f) + eps;
  if (feature == kLinElu) return x > 0.f ? x + 1.f : expf(x);
  return x;  // identity, and the raw coordinates of both Lorentz maps
}

// Feature rows of tokens t0 .. t0 + rows - 1 into f[rows][n]; rows at or past
// `tlim` are all zeros (a padded token carries no feature).  Block-wide.
template <typename Tin>
__device__ void lin_feature_rows(const Tin* x, float* f, long long t0, int rows, long long tlim,
                                 int d, int n, int feature, float eps) {
  for (int i = threadIdx.x; i < rows * d; i += blockDim.x) {
    const int r = i / d, a = i % d;
    const long long t = t0 + r;
    f[r * n + a] = (t < tlim) ? lin_psi_scalar(load_f32(x, t * d + a), feature, eps) : 0.f;
  }
  __syncthreads();
  if (feature == kLinLorentz || feature == kLinLorentzS) {
    const int m = (feature == kLinLorentz) ? d : d - 1;  // coordinates inside the norm
    for (int r = threadIdx.x; r < rows; r += blockDim.x) {
      float s = 0.f;
      for (int a = 0; a < m; ++a) s += f[r * n + a] * f[r * n + a];
      const bool live = t0 + r < tlim;
      if (feature == kLinLorentz) {
        f[r * n + d] = live ? sqrtf(s) : 0.f;
      } else {
        const float z = f[r * n + d - 1];
        f[r * n + d - 1] = live ? sqrtf(s) * (1.f + z * z) : 0.f;
      }
    }
  }
  __syncthreads();
}

// Chunk-state stage: rec[bh][c] = (psi(K_c)^T V_c, psi(K_c)^T 1).
// grid (NC, BH), block 256, dynamic LDS C * n floats.
template <typename Tin>
__global__ __launch_bounds__(256) void lin_state_f32(const Tin* k, const Tin* v, float* rec, int T,
                                                     int d, int dv, int C, int feature, float eps,
                                                     long long bh_stride, long long E) {
  extern __shared__ float lin_sm[];
  const int n = lin_dim(d, feature);
  float* fk = lin_sm;  // [C][n]
  const int c = blockIdx.x, bh = blockIdx.y;
  const long long t0 = static_cast<long long>(c) * C;
  const Tin* kb = k + static_cast<long long>(bh) * T * d;
  const Tin* vb = v + static_cast<long long>(bh) * T * dv;
  lin_feature_rows(kb, fk, t0, C, T, d, n, feature, eps);
  const int rows = static_cast<int>(T - t0 < C ? T - t0 : C);
  float* r = rec + bh * bh_stride + c * E;
  const int nS = n * dv;
  for (int e = threadIdx.x; e < nS + n; e += blockDim.x) {
    float acc = 0.f;
    if (e < nS) {
      const int f = e / dv, j = e % dv;
      for (int s = 0; s < rows; ++s) acc += fk[s * n + f] * load_f32(vb, (t0 + s) * dv + j);
    } else {
      const int f = e - nS;
      for (int s = 0; s < rows; ++s) acc += fk[s * n + f];
    }
    r[e] = acc;
  }
}

// Chunk-output stage for 32 queries of chunk c: prefix readout plus the causal
// in-chunk weights, then the normalisation.  grid (NC * ceil(C / 32), BH),
// block 256, dynamic LDS (32 n + C n + 32 C + 32) floats.
template <typename Tin>
__global__ __launch_bounds__(256) void lin_out_f32(const Tin* q, const Tin* k, const Tin* v,
                                                   const float* rec, float* out, int T, int d,
                                                   int dv, int C, int feature, float eps,
                                                   int normalize, long long bh_stride,
                                                   long long E) {
  extern __shared__ float lin_sm[];
  const int n = lin_dim(d, feature);
  const int QT = (C + 31) / 32;
  const int c = blockIdx.x / QT, qt = blockIdx.x % QT, bh = blockIdx.y;
  const long long t0 = static_cast<long long>(c) * C;
  const int r0 = qt * 32;                       // first query row inside the chunk
  const int qrows = C - r0 < 32 ? C - r0 : 32;  // query rows of this block
  float* fq = lin_sm;          // [32][n]
  float* fk = fq + 32 * n;     // [C][n]
  float* w = fk + C * n;       // [32][C]
  float* den = w + 32 * C;     // [32]
  const Tin* qb = q + static_cast<long long>(bh) * T * d;
  const Tin* kb = k + static_cast<long long>(bh) * T * d;
  const Tin* vb = v + static_cast<long long>(bh) * T * dv;
  const long long qlim = t0 + r0 + qrows < T ? t0 + r0 + qrows : T;
  lin_feature_rows(qb, fq, t0 + r0, 32, qlim, d, n, feature, eps);
  lin_feature_rows(kb, fk, t0, C, T, d, n, feature, eps);
  for (int i = threadIdx.x; i < 32 * C; i += blockDim.x) {
    const int r = i / C, s = i % C;
    float a = 0.f;
    if (s <= r0 + r) {
      for (int f = 0; f < n; ++f) a += fq[r * n + f] * fk[s * n + f];
    }
    w[i] = a;  // keys past T have a zero feature row, so their weight is 0
  }
  __syncthreads();
  const float* pre = rec + bh * bh_stride + c * E;  // exclusive prefix (S_pre, z_pre)
  const float* zpre = pre + static_cast<long long>(n) * dv;
  if (threadIdx.x < 32) {
    const int r = threadIdx.x;
    float D = 0.f;
    for (int f = 0; f < n; ++f) D += fq[r * n + f] * zpre[f];
    for (int s = 0; s < C; ++s) D += w[r * C + s];
    den[r] = D;
  }
  __syncthreads();
  for (int i = threadIdx.x; i < 32 * dv; i += blockDim.x) {
    const int r = i / dv, j = i % dv;
    const long long t = t0 + r0 + r;
    if (r >= qrows || t >= T) continue;
    float o = 0.f;
    for (int f = 0; f < n; ++f) o += fq[r * n + f] * pre[f * dv + j];
    const int smax = r0 + r;
    for (int s = 0; s <= smax && t0 + s < T; ++s) o += w[r * C + s] * load_f32(vb, (t0 + s) * dv + j);
    if (normalize) o = den[r] > 0.f ? o / den[r] : 0.f;
    out[(static_cast<long long>(bh) * T + t) * dv + j] = o;
  }
}

size_t lin_fp32_workspace(int BH, int T, int d, int dv, int C, int feature) {
  const long long n = lin_dim(d, feature);
  const long long NC = (static_cast<long long>(T) + C - 1) / C;
  return static_cast<size_t>(BH) * NC * (n * dv + n) * sizeof(float);
}

template <typename Tin>
hipError_t launch_lin_fp32(const void* q, const void* k, const void* v, float* out, int BH, int T,
                           int d, int dv, int C, int feature, float eps, int normalize, void* ws,
                           hipStream_t st, hipEvent_t* ev) {
  const int n = lin_dim(d, feature);
  const int NC = (T + C - 1) / C;
  const long long E = static_cast<long long>(n) * dv + n;
  const long long bh_stride = E * NC;
  float* rec = static_cast<float*>(ws);
  hipError_t e = record(ev, 0, st);
  if (e != hipSuccess) return e;
  lin_state_f32<Tin><<<dim3(NC, BH), 256, static_cast<size_t>(C) * n * sizeof(float), st>>>(
      static_cast<const Tin*>(k), static_cast<const Tin*>(v), rec, T, d, dv, C, feature, eps,
      bh_stride, E);
  if ((e = record(ev, 1, st)) != hipSuccess) return e;
  scan_exclusive<float, LinUnitWeight><<<dim3(static_cast<unsigned>((E + kEB - 1) / kEB), BH),
                                         256, 0, st>>>(rec, rec, NC, E, bh_stride,
                                                       LinUnitWeight{});
  if ((e = record(ev, 2, st)) != hipSuccess) return e;
  const size_t shm = (static_cast<size_t>(32) * n + static_cast<size_t>(C) * n + 32 * C + 32) *
                     sizeof(float);
  const int QT = (C + 31) / 32;
  lin_out_f32<Tin><<<dim3(NC * QT, BH), 256, shm, st>>>(
      static_cast<const Tin*>(q), static_cast<const Tin*>(k), static_cast<const Tin*>(v), rec,
      out, T, d, dv, C, feature, eps, normalize, bh_stride, E);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  return record(ev, 3, st);
}

template hipError_t launch_lin_fp32<float>(const void*, const void*, const void*, float*, int,
                                           int, int, int, int, int, float, int, void*,
                                           hipStream_t, hipEvent_t*);
template hipError_t launch_lin_fp32<bf16_t>(const void*, const void*, const void*, float*, int,
                                            int, int, int, int, int, float, int, void*,
                                            hipStream_t, hipEvent_t*);

// ===========================================================================
// bf16 MFMA path (d = dv = 64, n_psi = 64)
//
// MFMA operand layout (v_mfma_f32_32x32x16_bf16): lane l holds, of A (32 x 16),
// row l % 32 and k = 8 (l / 32) .. +7; of B (16 x 32), column l % 32 and the
// same k; of the fp32 result, column l % 32 and rows 8 (i / 4) + 4 (l / 32) +
// i % 4 for i = 0..15.
//
// LDS tiles are 64 rows of 64 bf16 at a stride of kLS = 72 elements (144
// bytes), so that the 16-byte operand reads of 16 consecutive rows fall in
// distinct bank groups:
//   kt  psi(K)^T  [feature][token]   A of the state update S += psi(K)^T V
//   vt  V^T       [value col][token] B of the update, A of O^T += V^T P^T
//   kr  psi(K)    [token][feature]   A of the scores P^T = psi(K) psi(Q)^T
//   st  S^T       [value col][feature], bf16 copy of the running state, A of
//                 the readout O^T += S^T psi(Q)^T
// Queries enter as the B operand psi(Q)^T straight from HBM (a lane loads the
// 16-byte runs of its own query row), so O^T comes out with one query per
// lane and the denominator of that query is lane-local.
// ===========================================================================

constexpr int kLD = 64;   // feature / value width of the MFMA path
constexpr int kLCH = 64;  // tokens per chunk inside a span
constexpr int kLS = 72;   // LDS row stride (bf16 elements)
constexpr long long kLE = static_cast<long long>(kLD) * kLD + kLD;  // record: S then z
// Lorentz-lift record: the d x d record, then the extra state row
// sum ||k|| v^T (kLD values), then sum ||k|| and three zeros (a multiple of
// four elements for the scan's 16-byte accesses).
constexpr long long kLEL = kLE + kLD + 4;
template <int F>
constexpr long long lin_record() { return F == kLinLorentz ? kLEL : kLE; }
// Raw-buffer descriptor word 3 (32-bit data format, no swizzle) of gfx9-class
// buffer resources; out-of-range accesses are dropped.
constexpr int kBufWord3 = 0x00020000;
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
// Byte offsets into one head's output rows (up to T + 63 rows of 256 bytes)
// must fit 31 bits.
constexpr long long kLinMaxT = (1LL << 31) / (kLD * 4) - kLCH;

template <int F>
__device__ __forceinline__ float lin_psi(float x, float eps) {
  if constexpr (F == kLinRelu) return fmaxf(x, 0.f) + eps;
  else if constexpr (F == kLinElu) return x > 0.f ? x + 1.f : __expf(x);
  else return x;
}

__device__ __forceinline__ void unpack8(const uint4& u, float* x) {
  const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    x[2 * i] = bf16lo_f32(w[i]);
    x[2 * i + 1] = bf16hi_f32(w[i]);
  }
}

__device__ __forceinline__ bf16x8 pack8(const float* x) {
  uint4 u;
  u.x = pack_bf16x2(x[0], x[1]);
  u.y = pack_bf16x2(x[2], x[3]);
  u.z = pack_bf16x2(x[4], x[5]);
  u.w = pack_bf16x2(x[6], x[7]);
  return __builtin_bit_cast(bf16x8, u);
}

__device__ __forceinline__ float sum8(const bf16x8& a) {
  const uint4 u = __builtin_bit_cast(uint4, a);
  return bf16lo_f32(u.x) + bf16hi_f32(u.x) + bf16lo_f32(u.y) + bf16hi_f32(u.y) +
         bf16lo_f32(u.z) + bf16hi_f32(u.z) + bf16lo_f32(u.w) + bf16hi_f32(u.w);
}

__device__ __forceinline__ f32x16 lin_mfma(const bf16x8& a, const bf16x8& b, const f32x16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ bf16x8 lds8(const uint16_t* p) {
  return *reinterpret_cast<const bf16x8*>(p);
}

// Staging of one 64-token chunk of K and V by the whole workgroup: thread
// (fg = tid % 8, tp = tid / 8) loads features 8 fg .. 8 fg + 7 of tokens 2 tp
// and 2 tp + 1 (16 bytes each; eight consecutive lanes cover a 128-byte row).
struct LinStage {
  uint4 k[2], v[2];
  bool live[2];
};

// Loads are unconditional (a padded token re-reads the last real row; its
// values are zeroed when used), so that no branch joins a pending load and
// the loads of the next chunks stay in flight across the current one.
__device__ __forceinline__ void lin_stage_load(LinStage& s, const uint16_t* kb, const uint16_t* vb,
                                               long long tc, long long tend, int fg, int tp) {
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const long long t = tc + 2 * tp + i;
    s.live[i] = t < tend;
    const long long tr = s.live[i] ? t : tend - 1;
    s.k[i] = *reinterpret_cast<const uint4*>(kb + tr * kLD + 8 * fg);
    s.v[i] = *reinterpret_cast<const uint4*>(vb + tr * kLD + 8 * fg);
  }
}

// Staged value rows as fp32, zero rows for padded tokens.
__device__ __forceinline__ void lin_stage_values(const LinStage& s, float (*y)[8]) {
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    unpack8(s.v[i], y[i]);
#pragma unroll
    for (int e = 0; e < 8; ++e) y[i][e] = s.live[i] ? y[i][e] : 0.f;
  }
}

// psi of the staged key rows (fp32), zero rows for padded tokens.  The
// Lorentz variant's norm runs over the eight lanes that share a token.
template <int F>
__device__ __forceinline__ void lin_stage_features(const LinStage& s, float (*x)[8], float eps,
                                                   int fg) {
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    unpack8(s.k[i], x[i]);
    if constexpr (F == kLinLorentzS) {
      float nrm = 0.f;
#pragma unroll
      for (int e = 0; e < 8; ++e) nrm += (fg == 7 && e == 7) ? 0.f : x[i][e] * x[i][e];
      nrm += __shfl_xor(nrm, 1);
      nrm += __shfl_xor(nrm, 2);
      nrm += __shfl_xor(nrm, 4);
      if (fg == 7) x[i][7] = sqrtf(nrm) * (1.f + x[i][7] * x[i][7]);
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e) x[i][e] = lin_psi<F>(x[i][e], eps);
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) x[i][e] = s.live[i] ? x[i][e] : 0.f;
  }
}

// ||x|| of the thread's two staged key rows (raw coordinates, zero rows for
// padded tokens): the eight lanes that share a token combine their parts.
__device__ __forceinline__ void lin_row_norms(const float (*x)[8], float* nk) {
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    float s = 0.f;
#pragma unroll
    for (int e = 0; e < 8; ++e) s += x[i][e] * x[i][e];
    s += __shfl_xor(s, 1);
    s += __shfl_xor(s, 2);
    s += __shfl_xor(s, 4);
    nk[i] = sqrtf(s);
  }
}

// Wave w's share of a chunk's Lorentz-lift state row: lane j sums
// nk[t] * V^T[j][t] over the chunk's tokens 16 w .. 16 w + 15 (V^T rows of
// stride kLS in LDS, bf16).
__device__ __forceinline__ float lin_lift_part(const uint16_t* vt, const float* nk, int w,
                                               int lane) {
  const uint4 u0 = *reinterpret_cast<const uint4*>(&vt[lane * kLS + 16 * w]);
  const uint4 u1 = *reinterpret_cast<const uint4*>(&vt[lane * kLS + 16 * w + 8]);
  float y[16];
  unpack8(u0, y);
  unpack8(u1, y + 8);
  float acc = 0.f;
#pragma unroll
  for (int t = 0; t < 16; ++t) acc += nk[16 * w + t] * y[t];
  return acc;
}

// Transposed LDS writes: element e of the thread's two tokens goes to row
// 8 fg + e, columns 2 tp and 2 tp + 1 (one 4-byte write).
__device__ __forceinline__ void lin_write_t(uint16_t* dst, const float (*x)[8], int fg, int tp) {
#pragma unroll
  for (int e = 0; e < 8; ++e)
    *reinterpret_cast<uint32_t*>(dst + (8 * fg + e) * kLS + 2 * tp) = pack_bf16x2(x[0][e], x[1][e]);
}

// ---------------------------------------------------------------------------
// Span-state stage: rec[bh][s] = (psi(K)^T V, psi(K)^T 1) over the span's
// tokens.  Wave w owns the 32 x 32 tile (feature block w / 2, value block
// w % 2) of S; waves 0 and 2 also sum their feature rows into z.
// grid BH * NS (1-D), block 256.
// ---------------------------------------------------------------------------
template <int F>
__global__ __launch_bounds__(256) void lin_span_state(const uint16_t* k, const uint16_t* v,
                                                      float* rec, int T, int L, int NS, float eps) {
  __shared__ __align__(16) uint16_t kt[2][kLD * kLS];
  __shared__ __align__(16) uint16_t vt[2][kLD * kLS];
  constexpr bool LIFT = F == kLinLorentz;
  __shared__ __align__(16) float nks[LIFT ? 2 : 1][LIFT ? kLCH : 1];  // ||k|| per chunk token
  __shared__ float red[LIFT ? 4 : 1][LIFT ? kLD + 1 : 1];
  const int bh = blockIdx.x / NS, sp = blockIdx.x % NS;
  const long long tbeg = static_cast<long long>(sp) * L;
  const long long tend = tbeg + L < T ? tbeg + L : T;
  const int nch = static_cast<int>((tend - tbeg + kLCH - 1) / kLCH);
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, h = lane >> 5, l32 = lane & 31;
  const int fg = tid & 7, tp = tid >> 3;
  const int fb = w >> 1, vb2 = w & 1;
  const uint16_t* kb = k + static_cast<long long>(bh) * T * kLD;
  const uint16_t* vb = v + static_cast<long long>(bh) * T * kLD;

  f32x16 acc;
#pragma unroll
  for (int i = 0; i < 16; ++i) acc[i] = 0.f;
  float zp = 0.f;
  float lift = 0.f, liftz = 0.f;  // lane j: sum ||k|| v_j and sum ||k|| over the wave's tokens
  // two chunks in flight: chunk ch + 2 is loaded into the registers chunk ch
  // has just left, right after the barrier that publishes chunk ch
  LinStage s0, s1;
  lin_stage_load(s0, kb, vb, tbeg, tend, fg, tp);
  if (nch > 1) lin_stage_load(s1, kb, vb, tbeg + kLCH, tend, fg, tp);
  auto step = [&](LinStage& sg, int ch) {
    const int buf = ch & 1;
    float x[2][8], y[2][8];
    lin_stage_features<F>(sg, x, eps, fg);
    lin_stage_values(sg, y);
    lin_write_t(kt[buf], x, fg, tp);
    lin_write_t(vt[buf], y, fg, tp);
    if constexpr (LIFT) {
      float nk[2];
      lin_row_norms(x, nk);
      if (fg == 0) {
        nks[buf][2 * tp] = nk[0];
        nks[buf][2 * tp + 1] = nk[1];
      }
    }
    __syncthreads();
    // unconditional (the last chunk is re-read near the end), so that no
    // branch joins the pending loads
    const int nx = ch + 2 < nch ? ch + 2 : nch - 1;
    lin_stage_load(sg, kb, vb, tbeg + static_cast<long long>(nx) * kLCH, tend, fg, tp);
#pragma unroll
    for (int ks = 0; ks < kLCH / 16; ++ks) {
      const bf16x8 a = lds8(&kt[buf][(32 * fb + l32) * kLS + 16 * ks + 8 * h]);
      const bf16x8 b = lds8(&vt[buf][(32 * vb2 + l32) * kLS + 16 * ks + 8 * h]);
      acc = lin_mfma(a, b, acc);
      if (vb2 == 0) zp += sum8(a);
    }
    if constexpr (LIFT) {
      lift += lin_lift_part(vt[buf], nks[buf], w, lane);
#pragma unroll
      for (int t = 0; t < 16; ++t) liftz += nks[buf][16 * w + t];
    }
  };
  for (int ch = 0; ch < nch; ch += 2) {
    step(s0, ch);
    if (ch + 1 < nch) step(s1, ch + 1);
  }
  float* r = rec + (static_cast<long long>(bh) * NS + sp) * lin_record<F>();
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    const int f = 32 * fb + 8 * (i >> 2) + 4 * h + (i & 3);
    r[f * kLD + 32 * vb2 + l32] = acc[i];
  }
  zp += __shfl_xor(zp, 32);
  if (vb2 == 0 && h == 0) r[kLD * kLD + 32 * fb + l32] = zp;
  if constexpr (LIFT) {
    red[w][lane] = lift;
    if (lane == 0) red[w][kLD] = liftz;
    __syncthreads();
    if (tid < kLD + 4) {
      float t = 0.f;
      if (tid <= kLD) t = red[0][tid] + red[1][tid] + red[2][tid] + red[3][tid];
      r[kLE + tid] = t;  // the row, the normaliser term, three zeros
    }
  }
}

// psi of the wave's query rows in B-operand order (kk-th 16-feature step,
// half h: features 16 kk + 8 h .. +7); the Lorentz variant's norm combines the
// two halves of a row (lanes l and l ^ 32).
template <int F>
__device__ __forceinline__ void lin_query_features(const uint4* raw, bf16x8* qa, float eps, int h,
                                                   float& nq) {
  float x[4][8];
#pragma unroll
  for (int kk = 0; kk < 4; ++kk) unpack8(raw[kk], x[kk]);
  if constexpr (F == kLinLorentz) {  // raw coordinates, plus ||q|| of the whole row
    float nrm = 0.f;
#pragma unroll
    for (int kk = 0; kk < 4; ++kk)
#pragma unroll
      for (int e = 0; e < 8; ++e) nrm += x[kk][e] * x[kk][e];
    nrm += __shfl_xor(nrm, 32);
    nq = sqrtf(nrm);
  } else if constexpr (F == kLinLorentzS) {
    float nrm = 0.f;
#pragma unroll
    for (int kk = 0; kk < 4; ++kk)
#pragma unroll
      for (int e = 0; e < 8; ++e) nrm += (h == 1 && kk == 3 && e == 7) ? 0.f : x[kk][e] * x[kk][e];
    nrm += __shfl_xor(nrm, 32);
    if (h == 1) x[3][7] = sqrtf(nrm) * (1.f + x[3][7] * x[3][7]);
  } else {
#pragma unroll
    for (int kk = 0; kk < 4; ++kk)
#pragma unroll
      for (int e = 0; e < 8; ++e) x[kk][e] = lin_psi<F>(x[kk][e], eps);
  }
#pragma unroll
  for (int kk = 0; kk < 4; ++kk) qa[kk] = pack8(x[kk]);
}

// A query row past the span end re-reads the last real row (its output is
// never stored); unconditional, like the staging loads.
__device__ __forceinline__ void lin_query_load(uint4* raw, const uint16_t* qb, long long t,
                                               long long tend, int h) {
  const long long tr = t < tend ? t : tend - 1;
#pragma unroll
  for (int kk = 0; kk < 4; ++kk)
    raw[kk] = *reinterpret_cast<const uint4*>(qb + tr * kLD + 16 * kk + 8 * h);
}

// ---------------------------------------------------------------------------
// Span-output stage.  Wave w: query block qb = w / 2 of each chunk (32 rows),
// value block vb2 = w % 2 (32 columns), and the running-state tile (feature
// block w / 2, value block w % 2).  Per chunk:
//   P^T(kb) = psi(K_kb) psi(Q_qb)^T for key blocks kb <= qb, causal mask on
//     kb = qb (key rows are permuted so that the accumulator registers are
//     directly the B operand of the next product);
//   O^T = sum_kb V_kb^T P^T(kb) + S_run^T psi(Q)^T;
//   D = sum of the P^T column + psi(q) . z_run (normalised readout);
//   then S_run += psi(K_c)^T V_c and z_run += psi(K_c)^T 1 for the next chunk.
// The Lorentz lift adds ||k|| ||q|| to each score, ||q|| l_run to O (l_run =
// sum ||k|| v, fp32 in LDS) and ||q|| m_run to D (m_run = sum ||k||).
// grid BH * NS (1-D), block 256.
// ---------------------------------------------------------------------------
template <int F, bool NORM>
__global__ __launch_bounds__(256) void lin_span_output(const uint16_t* q, const uint16_t* k,
                                                       const uint16_t* v, const float* rec,
                                                       float* out, int T, int L, int NS,
                                                       float eps) {
  __shared__ __align__(16) uint16_t kt[kLD * kLS];
  __shared__ __align__(16) uint16_t vt[kLD * kLS];
  __shared__ __align__(16) uint16_t kr[kLCH * kLS];
  __shared__ __align__(16) uint16_t st[kLD * kLS];
  __shared__ __align__(16) float zs[kLD];
  constexpr bool LIFT = F == kLinLorentz;
  constexpr int LX = LIFT ? kLD : 1;
  __shared__ __align__(16) float nks[LIFT ? kLCH : 1];  // ||k|| of the staged chunk's tokens
  __shared__ __align__(16) float lrun[LX];              // l_run
  __shared__ float lpart[LIFT ? 4 : 1][LX + 1];         // per-wave chunk sums of l and m
  __shared__ float mrun;                                // m_run
  const int bh = blockIdx.x / NS, sp = blockIdx.x % NS;
  const long long tbeg = static_cast<long long>(sp) * L;
  const long long tend = tbeg + L < T ? tbeg + L : T;
  const int nch = static_cast<int>((tend - tbeg + kLCH - 1) / kLCH);
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, h = lane >> 5, l32 = lane & 31;
  const int fg = tid & 7, tp = tid >> 3;
  const int qb = w >> 1, vb2 = w & 1, fb = w >> 1;
  const long long hoff = static_cast<long long>(bh) * T * kLD;
  // this head's output rows as a raw buffer of T * 256 bytes
  const __amdgpu_buffer_rsrc_t orsrc =
      __builtin_amdgcn_make_buffer_rsrc(out + hoff, 0, T * (kLD * 4), kBufWord3);
  const uint16_t* qh = q + hoff;
  const uint16_t* kh = k + hoff;
  const uint16_t* vh = v + hoff;
  // key row supplied by this lane to the score product: accumulator row m of
  // the result then holds key 16 (m / 16) + 8 h + m % 8 with m = 8 j + 4 h + r
  const int krow = 16 * (l32 >> 4) + 8 * ((l32 >> 2) & 1) + 4 * ((l32 >> 3) & 1) + (l32 & 3);

  // running state tile from the exclusive prefix
  const float* r = rec + (static_cast<long long>(bh) * NS + sp) * lin_record<F>();
  f32x16 sacc;
#pragma unroll
  for (int i = 0; i < 16; ++i)
    sacc[i] = r[(32 * fb + 8 * (i >> 2) + 4 * h + (i & 3)) * kLD + 32 * vb2 + l32];
  float zp = 0.f;
  if (NORM && tid < kLD) zs[tid] = r[kLD * kLD + tid];
  if constexpr (LIFT) {
    if (tid < kLD) lrun[tid] = r[kLE + tid];
    if (tid == kLD) mrun = r[kLE + kLD];
  }
  auto write_state = [&]() {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      uint2 u;
      u.x = pack_bf16x2(sacc[4 * j], sacc[4 * j + 1]);
      u.y = pack_bf16x2(sacc[4 * j + 2], sacc[4 * j + 3]);
      *reinterpret_cast<uint2*>(&st[(32 * vb2 + l32) * kLS + 32 * fb + 8 * j + 4 * h]) = u;
    }
  };
  write_state();

  // Chunk ch + 1 is staged into LDS at the end of iteration ch (after the
  // barrier that retires chunk ch's operands) from registers loaded one
  // iteration earlier; the loads for chunk ch + 2 follow at once.  Loads are
  // unconditional (the last chunk is re-read near the end) and stores go
  // through the buffer unit without a branch, so no control-flow join forces
  // an early wait on the pending loads.
  LinStage sg;
  uint4 qraw[4];
  bf16x8 qa[4];
  float nq = 0.f;  // ||q|| of this lane's query (Lorentz lift)
  auto stage_in = [&]() {
    float x[2][8], y[2][8];
    lin_stage_features<F>(sg, x, eps, fg);
    lin_stage_values(sg, y);
    lin_write_t(kt, x, fg, tp);
    lin_write_t(vt, y, fg, tp);
#pragma unroll
    for (int i = 0; i < 2; ++i)
      *reinterpret_cast<bf16x8*>(&kr[(2 * tp + i) * kLS + 8 * fg]) = pack8(x[i]);
    if constexpr (LIFT) {
      float nk[2];
      lin_row_norms(x, nk);
      if (fg == 0) {
        nks[2 * tp] = nk[0];
        nks[2 * tp + 1] = nk[1];
      }
    }
    lin_query_features<F>(qraw, qa, eps, h, nq);
  };
  auto load_chunk = [&](int c) {
    const long long tn = tbeg + static_cast<long long>(c < nch ? c : nch - 1) * kLCH;
    lin_stage_load(sg, kh, vh, tn, tend, fg, tp);
    lin_query_load(qraw, qh, tn + 32 * qb + l32, tend, h);
  };
  load_chunk(0);
  stage_in();
  load_chunk(1);

  for (int ch = 0; ch < nch; ++ch) {
    const long long tc = tbeg + static_cast<long long>(ch) * kLCH;
    __syncthreads();

    f32x16 oacc;
#pragma unroll
    for (int i = 0; i < 16; ++i) oacc[i] = 0.f;
    float dsum = 0.f;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      if (kb > qb) break;
      f32x16 p;
#pragma unroll
      for (int i = 0; i < 16; ++i) p[i] = 0.f;
#pragma unroll
      for (int kk = 0; kk < 4; ++kk)
        p = lin_mfma(lds8(&kr[(32 * kb + krow) * kLS + 16 * kk + 8 * h]), qa[kk], p);
      if constexpr (LIFT) {
        // + ||k|| ||q||: p[i] holds key 32 kb + 16 (i / 8) + 8 h + i % 8
#pragma unroll
        for (int i = 0; i < 16; ++i) p[i] += nks[32 * kb + 16 * (i >> 3) + 8 * h + (i & 7)] * nq;
      }
      if (kb == qb) {
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const int key = 16 * (i >> 3) + 8 * h + (i & 7);
          if (key > l32) p[i] = 0.f;
        }
      }
      if constexpr (NORM) {
#pragma unroll
        for (int i = 0; i < 16; ++i) dsum += p[i];
      }
#pragma unroll
      for (int pp = 0; pp < 2; ++pp) {
        float pv[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) pv[e] = p[8 * pp + e];
        oacc = lin_mfma(lds8(&vt[(32 * vb2 + l32) * kLS + 32 * kb + 16 * pp + 8 * h]), pack8(pv),
                        oacc);
      }
    }
#pragma unroll
    for (int kk = 0; kk < 4; ++kk)
      oacc = lin_mfma(lds8(&st[(32 * vb2 + l32) * kLS + 16 * kk + 8 * h]), qa[kk], oacc);
    if constexpr (LIFT) {
      // + ||q|| l_run: oacc[i] holds value column 32 vb2 + 8 (i / 4) + 4 h + i % 4
#pragma unroll
      for (int i = 0; i < 16; ++i) oacc[i] += lrun[32 * vb2 + 8 * (i >> 2) + 4 * h + (i & 3)] * nq;
    }
    if constexpr (NORM) {
      float dz = 0.f;
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) {
        const uint4 u = __builtin_bit_cast(uint4, qa[kk]);
        const float4 z0 = *reinterpret_cast<const float4*>(&zs[16 * kk + 8 * h]);
        const float4 z1 = *reinterpret_cast<const float4*>(&zs[16 * kk + 8 * h + 4]);
        dz += bf16lo_f32(u.x) * z0.x + bf16hi_f32(u.x) * z0.y + bf16lo_f32(u.y) * z0.z +
              bf16hi_f32(u.y) * z0.w + bf16lo_f32(u.z) * z1.x + bf16hi_f32(u.z) * z1.y +
              bf16lo_f32(u.w) * z1.z + bf16hi_f32(u.w) * z1.w;
      }
      if constexpr (LIFT) dz += h == 0 ? nq * mrun : 0.f;
      float den = dsum + dz;
      den += __shfl_xor(den, 32);
      const float inv = den > 0.f ? 1.f / den : 0.f;
#pragma unroll
      for (int i = 0; i < 16; ++i) oacc[i] *= inv;
    }
    {
      // rows past T fall outside the head's buffer range and are dropped by
      // the buffer unit (no branch, so the stores never join a pending load)
      const int ob = static_cast<int>((tc + 32 * qb + l32) * (kLD * 4)) + (32 * vb2 + 4 * h) * 4;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        u32x4 d;
        d[0] = __float_as_uint(oacc[4 * j]);
        d[1] = __float_as_uint(oacc[4 * j + 1]);
        d[2] = __float_as_uint(oacc[4 * j + 2]);
        d[3] = __float_as_uint(oacc[4 * j + 3]);
        __builtin_amdgcn_raw_buffer_store_b128(d, orsrc, ob + 32 * j, 0, 0);
      }
    }

    // running state += this chunk (read before the barrier, written after)
#pragma unroll
    for (int ks = 0; ks < kLCH / 16; ++ks) {
      const bf16x8 a = lds8(&kt[(32 * fb + l32) * kLS + 16 * ks + 8 * h]);
      sacc = lin_mfma(a, lds8(&vt[(32 * vb2 + l32) * kLS + 16 * ks + 8 * h]), sacc);
      if (NORM && vb2 == 0) zp += sum8(a);
    }
    if constexpr (LIFT) {
      lpart[w][lane] = lin_lift_part(vt, nks, w, lane);
      if (lane == 0) {
        float m = 0.f;
#pragma unroll
        for (int t = 0; t < 16; ++t) m += nks[16 * w + t];
        lpart[w][kLD] = m;
      }
    }
    __syncthreads();
    if (ch + 1 < nch) {
      if constexpr (LIFT) {
        if (tid < kLD) lrun[tid] += lpart[0][tid] + lpart[1][tid] + lpart[2][tid] + lpart[3][tid];
        if (tid == kLD) mrun += lpart[0][kLD] + lpart[1][kLD] + lpart[2][kLD] + lpart[3][kLD];
      }
      write_state();
      if constexpr (NORM) {
        zp += __shfl_xor(zp, 32);
        if (vb2 == 0 && h == 0) zs[32 * fb + l32] += zp;
        zp = 0.f;
      }
      stage_in();
      load_chunk(ch + 2);
    }
  }
}

bool lin_mfma_supported(int T, int d, int dv, int C, int feature) {
  return d == kLD && dv == kLD && C % kLCH == 0 && C <= 1024 && T < kLinMaxT;
}

size_t lin_mfma_workspace(int BH, int T, int L, int feature) {
  const long long NS = (static_cast<long long>(T) + L - 1) / L;
  const long long E = feature == kLinLorentz ? kLEL : kLE;
  return static_cast<size_t>(BH) * NS * E * sizeof(float);
}

template <int F, bool NORM>
static hipError_t run_lin_mfma(const void* q, const void* k, const void* v, float* out, int BH,
                               int T, int L, float eps, void* ws, hipStream_t st,
                               hipEvent_t* ev) {
  const int NS = (T + L - 1) / L;
  float* rec = static_cast<float*>(ws);
  const unsigned grid = static_cast<unsigned>(BH) * NS;
  hipError_t e = record(ev, 0, st);
  if (e != hipSuccess) return e;
  lin_span_state<F><<<grid, 256, 0, st>>>(static_cast<const uint16_t*>(k),
                                         static_cast<const uint16_t*>(v), rec, T, L, NS, eps);
  if ((e = record(ev, 1, st)) != hipSuccess) return e;
  constexpr long long E = lin_record<F>();
  static_assert(E % 4 == 0, "the fp32 scan moves 16-byte pieces");
  scan_exclusive_f32x4<LinUnitWeight>
      <<<dim3(static_cast<unsigned>((E + kEB4 - 1) / kEB4), BH), 256, 0, st>>>(
          rec, NS, E, E * NS, LinUnitWeight{});
  if ((e = record(ev, 2, st)) != hipSuccess) return e;
  lin_span_output<F, NORM><<<grid, 256, 0, st>>>(
      static_cast<const uint16_t*>(q), static_cast<const uint16_t*>(k),
      static_cast<const uint16_t*>(v), rec, out, T, L, NS, eps);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  return record(ev, 3, st);
}

hipError_t launch_lin_mfma(const void* q, const void* k, const void* v, float* out, int BH, int T,
                           int feature, float eps, int normalize, int L, void* ws, hipStream_t st,
                           hipEvent_t* ev) {
  if (L <= 0 || L % kLCH != 0) return hipErrorInvalidValue;
#define KATA_LIN_CASE(FF)                                                                       \
  case FF:                                                                                      \
    return normalize ? run_lin_mfma<FF, true>(q, k, v, out, BH, T, L, eps, ws, st, ev)          \
                     : run_lin_mfma<FF, false>(q, k, v, out, BH, T, L, eps, ws, st, ev);
  switch (feature) {
    KATA_LIN_CASE(kLinIdentity)
    KATA_LIN_CASE(kLinRelu)
    KATA_LIN_CASE(kLinElu)
    KATA_LIN_CASE(kLinLorentz)
    KATA_LIN_CASE(kLinLorentzS)
    default:
      return hipErrorInvalidValue;
  }
#undef KATA_LIN_CASE
}

}  // namespace kata
