// kata_fp32.hip -- fp32 VALU kernels of libkata: the general-shape chunked
// forward (any d <= 64, dv <= 256, C <= 128, fp32 or bf16 inputs), the state
// prefill, the recurrent decode step, and the exclusive associative scan over
// chunk states that both forward paths use.
//
// Feature layout: packed row-major upper triangle, f(a, b) = a*d - a(a-1)/2 + b - a.
// With g > 1 feature blocks (KATA-Mg, section "From rank-one rays to low-rank
// PSD packing": one rank-one factor per block of m = d/g coordinates) the
// features of block i are the pairs of coordinates inside it, packed the same
// way over m, at offset i*m(m+1)/2; n = g*m(m+1)/2, and the score of a
// (query, key) pair is sum_i (q_i . k_i)^2.  g = 1 is KATA-M1.
// A chunk-state record is S[f][j] (n x dv) followed by z[f] (n), fp32.
#include "kata_common.hpp"
#include "kata_internal.hpp"
#include "kata_scan.hpp"

namespace kata {

// Pair table for packed features: entry f holds (a, b) in the low/high byte.
__device__ __forceinline__ void build_pair_table(uint16_t* tab, int d, int g) {
  const int m = d / g, nm = m * (m + 1) / 2;
  for (int x = threadIdx.x; x < d; x += blockDim.x) {
    const int blk = x / m, a = x % m;
    for (int b = a; b < m; ++b)
      tab[blk * nm + packed_index(a, b, m)] =
          static_cast<uint16_t>((blk * m + a) | ((blk * m + b) << 8));
  }
}

// The pair (a, b) of feature f (one thread's lookup, no table).
__device__ __forceinline__ uint16_t pair_of(int f, int d, int g) {
  const int m = d / g, nm = m * (m + 1) / 2;
  const int blk = f / nm, fl = f % nm;
  int a = 0;
  while (a + 1 < m && packed_index(a + 1, a + 1, m) <= fl) ++a;
  const int b = a + (fl - packed_index(a, a, m));
  return static_cast<uint16_t>((blk * m + a) | ((blk * m + b) << 8));
}

// ---------------------------------------------------------------------------
// Chunk state (eq. chunk-SZ): for chunk c of head bh, over tokens
// [c*C, min(c*C + C, T)),  S[f][j] = sum_t k_a k_b v_j,  z[f] = sum_t k_a k_b.
// With C >= T and one chunk this is the prefill state.
// grid (ceil(n/FB), NC, BH), block 256.  Record stride rec = n*dv + n.
// ---------------------------------------------------------------------------
constexpr int kFB = 16;   // features per workgroup
constexpr int kTB = 32;   // tokens staged per pass

template <typename Tin>
__global__ __launch_bounds__(256) void chunk_state_f32(
    const Tin* __restrict__ k, const Tin* __restrict__ v, float* __restrict__ S_out,
    float* __restrict__ z_out, int T, int d, int dv, int C, int g, long long S_bh_stride,
    long long S_chunk_stride, long long z_bh_stride, long long z_chunk_stride) {
  __shared__ float ks[kTB][65];
  __shared__ float vs[kTB][257];
  __shared__ uint16_t pairs[kFB];
  const int n = g * ((d / g) * (d / g + 1) / 2);
  const int f0 = blockIdx.x * kFB;
  const int c = blockIdx.y;
  const int bh = blockIdx.z;
  const int tid = threadIdx.x;
  if (tid < kFB && f0 + tid < n) pairs[tid] = pair_of(f0 + tid, d, g);
  const int nf = min(kFB, n - f0);
  const int nout = nf * dv;
  constexpr int R = (kFB * 256) / 256;  // at most 16 outputs per thread
  float acc[R];
#pragma unroll
  for (int r = 0; r < R; ++r) acc[r] = 0.f;
  float zacc = 0.f;
  const long long t_begin = static_cast<long long>(c) * C;
  const long long t_end = min(static_cast<long long>(T), t_begin + C);
  const Tin* kh = k + static_cast<long long>(bh) * T * d;
  const Tin* vh = v + static_cast<long long>(bh) * T * dv;
  for (long long t0 = t_begin; t0 < t_end; t0 += kTB) {
    const int nt = static_cast<int>(min(static_cast<long long>(kTB), t_end - t0));
    __syncthreads();
    for (int i = tid; i < kTB * d; i += 256) {
      int t = i / d, a = i % d;
      ks[t][a] = (t < nt) ? load_f32(kh, (t0 + t) * d + a) : 0.f;
    }
    for (int i = tid; i < kTB * dv; i += 256) {
      int t = i / dv, j = i % dv;
      vs[t][j] = (t < nt) ? load_f32(vh, (t0 + t) * dv + j) : 0.f;
    }
    __syncthreads();
#pragma unroll
    for (int r = 0; r < R; ++r) {
      int o = tid + 256 * r;
      if (o < nout) {
        int fl = o / dv, j = o % dv;
        int a = pairs[fl] & 0xFF, b = pairs[fl] >> 8;
        float s = acc[r];
        for (int t = 0; t < nt; ++t) s += (ks[t][a] * ks[t][b]) * vs[t][j];
        acc[r] = s;
      }
    }
    if (tid < nf) {
      int a = pairs[tid] & 0xFF, b = pairs[tid] >> 8;
      for (int t = 0; t < nt; ++t) zacc += ks[t][a] * ks[t][b];
    }
  }
  float* So = S_out + bh * S_bh_stride + c * S_chunk_stride;
  float* zo = z_out + bh * z_bh_stride + c * z_chunk_stride;
#pragma unroll
  for (int r = 0; r < R; ++r) {
    int o = tid + 256 * r;
    if (o < nout) So[static_cast<long long>(f0) * dv + o] = acc[r];
  }
  if (tid < nf) zo[f0 + tid] = zacc;
}

// ---------------------------------------------------------------------------
// Chunk output (eq. chunk-out): for chunk c of head bh,
//   P[r][s] = sum_i (q_{r,i} . k_{s,i})^2 over the g blocks, for s <= r
//   (lower-triangular mask incl. diagonal),
//   N = Phi_w(Q_c) S_pre + P V_c,  D = Phi_w(Q_c) z_pre + P 1,  O = N / D (0 if D = 0),
// Phi_w the query-side packed feature (weight 2 off the diagonal).
// grid (NC, BH), block 256; C <= 128, d <= 64.
// ---------------------------------------------------------------------------
template <typename Tin>
__global__ __launch_bounds__(256) void chunk_out_f32(
    const Tin* __restrict__ q, const Tin* __restrict__ k, const Tin* __restrict__ v,
    const float* __restrict__ pre, float* __restrict__ out, int T, int d, int dv, int C, int g,
    long long bh_stride, long long chunk_stride) {
  extern __shared__ float smem[];
  const int m = d / g;
  const int n = g * (m * (m + 1) / 2);
  float* qs = smem;                 // [C][d]
  float* ks = qs + C * d;           // [C][d]
  float* P = ks + C * d;            // [C][C]
  float* Dn = P + C * C;            // [C]
  uint16_t* pairs = reinterpret_cast<uint16_t*>(Dn + C);  // [n]
  const int c = blockIdx.x;
  const int bh = blockIdx.y;
  const int tid = threadIdx.x;
  const long long t0 = static_cast<long long>(c) * C;
  const int nt = static_cast<int>(min(static_cast<long long>(C), T - t0));
  const Tin* qh = q + static_cast<long long>(bh) * T * d;
  const Tin* kh = k + static_cast<long long>(bh) * T * d;
  const Tin* vh = v + static_cast<long long>(bh) * T * dv;
  build_pair_table(pairs, d, g);
  for (int i = tid; i < C * d; i += 256) {
    int r = i / d, a = i % d;
    qs[i] = (r < nt) ? load_f32(qh, (t0 + r) * d + a) : 0.f;
    ks[i] = (r < nt) ? load_f32(kh, (t0 + r) * d + a) : 0.f;
  }
  __syncthreads();
  for (int i = tid; i < C * C; i += 256) {
    int r = i / C, s = i % C;
    float p = 0.f;
    if (s <= r)
      for (int blk = 0; blk < g; ++blk) {
        float a = 0.f;
        for (int x = blk * m; x < blk * m + m; ++x) a += qs[r * d + x] * ks[s * d + x];
        p += a * a;
      }
    P[i] = p;
  }
  __syncthreads();
  const float* Sp = pre + bh * bh_stride + c * chunk_stride;
  const float* zp = Sp + static_cast<long long>(n) * dv;
  for (int r = tid; r < C; r += 256) {
    float D = 0.f;
    for (int f = 0; f < n; ++f) {
      int a = pairs[f] & 0xFF, b = pairs[f] >> 8;
      float w = (a == b) ? 1.f : 2.f;
      D += (w * qs[r * d + a] * qs[r * d + b]) * zp[f];
    }
    for (int s = 0; s < C; ++s) D += P[r * C + s];
    Dn[r] = D;
  }
  __syncthreads();
  for (int o = tid; o < nt * dv; o += 256) {
    int r = o / dv, j = o % dv;
    float acc = 0.f;
    for (int f = 0; f < n; ++f) {
      int a = pairs[f] & 0xFF, b = pairs[f] >> 8;
      float w = (a == b) ? 1.f : 2.f;
      acc += (w * qs[r * d + a] * qs[r * d + b]) * Sp[static_cast<long long>(f) * dv + j];
    }
    for (int s = 0; s <= r; ++s) acc += P[r * C + s] * load_f32(vh, (t0 + s) * dv + j);
    float D = Dn[r];
    out[(static_cast<long long>(bh) * T + t0 + r) * dv + j] = (D > 0.f) ? acc / D : 0.f;
  }
}

// ---------------------------------------------------------------------------
// Decode step (eq. linatt's recurrence + normalised readout with the updated
// state).  One workgroup per head; S is streamed once (read-modify-write).
// grid BH, block 256; d <= 64, dv <= 256.
// ---------------------------------------------------------------------------
// S rows per thread whose loads are in flight together.  26 divides the 130
// rows each thread walks at n = 2080, dv = 64 and still fits 256 VGPRs
// (measured against 8, 16, 32, 40 and 48).
constexpr int kDecodeUnroll = 26;

// The state is touched once per step: stream it past the caches (non-temporal
// loads and stores; together they raise the step from 5.1 to 5.85 TB/s).
typedef float decode_f4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ float4 stream_load4(const float* p) {
  const decode_f4 t = __builtin_nontemporal_load(reinterpret_cast<const decode_f4*>(p));
  return make_float4(t.x, t.y, t.z, t.w);
}
__device__ __forceinline__ void stream_store4(float* p, float4 s) {
  const decode_f4 t = {s.x, s.y, s.z, s.w};
  __builtin_nontemporal_store(t, reinterpret_cast<decode_f4*>(p));
}

template <typename Tin>
__global__ __launch_bounds__(256) void decode_step_f32(float* __restrict__ S,
                                                       float* __restrict__ z,
                                                       const Tin* __restrict__ q,
                                                       const Tin* __restrict__ k,
                                                       const Tin* __restrict__ v,
                                                       float* __restrict__ out, int d, int dv,
                                                       int g) {
  __shared__ float qs[64], ks[64], vs[256];
  __shared__ uint16_t pairs[2080];
  __shared__ float red[256][5];
  const int n = g * ((d / g) * (d / g + 1) / 2);
  const int bh = blockIdx.x;
  const int tid = threadIdx.x;
  build_pair_table(pairs, d, g);
  if (tid < d) {
    qs[tid] = load_f32(q, static_cast<long long>(bh) * d + tid);
    ks[tid] = load_f32(k, static_cast<long long>(bh) * d + tid);
  }
  for (int j = tid; j < dv; j += 256) vs[j] = load_f32(v, static_cast<long long>(bh) * dv + j);
  __syncthreads();
  float* Sh = S + static_cast<long long>(bh) * n * dv;
  float* zh = z + static_cast<long long>(bh) * n;
  float num[4] = {0.f, 0.f, 0.f, 0.f};
  float den = 0.f;
  int jbase = 0;
  const bool vec = (dv % 4 == 0) && (256 % (dv / 4) == 0);
  if (vec) {
    // float4 stream: thread owns columns [4*(tid % (dv/4)), +4) of rows
    // tid / (dv/4), + 256/(dv/4), ...
    const int g = dv / 4;
    const int rows_per_pass = 256 / g;
    jbase = 4 * (tid % g);
    const float v0 = vs[jbase + 0], v1 = vs[jbase + 1], v2 = vs[jbase + 2], v3 = vs[jbase + 3];
    auto row = [&](int f, float4 s) {
      const int a = pairs[f] & 0xFF, b = pairs[f] >> 8;
      const float pk = ks[a] * ks[b];
      const float pq = ((a == b) ? 1.f : 2.f) * qs[a] * qs[b];
      s.x += pk * v0;
      s.y += pk * v1;
      s.z += pk * v2;
      s.w += pk * v3;
      stream_store4(Sh + static_cast<long long>(f) * dv + jbase, s);
      num[0] += pq * s.x;
      num[1] += pq * s.y;
      num[2] += pq * s.z;
      num[3] += pq * s.w;
    };
    // kDecodeUnroll rows per thread in flight: their loads are issued together
    int f = tid / g;
    for (; f + (kDecodeUnroll - 1) * rows_per_pass < n; f += kDecodeUnroll * rows_per_pass) {
      float4 s[kDecodeUnroll];
#pragma unroll
      for (int u = 0; u < kDecodeUnroll; ++u)
        s[u] = stream_load4(Sh + static_cast<long long>(f + u * rows_per_pass) * dv + jbase);
#pragma unroll
      for (int u = 0; u < kDecodeUnroll; ++u) row(f + u * rows_per_pass, s[u]);
    }
    for (; f < n; f += rows_per_pass)
      row(f, stream_load4(Sh + static_cast<long long>(f) * dv + jbase));
  } else {
    const int rows_per_pass = 256 / dv;  // dv <= 256
    jbase = tid % dv;
    if (tid < rows_per_pass * dv) {
      for (int f = tid / dv; f < n; f += rows_per_pass) {
        int a = pairs[f] & 0xFF, b = pairs[f] >> 8;
        float pk = ks[a] * ks[b];
        float pq = ((a == b) ? 1.f : 2.f) * qs[a] * qs[b];
        float s = Sh[static_cast<long long>(f) * dv + jbase] + pk * vs[jbase];
        Sh[static_cast<long long>(f) * dv + jbase] = s;
        num[0] += pq * s;
      }
    }
  }
  for (int f = tid; f < n; f += 256) {
    int a = pairs[f] & 0xFF, b = pairs[f] >> 8;
    float zz = zh[f] + ks[a] * ks[b];
    zh[f] = zz;
    den += ((a == b) ? 1.f : 2.f) * qs[a] * qs[b] * zz;
  }
  red[tid][0] = num[0];
  red[tid][1] = num[1];
  red[tid][2] = num[2];
  red[tid][3] = num[3];
  red[tid][4] = den;
  __syncthreads();
  // denominator: tree over all threads
  for (int s = 128; s >= 1; s >>= 1) {
    if (tid < s) red[tid][4] += red[tid + s][4];
    __syncthreads();
  }
  const float D = red[0][4];
  if (vec) {
    const int g = dv / 4;
    if (tid < g) {
      float acc[4] = {0.f, 0.f, 0.f, 0.f};
      for (int t = tid; t < 256; t += g)
        for (int x = 0; x < 4; ++x) acc[x] += red[t][x];
      for (int x = 0; x < 4; ++x)
        out[static_cast<long long>(bh) * dv + 4 * tid + x] = (D > 0.f) ? acc[x] / D : 0.f;
    }
  } else {
    const int rows_per_pass = 256 / dv;
    if (tid < dv) {
      float acc = 0.f;
      for (int t = tid; t < rows_per_pass * dv; t += dv) acc += red[t][0];
      out[static_cast<long long>(bh) * dv + tid] = (D > 0.f) ? acc / D : 0.f;
    }
  }
}

// ---------------------------------------------------------------------------
// Host launchers
// ---------------------------------------------------------------------------
size_t fp32_forward_workspace(int BH, int T, int d, int dv, int C, int g) {
  const size_t n = static_cast<size_t>(g) * (d / g) * (d / g + 1) / 2;
  const size_t NC = (static_cast<size_t>(T) + C - 1) / C;
  return static_cast<size_t>(BH) * NC * (n * dv + n) * sizeof(float);
}

size_t fp32_forward_smem(int d, int C, int g) {
  const size_t n = static_cast<size_t>(g) * (d / g) * (d / g + 1) / 2;
  return (static_cast<size_t>(C) * d * 2 + static_cast<size_t>(C) * C + C) * sizeof(float) +
         n * sizeof(uint16_t);
}

template <typename Tin>
hipError_t launch_fp32_forward(const void* q, const void* k, const void* v, float* out, int BH,
                               int T, int d, int dv, int C, int g, void* ws, hipStream_t st,
                               hipEvent_t* ev) {
  const int n = g * ((d / g) * (d / g + 1) / 2);
  const int NC = (T + C - 1) / C;
  const long long rec = static_cast<long long>(n) * dv + n;
  float* states = static_cast<float*>(ws);
  const long long bh_stride = rec * NC;
  dim3 g1((n + kFB - 1) / kFB, NC, BH);
  hipError_t e = record(ev, 0, st);
  if (e != hipSuccess) return e;
  chunk_state_f32<Tin><<<g1, 256, 0, st>>>(static_cast<const Tin*>(k), static_cast<const Tin*>(v),
                                           states, states + static_cast<long long>(n) * dv, T, d,
                                           dv, C, g, bh_stride, rec, bh_stride, rec);
  if ((e = record(ev, 1, st)) != hipSuccess) return e;
  dim3 g2(static_cast<unsigned>((rec + kEB - 1) / kEB), BH);
  scan_exclusive<float, UnitWeight><<<g2, 256, 0, st>>>(states, states, NC, rec, bh_stride,
                                                        UnitWeight{});
  if ((e = record(ev, 2, st)) != hipSuccess) return e;
  const size_t shm = fp32_forward_smem(d, C, g);
  if (shm > 65536) {
    e = hipFuncSetAttribute(reinterpret_cast<const void*>(&chunk_out_f32<Tin>),
                                       hipFuncAttributeMaxDynamicSharedMemorySize,
                                       static_cast<int>(shm));
    if (e != hipSuccess) return e;
  }
  chunk_out_f32<Tin><<<dim3(NC, BH), 256, shm, st>>>(
      static_cast<const Tin*>(q), static_cast<const Tin*>(k), static_cast<const Tin*>(v), states,
      out, T, d, dv, C, g, bh_stride, rec);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  return record(ev, 3, st);
}

template <typename Tin>
hipError_t launch_prefill(const void* k, const void* v, float* S, float* z, int BH, int T, int d,
                          int dv, int g, hipStream_t st) {
  const int n = g * ((d / g) * (d / g + 1) / 2);
  dim3 grid((n + kFB - 1) / kFB, 1, BH);
  // one chunk covering all T tokens; S and z are separate arrays
  chunk_state_f32<Tin><<<grid, 256, 0, st>>>(static_cast<const Tin*>(k), static_cast<const Tin*>(v),
                                           S, z, T, d, dv, T, g, static_cast<long long>(n) * dv, 0,
                                           static_cast<long long>(n), 0);
  return hipGetLastError();
}

template <typename Tin>
hipError_t launch_decode(float* S, float* z, const void* q, const void* k, const void* v,
                         float* out, int BH, int d, int dv, int g, hipStream_t st) {
  decode_step_f32<Tin><<<BH, 256, 0, st>>>(S, z, static_cast<const Tin*>(q),
                                           static_cast<const Tin*>(k), static_cast<const Tin*>(v),
                                           out, d, dv, g);
  return hipGetLastError();
}

template hipError_t launch_fp32_forward<float>(const void*, const void*, const void*, float*, int,
                                               int, int, int, int, int, void*, hipStream_t,
                                               hipEvent_t*);
template hipError_t launch_fp32_forward<bf16_t>(const void*, const void*, const void*, float*, int,
                                                int, int, int, int, int, void*, hipStream_t,
                                                hipEvent_t*);
template hipError_t launch_prefill<float>(const void*, const void*, float*, float*, int, int,
                                          int, int, int, hipStream_t);
template hipError_t launch_prefill<bf16_t>(const void*, const void*, float*, float*, int, int,
                                           int, int, int, hipStream_t);
template hipError_t launch_decode<float>(float*, float*, const void*, const void*, const void*,
                                         float*, int, int, int, int, hipStream_t);
template hipError_t launch_decode<bf16_t>(float*, float*, const void*, const void*, const void*,
                                          float*, int, int, int, int, hipStream_t);

}  // namespace kata
