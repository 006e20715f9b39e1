// kata_mfma.hip -- bf16 MFMA path of the causal KATA-M1 forward on gfx950.
//
// The chunked-state form (eq. chunk-SZ, eq. chunk-out; the three-stage
// pipeline of the tree-scan section) with one change of granularity: the state
// written to HBM covers a span of L = G*C tokens instead of one chunk.  By
// bilinearity this is exact: a span state is the sum of its chunk states, the
// prefix scan runs over span states, and inside a span the contribution of the
// earlier chunks, phi(Q_c)^T sum_{c'<c} S_c' = sum_{c'<c} P_cc' V_c', is taken
// from the causal squared-score blocks directly.  G = 1 is the per-chunk form.
//
//   K2  span_state : S_span = Phi(K)^T V and Z_span = K^T K, MFMA over the span,
//                    Phi(K) generated on chip (never written to HBM).
//   K3  scan       : exclusive prefix over spans (kata_fp32.hip's Blelloch scan),
//                    written as bf16 MFMA operands with the feature weights.
//   K4  span_output: squared-score attention inside the span (QK^T on MFMA,
//                    squared and masked in registers, P V back through MFMA),
//                    plus the readout Phi_w(Q) S_pre and q^T Z_pre q, then the
//                    normalisation O = N / D.
//
// Feature ("slot") order.  Instead of the row-major packed triangle, the
// state is kept in an order that lets every lane build its query features from
// registers.  A query row is held per lane in fp32 registers rotated by
// R = d/2 per lane group g of the 32x32x16 MFMA (register x holds q[(x+R*g) % d]).
// Slot s (K-step kappa = s/16, lane group g = (s/8)%2, j = s%8) has
//   P = 8*kappa + j,  delta = P / R,  r1 = P % R,
//   pair (x, y) = ((r1 + R*g) % d, (r1 + delta + R*g) % d),
// i.e. registers r1+j and r1+j+delta of the rotated row.  Pairs are grouped by
// cyclic difference delta = 0..R; every unordered pair appears once, except
// that for delta = R the g = 1 slots repeat the g = 0 pairs.  Those d/2 slots
// get weight 0, diagonal slots weight 1 and the rest weight 2 (exact powers of
// two), so sum_s w_s phi_s(q) phi_s(k) = (q . k)^2.  n_slot = (R+1)*d.
#include <utility>

#include "kata_common.hpp"
#include "kata_internal.hpp"
#include "kata_scan.hpp"

namespace kata {

template <int I, int N, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (I < N) {
    f(std::integral_constant<int, I>{});
    static_for<I + 1, N>(f);
  }
}

// Two state features k_x(t) k_y(t), k_x(t+1) k_y(t+1) from a bf16 pair of y
// values and the matching packed pair of x values, rounded to one bf16 pair.
// Each v_dot2 has one zero lane, so it returns the exact product.
__device__ __forceinline__ uint32_t gen_pair(bf16x2 y2, uint32_t xw) {
  const float p0 = __builtin_amdgcn_fdot2_f32_bf16(y2, __builtin_bit_cast(bf16x2, xw & 0x0000FFFFu),
                                                   0.f, false);
  const float p1 = __builtin_amdgcn_fdot2_f32_bf16(y2, __builtin_bit_cast(bf16x2, xw & 0xFFFF0000u),
                                                   0.f, false);
  return pack_bf16x2(p0, p1);
}

__device__ __forceinline__ f32x16 mfma32(const bf16x8& a, const bf16x8& b, const f32x16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

template <int D, int DV>
struct Geo {
  static constexpr int R = D / 2;
  static constexpr int NKS = (R + 1) * D / 16;   // readout K-steps (16 slots each)
  static constexpr int NSLOT = 16 * NKS;         // (R+1)*d
  static constexpr int NST = NSLOT / 32;         // 32-slot tiles
  static constexpr int MT = DV / 32;             // dv tiles
  static constexpr int ZM = D / 32;              // 32-dim tiles of Z
  static constexpr int KZ = D / 16;              // K-steps over d
  static constexpr long long ES = static_cast<long long>(DV) * NSLOT;
  static constexpr long long EZ = static_cast<long long>(D) * D;
  static constexpr long long E = ES + EZ;        // one span record
  static_assert(D % 32 == 0 && DV % 32 == 0, "tile shapes");
};

// Slot -> (x, y) dims of its pair (see the header comment).
template <int D>
__host__ __device__ __forceinline__ void slot_pair(int s, int& x, int& y) {
  constexpr int R = D / 2;
  const int kappa = s >> 4, g = (s >> 3) & 1, j = s & 7;
  const int P = 8 * kappa + j;
  const int delta = P / R, r1 = P % R;
  x = (r1 + R * g) % D;
  y = (r1 + delta + R * g) % D;
}

template <int D>
__host__ __device__ __forceinline__ float slot_weight(int s) {
  constexpr int R = D / 2;
  const int kappa = s >> 4, g = (s >> 3) & 1, j = s & 7;
  const int delta = (8 * kappa + j) / R;
  if (delta == 0) return 1.f;
  if (delta < R) return 2.f;
  return g == 0 ? 2.f : 0.f;
}

// Position of Z[a][b] in the operand-ordered Z record that K4 reads as the A
// operand of Y^T = Z Q^T: row m of the MFMA A tile stands for a = sigma(m)
// with sigma(32*mu + 8*(r/4) + 4*g + r%4) = 16*mu + r + R*g, so that the
// accumulator row each lane holds pairs with a register of its rotated query.
template <int D>
__host__ __device__ __forceinline__ int zop_index(int a, int b) {
  constexpr int R = D / 2, KZ = D / 16;
  const int ga = a / R, rem = a % R, mu = rem / 16, rr = rem % 16;
  const int m = 8 * (rr / 4) + 4 * ga + (rr % 4);  // row inside the 32-row tile
  const int gb = b / R, kap = (b % R) / 8, jb = b % 8;
  const int lane = m + 32 * gb;
  return ((mu * KZ + kap) * 64 + lane) * 8 + jb;
}

// Scan output weights: S region by slot, Z region 1.
template <int D, int DV>
struct SlotWeight {
  __device__ __forceinline__ float operator()(long long e) const {
    using G = Geo<D, DV>;
    if (e >= G::ES) return 1.f;
    return slot_weight<D>(static_cast<int>(e % G::NSLOT));
  }
};

// ---------------------------------------------------------------------------
// K2: span state.  grid (unit blocks, NS, BH), block 256 (4 waves).
// Units: slot tiles 0..NST-1 (32 slots x dv) and Z tiles NST..NST+ZM-1
// (32 dims x d).  Wave w of unit block ub owns units [ (4*ub + w)*UW, +UW ).
// Output spanst[bh][s][E] fp32: S^T as [dv][NSLOT], then Z in operand order.
// ---------------------------------------------------------------------------
constexpr int kTB2 = 64;            // tokens per staged block
constexpr int kRow2 = kTB2 + 8;     // LDS row length (bf16), 144 B

template <int D, int DV, int UW>
__global__ __launch_bounds__(256) void span_state_kernel(const uint16_t* __restrict__ k,
                                                         const uint16_t* __restrict__ v,
                                                         float* __restrict__ spanst, int T,
                                                         int L) {
  using G = Geo<D, DV>;
  constexpr int NUNITS = G::NST + G::ZM;
  __shared__ __attribute__((aligned(16))) uint16_t kT[2][D][kRow2];
  __shared__ __attribute__((aligned(16))) uint16_t vT[2][DV][kRow2];
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int c = lane & 31, g = lane >> 5;
  const int s = blockIdx.y, bh = blockIdx.z;
  const long long span0 = static_cast<long long>(s) * L;
  const long long span_end = min(static_cast<long long>(T), span0 + L);
  const uint16_t* kh = k + static_cast<long long>(bh) * T * D;
  const uint16_t* vh = v + static_cast<long long>(bh) * T * DV;
  const int unit0 = (blockIdx.x * 4 + wave) * UW;

  // per-unit constants: LDS rows of x and y for slot units
  int ux[UW], uy[UW];
#pragma unroll
  for (int u = 0; u < UW; ++u) {
    const int unit = unit0 + u;
    ux[u] = 0;
    uy[u] = 0;
    if (unit < G::NST) slot_pair<D>(32 * unit + c, ux[u], uy[u]);
  }
  f32x16 acc[UW][G::MT];
#pragma unroll
  for (int u = 0; u < UW; ++u)
#pragma unroll
    for (int m = 0; m < G::MT; ++m)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[u][m][r] = 0.f;

  // staging: task -> (pair p of tokens, 8-wide column group); K then V
  constexpr int KG = D / 8, VG = DV / 8;
  constexpr int NTASK = 32 * (KG + VG);
  constexpr int TPT = (NTASK + 255) / 256;
  u32x4 st_lo[TPT], st_hi[TPT];
  auto fetch = [&](long long t0) {
#pragma unroll
    for (int i = 0; i < TPT; ++i) {
      const int task = tid + 256 * i;
      const int cg = task >> 5, p = task & 31;
      const long long ta = t0 + 2 * p, tb = ta + 1;
      u32x4 zero = {0u, 0u, 0u, 0u};
      st_lo[i] = zero;
      st_hi[i] = zero;
      if (task < NTASK) {
        if (cg < KG) {
          if (ta < span_end) st_lo[i] = *reinterpret_cast<const u32x4*>(kh + ta * D + 8 * cg);
          if (tb < span_end) st_hi[i] = *reinterpret_cast<const u32x4*>(kh + tb * D + 8 * cg);
        } else {
          const int vg = cg - KG;
          if (ta < span_end) st_lo[i] = *reinterpret_cast<const u32x4*>(vh + ta * DV + 8 * vg);
          if (tb < span_end) st_hi[i] = *reinterpret_cast<const u32x4*>(vh + tb * DV + 8 * vg);
        }
      }
    }
  };
  auto commit = [&](int buf) {
#pragma unroll
    for (int i = 0; i < TPT; ++i) {
      const int task = tid + 256 * i;
      if (task >= NTASK) continue;
      const int cg = task >> 5, p = task & 31;
      uint16_t* base = (cg < KG) ? &kT[buf][8 * cg][0] : &vT[buf][8 * (cg - KG)][0];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const uint32_t a = st_lo[i][e], b = st_hi[i][e];
        // element 2e: (a.lo, b.lo); element 2e+1: (a.hi, b.hi)
        const uint32_t w0 = (a & 0xFFFFu) | (b << 16);
        const uint32_t w1 = (a >> 16) | (b & 0xFFFF0000u);
        *reinterpret_cast<uint32_t*>(base + (2 * e) * kRow2 + 2 * p) = w0;
        *reinterpret_cast<uint32_t*>(base + (2 * e + 1) * kRow2 + 2 * p) = w1;
      }
    }
  };

  const int nblk = static_cast<int>((span_end - span0 + kTB2 - 1) / kTB2);
  fetch(span0);
  commit(0);
  __syncthreads();
  for (int bi = 0; bi < nblk; ++bi) {
    const int buf = bi & 1;
    if (bi + 1 < nblk) fetch(span0 + static_cast<long long>(bi + 1) * kTB2);
#pragma unroll
    for (int ks = 0; ks < kTB2 / 16; ++ks) {
      const int col = 16 * ks + 8 * g;  // first token of this lane's 8
      bf16x8 va[G::MT];
#pragma unroll
      for (int m = 0; m < G::MT; ++m)
        va[m] = *reinterpret_cast<const bf16x8*>(&vT[buf][32 * m + c][col]);
#pragma unroll
      for (int u = 0; u < UW; ++u) {
        const int unit = unit0 + u;
        if (unit < G::NST) {
          const u32x4 X = *reinterpret_cast<const u32x4*>(&kT[buf][ux[u]][col]);
          const bf16x8 Y = *reinterpret_cast<const bf16x8*>(&kT[buf][uy[u]][col]);
          u32x4 Bw;
          // (k_y(t), k_y(t+1)) . (k_x(t), 0) and . (0, k_x(t+1)): exact single products
          Bw[0] = gen_pair(__builtin_shufflevector(Y, Y, 0, 1), X[0]);
          Bw[1] = gen_pair(__builtin_shufflevector(Y, Y, 2, 3), X[1]);
          Bw[2] = gen_pair(__builtin_shufflevector(Y, Y, 4, 5), X[2]);
          Bw[3] = gen_pair(__builtin_shufflevector(Y, Y, 6, 7), X[3]);
          const bf16x8 Bf = __builtin_bit_cast(bf16x8, Bw);
#pragma unroll
          for (int m = 0; m < G::MT; ++m) acc[u][m] = mfma32(va[m], Bf, acc[u][m]);
        } else if (unit < NUNITS) {
          const int nz = unit - G::NST;
          const bf16x8 Bz = *reinterpret_cast<const bf16x8*>(&kT[buf][32 * nz + c][col]);
#pragma unroll
          for (int m = 0; m < G::ZM; ++m) {
            const bf16x8 Az = *reinterpret_cast<const bf16x8*>(&kT[buf][32 * m + c][col]);
            acc[u][m] = mfma32(Az, Bz, acc[u][m]);
          }
        }
      }
    }
    if (bi + 1 < nblk) {
      commit(buf ^ 1);
    }
    __syncthreads();
  }

  // write the span record
  float* rec = spanst + (static_cast<long long>(bh) * gridDim.y + s) * G::E;
#pragma unroll
  for (int u = 0; u < UW; ++u) {
    const int unit = unit0 + u;
    if (unit < G::NST) {
#pragma unroll
      for (int m = 0; m < G::MT; ++m)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int dvrow = 32 * m + 8 * (r >> 2) + 4 * g + (r & 3);
          rec[static_cast<long long>(dvrow) * G::NSLOT + 32 * unit + c] = acc[u][m][r];
        }
    } else if (unit < NUNITS) {
      const int nz = unit - G::NST;
#pragma unroll
      for (int m = 0; m < G::ZM; ++m)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int a = 32 * m + 8 * (r >> 2) + 4 * g + (r & 3);
          const int b = 32 * nz + c;
          rec[G::ES + zop_index<D>(a, b)] = acc[u][m][r];
        }
    }
  }
}

// ---------------------------------------------------------------------------
// K4: span output.  grid (query blocks per span, NS, BH), block 64*W.
// The workgroup owns NTILE = W*NQ query tiles of 32 (span-relative tile index
// qb*NTILE + i); wave w takes tiles {w, 2W-1-w} (NQ = 2) or {w} (NQ = 1), which
// balances the causal work across waves.
// pre[bh][s][E] bf16: weighted S_pre^T as [dv][NSLOT], then Z_pre (operand order).
// ---------------------------------------------------------------------------
constexpr int kKC = 8;  // readout K-steps per staged block of S_pre

template <int D, int DV, int NQ, int W>
__global__ __launch_bounds__(64 * W) void span_output_kernel(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ k,
    const uint16_t* __restrict__ v, const uint16_t* __restrict__ pre, float* __restrict__ out,
    int T, int L) {
  using G = Geo<D, DV>;
  constexpr int R = G::R;
  constexpr int SROW = 16 * kKC + 8;        // bf16 per staged S_pre row (272 B)
  constexpr int KROW = D + 8;               // staged key row (bf16)
  constexpr int VROW = 32 + 8;              // staged V^T row (bf16)
  constexpr int SBUF = DV * SROW;           // one S_pre buffer (bf16 elements)
  constexpr int KVBUF = 32 * KROW + DV * VROW;
  constexpr int LDS_ELEMS = (2 * SBUF > 2 * KVBUF) ? 2 * SBUF : 2 * KVBUF;
  __shared__ __attribute__((aligned(16))) uint16_t lds[LDS_ELEMS];

  constexpr int NTH = 64 * W;
  constexpr int NT = W * NQ;
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int c = lane & 31, g = lane >> 5;
  const int qb = blockIdx.x, s = blockIdx.y, bh = blockIdx.z;
  const long long span0 = static_cast<long long>(s) * L;
  const long long span_end = min(static_cast<long long>(T), span0 + L);
  const long long wg_q0 = span0 + static_cast<long long>(qb) * NT * 32;
  if (wg_q0 >= span_end) return;  // whole workgroup beyond the sequence
  const uint16_t* qh = q + static_cast<long long>(bh) * T * D;
  const uint16_t* kh = k + static_cast<long long>(bh) * T * D;
  const uint16_t* vh = v + static_cast<long long>(bh) * T * DV;
  const uint16_t* rec = pre + (static_cast<long long>(bh) * gridDim.y + s) * G::E;

  int tile[NQ];           // span-relative tile index
  long long tq0[NQ];      // absolute first query of the tile
  bool tlive[NQ];
#pragma unroll
  for (int i = 0; i < NQ; ++i) {
    const int local = (NQ == 2) ? (i == 0 ? wave : 2 * W - 1 - wave) : wave;
    tile[i] = qb * NT + local;
    tq0[i] = span0 + 32LL * tile[i];
    tlive[i] = tq0[i] < span_end;
  }

  // bf16 query fragments for the d-contractions: qf[i][kz] holds
  // q[t][8*kz + R*g .. +7] of this lane's query t = tq0 + c.
  bf16x8 qf[NQ][G::KZ];
#pragma unroll
  for (int i = 0; i < NQ; ++i) {
    const long long t = tq0[i] + c;
#pragma unroll
    for (int kz = 0; kz < G::KZ; ++kz) {
      u32x4 w = {0u, 0u, 0u, 0u};
      if (t < span_end) w = *reinterpret_cast<const u32x4*>(qh + t * D + 8 * kz + R * g);
      qf[i][kz] = __builtin_bit_cast(bf16x8, w);
    }
  }

  f32x16 acc[G::MT][NQ];
#pragma unroll
  for (int m = 0; m < G::MT; ++m)
#pragma unroll
    for (int i = 0; i < NQ; ++i)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[m][i][r] = 0.f;
  float dpart[NQ];

  // ---- denominator from the prefix: q^T Z_pre q ------------------------------
  {
    f32x16 az[G::ZM][NQ];
#pragma unroll
    for (int m = 0; m < G::ZM; ++m)
#pragma unroll
      for (int i = 0; i < NQ; ++i)
#pragma unroll
        for (int r = 0; r < 16; ++r) az[m][i][r] = 0.f;
    const uint16_t* zop = rec + G::ES;
#pragma unroll
    for (int m = 0; m < G::ZM; ++m)
#pragma unroll
      for (int kz = 0; kz < G::KZ; ++kz) {
        const bf16x8 A =
            *reinterpret_cast<const bf16x8*>(zop + ((m * G::KZ + kz) * 64 + lane) * 8);
#pragma unroll
        for (int i = 0; i < NQ; ++i) az[m][i] = mfma32(A, qf[i][kz], az[m][i]);
      }
#pragma unroll
    for (int i = 0; i < NQ; ++i) {
      float dsum = 0.f;
#pragma unroll
      for (int m = 0; m < G::ZM; ++m)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          // row sigma = 16m + r + R*g, i.e. element (16m + r) % 8 of fragment (16m + r) / 8
          const int x = 16 * m + r;
          const uint32_t w = __builtin_bit_cast(u32x4, qf[i][x >> 3])[(x & 7) >> 1];
          const float qa = (x & 1) ? bf16hi_f32(w) : bf16lo_f32(w);
          dsum += qa * az[m][i][r];
        }
      dpart[i] = dsum;
    }
  }

  // ---- causal squared-score attention inside the span -----------------------
  {
    int last_tile = qb * NT + NT - 1;
    const int last_key_tile = static_cast<int>((span_end - 1 - span0) / 32);
    if (last_tile > last_key_tile) last_tile = last_key_tile;
    const int nkb = last_tile + 1;
    // staging: K rows (D/8 chunks of 16 B per key) and V^T (pairs of keys x 8 dv)
    constexpr int KT = 32 * (D / 8);
    constexpr int VT = 16 * (DV / 8);
    u32x4 sk[(KT + NTH - 1) / NTH], sva[(VT + NTH - 1) / NTH], svb[(VT + NTH - 1) / NTH];
    auto fetch = [&](int kb) {
      const long long key0 = span0 + 32LL * kb;
      #pragma unroll
      for (int i = 0; i * NTH < KT; ++i) {
        const int task = tid + i * NTH;
        u32x4 w = {0u, 0u, 0u, 0u};
        if (task < KT) {
          const int row = task / (D / 8), ch = task % (D / 8);
          if (key0 + row < span_end)
            w = *reinterpret_cast<const u32x4*>(kh + (key0 + row) * D + 8 * ch);
        }
        sk[i] = w;
      }
      #pragma unroll
      for (int i = 0; i * NTH < VT; ++i) {
        const int task = tid + i * NTH;
        u32x4 a = {0u, 0u, 0u, 0u}, b = {0u, 0u, 0u, 0u};
        if (task < VT) {
          const int cg = task >> 4, p = task & 15;
          const long long ka = key0 + 2 * p;
          if (ka < span_end) a = *reinterpret_cast<const u32x4*>(vh + ka * DV + 8 * cg);
          if (ka + 1 < span_end) b = *reinterpret_cast<const u32x4*>(vh + (ka + 1) * DV + 8 * cg);
        }
        sva[i] = a;
        svb[i] = b;
      }
    };
    auto commit = [&](int buf) {
      uint16_t* Ks = lds + buf * KVBUF;
      uint16_t* Vs = Ks + 32 * KROW;
      #pragma unroll
      for (int i = 0; i * NTH < KT; ++i) {
        const int task = tid + i * NTH;
        if (task < KT) {
          const int row = task / (D / 8), ch = task % (D / 8);
          *reinterpret_cast<u32x4*>(Ks + row * KROW + 8 * ch) = sk[i];
        }
      }
      #pragma unroll
      for (int i = 0; i * NTH < VT; ++i) {
        const int task = tid + i * NTH;
        if (task < VT) {
          const int cg = task >> 4, p = task & 15;
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const uint32_t a = sva[i][e], b = svb[i][e];
            *reinterpret_cast<uint32_t*>(Vs + (8 * cg + 2 * e) * VROW + 2 * p) =
                (a & 0xFFFFu) | (b << 16);
            *reinterpret_cast<uint32_t*>(Vs + (8 * cg + 2 * e + 1) * VROW + 2 * p) =
                (a >> 16) | (b & 0xFFFF0000u);
          }
        }
      }
    };
    fetch(0);
    commit(0);
    __syncthreads();
    for (int kb = 0; kb < nkb; ++kb) {
      const int buf = kb & 1;
      if (kb + 1 < nkb) fetch(kb + 1);
      const uint16_t* Ks = lds + buf * KVBUF;
      const uint16_t* Vs = Ks + 32 * KROW;
      bool need[NQ];
      bool any = false;
#pragma unroll
      for (int i = 0; i < NQ; ++i) {
        need[i] = tlive[i] && kb <= tile[i];
        any = any || need[i];
      }
      if (any) {
        // S^T = K_blk Q^T : rows = keys, columns = queries
        f32x16 sc[NQ];
#pragma unroll
        for (int i = 0; i < NQ; ++i)
#pragma unroll
          for (int r = 0; r < 16; ++r) sc[i][r] = 0.f;
#pragma unroll
        for (int kz = 0; kz < G::KZ; ++kz) {
          const bf16x8 A = *reinterpret_cast<const bf16x8*>(Ks + c * KROW + 8 * kz + R * g);
#pragma unroll
          for (int i = 0; i < NQ; ++i)
            if (need[i]) sc[i] = mfma32(A, qf[i][kz], sc[i]);
        }
        // V^T fragments: keys 16*kv + 4g + (0..3) and 16*kv + 8 + 4g + (0..3)
        bf16x8 va[G::MT][2];
#pragma unroll
        for (int m = 0; m < G::MT; ++m)
#pragma unroll
          for (int kv = 0; kv < 2; ++kv) {
            const uint16_t* row = Vs + (32 * m + c) * VROW + 16 * kv + 4 * g;
            const uint2 lo = *reinterpret_cast<const uint2*>(row);
            const uint2 hi = *reinterpret_cast<const uint2*>(row + 8);
            u32x4 w = {lo.x, lo.y, hi.x, hi.y};
            va[m][kv] = __builtin_bit_cast(bf16x8, w);
          }
#pragma unroll
        for (int i = 0; i < NQ; ++i) {
          if (!need[i]) continue;
          const bool diag = (kb == tile[i]);
          float p[16];
          float dsum = 0.f;
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int key = 8 * (r >> 2) + 4 * g + (r & 3);
            float x = sc[i][r] * sc[i][r];
            if (diag && key > c) x = 0.f;
            p[r] = x;
            dsum += x;
          }
          dpart[i] += dsum;
#pragma unroll
          for (int kv = 0; kv < 2; ++kv) {
            u32x4 w;
#pragma unroll
            for (int e = 0; e < 4; ++e) w[e] = pack_bf16x2(p[8 * kv + 2 * e], p[8 * kv + 2 * e + 1]);
            const bf16x8 Bp = __builtin_bit_cast(bf16x8, w);
#pragma unroll
            for (int m = 0; m < G::MT; ++m) acc[m][i] = mfma32(va[m][kv], Bp, acc[m][i]);
          }
        }
      }
      if (kb + 1 < nkb) commit(buf ^ 1);
      __syncthreads();
    }
  }

  // ---- readout of the span prefix: Phi_w(Q) S_pre ----------------------------
  {
    // rotated fp32 query rows: qr[i][x] = q[t][(x + R*g) % D]
    float qr[NQ][D];
#pragma unroll
    for (int i = 0; i < NQ; ++i) {
      const long long t = tq0[i] + c;
#pragma unroll
      for (int ch = 0; ch < D / 8; ++ch) {
        u32x4 w = {0u, 0u, 0u, 0u};
        if (t < span_end)
          w = *reinterpret_cast<const u32x4*>(qh + t * D + ((8 * ch + R * g) % D));
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          qr[i][8 * ch + 2 * e] = bf16lo_f32(w[e]);
          qr[i][8 * ch + 2 * e + 1] = bf16hi_f32(w[e]);
        }
      }
    }
    const uint16_t* Sg = rec;  // [DV][NSLOT]
    constexpr int NSTAGE = (G::NKS + kKC - 1) / kKC;
    // staging of one block: DV rows x (16*kKC) slots, 16 B per task
    constexpr int CH = 2 * kKC;  // 16-byte chunks per row
    constexpr int STASK = DV * CH;
    u32x4 sst[(STASK + NTH - 1) / NTH];
    auto sfetch = [&](int stg) {
      const int kc = (G::NKS - stg * kKC < kKC) ? (G::NKS - stg * kKC) : kKC;
      #pragma unroll
      for (int i = 0; i * NTH < STASK; ++i) {
        const int task = tid + i * NTH;
        u32x4 w = {0u, 0u, 0u, 0u};
        if (task < STASK) {
          const int row = task / CH, ch = task % CH;
          if (ch < 2 * kc)
            w = *reinterpret_cast<const u32x4*>(Sg + static_cast<long long>(row) * G::NSLOT +
                                                 16 * kKC * stg + 8 * ch);
        }
        sst[i] = w;
      }
    };
    auto scommit = [&](int buf) {
      uint16_t* Sb = lds + buf * SBUF;
      #pragma unroll
      for (int i = 0; i * NTH < STASK; ++i) {
        const int task = tid + i * NTH;
        if (task < STASK) {
          const int row = task / CH, ch = task % CH;
          *reinterpret_cast<u32x4*>(Sb + row * SROW + 8 * ch) = sst[i];
        }
      }
    };
    sfetch(0);
    scommit(0);
    __syncthreads();
    static_for<0, NSTAGE>([&](auto stg_c) {
      constexpr int stg = decltype(stg_c)::value;
      constexpr int k0 = stg * kKC;
      constexpr int kc = (G::NKS - k0 < kKC) ? (G::NKS - k0) : kKC;
      if constexpr (stg + 1 < NSTAGE) sfetch(stg + 1);
      const uint16_t* Sb = lds + (stg & 1) * SBUF;
      static_for<0, kc>([&](auto kk_c) {
        constexpr int kk = decltype(kk_c)::value;
        constexpr int kap = k0 + kk;
        constexpr int r1 = (8 * kap) % R;
        constexpr int dl = (8 * kap) / R;
        bf16x8 A[G::MT];
#pragma unroll
        for (int m = 0; m < G::MT; ++m)
          A[m] = *reinterpret_cast<const bf16x8*>(Sb + (32 * m + c) * SROW + 16 * kk + 8 * g);
#pragma unroll
        for (int i = 0; i < NQ; ++i) {
          u32x4 w;
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const float p0 = qr[i][r1 + 2 * e] * qr[i][r1 + 2 * e + dl];
            const float p1 = qr[i][r1 + 2 * e + 1] * qr[i][r1 + 2 * e + 1 + dl];
            w[e] = pack_bf16x2(p0, p1);
          }
          const bf16x8 B = __builtin_bit_cast(bf16x8, w);
#pragma unroll
          for (int m = 0; m < G::MT; ++m) acc[m][i] = mfma32(A[m], B, acc[m][i]);
        }
      });
      if constexpr (stg + 1 < NSTAGE) scommit((stg + 1) & 1);
      __syncthreads();
    });
  }

  // ---- normalise and store ---------------------------------------------------
#pragma unroll
  for (int i = 0; i < NQ; ++i) {
    const float Dt = dpart[i] + __shfl_xor(dpart[i], 32);
    const long long t = tq0[i] + c;
    if (!tlive[i] || t >= span_end) continue;
    const float inv = (Dt > 0.f) ? 1.f / Dt : 0.f;
    float* orow = out + (static_cast<long long>(bh) * T + t) * DV;
#pragma unroll
    for (int m = 0; m < G::MT; ++m)
#pragma unroll
      for (int r4 = 0; r4 < 4; ++r4) {
        float4 o;
        o.x = acc[m][i][4 * r4 + 0] * inv;
        o.y = acc[m][i][4 * r4 + 1] * inv;
        o.z = acc[m][i][4 * r4 + 2] * inv;
        o.w = acc[m][i][4 * r4 + 3] * inv;
        *reinterpret_cast<float4*>(orow + 32 * m + 8 * r4 + 4 * g) = o;
      }
  }
}

// ---------------------------------------------------------------------------
// Host side
// ---------------------------------------------------------------------------
bool mfma_supported(int d, int dv, int C) {
  return (d == 64 || d == 32) && dv == 64 && C > 0 && C % 32 == 0 && C <= 1024;
}

template <int D, int DV>
static long long record_elems() {
  return Geo<D, DV>::E;
}

static long long mfma_record(int d, int dv) {
  if (d == 64) return record_elems<64, 64>();
  return record_elems<32, 64>();
  (void)dv;
}

static size_t align256(size_t x) { return (x + 255) & ~static_cast<size_t>(255); }

size_t mfma_forward_workspace(int BH, int T, int d, int dv, int L) {
  const size_t NS = (static_cast<size_t>(T) + L - 1) / L;
  const size_t recs = static_cast<size_t>(BH) * NS * static_cast<size_t>(mfma_record(d, dv));
  return align256(recs * sizeof(float)) + align256(recs * sizeof(uint16_t));
}

template <int D, int DV>
static hipError_t run_mfma(const void* q, const void* k, const void* v, float* out, int BH, int T,
                           int L, void* ws, hipStream_t st, hipEvent_t* ev) {
  using G = Geo<D, DV>;
  const int NS = (T + L - 1) / L;
  const size_t recs = static_cast<size_t>(BH) * NS * G::E;
  float* spanst = static_cast<float*>(ws);
  uint16_t* pre = reinterpret_cast<uint16_t*>(static_cast<char*>(ws) + align256(recs * sizeof(float)));
  constexpr int UW = (D == 64) ? 6 : 5;
  constexpr int NUNITS = G::NST + G::ZM;
  const int ub = (NUNITS + 4 * UW - 1) / (4 * UW);
  hipError_t e = record(ev, 0, st);
  if (e != hipSuccess) return e;
  span_state_kernel<D, DV, UW><<<dim3(ub, NS, BH), 256, 0, st>>>(
      static_cast<const uint16_t*>(k), static_cast<const uint16_t*>(v), spanst, T, L);
  if ((e = record(ev, 1, st)) != hipSuccess) return e;
  dim3 g3(static_cast<unsigned>((G::E + kEB - 1) / kEB), BH);
  scan_exclusive<bf16_t, SlotWeight<D, DV>><<<g3, 256, 0, st>>>(
      spanst, reinterpret_cast<bf16_t*>(pre), NS, G::E, static_cast<long long>(NS) * G::E,
      SlotWeight<D, DV>{});
  if ((e = record(ev, 2, st)) != hipSuccess) return e;
  // query tiles: W waves x NQ tiles of 32 per workgroup, within one span
  const int tiles = (L + 31) / 32;
  const uint16_t* qq = static_cast<const uint16_t*>(q);
  const uint16_t* kk = static_cast<const uint16_t*>(k);
  const uint16_t* vv = static_cast<const uint16_t*>(v);
  if (tiles >= 8) {
    span_output_kernel<D, DV, 2, 4><<<dim3((tiles + 7) / 8, NS, BH), 256, 0, st>>>(qq, kk, vv, pre, out, T, L);
  } else if (tiles >= 4) {
    span_output_kernel<D, DV, 2, 2><<<dim3((tiles + 3) / 4, NS, BH), 128, 0, st>>>(qq, kk, vv, pre, out, T, L);
  } else if (tiles >= 2) {
    span_output_kernel<D, DV, 2, 1><<<dim3((tiles + 1) / 2, NS, BH), 64, 0, st>>>(qq, kk, vv, pre, out, T, L);
  } else {
    span_output_kernel<D, DV, 1, 1><<<dim3(1, NS, BH), 64, 0, st>>>(qq, kk, vv, pre, out, T, L);
  }
  if ((e = hipGetLastError()) != hipSuccess) return e;
  return record(ev, 3, st);
}

hipError_t launch_mfma_forward(const void* q, const void* k, const void* v, float* out, int BH,
                               int T, int d, int dv, int L, void* ws, hipStream_t st,
                               hipEvent_t* ev) {
  if (d == 64 && dv == 64) return run_mfma<64, 64>(q, k, v, out, BH, T, L, ws, st, ev);
  if (d == 32 && dv == 64) return run_mfma<32, 64>(q, k, v, out, BH, T, L, ws, st, ev);
  return hipErrorInvalidValue;
}

}  // namespace kata
