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
//                    Phi(K) generated on chip (never written to HBM); writes the
//                    span record in bf16 and the span's V^T for K4.
//   K3  scan       : in-place exclusive Blelloch prefix over the span records
//                    (kata_scan.hpp), fp32 sums, written back as bf16 MFMA
//                    operands with the feature weights.
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
// Small device helpers
// ---------------------------------------------------------------------------
typedef __attribute__((address_space(3))) void lds_void_t;

// One 16-byte global -> LDS copy per lane (gfx950 global_load_lds_dwordx4):
// lane l of the wave lands at lds_wave_base + 16*l; lds_wave_base must be the
// same for the whole wave.  Counted by vmcnt.  Issued from inline assembly so
// that the compiler's wait-count pass does not track these copies: it cannot
// tell which stage buffer a copy targets and would drain every copy in flight
// before each LDS read.  Callers therefore (1) wait for vmcnt 0 before a
// pipeline starts, so no compiler-issued vector-memory load is outstanding
// underneath the copies, (2) issue no other vector-memory operations while
// copies are in flight, and (3) consume a stage only after wait_vmcnt + an LDS
// barrier.  The "memory" clobber keeps the compiler from moving LDS accesses
// across the copy.
__device__ __forceinline__ void g2lds16(const void* gsrc, void* lds_wave_base) {
  const uint32_t lds = static_cast<uint32_t>(reinterpret_cast<uintptr_t>((lds_void_t*)lds_wave_base));
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off"
               :
               : "v"(gsrc), "s"(lds)
               : "memory", "m0");
}

// Wait until at most N vector-memory operations of this wave are in flight
// (lgkm and exp counters left alone).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 0xF) | (((N >> 4) & 3) << 14) | (0x7 << 4) | (0xF << 8));
}

// Workgroup barrier that orders LDS only: this wave's LDS operations are
// complete (lgkmcnt 0), then s_barrier.  Unlike __syncthreads() it does not
// wait for outstanding vector-memory operations, so global -> LDS copies of
// later stages stay in flight; callers wait for the stage they consume with
// wait_vmcnt first.  The signal fences keep the compiler from moving memory
// accesses across the barrier.
__device__ __forceinline__ void lds_barrier() {
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
  __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0), vmcnt and expcnt unchanged
  __builtin_amdgcn_s_barrier();
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
}

// 32-bit word j (0..3) of a 16-byte fragment, j known at compile time after
// unrolling.
__device__ __forceinline__ uint32_t word_of(const bf16x8& f, int j) {
  const uint4 w = __builtin_bit_cast(uint4, f);
  return j == 0 ? w.x : (j == 1 ? w.y : (j == 2 ? w.z : w.w));
}

// The eight state features of one lane's B fragment: for token pairs
// e = 0..3, y[e] holds (k_y(t), k_y(t+1)) and xl/xh the masked pairs
// (k_x(t), 0) and (0, k_x(t+1)).  v_dot2_f32_bf16 with a zero accumulator and
// one zero lane returns the exact fp32 product.  The eight dot products are
// issued back to back and followed by s_nop: the hardware does not interlock a
// dot-product result read by the next few VALU instructions, and the compiler
// cannot insert those wait states for instructions it does not see.
__device__ __forceinline__ void dot2x8(const uint32_t y[4], const uint32_t xl[4],
                                       const uint32_t xh[4], float p[8]) {
  asm volatile(
      "v_dot2_f32_bf16 %0, %8, %12, 0\n\t"
      "v_dot2_f32_bf16 %1, %8, %16, 0\n\t"
      "v_dot2_f32_bf16 %2, %9, %13, 0\n\t"
      "v_dot2_f32_bf16 %3, %9, %17, 0\n\t"
      "v_dot2_f32_bf16 %4, %10, %14, 0\n\t"
      "v_dot2_f32_bf16 %5, %10, %18, 0\n\t"
      "v_dot2_f32_bf16 %6, %11, %15, 0\n\t"
      "v_dot2_f32_bf16 %7, %11, %19, 0\n\t"
      "s_nop 4"
      : "=&v"(p[0]), "=&v"(p[1]), "=&v"(p[2]), "=&v"(p[3]), "=&v"(p[4]), "=&v"(p[5]),
        "=&v"(p[6]), "=&v"(p[7])
      : "v"(y[0]), "v"(y[1]), "v"(y[2]), "v"(y[3]), "v"(xl[0]), "v"(xl[1]), "v"(xl[2]),
        "v"(xl[3]), "v"(xh[0]), "v"(xh[1]), "v"(xh[2]), "v"(xh[3]));
}

// XOR swizzles of 16-byte chunks inside LDS rows; a row's logical chunk c is
// stored at position c ^ swz(row), which spreads the rows that one ds_read_b128
// touches over distinct bank groups.
template <int D>
__device__ __forceinline__ int kswz(int r) {
  if constexpr (D == 64) return (r ^ (r >> 3)) & 7;  // 8 chunks per key row
  else return ((r >> 1) ^ (r >> 3)) & 3;             // 4 chunks per key row
}
__device__ __forceinline__ int rswz(int m) { return m & 15; }  // rows of >= 16 chunks

// ---------------------------------------------------------------------------
// K2: span state.  grid (UB + 1, NS, BH), block 256 (4 waves).
// Blocks 0..UB-1: slot tiles.  Wave w of block ub owns tiles
// [(4*ub + w)*UW, +UW); every wave runs the same branch-free MFMA loop (tiles
// past the last one compute on a valid row and skip their store), so the
// accumulators stay in place.  Block UB: Z = K^T K (one 32x32 tile per wave)
// and the span's V^T (bf16, [dv][LV], keys of every 16-key group in the order
// 0-3, 8-11, 4-7, 12-15, the K order of the output kernel's P V product).
// Writes the span record (bf16): S^T as [dv][NSLOT], then Z in operand order.
// ---------------------------------------------------------------------------
constexpr int kTB2 = 64;            // tokens per staged block
constexpr int kRow2 = kTB2 + 8;     // LDS row length (bf16), 144 B

template <int D, int DV, int UW>
__global__ __launch_bounds__(256) void span_state_kernel(const uint16_t* __restrict__ k,
                                                         const uint16_t* __restrict__ v,
                                                         uint16_t* __restrict__ spanst,
                                                         uint16_t* __restrict__ vtp, int T,
                                                         int L, int LV) {
  using G = Geo<D, DV>;
  constexpr int NXR = D / 32;  // distinct x rows per lane (x depends on tile % NXR)
  static_assert(UW % NXR == 0, "unit parity must be static");
  __shared__ __attribute__((aligned(16))) uint16_t kT[2][D][kRow2];
  __shared__ __attribute__((aligned(16))) uint16_t vT[2][DV][kRow2];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int c = lane & 31, g = lane >> 5;
  const int s = blockIdx.y, bh = blockIdx.z;
  const bool zblock = blockIdx.x == gridDim.x - 1;
  const long long span0 = static_cast<long long>(s) * L;
  const long long span_end = min(static_cast<long long>(T), span0 + L);
  const uint16_t* kh = k + static_cast<long long>(bh) * T * D;
  const uint16_t* vh = v + static_cast<long long>(bh) * T * DV;
  const int unit0 = (blockIdx.x * 4 + wave) * UW;

  int xrow[NXR];
#pragma unroll
  for (int p = 0; p < NXR; ++p) {
    int yy;
    slot_pair<D>(32 * p + c, xrow[p], yy);
  }
  int yrow[UW];
#pragma unroll
  for (int u = 0; u < UW; ++u) {
    int xx;
    const int unit = unit0 + u < G::NST ? unit0 + u : G::NST - 1;  // valid row; store skipped
    slot_pair<D>(32 * unit + c, xx, yrow[u]);
  }

  // staging: task -> (pair p of tokens, 8-wide column group); K then V
  constexpr int KG = D / 8, VG = DV / 8;
  constexpr int NTASK = 32 * (KG + VG);
  constexpr int TPT = (NTASK + 255) / 256;
  uint4 st_lo[TPT], st_hi[TPT];
  auto fetch = [&](long long t0) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < TPT; ++i) {
      const int task = tid + 256 * i;
      const int cg = task >> 5, p = task & 31;
      const long long ta = t0 + 2 * p, tb = ta + 1;
      st_lo[i] = make_uint4(0u, 0u, 0u, 0u);
      st_hi[i] = make_uint4(0u, 0u, 0u, 0u);
      if (task < NTASK) {
        if (cg < KG) {
          if (ta < span_end) st_lo[i] = *reinterpret_cast<const uint4*>(kh + ta * D + 8 * cg);
          if (tb < span_end) st_hi[i] = *reinterpret_cast<const uint4*>(kh + tb * D + 8 * cg);
        } else {
          const int vg = cg - KG;
          if (ta < span_end) st_lo[i] = *reinterpret_cast<const uint4*>(vh + ta * DV + 8 * vg);
          if (tb < span_end) st_hi[i] = *reinterpret_cast<const uint4*>(vh + tb * DV + 8 * vg);
        }
      }
    }
  };
  auto commit = [&](int buf) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < TPT; ++i) {
      const int task = tid + 256 * i;
      if (task >= NTASK) continue;
      const int cg = task >> 5, p = task & 31;
      uint16_t* base = (cg < KG) ? &kT[buf][8 * cg][0] : &vT[buf][8 * (cg - KG)][0];
      const uint32_t a[4] = {st_lo[i].x, st_lo[i].y, st_lo[i].z, st_lo[i].w};
      const uint32_t b[4] = {st_hi[i].x, st_hi[i].y, st_hi[i].z, st_hi[i].w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        // element 2e: (a.lo, b.lo); element 2e+1: (a.hi, b.hi)
        *reinterpret_cast<uint32_t*>(base + (2 * e) * kRow2 + 2 * p) =
            __builtin_amdgcn_perm(b[e], a[e], 0x05040100u);
        *reinterpret_cast<uint32_t*>(base + (2 * e + 1) * kRow2 + 2 * p) =
            __builtin_amdgcn_perm(b[e], a[e], 0x07060302u);
      }
    }
  };
  const int nblk = static_cast<int>((span_end - span0 + kTB2 - 1) / kTB2);
  uint16_t* rec = spanst + (static_cast<long long>(bh) * gridDim.y + s) * G::E;

  if (zblock) {
    // ---- Z = K^T K over the span, and the span's V^T for the output kernel ----
    uint16_t* vt_rec = vtp + (static_cast<long long>(bh) * gridDim.y + s) * DV * LV;
    const int zm = wave / G::ZM, zn = wave % G::ZM;  // this wave's 32x32 tile of Z
    const bool zwave = wave < G::ZM * G::ZM;
    f32x16 zacc;
#pragma unroll
    for (int r = 0; r < 16; ++r) zacc[r] = 0.f;
    fetch(span0);
    commit(0);
    lds_barrier();
    for (int bi = 0; bi < nblk; ++bi) {
      const int buf = bi & 1;
      if (bi + 1 < nblk) fetch(span0 + static_cast<long long>(bi + 1) * kTB2);
#pragma unroll
      for (int i = 0; i < (DV * 8) / 256; ++i) {
        const int task = tid + 256 * i;
        const int m = task >> 3, h = task & 7;  // row, output chunk of 8 keys
        const int grp = h >> 1, hg = h & 1;
        const uint16_t* row = &vT[buf][m][16 * grp + 4 * hg];
        const uint2 lo = *reinterpret_cast<const uint2*>(row);
        const uint2 hi = *reinterpret_cast<const uint2*>(row + 8);
        *reinterpret_cast<uint4*>(vt_rec + static_cast<long long>(m) * LV + kTB2 * bi + 8 * h) =
            make_uint4(lo.x, lo.y, hi.x, hi.y);
      }
      if (zwave) {
#pragma unroll
        for (int ks = 0; ks < kTB2 / 16; ++ks) {
          const int col = 16 * ks + 8 * g;
          const bf16x8 Az = *reinterpret_cast<const bf16x8*>(&kT[buf][32 * zm + c][col]);
          const bf16x8 Bz = *reinterpret_cast<const bf16x8*>(&kT[buf][32 * zn + c][col]);
          zacc = mfma32(Az, Bz, zacc);
        }
      }
      if (bi + 1 < nblk) commit(buf ^ 1);
      lds_barrier();
    }
    if (zwave) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int a = 32 * zm + 8 * (r >> 2) + 4 * g + (r & 3);
        const int b = 32 * zn + c;
        __bf16 h = static_cast<__bf16>(zacc[r]);
        rec[G::ES + zop_index<D>(a, b)] = __builtin_bit_cast(uint16_t, h);
      }
    }
    return;
  }

  // ---- S_span^T = V^T Phi(K) for this wave's slot tiles ----------------------
  f32x16 acc[UW][G::MT];
#pragma unroll
  for (int u = 0; u < UW; ++u)
#pragma unroll
    for (int m = 0; m < G::MT; ++m)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[u][m][r] = 0.f;
  fetch(span0);
  commit(0);
  lds_barrier();
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
      // masked x pairs: (x_t, 0) and (0, x_{t+1}) for each token pair
      uint32_t xl[NXR][4], xh[NXR][4];
#pragma unroll
      for (int p = 0; p < NXR; ++p) {
        const uint4 X4 = *reinterpret_cast<const uint4*>(&kT[buf][xrow[p]][col]);
        const uint32_t X[4] = {X4.x, X4.y, X4.z, X4.w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          xl[p][e] = X[e] & 0x0000FFFFu;
          xh[p][e] = X[e] & 0xFFFF0000u;
        }
      }
#pragma unroll
      for (int u = 0; u < UW; ++u) {
        const int p = u % NXR;
        const uint4 Y4 = *reinterpret_cast<const uint4*>(&kT[buf][yrow[u]][col]);
        const uint32_t Y[4] = {Y4.x, Y4.y, Y4.z, Y4.w};
        float pr[8];
        dot2x8(Y, xl[p], xh[p], pr);
        const bf16x8 Bf = __builtin_bit_cast(
            bf16x8, make_uint4(pack_bf16x2(pr[0], pr[1]), pack_bf16x2(pr[2], pr[3]),
                               pack_bf16x2(pr[4], pr[5]), pack_bf16x2(pr[6], pr[7])));
#pragma unroll
        for (int m = 0; m < G::MT; ++m) acc[u][m] = mfma32(va[m], Bf, acc[u][m]);
      }
    }
    if (bi + 1 < nblk) commit(buf ^ 1);
    lds_barrier();
  }

  // write this wave's tiles of the span record (bf16)
#pragma unroll
  for (int u = 0; u < UW; ++u) {
    const int unit = unit0 + u;
    if (unit < G::NST) {
#pragma unroll
      for (int m = 0; m < G::MT; ++m)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int dvrow = 32 * m + 8 * (r >> 2) + 4 * g + (r & 3);
          __bf16 h = static_cast<__bf16>(acc[u][m][r]);
          rec[static_cast<long long>(dvrow) * G::NSLOT + 32 * unit + c] =
              __builtin_bit_cast(uint16_t, h);
        }
    }
  }
}

// ---------------------------------------------------------------------------
// K4: span output.  grid (query blocks per span, NS, BH), block 256 (4 waves),
// one workgroup per CU (96 KB of LDS in three 32 KB stage buffers).
// The workgroup owns 8 query tiles of 32 (span-relative tile index 8*qb + i);
// wave w takes tiles {w, 7-w}, which balances the causal work.
// Operands are staged by direct global -> LDS copies, three stages deep, so no
// registers hold staged data and the copies of stage s+2 overlap the
// arithmetic of stage s.
// pre[bh][s][E] bf16: weighted S_pre^T as [dv][NSLOT], then Z_pre (operand order).
// vtp[bh][s][dv][L] bf16: the span's V^T (permuted keys, see K2).
// ---------------------------------------------------------------------------
constexpr int kKB = 128;        // keys per intra stage
constexpr int kUnrolledStages = 8;  // intra stages handled in straight-line code
constexpr int kKC = 16;         // readout K-steps per stage
constexpr int kStageBytes = 32768;

__shared__ __attribute__((aligned(16))) uint16_t g_stage0[kStageBytes / 2];
__shared__ __attribute__((aligned(16))) uint16_t g_stage1[kStageBytes / 2];
__shared__ __attribute__((aligned(16))) uint16_t g_stage2[kStageBytes / 2];

template <int D, int DV>
__global__ __launch_bounds__(256) void span_output_kernel(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ k,
    const uint16_t* __restrict__ pre, const uint16_t* __restrict__ vtp, float* __restrict__ out,
    int T, int L, int LV) {
  using G = Geo<D, DV>;
  constexpr int R = G::R;
  constexpr int NQ = 2, W = 4, NT = 8;
  constexpr int KCH = D / 8;                    // 16-byte chunks per key row
  constexpr int KCHUNKS = kKB * KCH;            // K rows of one intra stage
  constexpr int VCH = kKB / 8;                  // chunks per V^T row of one stage (16)
  constexpr int VCHUNKS = DV * VCH;
  constexpr int ICH = KCHUNKS + VCHUNKS;        // chunks per intra stage
  static_assert(ICH * 16 <= kStageBytes && ICH % 256 == 0, "intra stage size");
  constexpr int IPW_I = ICH / 256;              // copy instructions per wave, intra
  constexpr int SCH = 2 * kKC;                  // chunks per S_pre row of one stage (32)
  constexpr int SCHUNKS = DV * SCH;
  static_assert(SCHUNKS * 16 <= kStageBytes && SCHUNKS % 256 == 0, "readout stage size");
  constexpr int IPW_R = SCHUNKS / 256;
  constexpr int NSTAGE_R = (G::NKS + kKC - 1) / kKC;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int c = lane & 31, g = lane >> 5;
  const int qb = blockIdx.x, s = blockIdx.y, bh = blockIdx.z;
  const long long span0 = static_cast<long long>(s) * L;
  const long long span_end = min(static_cast<long long>(T), span0 + L);
  const long long wg_q0 = span0 + static_cast<long long>(qb) * NT * 32;
  if (wg_q0 >= span_end) return;  // whole workgroup beyond the sequence
  const uint16_t* qh = q + static_cast<long long>(bh) * T * D;
  const uint16_t* kh = k + static_cast<long long>(bh) * T * D;
  const uint16_t* rec = pre + (static_cast<long long>(bh) * gridDim.y + s) * G::E;
  const uint16_t* vt_rec = vtp + (static_cast<long long>(bh) * gridDim.y + s) * DV * LV;

  int tile[NQ];
  long long tq0[NQ];
  bool tlive[NQ];
#pragma unroll
  for (int i = 0; i < NQ; ++i) {
    const int local = (i == 0) ? wave : 2 * W - 1 - wave;
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
      uint4 w = make_uint4(0u, 0u, 0u, 0u);
      if (t < span_end) w = *reinterpret_cast<const uint4*>(qh + t * D + 8 * kz + R * g);
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
          // row sigma = 16m + r + R*g: element (16m + r) % 8 of fragment (16m + r) / 8
          const int x = 16 * m + r;
          const uint32_t w = word_of(qf[i][x >> 3], (x & 7) >> 1);
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
    const int nstage = (last_tile + 1 + 3) / 4;  // 128-key stages
    // issue the copies of intra stage st into buffer `buf`
    auto issue = [&](int st, uint16_t* buf) __attribute__((always_inline)) {
      const long long key0 = span0 + static_cast<long long>(st) * kKB;
#pragma unroll
      for (int i = 0; i < IPW_I; ++i) {
        const int P = (i * W + wave) * 64 + lane;  // LDS chunk written by this lane
        const void* src;
        if (P < KCHUNKS) {
          const int r = P / KCH, pos = P % KCH;
          const int cl = pos ^ kswz<D>(r);
          long long key = key0 + r;
          if (key > T - 1) key = T - 1;  // in bounds; such keys are never used
          src = kh + key * D + 8 * cl;
        } else {
          const int P2 = P - KCHUNKS;
          const int m = P2 / VCH, pos = P2 % VCH;
          const int cl = pos ^ rswz(m);
          src = vt_rec + static_cast<long long>(m) * LV + st * kKB + 8 * cl;
        }
        g2lds16(src, buf + (i * W + wave) * 512);
      }
    };
    auto compute = [&](int st, const uint16_t* Ks) __attribute__((always_inline)) {
      const uint16_t* Vs = Ks + KCHUNKS * 8;
#pragma unroll
      for (int sb = 0; sb < kKB / 32; ++sb) {
        const int kb = 4 * st + sb;  // 32-key block inside the span
        bool need[NQ];
        bool any = false;
#pragma unroll
        for (int i = 0; i < NQ; ++i) {
          need[i] = tlive[i] && kb <= tile[i];
          any = any || need[i];
        }
        if (!any) continue;
        // S^T = K_blk Q^T : rows = keys, columns = queries
        f32x16 sc[NQ];
#pragma unroll
        for (int i = 0; i < NQ; ++i)
#pragma unroll
          for (int r = 0; r < 16; ++r) sc[i][r] = 0.f;
        const int krow = 32 * sb + c;
#pragma unroll
        for (int kz = 0; kz < G::KZ; ++kz) {
          const int cl = kz + (R / 8) * g;
          const bf16x8 A = *reinterpret_cast<const bf16x8*>(
              Ks + (krow * KCH + (cl ^ kswz<D>(krow))) * 8);
#pragma unroll
          for (int i = 0; i < NQ; ++i)
            if (need[i]) sc[i] = mfma32(A, qf[i][kz], sc[i]);
        }
        // V^T fragments (keys already in the P V K order)
        bf16x8 va[G::MT][2];
#pragma unroll
        for (int m = 0; m < G::MT; ++m)
#pragma unroll
          for (int kv = 0; kv < 2; ++kv) {
            const int vrow = 32 * m + c;
            const int cl = 4 * sb + 2 * kv + g;
            va[m][kv] = *reinterpret_cast<const bf16x8*>(Vs + (vrow * VCH + (cl ^ rswz(vrow))) * 8);
          }
#pragma unroll
        for (int i = 0; i < NQ; ++i) {
          if (!need[i]) continue;
          float p[16];
          float dsum = 0.f;
          if (kb == tile[i]) {
#pragma unroll
            for (int r = 0; r < 16; ++r) {
              const int key = 8 * (r >> 2) + 4 * g + (r & 3);
              const float x = sc[i][r] * sc[i][r];
              p[r] = (key > c) ? 0.f : x;
              dsum += p[r];
            }
          } else {
#pragma unroll
            for (int r = 0; r < 16; ++r) {
              p[r] = sc[i][r] * sc[i][r];
              dsum += p[r];
            }
          }
          dpart[i] += dsum;
#pragma unroll
          for (int kv = 0; kv < 2; ++kv) {
            uint4 w;
            w.x = pack_bf16x2(p[8 * kv + 0], p[8 * kv + 1]);
            w.y = pack_bf16x2(p[8 * kv + 2], p[8 * kv + 3]);
            w.z = pack_bf16x2(p[8 * kv + 4], p[8 * kv + 5]);
            w.w = pack_bf16x2(p[8 * kv + 6], p[8 * kv + 7]);
            const bf16x8 Bp = __builtin_bit_cast(bf16x8, w);
#pragma unroll
            for (int m = 0; m < G::MT; ++m) acc[m][i] = mfma32(va[m][kv], Bp, acc[m][i]);
          }
        }
      }
    };
    // three-deep pipeline over the stages; buffers chosen statically
    wait_vmcnt<0>();  // no compiler-issued loads underneath the copies
    issue(0, g_stage0);
    if (nstage > 1) issue(1, g_stage1);
    if (nstage <= kUnrolledStages) {
      // straight-line form (spans up to 1024 keys): the compiler can tell the
      // three buffers apart and inserts no extra waits on in-flight copies
      static_for<0, kUnrolledStages>([&](auto st_c) {
        constexpr int j = decltype(st_c)::value;
        if (j < nstage) {
          if (j + 1 < nstage) wait_vmcnt<IPW_I>(); else wait_vmcnt<0>();
          lds_barrier();
          if (j + 2 < nstage)
            issue(j + 2, (j + 2) % 3 == 0 ? g_stage0 : ((j + 2) % 3 == 1 ? g_stage1 : g_stage2));
          compute(j, j % 3 == 0 ? g_stage0 : (j % 3 == 1 ? g_stage1 : g_stage2));
        }
      });
    } else {
      for (int st = 0; st < nstage; st += 3) {
#pragma unroll
        for (int j = 0; j < 3; ++j) {
          const int cur = st + j;
          if (cur < nstage) {
            if (cur + 1 < nstage) wait_vmcnt<IPW_I>(); else wait_vmcnt<0>();
            lds_barrier();
            if (cur + 2 < nstage)
              issue(cur + 2, j == 0 ? g_stage2 : (j == 1 ? g_stage0 : g_stage1));
            compute(cur, j == 0 ? g_stage0 : (j == 1 ? g_stage1 : g_stage2));
          }
        }
      }
    }
    lds_barrier();  // every wave is done with the intra buffers
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
        uint4 w4 = make_uint4(0u, 0u, 0u, 0u);
        if (t < span_end)
          w4 = *reinterpret_cast<const uint4*>(qh + t * D + ((8 * ch + R * g) % D));
        const uint32_t w[4] = {w4.x, w4.y, w4.z, w4.w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          qr[i][8 * ch + 2 * e] = bf16lo_f32(w[e]);
          qr[i][8 * ch + 2 * e + 1] = bf16hi_f32(w[e]);
        }
      }
    }
    // stage stg holds slots [16*kKC*stg, +16*kKC) of every dv row
    auto issue = [&](int stg, uint16_t* buf) __attribute__((always_inline)) {
      const int kc = (G::NKS - stg * kKC < kKC) ? (G::NKS - stg * kKC) : kKC;
#pragma unroll
      for (int i = 0; i < IPW_R; ++i) {
        const int P = (i * W + wave) * 64 + lane;
        const int m = P / SCH, pos = P % SCH;
        int cl = pos ^ rswz(m);
        if (cl >= 2 * kc) cl = 0;  // past the last K-step: any in-record chunk, never read
        const void* src = rec + static_cast<long long>(m) * G::NSLOT + 16 * kKC * stg + 8 * cl;
        g2lds16(src, buf + (i * W + wave) * 512);
      }
    };
    auto compute = [&](auto stg_c, const uint16_t* Sb) __attribute__((always_inline)) {
      constexpr int stg = decltype(stg_c)::value;
      constexpr int k0 = stg * kKC;
      constexpr int kc = (G::NKS - k0 < kKC) ? (G::NKS - k0) : kKC;
      static_for<0, kc>([&](auto kk_c) {
        constexpr int kk = decltype(kk_c)::value;
        constexpr int kap = k0 + kk;
        constexpr int r1 = (8 * kap) % R;
        constexpr int dl = (8 * kap) / R;
        bf16x8 A[G::MT];
#pragma unroll
        for (int m = 0; m < G::MT; ++m) {
          const int row = 32 * m + c;
          const int cl = 2 * kk + g;
          A[m] = *reinterpret_cast<const bf16x8*>(Sb + (row * SCH + (cl ^ rswz(row))) * 8);
        }
#pragma unroll
        for (int i = 0; i < NQ; ++i) {
          uint32_t wv[4];
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const float p0 = qr[i][r1 + 2 * e] * qr[i][r1 + 2 * e + dl];
            const float p1 = qr[i][r1 + 2 * e + 1] * qr[i][r1 + 2 * e + 1 + dl];
            wv[e] = pack_bf16x2(p0, p1);
          }
          const bf16x8 B = __builtin_bit_cast(bf16x8, make_uint4(wv[0], wv[1], wv[2], wv[3]));
#pragma unroll
          for (int m = 0; m < G::MT; ++m) acc[m][i] = mfma32(A[m], B, acc[m][i]);
        }
      });
    };
    wait_vmcnt<0>();  // the query rows are loaded; no compiler loads in flight
    issue(0, g_stage0);
    if constexpr (NSTAGE_R > 1) issue(1, g_stage1);
    static_for<0, NSTAGE_R>([&](auto stg_c) {
      constexpr int stg = decltype(stg_c)::value;
      if constexpr (stg + 1 < NSTAGE_R) wait_vmcnt<IPW_R>(); else wait_vmcnt<0>();
      lds_barrier();
      if constexpr (stg + 2 < NSTAGE_R)
        issue(stg + 2, (stg + 2) % 3 == 0 ? g_stage0 : ((stg + 2) % 3 == 1 ? g_stage1 : g_stage2));
      compute(stg_c, stg % 3 == 0 ? g_stage0 : (stg % 3 == 1 ? g_stage1 : g_stage2));
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

static long long mfma_record(int d) {
  return d == 64 ? Geo<64, 64>::E : Geo<32, 64>::E;
}

static size_t align256(size_t x) { return (x + 255) & ~static_cast<size_t>(255); }

// Span length rounded up to whole intra stages so that every staged key
// block lies inside the span's V^T record.
static int span_alloc(int L) { return (L + kKB - 1) / kKB * kKB; }

size_t mfma_forward_workspace(int BH, int T, int d, int dv, int L) {
  const size_t NS = (static_cast<size_t>(T) + L - 1) / L;
  const size_t recs = static_cast<size_t>(BH) * NS * static_cast<size_t>(mfma_record(d));
  const size_t vt = static_cast<size_t>(BH) * NS * dv * span_alloc(L);
  return align256(recs * sizeof(uint16_t)) + align256(vt * sizeof(uint16_t));
}

template <int D, int DV>
static hipError_t run_mfma(const void* q, const void* k, const void* v, float* out, int BH, int T,
                           int L, void* ws, hipStream_t st, hipEvent_t* ev) {
  using G = Geo<D, DV>;
  const int NS = (T + L - 1) / L;
  const int LA = span_alloc(L);
  const size_t recs = static_cast<size_t>(BH) * NS * G::E;
  uint16_t* spanst = static_cast<uint16_t*>(ws);
  uint16_t* vtp =
      reinterpret_cast<uint16_t*>(static_cast<char*>(ws) + align256(recs * sizeof(uint16_t)));
  const uint16_t* qq = static_cast<const uint16_t*>(q);
  const uint16_t* kk = static_cast<const uint16_t*>(k);
  const uint16_t* vv = static_cast<const uint16_t*>(v);
  constexpr int UW = 6;
  const int ub = (G::NST + 4 * UW - 1) / (4 * UW);  // slot-tile blocks; one more for Z
  hipError_t e = record(ev, 0, st);
  if (e != hipSuccess) return e;
  span_state_kernel<D, DV, UW><<<dim3(ub + 1, NS, BH), 256, 0, st>>>(kk, vv, spanst, vtp, T, L,
                                                                     LA);
  if ((e = record(ev, 1, st)) != hipSuccess) return e;
  dim3 g3(static_cast<unsigned>((G::E + kEB16 - 1) / kEB16), BH);
  scan_exclusive_bf16<SlotWeight<D, DV>><<<g3, 256, 0, st>>>(
      spanst, NS, G::E, static_cast<long long>(NS) * G::E, SlotWeight<D, DV>{});
  if ((e = record(ev, 2, st)) != hipSuccess) return e;
  const int qblocks = (L + 255) / 256;
  span_output_kernel<D, DV><<<dim3(qblocks, NS, BH), 256, 0, st>>>(qq, kk, spanst, vtp, out, T,
                                                                   L, LA);
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
