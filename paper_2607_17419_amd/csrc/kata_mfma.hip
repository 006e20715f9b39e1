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
//                    span record in bf16.
//   K3  scan       : in-place exclusive Blelloch prefix over the span records
//                    (kata_scan.hpp), fp32 sums, written back as bf16 MFMA
//                    operands with the feature weights.
//   K4  span_output: squared-score attention inside the span (QK^T on MFMA,
//                    squared and masked in registers, P V back through MFMA,
//                    V^T operands by transposing LDS reads of the V rows),
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

// Block-diagonal feature of KATA-Mg (section "From rank-one rays to low-rank
// PSD packing"): NG blocks of DM = D/NG consecutive coordinates, each with the
// slot layout of Geo<DM> (its own rotation R = DM/2), blocks side by side in a
// span record: S^T as [dv][NG * NSLOT_block], then NG Z blocks of DM x DM in
// operand order.  NG = 1 is KATA-M1 (GeoG<D, DV, 1> matches Geo<D, DV>).
template <int D, int DV, int NG>
struct GeoG {
  using Blk = Geo<D / NG, DV>;
  static constexpr int DM = D / NG;          // coordinates per block
  static constexpr int RM = Blk::R;          // rotation of a block's slots
  static constexpr int KZM = Blk::KZ;        // 16-wide K-steps over one block
  static constexpr int KZ = NG * KZM;        // score MFMAs per query tile and key block
  static constexpr int NKSM = Blk::NKS;      // readout K-steps of one block
  static constexpr int NKS = NG * NKSM;
  static constexpr int NSLOTM = Blk::NSLOT;
  static constexpr int NSLOT = NG * NSLOTM;
  static constexpr int NSTM = Blk::NST;      // 32-slot tiles of one block
  static constexpr int NST = NG * NSTM;
  static constexpr int MT = Blk::MT;
  static constexpr int ZMB = Blk::ZM;        // 32-wide Z tiles per block dim
  static constexpr long long ES = static_cast<long long>(DV) * NSLOT;
  static constexpr long long EZ = static_cast<long long>(NG) * DM * DM;
  static constexpr long long E = ES + EZ;
  static_assert(D % NG == 0 && DM % 32 == 0, "blocks of a multiple of 32 coordinates");
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

// Scan output weights: S region by slot (inside its block), Z region 1.
template <int D, int DV, int NG>
struct SlotWeight {
  __device__ __forceinline__ float operator()(long long e) const {
    using G = GeoG<D, DV, NG>;
    if (e >= G::ES) return 1.f;
    return slot_weight<G::DM>(static_cast<int>(e % G::NSLOT % G::NSLOTM));
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


// 32-bit word j (0..3) of a 16-byte fragment, j known at compile time after
// unrolling.
__device__ __forceinline__ uint32_t word_of(const bf16x8& f, int j) {
  const uint4 w = __builtin_bit_cast(uint4, f);
  return j == 0 ? w.x : (j == 1 ? w.y : (j == 2 ? w.z : w.w));
}

// Single MFMAs for sequences whose order the caller fixes with scheduling
// barriers (compiler builtins: the compiler inserts the wait states between
// an MFMA and the VALU instructions around it): mfma_a and mfma_v accumulate,
// mfma_vz starts a chain from zero.
__device__ __forceinline__ void mfma_a(f32x16& acc, const bf16x8& a, const bf16x8& b) {
  acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc, 0, 0, 0);
}
__device__ __forceinline__ void mfma_vz(f32x16& acc, const bf16x8& a, const bf16x8& b) {
  const f32x16 z = {};
  acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, z, 0, 0, 0);
}
__device__ __forceinline__ void mfma_v(f32x16& acc, const bf16x8& a, const bf16x8& b) {
  acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc, 0, 0, 0);
}

// Keeps the operand registers of recently issued MFMAs live up to this point,
// so the compiler does not reuse them for new values: an instruction that
// writes a register an MFMA in flight still reads waits for that MFMA to
// finish.  Emits nothing.
template <typename T>
__device__ __forceinline__ void hold1(const T& x) {
  asm volatile("" ::"v"(x));
}
template <typename... Ts>
__device__ __forceinline__ void hold(const Ts&... xs) {
  (hold1(xs), ...);
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
// K2: span state.  1-D grid of workgroups of 256 threads (4 waves).  A span
// gets NB blocks: NUW = ceil(NST / kUW) slot waves, then one wave for Z (any
// further wave only helps stage).  Block id -> (span, part) keeps the blocks
// of one span on one XCD (equal id % 8), dispatched back to back, so the later
// blocks' reads of the span's K and V hit that XCD's L2.
// Slot wave gw owns slot tiles [gw*kUW, +kUW); tiles past the last one
// compute on a valid row and skip their store, so every wave runs the same
// branch-free MFMA loop.  The Z wave computes Z = K^T K.
//
// Arithmetic.  K and V are staged transposed ([dim][token]) in fp16 through a
// three-buffer LDS ring in blocks of kTB2 tokens, and the state is an fp16
// MFMA product with fp32 accumulation: a feature k_x k_y of two tokens is one
// packed fp16 multiply (v_pk_mul_f16) of two staged fp16 pairs, the B operand
// as it stands, with no conversion step.  bf16 inputs convert to fp16 exactly
// within fp16's exponent range, so each span gets power-of-two scales:
//   * if the first staged block's largest |k| lies in [2^-4, 2^4) and its
//     largest |v| in [2^-8, 2^8), the span runs unscaled (no extra work);
//   * otherwise, or if the unscaled pass produced a non-finite state (a later
//     block outgrew fp16: an fp16 overflow becomes inf, caught when the state
//     is written), the workgroup reads the span once for its exact maxima and
//     runs again with k -> k 2^-ek, v -> v 2^-ev (largest |k|, |v| in [1, 2)),
//     undoing the scales exactly when it writes the record.
// Features are rounded once, to fp16 (unit roundoff 2^-11, finer than a bf16
// rounding); the records are written in bf16 as before.
//
// Writes the span record (bf16): S^T as [dv][NSLOT], then Z in operand order.
// ---------------------------------------------------------------------------
constexpr int kTB2 = 128;           // tokens per staged block
constexpr int kRow2 = kTB2 + 8;     // K^T / V^T row length in LDS (fp16): rows 272 B apart
constexpr int kGapK2 = 64;          // fp16 gap (32 banks) before key rows DM/2, DM, ... (krow)
constexpr int kUW = 6;              // slot tiles per slot wave (four-wave form)
constexpr int kNBuf2 = 3;           // LDS ring of staged blocks

typedef __attribute__((__vector_size__(8 * sizeof(_Float16)))) _Float16 f16x8;
typedef __attribute__((__vector_size__(4 * sizeof(_Float16)))) _Float16 f16x4;

// Workgroup shape of K2.  d = 64 runs eight waves of three slot tiles (two
// waves per SIMD: one wave's feature products and staging issue while the
// other's MFMAs run); d = 32 runs four waves of six tiles, one per SIMD (its
// staging tasks do not divide over 512 threads).
template <int D, int DV, int NG>
struct StateGrid {
  static constexpr int NW = D == 64 ? 8 : 4;  // waves per workgroup
  static constexpr int UW = NW == 8 ? 3 : kUW;  // slot tiles per slot wave
  // slot waves per feature block (a wave's tiles never straddle two blocks)
  static constexpr int NUWB = (GeoG<D, DV, NG>::NSTM + UW - 1) / UW;
  static constexpr int NUW = NG * NUWB;                   // slot waves per span
  static constexpr int NB = (NUW + 1 + NW - 1) / NW;      // workgroups per span
};

// Largest |x| of the bf16 values in the 32-bit words of v, as a bf16 bit
// pattern (the magnitude bits order like the magnitudes).
__device__ __forceinline__ uint32_t absmax_bits(uint32_t m, uint4 v) {
  const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const uint32_t lo = w[i] & 0x7FFFu, hi = (w[i] >> 16) & 0x7FFFu;
    m = max(m, max(lo, hi));
  }
  return m;
}

__device__ __forceinline__ uint32_t wave_max_u32(uint32_t x) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) x = max(x, static_cast<uint32_t>(__shfl_xor(static_cast<int>(x), o)));
  return x;
}

template <int D, int DV, int NG>
__global__ __launch_bounds__((64 * StateGrid<D, DV, NG>::NW)) void span_state_kernel(const uint16_t* __restrict__ k,
                                                         const uint16_t* __restrict__ v,
                                                         uint16_t* __restrict__ spanst,
                                                         int T, int L, int NS, int BH,
                                                         int sp0, int nsp) {
  using G = GeoG<D, DV, NG>;
  using SG = StateGrid<D, DV, NG>;
  constexpr int UW = SG::UW;
  constexpr int NW = SG::NW;
  constexpr int NTH = 64 * NW;  // threads per workgroup
  constexpr int DM = G::DM;
  constexpr int NXR = DM / 32;  // distinct x rows per lane (x depends on tile % NXR)
  static_assert(G::MT == 2, "the slot loop issues the two dv tiles of a slot tile together");
  constexpr int KS = kTB2 / 16;                      // K-steps per staged block
  // Key row r of a K buffer starts at krow(r) (fp16 elements).  The slot tiles
  // read rows r and r + DM/2 of a feature block in the same 16-lane phase of a
  // ds_read_b128; a gap of kGapK2 halves (32 banks) after every DM/2 rows moves
  // alternate half-blocks to the other half of the banks.
  constexpr int KBUFE = D * kRow2 + (2 * NG - 1) * kGapK2;  // halves of one K buffer
  constexpr unsigned KBUF = KBUFE * 2;               // bytes of one K buffer
  constexpr unsigned VBUF = DV * kRow2 * 2;          // bytes of one V buffer
  auto krow = [](int r) { return r * kRow2 + (r / (DM / 2)) * kGapK2; };
  // K and V buffers in one array: the record epilogue reuses it as a whole
  constexpr int POOL = kNBuf2 * KBUFE + kNBuf2 * DV * kRow2;
  __shared__ __attribute__((aligned(16))) uint16_t pool[POOL];
  auto& kT = *reinterpret_cast<uint16_t(*)[kNBuf2][KBUFE]>(&pool[0]);
  auto& vT = *reinterpret_cast<uint16_t(*)[kNBuf2][DV][kRow2]>(&pool[kNBuf2 * KBUFE]);
  __shared__ uint32_t red[4];  // K and V magnitude maxima, non-finite flag
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int c = lane & 31, g = lane >> 5;
  const int id = blockIdx.x;
  const int jx = id >> 3;
  const int part = jx % SG::NB;
  // Work item li over the NS - 1 spans per head that enter a prefix (each
  // head's last span is left out), head by head.  All of these spans carry the same work, so the XCD a work item
  // lands on (work item mod 8) needs no balancing.
  const int li = sp0 + 8 * (jx / SG::NB) + (id & 7);
  if (li >= nsp) return;  // whole workgroup: padding of the grid
  const int s = li % (NS - 1), bh = li / (NS - 1);
  const int sp = bh * NS + s;  // span record index
  const int gw = part * NW + wave;  // wave index inside the span
  const long long span0 = static_cast<long long>(s) * L;
  const long long span_end = min(static_cast<long long>(T), span0 + L);
  const uint16_t* kh = k + static_cast<long long>(bh) * T * D;
  const uint16_t* vh = v + static_cast<long long>(bh) * T * DV;
  uint16_t* rec = spanst + static_cast<long long>(sp) * G::E;
  const int nblk = static_cast<int>((span_end - span0 + kTB2 - 1) / kTB2);

  // staging: task -> (pair p of tokens, 8-wide column group cg); K then V
  constexpr int KG = D / 8, VG = DV / 8;
  constexpr int NPAIR = kTB2 / 2;
  constexpr int NTASK = NPAIR * (KG + VG);
  static_assert(NTASK % NTH == 0 && NPAIR == 64, "staging: one token pair per lane");
  constexpr int TPT = NTASK / NTH;
  uint4 st_lo[TPT], st_hi[TPT];
  // Fetch / commit the staging tasks [i0, i1) of this thread for the block
  // starting at token t0.  The loads are unconditional (token index clamped
  // into the sequence) so that the number of loads in flight is the same on
  // every path and waits can count them; tokens at or past the span end are
  // zeroed by the byte selectors of the commit's permutes.
  auto fetch = [&](long long t0, auto i0_c, auto i1_c) __attribute__((always_inline)) {
#pragma unroll
    for (int i = decltype(i0_c)::value; i < decltype(i1_c)::value; ++i) {
      const int cg = wave + NW * i, p = lane;  // wave-uniform column group
      const long long ta = min(t0 + 2 * p, static_cast<long long>(T) - 1);
      const long long tb = min(t0 + 2 * p + 1, static_cast<long long>(T) - 1);
      if (cg < KG) {
        st_lo[i] = *reinterpret_cast<const uint4*>(kh + ta * D + 8 * cg);
        st_hi[i] = *reinterpret_cast<const uint4*>(kh + tb * D + 8 * cg);
      } else {
        const int vg = cg - KG;
        st_lo[i] = *reinterpret_cast<const uint4*>(vh + ta * DV + 8 * vg);
        st_hi[i] = *reinterpret_cast<const uint4*>(vh + tb * DV + 8 * vg);
      }
    }
  };
  // Commit: write the fetched pairs into LDS as fp16 (times the span's scale
  // when SC).
  auto commit = [&](auto sc_c, int buf, long long t0, float sk, float sv,
                    auto i0_c, auto i1_c) __attribute__((always_inline)) {
    constexpr bool SC = decltype(sc_c)::value;
#pragma unroll
    for (int i = decltype(i0_c)::value; i < decltype(i1_c)::value; ++i) {
      const int cg = wave + NW * i, p = lane;
      const bool va = t0 + 2 * p < span_end, vb = t0 + 2 * p + 1 < span_end;
      const uint32_t a[4] = {st_lo[i].x, st_lo[i].y, st_lo[i].z, st_lo[i].w};
      const uint32_t b[4] = {st_hi[i].x, st_hi[i].y, st_hi[i].z, st_hi[i].w};
      // v_perm byte selectors: 0-3 pick bytes of the second operand, 4-7 of
      // the first, 0x0c gives a zero byte; tokens at or past the span end
      // become zeros.  lo / hi: the low / high bf16 of a word as an fp32
      // bit pattern.
      const uint32_t lo_a = va ? 0x01000c0cu : 0x0c0c0c0cu, hi_a = va ? 0x03020c0cu : 0x0c0c0c0cu;
      const uint32_t lo_b = vb ? 0x01000c0cu : 0x0c0c0c0cu, hi_b = vb ? 0x03020c0cu : 0x0c0c0c0cu;
      const float scale = (cg < KG) ? sk : sv;
      uint16_t* base = (cg < KG) ? &kT[buf][krow(8 * cg) + 2 * p]
                                 : &vT[buf][8 * (cg - KG)][2 * p];
      // rows 8cg .. 8cg+7 of a K buffer lie between two gaps (DM/2 is a
      // multiple of 8), as do all rows of a V buffer
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        float xl = __uint_as_float(__builtin_amdgcn_perm(0u, a[e], lo_a));
        float yl = __uint_as_float(__builtin_amdgcn_perm(0u, b[e], lo_b));
        float xh = __uint_as_float(__builtin_amdgcn_perm(0u, a[e], hi_a));
        float yh = __uint_as_float(__builtin_amdgcn_perm(0u, b[e], hi_b));
        if constexpr (SC) {
          xl *= scale;
          yl *= scale;
          xh *= scale;
          yh *= scale;
        }
        // the conversions are exact in fp16's range (round-toward-zero only
        // below it)
        *reinterpret_cast<uint32_t*>(base + (2 * e) * kRow2) =
            __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_pkrtz(xl, yl));
        *reinterpret_cast<uint32_t*>(base + (2 * e + 1) * kRow2) =
            __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_pkrtz(xh, yh));
      }
    }
  };
  using I0 = std::integral_constant<int, 0>;
  using IT = std::integral_constant<int, TPT>;
  using Yes = std::true_type;
  using No = std::false_type;
  static_assert(TPT <= KS, "one staging piece per K-step at most");
  const char* kbase = reinterpret_cast<const char*>(&kT[0][0]);  // fp16 K buffers
  const char* vbase = reinterpret_cast<const char*>(&vT[0][0][0]);

  // ---- scales of the span --------------------------------------------------
  if (tid < 4) red[tid] = 0u;
  fetch(span0, I0{}, IT{});  // block 0, kept in the staging registers
  uint32_t mk = 0u, mv = 0u;
#pragma unroll
  for (int i = 0; i < TPT; ++i) {
    if (wave + NW * i < KG) {
      mk = absmax_bits(absmax_bits(mk, st_lo[i]), st_hi[i]);
    } else {
      mv = absmax_bits(absmax_bits(mv, st_lo[i]), st_hi[i]);
    }
  }
  mk = wave_max_u32(mk);
  mv = wave_max_u32(mv);
  __syncthreads();
  if (lane == 0) {
    atomicMax(&red[0], mk);
    atomicMax(&red[1], mv);
  }
  __syncthreads();
  // bf16 exponent fields of the largest |k|, |v| of block 0 (255: inf / NaN)
  int ek = static_cast<int>(red[0] >> 7), ev = static_cast<int>(red[1] >> 7);
  const bool nonfinite_in = ek >= 255 || ev >= 255;
  bool scaled = !nonfinite_in && !(ek >= 127 - 4 && ek < 127 + 4 && ev >= 127 - 8 && ev < 127 + 8);
  // Exact maxima of the whole span (read once more; only for spans outside
  // the unscaled range) -> exponents of the scales.
  auto span_scales = [&]() __attribute__((always_inline)) {
    uint32_t m2k = 0u, m2v = 0u;
    const long long n16 = (span_end - span0) * ((D + DV) / 8);  // 16-byte pieces
    for (long long j = tid; j < n16; j += NTH) {
      const long long t = span0 + j / ((D + DV) / 8);
      const int pc = static_cast<int>(j % ((D + DV) / 8));
      if (pc < KG) m2k = absmax_bits(m2k, *reinterpret_cast<const uint4*>(kh + t * D + 8 * pc));
      else m2v = absmax_bits(m2v, *reinterpret_cast<const uint4*>(vh + t * DV + 8 * (pc - KG)));
    }
    m2k = wave_max_u32(m2k);
    m2v = wave_max_u32(m2v);
    __syncthreads();
    if (tid < 2) red[tid] = 0u;
    __syncthreads();
    if (lane == 0) {
      atomicMax(&red[0], m2k);
      atomicMax(&red[1], m2v);
    }
    __syncthreads();
    ek = static_cast<int>(red[0] >> 7);
    ev = static_cast<int>(red[1] >> 7);
    fetch(span0, I0{}, IT{});  // block 0 again, for the scaled pass
  };
  if (scaled) span_scales();

  // ---- the span's passes ------------------------------------------------------
  // Three-deep ring: block bi is read from buffer bi % 3 while block bi+1 is
  // published into the next buffer piece by piece (staging task j of each
  // thread), and each piece's registers are refilled with block bi+2 right
  // away, so a global load has a whole block of compute to arrive.
  // Every block issues the same loads whether or not their data is used
  // (past the span's last block they re-read clamped, valid addresses), so the
  // count of loads in flight is the same on every path.
  // (straight-line code, at most one unscaled and one scaled pass: a loop
  // around the passes would keep every register of a pass live across it)
  float fin = 0.f;  // sum of the written state: non-finite iff some value is
  auto run = [&](auto sc_c) __attribute__((always_inline)) {
      constexpr bool SC = decltype(sc_c)::value;
      // scales: 2^-e maps the largest |k| (|v|) of the span into [1, 2)
      const int xk = SC ? max(ek, 1) - 127 : 0, xv = SC ? max(ev, 1) - 127 : 0;
      const float sk = ldexpf(1.f, -xk), sv = ldexpf(1.f, -xv);
      commit(sc_c, 0, span0, sk, sv, I0{}, IT{});
      fetch(span0 + kTB2, I0{}, IT{});
      lds_barrier();

      if (gw >= SG::NUW) {
        // ---- Z = K^T K over the span (wave NUW) ---------------------------------
        const bool zwave = gw == SG::NUW;
        // Z_blk = K_blk^T K_blk for each feature block: the diagonal ZMB x ZMB
        // tile blocks of K^T K
        constexpr int ZT = D / 32;  // 32-row tiles of K
        f32x16 zacc[NG][G::ZMB][G::ZMB];
#pragma unroll
        for (int bb = 0; bb < NG; ++bb)
#pragma unroll
          for (int a = 0; a < G::ZMB; ++a)
#pragma unroll
            for (int b = 0; b < G::ZMB; ++b)
#pragma unroll
              for (int r = 0; r < 16; ++r) zacc[bb][a][b][r] = 0.f;
        for (int bi = 0; bi < nblk; ++bi) {
          const int buf = bi % kNBuf2;
          if (bi + 1 < nblk)
            commit(sc_c, (bi + 1) % kNBuf2, span0 + static_cast<long long>(bi + 1) * kTB2, sk,
                   sv, I0{}, IT{});
          fetch(span0 + static_cast<long long>(bi + 2) * kTB2, I0{}, IT{});
          if (zwave) {
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) {
              f16x8 A[ZT];
#pragma unroll
              for (int a = 0; a < ZT; ++a)
                A[a] = *reinterpret_cast<const f16x8*>(&kT[buf][krow(32 * a + c) + 16 * ks + 8 * g]);
#pragma unroll
              for (int bb = 0; bb < NG; ++bb)
#pragma unroll
                for (int a = 0; a < G::ZMB; ++a)
#pragma unroll
                  for (int b = 0; b < G::ZMB; ++b)
                    zacc[bb][a][b] = __builtin_amdgcn_mfma_f32_32x32x16_f16(
                        A[bb * G::ZMB + a], A[bb * G::ZMB + b], zacc[bb][a][b], 0, 0, 0);
            }
          }
          lds_barrier();
        }
        if (zwave) {
#pragma unroll
          for (int bb = 0; bb < NG; ++bb)
#pragma unroll
            for (int za = 0; za < G::ZMB; ++za)
#pragma unroll
              for (int zb = 0; zb < G::ZMB; ++zb)
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                  const int a = 32 * za + 8 * (r >> 2) + 4 * g + (r & 3);  // inside the block
                  const int b = 32 * zb + c;
                  float x = zacc[bb][za][zb][r];
                  if constexpr (decltype(sc_c)::value) x = ldexpf(x, 2 * xk);
                  fin += x;
                  __bf16 h = static_cast<__bf16>(x);
                  rec[G::ES + static_cast<long long>(bb) * DM * DM + zop_index<DM>(a, b)] =
                      __builtin_bit_cast(uint16_t, h);
                }
        }
        return;
      }

      // ---- S_span^T = V^T Phi(K) for this wave's slot tiles --------------------
      // slot wave gw covers tiles [unit0, unit0 + UW) of feature block blk
      // (tiles past the block's last one are computed on a valid row and not
      // stored)
      const int blk = gw / SG::NUWB;
      const int unit0 = (gw % SG::NUWB) * UW;
      // per-lane byte offsets of the fragments inside buffer 0, column 8*g
      unsigned xo[NXR], yo[UW], vo[G::MT];
      // fx[p] serves the local tiles u with u % NXR == p, whose x row is that
      // of global tile parity (unit0 + p) % NXR
#pragma unroll
      for (int p = 0; p < NXR; ++p) {
        int xr, yy;
        slot_pair<DM>(32 * ((unit0 + p) % NXR) + c, xr, yy);
        xo[p] = static_cast<unsigned>((krow(DM * blk + xr) + 8 * g) * 2);
      }
#pragma unroll
      for (int u = 0; u < UW; ++u) {
        int xx, yr;
        const int unit = unit0 + u < G::NSTM ? unit0 + u : G::NSTM - 1;  // valid row; no store
        slot_pair<DM>(32 * unit + c, xx, yr);
        yo[u] = static_cast<unsigned>((krow(DM * blk + yr) + 8 * g) * 2);
      }
#pragma unroll
      for (int m = 0; m < G::MT; ++m)
        vo[m] = static_cast<unsigned>(((32 * m + c) * kRow2 + 8 * g) * 2);

      // Accumulators fed by compiler-builtin MFMAs: the compiler places them
      // and inserts the wait states.
      f32x16 acc[UW][G::MT];
#pragma unroll
      for (int u = 0; u < UW; ++u)
#pragma unroll
        for (int m = 0; m < G::MT; ++m)
#pragma unroll
          for (int r = 0; r < 16; ++r) acc[u][m][r] = 0.f;
      auto mf = [](f32x16& a, const f16x8& x, const f16x8& y) __attribute__((always_inline)) {
        a = __builtin_amdgcn_mfma_f32_32x32x16_f16(x, y, a, 0, 0, 0);
      };

      // LDS fragments: the y rows of the slot tiles (8 fp16 tokens each,
      // reloaded for the next K-step as soon as the features they feed are
      // computed), the x rows (reloaded for the next K-step after their last
      // use in this one) and V^T double buffered by K-step parity.
      f16x8 fy[UW], fx[NXR], fv[2][G::MT];
      auto ld16 = [](const char* p) __attribute__((always_inline)) {
        return *reinterpret_cast<const f16x8*>(p);
      };
      auto ldv = [&](int set, const char* vb, unsigned ko) __attribute__((always_inline)) {
#pragma unroll
        for (int m = 0; m < G::MT; ++m) fv[set][m] = ld16(vb + vo[m] + ko);
      };
      // tile u of a K-step computes the features of tile u+1, whose x row has
      // parity (u+1) % NXR; the x row of parity p is reloaded for the next
      // K-step after xlast(p), the last tile of this K-step that uses it
      auto xlast = [](int p) {
        int last = -1;
        for (int u = 0; u + 1 < UW; ++u)
          if ((u + 1) % NXR == p) last = u;
        return last;
      };
      // Per staged block: publish block bi+1 and fetch block bi+2 piece by
      // piece; the features of tile u+1 are computed between the two MFMAs of
      // tile u (the block's first tile beforehand).
      for (int bi = 0; bi < nblk; ++bi) {
        const int buf = bi % kNBuf2;
        const int nbuf = (bi + 1) % kNBuf2;
        const char* kb = kbase + buf * KBUF;
        const char* vb = vbase + buf * VBUF;
        const bool more1 = bi + 1 < nblk;
        const long long t1 = span0 + static_cast<long long>(bi + 1) * kTB2;
        const long long t2 = t1 + kTB2;
        ldv(0, vb, 0u);
#pragma unroll
        for (int p = 0; p < NXR; ++p) fx[p] = ld16(kb + xo[p]);
#pragma unroll
        for (int u = 0; u < UW; ++u) fy[u] = ld16(kb + yo[u]);
        // B fragments: bq[0] the next tile's, bq[1], bq[2] the two before
        // (kept live so that a new fragment never reuses the registers of an
        // MFMA that may still be running, see hold)
        f16x8 bq[3];
        bq[0] = fx[0] * fy[0];
        bq[1] = bq[0];
        bq[2] = bq[0];
        auto push = [&](const f16x8& nb) __attribute__((always_inline)) {
          bq[2] = bq[1];
          bq[1] = bq[0];
          bq[0] = nb;
          hold(bq[1], bq[2]);
        };
        static_for<0, KS>([&](auto ks_c) {
          constexpr int ks = decltype(ks_c)::value;
          constexpr int cur = ks & 1;
          constexpr unsigned kn = 32u * (ks + 1);  // byte column of K-step ks+1 (16 fp16)
          static_for<0, TPT>([&](auto j_c) {  // staging piece j at K-step j*KS/TPT
            constexpr int j = decltype(j_c)::value;
            if constexpr (j * KS / TPT == ks) {
              using J = std::integral_constant<int, j>;
              using J1 = std::integral_constant<int, j + 1>;
              if (more1) commit(sc_c, nbuf, t1, sk, sv, J{}, J1{});
              fetch(t2, J{}, J1{});
            }
          });
          const f16x8 va0 = fv[cur][0];
          const f16x8 va1 = fv[cur][1];
          static_for<0, UW>([&](auto u_c) {
            constexpr int u = decltype(u_c)::value;
            // fy[u] fed the features of (ks, u): reload it for (ks+1, u)
            if constexpr (ks + 1 < KS && u > 0) fy[u] = ld16(kb + yo[u] + kn);
            if constexpr (u + 1 < UW || ks + 1 < KS) {
              // the next tile's features (tile u+1 of this K-step, or tile 0
              // of the next one) between the tile's two MFMAs
              constexpr int un = (u + 1 < UW) ? u + 1 : 0;
              mf(acc[u][0], va0, bq[0]);
              __builtin_amdgcn_sched_barrier(0);
              const f16x8 nb = fx[un % NXR] * fy[un];
              __builtin_amdgcn_sched_barrier(0);
              mf(acc[u][1], va1, bq[0]);
              __builtin_amdgcn_sched_barrier(0);
              push(nb);
            } else {
              // the block's last tile: its features are one instruction old
              mf(acc[u][0], va0, bq[0]);
              mf(acc[u][1], va1, bq[0]);
            }
            if constexpr (u + 1 < UW && ks + 1 < KS) {
              if constexpr (u == 0) fy[0] = ld16(kb + yo[0] + kn);
              // V^T of K-step ks+1 into the other buffer, whose last readers
              // (the previous K-step's final tile) are two tiles old now
              if constexpr (u == 1) ldv(cur ^ 1, vb, kn);
#pragma unroll
              for (int p = 0; p < NXR; ++p)
                if (u == xlast(p)) fx[p] = ld16(kb + xo[p] + kn);
            }
          });
        });
        lds_barrier();
      }

      // Write this wave's tiles of the span record (bf16), undoing the scales.
      // The accumulators hold 4 consecutive dv rows of one slot per lane; they
      // go through LDS (this wave's own region of the free staging buffers,
      // [dv][HU*32 + 8] bf16, HU tiles at a time) so that the record is
      // written in 16-byte pieces of 8 consecutive slots.
      constexpr int HU = (UW + 1) / 2;  // tiles per round (the second may have fewer)
      constexpr int RS = HU * 32 + 8;   // bf16 per LDS row (16-byte aligned rows)
      static_assert(NW * DV * RS <= POOL, "record rounds fit the staging LDS");
      uint16_t* ep = &pool[wave * DV * RS];
      constexpr int CPR = HU * 4;  // 16-byte pieces per row and round
      static_for<0, 2>([&](auto h_c) {
        constexpr int h = decltype(h_c)::value;
        constexpr int NU = (h == 0) ? HU : UW - HU;  // tiles of this round
#pragma unroll
        for (int uu = 0; uu < NU; ++uu) {
          const int u = h * HU + uu;
#pragma unroll
          for (int m = 0; m < G::MT; ++m)
#pragma unroll
            for (int r = 0; r < 16; r += 2) {
              const int dvrow = 32 * m + 8 * (r >> 2) + 4 * g + (r & 3);
              float x0 = acc[u][m][r], x1 = acc[u][m][r + 1];
              if constexpr (decltype(sc_c)::value) {
                x0 = ldexpf(x0, 2 * xk + xv);
                x1 = ldexpf(x1, 2 * xk + xv);
              }
              if (unit0 + u < G::NSTM) fin += x0 + x1;
              const uint32_t w = pack_bf16x2(x0, x1);  // rows dvrow, dvrow + 1
              ep[dvrow * RS + 32 * uu + c] = static_cast<uint16_t>(w);
              ep[(dvrow + 1) * RS + 32 * uu + c] = static_cast<uint16_t>(w >> 16);
            }
        }
        __builtin_amdgcn_s_waitcnt(0xC07F);  // this wave's LDS writes are done
        __builtin_amdgcn_wave_barrier();
#pragma unroll
        for (int i = 0; i < DV * CPR / 64; ++i) {
          const int kc = lane + 64 * i;
          const int row = kc / CPR, pc = kc % CPR;
          const uint4 w = *reinterpret_cast<const uint4*>(ep + row * RS + 8 * pc);
          if (pc / 4 < NU && unit0 + h * HU + pc / 4 < G::NSTM)
            *reinterpret_cast<uint4*>(rec + static_cast<long long>(row) * G::NSLOT +
                                      32 * (blk * G::NSTM + unit0 + h * HU) + 8 * pc) = w;
        }
        __builtin_amdgcn_s_waitcnt(0xC07F);  // reads done before the next round's writes
        __builtin_amdgcn_wave_barrier();
      });
  };
  if (!scaled) {
    run(No{});
    // A non-finite state from finite inputs means an fp16 overflow in the
    // unscaled pass: run the span again with its scales.
    if (!nonfinite_in) {
      const bool bad = !(fabsf(fin) <= 3.0e38f);
      __syncthreads();
      if (bad) red[2] = 1u;
      __syncthreads();
      if (red[2] != 0u) {
        scaled = true;
        span_scales();
        run(Yes{});
      }
    }
  } else {
    run(Yes{});
  }
}

// ---------------------------------------------------------------------------
// Quadratic form (and the stage buffers of K4).  quadratic_kernel: 1-D grid
// of workgroups of 256 threads (4 waves), one per CU (LDS: the five 32 KB
// stage buffers, of which it uses three).  A head (one span covering the
// sequence) has QB = T/256 query blocks; block id -> (head, query block)
// keeps the query blocks of a head on one XCD (equal id % 8) so they share
// its keys in that XCD's L2.  The workgroup owns 8 query tiles of 32; wave w
// takes tiles {w, 7-w}, which balances the causal work.  Operands are staged
// by direct global -> LDS copies, three stages deep, so no registers hold
// staged data and the copies of stage s+2 overlap the arithmetic of stage s.
// LDS fragment reads use per-lane offsets computed once, so every read is a
// base register plus an immediate.
// pre[bh][s][E] bf16 (K4): weighted S_pre^T as [dv][NSLOT], then Z_pre
// (operand order).  K4 stages K and V rows as they are in HBM; the quadratic
// form reads vtp[bh][dv][LA] bf16, a permuted V^T (vt_permute_kernel).
// ---------------------------------------------------------------------------
constexpr int kKB = 128;        // keys per intra stage (four 32-key blocks)
constexpr int kKC = 16;         // readout K-steps per stage
constexpr int kStageBytes = 32768;

__shared__ __attribute__((aligned(16))) uint16_t g_stage0[kStageBytes / 2];
__shared__ __attribute__((aligned(16))) uint16_t g_stage1[kStageBytes / 2];
__shared__ __attribute__((aligned(16))) uint16_t g_stage2[kStageBytes / 2];
__shared__ __attribute__((aligned(16))) uint16_t g_stage3[kStageBytes / 2];
__shared__ __attribute__((aligned(16))) uint16_t g_stage4[kStageBytes / 2];

// Stage buffers 0-2 serve the intra-span stages; the readout's stage s uses
// buffer (3 + s) % 5, so its first two stages (buffers 3 and 4) can be copied
// in at the start of the kernel while the other phases run.
__device__ __forceinline__ uint16_t* stage_buf(int j) {
  return j == 0 ? g_stage0
                : (j == 1 ? g_stage1 : (j == 2 ? g_stage2 : (j == 3 ? g_stage3 : g_stage4)));
}

// Transposing LDS read of 16-bit elements (gfx950 ds_read_b64_tr_b16): in each
// group of 16 lanes, lane j receives in slot s = 0..3 element j % 4 of the
// 8-byte piece addressed by lane 4 s + j / 4 of its group.
typedef short i16x4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ uint2 lds_tr16(const void* p) {
  const i16x4 r = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (__attribute__((address_space(3))) i16x4*)(const_cast<void*>(p)));
  return __builtin_bit_cast(uint2, r);
}


// Scores of two query tiles against one 32-key block: sc_i = K_blk Q_i^T
// over the d-contraction, the two accumulation chains interleaved (compiler
// builtins; the compiler inserts the wait states before the VALU reads them).
template <int KZ>
__device__ __forceinline__ void score2(f32x16& sc0, f32x16& sc1, const bf16x8 (&A)[KZ],
                                       const bf16x8 (&q0)[KZ], const bf16x8 (&q1)[KZ]) {
  mfma_vz(sc0, A[0], q0[0]);
  mfma_vz(sc1, A[0], q1[0]);
#pragma unroll
  for (int kz = 1; kz < KZ; ++kz) {
    mfma_v(sc0, A[kz], q0[kz]);
    mfma_v(sc1, A[kz], q1[kz]);
  }
}

// Scores of two query tiles against one 32-key block with two feature blocks
// of 32 coordinates (K-steps 0, 1 of block 0 and 2, 3 of block 1): four
// chains, interleaved.
__device__ __forceinline__ void score2b2(f32x16& s00, f32x16& s01, f32x16& s10, f32x16& s11,
                                         const bf16x8 (&A)[4], const bf16x8 (&q0)[4],
                                         const bf16x8 (&q1)[4]) {
  mfma_vz(s00, A[0], q0[0]);
  mfma_vz(s10, A[0], q1[0]);
  mfma_vz(s01, A[2], q0[2]);
  mfma_vz(s11, A[2], q1[2]);
  mfma_v(s00, A[1], q0[1]);
  mfma_v(s10, A[1], q1[1]);
  mfma_v(s01, A[3], q0[3]);
  mfma_v(s11, A[3], q1[3]);
}

template <int D, int DV>
struct OutGrid {
  static constexpr int QB_TOKENS = 256;  // queries per workgroup
};

template <int D, int DV, int NG>
__global__ __launch_bounds__(256) void quadratic_kernel(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ k,
    const uint16_t* __restrict__ vtp, float* __restrict__ out, int T, int L, int LV, int NS,
    int QB, int sp0, int nsp) {
  using G = GeoG<D, DV, NG>;
  constexpr int DM = G::DM, RM = G::RM, KZM = G::KZM;
  constexpr int NQ = 2, W = 4, NT = 8;
  constexpr int KCH = D / 8;                    // 16-byte chunks per key row
  constexpr int KCHUNKS = kKB * KCH;            // K rows of one intra stage
  constexpr int VCH = kKB / 8;                  // chunks per V^T row of one stage (16)
  constexpr int VCHUNKS = DV * VCH;
  constexpr int ICH = KCHUNKS + VCHUNKS;        // chunks per intra stage
  static_assert(ICH * 16 <= kStageBytes && KCHUNKS % 256 == 0 && VCHUNKS % 256 == 0,
                "intra stage size");
  constexpr int IPW_K = KCHUNKS / 256;          // copy instructions per wave: K rows
  constexpr int IPW_I = ICH / 256;              // ... K rows then V^T rows
  static_assert(G::MT == 2, "two dv tiles");

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int c = lane & 31, g = lane >> 5;
  const int id = blockIdx.x;
  const int jx = id >> 3;
  // query blocks differ in work by up to a factor QB: the longest go first
  const int qb = QB - 1 - jx % QB;
  const int sp = sp0 + 8 * (jx / QB) + (id & 7);
  if (sp >= nsp) return;  // whole workgroup: padding of the grid
  const int s = sp % NS, bh = sp / NS;
  const long long span0 = static_cast<long long>(s) * L;
  const long long span_end = min(static_cast<long long>(T), span0 + L);
  const long long wg_q0 = span0 + static_cast<long long>(qb) * NT * 32;
  if (wg_q0 >= span_end) return;  // whole workgroup beyond the sequence
  const uint16_t* qh = q + static_cast<long long>(bh) * T * D;
  const uint16_t* kh = k + static_cast<long long>(bh) * T * D;
  const uint16_t* vt_rec = vtp + static_cast<long long>(sp) * DV * LV;

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

  // ---- staging copies of both phases ------------------------------------------
  // Stages cover the key blocks of the workgroup's last live tile; every
  // wave runs all of them (the stage barriers are workgroup-wide).
  int last_tile = qb * NT + NT - 1;
  const int last_key_tile = static_cast<int>((span_end - 1 - span0) / 32);
  if (last_tile > last_key_tile) last_tile = last_key_tile;
  const int nstage = (last_tile + 1 + 3) / 4;  // 128-key intra stages
  // intra copy i of this lane: K row / V^T row and the chunk it fetches
  int ksrc[IPW_K];  // element offset of the K chunk from the stage's first key row
  int vsrc[IPW_I - IPW_K];
#pragma unroll
  for (int i = 0; i < IPW_I; ++i) {
    const int P = (i * W + wave) * 64 + lane;  // LDS chunk written by this lane
    if (i < IPW_K) {
      const int r = P / KCH, pos = P % KCH;
      ksrc[i] = r * D + 8 * (pos ^ kswz<D>(r));
    } else {
      const int P2 = P - KCHUNKS;
      const int m = P2 / VCH, pos = P2 % VCH;
      vsrc[i - IPW_K] = m * LV + 8 * (pos ^ rswz(m));
    }
  }
  auto issue_i = [&](int st, uint16_t* buf) __attribute__((always_inline)) {
    const long long key0 = span0 + static_cast<long long>(st) * kKB;
#pragma unroll
    for (int i = 0; i < IPW_I; ++i) {
      const void* src;
      if (i < IPW_K) {
        // keys past the sequence: re-read the last row (never used)
        const long long over = key0 + ksrc[i] / D - (T - 1);
        src = kh + key0 * D + ksrc[i] - (over > 0 ? over * D : 0);
      } else {
        src = vt_rec + st * kKB + vsrc[i - IPW_K];
      }
      g2lds16(src, buf + (i * W + wave) * 512);
    }
  };
  // Stage 0 is issued first and the query fragments are loaded behind it;
  // the workgroup waits for that one memory round trip (the compiler's wait
  // before the empty asm below: loads complete in order, so it also covers
  // the copies issued before them), and only then issues stage 1, which
  // arrives under the first stage's work.  From here on the only vector
  // memory operations in flight are copies (and the final stores), which the
  // pipeline's own waits count.
  issue_i(0, g_stage0);

  // bf16 query fragments for the d-contractions, per feature block:
  // qf[i][KZM*bb + kz] holds q[t][DM*bb + 8*kz + RM*g .. +7] of this lane's
  // query t = tq0 + c (with one block: q[t][8*kz + R*g ..]).
  bf16x8 qf[NQ][G::KZ];
#pragma unroll
  for (int i = 0; i < NQ; ++i) {
    const long long t = min(tq0[i] + c, static_cast<long long>(T) - 1);
#pragma unroll
    for (int kz = 0; kz < G::KZ; ++kz)
      qf[i][kz] = *reinterpret_cast<const bf16x8*>(qh + t * D + DM * (kz / KZM) +
                                                   8 * (kz % KZM) + RM * g);
  }

#pragma unroll
  for (int i = 0; i < NQ; ++i)
#pragma unroll
    for (int kz = 0; kz < G::KZ; ++kz) asm volatile("" ::"v"(qf[i][kz]));
  if (nstage > 1) issue_i(1, g_stage1);

  // the P V accumulators
  f32x16 acc[G::MT][NQ];
#pragma unroll
  for (int m = 0; m < G::MT; ++m)
#pragma unroll
    for (int i = 0; i < NQ; ++i)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[m][i][r] = 0.f;
  float dpart[NQ];  // the denominators' row sums
#pragma unroll
  for (int i = 0; i < NQ; ++i) dpart[i] = 0.f;

  // ---- causal squared-score attention inside the span -----------------------
  // Per 32-key block kb and query tile i: S_i = K_kb Q_i^T (a chain of KZ
  // MFMAs into VGPRs), P_i = S_i^2 masked above the diagonal on the tile's
  // diagonal block (VALU, with the row sums for the denominator), and
  // O_i += V_kb^T P_i (four MFMAs: two dv halves x two 16-key halves).  The
  // wave's two tiles run half a block apart, so every VALU step has MFMAs of
  // the other tile to issue between:
  //   group A of block kb: S_0(kb) and P V of tile 0 at kb-1; P_1(kb-1)
  //   group B of block kb: S_1(kb) and P V of tile 1 at kb-1; P_0(kb)
  // A wave issues in order and an MFMA holds the matrix pipe for 32 cycles;
  // each group alternates its two MFMA chains (never two dependent MFMAs in a
  // row) and places a quarter of the P work after each MFMA (scheduling
  // barriers keep that order).  A tile whose diagonal block is past, or that
  // lies beyond the sequence, gets zero P fragments: its MFMAs still run, so
  // no branch surrounds an accumulator.
  {
    // fragment byte offsets inside a stage buffer
    //  K rows 32*sb + c, chunk (DM/8)*bb + kz' + (RM/8)*g of fragment KZM*bb + kz'
    //  (the layout of qf), ^ kswz: depends on sb only through sb & 1
    unsigned kfo[2][G::KZ];
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int kz = 0; kz < G::KZ; ++kz) {
        const int krow = 32 * h + c;
        const int chunk = (DM / 8) * (kz / KZM) + (kz % KZM) + (RM / 8) * g;
        kfo[h][kz] = static_cast<unsigned>((krow * KCH + (chunk ^ kswz<D>(krow))) * 16);
      }
    //  V^T rows 32*m + c, chunk (4*sb + 2*kv + g) ^ (c & 15); the row part of m is immediate
    unsigned vfo[4][2];
#pragma unroll
    for (int sb = 0; sb < 4; ++sb)
#pragma unroll
      for (int kv = 0; kv < 2; ++kv)
        vfo[sb][kv] = static_cast<unsigned>(
            (KCHUNKS + c * VCH + ((4 * sb + 2 * kv + g) ^ rswz(c))) * 16);

    // a tile's diagonal block, -1 for a tile beyond the sequence (wave-uniform)
    int tdiag[NQ];
#pragma unroll
    for (int i = 0; i < NQ; ++i) tdiag[i] = __builtin_amdgcn_readfirstlane(tlive[i] ? tile[i] : -1);
    // Fragment loads of block kb at stage position sb (known at compile time)
    // from its stage buffer; one 16-byte read per call, so that the callers
    // can spread them over the MFMA slots of a group.
    auto ldA1 = [&](const char* buf, auto sb_c, int kz, bf16x8& dst) __attribute__((always_inline)) {
      constexpr int sb = decltype(sb_c)::value;
      dst = *reinterpret_cast<const bf16x8*>(buf + (sb >> 1) * (64 * KCH * 16) + kfo[sb & 1][kz]);
    };
    auto ldV1 = [&](const char* buf, auto sb_c, int m, int kv, bf16x8& dst)
                    __attribute__((always_inline)) {
      constexpr int sb = decltype(sb_c)::value;
      dst = *reinterpret_cast<const bf16x8*>(buf + vfo[sb][kv] + m * (32 * VCH * 16));
    };
    auto ldA = [&](const char* buf, auto sb_c, bf16x8 (&A)[G::KZ]) __attribute__((always_inline)) {
#pragma unroll
      for (int kz = 0; kz < G::KZ; ++kz) ldA1(buf, sb_c, kz, A[kz]);
    };
    auto ldV = [&](const char* buf, auto sb_c, bf16x8 (&va)[G::MT][2]) __attribute__((always_inline)) {
#pragma unroll
      for (int m = 0; m < G::MT; ++m)
#pragma unroll
        for (int kv = 0; kv < 2; ++kv) ldV1(buf, sb_c, m, kv, va[m][kv]);
    };
    // Score accumulators of one query tile: one per feature block; the weight
    // of a (query, key) pair is the sum over blocks of the squared scores.
    struct Sc {
      f32x16 b[NG];
    };
    auto p_of = [](const Sc& sc, int r) __attribute__((always_inline)) {
      float p = sc.b[0][r] * sc.b[0][r];
#pragma unroll
      for (int bb = 1; bb < NG; ++bb) p += sc.b[bb][r] * sc.b[bb][r];
      return p;
    };
    // P elements 2j and 2j+1 of a tile on a block before its diagonal, packed.
    // The empty asm statement consumes the results before the next asm (an
    // MFMA), so the compiler can neither sink the part below it nor merge it
    // into the fix-up that follows the group.
    auto ppart = [&](int j, const Sc& sc, float& dacc, uint32_t (&bw)[8])
                     __attribute__((always_inline)) {
      const float p0 = p_of(sc, 2 * j);
      const float p1 = p_of(sc, 2 * j + 1);
      dacc += p0 + p1;
      bw[j] = pack_bf16x2(p0, p1);
      asm volatile("" : "+v"(dacc), "+v"(bw[j]));
    };
    // on tile i's diagonal block (keys above the query masked) and past it
    // (zero; also a tile beyond the sequence) the tile's P of block kb is
    // redone after its group, VALU only; dsave is the row sum before the group
    auto fixup = [&](int kb, int i, const Sc& sc, float dsave, float& dacc, uint32_t (&bw)[8])
                     __attribute__((always_inline)) {
      if (__builtin_expect(kb < tdiag[i], 1)) return;  // nothing to redo (the common case)
      if (kb == tdiag[i]) {
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const int r0 = 2 * j, r1 = 2 * j + 1;
          const float p0 = (8 * (r0 >> 2) + 4 * g + (r0 & 3) > c) ? 0.f : p_of(sc, r0);
          const float p1 = (8 * (r1 >> 2) + 4 * g + (r1 & 3) > c) ? 0.f : p_of(sc, r1);
          dsave += p0 + p1;
          bw[j] = pack_bf16x2(p0, p1);
        }
        dacc = dsave;
      } else {
#pragma unroll
        for (int j = 0; j < 8; ++j) bw[j] = 0u;
        dacc = dsave;
      }
    };
    auto bfrag = [](const uint32_t (&bw)[8], int kv) __attribute__((always_inline)) {
      return __builtin_bit_cast(bf16x8, make_uint4(bw[4 * kv], bw[4 * kv + 1], bw[4 * kv + 2],
                                                   bw[4 * kv + 3]));
    };
    // one group: score chains into scs (if S), P V into (a0, a1) from fragments
    // vb and P words bv (if V), and the P words bw of the other tile from scp
    // (full mode; the caller fixes them up for the other modes); extra(i)
    // adds the caller's work (fragment loads) to slot i.  Score MFMA i is
    // K-step i / NG of block i % NG, so consecutive MFMAs of one chain are NG
    // slots apart.
    auto group = [&](auto s_c, auto v_c, Sc& scs, const bf16x8 (&Ab)[G::KZ],
                     const bf16x8 (&qs)[G::KZ], f32x16& a0, f32x16& a1,
                     const bf16x8 (&vb)[G::MT][2], const uint32_t (&bv)[8], Sc& scp,
                     float& dacc, uint32_t (&bw)[8], auto&& extra) __attribute__((always_inline)) {
      constexpr bool HS = decltype(s_c)::value, HV = decltype(v_c)::value;
      bf16x8 Bv[2];
      if constexpr (HV) {
        Bv[0] = bfrag(bv, 0);
        Bv[1] = bfrag(bv, 1);
      }
      static_for<0, 4>([&](auto i_c) {
        constexpr int i = decltype(i_c)::value;
        if constexpr (HS && i < G::KZ) {
          constexpr int bb = i % NG, kz = KZM * bb + i / NG;
          if constexpr (i / NG == 0) mfma_vz(scs.b[bb], Ab[kz], qs[kz]);
          else mfma_v(scs.b[bb], Ab[kz], qs[kz]);
        }
        // without a score chain the P V MFMA goes first, so that the VALU
        // reads scp two MFMA issues after the chain that wrote it
        if constexpr (!HS && HV) mfma_a((i & 1) ? a1 : a0, vb[i & 1][i >> 1], Bv[i >> 1]);
        // the scores become available to the VALU only after the first MFMA
        if constexpr (i == 0) {
#pragma unroll
          for (int bb = 0; bb < NG; ++bb) asm volatile("" : "+v"(scp.b[bb]));
        }
        __builtin_amdgcn_sched_barrier(0);
        ppart(2 * i, scp, dacc, bw);
        __builtin_amdgcn_sched_barrier(0);
        if constexpr (HS && HV) mfma_a((i & 1) ? a1 : a0, vb[i & 1][i >> 1], Bv[i >> 1]);
        __builtin_amdgcn_sched_barrier(0);
        ppart(2 * i + 1, scp, dacc, bw);
        extra(i_c);
        __builtin_amdgcn_sched_barrier(0);
      });
    };
    auto none = [](auto) {};
    using Yes = std::true_type;
    using No = std::false_type;
    using std::integral_constant;

    const int NB = 4 * nstage;  // 32-key blocks, all waves alike (stage barriers)
    bf16x8 A[2][G::KZ], va[2][G::MT][2];
    Sc sc[NQ];
    uint32_t bw[NQ][8];
    // stage buffers of stages st, st+1, st+2 (rotated once per stage)
    const char* b0 = reinterpret_cast<const char*>(g_stage0);
    const char* b1 = reinterpret_cast<const char*>(g_stage1);
    const char* b2 = reinterpret_cast<const char*>(g_stage2);
    // stage 0 (its copies were waited for with the query fragments)
    lds_barrier();
    if (nstage > 2) issue_i(2, g_stage2);
    ldA(b0, integral_constant<int, 0>{}, A[0]);
    ldA(b0, integral_constant<int, 1>{}, A[1]);
    ldV(b0, integral_constant<int, 0>{}, va[0]);
    // block 0: both score chains interleaved (no earlier block to finish),
    // then P_0(0); score2 leaves sc[0] readable by VALU
    if constexpr (NG == 1) score2<G::KZ>(sc[0].b[0], sc[1].b[0], A[0], qf[0], qf[1]);
    else score2b2(sc[0].b[0], sc[0].b[1], sc[1].b[0], sc[1].b[1], A[0], qf[0], qf[1]);
    {
      const float dsave = dpart[0];
#pragma unroll
      for (int j = 0; j < 8; ++j) ppart(j, sc[0], dpart[0], bw[0]);
      fixup(0, 0, sc[0], dsave, dpart[0], bw[0]);
    }
    // block kb >= 1 at stage position sb: A[sb & 1] holds A(kb) and V(kb) is
    // loaded into va[sb & 1]; P V of block kb-1 uses va[(sb & 1) ^ 1].  Inside
    // a stage the loads of V(kb) and A(kb+1) ride in group A's MFMA slots; the
    // last block of a stage loads up front, around the stage change.
    auto step = [&](auto sb_c, int kb) __attribute__((always_inline)) {
      constexpr int sb = decltype(sb_c)::value;
      constexpr int cur = sb & 1;
      auto loads = [&](auto i_c) __attribute__((always_inline)) {
        constexpr int i = decltype(i_c)::value;
        if constexpr (sb != 3) {
          if constexpr (i < 2) {
            ldV1(b0, sb_c, i, 0, va[cur][i][0]);
            ldV1(b0, sb_c, i, 1, va[cur][i][1]);
          } else {
#pragma unroll
            for (int kz = 2 * (i - 2); kz < 2 * (i - 2) + 2; ++kz)
              if (kz < G::KZ) ldA1(b0, integral_constant<int, sb + 1>{}, kz, A[cur ^ 1][kz]);
          }
        }
      };
      if constexpr (sb == 3) {
        ldV(b0, sb_c, va[cur]);
        if (kb + 1 < NB) {  // block kb+1 opens stage st
          const int st = (kb + 1) >> 2;
          if (st + 1 < nstage) wait_vmcnt<IPW_I>(); else wait_vmcnt<0>();
          lds_barrier();  // also: every wave has read stage st-1 (V(kb) above)
          if (st + 2 < nstage) issue_i(st + 2, const_cast<uint16_t*>(reinterpret_cast<const uint16_t*>(b0)));
          ldA(b1, integral_constant<int, 0>{}, A[cur ^ 1]);
        }
      }
      {
        const float dsave = dpart[1];
        group(Yes{}, Yes{}, sc[0], A[cur], qf[0], acc[0][0], acc[1][0], va[cur ^ 1], bw[0], sc[1],
              dpart[1], bw[1], loads);
        fixup(kb - 1, 1, sc[1], dsave, dpart[1], bw[1]);
      }
      {
        const float dsave = dpart[0];
        group(Yes{}, Yes{}, sc[1], A[cur], qf[1], acc[0][1], acc[1][1], va[cur ^ 1], bw[1], sc[0],
              dpart[0], bw[0], none);
        fixup(kb, 0, sc[0], dsave, dpart[0], bw[0]);
      }
    };
    auto rotate = [&]() __attribute__((always_inline)) {
      const char* t = b0;
      b0 = b1;
      b1 = b2;
      b2 = t;
    };
    step(integral_constant<int, 1>{}, 1);
    step(integral_constant<int, 2>{}, 2);
    step(integral_constant<int, 3>{}, 3);
    rotate();
    for (int st = 1; st < nstage; ++st) {
      step(integral_constant<int, 0>{}, 4 * st);
      step(integral_constant<int, 1>{}, 4 * st + 1);
      step(integral_constant<int, 2>{}, 4 * st + 2);
      step(integral_constant<int, 3>{}, 4 * st + 3);
      rotate();
    }
    // finish the last block (kb = NB - 1, odd): P V of both tiles
    {
      const float dsave = dpart[1];
      group(No{}, Yes{}, sc[0], A[0], qf[0], acc[0][0], acc[1][0], va[1], bw[0], sc[1], dpart[1],
            bw[1], none);
      fixup(NB - 1, 1, sc[1], dsave, dpart[1], bw[1]);
    }
    {
      // no P left to compute: the VALU parts of this group redo P_0 of the
      // last block into a scratch copy, which is discarded
      float dd = 0.f;
      uint32_t bx[8];
      group(No{}, Yes{}, sc[1], A[0], qf[1], acc[0][1], acc[1][1], va[1], bw[1], sc[0], dd, bx,
            none);
      hold(bx[0]);
    }
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
// K4: span output, eight-wave form (dv = 64; d = 64 with one or two feature
// blocks, d = 32).  The in-span loop and stage buffers of quadratic_kernel
// with the prefix readout added, and 512 threads owning 512
// queries (16 tiles of 32): wave w holds tiles w and 15 - w, so two waves
// share each SIMD with balanced causal work (waves w and w + 4 hold tiles
// adding up to 30), and one wave's VALU work (squared scores, query feature
// products) issues while the other's MFMAs run.  With a single wave per SIMD
// VALU issues at about half the rate and largely adds to the MFMA time.
// Twice the queries per workgroup halve the prefix-record bytes streamed
// into LDS per query (the readout's dominant copy traffic) and the in-span
// K / V copies; every LDS fragment feeds two tiles.  V rows are staged as they
// are in HBM and turned into V^T operands by transposing LDS reads, so no
// transposed copy of V goes through HBM.  A wave skips the MFMAs
// of key blocks past a tile's diagonal (it still takes part in every stage
// barrier and copy).  MFMAs are compiler builtins (the compiler inserts the
// wait states).  Grid: 8 * ceil(L / 512) * ceil(spans / 8) workgroups, one
// per CU (160 KB of LDS), a span's workgroups on one XCD.
// ---------------------------------------------------------------------------
constexpr int kQB8 = 512;  // queries per workgroup of the eight-wave form

template <int D, int DV, int NG>
__global__ __launch_bounds__(512) void span_output8_kernel(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ k,
    const uint16_t* __restrict__ v, const uint16_t* __restrict__ pre, float* __restrict__ out,
    float* __restrict__ den, int T, int L, int NS, int BH, int QB, int sp0, int nsp) {
  using G = GeoG<D, DV, NG>;
  static_assert(DV == 64, "the eight-wave form covers dv = 64");
  constexpr int DM = G::DM, RM = G::RM, KZM = G::KZM, KZ = G::KZ;
  constexpr int W = 8, NQ = 2, NT = kQB8 / 32;
  constexpr int KCH = D / 8;                    // 16-byte chunks per key row
  constexpr int KCHUNKS = kKB * KCH;            // K rows of one intra stage
  constexpr int VRCH = DV / 8;                  // 16-byte chunks per V row (8)
  constexpr int VCHUNKS = kKB * VRCH;           // V rows of one intra stage
  constexpr int ICH = KCHUNKS + VCHUNKS;        // chunks per intra stage
  static_assert(ICH * 16 <= kStageBytes && KCHUNKS % (64 * W) == 0 && VCHUNKS % (64 * W) == 0,
                "intra stage size");
  constexpr int IPW_K = KCHUNKS / (64 * W);     // copy instructions per wave: K rows
  constexpr int IPW_I = ICH / (64 * W);         // ... K rows then V^T rows
  constexpr int SCH = 2 * kKC;                  // chunks per S_pre row of one stage (32)
  constexpr int SCHUNKS = DV * SCH;
  static_assert(SCHUNKS * 16 <= kStageBytes && SCHUNKS % (64 * W) == 0, "readout stage size");
  constexpr int IPW_R = SCHUNKS / (64 * W);
  constexpr int NSTAGE_R = (G::NKS + kKC - 1) / kKC;
  static_assert(G::MT == 2, "two dv tiles");

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int c = lane & 31, g = lane >> 5;
  const int id = blockIdx.x;
  const int jx = id >> 3;
  const int qb = jx % QB;
  // Work item li in span-major order, last spans first: the first spans (no
  // readout) come last and fill the tail, and the eight XCDs (work item mod
  // 8) get equal shares of every span position.
  const int li = sp0 + 8 * (jx / QB) + (id & 7);
  if (li >= nsp) return;  // whole workgroup: padding of the grid
  const int s = NS - 1 - li / BH, bh = li % BH;
  const int sp = bh * NS + s;  // span record index (head-major)
  const long long span0 = static_cast<long long>(s) * L;
  const long long span_end = min(static_cast<long long>(T), span0 + L);
  const long long wg_q0 = span0 + static_cast<long long>(qb) * kQB8;
  if (wg_q0 >= span_end) return;  // whole workgroup beyond the sequence
  const uint16_t* qh = q + static_cast<long long>(bh) * T * D;
  const uint16_t* kh = k + static_cast<long long>(bh) * T * D;
  const uint16_t* vh = v + static_cast<long long>(bh) * T * DV;
  const uint16_t* rec = pre + static_cast<long long>(sp) * G::E;

  int tile[NQ];
  long long tq0[NQ];
  bool tlive[NQ];
#pragma unroll
  for (int i = 0; i < NQ; ++i) {
    tile[i] = qb * NT + (i == 0 ? wave : NT - 1 - wave);
    tq0[i] = span0 + 32LL * tile[i];
    tlive[i] = tq0[i] < span_end;
  }

  // ---- staging copies of both phases ------------------------------------------
  int last_tile = qb * NT + NT - 1;
  const int last_key_tile = static_cast<int>((span_end - 1 - span0) / 32);
  if (last_tile > last_key_tile) last_tile = last_key_tile;
  const int nstage = (last_tile + 1 + 3) / 4;  // 128-key intra stages
  // Copy i of a lane writes LDS chunk P = 512 i + 64 wave + lane.  K rows are
  // KCH chunks long and their copies are formed per copy (one or two per
  // stage).  For V and S^T the source row grows by a constant with i and the
  // XOR swizzle of the lane's chunk does not depend on i, so one offset per
  // operand serves all of a lane's copies:
  //   V    row 64 i' + 8 wave + lane / 8,  chunk (lane % 8) ^ vswz (i' = i - IPW_K)
  //   S^T  row 16 i + 2 wave + lane / 32,  chunk lane % 32
  // V rows are stored as they are in HBM, 128 bytes each, with chunk c of key
  // row r at chunk c ^ 4 ((r >> 1) & 1); bit 1 of the row is bit 4 of the lane.
  static_assert(VRCH == 8 && SCH == 32 && W == 8 && KCHUNKS % 512 == 0, "copy geometry");
  const int vrow0 = 8 * wave + (lane >> 3);
  const int vsrc0 = vrow0 * DV + 8 * ((lane & 7) ^ (4 * ((lane >> 4) & 1)));
  const int rrow0 = 2 * wave + g;
  const int rcl = c ^ rswz(rrow0);  // the chunk a lane copies of its S^T row
  const int rsrc0 = rrow0 * G::NSLOT + 8 * rcl;
  auto issue_i = [&](int st, uint16_t* buf) __attribute__((always_inline)) {
    const long long key0 = span0 + static_cast<long long>(st) * kKB;
#pragma unroll
    for (int i = 0; i < IPW_I; ++i) {
      const void* src;
      if (i < IPW_K) {
        const int P = (i * W + wave) * 64 + lane;
        const int r = P / KCH, pos = P % KCH;
        // keys past the sequence: re-read the last row (never used)
        const long long over = key0 + r - (T - 1);
        src = kh + (key0 + r) * D + 8 * (pos ^ kswz<D>(r)) - (over > 0 ? over * D : 0);
      } else {
        // keys past the sequence: re-read the last row (their weights are zero)
        const int r = 64 * (i - IPW_K) + vrow0;
        const long long over = key0 + r - (T - 1);
        src = vh + key0 * DV + vsrc0 + 64 * (i - IPW_K) * DV - (over > 0 ? over * DV : 0);
      }
      g2lds16(src, buf + (i * W + wave) * 512);
    }
  };
  auto issue_r = [&](auto stg_c) __attribute__((always_inline)) {
    constexpr int stg = decltype(stg_c)::value;
    constexpr int kc = (G::NKS - stg * kKC < kKC) ? (G::NKS - stg * kKC) : kKC;
    uint16_t* buf = stage_buf((3 + stg) % 5);
    // chunks past the last K-step: re-read the row's first chunk (never used)
    int off = rsrc0;
    if constexpr (kc < kKC) {
      if (rcl >= 2 * kc) off -= 8 * rcl;
    }
#pragma unroll
    for (int i = 0; i < IPW_R; ++i)
      g2lds16(rec + 16 * kKC * stg + off + 16 * i * G::NSLOT, buf + (i * W + wave) * 512);
  };
  // Stage 0 of the in-span phase first, the query and Z fragments behind it;
  // the wave waits for that one round trip (loads complete in order, so the
  // compiler's wait for the fragments covers the copies issued before them;
  // every fragment is consumed, so no load is left to be waited for behind
  // later copies), then issues in-span stage 1 and readout stages 0 and 1.
  issue_i(0, g_stage0);
  // qf[i][KZM bb + kz] holds q[t][DM bb + 8 kz + RM g .. +7] of this lane's
  // query t = tq0 + c, per feature block bb
  bf16x8 qf[NQ][KZ];
#pragma unroll
  for (int i = 0; i < NQ; ++i) {
    const long long t = min(tq0[i] + c, static_cast<long long>(T) - 1);
#pragma unroll
    for (int kz = 0; kz < KZ; ++kz)
      qf[i][kz] = *reinterpret_cast<const bf16x8*>(qh + t * D + DM * (kz / KZM) +
                                                   8 * (kz % KZM) + RM * g);
  }
  // The first span of a head has a zero prefix: its workgroups read no
  // prefix record and skip the readout (wave-uniform).
  const bool pfx = s > 0;
  // Z_pre operand fragments of each feature block
  bf16x8 zA[NG][G::ZMB][KZM];
  if (pfx) {
#pragma unroll
    for (int bb = 0; bb < NG; ++bb)
#pragma unroll
      for (int m = 0; m < G::ZMB; ++m)
#pragma unroll
        for (int kz = 0; kz < KZM; ++kz)
          zA[bb][m][kz] = *reinterpret_cast<const bf16x8*>(
              rec + G::ES + static_cast<long long>(bb) * DM * DM + ((m * KZM + kz) * 64 + lane) * 8);
  }
#pragma unroll
  for (int i = 0; i < NQ; ++i)
#pragma unroll
    for (int kz = 0; kz < KZ; ++kz) asm volatile("" ::"v"(qf[i][kz]));
  if (pfx) {
#pragma unroll
    for (int bb = 0; bb < NG; ++bb)
#pragma unroll
      for (int m = 0; m < G::ZMB; ++m)
#pragma unroll
        for (int kz = 0; kz < KZM; ++kz) asm volatile("" ::"v"(zA[bb][m][kz]));
  }
  if (nstage > 1) issue_i(1, g_stage1);
  if (pfx) {
    issue_r(std::integral_constant<int, 0>{});
    if constexpr (NSTAGE_R > 1) issue_r(std::integral_constant<int, 1>{});
  }

  // ---- denominator from the prefix: sum over blocks of q_bb^T Z_bb q_bb ------
  float dpart[NQ];
#pragma unroll
  for (int i = 0; i < NQ; ++i) {
    float dsum = 0.f;
    if (!pfx) {
      dpart[i] = 0.f;
      continue;
    }
#pragma unroll
    for (int bb = 0; bb < NG; ++bb)
#pragma unroll
      for (int m = 0; m < G::ZMB; ++m) {
        f32x16 az;
#pragma unroll
        for (int r = 0; r < 16; ++r) az[r] = 0.f;
#pragma unroll
        for (int kz = 0; kz < KZM; ++kz) az = mfma32(zA[bb][m][kz], qf[i][KZM * bb + kz], az);
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          // row sigma = 16m + r + RM g of block bb: element (16m + r) % 8 of the
          // block's fragment (16m + r) / 8
          const int x = 16 * m + r;
          const uint32_t w = word_of(qf[i][KZM * bb + (x >> 3)], (x & 7) >> 1);
          dsum += ((x & 1) ? bf16hi_f32(w) : bf16lo_f32(w)) * az[r];
        }
      }
    dpart[i] = dsum;
  }

  f32x16 acc[2][NQ];  // O^T of tile i, dv columns 32 m .. 32 m + 31
#pragma unroll
  for (int m = 0; m < 2; ++m)
#pragma unroll
    for (int i = 0; i < NQ; ++i)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[m][i][r] = 0.f;

  // ---- causal squared-score attention inside the span -----------------------
  // Per 32-key block kb and live tile i with kb up to its diagonal:
  // S = K_kb Q_i^T (KZ MFMAs), P = S^2 (masked above the diagonal on the
  // diagonal block; the row sums go to the denominator), O_i^T += V_kb^T P
  // (four MFMAs: two dv halves x two 16-key halves; the lane's score
  // registers are directly the P fragment, and the V^T fragments are read in
  // the same permuted key order).  The block's K and V fragments are read from
  // LDS once for both tiles.
  {
    unsigned kfo[2][KZ];
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int kz = 0; kz < KZ; ++kz) {
        const int krow = 32 * h + c;
        const int chunk = (DM / 8) * (kz / KZM) + (kz % KZM) + (RM / 8) * g;
        kfo[h][kz] = static_cast<unsigned>((krow * KCH + (chunk ^ kswz<D>(krow))) * 16);
      }
    // V^T fragments come from transposing reads of the V rows
    // (ds_read_b64_tr_b16: lane j of a 16-lane group receives, in slot s,
    // 16-bit element j % 4 of the 8-byte piece that lane 4 s + j / 4 of the
    // group addresses).  Lane j of group G addresses key row 4 g + j / 4 of a
    // 16-key half (plus 8 for the second read) and the piece holding dv
    // 32 m + 16 (G % 2) + 4 (j % 4) .. + 3, so it receives dv 32 m + 16 (G % 2) + j
    // of keys 4 g + 0..3 and 8 + 4 g + 0..3: the A operand in the key order of
    // the score fragments (rows 8 (r / 4) + 4 g + r % 4).  The four rows a group
    // reads fall in distinct banks under the chunk swizzle.
    const int jl = lane & 15;
    unsigned vfo[2];
#pragma unroll
    for (int m = 0; m < 2; ++m) {
      const int ch = 4 * m + 2 * ((lane >> 4) & 1) + ((jl & 3) >> 1);
      vfo[m] = static_cast<unsigned>(KCHUNKS * 16 + (4 * g + (jl >> 2)) * (VRCH * 16) +
                                     16 * (ch ^ (4 * ((jl >> 3) & 1))) + 8 * (jl & 1));
    }
    int tdiag[NQ];  // a tile's diagonal block, -1 for a tile beyond the sequence
#pragma unroll
    for (int i = 0; i < NQ; ++i) tdiag[i] = __builtin_amdgcn_readfirstlane(tlive[i] ? tile[i] : -1);
    const int tmax = tdiag[0] > tdiag[1] ? tdiag[0] : tdiag[1];

    auto block = [&](const char* buf, auto sb_c, int kb) __attribute__((always_inline)) {
      constexpr int sb = decltype(sb_c)::value;
      if (kb > tmax) return;  // wave-uniform: past both diagonals
      bf16x8 A[KZ];
#pragma unroll
      for (int kz = 0; kz < KZ; ++kz)
        A[kz] = *reinterpret_cast<const bf16x8*>(buf + (sb >> 1) * (64 * KCH * 16) +
                                                 kfo[sb & 1][kz]);
      bf16x8 V[2][2];
#pragma unroll
      for (int m = 0; m < 2; ++m)
#pragma unroll
        for (int kv = 0; kv < 2; ++kv) {
          const char* vp = buf + vfo[m] + (32 * sb + 16 * kv) * (VRCH * 16);
          const uint2 lo = lds_tr16(vp), hi = lds_tr16(vp + 8 * (VRCH * 16));
          V[m][kv] = __builtin_bit_cast(bf16x8, make_uint4(lo.x, lo.y, hi.x, hi.y));
        }
#pragma unroll
      for (int i = 0; i < NQ; ++i) {
        if (kb > tdiag[i]) continue;  // wave-uniform
        // scores per feature block; the weight is the sum of their squares
        f32x16 sc[NG];
#pragma unroll
        for (int bb = 0; bb < NG; ++bb) {
#pragma unroll
          for (int r = 0; r < 16; ++r) sc[bb][r] = 0.f;
#pragma unroll
          for (int kz = 0; kz < KZM; ++kz)
            sc[bb] = mfma32(A[KZM * bb + kz], qf[i][KZM * bb + kz], sc[bb]);
        }
        auto p_of = [&](int r) __attribute__((always_inline)) {
          float p = sc[0][r] * sc[0][r];
#pragma unroll
          for (int bb = 1; bb < NG; ++bb) p += sc[bb][r] * sc[bb][r];
          return p;
        };
        uint32_t bw[8];
        if (kb < tdiag[i]) {
#pragma unroll
          for (int j = 0; j < 8; ++j) {
            const float p0 = p_of(2 * j);
            const float p1 = p_of(2 * j + 1);
            dpart[i] += p0 + p1;
            bw[j] = pack_bf16x2(p0, p1);
          }
        } else {
#pragma unroll
          for (int j = 0; j < 8; ++j) {
            const int r0 = 2 * j, r1 = 2 * j + 1;
            const float p0 = (8 * (r0 >> 2) + 4 * g + (r0 & 3) > c) ? 0.f : p_of(r0);
            const float p1 = (8 * (r1 >> 2) + 4 * g + (r1 & 3) > c) ? 0.f : p_of(r1);
            dpart[i] += p0 + p1;
            bw[j] = pack_bf16x2(p0, p1);
          }
        }
#pragma unroll
        for (int kv = 0; kv < 2; ++kv) {
          const bf16x8 Bp = __builtin_bit_cast(
              bf16x8, make_uint4(bw[4 * kv], bw[4 * kv + 1], bw[4 * kv + 2], bw[4 * kv + 3]));
          acc[0][i] = mfma32(V[0][kv], Bp, acc[0][i]);
          acc[1][i] = mfma32(V[1][kv], Bp, acc[1][i]);
        }
      }
    };

    const char* b0 = reinterpret_cast<const char*>(g_stage0);
    const char* b1 = reinterpret_cast<const char*>(g_stage1);
    const char* b2 = reinterpret_cast<const char*>(g_stage2);
    lds_barrier();  // stage 0 (its copies were waited for with the fragments)
    if (nstage > 2) issue_i(2, g_stage2);
    for (int st = 0; st < nstage; ++st) {
      if (st > 0) {
        if (st + 1 < nstage) wait_vmcnt<IPW_I>(); else wait_vmcnt<0>();
        lds_barrier();  // stage st has landed; every wave is done with stage st - 1
        if (st + 2 < nstage)
          issue_i(st + 2, const_cast<uint16_t*>(reinterpret_cast<const uint16_t*>(b2)));
      }
      block(b0, std::integral_constant<int, 0>{}, 4 * st);
      block(b0, std::integral_constant<int, 1>{}, 4 * st + 1);
      block(b0, std::integral_constant<int, 2>{}, 4 * st + 2);
      block(b0, std::integral_constant<int, 3>{}, 4 * st + 3);
      const char* t = b0;
      b0 = b1;
      b1 = b2;
      b2 = t;
    }
    wait_vmcnt<0>();  // the readout's first stages
    lds_barrier();    // every wave is done with the intra buffers
  }
  // Readout stage s sits in buffer (3 + s) % 5 and is copied in four stages
  // ahead: stages 0 and 1 came with the prologue, 2 to 4 go now (into the
  // in-span buffers), and stage s + 4 is issued once every wave is done with
  // stage s - 1, whose buffer it takes.
  if (pfx) static_for<2, (NSTAGE_R < 5 ? NSTAGE_R : 5)>([&](auto stg_c) { issue_r(stg_c); });

  if (pfx) {  // the first span's prefix is zero: no readout
    // ---- readout of the span prefix: Phi_w(Q) S_pre ----------------------------
    // rotated fp32 query rows per feature block:
    // qr[i][DM bb + x] = q[t][DM bb + (x + RM g) % DM]; the lane's own
    // fragments of block bb hold x < RM, the lane 32 away holds the rest
    float qr[NQ][D];
#pragma unroll
    for (int i = 0; i < NQ; ++i)
#pragma unroll
      for (int kz = 0; kz < KZ; ++kz) {
        const int base = DM * (kz / KZM) + 8 * (kz % KZM);
        const uint4 w4 = __builtin_bit_cast(uint4, qf[i][kz]);
        const uint32_t w[4] = {w4.x, w4.y, w4.z, w4.w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const uint32_t pw = static_cast<uint32_t>(__shfl_xor(static_cast<int>(w[e]), 32));
          qr[i][base + 2 * e] = bf16lo_f32(w[e]);
          qr[i][base + 2 * e + 1] = bf16hi_f32(w[e]);
          qr[i][base + RM + 2 * e] = bf16lo_f32(pw);
          qr[i][base + RM + 2 * e + 1] = bf16hi_f32(pw);
        }
      }
    // A fragment of K-step kk: row c (and c + 32), chunk (2 (kk % 8) + g) ^ (c % 16)
    // of the 32 in the row, plus 256 bytes for kk >= 8; formed per K-step (a
    // XOR and an add) rather than held in eight registers
    const unsigned arow = static_cast<unsigned>(c * SCH * 16);
    const unsigned asw = static_cast<unsigned>(g ^ rswz(c));
    const bool any_live = tlive[0] || tlive[1];
    static_for<0, NSTAGE_R>([&](auto stg_c) {
      constexpr int stg = decltype(stg_c)::value;
      constexpr int k0 = stg * kKC;
      constexpr int kc = (G::NKS - k0 < kKC) ? (G::NKS - k0) : kKC;
      if constexpr (stg >= 2) {
        // stages stg + 1 .. min(stg + 3, last) may stay in flight
        constexpr int later = (NSTAGE_R - 1 - stg < 3) ? NSTAGE_R - 1 - stg : 3;
        wait_vmcnt<IPW_R * later>();
      }
      if constexpr (stg >= 1) lds_barrier();  // stage stg landed; stage stg - 1 consumed
      if constexpr (stg >= 1 && stg + 4 < NSTAGE_R) issue_r(std::integral_constant<int, stg + 4>{});
      if (!any_live) return;  // wave-uniform: dead tiles only take part in the staging
      const char* Sb = reinterpret_cast<const char*>(stage_buf((3 + stg) % 5));
      static_for<0, kc>([&](auto kk_c) {
        constexpr int kk = decltype(kk_c)::value;
        constexpr int kap = k0 + kk;
        // K-step kl of feature block bb: slots 16 kl + 8 g + j pair registers
        // r1 + j and r1 + j + dl of the block's rotated row
        constexpr int bb = kap / G::NKSM, kl = kap % G::NKSM;
        constexpr int r1 = (8 * kl) % RM, dl = (8 * kl) / RM;
        const char* ap = Sb + arow + ((static_cast<unsigned>(2 * (kk & 7)) ^ asw) << 4) + (kk >> 3) * 256;
        const bf16x8 A0 = *reinterpret_cast<const bf16x8*>(ap);
        const bf16x8 A1 = *reinterpret_cast<const bf16x8*>(ap + 32 * SCH * 16);
#pragma unroll
        for (int i = 0; i < NQ; ++i) {
          float pr[8];
#pragma unroll
          for (int j = 0; j < 8; ++j)
            pr[j] = qr[i][DM * bb + r1 + j] * qr[i][DM * bb + (r1 + j + dl) % DM];
          const bf16x8 bq = __builtin_bit_cast(
              bf16x8, make_uint4(pack_bf16x2(pr[0], pr[1]), pack_bf16x2(pr[2], pr[3]),
                                 pack_bf16x2(pr[4], pr[5]), pack_bf16x2(pr[6], pr[7])));
          acc[0][i] = mfma32(A0, bq, acc[0][i]);
          acc[1][i] = mfma32(A1, bq, acc[1][i]);
        }
      });
    });

  }

  // ---- normalise and store ---------------------------------------------------
  // A tile's accumulators hold 4 consecutive dv columns of one query per
  // lane; they go through this wave's own 16 KB of the (now idle) stage
  // buffers, [32 queries][68 floats] per tile, so that each store
  // instruction writes four whole 256-byte output rows.
  lds_barrier();  // every wave is done with the readout buffers
  float* ost = reinterpret_cast<float*>(stage_buf(wave >> 1)) + (wave & 1) * 4096;
  constexpr int OS = DV + 4;  // floats per LDS row (16-byte aligned rows)
  static_assert(32 * OS <= 4096, "one tile per round fits the wave's 16 KB");
#pragma unroll
  for (int i = 0; i < NQ; ++i) {
    const float Dt = dpart[i] + __shfl_xor(dpart[i], 32);
    if (!tlive[i]) continue;  // wave-uniform
    if (den != nullptr && g == 0) {  // the denominators, for a backward pass
      const long long t = tq0[i] + c;
      if (t < span_end) den[static_cast<long long>(bh) * T + t] = Dt;
    }
    const float inv = (Dt > 0.f) ? 1.f / Dt : 0.f;
#pragma unroll
    for (int m = 0; m < 2; ++m)
#pragma unroll
      for (int r4 = 0; r4 < 4; ++r4) {
        float4 o;
        o.x = acc[m][i][4 * r4 + 0] * inv;
        o.y = acc[m][i][4 * r4 + 1] * inv;
        o.z = acc[m][i][4 * r4 + 2] * inv;
        o.w = acc[m][i][4 * r4 + 3] * inv;
        *reinterpret_cast<float4*>(ost + c * OS + 32 * m + 8 * r4 + 4 * g) = o;
      }
    __builtin_amdgcn_s_waitcnt(0xC07F);  // this wave's LDS writes are done
    __builtin_amdgcn_wave_barrier();
    // lane l: rows 4 j + l / 16 of the tile, 16-byte piece l % 16 of the row
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int row = 4 * j + (lane >> 4), pc = lane & 15;
      const float4 o = *reinterpret_cast<const float4*>(ost + row * OS + 4 * pc);
      const long long t = tq0[i] + row;
      if (t < span_end)
        *reinterpret_cast<float4*>(out + (static_cast<long long>(bh) * T + t) * DV + 4 * pc) = o;
    }
    __builtin_amdgcn_s_waitcnt(0xC07F);  // reads done before the next tile's writes
    __builtin_amdgcn_wave_barrier();
  }
}

// ---------------------------------------------------------------------------
// V^T of the keys key_base .. key_base + LV - 1 of every head, into
// vtp + bh out_bh + out0 as [dv][LV] bf16, keys of every 16-key group in the
// order 0-3, 8-11, 4-7, 12-15 (the key order of the quadratic kernel's P V
// product), keys at or past T zero: the whole head for the quadratic form.
// A workgroup transposes 64 keys through LDS.
// grid (LV / 64, BH), block 256.
// ---------------------------------------------------------------------------
template <int DV>
__global__ __launch_bounds__(256) void vt_permute_kernel(const uint16_t* __restrict__ v,
                                                         uint16_t* __restrict__ vtp, int T,
                                                         int LV, int key_base,
                                                         long long out_bh, long long out0) {
  constexpr int KEYS = 64, CH = DV / 8;  // keys per workgroup, 16-byte chunks per V row
  __shared__ uint32_t tile[KEYS][DV / 2 + 1];  // [key][dv pair], one word of padding
  const int bh = blockIdx.y;
  const long long key0 = static_cast<long long>(blockIdx.x) * KEYS;
  const uint16_t* vh = v + (static_cast<long long>(bh) * T + key_base) * DV;
  const long long nkeys = static_cast<long long>(T) - key_base;
  for (int i = threadIdx.x; i < KEYS * CH; i += 256) {
    const int key = i / CH, ch = i % CH;
    uint4 x = make_uint4(0u, 0u, 0u, 0u);
    if (key0 + key < nkeys) x = *reinterpret_cast<const uint4*>(vh + (key0 + key) * DV + 8 * ch);
    tile[key][4 * ch + 0] = x.x;
    tile[key][4 * ch + 1] = x.y;
    tile[key][4 * ch + 2] = x.z;
    tile[key][4 * ch + 3] = x.w;
  }
  __syncthreads();
  uint16_t* out = vtp + bh * out_bh + out0;
  for (int i = threadIdx.x; i < DV * (KEYS / 8); i += 256) {
    const int m = i / (KEYS / 8), h = i % (KEYS / 8);  // dv row, output chunk of 8 keys
    const int base = 16 * (h >> 1) + 4 * (h & 1);        // keys base+0..3, base+8..11
    uint16_t e[8];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const uint32_t w0 = tile[base + j][m >> 1], w1 = tile[base + 8 + j][m >> 1];
      e[j] = static_cast<uint16_t>((m & 1) ? (w0 >> 16) : w0);
      e[4 + j] = static_cast<uint16_t>((m & 1) ? (w1 >> 16) : w1);
    }
    *reinterpret_cast<uint4*>(out + static_cast<long long>(m) * LV + key0 + 8 * h) =
        make_uint4(e[0] | (static_cast<uint32_t>(e[1]) << 16), e[2] | (static_cast<uint32_t>(e[3]) << 16),
                   e[4] | (static_cast<uint32_t>(e[5]) << 16), e[6] | (static_cast<uint32_t>(e[7]) << 16));
  }
}

// ---------------------------------------------------------------------------
// Host side
// ---------------------------------------------------------------------------
bool mfma_supported(int d, int dv, int C, int g) {
  const bool shape = (d == 64 && (g == 1 || g == 2)) || (d == 32 && g == 1);
  return shape && dv == 64 && C > 0 && C % 32 == 0 && C <= 1024;
}

static long long mfma_record(int d, int g) {
  if (d == 64) return g == 2 ? GeoG<64, 64, 2>::E : GeoG<64, 64, 1>::E;
  return GeoG<32, 64, 1>::E;
}

static size_t align256(size_t x) { return (x + 255) & ~static_cast<size_t>(255); }

// Sequence length rounded up to whole intra stages so that every staged key
// block of the quadratic form lies inside its V^T copy.
static int span_alloc(int L) { return (L + kKB - 1) / kKB * kKB; }

constexpr int kSpansPerLaunch = 1 << 20;

size_t mfma_forward_workspace(int BH, int T, int d, int /*dv*/, int L, int g) {
  const size_t NS = (static_cast<size_t>(T) + L - 1) / L;
  const size_t recs = static_cast<size_t>(BH) * NS * static_cast<size_t>(mfma_record(d, g));
  return align256(recs * sizeof(uint16_t));
}

template <int D, int DV, int NG>
static hipError_t run_mfma(const void* q, const void* k, const void* v, float* out, float* den,
                           int BH, int T, int L, void* ws, hipStream_t st, hipEvent_t* ev) {
  using G = GeoG<D, DV, NG>;
  const int NS = (T + L - 1) / L;
  uint16_t* spanst = static_cast<uint16_t*>(ws);
  const uint16_t* qq = static_cast<const uint16_t*>(q);
  const uint16_t* kk = static_cast<const uint16_t*>(k);
  const uint16_t* vv = static_cast<const uint16_t*>(v);
  const int nsp = BH * NS;
  hipError_t e = record(ev, 0, st);
  if (e != hipSuccess) return e;
  // K2 over the BH (NS - 1) spans that enter a prefix, in launches of at most
  // kSpansPerLaunch spans (1-D grid size limit); none when every head is one
  // span
  const int nst = BH * (NS - 1);
  for (int sp0 = 0; sp0 < nst; sp0 += kSpansPerLaunch) {
    const int cnt = nst - sp0 < kSpansPerLaunch ? nst - sp0 : kSpansPerLaunch;
    const unsigned nb2 = 8u * StateGrid<D, DV, NG>::NB * static_cast<unsigned>((cnt + 7) / 8);
    span_state_kernel<D, DV, NG><<<nb2, 64 * StateGrid<D, DV, NG>::NW, 0, st>>>(
        kk, vv, spanst, T, L, NS, BH, sp0, sp0 + cnt);
  }
  if ((e = record(ev, 1, st)) != hipSuccess) return e;
  // one span per head: its prefix is zero and the output kernel reads none
  if (NS > 1)
    launch_scan_exclusive_bf16(spanst, NS, G::E, static_cast<long long>(NS) * G::E, BH,
                               SlotWeight<D, DV, NG>{}, st);
  if ((e = record(ev, 2, st)) != hipSuccess) return e;
  const int qb8 = (L + kQB8 - 1) / kQB8;
  for (int sp0 = 0; sp0 < nsp; sp0 += kSpansPerLaunch) {
    const int cnt = nsp - sp0 < kSpansPerLaunch ? nsp - sp0 : kSpansPerLaunch;
    const unsigned nb8 = 8u * static_cast<unsigned>(qb8) * static_cast<unsigned>((cnt + 7) / 8);
    span_output8_kernel<D, DV, NG><<<nb8, 512, 0, st>>>(qq, kk, vv, spanst, out, den, T, L, NS,
                                                        BH, qb8, sp0, sp0 + cnt);
  }
  if ((e = hipGetLastError()) != hipSuccess) return e;
  return record(ev, 3, st);
}

// Quadratic form: one span per head covering the whole sequence, no state,
// no scan, no prefix readout; the workspace holds the permuted V^T.
size_t mfma_quadratic_workspace(int BH, int T, int dv) {
  return align256(static_cast<size_t>(BH) * dv * span_alloc(T) * sizeof(uint16_t));
}

template <int D, int DV, int NG>
static hipError_t run_quadratic(const void* q, const void* k, const void* v, float* out, int BH,
                                int T, void* ws, hipStream_t st) {
  const int LA = span_alloc(T);
  static_assert(kKB % 64 == 0, "the transpose writes whole 64-key groups");
  uint16_t* vtp = static_cast<uint16_t*>(ws);
  vt_permute_kernel<DV><<<dim3(static_cast<unsigned>(LA / 64), static_cast<unsigned>(BH)), 256, 0,
                          st>>>(static_cast<const uint16_t*>(v), vtp, T, LA, 0,
                                static_cast<long long>(DV) * LA, 0LL);
  const int qblocks = (T + OutGrid<D, DV>::QB_TOKENS - 1) / OutGrid<D, DV>::QB_TOKENS;
  // 8 * qblocks * ceil(cnt / 8) workgroups per launch, below 2^31
  int per = static_cast<int>((0x7fffffffLL / (8LL * qblocks)) * 8);
  if (per > kSpansPerLaunch) per = kSpansPerLaunch;
  for (int sp0 = 0; sp0 < BH; sp0 += per) {
    const int cnt = BH - sp0 < per ? BH - sp0 : per;
    const unsigned nb4 = 8u * static_cast<unsigned>(qblocks) * static_cast<unsigned>((cnt + 7) / 8);
    quadratic_kernel<D, DV, NG><<<nb4, 256, 0, st>>>(static_cast<const uint16_t*>(q),
                                                     static_cast<const uint16_t*>(k), vtp, out, T,
                                                     T, LA, 1, qblocks, sp0, sp0 + cnt);
  }
  return hipGetLastError();
}

hipError_t launch_mfma_quadratic(const void* q, const void* k, const void* v, float* out, int BH,
                                 int T, int d, int dv, int g, void* ws, hipStream_t st) {
  if (d == 64 && dv == 64 && g == 1) return run_quadratic<64, 64, 1>(q, k, v, out, BH, T, ws, st);
  if (d == 64 && dv == 64 && g == 2) return run_quadratic<64, 64, 2>(q, k, v, out, BH, T, ws, st);
  if (d == 32 && dv == 64 && g == 1) return run_quadratic<32, 64, 1>(q, k, v, out, BH, T, ws, st);
  return hipErrorInvalidValue;
}

hipError_t launch_mfma_forward(const void* q, const void* k, const void* v, float* out, float* den,
                               int BH, int T, int d, int dv, int g, int L, void* ws,
                               hipStream_t st, hipEvent_t* ev) {
  if (d == 64 && dv == 64 && g == 1)
    return run_mfma<64, 64, 1>(q, k, v, out, den, BH, T, L, ws, st, ev);
  if (d == 64 && dv == 64 && g == 2)
    return run_mfma<64, 64, 2>(q, k, v, out, den, BH, T, L, ws, st, ev);
  if (d == 32 && dv == 64 && g == 1)
    return run_mfma<32, 64, 1>(q, k, v, out, den, BH, T, L, ws, st, ev);
  return hipErrorInvalidValue;
}

}  // namespace kata
