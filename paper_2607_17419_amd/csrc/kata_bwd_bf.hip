// kata_bwd_bf.hip -- gradients (dq, dk, dv) of the O(T) chunked backward of
// KATA-M1 on the bf16 matrix cores of gfx950, for bf16 inputs with d = dv = 64
// and chunks of C = 64 tokens.  The other launches of the backward (chunk
// states, scans, coefficients) and every other shape are in kata_bwd.hip; this
// file is built with the MFMA results in VGPRs (the accumulators are updated
// by VALU code between MFMAs).
#include <type_traits>

#include "kata_common.hpp"
#include "kata_internal.hpp"

namespace kata {

namespace {

// ---------------------------------------------------------------------------
// Gradients of chunk c on the bf16 matrix cores (v_mfma_f32_32x32x16_bf16,
// fp32 accumulation): bf16 inputs, d = dv = C = 64, one feature block.  The
// prefix and suffix records come from the scans with S in bf16 (z in fp32)
// and the in-chunk score products are rounded to bf16 once in LDS.  The
// coefficients a_t, b_t enter as a bf16 pair hi + lo (lo = the rounding residue
// of hi) wherever they multiply a state or a value: <a_t, v_s> + b_t and
// S a_t + b_t z cancel to small values when the attention of row t is peaked
// (exactly at t = 0), and one bf16 rounding of a_t, b_t (unit roundoff 2^-8)
// would leave a residue of that order of the cancelling terms; the pair
// represents them within 2^-16.
//
// In-chunk terms as five 64 x 64 x 64 products: Sc = Q K^T and Cw = A V^T + b
// (dL/dw_ts), the masked Pm = 2 Cw * Sc and W = Sc^2 (s <= t), then
//   dq^T += K^T Pm^T,  dk^T += Q^T Pm,  dv^T += A^T W.
// Inter-chunk terms slab by slab: slab y holds the packed record rows
// {y, x}, x >= y, which are the consecutive rows packed(y, y) .. packed(y, 63)
// (the row-major upper triangle), with z (dz) as a 65th column; the diagonal
// row arrives halved from the scan.  For the query side, with G_t[{y,x}] =
// S[{y,x}] . a_t + b_t z[{y,x}],
//   P^T[x][t] = sum_j S_slab[x][j] a_t[j] + z_slab[x] b_t          (MFMA, K = 80)
//   dq^T[x][t] += 2 q_t[y] P^T[x][t]                 (pair {x,y}, coordinate x)
//   dq[t][y]   += 2 sum_x q_t[x] P^T[x][t]           (pair {x,y}, coordinate y)
// which together count every off-diagonal pair from both sides and the
// diagonal pair once (the halving).  The key side is the same with the suffix
// record, v_i and a unit coefficient for dz.  The value gradient takes the
// slab transposed, DT[j][x] = dS_slab[x][j] (1/2 on the diagonal, 1 off it, 0
// below), so that with the pair weights (1 on the diagonal, 2 off it)
//   dv^T[j][i] += 2 k_i[y] sum_x DT[j][x] k_i[x].
// Two groups of four waves; group g takes the slabs y = g, g + 2, ... in its own
// LDS slab buffer, so each SIMD runs two waves (one per group).  The groups
// stage and compute in step: two computing waves on a SIMD hide each other's
// MFMA and epilogue latency (running them a phase apart was slower).  In a group,
// the waves of role 0-1 own dq of token tile role, 2-3 dk of key tile role - 2,
// and every wave one 32 x 32 tile (value tile role >> 1, key tile role & 1) of
// dv; role = w in group 0 and w + 2 (mod 4) in group 1, so that every SIMD
// pairs a dq and a dk wave (dq has twice the slab MFMAs).  Group 0 also
// stages the chunk rows and takes the in-chunk terms; at the end group 1 adds
// its accumulators through LDS.  The record rows of a group's next slab are
// fetched into registers (buffer loads) while the current one is used.
// grid (NC, BH), block 512, dynamic LDS kBfLds bytes (one workgroup per CU).
// ---------------------------------------------------------------------------
constexpr int kBP = 72;         // bf16 row stride of a 64 x 64 operand tile
constexpr int kBW = 88;         // bf16 row stride of a tile with a 65th column (K = 80)
constexpr int kBR = 68;         // fp32 row stride of the per-slab row-sum tiles
constexpr int kBT = 64 * kBP;   // elements of a kBP tile
constexpr int kBTW = 64 * kBW;  // elements of a kBW tile
constexpr int kBfOffK = 2 * kBT;
constexpr int kBfOffV = kBfOffK + 2 * kBT;
constexpr int kBfOffA = kBfOffV + 2 * kBTW;
constexpr int kBfOffAl = kBfOffA + 2 * kBTW;
constexpr int kBfOffSlab = kBfOffAl + 2 * kBTW;
constexpr int kBfSlab = 2 * (2 * kBTW + kBT);  // bytes of one slab buffer (S, dS, dS^T)
constexpr int kBfOffR = kBfOffSlab + 2 * kBfSlab;
constexpr int kBfLds = kBfOffR + 2 * 64 * kBR * 4;
constexpr int kBfN = 2080;      // packed features of d = 64
constexpr int kBfWord3 = 0x00020000;  // buffer resource word 3 (raw dword access)
// Chunk records of this path: S as bf16 rows of 64 (128 bytes), then z as fp32;
// the scans write the diagonal features f = (a, a) halved (weight 1/2).
constexpr int kRecSB = kBfN * 64 * 2;    // bytes of the S part
constexpr int kRecB = kRecSB + kBfN * 4;  // bytes of a record
constexpr int kRecS16 = kRecSB / 16;      // 16-byte chunks of the S part
constexpr int kRec16 = kRecB / 16;        // 16-byte chunks of a record
static_assert(kRecB % 16 == 0, "records are 16-byte aligned");
static_assert(6 * kBT * 2 <= 2 * kBfSlab, "in-chunk tiles fit the slab buffers");

__device__ __forceinline__ f32x16 mfma_bf(const bf16x8& a, const bf16x8& b, const f32x16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ bf16x8 ld8(const uint16_t* p) {
  return *reinterpret_cast<const bf16x8*>(p);
}
__device__ __forceinline__ uint16_t bf_bits(float x) {
  return static_cast<uint16_t>(pack_bf16x2(x, 0.f) & 0xFFFFu);
}
__device__ __forceinline__ float bf_f32(uint16_t b) {
  return __uint_as_float(static_cast<uint32_t>(b) << 16);
}
// bf16 pairs: the low / high halves of two words as one word
__device__ __forceinline__ uint32_t lo_pair(uint32_t a, uint32_t b) {
  return (a & 0xFFFFu) | (b << 16);
}
__device__ __forceinline__ uint32_t hi_pair(uint32_t a, uint32_t b) {
  return (a >> 16) | (b & 0xFFFF0000u);
}

// One slab's record values in registers: rows 8 rg .. 8 rg + 7 of the slab
// tile, columns 2 cp, 2 cp + 1 of S and dS (bf16 pairs), and the z / dz of
// row lane.
struct BfSlabRegs {
  uint32_t a[8], b[8];
  float za, zb;
};

__global__ __launch_bounds__(512, 1) void bwd_grad_bf(const uint16_t* __restrict__ q,
                                                      const uint16_t* __restrict__ k,
                                                      const uint16_t* __restrict__ v,
                                                      const float* __restrict__ ab,
                                                      const unsigned char* __restrict__ frec,
                                                      const unsigned char* __restrict__ brec,
                                                      float* __restrict__ dq,
                                                      float* __restrict__ dk,
                                                      float* __restrict__ dvo, int T,
                                                      long long rec_bh) {
  extern __shared__ __align__(16) unsigned char gsm[];
  uint16_t* Qs = reinterpret_cast<uint16_t*>(gsm);
  uint16_t* Ks = reinterpret_cast<uint16_t*>(gsm + kBfOffK);
  uint16_t* Vs = reinterpret_cast<uint16_t*>(gsm + kBfOffV);  // column 64: 1 (valid rows)
  uint16_t* As = reinterpret_cast<uint16_t*>(gsm + kBfOffA);  // column 64: b_t
  uint16_t* Al = reinterpret_cast<uint16_t*>(gsm + kBfOffAl);  // a_t, b_t - (their bf16)
  uint16_t* slab = reinterpret_cast<uint16_t*>(gsm + kBfOffSlab);
  float* dqR = reinterpret_cast<float*>(gsm + kBfOffR);
  float* dkR = dqR + 64 * kBR;
  // in-chunk tiles, on the slab buffers before the first slab is staged
  uint16_t* QT = slab;
  uint16_t* KT = QT + kBT;
  uint16_t* AT = KT + kBT;
  uint16_t* Pm = AT + kBT;
  uint16_t* PmT = Pm + kBT;
  uint16_t* WT = PmT + kBT;

  // two groups of four waves: group g takes the slabs y = g, g + 2, ...
  const int c = blockIdx.x, bh = blockIdx.y, tid = threadIdx.x & 255;
  const int grp = __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x) >> 8);
  const int lane = tid & 63, w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int h = lane >> 5, l32 = lane & 31;
  const long long t0 = static_cast<long long>(c) * 64;
  const int nt = static_cast<int>(min(64LL, static_cast<long long>(T) - t0));
  const long long hb = static_cast<long long>(bh) * T;
  const unsigned char* Sp = frec + bh * rec_bh + static_cast<long long>(c) * kRecB;
  const unsigned char* Bs = brec + bh * rec_bh + static_cast<long long>(c) * kRecB;
  const int rg = tid >> 5, cp = tid & 31;  // staging: rows 8 rg + r, columns 2 cp, 2 cp + 1

  // record rows through buffer loads: the chunk's record as the resource, the
  // slab's first row as the scalar offset, row and column as the vector offset
  const __amdgpu_buffer_rsrc_t rS =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<unsigned char*>(Sp), 0, kRecB, kBfWord3);
  const __amdgpu_buffer_rsrc_t rB =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<unsigned char*>(Bs), 0, kRecB, kBfWord3);
  auto fetch = [&](BfSlabRegs& p, int y) {
    const int f0 = y * 64 - (y * (y - 1)) / 2;  // packed(y, y)
    const int so = f0 * 128;
#pragma unroll
    for (int r = 0; r < 8; ++r) {
      const int vo = max(8 * rg + r - y, 0) * 128 + 4 * cp;  // rows below y: row f0, staged 0
      p.a[r] = __builtin_amdgcn_raw_buffer_load_b32(rS, vo, so, 0);
      p.b[r] = __builtin_amdgcn_raw_buffer_load_b32(rB, vo, so, 0);
    }
    const int zo = max(lane - y, 0) * 4;
    p.za = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rS, zo, kRecSB + f0 * 4, 0));
    p.zb = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rB, zo, kRecSB + f0 * 4, 0));
  };
  auto stage = [&](const BfSlabRegs& p, int y, uint16_t* buf) {
    uint16_t* Ss = buf;
    uint16_t* Ds = buf + kBTW;
    uint16_t* DT = Ds + kBTW;
    // rows below y are zero; the diagonal row arrives halved from the scan
    uint32_t sa[8], sb[8];
#pragma unroll
    for (int r = 0; r < 8; ++r) {
      const int x = 8 * rg + r;
      sa[r] = x < y ? 0u : p.a[r];
      sb[r] = x < y ? 0u : p.b[r];
      *reinterpret_cast<uint32_t*>(Ss + x * kBW + 2 * cp) = sa[r];
      *reinterpret_cast<uint32_t*>(Ds + x * kBW + 2 * cp) = sb[r];
    }
    *reinterpret_cast<uint4*>(DT + (2 * cp) * kBP + 8 * rg) =
        make_uint4(lo_pair(sb[0], sb[1]), lo_pair(sb[2], sb[3]), lo_pair(sb[4], sb[5]),
                   lo_pair(sb[6], sb[7]));
    *reinterpret_cast<uint4*>(DT + (2 * cp + 1) * kBP + 8 * rg) =
        make_uint4(hi_pair(sb[0], sb[1]), hi_pair(sb[2], sb[3]), hi_pair(sb[4], sb[5]),
                   hi_pair(sb[6], sb[7]));
    if (w == 3) {  // z column and the zero columns 65..79 of row lane (wave 3
                   // stages every slab)
      const int x = lane;
      const float mz = x < y ? 0.f : 1.f;
      const uint4 zero = make_uint4(0u, 0u, 0u, 0u);
      *reinterpret_cast<uint4*>(Ss + x * kBW + 64) = make_uint4(pack_bf16x2(p.za * mz, 0.f), 0u, 0u, 0u);
      *reinterpret_cast<uint4*>(Ss + x * kBW + 72) = zero;
      *reinterpret_cast<uint4*>(Ds + x * kBW + 64) = make_uint4(pack_bf16x2(p.zb * mz, 0.f), 0u, 0u, 0u);
      *reinterpret_cast<uint4*>(Ds + x * kBW + 72) = zero;
    }
  };

  // ---- chunk rows: q, k, v, a (bf16) row-major and q, k, a transposed ----------
  if (grp == 0) {
    const uint16_t* qh = q + (hb + t0) * 64;
    const uint16_t* kh = k + (hb + t0) * 64;
    const uint16_t* vh = v + (hb + t0) * 64;
    const float* abh = ab + (hb + t0) * 65;
    uint32_t qv[8], kv[8], vv[8], av[8], al[8];
#pragma unroll
    for (int r = 0; r < 8; ++r) {
      const int t = 8 * rg + r;
      const int tc = min(t, nt - 1);
      const bool in = t < nt;
      const uint32_t q2 = *reinterpret_cast<const uint32_t*>(qh + tc * 64 + 2 * cp);
      const uint32_t k2 = *reinterpret_cast<const uint32_t*>(kh + tc * 64 + 2 * cp);
      const uint32_t v2 = *reinterpret_cast<const uint32_t*>(vh + tc * 64 + 2 * cp);
      const float a0 = abh[tc * 65 + 2 * cp], a1 = abh[tc * 65 + 2 * cp + 1];
      qv[r] = in ? q2 : 0u;
      kv[r] = in ? k2 : 0u;
      vv[r] = in ? v2 : 0u;
      av[r] = in ? pack_bf16x2(a0, a1) : 0u;
      al[r] = in ? pack_bf16x2(a0 - bf16lo_f32(av[r]), a1 - bf16hi_f32(av[r])) : 0u;
    }
    float bcol = 0.f;
    if (w == 0) bcol = abh[min(tid, nt - 1) * 65 + 64];
#pragma unroll
    for (int r = 0; r < 8; ++r) {
      const int t = 8 * rg + r;
      *reinterpret_cast<uint32_t*>(Qs + t * kBP + 2 * cp) = qv[r];
      *reinterpret_cast<uint32_t*>(Ks + t * kBP + 2 * cp) = kv[r];
      *reinterpret_cast<uint32_t*>(Vs + t * kBW + 2 * cp) = vv[r];
      *reinterpret_cast<uint32_t*>(As + t * kBW + 2 * cp) = av[r];
      *reinterpret_cast<uint32_t*>(Al + t * kBW + 2 * cp) = al[r];
    }
    auto put_t = [&](uint16_t* dst, const uint32_t* s) {
      *reinterpret_cast<uint4*>(dst + (2 * cp) * kBP + 8 * rg) =
          make_uint4(lo_pair(s[0], s[1]), lo_pair(s[2], s[3]), lo_pair(s[4], s[5]),
                     lo_pair(s[6], s[7]));
      *reinterpret_cast<uint4*>(dst + (2 * cp + 1) * kBP + 8 * rg) =
          make_uint4(hi_pair(s[0], s[1]), hi_pair(s[2], s[3]), hi_pair(s[4], s[5]),
                     hi_pair(s[6], s[7]));
    };
    put_t(QT, qv);
    put_t(KT, kv);
    put_t(AT, av);
    if (w == 0) {
      const bool in = tid < nt;
      const uint4 zero = make_uint4(0u, 0u, 0u, 0u);
      *reinterpret_cast<uint4*>(Vs + tid * kBW + 64) = make_uint4(in ? 0x3F80u : 0u, 0u, 0u, 0u);
      *reinterpret_cast<uint4*>(Vs + tid * kBW + 72) = zero;
      const uint32_t bh16 = in ? pack_bf16x2(bcol, 0.f) : 0u;
      const uint32_t bl16 = in ? pack_bf16x2(bcol - bf16lo_f32(bh16), 0.f) : 0u;
      *reinterpret_cast<uint4*>(As + tid * kBW + 64) = make_uint4(bh16, 0u, 0u, 0u);
      *reinterpret_cast<uint4*>(As + tid * kBW + 72) = zero;
      *reinterpret_cast<uint4*>(Al + tid * kBW + 64) = make_uint4(bl16, 0u, 0u, 0u);
      *reinterpret_cast<uint4*>(Al + tid * kBW + 72) = zero;
    }
  }
  // each group's first slab is on its way during the in-chunk terms
  BfSlabRegs pf0;
  fetch(pf0, grp);
  __syncthreads();

  // ---- in-chunk scores: wave w takes the (key tile w >> 1, token tile w & 1)
  // tile of Sc^T and Cw^T, then writes Pm, Pm^T and W^T (group 0) ---------------
  if (grp == 0) {
    const int S = w >> 1, Tt = w & 1;
    f32x16 sc = {}, cw = {};
#pragma unroll
    for (int ks = 0; ks < 4; ++ks)
      sc = mfma_bf(ld8(Ks + (32 * S + l32) * kBP + 16 * ks + 8 * h),
                   ld8(Qs + (32 * Tt + l32) * kBP + 16 * ks + 8 * h), sc);
#pragma unroll
    for (int ks = 0; ks < 5; ++ks) {
      const bf16x8 vf = ld8(Vs + (32 * S + l32) * kBW + 16 * ks + 8 * h);
      cw = mfma_bf(vf, ld8(As + (32 * Tt + l32) * kBW + 16 * ks + 8 * h), cw);
      cw = mfma_bf(vf, ld8(Al + (32 * Tt + l32) * kBW + 16 * ks + 8 * h), cw);
    }
    const int t = 32 * Tt + l32;
#pragma unroll
    for (int mq = 0; mq < 4; ++mq) {
      const int s0 = 32 * S + 8 * mq + 4 * h;
      float pm[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int i = 4 * mq + e, s = s0 + e;
        const bool live = s <= t;
        pm[e] = live ? 2.f * cw[i] * sc[i] : 0.f;
        const float wv = live ? sc[i] * sc[i] : 0.f;
        PmT[s * kBP + t] = bf_bits(pm[e]);
        WT[s * kBP + t] = bf_bits(wv);
      }
      *reinterpret_cast<uint2*>(Pm + t * kBP + s0) =
          make_uint2(pack_bf16x2(pm[0], pm[1]), pack_bf16x2(pm[2], pm[3]));
    }
  }
  __syncthreads();

  // ---- in-chunk products and the per-wave operands of the slab loop ------------
  // compute role: group 1 is rotated by two, so that each SIMD (wave w of
  // both groups) runs one dq wave and one dk wave (the dq side has twice the
  // slab MFMAs: a_t enters as hi + lo)
  const int role = (w + 2 * grp) & 3;
  const bool dqw = role < 2;
  const int Tw = role & 1;  // token tile (dq) / key tile (dk) / key tile of dv
  const int J = role >> 1;  // value tile of dv
  f32x16 acc0 = {}, acc1 = {}, dvacc = {};
  if (grp == 0) {
    const uint16_t* Xa = dqw ? KT : QT;
    const uint16_t* Xb = (dqw ? Pm : PmT) + (32 * Tw + l32) * kBP + 8 * h;
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      const bf16x8 bfrag = ld8(Xb + 16 * ks);
      acc0 = mfma_bf(ld8(Xa + l32 * kBP + 16 * ks + 8 * h), bfrag, acc0);
      acc1 = mfma_bf(ld8(Xa + (32 + l32) * kBP + 16 * ks + 8 * h), bfrag, acc1);
    }
#pragma unroll
    for (int ks = 0; ks < 4; ++ks)
      dvacc = mfma_bf(ld8(AT + (32 * J + l32) * kBP + 16 * ks + 8 * h),
                      ld8(WT + (32 * Tw + l32) * kBP + 16 * ks + 8 * h), dvacc);
  }
  bf16x8 bfr[5], bfl[5];  // a_t | b_t as hi, lo (dq) or v_i | 1 (dk) of this lane's row, K = 80
  {
    const uint16_t* src = (dqw ? As : Vs) + (32 * Tw + l32) * kBW + 8 * h;
    const uint16_t* srl = Al + (32 * Tw + l32) * kBW + 8 * h;
#pragma unroll
    for (int ks = 0; ks < 5; ++ks) {
      bfr[ks] = ld8(src + 16 * ks);
      bfl[ks] = ld8(srl + 16 * ks);
    }
  }
  const uint16_t* xrow = (dqw ? Qs : Ks) + (32 * Tw + l32) * kBP;  // q_t or k_i of this lane
  const uint16_t* krow = Ks + (32 * Tw + l32) * kBP;               // k_i of the dv column
  float* Rout = (dqw ? dqR : dkR) + (32 * Tw + l32) * kBR;
  float xr[2][16];  // x_t[x] (q or k of this lane's token) for its accumulator rows x
#pragma unroll
  for (int X = 0; X < 2; ++X)
#pragma unroll
    for (int i = 0; i < 16; ++i) xr[X][i] = bf_f32(xrow[32 * X + 8 * (i >> 2) + 4 * h + (i & 3)]);
  __syncthreads();  // the in-chunk tiles are dead: the slab buffers take over

  // x0: x tile 0 still holds rows x >= y (y < 32), a compile-time switch
  auto compute = [&](auto x0c, int y, const uint16_t* buf) {
    constexpr bool x0 = decltype(x0c)::value;
    const uint16_t* Sl = buf + (dqw ? 0 : kBTW);
    const uint16_t* DT = buf + 2 * kBTW;
    f32x16 P0 = {}, P1 = {}, Qy = {};
    if constexpr (x0) {
#pragma unroll
      for (int ks = 0; ks < 5; ++ks) {
        const bf16x8 sf = ld8(Sl + l32 * kBW + 16 * ks + 8 * h);
        P0 = mfma_bf(sf, bfr[ks], P0);
        if (dqw) P0 = mfma_bf(sf, bfl[ks], P0);
      }
    }
#pragma unroll
    for (int ks = 0; ks < 5; ++ks) {
      const bf16x8 sf = ld8(Sl + (32 + l32) * kBW + 16 * ks + 8 * h);
      P1 = mfma_bf(sf, bfr[ks], P1);
      if (dqw) P1 = mfma_bf(sf, bfl[ks], P1);
    }
#pragma unroll
    for (int ks = x0 ? 0 : 2; ks < 4; ++ks)  // rows below y are zero (all of x < 32 once y >= 32)
      Qy = mfma_bf(ld8(DT + (32 * J + l32) * kBP + 16 * ks + 8 * h), ld8(krow + 16 * ks + 8 * h), Qy);
    const float s2 = 2.f * bf_f32(xrow[y]);
    float R = 0.f;
    if constexpr (x0) {
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        acc0[i] += s2 * P0[i];
        R += xr[0][i] * P0[i];
      }
    }
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      acc1[i] += s2 * P1[i];
      R += xr[1][i] * P1[i];
    }
    R += __shfl_xor(R, 32);
    if (h == 0) Rout[y] = 2.f * R;
    const float ky = 2.f * bf_f32(krow[y]);  // DT holds dS with the diagonal halved
#pragma unroll
    for (int i = 0; i < 16; ++i) dvacc[i] += ky * Qy[i];
  };

  uint16_t* mybuf = slab + grp * (kBfSlab / 2);
  // wave w stages rows 16 w .. 16 w + 15; once the group's previous slab
  // (y - 2) has zeroed them all (16 w + 16 <= y - 2) they stay zero, and the
  // wave stages and fetches nothing more (wave 3 also stages z every slab)
  auto live = [&](int y) { return 16 * w + 18 > y; };
  for (int i = 0; i < 16; ++i) {
    const int y = 2 * i + grp;
    if (live(y)) {
      stage(pf0, y, mybuf);
      fetch(pf0, y + 2);
    }
    __syncthreads();
    compute(std::true_type{}, y, mybuf);
    __syncthreads();
  }
  for (int i = 16; i < 32; ++i) {
    const int y = 2 * i + grp;
    if (live(y)) {
      stage(pf0, y, mybuf);
      fetch(pf0, min(y + 2, 63));
    }
    __syncthreads();
    compute(std::false_type{}, y, mybuf);
    __syncthreads();
  }
  // group 1 hands its accumulators to group 0 through the (free) slab buffers
  float* red = reinterpret_cast<float*>(slab) + (role * 64 + lane) * 48;
  if (grp == 1) {
#pragma unroll
    for (int mq = 0; mq < 4; ++mq) {
      *reinterpret_cast<float4*>(red + 4 * mq) =
          make_float4(acc0[4 * mq], acc0[4 * mq + 1], acc0[4 * mq + 2], acc0[4 * mq + 3]);
      *reinterpret_cast<float4*>(red + 16 + 4 * mq) =
          make_float4(acc1[4 * mq], acc1[4 * mq + 1], acc1[4 * mq + 2], acc1[4 * mq + 3]);
      *reinterpret_cast<float4*>(red + 32 + 4 * mq) =
          make_float4(dvacc[4 * mq], dvacc[4 * mq + 1], dvacc[4 * mq + 2], dvacc[4 * mq + 3]);
    }
  }
  __syncthreads();
  if (grp == 1) return;
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    acc0[i] += red[i];
    acc1[i] += red[16 + i];
    dvacc[i] += red[32 + i];
  }

  // ---- outputs: accumulators plus the slab row sums ----------------------------
  {
    float* G = dqw ? dq : dk;
    const int tok = 32 * Tw + l32;
    const float* Rr = (dqw ? dqR : dkR) + tok * kBR;
    if (tok < nt) {
      float* g = G + (hb + t0 + tok) * 64;
#pragma unroll
      for (int mq = 0; mq < 4; ++mq) {
        const int xa = 8 * mq + 4 * h;
        const float4 r0 = *reinterpret_cast<const float4*>(Rr + xa);
        const float4 r1 = *reinterpret_cast<const float4*>(Rr + 32 + xa);
        *reinterpret_cast<float4*>(g + xa) =
            make_float4(acc0[4 * mq] + r0.x, acc0[4 * mq + 1] + r0.y, acc0[4 * mq + 2] + r0.z,
                        acc0[4 * mq + 3] + r0.w);
        *reinterpret_cast<float4*>(g + 32 + xa) =
            make_float4(acc1[4 * mq] + r1.x, acc1[4 * mq + 1] + r1.y, acc1[4 * mq + 2] + r1.z,
                        acc1[4 * mq + 3] + r1.w);
      }
    }
    if (tok < nt) {
      float* gv = dvo + (hb + t0 + tok) * 64 + 32 * J;
#pragma unroll
      for (int mq = 0; mq < 4; ++mq)
        *reinterpret_cast<float4*>(gv + 8 * mq + 4 * h) =
            make_float4(dvacc[4 * mq], dvacc[4 * mq + 1], dvacc[4 * mq + 2], dvacc[4 * mq + 3]);
    }
  }
}

// ---------------------------------------------------------------------------
// Chunk states on the bf16 matrix cores, d = dv = C = 64: for the packed
// pairs f = (a, b), a <= b (row-major upper triangle),
//   S[f][j] = sum_t x_ta x_tb y_tj,   z[f] = sum_t wt_t x_ta x_tb,
// written as one record per chunk: S rounded to bf16 (rows of 64, through a
// per-wave LDS tile so that a wave stores 32 whole rows), then z in fp32.  Forward states (kBwd =
// false): x = k, y = v, wt = 1.  Backward states (kBwd): x = q, y = a_t and
// wt = b_t from the coefficient rows; a_t enters as a bf16 pair hi + lo like
// in the gradients.  The feature products are exact in fp32 and rounded to
// bf16 once as the MFMA operand; z sums the fp32 products.  x and y are
// staged transposed ([dim][token], bf16), so a lane reads the eight tokens of
// its K slice with one 16-byte load.  Wave w takes the 32-feature tiles
// w, w + 4, ...  grid (NC, BH), block 256.
// ---------------------------------------------------------------------------
template <bool kBwd>
__global__ __launch_bounds__(256) void bwd_state_bf(const uint16_t* __restrict__ x,
                                                    const void* __restrict__ yv,
                                                    unsigned char* __restrict__ rec, int T,
                                                    long long rec_bh) {
  __shared__ __align__(16) uint16_t ot[4 * 32 * kBP];  // per-wave output rows
  __shared__ __align__(16) uint16_t xT[64 * kBP];
  __shared__ __align__(16) uint16_t yT[64 * kBP];
  __shared__ __align__(16) uint16_t yL[kBwd ? 64 * kBP : 8];
  __shared__ __align__(16) float wt[64];
  __shared__ uint16_t pairs[kBfN];
  const int c = blockIdx.x, bh = blockIdx.y, tid = threadIdx.x;
  const int lane = tid & 63, w = tid >> 6, h = lane >> 5, l32 = lane & 31;
  const long long t0 = static_cast<long long>(c) * 64;
  const int nt = static_cast<int>(min(64LL, static_cast<long long>(T) - t0));
  const long long hb = static_cast<long long>(bh) * T;
  for (int a = tid; a < 64; a += 256)
    for (int b = a; b < 64; ++b)
      pairs[a * 64 - a * (a - 1) / 2 + (b - a)] = static_cast<uint16_t>(a | (b << 8));
  {
    const int rg = tid >> 5, cp = tid & 31;  // rows 8 rg + r, columns 2 cp, 2 cp + 1
    const uint16_t* xh = x + (hb + t0) * 64;
    uint32_t xv[8], yh[8], yl[8];
#pragma unroll
    for (int r = 0; r < 8; ++r) {
      const int t = 8 * rg + r, tc = min(t, nt - 1);
      const bool in = t < nt;
      const uint32_t x2 = *reinterpret_cast<const uint32_t*>(xh + tc * 64 + 2 * cp);
      xv[r] = in ? x2 : 0u;
      if constexpr (kBwd) {
        const float* ar = static_cast<const float*>(yv) + (hb + t0 + tc) * 65;
        const float a0 = ar[2 * cp], a1 = ar[2 * cp + 1];
        const uint32_t hi = pack_bf16x2(a0, a1);
        yh[r] = in ? hi : 0u;
        yl[r] = in ? pack_bf16x2(a0 - bf16lo_f32(hi), a1 - bf16hi_f32(hi)) : 0u;
      } else {
        const uint16_t* vh = static_cast<const uint16_t*>(yv) + (hb + t0) * 64;
        const uint32_t v2 = *reinterpret_cast<const uint32_t*>(vh + tc * 64 + 2 * cp);
        yh[r] = in ? v2 : 0u;
        yl[r] = 0u;
      }
    }
    auto put_t = [&](uint16_t* dst, const uint32_t* s2) {
      *reinterpret_cast<uint4*>(dst + (2 * cp) * kBP + 8 * rg) =
          make_uint4(lo_pair(s2[0], s2[1]), lo_pair(s2[2], s2[3]), lo_pair(s2[4], s2[5]),
                     lo_pair(s2[6], s2[7]));
      *reinterpret_cast<uint4*>(dst + (2 * cp + 1) * kBP + 8 * rg) =
          make_uint4(hi_pair(s2[0], s2[1]), hi_pair(s2[2], s2[3]), hi_pair(s2[4], s2[5]),
                     hi_pair(s2[6], s2[7]));
    };
    put_t(xT, xv);
    put_t(yT, yh);
    if constexpr (kBwd) put_t(yL, yl);
    if (tid < 64) {
      float b = 1.f;
      if constexpr (kBwd)
        b = tid < nt ? static_cast<const float*>(yv)[(hb + t0 + tid) * 65 + 64] : 0.f;
      wt[tid] = b;
    }
  }
  __syncthreads();
  unsigned char* r0 = rec + bh * rec_bh + static_cast<long long>(c) * kRecB;
  uint16_t* ow = ot + w * 32 * kBP;
  for (int ft = w; ft < kBfN / 32; ft += 4) {
    const int f = 32 * ft + l32;
    const int pa = pairs[f] & 0xFF, pb = pairs[f] >> 8;
    f32x16 acc0 = {}, acc1 = {};
    float zp = 0.f;
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      const int tk = 16 * ks + 8 * h;
      const uint4 xa = *reinterpret_cast<const uint4*>(xT + pa * kBP + tk);
      const uint4 xb = *reinterpret_cast<const uint4*>(xT + pb * kBP + tk);
      const uint32_t wa[4] = {xa.x, xa.y, xa.z, xa.w}, wb[4] = {xb.x, xb.y, xb.z, xb.w};
      uint32_t pk[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float p0 = bf16lo_f32(wa[e]) * bf16lo_f32(wb[e]);
        const float p1 = bf16hi_f32(wa[e]) * bf16hi_f32(wb[e]);
        pk[e] = pack_bf16x2(p0, p1);
        if constexpr (kBwd)  // padded tokens have x = 0 and wt = 0
          zp += wt[tk + 2 * e] * p0 + wt[tk + 2 * e + 1] * p1;
        else
          zp += p0 + p1;
      }
      const bf16x8 A = __builtin_bit_cast(bf16x8, make_uint4(pk[0], pk[1], pk[2], pk[3]));
      acc0 = mfma_bf(A, ld8(yT + l32 * kBP + tk), acc0);
      acc1 = mfma_bf(A, ld8(yT + (32 + l32) * kBP + tk), acc1);
      if constexpr (kBwd) {
        acc0 = mfma_bf(A, ld8(yL + l32 * kBP + tk), acc0);
        acc1 = mfma_bf(A, ld8(yL + (32 + l32) * kBP + tk), acc1);
      }
    }
    zp += __shfl_xor(zp, 32);
    // the tile's 32 rows as bf16 into this wave's LDS rows, then 16-byte
    // pieces of whole rows to HBM (a wave's LDS accesses complete in order)
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int r = 8 * (i >> 2) + 4 * h + (i & 3);
      ow[r * kBP + l32] = bf_bits(acc0[i]);
      ow[r * kBP + 32 + l32] = bf_bits(acc1[i]);
    }
#pragma unroll
    for (int q4 = 0; q4 < 4; ++q4) {
      const int ch = lane + 64 * q4, r = ch >> 3, part = ch & 7;
      *reinterpret_cast<uint4*>(r0 + static_cast<long long>(32 * ft + r) * 128 + 16 * part) =
          *reinterpret_cast<const uint4*>(ow + r * kBP + 8 * part);
    }
    if (h == 0) reinterpret_cast<float*>(r0 + kRecSB)[f] = zp;
  }
}

// ---------------------------------------------------------------------------
// Exclusive prefix (or, kReverse, suffix) over the chunk records of this path,
// in place: record c receives w(e) x the sum over the records before (after)
// it, summed in fp32; S elements are read and written as bf16, z as fp32, and
// w = 1/2 on the diagonal features (a, a), 1 elsewhere.  A thread takes one
// 16-byte piece of the record (8 bf16 of S or 4 fp32 of z) in kSR consecutive
// records of a kSG x kSR-record block: an up- and down-sweep in registers, then
// the kSG row groups of the workgroup join their block sums through LDS (kSR
// shrinks for short sequences so that every row group has records).  The S / z
// boundary falls on a workgroup boundary (kRecS16 is a multiple of kSC).
// grid (ceil(kRec16 / kSC), BH), block kSC x kSG.
// ---------------------------------------------------------------------------
constexpr int kSC = 32;  // 16-byte pieces per workgroup (512 contiguous bytes of a record)
constexpr int kSG = 2;   // row groups (one wave per workgroup: measured fastest)
static_assert(kRecS16 % kSC == 0, "a workgroup reads one element type");

// Whether packed index f (0 <= f < 2080) is a diagonal pair: f = D(a) =
// 64 a - a (a - 1) / 2 for the row a with D(a) <= f < D(a + 1), which solves
// a^2 - 129 a + 2 f = 0 (the square root estimate is corrected by one either
// way, then checked exactly).
__device__ __forceinline__ bool diag_feature(int f) {
  auto D = [](int a) { return 64 * a - a * (a - 1) / 2; };
  int a = static_cast<int>((129.f - sqrtf(16641.f - 8.f * static_cast<float>(f))) * 0.5f);
  a = max(0, min(63, a));
  if (a < 63 && D(a + 1) <= f) ++a;
  if (a > 0 && D(a) > f) --a;
  return D(a) == f;
}

// Every record piece is read once and written once per scan, so both go past
// the caches (non-temporal).  With the one-wave, 512-byte workgroup shape above
// a scan at B8 H16 T4096 measured 0.79 ms, against 0.94 ms with cached access
// and 16 x 8 workgroups.
typedef unsigned scan_u4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ uint4 stream_load_u4(const unsigned char* p) {
  const scan_u4 t = __builtin_nontemporal_load(reinterpret_cast<const scan_u4*>(p));
  return make_uint4(t.x, t.y, t.z, t.w);
}
__device__ __forceinline__ void stream_store_u4(unsigned char* p, uint4 u) {
  const scan_u4 t = {u.x, u.y, u.z, u.w};
  __builtin_nontemporal_store(t, reinterpret_cast<scan_u4*>(p));
}

template <bool kReverse, int kSR>
__global__ __launch_bounds__(kSC * kSG) void scan_bf(unsigned char* __restrict__ rec, int N,
                                               long long rec_bh) {
  __shared__ float4 tot[kSG][kSC][2];
  const int tid = threadIdx.x, cg = tid % kSC, rg = tid / kSC;
  const int pc = blockIdx.x * kSC + cg;
  const bool active = pc < kRec16;
  const bool isS = blockIdx.x * kSC < kRecS16;  // uniform over the workgroup
  unsigned char* rb = rec + blockIdx.y * rec_bh + 16LL * pc;
  float w[8], carry[8];
  if (isS) {
    const float wv = diag_feature(pc >> 3) ? 0.5f : 1.f;  // 8 pieces per 64-wide row
#pragma unroll
    for (int x = 0; x < 8; ++x) w[x] = wv;
  } else {
    const int zf = 4 * (pc - kRecS16);
#pragma unroll
    for (int x = 0; x < 8; ++x) w[x] = (x < 4 && diag_feature(zf + x)) ? 0.5f : 1.f;
  }
#pragma unroll
  for (int x = 0; x < 8; ++x) carry[x] = 0.f;
  for (int r0 = 0; r0 < N; r0 += kSG * kSR) {
    const int rbase = r0 + rg * kSR;
    float v[kSR][8];
#pragma unroll
    for (int j = 0; j < kSR; ++j) {
      const int rr = rbase + j;
      uint4 u = make_uint4(0u, 0u, 0u, 0u);
      if (active && rr < N)
        u = stream_load_u4(rb + static_cast<long long>(kReverse ? N - 1 - rr : rr) * kRecB);
      const uint32_t uw[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        if (isS) {
          v[j][2 * e] = bf16lo_f32(uw[e]);
          v[j][2 * e + 1] = bf16hi_f32(uw[e]);
        } else {
          v[j][e] = __uint_as_float(uw[e]);
          v[j][4 + e] = 0.f;
        }
      }
    }
#pragma unroll
    for (int d = 1; d < kSR; d <<= 1)
#pragma unroll
      for (int j = 2 * d - 1; j < kSR; j += 2 * d)
#pragma unroll
        for (int x = 0; x < 8; ++x) v[j][x] += v[j - d][x];
    float gsum[8];
#pragma unroll
    for (int x = 0; x < 8; ++x) {
      gsum[x] = v[kSR - 1][x];
      v[kSR - 1][x] = 0.f;
    }
#pragma unroll
    for (int d = kSR / 2; d >= 1; d >>= 1)
#pragma unroll
      for (int j = 2 * d - 1; j < kSR; j += 2 * d)
#pragma unroll
        for (int x = 0; x < 8; ++x) {
          const float left = v[j - d][x];
          v[j - d][x] = v[j][x];
          v[j][x] += left;
        }
    tot[rg][cg][0] = make_float4(gsum[0], gsum[1], gsum[2], gsum[3]);
    tot[rg][cg][1] = make_float4(gsum[4], gsum[5], gsum[6], gsum[7]);
    __syncthreads();
    float pre[8], blk[8];
#pragma unroll
    for (int x = 0; x < 8; ++x) {
      pre[x] = carry[x];
      blk[x] = 0.f;
    }
#pragma unroll
    for (int g2 = 0; g2 < kSG; ++g2) {
      const float4 t0 = tot[g2][cg][0], t1 = tot[g2][cg][1];
      const float tv[8] = {t0.x, t0.y, t0.z, t0.w, t1.x, t1.y, t1.z, t1.w};
#pragma unroll
      for (int x = 0; x < 8; ++x) {
        if (g2 < rg) pre[x] += tv[x];
        blk[x] += tv[x];
      }
    }
    __syncthreads();  // tot is rewritten by the next block
#pragma unroll
    for (int j = 0; j < kSR; ++j) {
      const int rr = rbase + j;
      if (!(active && rr < N)) continue;
      float o[8];
#pragma unroll
      for (int x = 0; x < 8; ++x) o[x] = w[x] * (pre[x] + v[j][x]);
      const uint4 u = isS ? make_uint4(pack_bf16x2(o[0], o[1]), pack_bf16x2(o[2], o[3]),
                                       pack_bf16x2(o[4], o[5]), pack_bf16x2(o[6], o[7]))
                          : make_uint4(__float_as_uint(o[0]), __float_as_uint(o[1]),
                                       __float_as_uint(o[2]), __float_as_uint(o[3]));
      stream_store_u4(rb + static_cast<long long>(kReverse ? N - 1 - rr : rr) * kRecB, u);
    }
#pragma unroll
    for (int x = 0; x < 8; ++x) carry[x] += blk[x];
  }
}

// ---------------------------------------------------------------------------
// Chunk-state prefixes in one pass (state and exclusive scan fused), on the
// bf16 matrix cores, d = dv = C = 64: record c receives w(f) x the sum of the
// chunk states S_c'[f][j] = sum_t x_ta x_tb y_tj, z_c'[f] = sum_t wt_t x_ta x_tb
// over the chunks c' < c (or, kBwd, c' > c), w = 1/2 on the diagonal features
// (a, a); S rounded to bf16 once from the fp32 running sum, z in fp32.  Forward
// (kBwd = false): x = k, y = v, wt = 1.  Backward (kBwd): x = q, y = a_t as a
// bf16 pair hi + lo, wt = b_t from the coefficient rows.
// Wave w of workgroup tg owns the kTW 32-feature tiles kTW (kPW tg + w) + u of
// one head (tiles past the 65th are skipped; a wave with none only stages)
// and walks the head's chunks in scan order with the running sums of its tiles
// in registers: per chunk it writes each running sum as the record (the
// exclusive prefix), then adds the chunk's state.  Two tiles per wave give two
// independent MFMA chains and share the y operands.  Each chunk's x and y are
// staged in LDS once per workgroup, transposed ([dim][token]), by all four
// waves (one per SIMD, so that every SIMD carries the same work), and the next
// chunks' rows are loaded into registers while the current one is
// contracted.  The kPG workgroups of a
// head read the same rows: they are given workgroup ids of one residue mod 8,
// which the dispatcher sends to one XCD, so the rows come from that XCD's L2.
// The records are written past the caches (non-temporal): only later launches
// read them, and cached they would evict from L2 the rows that the head's
// other workgroups are about to read.  grid (kPG x 8 ceil(BH / 8)), block 64 kPW.
// ---------------------------------------------------------------------------
constexpr int kPW = 4;                        // waves per workgroup
constexpr int kTW = 2;                        // feature tiles per wave
constexpr int kPT = kBfN / 32;                // feature tiles per record
constexpr int kPG = (kPT + kPW * kTW - 1) / (kPW * kTW);  // workgroups per head
static_assert(kPT * 32 == kBfN && kPW * 64 == 256, "tiles of 32 features; 256 stagers");

// Raw rows of one chunk held in registers between their loads and their
// staging (converted only when staged, so that the loads stay in flight over
// the contractions in between).
template <bool kBwd>
struct PrefixRaw {
  uint32_t x[8];
  uint32_t y[kBwd ? 1 : 8];
  float a[kBwd ? 16 : 1];
  float b;
};

template <bool kBwd>
__global__ __launch_bounds__(64 * kPW) void bwd_prefix_bf(const uint16_t* __restrict__ x,
                                                          const void* __restrict__ yv,
                                                          unsigned char* __restrict__ rec,
                                                          int T, int BH, long long rec_bh) {
  constexpr int kTile = 64 * kBP;                   // one staged 64 x 64 tile
  constexpr int kBuf = (kBwd ? 3 : 2) * kTile;      // x, y (and the y residue) of a chunk
  __shared__ __align__(16) uint16_t ot[kPW * 32 * kBP];  // per-wave output rows
  __shared__ __align__(16) uint16_t tiles[2 * kBuf];     // two chunks in flight
  __shared__ __align__(16) float wts[2][64];
  const int id = blockIdx.x, jx = id >> 3;
  const int bh = 8 * (jx / kPG) + (id & 7), tg = jx % kPG;
  if (bh >= BH) return;  // the whole workgroup
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, h = lane >> 5, l32 = lane & 31;
  const int NC = (T + 63) / 64;
  const long long hb = static_cast<long long>(bh) * T;
  const int ft0 = kTW * (kPW * tg + w);
  const int nlive = max(0, min(kTW, kPT - ft0));  // tiles of this wave (wave-uniform)
  int ft[kTW], f[kTW], pa[kTW], pb[kTW];
  uint32_t dmask[kTW];
  float wz[kTW];
#pragma unroll
  for (int u = 0; u < kTW; ++u) {
    ft[u] = min(ft0 + u, kPT - 1);
    f[u] = 32 * ft[u] + l32;
    // the pair (pa, pb) of feature f: the row pa of the upper triangle with
    // D(pa) <= f < D(pa + 1), D(a) = 64 a - a (a - 1) / 2
    int a = 0;
    while (a < 63 && 64 * (a + 1) - (a + 1) * a / 2 <= f[u]) ++a;
    pa[u] = a;
    pb[u] = a + f[u] - (64 * a - a * (a - 1) / 2);
    // diagonal features of the tile, one bit per lane's feature
    dmask[u] = static_cast<uint32_t>(__ballot(pa[u] == pb[u]));
    wz[u] = pa[u] == pb[u] ? 0.5f : 1.f;
  }
  // staging: thread tid takes rows 8 rg .. 8 rg + 7, columns 2 cp, 2 cp + 1
  const int rg = tid >> 5, cp = tid & 31;
  auto chunk = [&](int it) { return kBwd ? NC - 1 - it : it; };
  // rows through buffer loads: one resource per chunk whose range ends at the
  // chunk's last valid row, so rows past the sequence's end read as zero, and
  // one 32-bit lane offset plus the row number (an immediate) per row
  const uint32_t xo = static_cast<uint32_t>(2 * (8 * rg * 64 + 2 * cp));
  const uint32_t ao = static_cast<uint32_t>(4 * (8 * rg * 65 + 2 * cp));
  auto fetch = [&](PrefixRaw<kBwd>& R, int c) {
    const long long t0 = static_cast<long long>(c) * 64;
    const int nt = static_cast<int>(min(64LL, static_cast<long long>(T) - t0));
    const __amdgpu_buffer_rsrc_t rx = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint16_t*>(x + (hb + t0) * 64), 0, nt * 128, kBfWord3);
    if constexpr (kBwd) {
      const __amdgpu_buffer_rsrc_t ra = __builtin_amdgcn_make_buffer_rsrc(
          const_cast<float*>(static_cast<const float*>(yv) + (hb + t0) * 65), 0, nt * 260,
          kBfWord3);
#pragma unroll
      for (int r = 0; r < 8; ++r) {
        R.x[r] = __builtin_amdgcn_raw_buffer_load_b32(rx, xo + 128 * r, 0, 0);
        R.a[2 * r] = __builtin_bit_cast(
            float, __builtin_amdgcn_raw_buffer_load_b32(ra, ao + 260 * r, 0, 0));
        R.a[2 * r + 1] = __builtin_bit_cast(
            float, __builtin_amdgcn_raw_buffer_load_b32(ra, ao + 260 * r + 4, 0, 0));
      }
      if (tid < 64)
        R.b = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(ra, 260 * tid + 256,
                                                                             0, 0));
    } else {
      const __amdgpu_buffer_rsrc_t ry = __builtin_amdgcn_make_buffer_rsrc(
          const_cast<uint16_t*>(static_cast<const uint16_t*>(yv) + (hb + t0) * 64), 0, nt * 128,
          kBfWord3);
#pragma unroll
      for (int r = 0; r < 8; ++r) {
        R.x[r] = __builtin_amdgcn_raw_buffer_load_b32(rx, xo + 128 * r, 0, 0);
        R.y[r] = __builtin_amdgcn_raw_buffer_load_b32(ry, xo + 128 * r, 0, 0);
      }
    }
  };
  auto put_t = [&](uint16_t* dst, const uint32_t* s2) {
    *reinterpret_cast<uint4*>(dst + (2 * cp) * kBP + 8 * rg) =
        make_uint4(lo_pair(s2[0], s2[1]), lo_pair(s2[2], s2[3]), lo_pair(s2[4], s2[5]),
                   lo_pair(s2[6], s2[7]));
    *reinterpret_cast<uint4*>(dst + (2 * cp + 1) * kBP + 8 * rg) =
        make_uint4(hi_pair(s2[0], s2[1]), hi_pair(s2[2], s2[3]), hi_pair(s2[4], s2[5]),
                   hi_pair(s2[6], s2[7]));
  };
  auto stage = [&](const PrefixRaw<kBwd>& R, int buf) {
    uint32_t xv[8], yh[8], yl[8];
#pragma unroll
    for (int r = 0; r < 8; ++r) {
      xv[r] = R.x[r];
      if constexpr (kBwd) {
        yh[r] = pack_bf16x2(R.a[2 * r], R.a[2 * r + 1]);
        yl[r] = pack_bf16x2(R.a[2 * r] - bf16lo_f32(yh[r]), R.a[2 * r + 1] - bf16hi_f32(yh[r]));
      } else {
        yh[r] = R.y[r];
        yl[r] = 0u;
      }
    }

    uint16_t* tb = tiles + buf * kBuf;
    put_t(tb, xv);
    put_t(tb + kTile, yh);
    if constexpr (kBwd) put_t(tb + 2 * kTile, yl);
    if constexpr (kBwd)
      if (tid < 64) wts[buf][tid] = R.b;  // zero past the sequence's end
  };
  f32x16 run0[kTW], run1[kTW];
  float zrun[kTW];
#pragma unroll
  for (int u = 0; u < kTW; ++u) {
    run0[u] = f32x16{};
    run1[u] = f32x16{};
    zrun[u] = 0.f;
  }
  uint16_t* ow = ot + w * 32 * kBP;
  unsigned char* rh = rec + bh * rec_bh;
  // record c = the running sum of tile u (w = 1/2 on diagonal features), as
  // whole bf16 rows through this wave's LDS rows (a wave's LDS accesses
  // complete in order).  The running sums are the transposed tile: lane
  // (l32, h) holds feature f's values j = 8 g + 4 h + 0..3 (run0) and 32 +
  // those (run1), four consecutive bf16 of the record row per group g.
  auto put_record = [&](unsigned char* r0, int u) {
    auto put_row = [&](float sc) {
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        *reinterpret_cast<uint2*>(ow + l32 * kBP + 8 * g + 4 * h) =
            make_uint2(pack_bf16x2(sc * run0[u][4 * g], sc * run0[u][4 * g + 1]),
                       pack_bf16x2(sc * run0[u][4 * g + 2], sc * run0[u][4 * g + 3]));
        *reinterpret_cast<uint2*>(ow + l32 * kBP + 32 + 8 * g + 4 * h) =
            make_uint2(pack_bf16x2(sc * run1[u][4 * g], sc * run1[u][4 * g + 1]),
                       pack_bf16x2(sc * run1[u][4 * g + 2], sc * run1[u][4 * g + 3]));
      }
    };
    if (dmask[u] != 0u)
      put_row(wz[u]);
    else
      put_row(1.f);  // no diagonal feature in this tile: no weight
#pragma unroll
    for (int q4 = 0; q4 < 4; ++q4) {
      const int ch = lane + 64 * q4, r = ch >> 3, part = ch & 7;
      stream_store_u4(r0 + static_cast<long long>(32 * ft[u] + r) * 128 + 16 * part,
                      *reinterpret_cast<const uint4*>(ow + r * kBP + 8 * part));
    }
    if (h == 0) reinterpret_cast<float*>(r0 + kRecSB)[f[u]] = wz[u] * zrun[u];
  };
  // chunk it: write its records (the running sums), then add its state
  auto step = [&](int it) {
    if (nlive == 0) return;
    const int c = chunk(it), buf = it & 1;
    unsigned char* r0 = rh + static_cast<long long>(c) * kRecB;
    put_record(r0, 0);
    if (nlive == kTW) put_record(r0, 1);
    const uint16_t* xT = tiles + buf * kBuf;
    const uint16_t* yT = xT + kTile;
    const uint16_t* yL = xT + 2 * kTile;
    const float* wt = wts[buf];
    float zp[kTW] = {};
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      const int tk = 16 * ks + 8 * h;
      // the y rows j = l32 and 32 + l32 of this K step, shared by the tiles
      const bf16x8 y0 = ld8(yT + l32 * kBP + tk), y1 = ld8(yT + (32 + l32) * kBP + tk);
      bf16x8 l0, l1;
      if constexpr (kBwd) {
        l0 = ld8(yL + l32 * kBP + tk);
        l1 = ld8(yL + (32 + l32) * kBP + tk);
      }
#pragma unroll
      for (int u = 0; u < kTW; ++u) {
        const uint4 xa = *reinterpret_cast<const uint4*>(xT + pa[u] * kBP + tk);
        const uint4 xb = *reinterpret_cast<const uint4*>(xT + pb[u] * kBP + tk);
        const uint32_t wa[4] = {xa.x, xa.y, xa.z, xa.w}, wb[4] = {xb.x, xb.y, xb.z, xb.w};
        uint32_t pk[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float p0 = bf16lo_f32(wa[e]) * bf16lo_f32(wb[e]);
          const float p1 = bf16hi_f32(wa[e]) * bf16hi_f32(wb[e]);
          pk[e] = pack_bf16x2(p0, p1);
          if constexpr (kBwd)  // padded tokens: wt = 0
            zp[u] += wt[tk + 2 * e] * p0 + wt[tk + 2 * e + 1] * p1;
          else  // padded tokens: x = 0
            zp[u] += p0 + p1;
        }
        // S^T tile: rows j of y (A operand), columns the 32 features (B operand)
        const bf16x8 P = __builtin_bit_cast(bf16x8, make_uint4(pk[0], pk[1], pk[2], pk[3]));
        run0[u] = mfma_bf(y0, P, run0[u]);
        run1[u] = mfma_bf(y1, P, run1[u]);
        if constexpr (kBwd) {
          run0[u] = mfma_bf(l0, P, run0[u]);
          run1[u] = mfma_bf(l1, P, run1[u]);
        }
      }
    }
#pragma unroll
    for (int u = 0; u < kTW; ++u) zrun[u] += zp[u] + __shfl_xor(zp[u], 32);
  };
  // Chunk it + 1 is staged (LDS buffer (it + 1) & 1) while chunk it is
  // contracted from the other buffer, and the loads of chunk it + 1 + kAhead
  // are issued into the register set just staged: kAhead chunks' loads are in
  // flight (two for the forward states; one for the backward states, whose
  // fp32 a_t rows take twice the registers).  One LDS-only barrier per chunk;
  // the record stores and the loads stay in flight across it.
  constexpr int kAhead = kBwd ? 1 : 2;
  PrefixRaw<kBwd> Ra, Rb_;
  PrefixRaw<kBwd>& R0 = Ra;
  PrefixRaw<kBwd>& R1 = kAhead == 2 ? Rb_ : Ra;
  // Every fetch is issued, past the last chunk as a repeat of it (its values
  // are never staged): with the same loads on every path the compiler's wait
  // before each staging counts exactly the loads and stores issued after it.
  auto ahead = [&](int it) { return chunk(min(it, NC - 1)); };
  fetch(R0, chunk(0));
  stage(R0, 0);
  fetch(R1, ahead(1));
  if (kAhead == 2) fetch(R0, ahead(2));
  lds_barrier();
  for (int it = 0; it < NC; it += 2) {
    if (it + 1 < NC) stage(R1, 1);
    fetch(R1, ahead(it + 1 + kAhead));
    step(it);
    lds_barrier();  // buffer 0 is read by every wave; buffer 1 is staged
    if (it + 1 >= NC) break;
    if (it + 2 < NC) stage(R0, 0);
    fetch(R0, ahead(it + 2 + kAhead));
    step(it + 1);
    lds_barrier();
  }
}

}  // namespace

bool bwd_bf_ok(int d, int dv, int C, int g) { return d == 64 && dv == 64 && C == 64 && g == 1; }

size_t bwd_bf_record_bytes() { return kRecB; }

hipError_t launch_bwd_state_bf(bool backward, const void* x, const void* y, void* rec, int BH,
                               int T, hipStream_t st) {
  const int NC = (T + 63) / 64;
  const long long rec_bh = static_cast<long long>(NC) * kRecB;
  unsigned char* r = static_cast<unsigned char*>(rec);
  if (backward)
    bwd_state_bf<true><<<dim3(NC, BH), 256, 0, st>>>(static_cast<const uint16_t*>(x), y, r, T,
                                                     rec_bh);
  else
    bwd_state_bf<false><<<dim3(NC, BH), 256, 0, st>>>(static_cast<const uint16_t*>(x), y, r, T,
                                                      rec_bh);
  return hipGetLastError();
}

hipError_t launch_bwd_scan_bf(bool reverse, void* rec, int BH, int T, hipStream_t st) {
  const int NC = (T + 63) / 64;
  const long long rec_bh = static_cast<long long>(NC) * kRecB;
  const dim3 grid((kRec16 + kSC - 1) / kSC, BH);
  unsigned char* r = static_cast<unsigned char*>(rec);
  auto go = [&](auto rows) {
    constexpr int R = decltype(rows)::value;
    if (reverse)
      scan_bf<true, R><<<grid, kSC * kSG, 0, st>>>(r, NC, rec_bh);
    else
      scan_bf<false, R><<<grid, kSC * kSG, 0, st>>>(r, NC, rec_bh);
  };
  if (NC >= 8 * kSG)
    go(std::integral_constant<int, 8>{});
  else if (NC >= 4 * kSG)
    go(std::integral_constant<int, 4>{});
  else if (NC >= 2 * kSG)
    go(std::integral_constant<int, 2>{});
  else
    go(std::integral_constant<int, 1>{});
  return hipGetLastError();
}

// The fused launches run 9 workgroups per head, each sequential over the
// head's chunks, so their time hardly depends on the head count until the
// chip is full: forward + backward record streams at T = 4096 take 0.29 ms
// fused from 4 to 16 heads, while the chunk-parallel state launches and
// scans take 0.18 ms at 8 heads and 0.36 ms at 16 (0.43 against 0.67 ms at 32
// heads, 0.54 against 0.97 ms at 48).
int bwd_bf_fused_min_heads() { return 16; }

hipError_t launch_bwd_prefix_bf(bool backward, const void* x, const void* y, void* rec, int BH,
                                int T, hipStream_t st) {
  const int NC = (T + 63) / 64;
  const long long rec_bh = static_cast<long long>(NC) * kRecB;
  const unsigned grid = static_cast<unsigned>(kPG * 8 * ((BH + 7) / 8));
  unsigned char* r = static_cast<unsigned char*>(rec);
  const uint16_t* xs = static_cast<const uint16_t*>(x);
  if (backward)
    bwd_prefix_bf<true><<<grid, 64 * kPW, 0, st>>>(xs, y, r, T, BH, rec_bh);
  else
    bwd_prefix_bf<false><<<grid, 64 * kPW, 0, st>>>(xs, y, r, T, BH, rec_bh);
  return hipGetLastError();
}

hipError_t launch_bwd_grad_bf(const void* q, const void* k, const void* v, const float* ab,
                              const void* frec, const void* brec, float* dq, float* dk,
                              float* dv_out, int BH, int T, hipStream_t st) {
  const int NC = (T + 63) / 64;
  const long long rec_bh = static_cast<long long>(NC) * kRecB;
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&bwd_grad_bf),
                                     hipFuncAttributeMaxDynamicSharedMemorySize, kBfLds);
  if (e != hipSuccess) return e;
  bwd_grad_bf<<<dim3(NC, BH), 512, kBfLds, st>>>(
      static_cast<const uint16_t*>(q), static_cast<const uint16_t*>(k),
      static_cast<const uint16_t*>(v), ab, static_cast<const unsigned char*>(frec),
      static_cast<const unsigned char*>(brec), dq, dk, dv_out, T, rec_bh);
  return hipGetLastError();
}

}  // namespace kata
