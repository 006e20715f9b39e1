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
// operands that are not bf16 already (the prefix and suffix records, the
// in-chunk score products) are rounded to bf16 once, when staged in LDS.  The
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
// (the row-major upper triangle), with z (dz) as a 65th column and the
// diagonal row halved.  For the query side, with G_t[{y,x}] =
// S[{y,x}] . a_t + b_t z[{y,x}],
//   P^T[x][t] = sum_j S_slab[x][j] a_t[j] + z_slab[x] b_t          (MFMA, K = 80)
//   dq^T[x][t] += 2 q_t[y] P^T[x][t]                 (pair {x,y}, coordinate x)
//   dq[t][y]   += 2 sum_x q_t[x] P^T[x][t]           (pair {x,y}, coordinate y)
// which together count every off-diagonal pair from both sides and the
// diagonal pair once (the halving).  The key side is the same with the suffix
// record, v_i and a unit coefficient for dz.  The value gradient takes the
// slab transposed, DT[j][x] = 2 dS_slab[x][j] (weights 1 on the diagonal, 2
// off it, 0 below):
//   dv^T[j][i] += k_i[y] sum_x DT[j][x] k_i[x].
// Waves: 0-1 own dq of token tile w, 2-3 dk of key tile w - 2, and every wave
// one 32 x 32 tile (value tile w >> 1, key tile w & 1) of dv.  The record rows
// of the next slab are fetched into registers (buffer loads) while the current
// one is used, and the slabs are double-buffered in LDS, so one barrier per
// slab orders staging and use.  grid (NC, BH), block 256, dynamic LDS kBfLds
// bytes (one workgroup per CU).
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
// tile, columns 2 cp, 2 cp + 1 of S and dS, and the z / dz of row tid % 64.
struct BfSlabRegs {
  float2 a[8], b[8];
  float za, zb;
};

__global__ __launch_bounds__(256, 1) void bwd_grad_bf(const uint16_t* __restrict__ q,
                                                      const uint16_t* __restrict__ k,
                                                      const uint16_t* __restrict__ v,
                                                      const float* __restrict__ ab,
                                                      const float* __restrict__ frec,
                                                      const float* __restrict__ brec,
                                                      float* __restrict__ dq,
                                                      float* __restrict__ dk,
                                                      float* __restrict__ dvo, int T,
                                                      long long bh_stride, long long E) {
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

  const int c = blockIdx.x, bh = blockIdx.y, tid = threadIdx.x;
  const int lane = tid & 63, w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int h = lane >> 5, l32 = lane & 31;
  const long long t0 = static_cast<long long>(c) * 64;
  const int nt = static_cast<int>(min(64LL, static_cast<long long>(T) - t0));
  const long long hb = static_cast<long long>(bh) * T;
  const float* Sp = frec + bh * bh_stride + c * E;
  const float* Bs = brec + bh * bh_stride + c * E;
  const int rg = tid >> 5, cp = tid & 31;  // staging: rows 8 rg + r, columns 2 cp, 2 cp + 1

  // record rows through buffer loads: the chunk's record as the resource, the
  // slab's first row as the scalar offset, row and column as the vector offset
  const __amdgpu_buffer_rsrc_t rS =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(Sp), 0, static_cast<int>(E * 4), kBfWord3);
  const __amdgpu_buffer_rsrc_t rB =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(Bs), 0, static_cast<int>(E * 4), kBfWord3);
  auto fetch = [&](BfSlabRegs& p, int y) {
    const int f0 = y * 64 - (y * (y - 1)) / 2;  // packed(y, y)
    const int so = f0 * 256;
#pragma unroll
    for (int r = 0; r < 8; ++r) {
      const int vo = max(8 * rg + r - y, 0) * 256 + 8 * cp;  // rows below y: row f0, staged 0
      p.a[r] = __builtin_bit_cast(float2, __builtin_amdgcn_raw_buffer_load_b64(rS, vo, so, 0));
      p.b[r] = __builtin_bit_cast(float2, __builtin_amdgcn_raw_buffer_load_b64(rB, vo, so, 0));
    }
    const int zo = max((tid & 63) - y, 0) * 4;
    p.za = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rS, zo, kBfN * 256 + f0 * 4, 0));
    p.zb = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rB, zo, kBfN * 256 + f0 * 4, 0));
  };
  auto stage = [&](const BfSlabRegs& p, int y, uint16_t* buf) {
    uint16_t* Ss = buf;
    uint16_t* Ds = buf + kBTW;
    uint16_t* DT = Ds + kBTW;
    float m[8];
#pragma unroll
    for (int r = 0; r < 8; ++r) {
      const int x = 8 * rg + r;
      m[r] = x < y ? 0.f : (x == y ? 0.5f : 1.f);
    }
    uint32_t ta[4], tb[4];
#pragma unroll
    for (int r = 0; r < 8; ++r) {
      const int x = 8 * rg + r;
      *reinterpret_cast<uint32_t*>(Ss + x * kBW + 2 * cp) =
          pack_bf16x2(p.a[r].x * m[r], p.a[r].y * m[r]);
      *reinterpret_cast<uint32_t*>(Ds + x * kBW + 2 * cp) =
          pack_bf16x2(p.b[r].x * m[r], p.b[r].y * m[r]);
    }
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const float m0 = 2.f * m[2 * r], m1 = 2.f * m[2 * r + 1];
      ta[r] = pack_bf16x2(p.b[2 * r].x * m0, p.b[2 * r + 1].x * m1);
      tb[r] = pack_bf16x2(p.b[2 * r].y * m0, p.b[2 * r + 1].y * m1);
    }
    *reinterpret_cast<uint4*>(DT + (2 * cp) * kBP + 8 * rg) = make_uint4(ta[0], ta[1], ta[2], ta[3]);
    *reinterpret_cast<uint4*>(DT + (2 * cp + 1) * kBP + 8 * rg) =
        make_uint4(tb[0], tb[1], tb[2], tb[3]);
    if (w == 0) {  // z column and the zero columns 65..79 of row tid
      const int x = tid;
      const float mz = x < y ? 0.f : (x == y ? 0.5f : 1.f);
      const uint4 zero = make_uint4(0u, 0u, 0u, 0u);
      *reinterpret_cast<uint4*>(Ss + x * kBW + 64) = make_uint4(pack_bf16x2(p.za * mz, 0.f), 0u, 0u, 0u);
      *reinterpret_cast<uint4*>(Ss + x * kBW + 72) = zero;
      *reinterpret_cast<uint4*>(Ds + x * kBW + 64) = make_uint4(pack_bf16x2(p.zb * mz, 0.f), 0u, 0u, 0u);
      *reinterpret_cast<uint4*>(Ds + x * kBW + 72) = zero;
    }
  };

  // ---- chunk rows: q, k, v, a (bf16) row-major and q, k, a transposed ----------
  {
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
  // the first two slabs' record rows are on their way during the in-chunk terms
  BfSlabRegs pf0;
  fetch(pf0, 0);
  __syncthreads();

  // ---- in-chunk scores: wave w takes the (key tile w >> 1, token tile w & 1)
  // tile of Sc^T and Cw^T, then writes Pm, Pm^T and W^T ----------------------------
  {
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
  const bool dqw = w < 2;
  const int Tw = w & 1;  // token tile (dq waves) / key tile (dk waves) / key tile of dv
  const int J = w >> 1;  // value tile of dv
  f32x16 acc0 = {}, acc1 = {}, dvacc = {};
  {
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
  __syncthreads();  // the in-chunk tiles are dead: the slab buffers take over

  auto compute = [&](int y, const uint16_t* buf) {
    const uint16_t* Sl = buf + (dqw ? 0 : kBTW);
    const uint16_t* DT = buf + 2 * kBTW;
    f32x16 P0 = {}, P1 = {}, Qy = {};
    const bool x0 = y < 32;  // x tile 0 holds rows x >= y
    if (x0) {
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
    for (int ks = 0; ks < 4; ++ks)  // rows below y are staged as zeros
      Qy = mfma_bf(ld8(DT + (32 * J + l32) * kBP + 16 * ks + 8 * h), ld8(krow + 16 * ks + 8 * h), Qy);
    const float s2 = 2.f * bf_f32(xrow[y]);
    float R = 0.f;
    // x_t[x] of this lane's accumulator rows x = 32 X + 8 m + 4 h + e, four per read
    auto xq = [&](int X, int mq) { return *reinterpret_cast<const uint2*>(xrow + 32 * X + 8 * mq + 4 * h); };
    if (x0) {
#pragma unroll
      for (int mq = 0; mq < 4; ++mq) {
        const uint2 xw = xq(0, mq);
        const float xv[4] = {bf16lo_f32(xw.x), bf16hi_f32(xw.x), bf16lo_f32(xw.y), bf16hi_f32(xw.y)};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          acc0[4 * mq + e] += s2 * P0[4 * mq + e];
          R += xv[e] * P0[4 * mq + e];
        }
      }
    }
#pragma unroll
    for (int mq = 0; mq < 4; ++mq) {
      const uint2 xw = xq(1, mq);
      const float xv[4] = {bf16lo_f32(xw.x), bf16hi_f32(xw.x), bf16lo_f32(xw.y), bf16hi_f32(xw.y)};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        acc1[4 * mq + e] += s2 * P1[4 * mq + e];
        R += xv[e] * P1[4 * mq + e];
      }
    }
    R += __shfl_xor(R, 32);
    if (h == 0) Rout[y] = 2.f * R;
    const float ky = bf_f32(krow[y]);
#pragma unroll
    for (int i = 0; i < 16; ++i) dvacc[i] += ky * Qy[i];
  };

  uint16_t* buf0 = slab;
  uint16_t* buf1 = slab + kBfSlab / 2;
  stage(pf0, 0, buf0);
  fetch(pf0, 1);
  __syncthreads();
  for (int y = 0; y < 64; y += 2) {
    stage(pf0, y + 1, buf1);
    fetch(pf0, min(y + 2, 63));
    compute(y, buf0);
    __syncthreads();
    stage(pf0, y + 2, buf0);
    fetch(pf0, min(y + 3, 63));
    compute(y + 1, buf1);
    __syncthreads();
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

}  // namespace

bool bwd_bf_ok(int d, int dv, int C, int g) { return d == 64 && dv == 64 && C == 64 && g == 1; }

hipError_t launch_bwd_grad_bf(const void* q, const void* k, const void* v, const float* ab,
                              const float* frec, const float* brec, float* dq, float* dk,
                              float* dv_out, int BH, int T, long long bh_stride, long long E,
                              hipStream_t st) {
  const int NC = (T + 63) / 64;
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&bwd_grad_bf),
                                     hipFuncAttributeMaxDynamicSharedMemorySize, kBfLds);
  if (e != hipSuccess) return e;
  bwd_grad_bf<<<dim3(NC, BH), 256, kBfLds, st>>>(
      static_cast<const uint16_t*>(q), static_cast<const uint16_t*>(k),
      static_cast<const uint16_t*>(v), ab, frec, brec, dq, dk, dv_out, T, bh_stride, E);
  return hipGetLastError();
}

}  // namespace kata
