// kata_scan.hpp -- exclusive associative scan over chunk (or span) state
// records, shared by the fp32 and MFMA forward paths.
#pragma once

#include "kata_common.hpp"
#include "kata_internal.hpp"

namespace kata {

// ---------------------------------------------------------------------------
// Exclusive prefix along the record axis (section "Tree-scan inter-chunk
// reduction"; the three-stage pipeline's middle stage):
//   out[bh][c][e] = w(e) * sum_{c' < c} in[bh][c'][e],  out[.][0][.] = 0.
// kReverse runs the same scan over the records in reverse order (record c
// receives the sum over c' > c: the exclusive suffix of the backward pass).
// Each workgroup owns kEB consecutive elements of the record for every chunk;
// rows are processed in blocks of kNB with a work-efficient (Blelloch) tree in
// LDS: an up-sweep of log2(kNB) levels, then a down-sweep, plus a carry from
// earlier blocks.  HBM traffic: one coalesced read and one write per element.
// in and out may alias when OutT is float.
// grid (ceil(E / kEB), BH), block 256.
// ---------------------------------------------------------------------------
constexpr int kEB = 64;
constexpr int kNB = 128;

template <typename OutT, typename Weight, bool kReverse = false>
__global__ __launch_bounds__(256) void scan_exclusive(const float* in, OutT* out, int N,
                                                      long long E, long long bh_stride,
                                                      Weight weight) {
  __shared__ float tile[kNB][kEB + 1];
  __shared__ float carry_s[kEB];
  const int tid = threadIdx.x;
  const long long e0 = static_cast<long long>(blockIdx.x) * kEB;
  const int bh = blockIdx.y;
  const float* ib = in + bh * bh_stride;
  OutT* ob = out + bh * bh_stride;
  const int col = tid % kEB;
  const int rgrp = tid / kEB;  // 4 row groups
  const long long e = e0 + col;
  const bool active = e < E;
  float carry = 0.f;  // held by the threads with rgrp == 0
  for (int r0 = 0; r0 < N; r0 += kNB) {
    const int nr = min(kNB, N - r0);
    // load (zero beyond the last row)
    for (int r = rgrp; r < kNB; r += 4)
      tile[r][col] = (active && r < nr)
                         ? ib[static_cast<long long>(kReverse ? N - 1 - (r0 + r) : r0 + r) * E + e]
                         : 0.f;
    __syncthreads();
    // up-sweep: node i (right child index) accumulates its left sibling
    for (int step = 1; step < kNB; step <<= 1) {
      const int nodes = kNB / (2 * step);
      for (int i = tid; i < nodes * kEB; i += 256) {
        int node = i / kEB, cc = i % kEB;
        int right = (node + 1) * 2 * step - 1;
        tile[right][cc] += tile[right - step][cc];
      }
      __syncthreads();
    }
    float total = 0.f;
    if (rgrp == 0) {
      total = tile[kNB - 1][col];
      tile[kNB - 1][col] = 0.f;
    }
    __syncthreads();
    // down-sweep
    for (int step = kNB / 2; step >= 1; step >>= 1) {
      const int nodes = kNB / (2 * step);
      for (int i = tid; i < nodes * kEB; i += 256) {
        int node = i / kEB, cc = i % kEB;
        int right = (node + 1) * 2 * step - 1;
        float left = tile[right - step][cc];
        tile[right - step][cc] = tile[right][cc];
        tile[right][cc] += left;
      }
      __syncthreads();
    }
    // add the carry of earlier blocks and store
    if (rgrp == 0) carry_s[col] = carry;
    __syncthreads();
    const float cin = carry_s[col];
    for (int r = rgrp; r < nr; r += 4)
      if (active)
        store_weighted(ob, static_cast<long long>(kReverse ? N - 1 - (r0 + r) : r0 + r) * E + e,
                       tile[r][col] + cin, weight(e));
    if (rgrp == 0) carry += total;
    __syncthreads();
  }
}

}  // namespace kata

namespace kata {

// ---------------------------------------------------------------------------
// In-place exclusive prefix over bf16 records (the MFMA path's span states):
//   rec[bh][c][e] <- bf16( w(e) * sum_{c' < c} rec[bh][c'][e] ),  rec[.][0][.] = 0,
// with the sums carried in fp32.  Blocked Blelloch scan along the record
// axis: thread (column group cg, row group rg) holds 8 elements x kRPT16
// records in registers and runs the up-sweep / down-sweep over its records
// there; with RG > 1 row groups the row-group totals are scanned across the
// groups through LDS; blocks of RG * kRPT16 records are chained by an fp32
// carry.  A workgroup owns 8 * (256 / RG) consecutive elements of every
// record, so short record axes take few row groups and wide element slices
// (RG = 1 for up to 16 records: no idle row groups, no LDS exchange) and long
// ones take eight.  The last record's input never enters an exclusive prefix
// and is not read.  All of a thread's loads of a block are in flight together
// (16-byte accesses).  E must be a multiple of 8.
// grid (ceil(E / scan_bf16_elems(RG)), BH), block 256.
// ---------------------------------------------------------------------------
constexpr int kRPT16 = 16;  // records per thread and block

__host__ __device__ constexpr int scan_bf16_elems(int rg) { return 8 * (256 / rg); }

// Row groups for N records: the fewest that cover N in one block, at most 8.
inline int scan_bf16_row_groups(int N) {
  return N <= kRPT16 ? 1 : N <= 2 * kRPT16 ? 2 : N <= 4 * kRPT16 ? 4 : 8;
}

// Records are read once and written once: non-temporal 16-byte accesses keep
// them from lingering dirty in the caches, where their write-back would
// otherwise overlap the next kernel (measured: the span output kernel after
// this scan ran about 2% faster).
typedef unsigned scan_b128 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ uint4 stream_load_b128(const uint16_t* p) {
  const scan_b128 t = __builtin_nontemporal_load(reinterpret_cast<const scan_b128*>(p));
  return make_uint4(t.x, t.y, t.z, t.w);
}
__device__ __forceinline__ void stream_store_b128(uint16_t* p, uint4 u) {
  const scan_b128 t = {u.x, u.y, u.z, u.w};
  __builtin_nontemporal_store(t, reinterpret_cast<scan_b128*>(p));
}

template <int RG, typename Weight>
__global__ __launch_bounds__(256) void scan_exclusive_bf16(uint16_t* rec, int N, long long E,
                                                           long long bh_stride, Weight weight) {
  static_assert(RG == 1 || RG == 2 || RG == 4 || RG == 8, "row groups");
  constexpr int CG = 256 / RG;              // column groups of 8 elements
  constexpr int EB = scan_bf16_elems(RG);   // elements per workgroup
  constexpr int NB = RG * kRPT16;           // records per block
  __shared__ float tot[RG][EB];
  const int tid = threadIdx.x;
  const int cg = tid % CG, rg = tid / CG;
  const long long ec = static_cast<long long>(blockIdx.x) * EB + 8 * cg;
  uint16_t* rb = rec + blockIdx.y * bh_stride;
  const bool active = ec < E;
  float w[8], carry[8];
#pragma unroll
  for (int x = 0; x < 8; ++x) {
    w[x] = active ? weight(ec + x) : 0.f;
    carry[x] = 0.f;
  }
  for (int r0 = 0; r0 < N; r0 += NB) {
    const int rbase = r0 + rg * kRPT16;  // this thread's first record
    float v[kRPT16][8];
#pragma unroll
    for (int j = 0; j < kRPT16; ++j) {
      uint4 q4 = make_uint4(0u, 0u, 0u, 0u);
      if (active && rbase + j < N - 1)
        q4 = stream_load_b128(rb + static_cast<long long>(rbase + j) * E + ec);
      const uint32_t q[4] = {q4.x, q4.y, q4.z, q4.w};
#pragma unroll
      for (int x = 0; x < 4; ++x) {
        v[j][2 * x] = bf16lo_f32(q[x]);
        v[j][2 * x + 1] = bf16hi_f32(q[x]);
      }
    }
    // up-sweep: v[j] for j = 2^(l+1)-1 (mod 2^(l+1)) accumulates its left subtree
#pragma unroll
    for (int d = 1; d < kRPT16; d <<= 1)
#pragma unroll
      for (int j = 2 * d - 1; j < kRPT16; j += 2 * d)
#pragma unroll
        for (int x = 0; x < 8; ++x) v[j][x] += v[j - d][x];
    float gsum[8];
#pragma unroll
    for (int x = 0; x < 8; ++x) {
      gsum[x] = v[kRPT16 - 1][x];
      v[kRPT16 - 1][x] = 0.f;
    }
    // down-sweep: exclusive prefixes within the thread's records
#pragma unroll
    for (int d = kRPT16 / 2; d >= 1; d >>= 1)
#pragma unroll
      for (int j = 2 * d - 1; j < kRPT16; j += 2 * d)
#pragma unroll
        for (int x = 0; x < 8; ++x) {
          const float left = v[j - d][x];
          v[j - d][x] = v[j][x];
          v[j][x] += left;
        }
    float pre[8], blk[8];
#pragma unroll
    for (int x = 0; x < 8; ++x) {
      pre[x] = carry[x];
      blk[x] = gsum[x];
    }
    if constexpr (RG > 1) {
      // exclusive scan of the row-group totals, plus the block total for the carry
#pragma unroll
      for (int x = 0; x < 8; ++x) tot[rg][8 * cg + x] = gsum[x];
      __syncthreads();
#pragma unroll
      for (int x = 0; x < 8; ++x) blk[x] = 0.f;
#pragma unroll
      for (int g2 = 0; g2 < RG; ++g2)
#pragma unroll
        for (int x = 0; x < 8; ++x) {
          const float t = tot[g2][8 * cg + x];
          if (g2 < rg) pre[x] += t;
          blk[x] += t;
        }
      __syncthreads();  // tot is rewritten by the next block
    }
#pragma unroll
    for (int j = 0; j < kRPT16; ++j) {
      if (active && rbase + j < N) {
        uint32_t q[4];
#pragma unroll
        for (int x = 0; x < 4; ++x)
          q[x] = pack_bf16x2(w[2 * x] * (pre[2 * x] + v[j][2 * x]),
                             w[2 * x + 1] * (pre[2 * x + 1] + v[j][2 * x + 1]));
        stream_store_b128(rb + static_cast<long long>(rbase + j) * E + ec,
                          make_uint4(q[0], q[1], q[2], q[3]));
      }
    }
#pragma unroll
    for (int x = 0; x < 8; ++x) carry[x] += blk[x];
  }
}

// Launch the bf16 record scan with the row-group count scan_bf16_row_groups(N).
template <typename Weight>
void launch_scan_exclusive_bf16(uint16_t* rec, int N, long long E, long long bh_stride, int BH,
                                Weight weight, hipStream_t st) {
  const int rg = scan_bf16_row_groups(N);
  const dim3 grid(static_cast<unsigned>((E + scan_bf16_elems(rg) - 1) / scan_bf16_elems(rg)),
                  static_cast<unsigned>(BH));
  switch (rg) {
    case 1: scan_exclusive_bf16<1><<<grid, 256, 0, st>>>(rec, N, E, bh_stride, weight); break;
    case 2: scan_exclusive_bf16<2><<<grid, 256, 0, st>>>(rec, N, E, bh_stride, weight); break;
    case 4: scan_exclusive_bf16<4><<<grid, 256, 0, st>>>(rec, N, E, bh_stride, weight); break;
    default: scan_exclusive_bf16<8><<<grid, 256, 0, st>>>(rec, N, E, bh_stride, weight); break;
  }
}

}  // namespace kata

namespace kata {

// ---------------------------------------------------------------------------
// In-place exclusive prefix over fp32 records, register-blocked like the bf16
// scan above:  rec[bh][c][e] <- w(e) * sum_{c' < c} rec[bh][c'][e].
// Thread (column group cg, row group rg) holds 4 elements (one 16-byte
// access per record) x kRPT4 records; the up-sweep / down-sweep runs over its
// records in registers, the row-group totals are scanned through LDS, and
// blocks of kNB4 records are chained by a carry.  All of a thread's loads of
// a block are issued together.  E must be a multiple of 4.  kReverse scans the
// records in reverse order (record c receives the sum over c' > c).
// grid (ceil(E / kEB4), BH), block 256.
// ---------------------------------------------------------------------------
constexpr int kCG4 = 32;               // column groups of 4 elements
constexpr int kEB4 = 4 * kCG4;         // elements per workgroup (128)
constexpr int kRG4 = 256 / kCG4;       // row groups (8)
constexpr int kRPT4 = 8;               // records per thread and block
constexpr int kNB4 = kRG4 * kRPT4;     // records per block (64)

template <typename Weight, bool kReverse = false>
__global__ __launch_bounds__(256) void scan_exclusive_f32x4(float* rec, int N, long long E,
                                                            long long bh_stride, Weight weight) {
  __shared__ float4 tot[kRG4][kCG4];
  const int tid = threadIdx.x;
  const int cg = tid % kCG4, rg = tid / kCG4;
  const long long ec = static_cast<long long>(blockIdx.x) * kEB4 + 4 * cg;
  float* rb = rec + blockIdx.y * bh_stride;
  const bool active = ec < E;
  float w[4], carry[4];
#pragma unroll
  for (int x = 0; x < 4; ++x) {
    w[x] = active ? weight(ec + x) : 0.f;
    carry[x] = 0.f;
  }
  for (int r0 = 0; r0 < N; r0 += kNB4) {
    const int rbase = r0 + rg * kRPT4;
    float v[kRPT4][4];
#pragma unroll
    for (int j = 0; j < kRPT4; ++j) {
      float4 a = make_float4(0.f, 0.f, 0.f, 0.f);
      if (active && rbase + j < N)
        a = *reinterpret_cast<const float4*>(
            rb + static_cast<long long>(kReverse ? N - 1 - (rbase + j) : rbase + j) * E + ec);
      v[j][0] = a.x;
      v[j][1] = a.y;
      v[j][2] = a.z;
      v[j][3] = a.w;
    }
#pragma unroll
    for (int d = 1; d < kRPT4; d <<= 1)
#pragma unroll
      for (int j = 2 * d - 1; j < kRPT4; j += 2 * d)
#pragma unroll
        for (int x = 0; x < 4; ++x) v[j][x] += v[j - d][x];
    float gsum[4];
#pragma unroll
    for (int x = 0; x < 4; ++x) {
      gsum[x] = v[kRPT4 - 1][x];
      v[kRPT4 - 1][x] = 0.f;
    }
#pragma unroll
    for (int d = kRPT4 / 2; d >= 1; d >>= 1)
#pragma unroll
      for (int j = 2 * d - 1; j < kRPT4; j += 2 * d)
#pragma unroll
        for (int x = 0; x < 4; ++x) {
          const float left = v[j - d][x];
          v[j - d][x] = v[j][x];
          v[j][x] += left;
        }
    tot[rg][cg] = make_float4(gsum[0], gsum[1], gsum[2], gsum[3]);
    __syncthreads();
    float pre[4], blk[4];
#pragma unroll
    for (int x = 0; x < 4; ++x) {
      pre[x] = carry[x];
      blk[x] = 0.f;
    }
#pragma unroll
    for (int g2 = 0; g2 < kRG4; ++g2) {
      const float4 t = tot[g2][cg];
      const float tv[4] = {t.x, t.y, t.z, t.w};
#pragma unroll
      for (int x = 0; x < 4; ++x) {
        if (g2 < rg) pre[x] += tv[x];
        blk[x] += tv[x];
      }
    }
    __syncthreads();  // tot is rewritten by the next block
#pragma unroll
    for (int j = 0; j < kRPT4; ++j) {
      if (active && rbase + j < N)
        *reinterpret_cast<float4*>(
            rb + static_cast<long long>(kReverse ? N - 1 - (rbase + j) : rbase + j) * E + ec) =
            make_float4(w[0] * (pre[0] + v[j][0]), w[1] * (pre[1] + v[j][1]),
                        w[2] * (pre[2] + v[j][2]), w[3] * (pre[3] + v[j][3]));
    }
#pragma unroll
    for (int x = 0; x < 4; ++x) carry[x] += blk[x];
  }
}

}  // namespace kata
