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
// Each workgroup owns kEB consecutive elements of the record for every chunk;
// rows are processed in blocks of kNB with a work-efficient (Blelloch) tree in
// LDS: an up-sweep of log2(kNB) levels, then a down-sweep, plus a carry from
// earlier blocks.  HBM traffic: one coalesced read and one write per element.
// in and out may alias when OutT is float.
// grid (ceil(E / kEB), BH), block 256.
// ---------------------------------------------------------------------------
constexpr int kEB = 64;
constexpr int kNB = 128;

template <typename OutT, typename Weight>
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
      tile[r][col] = (active && r < nr) ? ib[static_cast<long long>(r0 + r) * E + e] : 0.f;
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
      if (active) store_weighted(ob, static_cast<long long>(r0 + r) * E + e, tile[r][col] + cin, weight(e));
    if (rgrp == 0) carry += total;
    __syncthreads();
  }
}

}  // namespace kata

namespace kata {

// ---------------------------------------------------------------------------
// In-place exclusive prefix over bf16 records (the MFMA path's span states):
//   rec[bh][c][e] <- bf16( w(e) * sum_{c' < c} rec[bh][c'][e] ),  rec[.][0][.] = 0,
// with the sums carried in fp32.  A workgroup owns kEB16 consecutive elements
// of every record (512-byte rows, 16-byte accesses); rows are processed in
// blocks of kNB16 with a Blelloch tree in LDS and an fp32 carry between blocks.
// E must be a multiple of 8.  grid (ceil(E / kEB16), BH), block 256.
// ---------------------------------------------------------------------------
constexpr int kEB16 = 256;
constexpr int kNB16 = 32;

template <typename Weight>
__global__ __launch_bounds__(256) void scan_exclusive_bf16(uint16_t* rec, int N, long long E,
                                                           long long bh_stride, Weight weight) {
  __shared__ float tile[kNB16][kEB16 + 4];
  __shared__ float total_s[kEB16];
  const int tid = threadIdx.x;
  const long long e0 = static_cast<long long>(blockIdx.x) * kEB16;
  uint16_t* rb = rec + blockIdx.y * bh_stride;
  const int cc = tid & 31;        // 8-element chunk of the column block
  const int r8 = tid >> 5;        // row inside a pass of 8 rows
  const long long ec = e0 + 8 * cc;
  const bool active = ec < E;
  float carry[8];
  float w[8];
#pragma unroll
  for (int x = 0; x < 8; ++x) {
    carry[x] = 0.f;
    w[x] = active ? weight(ec + x) : 0.f;
  }
  for (int r0 = 0; r0 < N; r0 += kNB16) {
    const int nr = min(kNB16, N - r0);
#pragma unroll
    for (int p = 0; p < kNB16 / 8; ++p) {
      const int r = r8 + 8 * p;
      uint4 q4 = make_uint4(0u, 0u, 0u, 0u);
      if (active && r < nr)
        q4 = *reinterpret_cast<const uint4*>(rb + static_cast<long long>(r0 + r) * E + ec);
      const uint32_t q[4] = {q4.x, q4.y, q4.z, q4.w};
#pragma unroll
      for (int x = 0; x < 4; ++x) {
        tile[r][8 * cc + 2 * x] = bf16lo_f32(q[x]);
        tile[r][8 * cc + 2 * x + 1] = bf16hi_f32(q[x]);
      }
    }
    __syncthreads();
    for (int step = 1; step < kNB16; step <<= 1) {
      const int nodes = kNB16 / (2 * step);
      for (int i = tid; i < nodes * kEB16; i += 256) {
        const int node = i / kEB16, col = i % kEB16;
        const int right = (node + 1) * 2 * step - 1;
        tile[right][col] += tile[right - step][col];
      }
      __syncthreads();
    }
    total_s[tid] = tile[kNB16 - 1][tid];
    tile[kNB16 - 1][tid] = 0.f;
    __syncthreads();
    for (int step = kNB16 / 2; step >= 1; step >>= 1) {
      const int nodes = kNB16 / (2 * step);
      for (int i = tid; i < nodes * kEB16; i += 256) {
        const int node = i / kEB16, col = i % kEB16;
        const int right = (node + 1) * 2 * step - 1;
        const float left = tile[right - step][col];
        tile[right - step][col] = tile[right][col];
        tile[right][col] += left;
      }
      __syncthreads();
    }
#pragma unroll
    for (int p = 0; p < kNB16 / 8; ++p) {
      const int r = r8 + 8 * p;
      if (active && r < nr) {
        uint32_t q[4];
#pragma unroll
        for (int x = 0; x < 4; ++x)
          q[x] = pack_bf16x2(w[2 * x] * (tile[r][8 * cc + 2 * x] + carry[2 * x]),
                             w[2 * x + 1] * (tile[r][8 * cc + 2 * x + 1] + carry[2 * x + 1]));
        *reinterpret_cast<uint4*>(rb + static_cast<long long>(r0 + r) * E + ec) =
            make_uint4(q[0], q[1], q[2], q[3]);
      }
    }
#pragma unroll
    for (int x = 0; x < 8; ++x) carry[x] += total_s[8 * cc + x];
    __syncthreads();
  }
}

}  // namespace kata
