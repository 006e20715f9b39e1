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
