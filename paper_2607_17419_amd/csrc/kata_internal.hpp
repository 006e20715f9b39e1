// kata_internal.hpp -- internal launch interface between the libkata host
// dispatch (kata_api.hip) and the kernel files.
#pragma once

#include "kata_common.hpp"

namespace kata {

// Per-element weight applied by the prefix scan when it writes its output.
struct UnitWeight {
  __device__ __forceinline__ float operator()(long long) const { return 1.f; }
};

__device__ __forceinline__ void store_weighted(float* p, long long i, float x, float w) {
  p[i] = x * w;
}
__device__ __forceinline__ void store_weighted(bf16_t* p, long long i, float x, float w) {
  __bf16 h = static_cast<__bf16>(x * w);
  p[i].bits = __builtin_bit_cast(uint16_t, h);
}

// ---- fp32 path (kata_fp32.hip) -------------------------------------------
// g: feature blocks of KATA-Mg (d % g == 0; 1 is KATA-M1)
size_t fp32_forward_workspace(int BH, int T, int d, int dv, int C, int g);
size_t fp32_forward_smem(int d, int C, int g);

// ev: null, or 4 events recorded on `st` before the state kernel and after
// each of the three stages (state, scan, output).
template <typename Tin>
hipError_t launch_fp32_forward(const void* q, const void* k, const void* v, float* out, int BH,
                               int T, int d, int dv, int C, int g, void* ws, hipStream_t st,
                               hipEvent_t* ev);
template <typename Tin>
hipError_t launch_prefill(const void* k, const void* v, float* S, float* z, int BH, int T, int d,
                          int dv, int g, hipStream_t st);
template <typename Tin>
hipError_t launch_decode(float* S, float* z, const void* q, const void* k, const void* v,
                         float* out, int BH, int d, int dv, int g, hipStream_t st);

// ---- bf16 MFMA path (kata_mfma.hip) ---------------------------------------
// g: feature blocks of KATA-Mg (1 or, at d = 64, 2)
bool mfma_supported(int d, int dv, int C, int g);
size_t mfma_forward_workspace(int BH, int T, int d, int dv, int L, int g);
// den (nullable): the per-row denominators D_t, fp32 [BH][T]
hipError_t launch_mfma_forward(const void* q, const void* k, const void* v, float* out, float* den,
                               int BH, int T, int d, int dv, int g, int L, void* ws,
                               hipStream_t st, hipEvent_t* ev);
size_t mfma_quadratic_workspace(int BH, int T, int dv);
hipError_t launch_mfma_quadratic(const void* q, const void* k, const void* v, float* out, int BH,
                                 int T, int d, int dv, int g, void* ws, hipStream_t st);

// ---- linear features (kata_linear.hip) ------------------------------------
// feature codes of kata_lin_feature_t
constexpr int kLinIdentity = 0, kLinRelu = 1, kLinElu = 2, kLinLorentz = 3, kLinLorentzS = 4;
__host__ __device__ inline int lin_dim(int d, int feature) {
  return feature == kLinLorentz ? d + 1 : d;
}
size_t lin_fp32_workspace(int BH, int T, int d, int dv, int C, int feature);
template <typename Tin>
hipError_t launch_lin_fp32(const void* q, const void* k, const void* v, float* out, int BH, int T,
                           int d, int dv, int C, int feature, float eps, int normalize, void* ws,
                           hipStream_t st, hipEvent_t* ev);
bool lin_mfma_supported(int T, int d, int dv, int C, int feature);
size_t lin_mfma_workspace(int BH, int T, int L, int feature);
hipError_t launch_lin_mfma(const void* q, const void* k, const void* v, float* out, int BH, int T,
                           int feature, float eps, int normalize, int L, void* ws, hipStream_t st,
                           hipEvent_t* ev);

// ---- backward (kata_bwd.hip; gradients of bf16 inputs in kata_bwd_bf.hip) ----
bool bwd_supported(int d, int dv, int C, int g);
// Shapes of the bf16 matrix-core gradients kernel: d = dv = C = 64, g = 1.
bool bwd_bf_ok(int d, int dv, int C, int g);
// Records of that path, per chunk and head: S as bf16 rows of 64, then z as
// fp32 (bwd_bf_record_bytes() bytes, chunk-major within a head).
size_t bwd_bf_record_bytes();
// Chunk records of every chunk on the bf16 matrix cores for bf16 x: forward
// states (x = k, y = v bf16) or backward states (x = q, y = the a_t | b_t
// rows, fp32, row stride 65).
hipError_t launch_bwd_state_bf(bool backward, const void* x, const void* y, void* rec, int BH,
                               int T, hipStream_t st);
// Exclusive prefix (reverse: suffix) of those records in place, diagonal
// features weighted 1/2.
hipError_t launch_bwd_scan_bf(bool reverse, void* rec, int BH, int T, hipStream_t st);
// The exclusive prefix (backward: suffix) records of the same chunk states in
// one pass, state and scan fused, diagonal features weighted 1/2; used from
// bwd_bf_fused_min_heads() heads (batch x heads) on.
int bwd_bf_fused_min_heads();
// Whether the backward of this shape fuses each state launch with its scan.
inline bool bwd_fused_scan(int BH, int d, int dv, int C, int g, bool bf16_inputs) {
  return bf16_inputs && bwd_bf_ok(d, dv, C, g) && BH >= bwd_bf_fused_min_heads();
}
hipError_t launch_bwd_prefix_bf(bool backward, const void* x, const void* y, void* rec, int BH,
                                int T, hipStream_t st);
// Gradients of every chunk from the scanned records, a_t | b_t rows (ab, row
// stride 65) and bf16 q, k, v; every tensor 16-byte aligned (as the C ABI
// requires).
hipError_t launch_bwd_grad_bf(const void* q, const void* k, const void* v, const float* ab,
                              const void* frec, const void* brec, float* dq, float* dk,
                              float* dv_out, int BH, int T, hipStream_t st);
size_t bwd_workspace(int BH, int T, int d, int dv, int C, int g);
// ev: null, or 7 events recorded before the first kernel and after each of the
// six launches (forward states, prefix scan, coefficients, backward states,
// suffix scan, gradients).  den: null, or the forward's denominators D_t
// (fp32 [BH][T]), which then replace the recomputed ones in the coefficients.
template <typename Tin>
hipError_t launch_bwd(const void* q, const void* k, const void* v, const float* out,
                      const float* dout, const float* den, float* dq, float* dk, float* dv_out,
                      int BH, int T, int d, int dv, int C, int g, void* ws, hipStream_t st,
                      hipEvent_t* ev);

inline hipError_t record(hipEvent_t* ev, int i, hipStream_t st) {
  return ev ? hipEventRecord(ev[i], st) : hipSuccess;
}

}  // namespace kata
