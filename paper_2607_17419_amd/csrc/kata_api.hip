// kata_api.hip -- host side of the libkata C ABI (include/kata.h): argument
// validation, path selection (bf16 MFMA fast path or fp32 path), workspace
// handling and error mapping.  Nothing here touches the GPU before the
// arguments have been validated.  Every entry point exists for KATA-M1 and,
// with a feature-block count g (kata_mg_*), for KATA-Mg; g = 1 is M1.
#include <climits>
#include <cmath>
#include <cstdint>
#include <cstring>
#include <mutex>

#include "kata.h"
#include "kata_internal.hpp"

namespace {

constexpr long long kMaxElems = 1LL << 40;  // per-tensor element bound
constexpr int kGridYZ = 65535;

enum class Path { kInvalid, kUnsupported, kMfma, kFp32 };

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

bool product_ok(long long a, long long b, long long c, long long d) {
  // a*b*c*d <= kMaxElems with every factor >= 1
  long long p = a;
  for (long long f : {b, c, d}) {
    if (p > kMaxElems / f) return false;
    p *= f;
  }
  return true;
}

bool blocks_ok(int d, int g) { return g >= 1 && d >= g && d % g == 0; }

// Default span on the MFMA path: about 1024 tokens per stored record at
// d = 64 and 512 at d = 32, whose records are a quarter the size, so that the
// in-span attention (growing with the span) and the record traffic (shrinking
// with it) balance; measured forwards: d = 32, C = 128, B1 H16 T131072 0.78 ms
// at 512 tokens against 0.81 at 1024 and 1.09 at 256; d = 64 (one or two
// feature blocks) fastest at 1024.
int default_span(int C, int d, Path path) {
  if (path != Path::kMfma) return 1;
  int s = (d <= 32 ? 512 : 1024) / C;
  return s < 1 ? 1 : s;
}

Path fwd_path(int B, int H, int T, int d, int dv, int C, int dtype, int g) {
  if (B < 1 || H < 1 || T < 1 || d < 1 || dv < 1 || C < 1) return Path::kInvalid;
  if (dtype != KATA_F32 && dtype != KATA_BF16) return Path::kInvalid;
  if (!blocks_ok(d, g)) return Path::kInvalid;
  if (!product_ok(B, H, T, d > dv ? d : dv)) return Path::kInvalid;
  if (static_cast<long long>(B) * H > kGridYZ) return Path::kUnsupported;
  if (dtype == KATA_BF16 && kata::mfma_supported(d, dv, C, g)) return Path::kMfma;
  if (d > 64 || dv > 256 || C > 128) return Path::kUnsupported;
  if ((static_cast<long long>(T) + C - 1) / C > kGridYZ) return Path::kUnsupported;
  return Path::kFp32;
}

int span_tokens(int T, int C, int span_chunks) {
  long long L = static_cast<long long>(C) * span_chunks;
  const long long Tc = (static_cast<long long>(T) + C - 1) / C * C;  // T rounded up to C
  if (L > Tc) L = Tc;
  return static_cast<int>(L);
}

size_t workspace_for(Path path, int B, int H, int T, int d, int dv, int C, int g,
                     int span_chunks) {
  const int BH = B * H;
  if (path == Path::kFp32) return kata::fp32_forward_workspace(BH, T, d, dv, C, g);
  if (path == Path::kMfma) {
    const int L = span_tokens(T, C, span_chunks);
    return kata::mfma_forward_workspace(BH, T, d, dv, L, g);
  }
  return 0;
}

kata_status_t from_hip(hipError_t e) { return e == hipSuccess ? KATA_OK : KATA_ERR_HIP; }

// Stream-ordered workspace of the allocating entry points.  A failed
// allocation returns KATA_ERR_HIP and clears the thread's last-error state, so
// that the failure is not reported again by a later call's hipGetLastError.
kata_status_t alloc_ws(void** ws, size_t bytes, hipStream_t stream) {
  *ws = nullptr;
  if (hipMallocAsync(ws, bytes, stream) != hipSuccess || *ws == nullptr) {
    (void)hipGetLastError();
    *ws = nullptr;
    return KATA_ERR_HIP;
  }
  return KATA_OK;
}

int default_span_of(int B, int H, int T, int d, int dv, int C, int dtype, int g) {
  const Path p = fwd_path(B, H, T, d, dv, C, dtype, g);
  if (p == Path::kInvalid || p == Path::kUnsupported) return 0;
  return default_span(C, d, p);
}

size_t fwd_workspace_bytes(int B, int H, int T, int d, int dv, int C, int dtype, int g,
                           int span_chunks) {
  const Path p = fwd_path(B, H, T, d, dv, C, dtype, g);
  if (p == Path::kInvalid || p == Path::kUnsupported || span_chunks < 0) return 0;
  if (span_chunks == 0) span_chunks = default_span(C, d, p);
  if (p == Path::kFp32) span_chunks = 1;
  return workspace_for(p, B, H, T, d, dv, C, g, span_chunks);
}

// den: null, or where the MFMA path writes the denominators D_t (fp32 [B][H][T])
kata_status_t fwd_ws(const void* q, const void* k, const void* v, float* out, int B, int H,
                     int T, int d, int dv, int C, int g, kata_dtype_t dtype, int span_chunks,
                     void* workspace, size_t workspace_bytes, hipEvent_t* ev,
                     hipStream_t stream, float* den = nullptr) {
  if (!q || !k || !v || !out) return KATA_ERR_INVALID_ARG;
  if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(out)) return KATA_ERR_INVALID_ARG;
  if (den && !aligned16(den)) return KATA_ERR_INVALID_ARG;
  if (span_chunks < 0) return KATA_ERR_INVALID_ARG;
  const Path p = fwd_path(B, H, T, d, dv, C, dtype, g);
  if (p == Path::kInvalid) return KATA_ERR_INVALID_ARG;
  if (p == Path::kUnsupported) return KATA_ERR_UNSUPPORTED;
  if (!workspace || (reinterpret_cast<uintptr_t>(workspace) & 255u) != 0) return KATA_ERR_INVALID_ARG;
  if (span_chunks == 0) span_chunks = default_span(C, d, p);
  if (p == Path::kFp32) span_chunks = 1;
  const size_t need = workspace_for(p, B, H, T, d, dv, C, g, span_chunks);
  if (workspace_bytes < need) return KATA_ERR_INVALID_ARG;
  const int BH = B * H;
  if (p == Path::kMfma) {
    const int L = span_tokens(T, C, span_chunks);
    if ((static_cast<long long>(T) + L - 1) / L > kGridYZ) return KATA_ERR_UNSUPPORTED;
    return from_hip(kata::launch_mfma_forward(q, k, v, out, den, BH, T, d, dv, g, L, workspace,
                                              stream, ev));
  }
  if (den) return KATA_ERR_UNSUPPORTED;  // denominators on the MFMA path only
  if (dtype == KATA_F32)
    return from_hip(kata::launch_fp32_forward<float>(q, k, v, out, BH, T, d, dv, C, g, workspace,
                                                     stream, ev));
  return from_hip(kata::launch_fp32_forward<kata::bf16_t>(q, k, v, out, BH, T, d, dv, C, g,
                                                          workspace, stream, ev));
}

kata_status_t fwd_timed(const void* q, const void* k, const void* v, float* out, int B, int H,
                        int T, int d, int dv, int C, int g, kata_dtype_t dtype, int span_chunks,
                        void* workspace, size_t workspace_bytes, hipEvent_t* stage_events,
                        hipStream_t stream) {
  if (!stage_events) return KATA_ERR_INVALID_ARG;
  for (int i = 0; i < 4; ++i)
    if (!stage_events[i]) return KATA_ERR_INVALID_ARG;
  return fwd_ws(q, k, v, out, B, H, T, d, dv, C, g, dtype, span_chunks, workspace,
                workspace_bytes, stage_events, stream);
}

kata_status_t fwd_alloc(const void* q, const void* k, const void* v, float* out, int B, int H,
                        int T, int d, int dv, int C, int g, kata_dtype_t dtype,
                        hipStream_t stream) {
  if (!q || !k || !v || !out) return KATA_ERR_INVALID_ARG;
  if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(out)) return KATA_ERR_INVALID_ARG;
  const Path p = fwd_path(B, H, T, d, dv, C, dtype, g);
  if (p == Path::kInvalid) return KATA_ERR_INVALID_ARG;
  if (p == Path::kUnsupported) return KATA_ERR_UNSUPPORTED;
  const int span = (p == Path::kFp32) ? 1 : default_span(C, d, p);
  const size_t bytes = workspace_for(p, B, H, T, d, dv, C, g, span);
  void* ws = nullptr;
  if (alloc_ws(&ws, bytes, stream) != KATA_OK) return KATA_ERR_HIP;
  const kata_status_t st =
      fwd_ws(q, k, v, out, B, H, T, d, dv, C, g, dtype, span, ws, bytes, nullptr, stream);
  const hipError_t fe = hipFreeAsync(ws, stream);
  if (st != KATA_OK) return st;
  return from_hip(fe);
}

// ---- allocation-free forward ------------------------------------------------
// The workspace of kata_fwd_chunked_noalloc is this file-scope device array:
// every GPU the library runs on holds its own copy until the process ends.
// Host code never passes the array's name to a kernel (on the host it is only
// a stand-in symbol); it uses the device address that hipGetSymbolAddress
// returns for the device the call runs on, looked up once per device.
constexpr size_t kNoAllocScratchBytes = static_cast<size_t>(256) << 20;
static __device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};  // device address of `scratch`, per device

// Device address of the scratch array on the device that `stream` belongs to
// (the current device for the null stream).  The first call on a device makes
// that device current for the lookup and restores the caller's device.
kata_status_t scratch_ptr(hipStream_t stream, void** out) {
  *out = nullptr;
  int cur = -1, dev = -1;
  if (hipGetDevice(&cur) != hipSuccess) {
    (void)hipGetLastError();
    return KATA_ERR_HIP;
  }
  dev = cur;
  if (stream != nullptr && hipStreamGetDevice(stream, &dev) != hipSuccess) {
    (void)hipGetLastError();
    return KATA_ERR_HIP;
  }
  if (dev < 0 || dev >= kMaxDevices) return KATA_ERR_UNSUPPORTED;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_ptr[dev] == nullptr) {
    if (dev != cur && hipSetDevice(dev) != hipSuccess) {
      (void)hipGetLastError();
      return KATA_ERR_HIP;
    }
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (dev != cur) (void)hipSetDevice(cur);
    if (e != hipSuccess || p == nullptr) {
      (void)hipGetLastError();
      return KATA_ERR_HIP;
    }
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return KATA_OK;
}

kata_status_t fwd_noalloc(const void* q, const void* k, const void* v, float* out, int B, int H,
                          int T, int d, int dv, int C, int g, kata_dtype_t dtype,
                          hipStream_t stream) {
  if (!q || !k || !v || !out) return KATA_ERR_INVALID_ARG;
  if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(out)) return KATA_ERR_INVALID_ARG;
  const Path p = fwd_path(B, H, T, d, dv, C, dtype, g);
  if (p == Path::kInvalid) return KATA_ERR_INVALID_ARG;
  if (p == Path::kUnsupported) return KATA_ERR_UNSUPPORTED;
  const int span = (p == Path::kFp32) ? 1 : default_span(C, d, p);
  const size_t bytes = workspace_for(p, B, H, T, d, dv, C, g, span);
  if (bytes > kNoAllocScratchBytes) return KATA_ERR_UNSUPPORTED;  // beyond the scratch array
  void* ws = nullptr;
  const kata_status_t st = scratch_ptr(stream, &ws);
  if (st != KATA_OK) return st;
  return fwd_ws(q, k, v, out, B, H, T, d, dv, C, g, dtype, span, ws, kNoAllocScratchBytes,
                nullptr, stream);
}

// Quadratic form: bf16 MFMA path only.
kata_status_t quad_check(int B, int H, int T, int d, int dv, int dtype, int g) {
  if (B < 1 || H < 1 || T < 1 || d < 1 || dv < 1) return KATA_ERR_INVALID_ARG;
  if (dtype != KATA_F32 && dtype != KATA_BF16) return KATA_ERR_INVALID_ARG;
  if (!blocks_ok(d, g)) return KATA_ERR_INVALID_ARG;
  if (!product_ok(B, H, T, d > dv ? d : dv)) return KATA_ERR_INVALID_ARG;
  if (static_cast<long long>(B) * H > kGridYZ) return KATA_ERR_UNSUPPORTED;
  if (dtype != KATA_BF16 || !kata::mfma_supported(d, dv, 64, g)) return KATA_ERR_UNSUPPORTED;
  return KATA_OK;
}

size_t quad_workspace_bytes(int B, int H, int T, int d, int dv, int dtype, int g) {
  if (quad_check(B, H, T, d, dv, dtype, g) != KATA_OK) return 0;
  return kata::mfma_quadratic_workspace(B * H, T, dv);
}

kata_status_t quad_ws(const void* q, const void* k, const void* v, float* out, int B, int H,
                      int T, int d, int dv, int g, kata_dtype_t dtype, void* workspace,
                      size_t workspace_bytes, hipStream_t stream) {
  if (!q || !k || !v || !out) return KATA_ERR_INVALID_ARG;
  if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(out)) return KATA_ERR_INVALID_ARG;
  const kata_status_t c = quad_check(B, H, T, d, dv, dtype, g);
  if (c != KATA_OK) return c;
  if (!workspace || (reinterpret_cast<uintptr_t>(workspace) & 255u) != 0) return KATA_ERR_INVALID_ARG;
  if (workspace_bytes < kata::mfma_quadratic_workspace(B * H, T, dv)) return KATA_ERR_INVALID_ARG;
  return from_hip(
      kata::launch_mfma_quadratic(q, k, v, out, B * H, T, d, dv, g, workspace, stream));
}

kata_status_t prefill(const void* k, const void* v, float* S, float* z, int B, int H, int T,
                      int d, int dv, int g, kata_dtype_t dtype, hipStream_t stream) {
  if (!k || !v || !S || !z) return KATA_ERR_INVALID_ARG;
  if (!aligned16(k) || !aligned16(v) || !aligned16(S) || !aligned16(z)) return KATA_ERR_INVALID_ARG;
  if (B < 1 || H < 1 || T < 1 || d < 1 || dv < 1) return KATA_ERR_INVALID_ARG;
  if (dtype != KATA_F32 && dtype != KATA_BF16) return KATA_ERR_INVALID_ARG;
  if (!blocks_ok(d, g)) return KATA_ERR_INVALID_ARG;
  if (!product_ok(B, H, T, d > dv ? d : dv)) return KATA_ERR_INVALID_ARG;
  if (d > 64 || dv > 256) return KATA_ERR_UNSUPPORTED;
  if (static_cast<long long>(B) * H > kGridYZ) return KATA_ERR_UNSUPPORTED;
  const int BH = B * H;
  if (dtype == KATA_F32)
    return from_hip(kata::launch_prefill<float>(k, v, S, z, BH, T, d, dv, g, stream));
  return from_hip(kata::launch_prefill<kata::bf16_t>(k, v, S, z, BH, T, d, dv, g, stream));
}

kata_status_t decode(float* S, float* z, const void* q, const void* k, const void* v, float* out,
                     int B, int H, int d, int dv, int g, kata_dtype_t dtype, hipStream_t stream) {
  if (!S || !z || !q || !k || !v || !out) return KATA_ERR_INVALID_ARG;
  if (!aligned16(S) || !aligned16(z) || !aligned16(q) || !aligned16(k) || !aligned16(v) ||
      !aligned16(out))
    return KATA_ERR_INVALID_ARG;
  if (B < 1 || H < 1 || d < 1 || dv < 1) return KATA_ERR_INVALID_ARG;
  if (dtype != KATA_F32 && dtype != KATA_BF16) return KATA_ERR_INVALID_ARG;
  if (!blocks_ok(d, g)) return KATA_ERR_INVALID_ARG;
  if (!product_ok(B, H, d * (d + 1) / 2, dv)) return KATA_ERR_INVALID_ARG;
  if (d > 64 || dv > 256) return KATA_ERR_UNSUPPORTED;
  if (static_cast<long long>(B) * H > INT_MAX) return KATA_ERR_UNSUPPORTED;
  const int BH = B * H;
  if (dtype == KATA_F32)
    return from_hip(kata::launch_decode<float>(S, z, q, k, v, out, BH, d, dv, g, stream));
  return from_hip(kata::launch_decode<kata::bf16_t>(S, z, q, k, v, out, BH, d, dv, g, stream));
}

// ---- linear features ----------------------------------------------------------

Path lin_path(int B, int H, int T, int d, int dv, int C, int feature, float eps, int normalize,
              int dtype) {
  if (B < 1 || H < 1 || T < 1 || d < 1 || dv < 1 || C < 1) return Path::kInvalid;
  if (dtype != KATA_F32 && dtype != KATA_BF16) return Path::kInvalid;
  if (feature < kata::kLinIdentity || feature > kata::kLinLorentzS) return Path::kInvalid;
  if (!std::isfinite(eps) || eps < 0.f) return Path::kInvalid;
  if (normalize != 0 && normalize != 1) return Path::kInvalid;
  if (!product_ok(B, H, T, d + 1 > dv ? d + 1 : dv)) return Path::kInvalid;
  if (static_cast<long long>(B) * H > kGridYZ) return Path::kUnsupported;
  if (dtype == KATA_BF16 && kata::lin_mfma_supported(T, d, dv, C, feature)) return Path::kMfma;
  if (d > 64 || dv > 256 || C > 128) return Path::kUnsupported;
  if ((static_cast<long long>(T) + C - 1) / C * ((C + 31) / 32) > INT_MAX) return Path::kUnsupported;
  return Path::kFp32;
}

// Default span on the MFMA path: about 1024 workgroups per launch (four per
// compute unit) while a span stays within 1024 tokens.
int lin_default_span(int B, int H, int T, int C, Path path) {
  if (path != Path::kMfma) return 1;
  const long long per_wg = static_cast<long long>(T) * B * H / 1024;
  long long s = per_wg / C;
  if (s > 1024 / C) s = 1024 / C;
  return s < 1 ? 1 : static_cast<int>(s);
}

size_t lin_workspace_for(Path p, int B, int H, int T, int d, int dv, int C, int feature,
                         int span_chunks) {
  if (p == Path::kFp32) return kata::lin_fp32_workspace(B * H, T, d, dv, C, feature);
  if (p == Path::kMfma)
    return kata::lin_mfma_workspace(B * H, T, span_tokens(T, C, span_chunks), feature);
  return 0;
}

kata_status_t lin_ws(const void* q, const void* k, const void* v, float* out, int B, int H, int T,
                     int d, int dv, int C, int feature, float eps, int normalize,
                     kata_dtype_t dtype, int span_chunks, void* workspace, size_t workspace_bytes,
                     hipEvent_t* ev, hipStream_t stream) {
  if (!q || !k || !v || !out) return KATA_ERR_INVALID_ARG;
  if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(out)) return KATA_ERR_INVALID_ARG;
  if (span_chunks < 0) return KATA_ERR_INVALID_ARG;
  const Path p = lin_path(B, H, T, d, dv, C, feature, eps, normalize, dtype);
  if (p == Path::kInvalid) return KATA_ERR_INVALID_ARG;
  if (p == Path::kUnsupported) return KATA_ERR_UNSUPPORTED;
  if (!workspace || (reinterpret_cast<uintptr_t>(workspace) & 255u) != 0) return KATA_ERR_INVALID_ARG;
  if (span_chunks == 0) span_chunks = lin_default_span(B, H, T, C, p);
  if (p == Path::kFp32) span_chunks = 1;
  if (workspace_bytes < lin_workspace_for(p, B, H, T, d, dv, C, feature, span_chunks))
    return KATA_ERR_INVALID_ARG;
  const int BH = B * H;
  if (p == Path::kMfma) {
    const int L = span_tokens(T, C, span_chunks);
    if (static_cast<long long>(BH) * ((static_cast<long long>(T) + L - 1) / L) > INT_MAX)
      return KATA_ERR_UNSUPPORTED;
    return from_hip(kata::launch_lin_mfma(q, k, v, out, BH, T, feature, eps, normalize, L,
                                          workspace, stream, ev));
  }
  if (dtype == KATA_F32)
    return from_hip(kata::launch_lin_fp32<float>(q, k, v, out, BH, T, d, dv, C, feature, eps,
                                                 normalize, workspace, stream, ev));
  return from_hip(kata::launch_lin_fp32<kata::bf16_t>(q, k, v, out, BH, T, d, dv, C, feature, eps,
                                                      normalize, workspace, stream, ev));
}

// ---- backward ---------------------------------------------------------------------

kata_status_t bwd_check(int B, int H, int T, int d, int dv, int C, int g, int dtype) {
  if (B < 1 || H < 1 || T < 1 || d < 1 || dv < 1 || C < 1) return KATA_ERR_INVALID_ARG;
  if (dtype != KATA_F32 && dtype != KATA_BF16) return KATA_ERR_INVALID_ARG;
  if (!blocks_ok(d, g)) return KATA_ERR_INVALID_ARG;
  if (!product_ok(B, H, T, d > dv ? d + 1 : dv + 1)) return KATA_ERR_INVALID_ARG;
  if (!kata::bwd_supported(d, dv, C, g)) return KATA_ERR_UNSUPPORTED;
  if (static_cast<long long>(B) * H > kGridYZ) return KATA_ERR_UNSUPPORTED;
  if ((static_cast<long long>(T) + C - 1) / C > kGridYZ) return KATA_ERR_UNSUPPORTED;
  return KATA_OK;
}

// Non-null, 16-byte aligned tensors of the backward (checked before any HIP call).
bool bwd_ptrs_ok(const void* q, const void* k, const void* v, const float* out,
                 const float* dout, const float* dq, const float* dk, const float* dvv) {
  for (const void* p : {q, k, v, static_cast<const void*>(out), static_cast<const void*>(dout),
                        static_cast<const void*>(dq), static_cast<const void*>(dk),
                        static_cast<const void*>(dvv)})
    if (!p || !aligned16(p)) return false;
  return true;
}

// den: null, or the forward's denominators D_t (fp32 [B][H][T])
kata_status_t bwd_ws(const void* q, const void* k, const void* v, const float* out,
                     const float* dout, float* dq, float* dk, float* dvv, int B, int H, int T,
                     int d, int dv, int C, int g, kata_dtype_t dtype, void* workspace,
                     size_t workspace_bytes, hipEvent_t* ev, hipStream_t stream,
                     const float* den = nullptr) {
  if (!bwd_ptrs_ok(q, k, v, out, dout, dq, dk, dvv)) return KATA_ERR_INVALID_ARG;
  if (den && !aligned16(den)) return KATA_ERR_INVALID_ARG;
  const kata_status_t c = bwd_check(B, H, T, d, dv, C, g, dtype);
  if (c != KATA_OK) return c;
  if (!workspace || (reinterpret_cast<uintptr_t>(workspace) & 255u) != 0) return KATA_ERR_INVALID_ARG;
  if (workspace_bytes < kata::bwd_workspace(B * H, T, d, dv, C, g)) return KATA_ERR_INVALID_ARG;
  const int BH = B * H;
  if (dtype == KATA_F32)
    return from_hip(kata::launch_bwd<float>(q, k, v, out, dout, den, dq, dk, dvv, BH, T, d, dv, C,
                                            g, workspace, stream, ev));
  return from_hip(kata::launch_bwd<kata::bf16_t>(q, k, v, out, dout, den, dq, dk, dvv, BH, T, d,
                                                 dv, C, g, workspace, stream, ev));
}

// Enum arguments arrive from C callers as plain ints and may hold any value;
// in C++ an enum object outside its enumerators' range must not be read as
// that enum type, so the entry points look at their bits first.
template <typename E>
int enum_bits(const E& e) {
  static_assert(sizeof(E) == sizeof(int), "enums of the C ABI are int-sized");
  int v;
  std::memcpy(&v, &e, sizeof v);
  return v;
}
bool dtype_ok(const kata_dtype_t& t) {
  const int v = enum_bits(t);
  return v == KATA_F32 || v == KATA_BF16;
}
bool feature_ok(const kata_lin_feature_t& f) {
  const int v = enum_bits(f);
  return v >= KATA_LIN_IDENTITY && v <= KATA_LIN_LORENTZ_S;
}

}  // namespace

extern "C" {

int kata_abi_version(void) { return 106; }

const char* kata_status_string(kata_status_t s) {
  switch (enum_bits(s)) {
    case KATA_OK: return "KATA_OK";
    case KATA_ERR_INVALID_ARG: return "KATA_ERR_INVALID_ARG";
    case KATA_ERR_UNSUPPORTED: return "KATA_ERR_UNSUPPORTED";
    case KATA_ERR_HIP: return "KATA_ERR_HIP";
  }
  return "KATA_UNKNOWN_STATUS";
}

// ---- KATA-M1 ----------------------------------------------------------------

int kata_fwd_default_span(int B, int H, int T, int d, int dv, int C, kata_dtype_t dtype) {
  if (!dtype_ok(dtype)) return 0;
  return default_span_of(B, H, T, d, dv, C, dtype, 1);
}

size_t kata_fwd_workspace_bytes(int B, int H, int T, int d, int dv, int C, kata_dtype_t dtype,
                                int span_chunks) {
  if (!dtype_ok(dtype)) return 0;
  return fwd_workspace_bytes(B, H, T, d, dv, C, dtype, 1, span_chunks);
}

kata_status_t kata_fwd_chunked_ws(const void* q, const void* k, const void* v, float* out, int B,
                                  int H, int T, int d, int dv, int C, kata_dtype_t dtype,
                                  int span_chunks, void* workspace, size_t workspace_bytes,
                                  hipStream_t stream) {
  if (!dtype_ok(dtype)) return KATA_ERR_INVALID_ARG;
  return fwd_ws(q, k, v, out, B, H, T, d, dv, C, 1, dtype, span_chunks, workspace,
                workspace_bytes, nullptr, stream);
}

kata_status_t kata_fwd_chunked_train_ws(const void* q, const void* k, const void* v, float* out,
                                        float* den, int B, int H, int T, int d, int dv, int C,
                                        kata_dtype_t dtype, int span_chunks, void* workspace,
                                        size_t workspace_bytes, hipStream_t stream) {
  if (!dtype_ok(dtype)) return KATA_ERR_INVALID_ARG;
  if (!den) return KATA_ERR_INVALID_ARG;
  return fwd_ws(q, k, v, out, B, H, T, d, dv, C, 1, dtype, span_chunks, workspace,
                workspace_bytes, nullptr, stream, den);
}

kata_status_t kata_fwd_chunked_timed(const void* q, const void* k, const void* v, float* out,
                                     int B, int H, int T, int d, int dv, int C,
                                     kata_dtype_t dtype, int span_chunks, void* workspace,
                                     size_t workspace_bytes, hipEvent_t* stage_events,
                                     hipStream_t stream) {
  if (!dtype_ok(dtype)) return KATA_ERR_INVALID_ARG;
  return fwd_timed(q, k, v, out, B, H, T, d, dv, C, 1, dtype, span_chunks, workspace,
                   workspace_bytes, stage_events, stream);
}

kata_status_t kata_fwd_chunked(const void* q, const void* k, const void* v, float* out, int B,
                               int H, int T, int d, int dv, int C, kata_dtype_t dtype,
                               hipStream_t stream) {
  if (!dtype_ok(dtype)) return KATA_ERR_INVALID_ARG;
  return fwd_alloc(q, k, v, out, B, H, T, d, dv, C, 1, dtype, stream);
}

kata_status_t kata_fwd_chunked_noalloc(const void* q, const void* k, const void* v, float* out,
                                       int B, int H, int T, int d, int dv, int C,
                                       kata_dtype_t dtype, hipStream_t stream) {
  if (!dtype_ok(dtype)) return KATA_ERR_INVALID_ARG;
  return fwd_noalloc(q, k, v, out, B, H, T, d, dv, C, 1, dtype, stream);
}

size_t kata_noalloc_scratch_bytes(void) { return kNoAllocScratchBytes; }

size_t kata_fwd_quadratic_workspace_bytes(int B, int H, int T, int d, int dv, kata_dtype_t dtype) {
  if (!dtype_ok(dtype)) return 0;
  return quad_workspace_bytes(B, H, T, d, dv, dtype, 1);
}

kata_status_t kata_fwd_quadratic_ws(const void* q, const void* k, const void* v, float* out, int B,
                                    int H, int T, int d, int dv, kata_dtype_t dtype,
                                    void* workspace, size_t workspace_bytes, hipStream_t stream) {
  if (!dtype_ok(dtype)) return KATA_ERR_INVALID_ARG;
  return quad_ws(q, k, v, out, B, H, T, d, dv, 1, dtype, workspace, workspace_bytes, stream);
}

kata_status_t kata_fwd_quadratic(const void* q, const void* k, const void* v, float* out, int B,
                                 int H, int T, int d, int dv, kata_dtype_t dtype,
                                 hipStream_t stream) {
  if (!dtype_ok(dtype)) return KATA_ERR_INVALID_ARG;
  if (!q || !k || !v || !out) return KATA_ERR_INVALID_ARG;
  if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(out)) return KATA_ERR_INVALID_ARG;
  const kata_status_t c = quad_check(B, H, T, d, dv, dtype, 1);
  if (c != KATA_OK) return c;
  const size_t bytes = kata::mfma_quadratic_workspace(B * H, T, dv);
  void* ws = nullptr;
  if (alloc_ws(&ws, bytes, stream) != KATA_OK) return KATA_ERR_HIP;
  const kata_status_t st = quad_ws(q, k, v, out, B, H, T, d, dv, 1, dtype, ws, bytes, stream);
  const hipError_t fe = hipFreeAsync(ws, stream);
  if (st != KATA_OK) return st;
  return from_hip(fe);
}

kata_status_t kata_prefill_state(const void* k, const void* v, float* S, float* z, int B, int H,
                                 int T, int d, int dv, kata_dtype_t dtype, hipStream_t stream) {
  if (!dtype_ok(dtype)) return KATA_ERR_INVALID_ARG;
  return prefill(k, v, S, z, B, H, T, d, dv, 1, dtype, stream);
}

kata_status_t kata_decode_step(float* S, float* z, const void* q, const void* k, const void* v,
                               float* out, int B, int H, int d, int dv, kata_dtype_t dtype,
                               hipStream_t stream) {
  if (!dtype_ok(dtype)) return KATA_ERR_INVALID_ARG;
  return decode(S, z, q, k, v, out, B, H, d, dv, 1, dtype, stream);
}

// ---- KATA-Mg -----------------------------------------------------------------

size_t kata_mg_fwd_workspace_bytes(int B, int H, int T, int d, int dv, int C, int g,
                                   kata_dtype_t dtype, int span_chunks) {
  if (!dtype_ok(dtype)) return 0;
  return fwd_workspace_bytes(B, H, T, d, dv, C, dtype, g, span_chunks);
}

kata_status_t kata_mg_fwd_chunked_ws(const void* q, const void* k, const void* v, float* out,
                                     int B, int H, int T, int d, int dv, int C, int g,
                                     kata_dtype_t dtype, int span_chunks, void* workspace,
                                     size_t workspace_bytes, hipStream_t stream) {
  if (!dtype_ok(dtype)) return KATA_ERR_INVALID_ARG;
  return fwd_ws(q, k, v, out, B, H, T, d, dv, C, g, dtype, span_chunks, workspace,
                workspace_bytes, nullptr, stream);
}

kata_status_t kata_mg_fwd_chunked_timed(const void* q, const void* k, const void* v, float* out,
                                        int B, int H, int T, int d, int dv, int C, int g,
                                        kata_dtype_t dtype, int span_chunks, void* workspace,
                                        size_t workspace_bytes, hipEvent_t* stage_events,
                                        hipStream_t stream) {
  if (!dtype_ok(dtype)) return KATA_ERR_INVALID_ARG;
  return fwd_timed(q, k, v, out, B, H, T, d, dv, C, g, dtype, span_chunks, workspace,
                   workspace_bytes, stage_events, stream);
}

kata_status_t kata_mg_fwd_chunked(const void* q, const void* k, const void* v, float* out, int B,
                                  int H, int T, int d, int dv, int C, int g, kata_dtype_t dtype,
                                  hipStream_t stream) {
  if (!dtype_ok(dtype)) return KATA_ERR_INVALID_ARG;
  return fwd_alloc(q, k, v, out, B, H, T, d, dv, C, g, dtype, stream);
}

size_t kata_mg_fwd_quadratic_workspace_bytes(int B, int H, int T, int d, int dv, int g,
                                             kata_dtype_t dtype) {
  if (!dtype_ok(dtype)) return 0;
  return quad_workspace_bytes(B, H, T, d, dv, dtype, g);
}

kata_status_t kata_mg_fwd_quadratic_ws(const void* q, const void* k, const void* v, float* out,
                                       int B, int H, int T, int d, int dv, int g,
                                       kata_dtype_t dtype, void* workspace,
                                       size_t workspace_bytes, hipStream_t stream) {
  if (!dtype_ok(dtype)) return KATA_ERR_INVALID_ARG;
  return quad_ws(q, k, v, out, B, H, T, d, dv, g, dtype, workspace, workspace_bytes, stream);
}

kata_status_t kata_mg_prefill_state(const void* k, const void* v, float* S, float* z, int B, int H,
                                    int T, int d, int dv, int g, kata_dtype_t dtype,
                                    hipStream_t stream) {
  if (!dtype_ok(dtype)) return KATA_ERR_INVALID_ARG;
  return prefill(k, v, S, z, B, H, T, d, dv, g, dtype, stream);
}

kata_status_t kata_mg_decode_step(float* S, float* z, const void* q, const void* k, const void* v,
                                  float* out, int B, int H, int d, int dv, int g,
                                  kata_dtype_t dtype, hipStream_t stream) {
  if (!dtype_ok(dtype)) return KATA_ERR_INVALID_ARG;
  return decode(S, z, q, k, v, out, B, H, d, dv, g, dtype, stream);
}

// ---- linear features -----------------------------------------------------------

int kata_lin_dim(int d, kata_lin_feature_t feature) {
  if (!feature_ok(feature)) return 0;
  if (d < 1 || feature < KATA_LIN_IDENTITY || feature > KATA_LIN_LORENTZ_S) return 0;
  return kata::lin_dim(d, feature);
}

int kata_lin_default_span(int B, int H, int T, int d, int dv, int C, kata_lin_feature_t feature,
                          kata_dtype_t dtype) {
  if (!dtype_ok(dtype)) return 0;
  if (!feature_ok(feature)) return 0;
  const Path p = lin_path(B, H, T, d, dv, C, feature, 0.f, 1, dtype);
  if (p == Path::kInvalid || p == Path::kUnsupported) return 0;
  return lin_default_span(B, H, T, C, p);
}

size_t kata_lin_fwd_workspace_bytes(int B, int H, int T, int d, int dv, int C,
                                    kata_lin_feature_t feature, kata_dtype_t dtype,
                                    int span_chunks) {
  if (!dtype_ok(dtype)) return 0;
  if (!feature_ok(feature)) return 0;
  const Path p = lin_path(B, H, T, d, dv, C, feature, 0.f, 1, dtype);
  if (p == Path::kInvalid || p == Path::kUnsupported || span_chunks < 0) return 0;
  if (span_chunks == 0) span_chunks = lin_default_span(B, H, T, C, p);
  if (p == Path::kFp32) span_chunks = 1;
  return lin_workspace_for(p, B, H, T, d, dv, C, feature, span_chunks);
}

kata_status_t kata_lin_fwd_chunked_ws(const void* q, const void* k, const void* v, float* out,
                                      int B, int H, int T, int d, int dv, int C,
                                      kata_lin_feature_t feature, float eps, int normalize,
                                      kata_dtype_t dtype, int span_chunks, void* workspace,
                                      size_t workspace_bytes, hipStream_t stream) {
  if (!dtype_ok(dtype)) return KATA_ERR_INVALID_ARG;
  if (!feature_ok(feature)) return KATA_ERR_INVALID_ARG;
  return lin_ws(q, k, v, out, B, H, T, d, dv, C, feature, eps, normalize, dtype, span_chunks,
                workspace, workspace_bytes, nullptr, stream);
}

kata_status_t kata_lin_fwd_chunked_timed(const void* q, const void* k, const void* v, float* out,
                                         int B, int H, int T, int d, int dv, int C,
                                         kata_lin_feature_t feature, float eps, int normalize,
                                         kata_dtype_t dtype, int span_chunks, void* workspace,
                                         size_t workspace_bytes, hipEvent_t* stage_events,
                                         hipStream_t stream) {
  if (!dtype_ok(dtype)) return KATA_ERR_INVALID_ARG;
  if (!feature_ok(feature)) return KATA_ERR_INVALID_ARG;
  if (!stage_events) return KATA_ERR_INVALID_ARG;
  for (int i = 0; i < 4; ++i)
    if (!stage_events[i]) return KATA_ERR_INVALID_ARG;
  return lin_ws(q, k, v, out, B, H, T, d, dv, C, feature, eps, normalize, dtype, span_chunks,
                workspace, workspace_bytes, stage_events, stream);
}

kata_status_t kata_lin_fwd_chunked(const void* q, const void* k, const void* v, float* out, int B,
                                   int H, int T, int d, int dv, int C, kata_lin_feature_t feature,
                                   float eps, int normalize, kata_dtype_t dtype,
                                   hipStream_t stream) {
  if (!dtype_ok(dtype)) return KATA_ERR_INVALID_ARG;
  if (!feature_ok(feature)) return KATA_ERR_INVALID_ARG;
  if (!q || !k || !v || !out) return KATA_ERR_INVALID_ARG;
  if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(out)) return KATA_ERR_INVALID_ARG;
  const Path p = lin_path(B, H, T, d, dv, C, feature, eps, normalize, dtype);
  if (p == Path::kInvalid) return KATA_ERR_INVALID_ARG;
  if (p == Path::kUnsupported) return KATA_ERR_UNSUPPORTED;
  const int span = lin_default_span(B, H, T, C, p);
  const size_t bytes = lin_workspace_for(p, B, H, T, d, dv, C, feature, span);
  void* ws = nullptr;
  if (alloc_ws(&ws, bytes, stream) != KATA_OK) return KATA_ERR_HIP;
  const kata_status_t st = lin_ws(q, k, v, out, B, H, T, d, dv, C, feature, eps, normalize, dtype,
                                  span, ws, bytes, nullptr, stream);
  const hipError_t fe = hipFreeAsync(ws, stream);
  if (st != KATA_OK) return st;
  return from_hip(fe);
}

// ---- backward -------------------------------------------------------------------

size_t kata_bwd_workspace_bytes(int B, int H, int T, int d, int dv, int C, int g,
                                kata_dtype_t dtype) {
  if (!dtype_ok(dtype)) return 0;
  if (bwd_check(B, H, T, d, dv, C, g, dtype) != KATA_OK) return 0;
  return kata::bwd_workspace(B * H, T, d, dv, C, g);
}

int kata_bwd_fused_scan(int B, int H, int T, int d, int dv, int C, int g, kata_dtype_t dtype) {
  if (!dtype_ok(dtype)) return -1;
  if (bwd_check(B, H, T, d, dv, C, g, dtype) != KATA_OK) return -1;
  return kata::bwd_fused_scan(B * H, d, dv, C, g, dtype == KATA_BF16) ? 1 : 0;
}

kata_status_t kata_bwd_chunked_ws(const void* q, const void* k, const void* v, const float* out,
                                  const float* dout, float* dq, float* dk, float* dv_out, int B,
                                  int H, int T, int d, int dv, int C, int g, kata_dtype_t dtype,
                                  void* workspace, size_t workspace_bytes, hipStream_t stream) {
  if (!dtype_ok(dtype)) return KATA_ERR_INVALID_ARG;
  return bwd_ws(q, k, v, out, dout, dq, dk, dv_out, B, H, T, d, dv, C, g, dtype, workspace,
                workspace_bytes, nullptr, stream);
}

kata_status_t kata_bwd_chunked_timed(const void* q, const void* k, const void* v,
                                     const float* out, const float* dout, float* dq, float* dk,
                                     float* dv_out, int B, int H, int T, int d, int dv, int C,
                                     int g, kata_dtype_t dtype, void* workspace,
                                     size_t workspace_bytes, hipEvent_t* stage_events,
                                     hipStream_t stream) {
  if (!dtype_ok(dtype)) return KATA_ERR_INVALID_ARG;
  if (!stage_events) return KATA_ERR_INVALID_ARG;
  for (int i = 0; i < 7; ++i)
    if (!stage_events[i]) return KATA_ERR_INVALID_ARG;
  return bwd_ws(q, k, v, out, dout, dq, dk, dv_out, B, H, T, d, dv, C, g, dtype, workspace,
                workspace_bytes, stage_events, stream);
}

kata_status_t kata_bwd_chunked_ex(const void* q, const void* k, const void* v, const float* out,
                                  const float* dout, const float* den, float* dq, float* dk,
                                  float* dv_out, int B, int H, int T, int d, int dv, int C, int g,
                                  kata_dtype_t dtype, void* workspace, size_t workspace_bytes,
                                  hipEvent_t* stage_events, hipStream_t stream) {
  if (!dtype_ok(dtype)) return KATA_ERR_INVALID_ARG;
  if (stage_events)
    for (int i = 0; i < 7; ++i)
      if (!stage_events[i]) return KATA_ERR_INVALID_ARG;
  return bwd_ws(q, k, v, out, dout, dq, dk, dv_out, B, H, T, d, dv, C, g, dtype, workspace,
                workspace_bytes, stage_events, stream, den);
}

kata_status_t kata_bwd_chunked(const void* q, const void* k, const void* v, const float* out,
                               const float* dout, float* dq, float* dk, float* dv_out, int B,
                               int H, int T, int d, int dv, int C, int g, kata_dtype_t dtype,
                               hipStream_t stream) {
  if (!dtype_ok(dtype)) return KATA_ERR_INVALID_ARG;
  if (!bwd_ptrs_ok(q, k, v, out, dout, dq, dk, dv_out)) return KATA_ERR_INVALID_ARG;
  const kata_status_t c = bwd_check(B, H, T, d, dv, C, g, dtype);
  if (c != KATA_OK) return c;
  const size_t bytes = kata::bwd_workspace(B * H, T, d, dv, C, g);
  void* ws = nullptr;
  if (alloc_ws(&ws, bytes, stream) != KATA_OK) return KATA_ERR_HIP;
  const kata_status_t st = bwd_ws(q, k, v, out, dout, dq, dk, dv_out, B, H, T, d, dv, C, g, dtype,
                                  ws, bytes, nullptr, stream);
  const hipError_t fe = hipFreeAsync(ws, stream);
  if (st != KATA_OK) return st;
  return from_hip(fe);
}

}  // extern "C"
