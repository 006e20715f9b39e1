/*
 * kata.h -- C ABI of libkata: causal KATA-M1 attention (rank-one PSD feature
 * map), and its block-diagonal KATA-Mg variant, on AMD Instinct MI355X (gfx950).
 *
 * The operation.  For every head, with query q_t, key k_t in R^d and value v_t
 * in R^dv, the feature map is the rank-one PSD lift phi(x) = vec(x x^T)
 * (section "Rank-one packing into the PSD cone"), whose inner product is
 * <phi(q), phi(k)> = (q . k)^2.  Normalised causal linear attention
 * (eq. linatt) with this map gives
 *
 *     o_t = sum_{i<=t} (q_t . k_i)^2 v_i  /  sum_{i<=t} (q_t . k_i)^2 ,
 *
 * a convex combination of the values (output-gate proposition).  A row whose
 * denominator is 0 (q_t orthogonal to every k_i, i <= t, e.g. q_t = 0) is
 * defined as all zeros; the paper leaves it undefined.
 *
 * Conventions shared by every entry point:
 *  - Tensors are contiguous, row-major, device-resident (HBM), 16-byte aligned:
 *      q, k : [B][H][T][d]     v : [B][H][T][dv]     out : [B][H][T][dv] fp32.
 *    q, k, v are fp32 or bf16 (kata_dtype_t); out, S and z are always fp32.
 *  - The caller owns every buffer.  `out` must not alias an input.
 *  - Every call validates its arguments on the host before touching the GPU;
 *    on an error nothing is launched and nothing is written.
 *  - Calls only enqueue work on `stream` and return; they never synchronise.
 *    A device fault surfaces at the caller's next synchronisation.
 *  - The calls that take a caller workspace (the _ws and _timed variants),
 *    kata_fwd_chunked_noalloc, kata_prefill_state and kata_decode_step
 *    enqueue kernel launches only (and the _timed variants event records), so
 *    a caller may capture them into a HIP graph and replay it; the variants
 *    without a workspace argument allocate theirs stream-ordered
 *    (hipMallocAsync / hipFreeAsync) on `stream`.
 *  - The library keeps no global mutable state (except the scratch array of
 *    kata_fwd_chunked_noalloc, see there); calls from several threads are
 *    safe.  NaN and Inf in inputs propagate; inputs are not normalised.
 *  - Packed state layout (decode and prefill): the n = d(d+1)/2 features of
 *    the pair (a, b), a <= b, in row-major upper-triangle order,
 *        f(a, b) = a*d - a*(a-1)/2 + (b - a),
 *    S : [B][H][n][dv] holds sum_i k_a k_b v_i (unscaled), z : [B][H][n]
 *    holds sum_i k_a k_b.
 */
#ifndef KATA_H
#define KATA_H

#include <stddef.h>
#include <hip/hip_runtime_api.h>

#ifndef KATA_API
#define KATA_API __attribute__((visibility("default")))
#endif

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  KATA_OK = 0,
  KATA_ERR_INVALID_ARG = 1, /* null pointer, size < 1, or a size product overflows */
  KATA_ERR_UNSUPPORTED = 2, /* valid arguments outside what is implemented */
  KATA_ERR_HIP = 3          /* a HIP launch or allocation failed */
} kata_status_t;

typedef enum { KATA_F32 = 0, KATA_BF16 = 1 } kata_dtype_t;

/*
 * Causal KATA-M1 forward in the exact O(T) chunked-state form (eq. chunk-SZ,
 * eq. chunk-out and the chunkwise algorithm of the appendix; the three-stage
 * state / associative-scan / output pipeline of the tree-scan section).
 * The final chunk is zero-padded on chip and the output is truncated to T rows.
 *   q, k, v, out : see the conventions above.
 *   B, H, T >= 1.  d in 1..64.  dv >= 1.  C >= 1 is the chunk size.
 *   Fast path (bf16 MFMA): dtype = KATA_BF16, d in {32, 64}, dv = 64,
 *   C a multiple of 32 up to 1024.  Every other shape with d <= 64, dv <= 256
 *   and C <= 128 runs on the fp32 path; anything else is KATA_ERR_UNSUPPORTED.
 *   Workspace (kata_fwd_workspace_bytes) is allocated stream-ordered with
 *   hipMallocAsync on `stream` and released with hipFreeAsync.
 */
KATA_API kata_status_t kata_fwd_chunked(const void* q, const void* k, const void* v, float* out,
                               int B, int H, int T, int d, int dv, int C,
                               kata_dtype_t dtype, hipStream_t stream);

/*
 * kata_fwd_chunked for callers that cannot allocate device memory: code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc.
 * Same arguments, default span and results as kata_fwd_chunked; it calls no
 * hipMalloc / hipFree or allocating library routine.  Its workspace is a
 * library-owned device array of kata_noalloc_scratch_bytes() bytes (256 MiB),
 * one per GPU, held by every GPU the library runs on until the process ends;
 * the first call on a device looks up that device's copy (the stream's device;
 * the current device for the null stream).
 *   Returns KATA_ERR_UNSUPPORTED when the workspace kata_fwd_chunked would
 *   allocate (kata_fwd_workspace_bytes at the default span) exceeds the array,
 *   e.g. B*H*T above about 650k head-tokens at d = dv = 64 on the bf16 path.
 *   Every call on one GPU shares that GPU's array and leaves its contents
 *   behind: calls that overlap on one GPU (different streams, or host
 *   threads) race and give undefined results.  No kernel reads scratch that
 *   the same call has not written, so nothing is cleared between calls.
 */
KATA_API kata_status_t kata_fwd_chunked_noalloc(const void* q, const void* k, const void* v,
                                                float* out, int B, int H, int T, int d, int dv,
                                                int C, kata_dtype_t dtype, hipStream_t stream);

/* Size in bytes of the per-device scratch array of kata_fwd_chunked_noalloc. */
KATA_API size_t kata_noalloc_scratch_bytes(void);

/*
 * The same forward with caller-provided workspace and an explicit span.
 *   span_chunks : number of chunks folded into one stored state (the state
 *                 written to HBM covers span_chunks*C tokens; the chunks inside
 *                 a span are combined on chip).  0 selects the default
 *                 (kata_fwd_default_span).  1 is the per-chunk form.  Results do
 *                 not depend on it beyond rounding.
 *   workspace   : device buffer of at least kata_fwd_workspace_bytes(...)
 *                 bytes, 256-byte aligned, owned by the caller, contents
 *                 ignored on entry and undefined on exit.  Two calls in flight
 *                 at once must not share it.
 */
KATA_API kata_status_t kata_fwd_chunked_ws(const void* q, const void* k, const void* v, float* out,
                                  int B, int H, int T, int d, int dv, int C,
                                  kata_dtype_t dtype, int span_chunks, void* workspace,
                                  size_t workspace_bytes, hipStream_t stream);

/*
 * kata_fwd_chunked_ws plus stage timing, for profiling: stage_events[0..3]
 * (caller-created HIP events, all non-null) are recorded on `stream` before the
 * state kernel and after each of the three stages (chunk or span state,
 * associative scan, output).  Nothing synchronises; the caller reads the
 * elapsed times with hipEventElapsedTime once the stream has reached them.
 */
KATA_API kata_status_t kata_fwd_chunked_timed(const void* q, const void* k, const void* v,
                                              float* out, int B, int H, int T, int d, int dv,
                                              int C, kata_dtype_t dtype, int span_chunks,
                                              void* workspace, size_t workspace_bytes,
                                              hipEvent_t* stage_events, hipStream_t stream);

/*
 * kata_fwd_chunked_ws for a training step: it also writes each row's
 * denominator D_t = sum_{i<=t} (q_t . k_i)^2 (the normaliser of eq. linatt,
 * fp32 as the forward computed it) to den, fp32 [B][H][T], caller-owned,
 * 16-byte aligned, for kata_bwd_chunked_ex, which then need not form it again
 * from the prefix states.  Supported on the bf16 MFMA path (the shapes of
 * kata_fwd_chunked_ws with dtype KATA_BF16, d in {32, 64}, dv = 64, C a
 * multiple of 32); other valid arguments give KATA_ERR_UNSUPPORTED.  den null:
 * KATA_ERR_INVALID_ARG.
 */
KATA_API kata_status_t kata_fwd_chunked_train_ws(const void* q, const void* k, const void* v,
                                                 float* out, float* den, int B, int H, int T,
                                                 int d, int dv, int C, kata_dtype_t dtype,
                                                 int span_chunks, void* workspace,
                                                 size_t workspace_bytes, hipStream_t stream);

/* Workspace bytes kata_fwd_chunked_ws needs for these arguments (0 when the
 * arguments are invalid or unsupported). */
KATA_API size_t kata_fwd_workspace_bytes(int B, int H, int T, int d, int dv, int C,
                                kata_dtype_t dtype, int span_chunks);

/* The span (in chunks) that span_chunks = 0 selects for these arguments. */
KATA_API int kata_fwd_default_span(int B, int H, int T, int d, int dv, int C, kata_dtype_t dtype);

/*
 * The same causal KATA-M1 forward in the quadratic (flash-style) form: the
 * O(T^2) definition above evaluated in 32x32 query-key blocks on chip
 * (squared scores, causal mask, P V and the row sums), never forming a
 * feature state (section "Synthetic induction and hardware microbenchmarks",
 * paragraph "Kernel latency and throughput ratios": the quadratic operating
 * point, preferable to the O(T) form at short T).  Same outputs as
 * kata_fwd_chunked up to rounding.
 *   Supported: dtype = KATA_BF16, d in {32, 64}, dv = 64 (bf16 MFMA);
 *   other valid arguments give KATA_ERR_UNSUPPORTED.  B*H <= 65535.
 *   workspace : device buffer of at least kata_fwd_quadratic_workspace_bytes(...)
 *               bytes, 256-byte aligned, caller-owned (it receives a permuted
 *               bf16 copy of V^T), contents undefined on exit.
 * kata_fwd_quadratic allocates that workspace stream-ordered (hipMallocAsync /
 * hipFreeAsync on `stream`).
 */
KATA_API kata_status_t kata_fwd_quadratic(const void* q, const void* k, const void* v, float* out,
                                          int B, int H, int T, int d, int dv,
                                          kata_dtype_t dtype, hipStream_t stream);
KATA_API kata_status_t kata_fwd_quadratic_ws(const void* q, const void* k, const void* v,
                                             float* out, int B, int H, int T, int d, int dv,
                                             kata_dtype_t dtype, void* workspace,
                                             size_t workspace_bytes, hipStream_t stream);
/* Workspace bytes kata_fwd_quadratic_ws needs (0 when the arguments are
 * invalid or unsupported). */
KATA_API size_t kata_fwd_quadratic_workspace_bytes(int B, int H, int T, int d, int dv,
                                                   kata_dtype_t dtype);

/*
 * State after T tokens by the additive recurrence of eq. linatt:
 *   S = sum_{t<T} phi(k_t) v_t^T,  z = sum_{t<T} phi(k_t)   (packed layout above).
 * Overwrites S : [B][H][n][dv] and z : [B][H][n] (fp32).  Products k_a k_b and
 * the sums are formed in fp32.  Bridges a prefill to kata_decode_step.
 *   k, v : [B][H][T][d], [B][H][T][dv];  d in 1..64, dv in 1..256.
 */
KATA_API kata_status_t kata_prefill_state(const void* k, const void* v, float* S, float* z,
                                 int B, int H, int T, int d, int dv,
                                 kata_dtype_t dtype, hipStream_t stream);

/*
 * One recurrent decode step for all B*H heads (eq. linatt's recurrence and its
 * normalised readout, using the updated state so the current token counts, as
 * in the forward):
 *   S <- S + phi(k) v^T,  z <- z + phi(k),  out = phi(q)^T S / phi(q)^T z.
 *   S : [B][H][n][dv] fp32 and z : [B][H][n] fp32, updated in place (packed
 *       layout above; caller-owned, so a failed step can be retried from the
 *       caller's copy).
 *   q, k : [B][H][d], v : [B][H][dv] in `dtype`;  out : [B][H][dv] fp32.
 *   d in 1..64, dv in 1..256.  State arithmetic is fp32.
 */
KATA_API kata_status_t kata_decode_step(float* S, float* z, const void* q, const void* k,
                               const void* v, float* out, int B, int H, int d, int dv,
                               kata_dtype_t dtype, hipStream_t stream);

/*
 * KATA-Mg, the block-diagonal PSD feature (section "From rank-one rays to
 * low-rank PSD packing").  Each query and key is split into g blocks of
 * m = d/g consecutive coordinates, u = (u_1, ..., u_g), and the feature keeps
 * one rank-one factor per block, psi(u) = (u_1 u_1^T, ..., u_g u_g^T), so
 *
 *     o_t = sum_{i<=t} w_ti v_i / sum_{i<=t} w_ti,   w_ti = sum_a (q_{t,a} . k_{i,a})^2 .
 *
 * g = 1 is KATA-M1 (the calls above).  g >= 1 must divide d, else
 * KATA_ERR_INVALID_ARG.  Packed state layout (prefill, decode): n = g*m(m+1)/2
 * features; block a's pair (i, j), i <= j < m, at a*m(m+1)/2 + f_m(i, j)
 * (the M1 order over m coordinates); S : [B][H][n][dv], z : [B][H][n].
 * Forward fast path (bf16 MFMA): dtype = KATA_BF16, dv = 64, C a multiple of
 * 32 up to 1024 and (d, g) in {(64, 1), (64, 2), (32, 1)}; other shapes with
 * d <= 64, dv <= 256 and C <= 128 run on the fp32 path.  The quadratic form
 * exists on the fast path only.  Arguments, workspace ownership, errors and
 * asynchrony otherwise as for the M1 call of the same name.
 */
KATA_API kata_status_t kata_mg_fwd_chunked(const void* q, const void* k, const void* v,
                                           float* out, int B, int H, int T, int d, int dv, int C,
                                           int g, kata_dtype_t dtype, hipStream_t stream);
KATA_API kata_status_t kata_mg_fwd_chunked_ws(const void* q, const void* k, const void* v,
                                              float* out, int B, int H, int T, int d, int dv,
                                              int C, int g, kata_dtype_t dtype, int span_chunks,
                                              void* workspace, size_t workspace_bytes,
                                              hipStream_t stream);
KATA_API kata_status_t kata_mg_fwd_chunked_timed(const void* q, const void* k, const void* v,
                                                 float* out, int B, int H, int T, int d, int dv,
                                                 int C, int g, kata_dtype_t dtype,
                                                 int span_chunks, void* workspace,
                                                 size_t workspace_bytes,
                                                 hipEvent_t* stage_events, hipStream_t stream);
KATA_API size_t kata_mg_fwd_workspace_bytes(int B, int H, int T, int d, int dv, int C, int g,
                                            kata_dtype_t dtype, int span_chunks);
KATA_API kata_status_t kata_mg_fwd_quadratic_ws(const void* q, const void* k, const void* v,
                                                float* out, int B, int H, int T, int d, int dv,
                                                int g, kata_dtype_t dtype, void* workspace,
                                                size_t workspace_bytes, hipStream_t stream);
KATA_API size_t kata_mg_fwd_quadratic_workspace_bytes(int B, int H, int T, int d, int dv, int g,
                                                      kata_dtype_t dtype);
KATA_API kata_status_t kata_mg_prefill_state(const void* k, const void* v, float* S, float* z,
                                             int B, int H, int T, int d, int dv, int g,
                                             kata_dtype_t dtype, hipStream_t stream);
KATA_API kata_status_t kata_mg_decode_step(float* S, float* z, const void* q, const void* k,
                                           const void* v, float* out, int B, int H, int d, int dv,
                                           int g, kata_dtype_t dtype, hipStream_t stream);

/*
 * Causal linear attention with a linear (n_psi ~ d) feature map: the orthant
 * maps and the Lorentz lift of section "Classical feature maps", the n_psi = d
 * Lorentz variant of the appendix KATA-Lorentz model, and the plain feature
 * psi(x) = x of the associative-scan measurements (appendix "Associative-scan
 * kernel", table of small-batch associative-scan throughput).  With
 * w_ti = <psi(q_t), psi(k_i)>:
 *     normalize = 1:  o_t = sum_{i<=t} w_ti v_i / sum_{i<=t} w_ti   (eq. linatt),
 *                     and o_t = 0 when the denominator is not positive;
 *     normalize = 0:  o_t = sum_{i<=t} w_ti v_i  (unnormalised; the usual
 *                     choice for KATA_LIN_IDENTITY, whose weights carry a sign).
 * Computed in the three-stage chunk-state / associative-scan / chunk-output
 * form (paragraph "Three-kernel pipeline" of that appendix).
 *   feature : a kata_lin_feature_t; eps (>= 0, finite) is used by
 *             KATA_LIN_RELU only.  n_psi = kata_lin_dim(d, feature).
 *   Fast path (bf16 MFMA): dtype = KATA_BF16, d = dv = 64, every feature, C a
 *   multiple of 64 up to 1024 (KATA_LIN_LORENTZ's extra coordinate ||x|| is
 *   carried as a rank-one fp32 term beside the d x d MFMA state).  Every
 *   other shape with d <= 64, dv <= 256 and C <= 128 runs on the fp32 path;
 *   anything else is KATA_ERR_UNSUPPORTED.
 *   span_chunks, workspace, stage_events: as for kata_fwd_chunked_ws and
 *   kata_fwd_chunked_timed (records of span_chunks * C tokens on the fast
 *   path; one per chunk on the fp32 path).  Tensors, ownership, errors and
 *   asynchrony as in the conventions at the top of this file.
 */
typedef enum {
  KATA_LIN_IDENTITY = 0,  /* psi(x) = x                                  n_psi = d     */
  KATA_LIN_RELU = 1,      /* psi(x) = ReLU(x) + eps                      n_psi = d     */
  KATA_LIN_ELU = 2,       /* psi(x) = ELU(x) + 1                         n_psi = d     */
  KATA_LIN_LORENTZ = 3,   /* psi(x) = (x, ||x||_2)                       n_psi = d + 1 */
  KATA_LIN_LORENTZ_S = 4  /* psi(x) = (y, ||y||_2 (1 + s^2)), y = x_1..x_{d-1},
                             s = x_d                                     n_psi = d     */
} kata_lin_feature_t;

/* n_psi of a feature at width d (0 when d < 1 or the feature is unknown). */
KATA_API int kata_lin_dim(int d, kata_lin_feature_t feature);
KATA_API kata_status_t kata_lin_fwd_chunked(const void* q, const void* k, const void* v,
                                            float* out, int B, int H, int T, int d, int dv,
                                            int C, kata_lin_feature_t feature, float eps,
                                            int normalize, kata_dtype_t dtype,
                                            hipStream_t stream);
KATA_API kata_status_t kata_lin_fwd_chunked_ws(const void* q, const void* k, const void* v,
                                               float* out, int B, int H, int T, int d, int dv,
                                               int C, kata_lin_feature_t feature, float eps,
                                               int normalize, kata_dtype_t dtype,
                                               int span_chunks, void* workspace,
                                               size_t workspace_bytes, hipStream_t stream);
KATA_API kata_status_t kata_lin_fwd_chunked_timed(const void* q, const void* k, const void* v,
                                                  float* out, int B, int H, int T, int d, int dv,
                                                  int C, kata_lin_feature_t feature, float eps,
                                                  int normalize, kata_dtype_t dtype,
                                                  int span_chunks, void* workspace,
                                                  size_t workspace_bytes,
                                                  hipEvent_t* stage_events, hipStream_t stream);
/* Workspace bytes for these arguments (0 when invalid or unsupported). */
KATA_API size_t kata_lin_fwd_workspace_bytes(int B, int H, int T, int d, int dv, int C,
                                             kata_lin_feature_t feature, kata_dtype_t dtype,
                                             int span_chunks);
/* The span (in chunks) that span_chunks = 0 selects (0 when invalid or unsupported). */
KATA_API int kata_lin_default_span(int B, int H, int T, int d, int dv, int C,
                                   kata_lin_feature_t feature, kata_dtype_t dtype);

/*
 * Backward of the causal KATA-Mg forward (g = 1: KATA-M1) in the O(T)
 * chunked form: the chunked backward of the appendix's chunkwise algorithm (a
 * reverse scan over chunks carrying the state cotangent, forward quantities
 * recomputed from chunk-boundary states, the feature-map VJP
 * dx = (dPsi + dPsi^T) x closing the chain).  For output cotangents
 * dout = dL/do it returns
 *     dq = dL/dq, dk = dL/dk, dv_out = dL/dv,
 * with a_t = dout_t / D_t, b_t = -<dout_t, o_t> / D_t, dL/dw_ti = <a_t, v_i> + b_t
 * (i <= t), w_ti = sum_blk (q_t,blk . k_i,blk)^2.  A row with D_t = 0 (whose
 * readout is the constant 0) passes no gradient.
 *   q, k, v : the forward's inputs (dtype), out : its fp32 output
 *             [B][H][T][dv] (kata_fwd_chunked or kata_mg_fwd_chunked), dout :
 *             fp32 [B][H][T][dv]; dq, dk : fp32 [B][H][T][d], dv_out : fp32
 *             [B][H][T][dv], overwritten, none aliasing an input.
 *   Supported: d <= 64, dv <= 256, C <= 64, g | d, fp32 or bf16 inputs.  Else
 *   KATA_ERR_UNSUPPORTED (shape) or KATA_ERR_INVALID_ARG.
 *   Arithmetic: fp32 throughout, except for bf16 inputs with d = dv = C = 64
 *   and g = 1, where the chunk states, the scanned state records (S rounded to
 *   bf16, z fp32, fp32 sums) and the gradient products run on the bf16 matrix
 *   cores with fp32 accumulation, a_t and b_t entering as bf16 hi + lo pairs;
 *   that path's gradients are within 2e-2 (per-head relative l2) of the exact
 *   ones, about 2e-3 on the test workloads.
 *   workspace : >= kata_bwd_workspace_bytes(...) bytes, 256-byte aligned,
 *   caller-owned, contents undefined on exit; kata_bwd_chunked allocates it
 *   stream-ordered.  stage_events : 7 caller-created events, recorded before
 *   the first launch and after each of the six (forward states, prefix scan,
 *   per-token coefficients, backward states, suffix scan, gradients); where
 *   kata_bwd_fused_scan() is 1 each state launch also writes the scanned
 *   records and the two scan intervals are empty.
 */
KATA_API kata_status_t kata_bwd_chunked(const void* q, const void* k, const void* v,
                                        const float* out, const float* dout, float* dq,
                                        float* dk, float* dv_out, int B, int H, int T, int d,
                                        int dv, int C, int g, kata_dtype_t dtype,
                                        hipStream_t stream);
KATA_API kata_status_t kata_bwd_chunked_ws(const void* q, const void* k, const void* v,
                                           const float* out, const float* dout, float* dq,
                                           float* dk, float* dv_out, int B, int H, int T, int d,
                                           int dv, int C, int g, kata_dtype_t dtype,
                                           void* workspace, size_t workspace_bytes,
                                           hipStream_t stream);
KATA_API kata_status_t kata_bwd_chunked_timed(const void* q, const void* k, const void* v,
                                              const float* out, const float* dout, float* dq,
                                              float* dk, float* dv_out, int B, int H, int T,
                                              int d, int dv, int C, int g, kata_dtype_t dtype,
                                              void* workspace, size_t workspace_bytes,
                                              hipEvent_t* stage_events, hipStream_t stream);
/*
 * kata_bwd_chunked_ws with two optional arguments: den, null or the
 * denominators D_t that kata_fwd_chunked_train_ws wrote for this forward
 * (fp32 [B][H][T], 16-byte aligned), from which the per-token coefficients
 * a_t, b_t are formed directly instead of from the prefix states (same values
 * up to rounding); stage_events, null or 7 events as for
 * kata_bwd_chunked_timed (all non-null).  Any supported backward shape.
 */
KATA_API kata_status_t kata_bwd_chunked_ex(const void* q, const void* k, const void* v,
                                           const float* out, const float* dout, const float* den,
                                           float* dq, float* dk, float* dv_out, int B, int H,
                                           int T, int d, int dv, int C, int g,
                                           kata_dtype_t dtype, void* workspace,
                                           size_t workspace_bytes, hipEvent_t* stage_events,
                                           hipStream_t stream);
KATA_API size_t kata_bwd_workspace_bytes(int B, int H, int T, int d, int dv, int C, int g,
                                         kata_dtype_t dtype);
/* 1 when kata_bwd_chunked* computes the prefix and suffix records of this
 * shape with the state and the scan in one launch each (bf16 inputs at
 * d = dv = C = 64, g = 1, from 16 heads B x H on), 0 when it runs a state launch
 * and a scan launch for each, -1 for an unsupported shape. */
KATA_API int kata_bwd_fused_scan(int B, int H, int T, int d, int dv, int C, int g,
                                 kata_dtype_t dtype);

/* Static, human-readable name of a status code. */
KATA_API const char* kata_status_string(kata_status_t s);

/* ABI version of this header (major*100 + minor). */
KATA_API int kata_abi_version(void);

#ifdef __cplusplus
}
#endif

#endif /* KATA_H */
