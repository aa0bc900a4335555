/*
 * llmv.h -- C ABI of libllmv, batched LLMVisor latency attribution on
 * AMD Instinct MI355X (gfx950).
 *
 * The method (LLMVisor, Sec. 2.1, Eq. 1): a batch B of co-scheduled requests
 * has latency
 *     T_B = beta + a1*sum_i p_i + a2*sum_i c_i + a3*sum_i p_i^2 + a4*sum_i |B|
 * with p_i the tokens request i processes in the step and c_i the context
 * tokens it attends to (Sec. 2.1).  The form has two segments per phase
 * (memory-bound MEM and compute-bound COMP), so four coefficient sets in all
 * (Sec. 2.1).  Because T_B is a sum of per-request terms, each request's
 * share f(i|B) is its own terms, the shares are nonnegative for nonnegative
 * coefficients and add up to T_B, and a tenant's usage L_u is the sum of its
 * requests' shares (Sec. 2, Problem formulation).  Features are scaled by
 * constants proportional to FLOPs and bytes (Sec. 2.1), derived from a model
 * shape (llmv_shape_constants).
 *
 * Readings of points the paper leaves open (the same in every entry point):
 *   - a4 term: |B| per request, |B|^2 per batch (Eq. 1 sums |B| over i);
 *   - beta: split equally, beta*S0/|B| per request;
 *   - segment: COMP when T_COMP > T_MEM (strictly), else MEM; T_B is the
 *     chosen segment's value, i.e. max(T_MEM, T_COMP);
 *   - phase: PREFILL when any request has p_i > 1 or c_i == 0, else DECODE;
 *   - an empty batch has T_B = 0 and regime LLMV_REGIME_EMPTY.
 *
 * Conventions for every entry point below:
 *   - Pointers marked "device" must point to device memory of the current
 *     HIP device; "host" pointers to host memory.  The caller owns all
 *     memory; the library allocates nothing on these paths.  The per-request
 *     arrays (p, c, tenant, share) must be 16-byte aligned (any hipMalloc or
 *     torch allocation is); they are read and written with 16-byte accesses.
 *   - `stream` is a hipStream_t (NULL = the null stream).  Work is enqueued
 *     on it and the call returns without waiting; outputs are valid once the
 *     stream has reached that point.  llmv_validate is the exception: it
 *     waits for its own result.
 *   - `ws` is a device workspace of at least llmv_workspace_size(...) bytes,
 *     256-byte aligned.  Its contents need no initialisation and are
 *     clobbered.  Two calls that overlap in time must not share a workspace.
 *   - Return value: LLMV_OK, or a negative LLMV_E* code.  Host-side argument
 *     checks run before anything is enqueued.  Device data are NOT checked
 *     by the attribution calls: data outside the limits below is undefined
 *     behaviour; check it with llmv_validate.  llmv_last_error() gives a
 *     message for the calling thread's last failure.
 */
#ifndef LLMV_H
#define LLMV_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Return codes. */
#define LLMV_OK 0
#define LLMV_EINVAL (-1)     /* bad host-side argument                        */
#define LLMV_ERANGE (-2)     /* device data outside the limits (llmv_validate) */
#define LLMV_EDEVICE (-3)    /* HIP runtime or launch error                   */
#define LLMV_EWORKSPACE (-4) /* workspace too small or misaligned             */

/* Phase / segment / regime numbering: regime = 2*phase + segment. */
#define LLMV_PREFILL 0
#define LLMV_DECODE 1
#define LLMV_MEM 0
#define LLMV_COMP 1
#define LLMV_REGIME_EMPTY 255

/* Data limits. */
#define LLMV_P_MAX (1 << 20)       /* 1 <= p_i <= 2^20                         */
#define LLMV_BATCH_MAX (1 << 22)   /* 0 <= |B| <= 2^22; c_i is any int32 >= 0  */
#define LLMV_TENANTS_MAX (1 << 24) /* 1 <= n_tenants <= 2^24                   */

/* Model shape (host struct).  Every field must be > 0.  weight_bytes and
 * kv_bytes are bytes per element (2 for bf16). */
typedef struct {
  int32_t n_layers, hidden, n_q_heads, n_kv_heads, head_dim, ffn, vocab,
      weight_bytes, kv_bytes;
} llmv_shape;

/* A trace of batches in CSR form (host struct holding device pointers).
 *   offsets [n_batches+1] int64, device: batch b holds requests
 *           offsets[b] .. offsets[b+1]-1; offsets[0] == 0, non-decreasing,
 *           offsets[n_batches] == n_requests.
 *   p, c    [n_requests] int32, device: tokens processed this step (p_i) and
 *           context tokens attended (c_i), Sec. 2.1.
 *   tenant  [n_requests] int32, device, or NULL when no tenant sums are
 *           requested: 0 <= tenant[i] < n_tenants.                        */
typedef struct {
  int64_t n_batches, n_requests;
  const int64_t *offsets;
  const int32_t *p, *c, *tenant;
} llmv_trace;

/* Host only; enqueues nothing.  Shape constants S[0..3] (host array):
 *   P_layer = hidden*head_dim*(2*Hq + 2*Hkv) + 3*hidden*ffn
 *   S0 = weight_bytes*(n_layers*P_layer + vocab*hidden)  weight bytes per step
 *   S1 = 2*n_layers*P_layer                            linear FLOPs per token
 *   S2 = 2*n_layers*Hkv*head_dim*kv_bytes              KV bytes per context token
 *   S3 = 2*n_layers*Hq*head_dim                        causal attention FLOPs per p^2
 * (Sec. 2.1: features proportional to FLOPs and I/O).  shape == NULL gives
 * (1,1,1,1), i.e. Eq. 1 on the raw sums.  LLMV_EINVAL for a field <= 0 or a
 * constant >= 2^53. */
int llmv_shape_constants(const llmv_shape *shape, double S[4]);

/* Bytes of device workspace every call below needs for a trace of this
 * size, except llmv_attribute_sweep (llmv_sweep_workspace_size). */
size_t llmv_workspace_size(int64_t n_batches, int64_t n_requests, int32_t n_tenants);

/* Bytes of device workspace llmv_attribute_sweep needs for a trace of this
 * size: llmv_workspace_size's (with a histogram per setting of a pass)
 * plus the (batch, tenant) groups: 20 bytes per request, 40 bytes per batch
 * and a few KiB. */
size_t llmv_sweep_workspace_size(int64_t n_batches, int64_t n_requests, int32_t n_tenants);

/* llmv_sweep_workspace_size for llmv_attribute_sweep_ext: 4 more bytes per
 * request (the groups' sums of p*c) and 8 more per batch. */
size_t llmv_sweep_workspace_size_ext(int64_t n_batches, int64_t n_requests, int32_t n_tenants);

/* Batched attribution (Sec. 2 Problem formulation; Sec. 2.1, Eq. 1).
 *   trace     host struct, device arrays as above.
 *   shape     host, or NULL for the unit shape.
 *   coeffs    host, 20 finite fp32: theta[phase][segment][k] at index
 *             (phase*2 + segment)*5 + k, k = (beta, a1, a2, a3, a4).
 *   latency   device [n_batches] fp32 T_B, or NULL.
 *   regime    device [n_batches] uint8 2*phase+segment / LLMV_REGIME_EMPTY,
 *             or NULL.
 *   share     device [n_requests] fp32 f(i|B), or NULL.
 *   n_tenants number of tenant ids; needed when tenant_sums != NULL.
 *   tenant_sums device [n_tenants] fp64 L_u, or NULL.  Overwritten (not
 *             accumulated); needs trace->tenant.
 * Per batch, the model and the share constants are evaluated in fp64 from
 * exact integer sums; the constants are rounded to fp32 and each share is
 * evaluated in fp32 (a few ulp); tenant sums add the fp32 shares in fp64.
 * Every output is independent of the others being requested.  A trace of
 * one scheduling step (at most 4096 requests and 1024 batches, and at most
 * 4096 tenants when tenant sums are requested) runs as one workgroup in one
 * launch and does not touch the workspace (ws may then be NULL). */
int llmv_attribute(const llmv_trace *trace, const llmv_shape *shape,
                   const float coeffs[20], float *latency, uint8_t *regime,
                   float *share, int32_t n_tenants, double *tenant_sums,
                   void *ws, size_t ws_bytes, void *stream);

/* Attribution of one scheduling step on the host, for a scheduler that
 * attributes each step as it is formed and cannot afford a device round trip
 * (Sec. 1: admission control and accounting inside the serving loop;
 * Sec. 2.1, last paragraph: the model runs once per step).  The outputs of
 * llmv_attribute, computed by the CPU from HOST arrays: every pointer in
 * trace, and latency, regime, share and tenant_sums, are host pointers (each
 * output optional, as in llmv_attribute).  Batch sums are exact integers,
 * the model and the share constants fp64 and the shares fp32 with the same
 * operations as the GPU kernels, so latency, regime and shares equal the
 * GPU's bit for bit; tenant sums add the shares in fp64 in request order.
 * Unlike the device entry points it checks the data first (LLMV_ERANGE for
 * data outside the limits, nothing written).  Synchronous, single-threaded,
 * no device use.  For traces of one step (a few thousand requests); large
 * traces belong on the GPU. */
int llmv_attribute_host(const llmv_trace *trace, const llmv_shape *shape,
                        const float coeffs[20], float *latency, uint8_t *regime,
                        float *share, int32_t n_tenants, double *tenant_sums);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc):
 * llmv_attribute with no workspace argument.  The scratch it needs (chunk
 * table, claim counter, per-workgroup tenant partials) is a static device
 * array of LLMV_NOALLOC_SCRATCH_BYTES in the library, one per GPU, held
 * until the process ends; its address is looked up once per device on the
 * first call there.  The call allocates nothing (no hipMalloc, no library
 * allocation); the caller still passes every input and output.  Outputs,
 * precision, ordering and errors are those of llmv_attribute; a trace whose
 * scratch (llmv_workspace_size of its sizes) exceeds the static array is
 * refused with LLMV_EINVAL before anything is enqueued.  Every call on one
 * GPU shares that GPU's array: calls that overlap in time on one GPU (other
 * streams, other host threads) race and must be serialised by the caller.
 * Each call rewrites what it reads of the array (the claim counter is
 * cleared by its first kernel), so no state carries over between calls. */
#define LLMV_NOALLOC_SCRATCH_BYTES ((size_t)16 << 20)
int llmv_attribute_noalloc(const llmv_trace *trace, const llmv_shape *shape,
                           const float coeffs[20], float *latency, uint8_t *regime,
                           float *share, int32_t n_tenants, double *tenant_sums,
                           void *stream);

/* Extended model (feature variants the paper leaves open; Sec. 2.1 defines
 * Eq. 1 only).  Two more features per batch, each with its own coefficient
 * in every (phase, segment) set:
 *   a5 * S5 * sum_i p_i*c_i   the processed tokens attending to the cached
 *                             context (a prefill chunk with a prefix);
 *   a6 * S6 * |B|             a per-request term: one position's logits
 *                             (with the unit shape, the other reading of
 *                             Eq. 1's a4 term, a4*|B| per batch).
 * Per request the features are
 *   x_i = (S0/|B|, S1*p_i, S2*c_i, S3*p_i^2, |B|, S5*p_i*c_i, S6),
 * so shares stay additive.  Phase, segment and empty-batch rules are those
 * of llmv_attribute. */

/* Host only.  S[0..3] as llmv_shape_constants; S[4] = S5 =
 * 4*L*Hq*head_dim (FLOPs per processed token and cached key: score and
 * value mix, every layer and query head), S[5] = S6 = 2*vocab*hidden
 * (output-projection FLOPs per request).  shape == NULL gives all ones. */
int llmv_shape_constants_ext(const llmv_shape *shape, double S[6]);

/* llmv_attribute under the extended model.
 *   coeffs  host, 28 finite fp32: theta[phase][segment][k] at index
 *           (phase*2 + segment)*7 + k, k = (beta, a1, a2, a3, a4, a5, a6).
 * Other arguments, outputs, precision and workspace as llmv_attribute.  The
 * batch sum of p_i*c_i is exact in uint64 and must stay below 2^63 (not
 * checked).  With a5 = a6 = 0 in every set, latency, regime and shares are
 * bit-identical to llmv_attribute's with the first five coefficients of each
 * set, and tenant sums equal up to the order of their fp64 additions. */
int llmv_attribute_ext(const llmv_trace *trace, const llmv_shape *shape,
                       const float coeffs[28], float *latency, uint8_t *regime,
                       float *share, int32_t n_tenants, double *tenant_sums,
                       void *ws, size_t ws_bytes, void *stream);

/* What-if sweep (Sec. 1: fast "what-if" planning over alternative model
 * and coefficient settings; Eq. 1 and Sec. 2 Problem formulation for each):
 * the tenant sums of one trace under every pair (shape s, coefficient vector
 * v).
 *   shapes   host [n_shapes] llmv_shape, or NULL with n_shapes == 1 for the
 *            unit shape.
 *   coeffs   host [n_coeffs][20] finite fp32, laid out as in llmv_attribute.
 *   n_tenants, trace->tenant as for llmv_attribute's tenant sums.
 *   out      device [n_shapes][n_coeffs][n_tenants] fp64, overwritten:
 *            out[(s*n_coeffs + v)*n_tenants + u] = L_u under (s, v).
 * Equivalent to n_shapes*n_coeffs calls of llmv_attribute with only
 * tenant_sums requested, up to rounding: the shares of one tenant's requests
 * in one batch are summed in closed form, k0*n + k1*sum p + k2*sum c +
 * k3*sum p^2 with the batch's fp32 constants and the group's sums rounded to
 * fp32, and added in fp64.  The (batch, tenant) groups are formed once per
 * call; each pass over them evaluates 8 consecutive settings (4 above 1024
 * tenants, 2 above 2048).  n_tenants must be <= 4096 here.  The workspace is
 * llmv_sweep_workspace_size's. */
int llmv_attribute_sweep(const llmv_trace *trace, const llmv_shape *shapes,
                         int32_t n_shapes, const float *coeffs, int32_t n_coeffs,
                         int32_t n_tenants, double *out, void *ws, size_t ws_bytes,
                         void *stream);

/* llmv_attribute_sweep under the extended model (readings X1-X3; Sec. 1
 * what-if planning):
 *   shapes   as llmv_attribute_sweep; each one's S5 and S6 as in
 *            llmv_shape_constants_ext.
 *   coeffs   host [n_coeffs][28] finite fp32, laid out as in
 *            llmv_attribute_ext.
 * Equivalent, up to rounding, to n_shapes*n_coeffs calls of
 * llmv_attribute_ext with only tenant_sums requested: a group's shares sum
 * to k0*n + k1*sum p + k2*sum c + k3*sum p^2 + k5*sum p*c, with k0 holding
 * the a6 term and k5 = fp32(a5*S5), the group's sums rounded to fp32.
 * Regimes come from the exact batch sums, as in llmv_attribute_ext.  Other
 * arguments, limits (sum p*c per batch below 2^63, not checked) and errors
 * as llmv_attribute_sweep; the workspace is llmv_sweep_workspace_size_ext's. */
int llmv_attribute_sweep_ext(const llmv_trace *trace, const llmv_shape *shapes,
                             int32_t n_shapes, const float *coeffs, int32_t n_coeffs,
                             int32_t n_tenants, double *out, void *ws, size_t ws_bytes,
                             void *stream);

/* Exact per-batch sums of Eq. 1 and the batch phase (Sec. 2.1), the state
 * an admission query starts from:
 *   sums    device [4][n_batches] int64, row k at sums[k*n_batches + b]:
 *           (|B|, sum p, sum c, sum p^2); zeros for an empty batch.
 *   phase   device [n_batches] uint8 LLMV_PREFILL / LLMV_DECODE (prefill iff
 *           some request has p > 1 or c = 0), LLMV_REGIME_EMPTY for an empty
 *           batch.
 * Either output may be NULL.  Workspace as for llmv_attribute. */
int llmv_batch_sums(const llmv_trace *trace, int64_t *sums, uint8_t *phase, void *ws,
                    size_t ws_bytes, void *stream);

/* llmv_batch_sums plus the extended model's cross sum (readings X1-X3), the
 * state llmv_fit_ext and llmv_fit_metrics_ext start from:
 *   sums    device [5][n_batches] int64: (|B|, sum p, sum c, sum p^2,
 *           sum p*c); zeros for an empty batch.  sum p*c must stay below
 *           2^63 (not checked).
 *   phase   as llmv_batch_sums.
 * Either output may be NULL.  Workspace as for llmv_attribute. */
int llmv_batch_sums_ext(const llmv_trace *trace, int64_t *sums, uint8_t *phase, void *ws,
                        size_t ws_bytes, void *stream);

/* Admission query (Sec. 1: admission control that rejects or defers a
 * request whose share would exceed its budget; Sec. 2 Problem formulation;
 * Eq. 1).  Candidate j, a request (cand_p[j], cand_c[j]), is proposed for
 * batch cand_batch[j]; B' is that batch with the candidate added.
 *   sums, phase  device, as written by llmv_batch_sums for n_batches batches.
 *   shape, coeffs  as for llmv_attribute.
 *   cand_batch, cand_p, cand_c  device [n_cand]; 1 <= cand_p <= 2^20,
 *                  cand_c >= 0 (not checked).
 *   t_after  device [n_cand] fp32 f(B'), or NULL.
 *   delta    device [n_cand] fp32 f(B') - f(B) (f of an empty batch is 0),
 *            or NULL.
 *   share    device [n_cand] fp32 f(candidate | B'), or NULL.
 *   regime   device [n_cand] uint8 2*phase + segment of B', or NULL.
 * B' is a prefill batch if B is one or the candidate has p > 1 or c = 0.
 * Everything is evaluated in fp64 and rounded once.  A candidate whose
 * batch index is outside [0, n_batches) gets NaN outputs and regime
 * LLMV_REGIME_EMPTY.  No workspace.  One thread per candidate. */
int llmv_admit(const int64_t *sums, const uint8_t *phase, int64_t n_batches,
               const llmv_shape *shape, const float coeffs[20], const int64_t *cand_batch,
               const int32_t *cand_p, const int32_t *cand_c, int64_t n_cand, float *t_after,
               float *delta, float *share, uint8_t *regime, void *stream);

/* llmv_admit under the extended model (readings X1-X3):
 *   sums    device [5][n_batches] as written by llmv_batch_sums_ext.
 *   coeffs  host, 28 finite fp32 as for llmv_attribute_ext.
 * B' also adds the candidate's p*c to sum p*c; the candidate's share gains
 * its a5*S5*p*c and a6*S6 terms.  Other arguments, outputs and rules as
 * llmv_admit. */
int llmv_admit_ext(const int64_t *sums, const uint8_t *phase, int64_t n_batches,
                   const llmv_shape *shape, const float coeffs[28], const int64_t *cand_batch,
                   const int32_t *cand_p, const int32_t *cand_c, int64_t n_cand, float *t_after,
                   float *delta, float *share, uint8_t *regime, void *stream);

/* Fitting Eq. 1 (Sec. 2.1: the coefficients are fitted by ordinary least
 * squares on profiled batch latencies, one set per phase and segment) and
 * the accuracy metrics (Sec. 3 and Appendix A: r^2 and the 90th / 99th
 * percentile of the relative error).  Both start from the batch state that
 * llmv_batch_sums writes, plus a measured latency per batch:
 *   sums, phase  device, as written by llmv_batch_sums for n_batches
 *                batches (n_batches <= 2^31).
 *   y            device [n_batches] fp64 measured latency (ignored for
 *                empty batches).
 * Readings of points the paper leaves open:
 *   - segment membership: fitting runs in rounds; a round assigns every
 *     nonempty batch to the segment whose prediction under the current
 *     coefficients is larger (ties to MEM), then refits each set;
 *   - identifiability: when every batch of a set has sum p^2 == sum p (all
 *     decode requests process one token), a3 keeps its current value; when
 *     every batch has sum c == 0, a2 does; the other coefficients are fitted
 *     to y minus the kept terms.  A set with fewer batches than free
 *     coefficients, or with (numerically) dependent free columns, keeps all
 *     of its coefficients;
 *   - r^2 = 1 - SSE / sum (y - mean y)^2 over a group's nonempty batches;
 *   - relative error |f(B) - y| / y over nonempty batches with y > 0,
 *     rounded to fp32; the p-th percentile of m errors is the
 *     ceil(p*m)-th smallest (nearest rank, exact integer ranks).
 * `ws` is a device workspace of llmv_fit_workspace_size(n_batches) bytes
 * (256-byte aligned, clobbered).  Results are written to device memory on
 * `stream`; nothing waits. */
size_t llmv_fit_workspace_size(int64_t n_batches);

/* Ordinary least squares for the four coefficient sets:
 *   shape    host, or NULL for the unit shape (as for llmv_attribute).
 *   theta0   host [20] finite fp64, the starting coefficients (layout of
 *            llmv_attribute's coeffs); they decide the first round's segment
 *            membership and the values of coefficients a set cannot fit.
 *   rounds   0..1024 rounds of (assign, refit); 0 copies theta0.
 *   theta    device [20] fp64 out: the fitted coefficients.
 *   counts   device [4] int64 out: batches of each (phase, segment) set in
 *            the last round (zeros for rounds == 0), or NULL.
 * Each round forms every set's normal equations (X^T X, X^T y over the
 * batch features of Eq. 1: S0, S1*sum p, S2*sum c, S3*sum p^2, |B|^2) in
 * fp64 and solves them by a Cholesky factorisation after scaling each
 * column to unit diagonal; the batch sums are added in a fixed order, so the
 * result does not depend on scheduling.  Coefficients are not constrained
 * to be nonnegative. */
int llmv_fit(const int64_t *sums, const uint8_t *phase, int64_t n_batches,
             const llmv_shape *shape, const double *y, const double theta0[20],
             int32_t rounds, double *theta, int64_t *counts, void *ws, size_t ws_bytes,
             void *stream);

/* Accuracy of fp32 coefficients (the model every other entry point
 * evaluates) against measured latencies:
 *   coeffs   host [20] finite fp32.
 *   rel_err  device [n_batches] fp32 out: the relative error of each batch,
 *            NaN for an empty batch or y <= 0; or NULL.
 *   out      device [12] fp64 out: for g = prefill, decode, all,
 *            out[4g .. 4g+3] = (r^2, p90, p99, nonempty batches); r^2 is NaN
 *            without batches or with all y equal, a percentile NaN without
 *            errors.
 * Predictions are Eq. 1 in fp64 with the segment max; percentiles are exact
 * (a radix select over the fp32 errors), r^2 takes two passes (mean, then
 * the sums of squares) with fixed-order sums. */
int llmv_fit_metrics(const int64_t *sums, const uint8_t *phase, int64_t n_batches,
                     const llmv_shape *shape, const float coeffs[20], const double *y,
                     float *rel_err, double *out, void *ws, size_t ws_bytes, void *stream);

/* llmv_fit and llmv_fit_metrics for the extended model (Eq. 1 plus a5*S5*
 * sum p*c and a6*S6*|B|; the feature variants the paper leaves open), with
 * the same rounds, identifiability rules, metrics and precision:
 *   sums          device [5][n_batches] int64 as written by
 *                 llmv_batch_sums_ext (the fifth row is sum p*c).
 *   theta0, theta fp64 [28], coeffs fp32 [28]: index (phase*2 + segment)*7
 *                 + k, k = (beta, a1, a2, a3, a4, a5, a6).
 * Two more coefficients can keep their starting values: a5 when sum p*c ==
 * sum c in every batch of a set (every request with a context processes one
 * token: the cross term is the c term), a6 when sum p == |B| (every request
 * processes one token: the per-request term is the p term).  Shape constants
 * as llmv_shape_constants_ext.  Workspace: llmv_fit_workspace_size. */
int llmv_fit_ext(const int64_t *sums, const uint8_t *phase, int64_t n_batches,
                 const llmv_shape *shape, const double *y, const double theta0[28],
                 int32_t rounds, double *theta, int64_t *counts, void *ws, size_t ws_bytes,
                 void *stream);
int llmv_fit_metrics_ext(const int64_t *sums, const uint8_t *phase, int64_t n_batches,
                         const llmv_shape *shape, const float coeffs[28], const double *y,
                         float *rel_err, double *out, void *ws, size_t ws_bytes, void *stream);

/* Request and batch features (Sec. 2.1), structure of arrays:
 *   x_req   device [5][n_requests] fp32, element k of request i at
 *           x_req[k*n_requests + i]: (S0/|B|, S1*p_i, S2*c_i, S3*p_i^2, |B|),
 *           or NULL.
 *   x_batch device [5][n_batches] fp64: the batch sums
 *           (S0, S1*sum p, S2*sum c, S3*sum p^2, |B|^2), zeros for an empty
 *           batch, or NULL.
 * Dotting x with a coefficient set gives Eq. 1's value (batch) or share
 * (request).  trace->tenant is ignored. */
int llmv_features(const llmv_trace *trace, const llmv_shape *shape, float *x_req,
                  double *x_batch, void *ws, size_t ws_bytes, void *stream);

/* Tenant sums of given shares (Sec. 2, Problem formulation: L_u):
 *   tenant  device [n] int32 in [0, n_tenants);  share device [n] fp32;
 *   tenant_sums device [n_tenants] fp64, overwritten. */
int llmv_tenant_sums(const int32_t *tenant, const float *share, int64_t n,
                     int32_t n_tenants, double *tenant_sums, void *ws,
                     size_t ws_bytes, void *stream);

/* Checks the device data of a trace against the limits above: offsets
 * (start at 0, non-decreasing, end at n_requests, batch sizes <= 2^22),
 * 1 <= p <= 2^20, c >= 0, and 0 <= tenant < n_tenants when trace->tenant is
 * not NULL.  Waits for the stream.  LLMV_OK when all hold, LLMV_ERANGE when
 * any does not, or an argument / device error code. */
int llmv_validate(const llmv_trace *trace, int32_t n_tenants, void *ws,
                  size_t ws_bytes, void *stream);

/* Message for the calling thread's last non-zero return (static storage,
 * valid until that thread's next call). */
const char *llmv_last_error(void);

/* Measurement hook, not part of the method.  For callers that time the main
 * kernel on its own: while set (per calling thread), llmv_attribute and
 * llmv_features record `before` (a hipEvent_t) on their stream right before
 * the tile kernel is enqueued and `after` right after it.  Pass NULL, NULL
 * to stop.  The events are the caller's; the library does not own them. */
int llmv_set_kernel_events(void *before, void *after);

#ifdef __cplusplus
}
#endif

#endif /* LLMV_H */
