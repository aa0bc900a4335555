/*
 * orc.h -- plain fp64 CPU oracle for LLMVisor batched latency attribution.
 *
 * TEST INFRASTRUCTURE ONLY.  This code exists to check the HIP path; it is
 * not part of the product.  Only the test suite, the smoke check and the
 * benchmark's CPU-baseline leg may load it.  It shares no code, header,
 * table or constant with the HIP library and includes nothing from it.
 *
 * What it computes (LLMVisor, "Piecewise roofline-guided linear latency
 * model", Sec. 2.1, Eq. 1; problem statement in Sec. 2 "Problem formulation"):
 *
 *   per batch B:   T_B = beta + a1*sum p + a2*sum c + a3*sum p^2 + a4*sum_i |B|
 *   per request:   f(i|B) = the request's own terms of that sum
 *   per tenant:    L_u = sum of f(i|B) over the tenant's requests
 *
 * with two coefficient sets per phase (memory-bound and compute-bound
 * segment) and features scaled by model-shape constants S0..S3.  Every
 * reading taken where the paper is silent is stated at the function that
 * applies it.  Arithmetic: IEEE fp64, round to nearest even, no FMA
 * contraction (built with -ffp-contract=off), single thread, request order.
 */
#ifndef ORC_H
#define ORC_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Error codes. */
#define ORC_OK 0
#define ORC_EINVAL (-1) /* bad argument (null pointer, negative size, bad shape) */
#define ORC_ERANGE (-2) /* trace data outside the stated limits               */

/* Phase, segment and regime numbering. regime = 2*phase + segment. */
#define ORC_PREFILL 0
#define ORC_DECODE 1
#define ORC_MEM 0
#define ORC_COMP 1
#define ORC_REGIME_EMPTY 255

/* Input limits (see orc_validate). */
#define ORC_P_MAX (1 << 20)        /* tokens processed by one request in one step */
#define ORC_BATCH_MAX (1 << 22)    /* requests in one batch                       */
#define ORC_TENANTS_MAX (1 << 24)  /* tenant id space                             */

/* Model shape; every field must be > 0.  weight_bytes / kv_bytes are bytes
 * per element (2 for bf16). */
typedef struct {
  int32_t n_layers, hidden, n_q_heads, n_kv_heads, head_dim, ffn, vocab,
      weight_bytes, kv_bytes;
} orc_shape;

/* Shape constants S[0..3] = (S0, S1, S2, S3), the proportionality factors of
 * the request features (Sec. 2.1: features proportional to FLOPs and memory
 * I/O rather than hand-computed FLOPs divided by peak rates):
 *   P_layer = hidden*head_dim*(2*Hq + 2*Hkv) + 3*hidden*ffn
 *   S0 = weight_bytes * (L*P_layer + vocab*hidden)   weight bytes per step
 *   S1 = 2*L*P_layer                                linear FLOPs per token
 *   S2 = 2*L*Hkv*head_dim*kv_bytes                  KV bytes per context token
 *   S3 = 2*L*Hq*head_dim                            causal attention FLOPs per p^2
 * shape == NULL gives the unit shape S = (1,1,1,1): Eq. 1 verbatim.
 * Returns ORC_EINVAL for a non-positive field or a constant >= 2^53. */
int orc_shape_constants(const orc_shape *shape, double S[4]);

/* First violation of the input limits, or ORC_OK.
 *   offsets[0] == 0, non-decreasing, offsets[nB] == N, batch size <= 2^22,
 *   1 <= p[i] <= 2^20, c[i] >= 0, 0 <= tenant[i] < n_tenants (tenant may be
 *   NULL, then n_tenants is not checked).  Returns ORC_EINVAL for null
 *   pointers or negative sizes, ORC_ERANGE for data outside the limits. */
int orc_validate(int64_t n_batches, int64_t n_requests, const int64_t *offsets,
                 const int32_t *p, const int32_t *c, const int32_t *tenant,
                 int32_t n_tenants);

/* Per-request and per-batch features.
 *   x_req  [5][N] : (S0/|B|, S1*p_i, S2*c_i, S3*p_i^2, |B|)   (may be NULL)
 *   x_batch[5][nB]: sums of x_req over the batch
 *                   = (S0, S1*P, S2*C, S3*Q, |B|^2), zeros for an empty batch
 *                                                           (may be NULL)
 * Layout is structure-of-arrays: element k of request i is x_req[k*N + i]. */
int orc_features(int64_t n_batches, int64_t n_requests, const int64_t *offsets,
                 const int32_t *p, const int32_t *c, const orc_shape *shape,
                 double *x_req, double *x_batch);

/* Attribution.  coeffs[20] holds theta[phase][segment][k] at index
 * (phase*2 + segment)*5 + k, k = (beta, a1, a2, a3, a4).  All outputs are
 * optional (NULL skips them):
 *   T[nB]       batch latency of the chosen segment
 *   TM[nB],TC[nB]  both segment values (0 for an empty batch)
 *   phase[nB]   ORC_PREFILL / ORC_DECODE (255 for an empty batch)
 *   regime[nB]  2*phase + segment, ORC_REGIME_EMPTY for an empty batch
 *   share[N]    per-request share under the chosen segment
 *   share_alt[N] per-request share under the other segment (used by parity
 *               checks inside the tie zone)
 *   tenant_sums[n_tenants]  sum of share over each tenant's requests,
 *               in request order; needs tenant != NULL.                    */
int orc_attribute(int64_t n_batches, int64_t n_requests, const int64_t *offsets,
                  const int32_t *p, const int32_t *c, const int32_t *tenant,
                  const orc_shape *shape, const float coeffs[20],
                  int32_t n_tenants, double *T, double *TM, double *TC,
                  uint8_t *phase, uint8_t *regime, double *share,
                  double *share_alt, double *tenant_sums);

/* Extended model (feature variants the paper leaves open; Sec. 2.1 defines
 * Eq. 1 only).  Two more features per batch, each with its own coefficient:
 *   a5 * S5 * sum_i p_i*c_i  attention of the processed tokens over the
 *                            cached context (chunked prefill with a prefix);
 *   a6 * S6 * |B|            per-request output projection (logits of one
 *                            position per request); with the unit shape this
 *                            is the other reading of Eq. 1's a4 term, a4*|B|
 *                            per batch.
 * S[0..5] = (S0, S1, S2, S3, S5, S6):
 *   S5 = 4*L*Hq*head_dim   FLOPs per (processed token, cached key) pair
 *   S6 = 2*vocab*hidden    output-projection FLOPs per request
 * shape == NULL gives all ones. */
int orc_shape_constants_ext(const orc_shape *shape, double S[6]);

/* Attribution under the extended model.  coeffs[28] holds
 * theta[phase][segment][k] at index (phase*2 + segment)*7 + k,
 * k = (beta, a1, a2, a3, a4, a5, a6).  Per request the features are
 *   x_i = (S0/|B|, S1*p_i, S2*c_i, S3*p_i^2, |B|, S5*p_i*c_i, S6),
 * per batch their sums; terms are added in order k = 0..6.  Phase, segment
 * and empty-batch rules, outputs and ownership as orc_attribute.  ORC_ERANGE
 * also when a batch's sum of p_i*c_i reaches 2^63. */
int orc_attribute_ext(int64_t n_batches, int64_t n_requests, const int64_t *offsets,
                      const int32_t *p, const int32_t *c, const int32_t *tenant,
                      const orc_shape *shape, const float coeffs[28], int32_t n_tenants,
                      double *T, double *TM, double *TC, uint8_t *phase, uint8_t *regime,
                      double *share, double *share_alt, double *tenant_sums);

/* Exact per-batch sums of Eq. 1 and the batch phase (Sec. 2.1):
 *   sums[4][nB] = (|B|, sum p, sum c, sum p^2), zeros for an empty batch;
 *   phase[nB]   ORC_PREFILL / ORC_DECODE, 255 for an empty batch.
 * Both outputs are optional. */
int orc_batch_sums(int64_t n_batches, int64_t n_requests, const int64_t *offsets,
                   const int32_t *p, const int32_t *c, int64_t *sums, uint8_t *phase);

/* orc_batch_sums plus the extended model's cross sum (readings X1-X3):
 *   sums[5][nB] = (|B|, sum p, sum c, sum p^2, sum p*c); ORC_ERANGE when a
 *   batch's sum p*c reaches 2^63. */
int orc_batch_sums_ext(int64_t n_batches, int64_t n_requests, const int64_t *offsets,
                       const int32_t *p, const int32_t *c, int64_t *sums, uint8_t *phase);

/* Admission query (Sec. 1: admission control that rejects or defers a
 * request whose share would exceed its budget; Sec. 2 Problem formulation).
 * B is the batch of the n requests (p, c) (n may be 0); B' is B with one more
 * request, the candidate (cp, cc).  Evaluated as that definition: the
 * attribution of B' and of B (orc_attribute on each, one batch).
 *   T_after    f(B')
 *   delta      f(B') - f(B), f of an empty batch being 0
 *   share      f(candidate | B'), the candidate's share in B'
 *   share_alt  the candidate's share under B''s other segment
 *   TM_after, TC_after  both segment values of B'
 *   regime     2*phase + segment of B'
 * Every output is optional. */
int orc_admit(int64_t n, const int32_t *p, const int32_t *c, int32_t cp, int32_t cc,
              const orc_shape *shape, const float coeffs[20], double *T_after,
              double *delta, double *share, double *share_alt, double *TM_after,
              double *TC_after, uint8_t *regime);

/* orc_admit under the extended model (readings X1-X3): coeffs [28], index
 * (phase*2 + segment)*7 + k; B and B' attributed by orc_attribute_ext. */
int orc_admit_ext(int64_t n, const int32_t *p, const int32_t *c, int32_t cp, int32_t cc,
                  const orc_shape *shape, const float coeffs[28], double *T_after,
                  double *delta, double *share, double *share_alt, double *TM_after,
                  double *TC_after, uint8_t *regime);

/* Tenant sums of given shares, in request order:
 * out[u] = sum_{i : tenant[i] == u} share[i].  ORC_ERANGE for a tenant id
 * outside [0, n_tenants). */
int orc_tenant_sums(const int32_t *tenant, const double *share,
                    int64_t n_requests, int32_t n_tenants, double *out);

#ifdef __cplusplus
}
#endif

#endif /* ORC_H */
