/*
 * orc.c -- plain fp64 CPU oracle for LLMVisor batched latency attribution.
 *
 * TEST INFRASTRUCTURE ONLY (see orc.h).  Single-threaded, request order,
 * IEEE fp64, built with -ffp-contract=off.  Written from the paper's
 * definitions (Sec. 2 "Problem formulation", Sec. 2.1 and Eq. 1); every
 * reading of a point the paper leaves open is stated where it is applied.
 *
 * Pins: every function here is pinned by the CPU test suite against
 * hand-worked batches, closed-form invariants of Eq. 1 and published model
 * parameter counts; none of those pins calls back into this file to make
 * its expected value.
 */
#include "orc.h"

#include <stdint.h>
#include <stdlib.h>

#include <stddef.h>

/* Largest integer below which every integer is exact in fp64. */
#define ORC_EXACT_LIMIT 9007199254740992LL /* 2^53 */

int orc_shape_constants(const orc_shape *sh, double S[4]) {
  if (!S) return ORC_EINVAL;
  if (!sh) {
    /* Unit shape: the features are the raw sums of Eq. 1. */
    S[0] = S[1] = S[2] = S[3] = 1.0;
    return ORC_OK;
  }
  if (sh->n_layers <= 0 || sh->hidden <= 0 || sh->n_q_heads <= 0 ||
      sh->n_kv_heads <= 0 || sh->head_dim <= 0 || sh->ffn <= 0 ||
      sh->vocab <= 0 || sh->weight_bytes <= 0 || sh->kv_bytes <= 0)
    return ORC_EINVAL;
  /* Integer arithmetic in int64 (long double would hide overflow). */
  const int64_t L = sh->n_layers, h = sh->hidden, hq = sh->n_q_heads,
                hkv = sh->n_kv_heads, d = sh->head_dim, f = sh->ffn,
                V = sh->vocab, wb = sh->weight_bytes, kb = sh->kv_bytes;
  /* Weights of one decoder layer: the q and o projections (h x Hq*d each),
   * the k and v projections (h x Hkv*d each) and the three gated-MLP
   * matrices (h x ffn each).  Norm vectors and biases are left out. */
  const int64_t p_layer = h * d * (2 * hq + 2 * hkv) + 3 * h * f;
  /* S0: bytes of weights streamed once per step: all layers plus the
   * output projection (vocab x hidden); the input embedding is a gather,
   * not a stream, and is left out. */
  const int64_t s0 = wb * (L * p_layer + V * h);
  /* S1: multiply-add FLOPs of the linear layers per processed token. */
  const int64_t s1 = 2 * L * p_layer;
  /* S2: KV-cache bytes read per context token (K and V, every layer). */
  const int64_t s2 = 2 * L * hkv * d * kb;
  /* S3: causal self-attention FLOPs per unit of p^2: a causal block of p
   * tokens has p(p+1)/2 query-key pairs, each costing 4*Hq*d FLOPs per layer
   * (2 for the score, 2 for the value mix); the p^2 part of that count is
   * 2*L*Hq*d*p^2.  The linear-in-p remainder is left to the a1 term. */
  const int64_t s3 = 2 * L * hq * d;
  if (s0 >= ORC_EXACT_LIMIT || s1 >= ORC_EXACT_LIMIT || s2 >= ORC_EXACT_LIMIT ||
      s3 >= ORC_EXACT_LIMIT)
    return ORC_EINVAL;
  S[0] = (double)s0;
  S[1] = (double)s1;
  S[2] = (double)s2;
  S[3] = (double)s3;
  return ORC_OK;
}

int orc_validate(int64_t nB, int64_t N, const int64_t *off, const int32_t *p,
                 const int32_t *c, const int32_t *tenant, int32_t n_tenants) {
  if (nB < 0 || N < 0 || !off) return ORC_EINVAL;
  if (N > 0 && (!p || !c)) return ORC_EINVAL;
  if (tenant && (n_tenants <= 0 || n_tenants > ORC_TENANTS_MAX)) return ORC_EINVAL;
  if (off[0] != 0) return ORC_ERANGE;
  for (int64_t b = 0; b < nB; ++b) {
    const int64_t n = off[b + 1] - off[b];
    if (n < 0 || n > ORC_BATCH_MAX) return ORC_ERANGE;
  }
  if (off[nB] != N) return ORC_ERANGE;
  for (int64_t i = 0; i < N; ++i) {
    if (p[i] < 1 || p[i] > ORC_P_MAX) return ORC_ERANGE;
    if (c[i] < 0) return ORC_ERANGE;
    if (tenant && (tenant[i] < 0 || tenant[i] >= n_tenants)) return ORC_ERANGE;
  }
  return ORC_OK;
}

/* Request-level feature vector x_i of Sec. 2.1, scaled by the shape:
 * x_i = (S0/|B|, S1*p_i, S2*c_i, S3*p_i^2, |B|).  Summing x_i over the batch
 * gives (S0, S1*sum p, S2*sum c, S3*sum p^2, |B|^2): the five terms of Eq. 1
 * with unit coefficients.
 * Reading of the beta term: beta is a per-batch constant, so the only split
 * that keeps the model a sum of per-request terms with no further data is
 * the equal one, S0/|B| per request.
 * Reading of the a4 term: Eq. 1 writes sum_i |B|, i.e. |B| per request and
 * |B|^2 per batch. */
static void request_features(const double S[4], int64_t n, int32_t p,
                             int32_t c, double x[5]) {
  const int64_t p2 = (int64_t)p * (int64_t)p; /* exact: p <= 2^20 */
  x[0] = S[0] / (double)n;
  x[1] = S[1] * (double)p;
  x[2] = S[2] * (double)c;
  x[3] = S[3] * (double)p2;
  x[4] = (double)n;
}

/* theta . x with the terms added in order k = 0..4. */
static double dot5(const double th[5], const double x[5]) {
  double acc = th[0] * x[0];
  acc = acc + th[1] * x[1];
  acc = acc + th[2] * x[2];
  acc = acc + th[3] * x[3];
  acc = acc + th[4] * x[4];
  return acc;
}

/* Per-batch sums of Eq. 1, exact in int64, plus the batch phase.
 * Phase reading: p_i is the number of tokens processed in this step (all of
 * the prompt in prefill, 1 in decode) and c_i is 0 in prefill (Sec. 2.1).
 * A request is therefore prefill-like when p_i > 1 or c_i == 0; a batch is a
 * prefill batch when any of its requests is prefill-like, a decode batch
 * otherwise (so a pure decode batch has every p_i == 1 and c_i >= 1). */
static void batch_sums(int64_t lo, int64_t hi, const int32_t *p,
                       const int32_t *c, int64_t *P, int64_t *C, int64_t *Q,
                       int *phase) {
  int64_t sp = 0, sc = 0, sq = 0;
  int prefill = 0;
  for (int64_t i = lo; i < hi; ++i) {
    sp += p[i];
    sc += c[i];
    sq += (int64_t)p[i] * (int64_t)p[i];
    if (p[i] > 1 || c[i] == 0) prefill = 1;
  }
  *P = sp;
  *C = sc;
  *Q = sq;
  *phase = prefill ? ORC_PREFILL : ORC_DECODE;
}

int orc_features(int64_t nB, int64_t N, const int64_t *off, const int32_t *p,
                 const int32_t *c, const orc_shape *shape, double *x_req,
                 double *x_batch) {
  double S[4];
  int rc = orc_shape_constants(shape, S);
  if (rc != ORC_OK) return rc;
  rc = orc_validate(nB, N, off, p, c, NULL, 0);
  if (rc != ORC_OK) return rc;
  for (int64_t b = 0; b < nB; ++b) {
    const int64_t lo = off[b], hi = off[b + 1], n = hi - lo;
    if (n == 0) {
      if (x_batch)
        for (int k = 0; k < 5; ++k) x_batch[k * nB + b] = 0.0;
      continue;
    }
    if (x_req) {
      for (int64_t i = lo; i < hi; ++i) {
        double x[5];
        request_features(S, n, p[i], c[i], x);
        for (int k = 0; k < 5; ++k) x_req[k * N + i] = x[k];
      }
    }
    if (x_batch) {
      int64_t P, C, Q;
      int ph;
      batch_sums(lo, hi, p, c, &P, &C, &Q, &ph);
      x_batch[0 * nB + b] = S[0];
      x_batch[1 * nB + b] = S[1] * (double)P;
      x_batch[2 * nB + b] = S[2] * (double)C;
      x_batch[3 * nB + b] = S[3] * (double)Q;
      x_batch[4 * nB + b] = (double)n * (double)n;
    }
  }
  return ORC_OK;
}

int orc_attribute(int64_t nB, int64_t N, const int64_t *off, const int32_t *p,
                  const int32_t *c, const int32_t *tenant,
                  const orc_shape *shape, const float coeffs[20],
                  int32_t n_tenants, double *T, double *TM, double *TC,
                  uint8_t *phase_out, uint8_t *regime, double *share,
                  double *share_alt, double *tenant_sums) {
  double S[4];
  if (!coeffs) return ORC_EINVAL;
  if (tenant_sums && !tenant) return ORC_EINVAL;
  int rc = orc_shape_constants(shape, S);
  if (rc != ORC_OK) return rc;
  rc = orc_validate(nB, N, off, p, c, tenant_sums ? tenant : NULL, n_tenants);
  if (rc != ORC_OK) return rc;

  /* theta[phase][segment][k] from the fp32 coefficient vector. */
  double th[2][2][5];
  for (int ph = 0; ph < 2; ++ph)
    for (int s = 0; s < 2; ++s)
      for (int k = 0; k < 5; ++k) th[ph][s][k] = (double)coeffs[(ph * 2 + s) * 5 + k];

  if (tenant_sums)
    for (int32_t u = 0; u < n_tenants; ++u) tenant_sums[u] = 0.0;

  for (int64_t b = 0; b < nB; ++b) {
    const int64_t lo = off[b], hi = off[b + 1], n = hi - lo;
    if (n == 0) {
      /* An empty batch runs no step: latency 0, no shares. */
      if (T) T[b] = 0.0;
      if (TM) TM[b] = 0.0;
      if (TC) TC[b] = 0.0;
      if (phase_out) phase_out[b] = ORC_REGIME_EMPTY;
      if (regime) regime[b] = ORC_REGIME_EMPTY;
      continue;
    }
    int64_t P, C, Q;
    int ph;
    batch_sums(lo, hi, p, c, &P, &C, &Q, &ph);
    /* Eq. 1 evaluated with each of the phase's two coefficient sets. */
    const double X[5] = {S[0], S[1] * (double)P, S[2] * (double)C,
                         S[3] * (double)Q, (double)n * (double)n};
    const double tm = dot5(th[ph][ORC_MEM], X);
    const double tc = dot5(th[ph][ORC_COMP], X);
    /* Segment choice.  The paper gives a two-segment linear form per phase
     * and calls the model roofline-guided, but names no breakpoint.  A
     * roofline is the larger of the memory-bound and the compute-bound time,
     * so the compute-bound segment is taken when it is strictly larger;
     * equality stays with the memory-bound segment. */
    const int seg = (tc > tm) ? ORC_COMP : ORC_MEM;
    if (T) T[b] = seg == ORC_COMP ? tc : tm;
    if (TM) TM[b] = tm;
    if (TC) TC[b] = tc;
    if (phase_out) phase_out[b] = (uint8_t)ph;
    if (regime) regime[b] = (uint8_t)(2 * ph + seg);
    if (share || share_alt || tenant_sums) {
      for (int64_t i = lo; i < hi; ++i) {
        double x[5];
        request_features(S, n, p[i], c[i], x);
        /* Closed-form additive share: the request's own terms of Eq. 1. */
        const double f = dot5(th[ph][seg], x);
        if (share) share[i] = f;
        if (share_alt) share_alt[i] = dot5(th[ph][1 - seg], x);
        /* L_u accumulates in request order (batches in order, requests in
         * order inside a batch). */
        if (tenant_sums) tenant_sums[tenant[i]] += f;
      }
    }
  }
  return ORC_OK;
}

int orc_shape_constants_ext(const orc_shape *sh, double S[6]) {
  if (!S) return ORC_EINVAL;
  double S4[4];
  const int rc = orc_shape_constants(sh, S4);
  if (rc != ORC_OK) return rc;
  for (int k = 0; k < 4; ++k) S[k] = S4[k];
  if (!sh) {
    S[4] = S[5] = 1.0;
    return ORC_OK;
  }
  const int64_t L = sh->n_layers, h = sh->hidden, hq = sh->n_q_heads, d = sh->head_dim,
                V = sh->vocab;
  /* S5: a processed token attending to one cached key costs, per layer and
   * query head, a head_dim-long dot product for the score and a head_dim-long
   * multiply-add into the output: 4*head_dim FLOPs. */
  const int64_t s5 = 4 * L * hq * d;
  /* S6: the logits of one position: a (vocab x hidden) matrix times a
   * vector, 2*vocab*hidden FLOPs per request. */
  const int64_t s6 = 2 * V * h;
  if (s5 >= ORC_EXACT_LIMIT || s6 >= ORC_EXACT_LIMIT) return ORC_EINVAL;
  S[4] = (double)s5;
  S[5] = (double)s6;
  return ORC_OK;
}

/* theta . x with the terms added in order k = 0..6. */
static double dot7(const double th[7], const double x[7]) {
  double acc = th[0] * x[0];
  for (int k = 1; k < 7; ++k) acc = acc + th[k] * x[k];
  return acc;
}

int orc_attribute_ext(int64_t nB, int64_t N, const int64_t *off, const int32_t *p,
                      const int32_t *c, const int32_t *tenant, const orc_shape *shape,
                      const float coeffs[28], int32_t n_tenants, double *T, double *TM,
                      double *TC, uint8_t *phase_out, uint8_t *regime, double *share,
                      double *share_alt, double *tenant_sums) {
  double S[6];
  if (!coeffs) return ORC_EINVAL;
  if (tenant_sums && !tenant) return ORC_EINVAL;
  int rc = orc_shape_constants_ext(shape, S);
  if (rc != ORC_OK) return rc;
  rc = orc_validate(nB, N, off, p, c, tenant_sums ? tenant : NULL, n_tenants);
  if (rc != ORC_OK) return rc;

  double th[2][2][7];
  for (int ph = 0; ph < 2; ++ph)
    for (int s = 0; s < 2; ++s)
      for (int k = 0; k < 7; ++k) th[ph][s][k] = (double)coeffs[(ph * 2 + s) * 7 + k];

  if (tenant_sums)
    for (int32_t u = 0; u < n_tenants; ++u) tenant_sums[u] = 0.0;

  for (int64_t b = 0; b < nB; ++b) {
    const int64_t lo = off[b], hi = off[b + 1], n = hi - lo;
    if (n == 0) {
      if (T) T[b] = 0.0;
      if (TM) TM[b] = 0.0;
      if (TC) TC[b] = 0.0;
      if (phase_out) phase_out[b] = ORC_REGIME_EMPTY;
      if (regime) regime[b] = ORC_REGIME_EMPTY;
      continue;
    }
    int64_t P, C, Q;
    int ph;
    batch_sums(lo, hi, p, c, &P, &C, &Q, &ph);
    /* sum of p_i*c_i, exact: each product is below 2^51; the sum is checked
     * against 2^63 as it grows */
    int64_t R = 0;
    for (int64_t i = lo; i < hi; ++i) {
      const int64_t pc = (int64_t)p[i] * (int64_t)c[i];
      if (R > INT64_MAX - pc) return ORC_ERANGE;
      R += pc;
    }
    const double X[7] = {S[0], S[1] * (double)P, S[2] * (double)C, S[3] * (double)Q,
                         (double)n * (double)n, S[4] * (double)R, S[5] * (double)n};
    const double tm = dot7(th[ph][ORC_MEM], X);
    const double tc = dot7(th[ph][ORC_COMP], X);
    /* The segment rule of orc_attribute: compute-bound when strictly larger. */
    const int seg = (tc > tm) ? ORC_COMP : ORC_MEM;
    if (T) T[b] = seg == ORC_COMP ? tc : tm;
    if (TM) TM[b] = tm;
    if (TC) TC[b] = tc;
    if (phase_out) phase_out[b] = (uint8_t)ph;
    if (regime) regime[b] = (uint8_t)(2 * ph + seg);
    if (share || share_alt || tenant_sums) {
      for (int64_t i = lo; i < hi; ++i) {
        const int64_t p2 = (int64_t)p[i] * (int64_t)p[i];
        const int64_t pc = (int64_t)p[i] * (int64_t)c[i];
        /* the request's own terms: summed over the batch they give X */
        const double x[7] = {S[0] / (double)n, S[1] * (double)p[i], S[2] * (double)c[i],
                             S[3] * (double)p2, (double)n, S[4] * (double)pc, S[5]};
        const double f = dot7(th[ph][seg], x);
        if (share) share[i] = f;
        if (share_alt) share_alt[i] = dot7(th[ph][1 - seg], x);
        if (tenant_sums) tenant_sums[tenant[i]] += f;
      }
    }
  }
  return ORC_OK;
}

int orc_batch_sums(int64_t nB, int64_t N, const int64_t *off, const int32_t *p,
                   const int32_t *c, int64_t *sums, uint8_t *phase) {
  int rc = orc_validate(nB, N, off, p, c, NULL, 0);
  if (rc != ORC_OK) return rc;
  for (int64_t b = 0; b < nB; ++b) {
    const int64_t n = off[b + 1] - off[b];
    int64_t P = 0, C = 0, Q = 0;
    int ph = ORC_REGIME_EMPTY;
    if (n > 0) batch_sums(off[b], off[b + 1], p, c, &P, &C, &Q, &ph);
    if (sums) {
      sums[0 * nB + b] = n;
      sums[1 * nB + b] = P;
      sums[2 * nB + b] = C;
      sums[3 * nB + b] = Q;
    }
    if (phase) phase[b] = (uint8_t)ph;
  }
  return ORC_OK;
}

int orc_batch_sums_ext(int64_t nB, int64_t N, const int64_t *off, const int32_t *p,
                       const int32_t *c, int64_t *sums, uint8_t *phase) {
  int rc = orc_batch_sums(nB, N, off, p, c, sums, phase);
  if (rc != ORC_OK || !sums) return rc;
  for (int64_t b = 0; b < nB; ++b) {
    /* sum of p_i*c_i, exact: each product is below 2^51; the sum is checked
     * against 2^63 as it grows */
    int64_t R = 0;
    for (int64_t i = off[b]; i < off[b + 1]; ++i) {
      const int64_t pc = (int64_t)p[i] * (int64_t)c[i];
      if (R > INT64_MAX - pc) return ORC_ERANGE;
      R += pc;
    }
    sums[4 * nB + b] = R;
  }
  return ORC_OK;
}

/* Admission query of either model (ext = 0: Eq. 1 with 20 coefficients,
 * ext = 1: the extended model with 28), by its definition: the attribution
 * of B' = B followed by the candidate, and of B. */
static int admit_query(int64_t n, const int32_t *p, const int32_t *c, int32_t cp, int32_t cc,
                       const orc_shape *shape, const float *coeffs, int ext, double *T_after,
                       double *delta, double *share, double *share_alt, double *TM_after,
                       double *TC_after, uint8_t *regime) {
  if (n < 0 || (n > 0 && (!p || !c)) || !coeffs) return ORC_EINVAL;
  int32_t *p1 = (int32_t *)malloc(sizeof(int32_t) * (size_t)(n + 1));
  int32_t *c1 = (int32_t *)malloc(sizeof(int32_t) * (size_t)(n + 1));
  double *f1 = (double *)malloc(sizeof(double) * (size_t)(n + 1));
  double *g1 = (double *)malloc(sizeof(double) * (size_t)(n + 1));
  if (!p1 || !c1 || !f1 || !g1) {
    free(p1); free(c1); free(f1); free(g1);
    return ORC_EINVAL;
  }
  for (int64_t i = 0; i < n; ++i) {
    p1[i] = p[i];
    c1[i] = c[i];
  }
  p1[n] = cp;
  c1[n] = cc;
  const int64_t off0[2] = {0, n}, off1[2] = {0, n + 1};
  double T0 = 0.0, T1 = 0.0, tm1 = 0.0, tc1 = 0.0;
  uint8_t reg1 = ORC_REGIME_EMPTY;
  int rc;
  if (ext) {
    rc = orc_attribute_ext(1, n, off0, p, c, NULL, shape, coeffs, 0, &T0, NULL, NULL, NULL,
                           NULL, NULL, NULL, NULL);
    if (rc == ORC_OK)
      rc = orc_attribute_ext(1, n + 1, off1, p1, c1, NULL, shape, coeffs, 0, &T1, &tm1, &tc1,
                             NULL, &reg1, f1, g1, NULL);
  } else {
    rc = orc_attribute(1, n, off0, p, c, NULL, shape, coeffs, 0, &T0, NULL, NULL, NULL, NULL,
                       NULL, NULL, NULL);
    if (rc == ORC_OK)
      rc = orc_attribute(1, n + 1, off1, p1, c1, NULL, shape, coeffs, 0, &T1, &tm1, &tc1, NULL,
                         &reg1, f1, g1, NULL);
  }
  if (rc == ORC_OK) {
    if (T_after) *T_after = T1;
    if (delta) *delta = T1 - T0;
    if (share) *share = f1[n];
    if (share_alt) *share_alt = g1[n];
    if (TM_after) *TM_after = tm1;
    if (TC_after) *TC_after = tc1;
    if (regime) *regime = reg1;
  }
  free(p1); free(c1); free(f1); free(g1);
  return rc;
}

int orc_admit(int64_t n, const int32_t *p, const int32_t *c, int32_t cp, int32_t cc,
              const orc_shape *shape, const float coeffs[20], double *T_after,
              double *delta, double *share, double *share_alt, double *TM_after,
              double *TC_after, uint8_t *regime) {
  return admit_query(n, p, c, cp, cc, shape, coeffs, 0, T_after, delta, share, share_alt,
                     TM_after, TC_after, regime);
}

int orc_admit_ext(int64_t n, const int32_t *p, const int32_t *c, int32_t cp, int32_t cc,
                  const orc_shape *shape, const float coeffs[28], double *T_after,
                  double *delta, double *share, double *share_alt, double *TM_after,
                  double *TC_after, uint8_t *regime) {
  return admit_query(n, p, c, cp, cc, shape, coeffs, 1, T_after, delta, share, share_alt,
                     TM_after, TC_after, regime);
}

int orc_tenant_sums(const int32_t *tenant, const double *share, int64_t N,
                    int32_t n_tenants, double *out) {
  if (N < 0 || n_tenants <= 0 || n_tenants > ORC_TENANTS_MAX || !out)
    return ORC_EINVAL;
  if (N > 0 && (!tenant || !share)) return ORC_EINVAL;
  for (int64_t i = 0; i < N; ++i)
    if (tenant[i] < 0 || tenant[i] >= n_tenants) return ORC_ERANGE;
  for (int32_t u = 0; u < n_tenants; ++u) out[u] = 0.0;
  for (int64_t i = 0; i < N; ++i) out[tenant[i]] += share[i];
  return ORC_OK;
}
