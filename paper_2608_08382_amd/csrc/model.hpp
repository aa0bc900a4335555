// model.hpp -- the per-batch model of LLMVisor Eq. 1 and the per-request
// share, shared by the GPU kernels and the host-side single-step
// attributor, so that both round alike.
//
// Per batch (Sec. 2.1): the phase's two coefficient sets (memory-bound and
// compute-bound) evaluated on the exact sums, X = (S0, S1*P, S2*C, S3*Q,
// n^2); the larger one is the latency (roofline max, ties memory-bound);
// each request's share is its own terms under the chosen set,
// k0 + k1*p + k2*c + k3*p^2 with k0 = beta*S0/n + a4*n (beta split equally,
// the a4 term |B| per request), k1 = a1*S1, k2 = a2*S2, k3 = a3*S3.
#pragma once

#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

namespace llmv {

// Eq. 1 with one coefficient set, terms added in order k = 0..4, every
// product rounded before its add (no contraction into fused multiply-adds:
// the host and the GPU give the same bits).
__host__ __device__ inline double eq1(const double* th, const double X[5]) {
#pragma clang fp contract(off)
  double acc = th[0] * X[0];
  acc = acc + th[1] * X[1];
  acc = acc + th[2] * X[2];
  acc = acc + th[3] * X[3];
  acc = acc + th[4] * X[4];
  return acc;
}

// The batch model from exact sums: the latency (*t, fp64), the regime
// (returned: 2*phase + segment) and the share constants k[0..3] (fp64).
// th: theta[phase][segment][k] at (phase*2 + segment)*5 + k; S: S0..S3.
__host__ __device__ inline int eq1_batch(const double* th, const double* S, int64_t n,
                                         uint64_t Psum, uint64_t Csum, uint64_t Qsum,
                                         bool prefill, double* t, double* k) {
#pragma clang fp contract(off)
  const double X[5] = {S[0], S[1] * (double)Psum, S[2] * (double)Csum, S[3] * (double)Qsum,
                       (double)n * (double)n};
  const int phase = prefill ? 0 : 1;
  const double* thm = th + (phase * 2 + 0) * 5;
  const double* thc = th + (phase * 2 + 1) * 5;
  const double tm = eq1(thm, X);
  const double tc = eq1(thc, X);
  // Roofline max of the two segments; ties stay memory-bound.
  const int seg = (tc > tm) ? 1 : 0;
  *t = seg ? tc : tm;
  const double* c = seg ? thc : thm;
  k[0] = c[0] * (S[0] / (double)n) + c[4] * (double)n;
  k[1] = c[1] * S[1];
  k[2] = c[2] * S[2];
  k[3] = c[3] * S[3];
  return 2 * phase + seg;
}

// fp32 share of one request from the fp32-rounded constants: three fused
// multiply-adds (correctly rounded on the host and the GPU alike).
__host__ __device__ inline float share_of(const float* k, int32_t p, int32_t c) {
#pragma clang fp contract(off)
  const float pf = (float)p;
  return fmaf(k[3], pf * pf, fmaf(k[2], (float)c, fmaf(k[1], pf, k[0])));
}

}  // namespace llmv
