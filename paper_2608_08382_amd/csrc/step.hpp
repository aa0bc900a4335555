// step.hpp -- one scheduler step, attributed with the least latency.
//
// The paper runs the attribution inside the serving loop, once per
// scheduling step, for admission control and accounting (Sec. 1; Sec. 2.1,
// last paragraph).  A step is one batch, or a handful, of at most a few
// thousand requests.  k_step attributes such a trace in one workgroup of
// kStepWG threads and one launch: every global load (offsets, p, c, tenant)
// is issued at once, the batch of each request is found by binary search in
// the offsets held in LDS, the exact sums go to LDS accumulators (a wave
// whose requests all lie in one batch adds them once), one thread per batch
// evaluates Eq. 1 (model.hpp), and each request's share and its tenant's
// sum follow.  No workspace, no chunk table, no second kernel.
#pragma once

#include "kernels.hpp"

namespace llmv {

constexpr int kStepWG = 1024;                            // threads of the one workgroup
constexpr int kStepPer = 4;                              // requests per thread
constexpr int64_t kStepN = (int64_t)kStepWG * kStepPer;  // requests per step, at most
constexpr int kStepB = 1024;                             // batches per step, at most
constexpr int kStepT = 4096;                             // tenants of the LDS histogram
// The packed (sum c, zero count) word of kernels.hpp holds for a step:
// fewer than 2^16 requests, each c < 2^31.
static_assert(kStepN < (1 << 16) && (uint64_t)kStepN * 0x7fffffffull < kZeroUnit,
              "a step's zero count and sum of c fit their fields");

// Eq. 1 attribution of a trace of at most kStepN requests and kStepB
// batches (and, with TEN, at most kStepT tenants): latency, regime, shares
// and tenant sums as llmv_attribute, each optional.  One workgroup.
template <bool TEN>
__global__ __launch_bounds__(kStepWG) void k_step(const Params P) {
  __shared__ int64_t s_off[kStepB + 1];
  __shared__ unsigned long long s_sum[3][kStepB];  // sum p, sum c | zero count << 48, sum p^2
  __shared__ v4f s_k[kStepB];                      // share constants per batch
  extern __shared__ double s_hist[];               // [n_tenants] with TEN
  const int tid = threadIdx.x, lane = tid & 63;
  const int64_t nB = P.nB, N = P.N;

  // ---- every global load first
  for (int64_t b = tid; b <= nB; b += kStepWG) s_off[b] = P.off[b];
  int32_t pv[kStepPer], cv[kStepPer], tv[kStepPer];
#pragma unroll
  for (int j = 0; j < kStepPer; ++j) {
    const int64_t i = tid + (int64_t)kStepWG * j;
    const bool v = i < N;
    pv[j] = v ? P.p[i] : 0;
    cv[j] = v ? P.c[i] : 0;
    tv[j] = (TEN && v) ? P.tenant[i] : 0;
  }
  for (int64_t b = tid; b < nB; b += kStepWG) s_sum[0][b] = s_sum[1][b] = s_sum[2][b] = 0ull;
  if (TEN)
    for (int u = tid; u < P.n_tenants; u += kStepWG) s_hist[u] = 0.0;
  __syncthreads();

  // ---- batch of each request: the last batch starting at or before it
  // (empty batches start where the next one does and are passed over)
  int32_t bid[kStepPer];
#pragma unroll
  for (int j = 0; j < kStepPer; ++j) {
    const int64_t i = tid + (int64_t)kStepWG * j;
    int32_t lo = 0, hi = (int32_t)nB - 1;
    while (lo < hi) {
      const int32_t mid = (lo + hi + 1) >> 1;
      if (s_off[mid] <= i) lo = mid;
      else hi = mid - 1;
    }
    bid[j] = lo;
  }

  // ---- exact batch sums
#pragma unroll
  for (int j = 0; j < kStepPer; ++j) {
    const int64_t i = tid + (int64_t)kStepWG * j;
    const bool v = i < N;
    const uint64_t p = (uint32_t)pv[j], c = (uint32_t)cv[j];
    uint64_t sp = v ? p : 0ull;
    uint64_t scz = v ? c + (c == 0 ? kZeroUnit : 0ull) : 0ull;
    uint64_t sq = v ? p * p : 0ull;
    // lanes hold consecutive requests: when every valid one is in lane 0's
    // batch, the wave adds its sums once
    const int32_t b0 = __shfl(bid[j], 0, 64);
    const bool one = __ballot(v && bid[j] != b0) == 0;
    if (one) {
      if (__ballot(v) != 0) {
        sp = wave_sum(sp);
        scz = wave_sum(scz);
        sq = wave_sum(sq);
        if (lane == 0) {
          atomicAdd(&s_sum[0][b0], (unsigned long long)sp);
          atomicAdd(&s_sum[1][b0], (unsigned long long)scz);
          atomicAdd(&s_sum[2][b0], (unsigned long long)sq);
        }
      }
    } else if (v) {
      atomicAdd(&s_sum[0][bid[j]], (unsigned long long)sp);
      atomicAdd(&s_sum[1][bid[j]], (unsigned long long)scz);
      atomicAdd(&s_sum[2][bid[j]], (unsigned long long)sq);
    }
  }
  __syncthreads();

  // ---- per batch: Eq. 1, the segment, the share constants
  for (int64_t b = tid; b < nB; b += kStepWG) {
    const int64_t n = s_off[b + 1] - s_off[b];
    if (n == 0) {
      if (P.latency) P.latency[b] = 0.0f;
      if (P.regime) P.regime[b] = 255;
      continue;
    }
    const uint64_t Ps = s_sum[0][b], CZ = s_sum[1][b], Qs = s_sum[2][b];
    // decode iff every request processes one token over a nonzero context
    const bool prefill = (Ps != (uint64_t)n) || ((CZ >> 48) != 0);
    double t, k[4];
    const int regime = eq1_batch(P.th, P.S, n, Ps, CZ & kCMask, Qs, prefill, &t, k);
    if (P.latency) P.latency[b] = (float)t;
    if (P.regime) P.regime[b] = (uint8_t)regime;
    s_k[b] = (v4f){(float)k[0], (float)k[1], (float)k[2], (float)k[3]};
  }
  __syncthreads();

  // ---- per request: the share, its tenant's sum
  if (P.share || TEN) {
#pragma unroll
    for (int j = 0; j < kStepPer; ++j) {
      const int64_t i = tid + (int64_t)kStepWG * j;
      if (i >= N) continue;
      const v4f k4 = s_k[bid[j]];
      const float K[4] = {k4.x, k4.y, k4.z, k4.w};
      const float s = share_of(K, pv[j], cv[j]);
      if (P.share) P.share[i] = s;
      if (TEN) atomicAdd(&s_hist[tv[j]], (double)s);
    }
  }
  if (TEN) {
    __syncthreads();
    for (int u = tid; u < P.n_tenants; u += kStepWG) P.tenant_sums[u] = s_hist[u];
  }
}

}  // namespace llmv
