// fit.hpp -- gfx950 kernels for fitting Eq. 1's coefficient sets by ordinary
// least squares and for the accuracy metrics of a coefficient set.
//
// The method (LLMVisor Sec. 2.1): the coefficients of Eq. 1 are fitted by OLS
// on profiled batch latencies, four sets (two phases x the memory-bound and
// the compute-bound segment); Sec. 3 / Appendix A report r^2 and the 90th /
// 99th percentile of the relative error.  Readings where the paper is silent:
//  * segment membership while fitting: rounds of (assign every nonempty
//    batch to the segment with the larger prediction under the current
//    coefficients, ties to the memory-bound one; refit each set);
//  * identifiability: when every batch of a set has sum p^2 == sum p (all
//    decode requests process one token), the p^2 coefficient keeps its
//    starting value; when every batch has sum c == 0, the c coefficient
//    does; the rest are fitted to y minus the kept terms; a set with fewer
//    batches than free coefficients, or with (numerically) dependent free
//    columns, keeps all its coefficients;
//  * r^2 = 1 - SSE / sum (y - mean y)^2 over the nonempty batches of a phase;
//  * relative error |yhat - y| / y over nonempty batches with y > 0, rounded
//    to fp32; percentile p = the ceil(p n)-th smallest (nearest rank).
//
// Work decomposition: the per-batch work is one pass over the batch sums
// (33 B per batch, plus 8 B of measured latency): k_fit_accum folds each
// batch into register accumulators of the normal equations of its set; one
// workgroup then reduces the per-workgroup sums in a fixed order and solves
// the four small systems.  Percentiles are exact: a radix select over the
// fp32 bit patterns (4 passes of 8 bits) for all six (phase, percentile)
// pairs at once.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace llmv {

constexpr int kFitSet = 23;            // per set: X X^T upper triangle (15), X y (5),
                                       // batches, batches with Q != P, batches with C != 0
constexpr int kFitVals = 4 * kFitSet;  // the four (phase, segment) sets
constexpr int kFitWG = 256;
constexpr int kFitReduceParts = 8;     // partial sums per column in the fixed-order reduction
constexpr int kMetricVals = 8;         // per phase: n, sum y, m (y > 0), unused; x2 phases
constexpr int kSelections = 6;         // (prefill, decode, all) x (p90, p99)

struct FitShape {
  double S[4];
};

// Shape constants and one fp64 coefficient vector theta[phase][segment][k].
struct FitModel {
  double S[4];
  double th[20];
};

// Eq. 1 under one coefficient set: the five terms added in order k = 0..4.
__device__ __forceinline__ double fit_eq1(const double* th, const double X[5]) {
  double acc = th[0] * X[0];
  acc = acc + th[1] * X[1];
  acc = acc + th[2] * X[2];
  acc = acc + th[3] * X[3];
  acc = acc + th[4] * X[4];
  return acc;
}

// Eq. 1's feature vector of batch b from its exact sums (Sec. 2.1).
__device__ __forceinline__ void fit_features(const double* S, const int64_t* __restrict__ sums,
                                             int64_t nB, int64_t b, double X[5]) {
  const int64_t n = sums[b];
  X[0] = S[0];
  X[1] = S[1] * (double)sums[nB + b];
  X[2] = S[2] * (double)sums[2 * nB + b];
  X[3] = S[3] * (double)sums[3 * nB + b];
  X[4] = (double)n * (double)n;
}

__device__ __forceinline__ double wave_sum_f64(double x) {
  for (int m = 32; m >= 1; m >>= 1) x += __shfl_xor(x, m, 64);
  return x;
}

// Per-workgroup sums of the normal equations of each set under the current
// coefficients theta (device [20]): partials[block][set*kFitSet + k].  Wave
// w of a workgroup owns set w: the four waves walk the same batches (one
// HBM read, the other three mostly cache hits), each lane adds the batches
// of its wave's set into 23 register accumulators.
__global__ __launch_bounds__(kFitWG) void k_fit_accum(const int64_t* __restrict__ sums,
                                                      const uint8_t* __restrict__ phase,
                                                      int64_t nB, const FitShape F,
                                                      const double* __restrict__ y,
                                                      const double* __restrict__ theta,
                                                      double* __restrict__ partials) {
  static_assert(kFitWG == 4 * 64, "one wave per (phase, segment) set");
  const int lane = threadIdx.x & 63, set = threadIdx.x >> 6;
  const int set_phase = set >> 1, set_seg = set & 1;
  double th[10];  // the two segment sets of this wave's phase
#pragma unroll
  for (int i = 0; i < 10; ++i) th[i] = theta[set_phase * 10 + i];
  double acc[kFitSet];
#pragma unroll
  for (int i = 0; i < kFitSet; ++i) acc[i] = 0.0;

  const int64_t stride = (int64_t)gridDim.x * 64;
  for (int64_t b = (int64_t)blockIdx.x * 64 + lane; b < nB; b += stride) {
    const int64_t n = sums[b];
    if (n == 0 || (phase[b] == 0 ? 0 : 1) != set_phase) continue;
    double X[5];
    fit_features(F.S, sums, nB, b, X);
    // Roofline max of the two segments; ties stay memory-bound.
    const int seg = fit_eq1(th + 5, X) > fit_eq1(th, X) ? 1 : 0;
    if (seg != set_seg) continue;
    const double yb = y[b];
    int k = 0;
#pragma unroll
    for (int i = 0; i < 5; ++i)
#pragma unroll
      for (int j = i; j < 5; ++j) acc[k++] += X[i] * X[j];
#pragma unroll
    for (int i = 0; i < 5; ++i) acc[15 + i] += X[i] * yb;
    acc[20] += 1.0;
    acc[21] += sums[3 * nB + b] != sums[nB + b] ? 1.0 : 0.0;
    acc[22] += sums[2 * nB + b] != 0 ? 1.0 : 0.0;
  }
#pragma unroll
  for (int i = 0; i < kFitSet; ++i) {
    const double t = wave_sum_f64(acc[i]);
    if (lane == 0) partials[(int64_t)blockIdx.x * kFitVals + set * kFitSet + i] = t;
  }
}

// Column sums of partials[grid][ncols] in a fixed order, by one workgroup of
// ncols * kFitReduceParts threads (ncols <= 128); the result lands in LDS
// tot[ncols].
__device__ __forceinline__ void reduce_columns(const double* __restrict__ partials, int grid,
                                               int ncols, double* red, double* tot) {
  const int t = threadIdx.x;
  if (t < ncols * kFitReduceParts) {
    const int col = t % ncols, part = t / ncols;
    double s = 0.0;
    for (int blk = part; blk < grid; blk += kFitReduceParts) s += partials[(int64_t)blk * ncols + col];
    red[part * ncols + col] = s;
  }
  __syncthreads();
  if (t < ncols) {
    double s = 0.0;
    for (int part = 0; part < kFitReduceParts; ++part) s += red[part * ncols + t];
    tot[t] = s;
  }
  __syncthreads();
}

// Solves one set's normal equations over its free coefficients (Jacobi
// scaling, then Cholesky); returns false when the set keeps its
// coefficients.  A: 15 upper-triangle entries, r: 5 entries of X y.
__device__ inline bool solve_set(const double* A15, const double* r, double cnt, double npq,
                                 double nc, double* th) {
  int free_[5], nf = 0;
  bool kept[5] = {false, false, false, false, false};
  if (nc == 0.0) kept[2] = true;
  if (npq == 0.0) kept[3] = true;
  for (int i = 0; i < 5; ++i)
    if (!kept[i]) free_[nf++] = i;
  if (cnt < (double)nf) return false;
  double A[5][5];
  int k = 0;
  for (int i = 0; i < 5; ++i)
    for (int j = i; j < 5; ++j) A[i][j] = A[j][i] = A15[k++];
  double M[5][5], b[5], d[5];
  for (int a = 0; a < nf; ++a) {
    const int i = free_[a];
    double rhs = r[i];
    for (int j = 0; j < 5; ++j)
      if (kept[j]) rhs -= A[i][j] * th[j];
    if (!(A[i][i] > 0.0)) return false;
    d[a] = sqrt(A[i][i]);
    b[a] = rhs / d[a];
  }
  for (int a = 0; a < nf; ++a)
    for (int c = 0; c < nf; ++c) M[a][c] = A[free_[a]][free_[c]] / (d[a] * d[c]);
  // Cholesky M = L L^T (unit diagonal after scaling); a tiny pivot means
  // dependent columns
  double L[5][5];
  for (int j = 0; j < nf; ++j) {
    double s = M[j][j];
    for (int q = 0; q < j; ++q) s -= L[j][q] * L[j][q];
    if (!(s > 1e-12)) return false;
    L[j][j] = sqrt(s);
    for (int i = j + 1; i < nf; ++i) {
      double t = M[i][j];
      for (int q = 0; q < j; ++q) t -= L[i][q] * L[j][q];
      L[i][j] = t / L[j][j];
    }
  }
  double z[5], x[5];
  for (int i = 0; i < nf; ++i) {
    double t = b[i];
    for (int q = 0; q < i; ++q) t -= L[i][q] * z[q];
    z[i] = t / L[i][i];
  }
  for (int i = nf - 1; i >= 0; --i) {
    double t = z[i];
    for (int q = i + 1; q < nf; ++q) t -= L[q][i] * x[q];
    x[i] = t / L[i][i];
  }
  for (int a = 0; a < nf; ++a) th[free_[a]] = x[a] / d[a];
  return true;
}

// One workgroup: the normal equations of the four sets summed over the
// per-workgroup partials in a fixed order, then each set solved; theta
// (device [20]) is updated in place and counts[4] receives each set's batch
// count.
__global__ __launch_bounds__(kFitVals * kFitReduceParts) void k_fit_solve(
    const double* __restrict__ partials, int grid, double* __restrict__ theta,
    long long* __restrict__ counts) {
  __shared__ double s_red[kFitReduceParts * kFitVals];
  __shared__ double s_tot[kFitVals];
  reduce_columns(partials, grid, kFitVals, s_red, s_tot);
  const int g = threadIdx.x;
  if (g < 4) {
    const double* a = s_tot + g * kFitSet;
    double th[5];
    for (int i = 0; i < 5; ++i) th[i] = theta[g * 5 + i];
    if (solve_set(a, a + 15, a[20], a[21], a[22], th))
      for (int i = 0; i < 5; ++i) theta[g * 5 + i] = th[i];
    counts[g] = (long long)a[20];
  }
}

// Fitting starts from theta0: copies it into theta (device [20]) and clears
// the set counts.
__global__ __launch_bounds__(64) void k_fit_init(const FitModel M, double* __restrict__ theta,
                                                 long long* __restrict__ counts) {
  const int t = threadIdx.x;
  if (t < 20) theta[t] = M.th[t];
  if (t < 4) counts[t] = 0;
}

// ------------------------------------------------------------ metrics

// Pass 1: prediction and relative error of every batch (NaN for an empty
// batch or y <= 0) and, per phase, the batch count, sum y and the count of
// relative errors: partials[block][8].
__global__ __launch_bounds__(kFitWG) void k_fit_metrics1(const int64_t* __restrict__ sums,
                                                         const uint8_t* __restrict__ phase,
                                                         int64_t nB, const FitModel A,
                                                         const double* __restrict__ y,
                                                         float* __restrict__ rel_err,
                                                         double* __restrict__ partials) {
  __shared__ double s_red[kFitWG / 64][kMetricVals];
  double acc[kMetricVals] = {0, 0, 0, 0, 0, 0, 0, 0};
  const int64_t stride = (int64_t)gridDim.x * kFitWG;
  for (int64_t b = (int64_t)blockIdx.x * kFitWG + threadIdx.x; b < nB; b += stride) {
    float e = __builtin_nanf("");
    if (sums[b] != 0) {
      double X[5];
      fit_features(A.S, sums, nB, b, X);
      const int ph = phase[b] == 0 ? 0 : 1;
      const double tm = fit_eq1(A.th + (ph * 2 + 0) * 5, X), tc = fit_eq1(A.th + (ph * 2 + 1) * 5, X);
      const double yhat = tc > tm ? tc : tm, yb = y[b];
      if (yb > 0) e = (float)(fabs(yhat - yb) / yb);
#pragma unroll
      for (int q = 0; q < 2; ++q) {
        acc[q * 4 + 0] += ph == q ? 1.0 : 0.0;
        acc[q * 4 + 1] += ph == q ? yb : 0.0;
        acc[q * 4 + 2] += (ph == q && yb > 0) ? 1.0 : 0.0;
      }
    }
    if (rel_err) rel_err[b] = e;
  }
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
  for (int i = 0; i < kMetricVals; ++i) {
    const double t = wave_sum_f64(acc[i]);
    if (lane == 0) s_red[wave][i] = t;
  }
  __syncthreads();
  if (threadIdx.x < kMetricVals) {
    double t = 0.0;
    for (int w = 0; w < kFitWG / 64; ++w) t += s_red[w][threadIdx.x];
    partials[(int64_t)blockIdx.x * kMetricVals + threadIdx.x] = t;
  }
}

// Sums pass-1 partials (fixed order) into tot[8].
__global__ __launch_bounds__(kMetricVals * kFitReduceParts) void k_fit_metrics_sum(
    const double* __restrict__ partials, int grid, int ncols, double* __restrict__ tot) {
  __shared__ double s_red[kFitReduceParts * kMetricVals];
  __shared__ double s_tot[kMetricVals];
  reduce_columns(partials, grid, ncols, s_red, s_tot);
  if (threadIdx.x < ncols) tot[threadIdx.x] = s_tot[threadIdx.x];
}

// Pass 2: per phase (and all), sum (y - mean)^2 and sum (y - yhat)^2 with
// the means of pass 1 (tot1[8]): partials[block][8] = (prefill tot, sse,
// decode tot, sse, all tot, sse, -, -).  Means per group are taken from the
// pass-1 sums.
__global__ __launch_bounds__(kFitWG) void k_fit_metrics2(const int64_t* __restrict__ sums,
                                                         const uint8_t* __restrict__ phase,
                                                         int64_t nB, const FitModel A,
                                                         const double* __restrict__ y,
                                                         const double* __restrict__ tot1,
                                                         double* __restrict__ partials) {
  __shared__ double s_red[kFitWG / 64][kMetricVals];
  const double n0 = tot1[0], n1 = tot1[4];
  const double mean[3] = {n0 > 0 ? tot1[1] / n0 : 0.0, n1 > 0 ? tot1[5] / n1 : 0.0,
                          n0 + n1 > 0 ? (tot1[1] + tot1[5]) / (n0 + n1) : 0.0};
  double acc[kMetricVals] = {0, 0, 0, 0, 0, 0, 0, 0};
  const int64_t stride = (int64_t)gridDim.x * kFitWG;
  for (int64_t b = (int64_t)blockIdx.x * kFitWG + threadIdx.x; b < nB; b += stride) {
    if (sums[b] == 0) continue;
    double X[5];
    fit_features(A.S, sums, nB, b, X);
    const int ph = phase[b] == 0 ? 0 : 1;
    const double tm = fit_eq1(A.th + (ph * 2 + 0) * 5, X), tc = fit_eq1(A.th + (ph * 2 + 1) * 5, X);
    const double yhat = tc > tm ? tc : tm, yb = y[b];
    const double r = yb - yhat;
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      const double dv = yb - mean[q];
      acc[q * 2 + 0] += ph == q ? dv * dv : 0.0;
      acc[q * 2 + 1] += ph == q ? r * r : 0.0;
    }
    const double da = yb - mean[2];
    acc[4] += da * da;
    acc[5] += r * r;
  }
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
  for (int i = 0; i < kMetricVals; ++i) {
    const double t = wave_sum_f64(acc[i]);
    if (lane == 0) s_red[wave][i] = t;
  }
  __syncthreads();
  if (threadIdx.x < kMetricVals) {
    double t = 0.0;
    for (int w = 0; w < kFitWG / 64; ++w) t += s_red[w][threadIdx.x];
    partials[(int64_t)blockIdx.x * kMetricVals + threadIdx.x] = t;
  }
}

// Radix select state of one selection: the bits chosen so far (prefix, the
// top 8*pass bits) and the rank still to find inside the prefix bucket
// (1-based; 0 = no values).
struct SelState {
  unsigned int prefix;
  unsigned int rank;
};

// One radix pass: hist[sel][digit] counts the relative errors of the
// selection's group whose top 8*pass bits equal its prefix, by the next 8
// bits.  Selection s: group s / 2 (0 prefill, 1 decode, 2 all).
__global__ __launch_bounds__(kFitWG) void k_select_hist(const float* __restrict__ rel_err,
                                                        const uint8_t* __restrict__ phase,
                                                        int64_t nB, int pass,
                                                        const SelState* __restrict__ st,
                                                        unsigned int* __restrict__ hist) {
  __shared__ unsigned int s_hist[kSelections * 256];
  for (int i = threadIdx.x; i < kSelections * 256; i += kFitWG) s_hist[i] = 0u;
  __syncthreads();
  unsigned int pre[kSelections];
#pragma unroll
  for (int s = 0; s < kSelections; ++s) pre[s] = st[s].prefix;
  const int shift = 24 - 8 * pass;
  const int64_t stride = (int64_t)gridDim.x * kFitWG;
  for (int64_t b = (int64_t)blockIdx.x * kFitWG + threadIdx.x; b < nB; b += stride) {
    const float e = rel_err[b];
    if (!(e >= 0.0f)) continue;  // NaN: empty batch or y <= 0
    const unsigned int u = __float_as_uint(e);
    const int grp = phase[b] == 0 ? 0 : 1;
    const unsigned int digit = (u >> shift) & 255u;
    const unsigned int top = pass == 0 ? 0u : (u >> (shift + 8));
#pragma unroll
    for (int s = 0; s < kSelections; ++s) {
      const int sg = s / 2;
      if ((sg == grp || sg == 2) && top == pre[s]) atomicAdd(&s_hist[s * 256 + digit], 1u);
    }
  }
  __syncthreads();
  for (int i = threadIdx.x; i < kSelections * 256; i += kFitWG)
    if (s_hist[i]) atomicAdd(&hist[i], s_hist[i]);
}

// After a radix pass: each selection moves into the bucket holding its rank;
// the histogram is cleared for the next pass.  One workgroup of 64 threads.
__global__ __launch_bounds__(64) void k_select_pick(SelState* __restrict__ st,
                                                    unsigned int* __restrict__ hist) {
  const int s = threadIdx.x;
  if (s < kSelections && st[s].rank > 0) {
    unsigned int below = 0, digit = 0;
    for (; digit < 256; ++digit) {
      const unsigned int h = hist[s * 256 + digit];
      if (below + h >= st[s].rank) break;
      below += h;
    }
    st[s].prefix = (st[s].prefix << 8) | (digit & 255u);
    st[s].rank -= below;
  }
  __syncthreads();
  for (int i = threadIdx.x; i < kSelections * 256; i += 64) hist[i] = 0u;
}

// The selections' starting ranks from the pass-1 counts (tot1: m at [2] and
// [6]): ceil(m * 9/10) and ceil(m * 99/100), 0 when m = 0.  Also clears the
// histogram.
__global__ __launch_bounds__(64) void k_select_init(const double* __restrict__ tot1,
                                                    SelState* __restrict__ st,
                                                    unsigned int* __restrict__ hist) {
  const int s = threadIdx.x;
  if (s < kSelections) {
    const int g = s / 2;
    const unsigned long long m0 = (unsigned long long)tot1[2], m1 = (unsigned long long)tot1[6];
    const unsigned long long m = g == 0 ? m0 : (g == 1 ? m1 : m0 + m1);
    const unsigned long long num = (s & 1) ? 99 : 9, den = (s & 1) ? 100 : 10;
    st[s].prefix = 0u;
    st[s].rank = (unsigned int)((num * m + den - 1) / den);
  }
  for (int i = threadIdx.x; i < kSelections * 256; i += 64) hist[i] = 0u;
}

// The metrics from the pass sums and the selected percentiles:
// out[g*4 + (0, 1, 2, 3)] = (r^2, p90, p99, batches) for g = prefill,
// decode, all.  r^2 is NaN without batches or when every y is equal; a
// percentile is NaN without relative errors.
__global__ __launch_bounds__(64) void k_fit_metrics_final(const double* __restrict__ tot1,
                                                          const double* __restrict__ tot2,
                                                          const SelState* __restrict__ st,
                                                          double* __restrict__ out) {
  const int g = threadIdx.x;
  if (g >= 3) return;
  const double n = g == 2 ? tot1[0] + tot1[4] : tot1[4 * g];
  const double sst = tot2[2 * g], sse = tot2[2 * g + 1];
  const double nan = __builtin_nan("");
  out[g * 4 + 0] = (n > 0 && sst > 0) ? 1.0 - sse / sst : nan;
  for (int q = 0; q < 2; ++q) {
    const SelState s = st[2 * g + q];
    out[g * 4 + 1 + q] = s.rank > 0 ? (double)__uint_as_float(s.prefix) : nan;
  }
  out[g * 4 + 3] = n;
}

}  // namespace llmv
