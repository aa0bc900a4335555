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
//  * the extended model (Eq. 1 plus a5*S5*sum p*c and a6*S6*|B|) is fitted
//    the same way with seven columns; a5 keeps its starting value when
//    sum p*c == sum c in every batch of a set, a6 when sum p == |B|;
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

// Accumulators of one (phase, segment) set for NC columns (5: Eq. 1, 7: the
// extended model): the upper triangle of X^T X, X^T y, the batch count and
// the identifiability counts (batches with Q != P, C != 0, and for NC = 7
// R != C, P != |B|).
template <int NC>
struct FitCols {
  static_assert(NC == 5 || NC == 7, "Eq. 1 or the extended model");
  static constexpr int kTri = NC * (NC + 1) / 2;
  static constexpr int kFlags = NC == 5 ? 3 : 5;
  static constexpr int kSet = kTri + NC + kFlags;
  static constexpr int kVals = 4 * kSet;  // the four (phase, segment) sets
};
constexpr int kFitValsMax = FitCols<7>::kVals;
constexpr int kFitWG = 256;
constexpr int kReduceWG = 1024;        // threads of the fixed-order column reductions
constexpr int kMetricVals = 8;         // per phase: n, sum y, m (y > 0), unused; x2 phases
constexpr int kSelections = 6;         // (prefill, decode, all) x (p90, p99)

// Shape constants: S0..S3, and for the extended model S5, S6.
struct FitShape {
  double S[6];
};

// Shape constants and one fp64 coefficient vector theta[phase][segment][k].
template <int NC>
struct FitModel {
  double S[6];
  double th[4 * NC];
};

// One coefficient set: the NC terms added in order k = 0, 1, ...
template <int NC>
__device__ __forceinline__ double fit_eq(const double* th, const double X[NC]) {
  double acc = th[0] * X[0];
#pragma unroll
  for (int k = 1; k < NC; ++k) acc = acc + th[k] * X[k];
  return acc;
}

// The feature vector of a batch from its exact sums (Sec. 2.1):
// (S0, S1*P, S2*C, S3*Q, |B|^2), and for the extended model (S5*R, S6*|B|).
template <int NC>
__device__ __forceinline__ void fit_features(const double* S, int64_t n, int64_t P, int64_t C,
                                             int64_t Q, int64_t R, double X[NC]) {
  X[0] = S[0];
  X[1] = S[1] * (double)P;
  X[2] = S[2] * (double)C;
  X[3] = S[3] * (double)Q;
  X[4] = (double)n * (double)n;
  if constexpr (NC == 7) {
    X[5] = S[4] * (double)R;
    X[6] = S[5] * (double)n;
  }
}

__device__ __forceinline__ double wave_sum_f64(double x) {
  for (int m = 32; m >= 1; m >>= 1) x += __shfl_xor(x, m, 64);
  return x;
}

// The state of one batch: exact sums, measured latency and phase.
struct BatchRegs {
  int64_t n, P, C, Q, R;
  double y;
  int ph;  // 0 prefill, 1 decode, -1 empty or past the end
};

// sums: [4][nB] (|B|, P, C, Q), for NC = 7 [5][nB] with R = sum p*c.
template <int NC>
__device__ __forceinline__ BatchRegs load_batch(const int64_t* __restrict__ sums,
                                                const uint8_t* __restrict__ phase,
                                                const double* __restrict__ y, int64_t nB,
                                                int64_t b) {
  BatchRegs r{0, 0, 0, 0, 0, 0.0, -1};
  if (b < nB) {
    r.n = sums[b];
    r.P = sums[nB + b];
    r.C = sums[2 * nB + b];
    r.Q = sums[3 * nB + b];
    if constexpr (NC == 7) r.R = sums[4 * nB + b];
    r.y = y[b];
    r.ph = r.n == 0 ? -1 : (phase[b] == 0 ? 0 : 1);
  }
  return r;
}

// Per-workgroup sums of the normal equations of each set under the current
// coefficients theta (device [4*NC]): partials[block][set*kSet + k].
// A workgroup walks chunks of kFitWG batches: the chunk is loaded once,
// coalesced (the next chunk's loads are issued before the current one is
// processed) and staged in LDS; wave w then folds the chunk's batches of set
// w (phase w/2, segment w%2) into kSet register accumulators per lane.
template <int NC>
__global__ __launch_bounds__(kFitWG) void k_fit_accum(const int64_t* __restrict__ sums,
                                                      const uint8_t* __restrict__ phase,
                                                      int64_t nB, const FitShape F,
                                                      const double* __restrict__ y,
                                                      const double* __restrict__ theta,
                                                      double* __restrict__ partials) {
  static_assert(kFitWG == 4 * 64, "one wave per (phase, segment) set");
  using Cols = FitCols<NC>;
  constexpr int kTri = Cols::kTri, kSet = Cols::kSet;
  __shared__ int64_t s_n[kFitWG], s_P[kFitWG], s_C[kFitWG], s_Q[kFitWG];
  __shared__ int64_t s_R[NC == 7 ? kFitWG : 1];
  __shared__ double s_y[kFitWG];
  __shared__ int s_ph[kFitWG];
  const int tid = threadIdx.x, lane = tid & 63, set = tid >> 6;
  const int set_phase = set >> 1, set_seg = set & 1;
  double th[2 * NC];  // the two segment sets of this wave's phase
#pragma unroll
  for (int i = 0; i < 2 * NC; ++i) th[i] = theta[set_phase * 2 * NC + i];
  double acc[kSet];
#pragma unroll
  for (int i = 0; i < kSet; ++i) acc[i] = 0.0;

  const int64_t stride = (int64_t)gridDim.x * kFitWG;
  int64_t base = (int64_t)blockIdx.x * kFitWG;
  BatchRegs cur = load_batch<NC>(sums, phase, y, nB, base + tid);
  for (; base < nB; base += stride) {
    s_n[tid] = cur.n;
    s_P[tid] = cur.P;
    s_C[tid] = cur.C;
    s_Q[tid] = cur.Q;
    if constexpr (NC == 7) s_R[tid] = cur.R;
    s_y[tid] = cur.y;
    s_ph[tid] = cur.ph;
    __syncthreads();
    cur = load_batch<NC>(sums, phase, y, nB, base + stride + tid);  // next chunk, in flight
#pragma unroll
    for (int k = 0; k < kFitWG / 64; ++k) {
      const int i = k * 64 + lane;
      if (s_ph[i] != set_phase) continue;
      const int64_t n = s_n[i], P = s_P[i], C = s_C[i], Q = s_Q[i];
      const int64_t R = NC == 7 ? s_R[i] : 0;
      double X[NC];
      fit_features<NC>(F.S, n, P, C, Q, R, X);
      // Roofline max of the two segments; ties stay memory-bound.
      const int seg = fit_eq<NC>(th + NC, X) > fit_eq<NC>(th, X) ? 1 : 0;
      if (seg != set_seg) continue;
      const double yb = s_y[i];
      int q = 0;
#pragma unroll
      for (int a = 0; a < NC; ++a)
#pragma unroll
        for (int c = a; c < NC; ++c) acc[q++] += X[a] * X[c];
#pragma unroll
      for (int a = 0; a < NC; ++a) acc[kTri + a] += X[a] * yb;
      acc[kTri + NC + 0] += 1.0;
      acc[kTri + NC + 1] += Q != P ? 1.0 : 0.0;
      acc[kTri + NC + 2] += C != 0 ? 1.0 : 0.0;
      if constexpr (NC == 7) {
        acc[kTri + NC + 3] += R != C ? 1.0 : 0.0;
        acc[kTri + NC + 4] += P != n ? 1.0 : 0.0;
      }
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < kSet; ++i) {
    const double t = wave_sum_f64(acc[i]);
    if (lane == 0) partials[(int64_t)blockIdx.x * Cols::kVals + set * kSet + i] = t;
  }
}

// Column sums of partials[grid][NCOLS] in a fixed order by one workgroup of
// kReduceWG threads: thread (part, col) adds rows part, part + PARTS, ...;
// then thread col adds the PARTS results in order.  The totals land in LDS
// tot[NCOLS].
template <int NCOLS>
__device__ __forceinline__ void reduce_columns(const double* __restrict__ partials, int grid,
                                               double* red, double* tot) {
  constexpr int PARTS = kReduceWG / NCOLS;
  const int t = threadIdx.x;
  if (t < PARTS * NCOLS) {
    const int col = t % NCOLS, part = t / NCOLS;
    double s = 0.0;
#pragma unroll 8
    for (int blk = part; blk < grid; blk += PARTS) s += partials[(int64_t)blk * NCOLS + col];
    red[part * NCOLS + col] = s;
  }
  __syncthreads();
  if (t < NCOLS) {
    double s = 0.0;
#pragma unroll 8
    for (int part = 0; part < PARTS; ++part) s += red[part * NCOLS + t];
    tot[t] = s;
  }
  __syncthreads();
}

// Solves one set's normal equations over its free coefficients; returns
// false when the set keeps its coefficients.  A: the upper triangle of
// X^T X, r: X^T y, f: the batch count and the identifiability counts
// (FitCols).  The free columns are scaled to unit diagonal and factorised by
// Cholesky; a kept column becomes an identity row (its term is moved to the
// right-hand side first), so the code is fully unrolled.  A pivot below
// 1e-12 (condition number of the scaled columns beyond ~1e6) counts as
// dependent columns.
template <int NC>
__device__ inline bool solve_set(const double* At, const double* r, const double* f,
                                 double th[NC]) {
  bool kept[NC];
#pragma unroll
  for (int k = 0; k < NC; ++k) kept[k] = false;
  kept[2] = f[2] == 0.0;  // sum c == 0 in every batch
  kept[3] = f[1] == 0.0;  // sum p^2 == sum p in every batch
  if constexpr (NC == 7) {
    kept[5] = f[3] == 0.0;  // sum p*c == sum c in every batch
    kept[6] = f[4] == 0.0;  // sum p == |B| in every batch
  }
  int nf = 0;
#pragma unroll
  for (int k = 0; k < NC; ++k) nf += kept[k] ? 0 : 1;
  if (f[0] < (double)nf) return false;
  double A[NC][NC];
  int q = 0;
#pragma unroll
  for (int i = 0; i < NC; ++i)
#pragma unroll
    for (int j = i; j < NC; ++j) {
      A[i][j] = At[q];
      A[j][i] = At[q];
      ++q;
    }
  double d[NC], b[NC];
#pragma unroll
  for (int i = 0; i < NC; ++i) {
    double rhs = r[i];
#pragma unroll
    for (int j = 0; j < NC; ++j)
      if (kept[j]) rhs -= A[i][j] * th[j];
    if (kept[i]) {
      d[i] = 1.0;
      b[i] = 0.0;
    } else {
      if (!(A[i][i] > 0.0)) return false;
      d[i] = sqrt(A[i][i]);
      b[i] = rhs / d[i];
    }
  }
  // scaled matrix, factorised in place (lower triangle)
#pragma unroll
  for (int i = 0; i < NC; ++i)
#pragma unroll
    for (int j = 0; j < NC; ++j)
      A[i][j] = (kept[i] || kept[j]) ? (i == j ? 1.0 : 0.0) : A[i][j] / (d[i] * d[j]);
#pragma unroll
  for (int j = 0; j < NC; ++j) {
    double s = A[j][j];
#pragma unroll
    for (int k = 0; k < j; ++k) s -= A[j][k] * A[j][k];
    if (!(s > 1e-12)) return false;
    A[j][j] = sqrt(s);
#pragma unroll
    for (int i = j + 1; i < NC; ++i) {
      double t = A[i][j];
#pragma unroll
      for (int k = 0; k < j; ++k) t -= A[i][k] * A[j][k];
      A[i][j] = t / A[j][j];
    }
  }
  double z[NC], x[NC];
#pragma unroll
  for (int i = 0; i < NC; ++i) {
    double t = b[i];
#pragma unroll
    for (int k = 0; k < i; ++k) t -= A[i][k] * z[k];
    z[i] = t / A[i][i];
  }
#pragma unroll
  for (int i = NC - 1; i >= 0; --i) {
    double t = z[i];
#pragma unroll
    for (int k = i + 1; k < NC; ++k) t -= A[k][i] * x[k];
    x[i] = t / A[i][i];
  }
#pragma unroll
  for (int i = 0; i < NC; ++i)
    if (!kept[i]) th[i] = x[i] / d[i];
  return true;
}

// One workgroup: the normal equations of the four sets summed over the
// per-workgroup partials in a fixed order, then each set solved; theta
// (device [4*NC]) is updated in place and counts[4] receives each set's
// batch count.
template <int NC>
__global__ __launch_bounds__(kReduceWG) void k_fit_solve(const double* __restrict__ partials,
                                                         int grid, double* __restrict__ theta,
                                                         long long* __restrict__ counts) {
  using Cols = FitCols<NC>;
  __shared__ double s_red[kReduceWG];
  __shared__ double s_tot[Cols::kVals];
  reduce_columns<Cols::kVals>(partials, grid, s_red, s_tot);
  const int g = threadIdx.x;
  if (g < 4) {
    const double* a = s_tot + g * Cols::kSet;
    double th[NC];
#pragma unroll
    for (int i = 0; i < NC; ++i) th[i] = theta[g * NC + i];
    if (solve_set<NC>(a, a + Cols::kTri, a + Cols::kTri + NC, th)) {
#pragma unroll
      for (int i = 0; i < NC; ++i) theta[g * NC + i] = th[i];
    }
    counts[g] = (long long)a[Cols::kTri + NC];
  }
}

// Fitting starts from theta0: copies it into theta (device [4*NC]) and
// clears the set counts.
template <int NC>
__global__ __launch_bounds__(64) void k_fit_init(const FitModel<NC> M, double* __restrict__ theta,
                                                 long long* __restrict__ counts) {
  const int t = threadIdx.x;
  if (t < 4 * NC) theta[t] = M.th[t];
  if (t < 4) counts[t] = 0;
}

// ------------------------------------------------------------ metrics

// The model's prediction (segment max) for a nonempty batch.
template <int NC>
__device__ __forceinline__ double predict(const FitModel<NC>& A, const BatchRegs& r) {
  double X[NC];
  fit_features<NC>(A.S, r.n, r.P, r.C, r.Q, r.R, X);
  const double tm = fit_eq<NC>(A.th + (r.ph * 2 + 0) * NC, X);
  const double tc = fit_eq<NC>(A.th + (r.ph * 2 + 1) * NC, X);
  return tc > tm ? tc : tm;
}

// The workgroup's sums of acc[kMetricVals] into partials[block][...].
__device__ __forceinline__ void block_partials(const double acc[kMetricVals],
                                               double* __restrict__ partials) {
  __shared__ double s_red[kFitWG / 64][kMetricVals];
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
// (1-based; 0 = no values).  Selection s: group s / 2 (0 prefill, 1 decode,
// 2 all), p90 for even s, p99 for odd s.
struct SelState {
  unsigned int prefix;
  unsigned int rank;
};

// Selections whose histogram has to be counted.  Two selections of one
// group with the same prefix have the same histogram (p99 reuses p90's);
// an "all" selection whose prefix equals both phase selections' of its
// percentile has the sum of theirs.  In pass 0 every prefix is empty, so
// only the prefill and decode p90 histograms are counted.
__device__ __forceinline__ unsigned int counted_selections(const unsigned int pre[kSelections]) {
  unsigned int m = 0;
#pragma unroll
  for (int s = 0; s < kSelections; ++s) {
    const bool same_group = (s & 1) && pre[s] == pre[s - 1];
    const bool both_phases = s >= 4 && pre[s] == pre[s - 4] && pre[s] == pre[s - 2];
    if (!same_group && !both_phases) m |= 1u << s;
  }
  return m;
}

// Adds one relative error (group grp, or -1 for none) to the LDS histograms
// of the counted selections whose prefix it matches.
__device__ __forceinline__ void select_add(unsigned int* s_hist, float e, int grp, int pass,
                                           const unsigned int pre[kSelections],
                                           unsigned int counted) {
  if (grp < 0) return;
  const unsigned int u = __float_as_uint(e);
  const int shift = 24 - 8 * pass;
  const unsigned int digit = (u >> shift) & 255u;
  const unsigned int top = pass == 0 ? 0u : (u >> (shift + 8));
#pragma unroll
  for (int s = 0; s < kSelections; ++s) {
    const int sg = s / 2;
    if (((counted >> s) & 1u) && (sg == grp || sg == 2) && top == pre[s])
      atomicAdd(&s_hist[s * 256 + digit], 1u);
  }
}

// Adds a workgroup's LDS histograms into the global ones.
__device__ __forceinline__ void flush_hist(const unsigned int* s_hist, unsigned int counted,
                                           unsigned int* __restrict__ hist) {
  for (int i = threadIdx.x; i < kSelections * 256; i += blockDim.x)
    if (((counted >> (i / 256)) & 1u) && s_hist[i]) atomicAdd(&hist[i], s_hist[i]);
}

// Pass 1: prediction and relative error of every batch (NaN for an empty
// batch or y <= 0) and, per phase, the batch count, sum y and the count of
// relative errors: partials[block][8] = (n, sum y, m, -) for prefill, then
// decode.  Also the first radix pass of the percentile selection (the top 8
// bits of every error; hist must be zero on entry).
template <int NC>
__global__ __launch_bounds__(kFitWG) void k_fit_metrics1(const int64_t* __restrict__ sums,
                                                         const uint8_t* __restrict__ phase,
                                                         int64_t nB, const FitModel<NC> A,
                                                         const double* __restrict__ y,
                                                         float* __restrict__ rel_err,
                                                         double* __restrict__ partials,
                                                         unsigned int* __restrict__ hist) {
  __shared__ unsigned int s_hist[kSelections * 256];
  for (int i = threadIdx.x; i < kSelections * 256; i += kFitWG) s_hist[i] = 0u;
  __syncthreads();
  const unsigned int pre0[kSelections] = {0, 0, 0, 0, 0, 0};
  const unsigned int counted = counted_selections(pre0);
  double acc[kMetricVals] = {0, 0, 0, 0, 0, 0, 0, 0};
  const int64_t stride = (int64_t)gridDim.x * kFitWG;
  for (int64_t b = (int64_t)blockIdx.x * kFitWG + threadIdx.x; b < nB; b += stride) {
    const BatchRegs r = load_batch<NC>(sums, phase, y, nB, b);
    float e = __builtin_nanf("");
    if (r.ph >= 0) {
      const double yhat = predict<NC>(A, r);
      if (r.y > 0) e = (float)(fabs(yhat - r.y) / r.y);
#pragma unroll
      for (int q = 0; q < 2; ++q) {
        acc[q * 4 + 0] += r.ph == q ? 1.0 : 0.0;
        acc[q * 4 + 1] += r.ph == q ? r.y : 0.0;
        acc[q * 4 + 2] += (r.ph == q && r.y > 0) ? 1.0 : 0.0;
      }
    }
    rel_err[b] = e;
    select_add(s_hist, e, (r.ph >= 0 && r.y > 0) ? r.ph : -1, 0, pre0, counted);
  }
  block_partials(acc, partials);  // synchronises the workgroup
  flush_hist(s_hist, counted, hist);
}

// Sums a pass's partials (fixed order) into tot[8].
__global__ __launch_bounds__(kReduceWG) void k_fit_metrics_sum(const double* __restrict__ partials,
                                                               int grid,
                                                               double* __restrict__ tot) {
  __shared__ double s_red[kReduceWG];
  __shared__ double s_tot[kMetricVals];
  reduce_columns<kMetricVals>(partials, grid, s_red, s_tot);
  if (threadIdx.x < kMetricVals) tot[threadIdx.x] = s_tot[threadIdx.x];
}

// Pass 2: per phase (and all), sum (y - mean)^2 and sum (y - yhat)^2 with
// the means of the pass-1 sums tot1[8]: partials[block][8] = (prefill
// sst, sse, decode sst, sse, all sst, sse, -, -).
template <int NC>
__global__ __launch_bounds__(kFitWG) void k_fit_metrics2(const int64_t* __restrict__ sums,
                                                         const uint8_t* __restrict__ phase,
                                                         int64_t nB, const FitModel<NC> A,
                                                         const double* __restrict__ y,
                                                         const double* __restrict__ tot1,
                                                         double* __restrict__ partials) {
  const double n0 = tot1[0], n1 = tot1[4];
  const double mean[3] = {n0 > 0 ? tot1[1] / n0 : 0.0, n1 > 0 ? tot1[5] / n1 : 0.0,
                          n0 + n1 > 0 ? (tot1[1] + tot1[5]) / (n0 + n1) : 0.0};
  double acc[kMetricVals] = {0, 0, 0, 0, 0, 0, 0, 0};
  const int64_t stride = (int64_t)gridDim.x * kFitWG;
  for (int64_t b = (int64_t)blockIdx.x * kFitWG + threadIdx.x; b < nB; b += stride) {
    const BatchRegs r = load_batch<NC>(sums, phase, y, nB, b);
    if (r.ph < 0) continue;
    const double res = r.y - predict<NC>(A, r);
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      const double dv = r.y - mean[q];
      acc[q * 2 + 0] += r.ph == q ? dv * dv : 0.0;
      acc[q * 2 + 1] += r.ph == q ? res * res : 0.0;
    }
    const double da = r.y - mean[2];
    acc[4] += da * da;
    acc[5] += res * res;
  }
  block_partials(acc, partials);
}

// One later radix pass (pass 1..3): hist[sel][digit] counts the relative
// errors of the selection's group whose top 8*pass bits equal its prefix, by
// the next 8 bits (counted selections only).  Four errors per thread per
// iteration, their loads issued together.
constexpr int kSelUnroll = 4;
__global__ __launch_bounds__(kFitWG) void k_select_hist(const float* __restrict__ rel_err,
                                                        const uint8_t* __restrict__ phase,
                                                        int64_t nB, int pass,
                                                        const SelState* __restrict__ st,
                                                        unsigned int* __restrict__ hist) {
  __shared__ unsigned int s_hist[kSelections * 256];
  for (int i = threadIdx.x; i < kSelections * 256; i += kFitWG) s_hist[i] = 0u;
  unsigned int pre[kSelections];
#pragma unroll
  for (int s = 0; s < kSelections; ++s) pre[s] = st[s].prefix;
  const unsigned int counted = counted_selections(pre);
  __syncthreads();
  const int64_t step = (int64_t)kFitWG * kSelUnroll;
  const int64_t stride = (int64_t)gridDim.x * step;
  for (int64_t b0 = (int64_t)blockIdx.x * step + threadIdx.x; b0 < nB; b0 += stride) {
    float e[kSelUnroll];
    int ph[kSelUnroll];
#pragma unroll
    for (int u = 0; u < kSelUnroll; ++u) {
      const int64_t b = b0 + (int64_t)u * kFitWG;
      e[u] = b < nB ? rel_err[b] : __builtin_nanf("");
      ph[u] = b < nB ? (int)phase[b] : 0;
    }
#pragma unroll
    for (int u = 0; u < kSelUnroll; ++u)
      select_add(s_hist, e[u], e[u] >= 0.0f ? (ph[u] == 0 ? 0 : 1) : -1, pass, pre, counted);
  }
  __syncthreads();
  flush_hist(s_hist, counted, hist);
}

// After a radix pass: each selection moves into the bucket holding its rank
// (thread t owns digit t of every selection; an inclusive scan over the 256
// counts finds the bucket), and the histogram is cleared for the next pass.
// A selection that was not counted takes the histogram it equals (see
// counted_selections).  After the first pass (tot1 != NULL) the ranks come
// from the pass-1 counts m (tot1[2], tot1[6]): ceil(9m/10) and
// ceil(99m/100), 0 when m = 0.
__global__ __launch_bounds__(256) void k_select_pick(SelState* __restrict__ st,
                                                     unsigned int* __restrict__ hist,
                                                     const double* __restrict__ tot1) {
  __shared__ unsigned int s_wave[kSelections][4];
  const int t = threadIdx.x, lane = t & 63, w = t >> 6;
  SelState cur[kSelections];
  unsigned int pre[kSelections];
#pragma unroll
  for (int s = 0; s < kSelections; ++s) {
    cur[s] = st[s];
    pre[s] = cur[s].prefix;
  }
  if (tot1) {
    const unsigned long long m0 = (unsigned long long)tot1[2], m1 = (unsigned long long)tot1[6];
#pragma unroll
    for (int s = 0; s < kSelections; ++s) {
      const int g = s / 2;
      const unsigned long long m = g == 0 ? m0 : (g == 1 ? m1 : m0 + m1);
      const unsigned long long num = (s & 1) ? 99 : 9, den = (s & 1) ? 100 : 10;
      cur[s].rank = (unsigned int)((num * m + den - 1) / den);
    }
  }
  const unsigned int counted = counted_selections(pre);
  unsigned int v[kSelections], incl[kSelections];
#pragma unroll
  for (int s = 0; s < kSelections; ++s) {
    if ((counted >> s) & 1u) {
      v[s] = hist[s * 256 + t];
      hist[s * 256 + t] = 0u;
    } else if ((s & 1) && pre[s] == pre[s - 1]) {
      v[s] = v[s - 1];
    } else {
      v[s] = v[s - 4] + v[s - 2];
    }
    unsigned int x = v[s];
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const unsigned int up = __shfl_up(x, off, 64);
      if (lane >= off) x += up;
    }
    incl[s] = x;
    if (lane == 63) s_wave[s][w] = x;
  }
  __syncthreads();  // every thread has read st[] before one of them rewrites it
#pragma unroll
  for (int s = 0; s < kSelections; ++s) {
    unsigned int before = 0;
    for (int k = 0; k < w; ++k) before += s_wave[s][k];
    const unsigned int hi = before + incl[s], lo = hi - v[s];
    const unsigned int rank = cur[s].rank;
    if (rank > 0 && lo < rank && rank <= hi) {
      st[s].prefix = (cur[s].prefix << 8) | (unsigned int)t;
      st[s].rank = rank - lo;
    } else if (t == 0 && rank == 0) {
      st[s].rank = 0;
    }
  }
}

// Clears the selection state (empty prefixes, no ranks) and the histogram
// before the first radix pass.
__global__ __launch_bounds__(256) void k_select_init(SelState* __restrict__ st,
                                                     unsigned int* __restrict__ hist) {
  const int t = threadIdx.x;
  if (t < kSelections) st[t] = SelState{0u, 0u};
  for (int i = t; i < kSelections * 256; i += 256) hist[i] = 0u;
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
