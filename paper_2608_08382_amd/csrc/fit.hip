// fit.hip -- host side of the fitting entry points of the libllmv C ABI
// (llmv_fit, llmv_fit_metrics and their extended-model forms; include/llmv.h):
// argument checks, workspace layout and the launches of the kernels in
// fit.hpp.
#include <hip/hip_runtime.h>

#include <cmath>

#include "fit.hpp"
#include "host.hpp"
#include "llmv.h"

using namespace llmv;
using namespace llmv::host;

namespace {

constexpr int kFitMaxGrid = 1024;
constexpr int kMaxRounds = 1024;
constexpr int64_t kFitMaxBatches = (int64_t)1 << 31;

struct FitLayout {
  size_t partials, tot1, tot2, sel, hist, counts, rel_err, total;
};

FitLayout fit_layout(int64_t nB) {
  FitLayout L{};
  size_t o = 0;
  L.partials = o;  // per-workgroup sums: [grid][FitCols::kVals], or [grid][kMetricVals]
  o += align_up((size_t)kFitMaxGrid * kFitValsMax * sizeof(double));
  L.tot1 = o;
  o += align_up(kMetricVals * sizeof(double));
  L.tot2 = o;
  o += align_up(kMetricVals * sizeof(double));
  L.sel = o;
  o += align_up(kSelections * sizeof(SelState));
  L.hist = o;
  o += align_up(kSelections * 256 * sizeof(unsigned int));
  L.counts = o;  // set counts when the caller asks for none
  o += align_up(4 * sizeof(long long));
  L.rel_err = o;  // relative errors when the caller asks for none
  o += align_up((size_t)(nB > 0 ? nB : 0) * sizeof(float));
  L.total = o;
  return L;
}

// One workgroup per kFitWG batches, at most kFitMaxGrid and at least one
// (the kernels write their partial sums even with no batches).  Every
// workgroup of the grid starts inside the batch range.
int fit_grid(int64_t nB) {
  const int64_t g = (nB + kFitWG - 1) / kFitWG;
  return g < 1 ? 1 : (g > kFitMaxGrid ? kFitMaxGrid : (int)g);
}

// Radix passes take kSelUnroll errors per thread per iteration.
int select_grid(int64_t nB) {
  const int64_t per = (int64_t)kFitWG * kSelUnroll;
  const int64_t g = (nB + per - 1) / per;
  return g < 1 ? 1 : (g > kFitMaxGrid ? kFitMaxGrid : (int)g);
}

int check_batches(const int64_t* sums, const uint8_t* phase, int64_t nB, const double* y) {
  if (nB < 0 || nB > kFitMaxBatches)
    return fail(LLMV_EINVAL, "n_batches=%lld outside [0, 2^31]", (long long)nB);
  if (nB > 0 && (!sums || !phase || !y)) return fail(LLMV_EINVAL, "sums, phase or y is NULL");
  return LLMV_OK;
}

// Shape constants of an NC-column model: S0..S3, and S5, S6 for NC = 7.
template <int NC>
int model_shape(const llmv_shape* shape, double S[6]) {
  for (int k = 0; k < 6; ++k) S[k] = 0.0;
  return NC == 7 ? shape_constants_ext(shape, S) : shape_constants(shape, S);
}

template <int NC>
int fit_run(const int64_t* sums, const uint8_t* phase, int64_t n_batches, const llmv_shape* shape,
            const double* y, const double* theta0, int32_t rounds, double* theta, int64_t* counts,
            void* ws, size_t ws_bytes, void* stream) {
  int rc = check_batches(sums, phase, n_batches, y);
  if (rc) return rc;
  if (rounds < 0 || rounds > kMaxRounds)
    return fail(LLMV_EINVAL, "rounds=%d outside [0, %d]", rounds, kMaxRounds);
  if (!theta0) return fail(LLMV_EINVAL, "theta0 is NULL");
  if (!theta) return fail(LLMV_EINVAL, "theta is NULL");
  FitModel<NC> M{};
  rc = model_shape<NC>(shape, M.S);
  if (rc) return rc;
  for (int i = 0; i < 4 * NC; ++i) {
    if (!std::isfinite(theta0[i])) return fail(LLMV_EINVAL, "theta0[%d] is not finite", i);
    M.th[i] = theta0[i];
  }
  const FitLayout L = fit_layout(n_batches);
  rc = check_ws(ws, ws_bytes, L.total);
  if (rc) return rc;
  char* base = (char*)ws;
  double* partials = (double*)(base + L.partials);
  long long* cnt = counts ? (long long*)counts : (long long*)(base + L.counts);
  hipStream_t s = (hipStream_t)stream;

  hipLaunchKernelGGL(k_fit_init<NC>, dim3(1), dim3(64), 0, s, M, theta, cnt);
  HIP_TRY(hipGetLastError(), "k_fit_init launch");
  FitShape F{};
  for (int k = 0; k < 6; ++k) F.S[k] = M.S[k];
  const int grid = fit_grid(n_batches);
  for (int r = 0; r < rounds; ++r) {
    hipLaunchKernelGGL(k_fit_accum<NC>, dim3(grid), dim3(kFitWG), 0, s, sums, phase, n_batches, F,
                       y, (const double*)theta, partials);
    HIP_TRY(hipGetLastError(), "k_fit_accum launch");
    hipLaunchKernelGGL(k_fit_solve<NC>, dim3(1), dim3(kReduceWG), 0, s,
                       (const double*)partials, grid, theta, cnt);
    HIP_TRY(hipGetLastError(), "k_fit_solve launch");
  }
  return LLMV_OK;
}

template <int NC>
int metrics_run(const int64_t* sums, const uint8_t* phase, int64_t n_batches,
                const llmv_shape* shape, const float* coeffs, const double* y, float* rel_err,
                double* out, void* ws, size_t ws_bytes, void* stream) {
  int rc = check_batches(sums, phase, n_batches, y);
  if (rc) return rc;
  if (!coeffs) return fail(LLMV_EINVAL, "coeffs is NULL");
  if (!out) return fail(LLMV_EINVAL, "out is NULL");
  FitModel<NC> M{};
  rc = model_shape<NC>(shape, M.S);
  if (rc) return rc;
  for (int i = 0; i < 4 * NC; ++i) {
    if (!std::isfinite(coeffs[i])) return fail(LLMV_EINVAL, "coeffs[%d] is not finite", i);
    M.th[i] = (double)coeffs[i];
  }
  const FitLayout L = fit_layout(n_batches);
  rc = check_ws(ws, ws_bytes, L.total);
  if (rc) return rc;
  char* base = (char*)ws;
  double* partials = (double*)(base + L.partials);
  double* tot1 = (double*)(base + L.tot1);
  double* tot2 = (double*)(base + L.tot2);
  SelState* sel = (SelState*)(base + L.sel);
  unsigned int* hist = (unsigned int*)(base + L.hist);
  float* err = rel_err ? rel_err : (float*)(base + L.rel_err);
  hipStream_t s = (hipStream_t)stream;
  const int grid = fit_grid(n_batches);

  // pass 1 (with the first radix pass of the percentile selection), its sums
  // and the first pick; then pass 2 for r^2
  hipLaunchKernelGGL(k_select_init, dim3(1), dim3(256), 0, s, sel, hist);
  HIP_TRY(hipGetLastError(), "k_select_init launch");
  hipLaunchKernelGGL(k_fit_metrics1<NC>, dim3(grid), dim3(kFitWG), 0, s, sums, phase, n_batches,
                     M, y, err, partials, hist);
  HIP_TRY(hipGetLastError(), "k_fit_metrics1 launch");
  hipLaunchKernelGGL(k_fit_metrics_sum, dim3(1), dim3(kReduceWG), 0, s, (const double*)partials,
                     grid, tot1);
  HIP_TRY(hipGetLastError(), "k_fit_metrics_sum launch");
  hipLaunchKernelGGL(k_select_pick, dim3(1), dim3(256), 0, s, sel, hist, (const double*)tot1);
  HIP_TRY(hipGetLastError(), "k_select_pick launch");
  hipLaunchKernelGGL(k_fit_metrics2<NC>, dim3(grid), dim3(kFitWG), 0, s, sums, phase, n_batches,
                     M, y, (const double*)tot1, partials);
  HIP_TRY(hipGetLastError(), "k_fit_metrics2 launch");
  hipLaunchKernelGGL(k_fit_metrics_sum, dim3(1), dim3(kReduceWG), 0, s, (const double*)partials,
                     grid, tot2);
  HIP_TRY(hipGetLastError(), "k_fit_metrics_sum launch");
  // the remaining radix passes of 8 bits over the fp32 errors
  const int sel_grid = select_grid(n_batches);
  for (int pass = 1; pass < 4; ++pass) {
    hipLaunchKernelGGL(k_select_hist, dim3(sel_grid), dim3(kFitWG), 0, s, (const float*)err, phase,
                       n_batches, pass, (const SelState*)sel, hist);
    HIP_TRY(hipGetLastError(), "k_select_hist launch");
    hipLaunchKernelGGL(k_select_pick, dim3(1), dim3(256), 0, s, sel, hist, (const double*)nullptr);
    HIP_TRY(hipGetLastError(), "k_select_pick launch");
  }
  hipLaunchKernelGGL(k_fit_metrics_final, dim3(1), dim3(64), 0, s, (const double*)tot1,
                     (const double*)tot2, (const SelState*)sel, out);
  HIP_TRY(hipGetLastError(), "k_fit_metrics_final launch");
  return LLMV_OK;
}

}  // namespace

extern "C" {

size_t llmv_fit_workspace_size(int64_t n_batches) { return fit_layout(n_batches).total; }

int llmv_fit(const int64_t* sums, const uint8_t* phase, int64_t n_batches,
             const llmv_shape* shape, const double* y, const double theta0[20], int32_t rounds,
             double* theta, int64_t* counts, void* ws, size_t ws_bytes, void* stream) {
  return fit_run<5>(sums, phase, n_batches, shape, y, theta0, rounds, theta, counts, ws, ws_bytes,
                    stream);
}

int llmv_fit_ext(const int64_t* sums, const uint8_t* phase, int64_t n_batches,
                 const llmv_shape* shape, const double* y, const double theta0[28],
                 int32_t rounds, double* theta, int64_t* counts, void* ws, size_t ws_bytes,
                 void* stream) {
  return fit_run<7>(sums, phase, n_batches, shape, y, theta0, rounds, theta, counts, ws, ws_bytes,
                    stream);
}

int llmv_fit_metrics(const int64_t* sums, const uint8_t* phase, int64_t n_batches,
                     const llmv_shape* shape, const float coeffs[20], const double* y,
                     float* rel_err, double* out, void* ws, size_t ws_bytes, void* stream) {
  return metrics_run<5>(sums, phase, n_batches, shape, coeffs, y, rel_err, out, ws, ws_bytes,
                        stream);
}

int llmv_fit_metrics_ext(const int64_t* sums, const uint8_t* phase, int64_t n_batches,
                         const llmv_shape* shape, const float coeffs[28], const double* y,
                         float* rel_err, double* out, void* ws, size_t ws_bytes, void* stream) {
  return metrics_run<7>(sums, phase, n_batches, shape, coeffs, y, rel_err, out, ws, ws_bytes,
                        stream);
}

}  // extern "C"
