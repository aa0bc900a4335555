// api.hip -- host side of the libllmv C ABI (include/llmv.h): argument
// checks, shape constants, workspace layout and kernel launches.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>

#include "host.hpp"
#include "groups.hpp"
#include "kernels.hpp"
#include "llmv.h"
#include "model.hpp"
#include "step.hpp"

namespace llmv {
// Scratch of llmv_attribute_noalloc, one copy per device (see llmv.h).
__device__ __align__(256) unsigned char scratch[LLMV_NOALLOC_SCRATCH_BYTES];
}  // namespace llmv

using namespace llmv;
using namespace llmv::host;

namespace {

thread_local hipEvent_t g_ev_before = nullptr;  // measurement hook
thread_local hipEvent_t g_ev_after = nullptr;

// Static scratch of llmv_attribute_noalloc: the device address of `scratch`
// on each device, looked up once per device (hipGetSymbolAddress with that
// device current).  Host code uses these addresses, never the array's name.
std::mutex g_scratch_mu;
void* g_scratch_dev[64] = {};

int scratch_address(void** out) {
  int dev = 0;
  HIP_TRY(hipGetDevice(&dev), "hipGetDevice");
  if (dev < 0 || dev >= 64) return fail(LLMV_EDEVICE, "device index %d out of range", dev);
  std::lock_guard<std::mutex> g(g_scratch_mu);
  if (!g_scratch_dev[dev]) {
    void* p = nullptr;
    HIP_TRY(hipGetSymbolAddress(&p, HIP_SYMBOL(llmv::scratch)), "hipGetSymbolAddress(scratch)");
    if (!p) return fail(LLMV_EDEVICE, "hipGetSymbolAddress(scratch) returned NULL");
    g_scratch_dev[dev] = p;
  }
  *out = g_scratch_dev[dev];
  return LLMV_OK;
}

// Upper bound of the persistent grid for n requests (sizes the workspace):
// no more than one workgroup per kWaves (narrow) wave tiles of requests, at
// most kMaxGrid.
int64_t grid_max_for(int64_t n) {
  const int64_t per = (int64_t)kCapNarrow * kWaves;
  const int64_t by_work = (n + per - 1) / per;
  return by_work < 1 ? 1 : (by_work > kMaxGrid ? kMaxGrid : by_work);
}

// Resident workgroups per compute unit for a kernel and its dynamic LDS.
template <typename K>
int blocks_per_cu(K kernel, size_t dyn, int block = kWG) {
  int nb = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, kernel, block, dyn) != hipSuccess || nb < 1)
    nb = 1;
  return nb;
}

// Persistent grid: exactly the workgroups that are resident at once (one
// wave of workgroups, no tail), capped by grid_max_for.
int64_t grid_for(int64_t n, int cus, int per_cu) {
  const int64_t g = (int64_t)cus * per_cu;
  const int64_t m = grid_max_for(n);
  return g < m ? g : m;
}

bool lds_hist(int32_t T) { return T > 0 && T <= kHistLdsMax; }

// Traces up to this many requests run as one workgroup in one launch (wave
// tiles of `cap` slots): two wave tiles per wave at most, so a longer serial
// walk never costs more than the launches it saves.
constexpr int64_t small_n(int64_t cap) { return 2 * cap * kWaves; }

// Replicas of the attribution path's LDS tenant histogram: 4, 2 or 1, within
// 32 KiB (two workgroups per CU keep fitting).
int hist_replicas(int32_t T) {
  for (int r = 4; r > 1; r /= 2)
    if ((size_t)r * (size_t)T * sizeof(double) <= 32 * 1024) return r;
  return 1;
}

// Settings per what-if pass for T tenants (T <= kHistLdsMax): 8, 4 or 2
// fp64 histograms of T + hot-tenant replicas, at most 65 KiB of LDS, so that
// with the kernel's own LDS two workgroups fit in a CU's 160 KiB.
constexpr size_t kSweepHistLds = 65 * 1024;
int sweep_group(int32_t T) {
  for (int g = kSweepG; g > 1; g /= 2)
    if ((size_t)g * (size_t)(T + kHotSlots) * sizeof(double) <= kSweepHistLds) return g;
  return 1;
}
static_assert(2 * (kHistLdsMax + kHotSlots) * sizeof(double) <= kSweepHistLds, "sweep LDS");

template <int NC>
using SweepKernel = void (*)(const GroupSweep, const VarTableOf<NC>);
template <int NC>
SweepKernel<NC> pick_sweep(int g) {
  if (g >= 8) return k_sweep_groups<8, NC>;
  if (g >= 4) return k_sweep_groups<4, NC>;
  return k_sweep_groups<2, NC>;
}

struct Layout {
  size_t wg_first, claims, partials, counts, hot, flag, big_list, big_seg, long_list, total;
};

// Chunks for `workers` wave workers over n requests, for wave tiles of `cap`
// slots.  When a worker's share is at least min_dyn_share(cap) requests:
// eighths/8 of the requests in static chunks, the rest in up to
// dyn_per_worker (at most kDynPerWorker) claimed chunks per worker of at
// least min_chunk(cap) requests.  The static part is one chunk per worker,
// or with `pieces` chunks of piece(cap) requests dealt round-robin (neighbouring
// waves then stream neighbouring memory).  Otherwise one static chunk per
// worker and no claims (a claim is a device-wide atomic on one counter;
// thousands of them cost more than a short launch can win back).
ChunkMap chunk_map(int64_t n, int64_t workers, bool pieces, int64_t cap,
                   int eighths = kStaticEighths, int dyn_per_worker = kDynPerWorker) {
  const int64_t kPiece = piece(cap), kMinChunk = min_chunk(cap);
  ChunkMap m{};
  m.n_static = workers;
  m.s2 = 1;
  if (n / workers < min_dyn_share(cap)) {
    m.s1 = (n + workers - 1) / workers;
    if (m.s1 < 1) m.s1 = 1;
    m.F = m.s1 * workers;
    m.n_chunks = workers;
    return m;
  }
  const int64_t n_static = n / 8 * eighths / kPiece;
  if (pieces && n_static >= workers) {
    m.n_static = n_static;
    m.s1 = kPiece;
  } else {
    m.s1 = n / 8 * eighths / workers;
  }
  m.F = m.s1 * m.n_static;
  const int64_t rest = n - m.F;
  int64_t dyn = (int64_t)min(dyn_per_worker, kDynPerWorker) * workers;
  if (dyn > rest / kMinChunk) dyn = rest / kMinChunk;
  if (dyn < 1) dyn = 1;
  m.s2 = (rest + dyn - 1) / dyn;
  if (m.s2 < 1) m.s2 = 1;
  m.n_chunks = m.n_static + dyn;
  return m;
}

// Workspace layout shared by every entry point for n requests; rows =
// histograms per workgroup (settings per pass in the what-if sweep, else 1).
Layout layout(int64_t n, int32_t T, int rows = 1) {
  Layout L{};
  size_t o = 0;
  const int64_t grid = grid_max_for(n);
  L.wg_first = o;  // first batch of each chunk (chunk_map's n_chunks + 1 at most)
  o += align_up((size_t)(n / piece(kCapNarrow) + grid * kWaves * (1 + kDynPerWorker) + 1) *
                sizeof(int64_t));
  L.claims = o;  // the launch's counters
  o += align_up(kCounters * sizeof(unsigned long long));
  L.partials = o;  // [grid][rows][T]
  if (lds_hist(T)) o += align_up((size_t)grid * (size_t)rows * (size_t)T * sizeof(double));
  L.counts = o;  // what-if sweep: requests per tenant, and the hot tenants
  if (lds_hist(T)) o += align_up((size_t)T * sizeof(unsigned long long));
  L.hot = o;
  o += align_up(kHot * sizeof(int32_t));
  L.flag = o;
  o += align_up(sizeof(int));
  // batches of more than kListMin requests, listed with their segments
  const size_t n_list = (size_t)(n / (kListMin + 1)) + 1;
  L.big_list = o;
  o += align_up(n_list * sizeof(BigEntry));
  L.big_seg = o;  // each listed batch of k requests: at most k / kBigSeg + 2 segments
  o += align_up(((size_t)(n / kBigSeg) + 2 * n_list) * sizeof(uint64_t));
  L.long_list = o;  // batches larger than a wave tile (each more than kCapNarrow - 3 requests)
  o += align_up((size_t)(n / (kCapNarrow - 3) + 1) * sizeof(int64_t));
  L.total = o;
  return L;
}

// The what-if sweep's groups after a Layout ending at o: slice table, slice
// group counts and offsets, batch group offsets, exact batch sums, scan tile
// sums, and the groups (at most one per request, plus a tile of slack that
// the sweep tiles read past the last group); under the extended model a
// fourth batch sum and the groups' sums of p*c.
struct GroupLayout {
  size_t first, scnt, soff, gofs, bsum, tsum, gw, gf, gr, part2, total;
};
// part2: a second set of pass partials ([grid][rows][T], as the Layout's),
// which a pass writes while the next pass folds the other.
GroupLayout group_layout(size_t o, int64_t nB, int64_t N, bool ext, int32_t T = 0, int rows = 1) {
  GroupLayout G{};
  const int64_t nS = (N + kSlice - 1) / kSlice;
  const int64_t nt = (nS + kScanTile - 1) / kScanTile;
  G.first = o;
  o += align_up((size_t)(nS + 1) * sizeof(int64_t));
  G.scnt = o;
  o += align_up((size_t)(nS + 1) * sizeof(int64_t));
  G.soff = o;
  o += align_up((size_t)(nS + 1) * sizeof(int64_t));
  G.gofs = o;
  o += align_up((size_t)(nB + 1) * sizeof(int64_t));
  G.bsum = o;
  o += align_up((size_t)((ext ? 5 : 4) * nB + 1) * sizeof(unsigned long long));
  G.tsum = o;
  o += align_up((size_t)(nt + 1) * sizeof(int64_t));
  G.gw = o;
  o += align_up((size_t)(N + kGT) * sizeof(uint32_t));
  G.gf = o;
  o += align_up((size_t)(N + kGT) * sizeof(v4f));
  G.gr = o;
  if (ext) o += align_up((size_t)(N + kGT) * sizeof(float));
  G.part2 = o;
  if (lds_hist(T)) o += align_up((size_t)grid_max_for(N) * (size_t)rows * (size_t)T * sizeof(double));
  G.total = o;
  return G;
}

int check_trace(const llmv_trace* tr, bool need_tenant) {
  if (!tr) return fail(LLMV_EINVAL, "trace is NULL");
  if (tr->n_batches < 0 || tr->n_requests < 0)
    return fail(LLMV_EINVAL, "negative sizes (n_batches=%lld, n_requests=%lld)",
                (long long)tr->n_batches, (long long)tr->n_requests);
  if (!tr->offsets) return fail(LLMV_EINVAL, "trace offsets is NULL");
  if (tr->n_requests > 0 && (!tr->p || !tr->c)) return fail(LLMV_EINVAL, "trace p or c is NULL");
  if (need_tenant && tr->n_requests > 0 && !tr->tenant)
    return fail(LLMV_EINVAL, "tenant sums requested but trace tenant is NULL");
  auto aligned = [](const void* ptr) { return ((uintptr_t)ptr & 15u) == 0; };
  if (!aligned(tr->p) || !aligned(tr->c) || (tr->tenant && !aligned(tr->tenant)))
    return fail(LLMV_EINVAL, "p, c and tenant must be 16-byte aligned");
  return LLMV_OK;
}

// Chunk table and cleared claim counter for one or more k_tiles launches.
int partition(const llmv_trace* tr, const ChunkMap& cm, int64_t* wg_first,
              unsigned long long* claims, hipStream_t stream) {
  int64_t blocks = (tr->n_batches + 1 + kWG - 1) / kWG;
  if (blocks > 4096) blocks = 4096;
  hipLaunchKernelGGL(k_partition, dim3((unsigned)blocks), dim3(kWG), 0, stream, tr->offsets,
                     tr->n_batches, cm, wg_first, claims);
  HIP_TRY(hipGetLastError(), "k_partition launch");
  return LLMV_OK;
}

typedef void (*TileKernel)(const Params, const NoVars);

TileKernel pick_tiles(int mode, int hist, bool share) {
  if (mode == MODE_FEAT) return k_tiles<MODE_FEAT, HIST_NONE, false>;
  if (mode == MODE_SUMS) return k_tiles<MODE_SUMS, HIST_NONE, false>;
  if (hist == HIST_NONE)
    return share ? k_tiles<MODE_ATTR, HIST_NONE, true> : k_tiles<MODE_ATTR, HIST_NONE, false>;
  if (hist == HIST_LDS)
    return share ? k_tiles<MODE_ATTR, HIST_LDS, true> : k_tiles<MODE_ATTR, HIST_LDS, false>;
  return share ? k_tiles<MODE_ATTR, HIST_GLOBAL, true> : k_tiles<MODE_ATTR, HIST_GLOBAL, false>;
}

// The tile kernel for a mode and its second argument's type.
template <typename VT> struct TilePick;
template <> struct TilePick<NoVars> {
  static TileKernel get(int mode, int hist, bool share) { return pick_tiles(mode, hist, share); }
};
template <> struct TilePick<ExtModel> {
  typedef void (*K)(const Params, const ExtModel);
  static K get(int, int hist, bool share) {
    if (hist == HIST_NONE)
      return share ? k_tiles<MODE_EXT, HIST_NONE, true> : k_tiles<MODE_EXT, HIST_NONE, false>;
    if (hist == HIST_LDS)
      return share ? k_tiles<MODE_EXT, HIST_LDS, true> : k_tiles<MODE_EXT, HIST_LDS, false>;
    return share ? k_tiles<MODE_EXT, HIST_GLOBAL, true> : k_tiles<MODE_EXT, HIST_GLOBAL, false>;
  }
};

// The long-batch kernel matching a tile kernel.
template <typename VT> struct LongPick;
template <> struct LongPick<NoVars> {
  typedef void (*K)(const Params, const NoVars, int64_t);
  static K get(int mode, int hist, bool share) {
    if (mode == MODE_FEAT) return k_long<MODE_FEAT, HIST_NONE, false>;
    if (mode == MODE_SUMS) return k_long<MODE_SUMS, HIST_NONE, false>;
    if (hist == HIST_NONE)
      return share ? k_long<MODE_ATTR, HIST_NONE, true> : k_long<MODE_ATTR, HIST_NONE, false>;
    if (hist == HIST_LDS)
      return share ? k_long<MODE_ATTR, HIST_LDS, true> : k_long<MODE_ATTR, HIST_LDS, false>;
    return share ? k_long<MODE_ATTR, HIST_GLOBAL, true> : k_long<MODE_ATTR, HIST_GLOBAL, false>;
  }
};
template <> struct LongPick<ExtModel> {
  typedef void (*K)(const Params, const ExtModel, int64_t);
  static K get(int, int hist, bool share) {
    if (hist == HIST_NONE)
      return share ? k_long<MODE_EXT, HIST_NONE, true> : k_long<MODE_EXT, HIST_NONE, false>;
    if (hist == HIST_LDS)
      return share ? k_long<MODE_EXT, HIST_LDS, true> : k_long<MODE_EXT, HIST_LDS, false>;
    return share ? k_long<MODE_EXT, HIST_GLOBAL, true> : k_long<MODE_EXT, HIST_GLOBAL, false>;
  }
};

// One scheduler step (at most kStepN requests, kStepB batches and, with
// tenant sums, kStepT tenants) runs in k_step: one workgroup, one launch.
bool step_fits(const llmv_trace* tr, bool want_tenant, int32_t T) {
  return tr->n_requests <= kStepN && tr->n_batches <= kStepB && (!want_tenant || T <= kStepT);
}

int run_step(const Params& P, bool want_tenant, hipStream_t stream) {
  const size_t dyn = want_tenant ? (size_t)P.n_tenants * sizeof(double) : 0;
  if (g_ev_before) HIP_TRY(hipEventRecord(g_ev_before, stream), "hipEventRecord");
  if (want_tenant)
    hipLaunchKernelGGL(k_step<true>, dim3(1), dim3(kStepWG), dyn, stream, P);
  else
    hipLaunchKernelGGL(k_step<false>, dim3(1), dim3(kStepWG), 0, stream, P);
  HIP_TRY(hipGetLastError(), "k_step launch");
  if (g_ev_after) HIP_TRY(hipEventRecord(g_ev_after, stream), "hipEventRecord");
  return LLMV_OK;
}

// Partition + tiles (+ tenant reduction) shared by attribute and features.
// V: the kernel's second argument (the extended model, or nothing).
template <typename VT>
int run_tiles(int mode, const llmv_trace* tr, Params& P, const VT& V, int32_t T,
              bool want_tenant, bool want_share, void* ws, size_t ws_bytes, hipStream_t stream) {
  int cus = 0;
  int rc = device_cus(&cus);
  if (rc) return rc;
  const int32_t Tl = want_tenant ? T : 0;
  const Layout L = layout(tr->n_requests, Tl);
  rc = check_ws(ws, ws_bytes, L.total);
  if (rc) return rc;
  const int hist = !want_tenant ? HIST_NONE : (lds_hist(T) ? HIST_LDS : HIST_GLOBAL);
  const int rep = hist == HIST_LDS ? hist_replicas(T) : 1;
  const size_t dyn = hist == HIST_LDS ? (size_t)rep * (size_t)T * sizeof(double)
                     : (hist == HIST_GLOBAL ? kCacheLds : 0);
  const auto kern = TilePick<VT>::get(mode, hist, want_share);
  const auto klong = LongPick<VT>::get(mode, hist, want_share);
  P.hist_rep = rep;
  char* base = (char*)ws;
  // batches larger than a wave tile, listed for k_long
  P.long_list = (int64_t*)(base + L.long_list);
  P.long_count = (unsigned long long*)(base + L.claims) + kLongCounter;
  P.big_list = nullptr;
  P.big_seg = nullptr;

  const int64_t cap = tile_cap(mode, hist);
  // a batch larger than a tile needs more than cap - 4 requests
  const bool longs = tr->n_requests > cap - 4;
  if (tr->n_requests <= small_n(cap) && hist != HIST_GLOBAL) {
    // A small trace (one scheduler step, say) in one launch: one workgroup,
    // its waves split the batches by count (no chunk table), and the
    // workgroup's tenant histogram is the result (no reduction); k_long
    // follows with one workgroup if a batch can be larger than a tile.
    P.split_by_count = 1;
    P.n_chunks = kWaves;
    P.n_static = kWaves;
    P.wg_first = nullptr;
    P.claims = nullptr;
    P.partials = hist == HIST_LDS ? P.tenant_sums : nullptr;
    if (g_ev_before) HIP_TRY(hipEventRecord(g_ev_before, stream), "hipEventRecord");
    hipLaunchKernelGGL(kern, dim3(1), dim3(kWG), dyn, stream, P, V);
    HIP_TRY(hipGetLastError(), "k_tiles launch");
    if (g_ev_after) HIP_TRY(hipEventRecord(g_ev_after, stream), "hipEventRecord");
    if (longs) {
      hipLaunchKernelGGL(klong, dim3(1), dim3(kWG), dyn, stream, P, V, (int64_t)1);
      HIP_TRY(hipGetLastError(), "k_long launch");
    }
    return LLMV_OK;
  }

  const int64_t grid = grid_for(tr->n_requests, cus, blocks_per_cu(kern, dyn));
  int64_t* wg_first = (int64_t*)(base + L.wg_first);
  const int n_chunks = want_tenant ? (T + kTenantChunk - 1) / kTenantChunk : 0;

  // When the mean batch is larger than a tile, most requests lie in batches
  // that the tile kernel only lists for k_long: a chunk then takes a few
  // microseconds, and chunk setups and claims (device-scope atomics) cost
  // more than the balance they buy.  One static chunk per wave over all but
  // the remainder, at most 2 claimed chunks per wave.
  const bool long_mean = tr->n_requests > tr->n_batches * (int64_t)cap;
  const ChunkMap cm = long_mean ? chunk_map(tr->n_requests, grid * kWaves, false, cap, 8, 2)
                                : chunk_map(tr->n_requests, grid * kWaves, true, cap);
  P.wg_first = wg_first;
  P.split_by_count = 0;
  P.claims = (unsigned long long*)(base + L.claims);
  P.claim_base = 0;
  P.n_chunks = cm.n_chunks;
  P.n_static = cm.n_static;
  P.partials = hist == HIST_LDS ? (double*)(base + L.partials) : nullptr;
  // Eq. 1 attribution: batches of more than kListMin requests are listed
  // for the segment kernels
  const bool listed = mode == MODE_ATTR && tr->n_requests > kListMin;
  P.big_list = listed ? (BigEntry*)(base + L.big_list) : nullptr;
  P.big_seg = listed ? (uint64_t*)(base + L.big_seg) : nullptr;

  rc = partition(tr, cm, wg_first, P.claims, stream);
  if (rc) return rc;
  if (hist == HIST_GLOBAL) {
    // the atomics path accumulates into the output: clear it first
    hipLaunchKernelGGL(k_zero_f64, dim3(16), dim3(kWG), 0, stream, P.tenant_sums, (int64_t)T);
    HIP_TRY(hipGetLastError(), "k_zero_f64 launch");
  }

  if (g_ev_before) HIP_TRY(hipEventRecord(g_ev_before, stream), "hipEventRecord");
  hipLaunchKernelGGL(kern, dim3((unsigned)grid), dim3(kWG), dyn, stream, P, V);
  HIP_TRY(hipGetLastError(), "k_tiles launch");
  if (g_ev_after) HIP_TRY(hipEventRecord(g_ev_after, stream), "hipEventRecord");

  if (listed) {
    // exact sums of the listed batches' segments
    hipLaunchKernelGGL(k_big_sums, dim3(kBigGrid), dim3(kBigWG), 0, stream, P);
    HIP_TRY(hipGetLastError(), "k_big_sums launch");
  }
  if (longs) {
    // the long batches, then the listed batches' per-request outputs
    const int64_t lgrid = grid_for(tr->n_requests, cus, blocks_per_cu(klong, dyn));
    hipLaunchKernelGGL(klong, dim3((unsigned)lgrid), dim3(kWG), dyn, stream, P, V, grid);
    HIP_TRY(hipGetLastError(), "k_long launch");
  }

  if (hist == HIST_LDS) {
    hipLaunchKernelGGL(k_tenant_reduce, dim3((unsigned)n_chunks), dim3(64 * kReduceWaves), 0, stream,
                       (const double*)P.partials, (int)grid, (int)T, P.tenant_sums);
    HIP_TRY(hipGetLastError(), "k_tenant_reduce launch");
  }
  return LLMV_OK;
}

// Checks and kernel parameters shared by llmv_attribute (20 coefficients)
// and llmv_attribute_ext (28).
int attribute_params(const llmv_trace* trace, const llmv_shape* shape, const float* coeffs,
                     int n_coeffs, float* latency, uint8_t* regime, float* share,
                     int32_t n_tenants, double* tenant_sums, Params& P) {
  const bool want_tenant = tenant_sums != nullptr;
  int rc = check_trace(trace, want_tenant);
  if (rc) return rc;
  if (!coeffs) return fail(LLMV_EINVAL, "coeffs is NULL");
  for (int i = 0; i < n_coeffs; ++i)
    if (!std::isfinite(coeffs[i])) return fail(LLMV_EINVAL, "coeffs[%d] is not finite", i);
  if (want_tenant && (n_tenants <= 0 || n_tenants > LLMV_TENANTS_MAX))
    return fail(LLMV_EINVAL, "n_tenants=%d outside [1, 2^24]", n_tenants);
  if (share && ((uintptr_t)share & 15u)) return fail(LLMV_EINVAL, "share must be 16-byte aligned");
  rc = shape_constants(shape, P.S);
  if (rc) return rc;
  P.off = trace->offsets;
  P.p = trace->p;
  P.c = trace->c;
  P.tenant = want_tenant ? trace->tenant : nullptr;
  P.nB = trace->n_batches;
  P.N = trace->n_requests;
  P.latency = latency;
  P.regime = regime;
  P.share = share;
  P.tenant_sums = tenant_sums;
  P.n_tenants = want_tenant ? n_tenants : 0;
  return LLMV_OK;
}

// The admission queries of Eq. 1 (NC = 5) or of the extended model (NC = 7).
template <int NC>
int admit_run(const int64_t* sums, const uint8_t* phase, int64_t n_batches,
              const llmv_shape* shape, const float* coeffs, const int64_t* cand_batch,
              const int32_t* cand_p, const int32_t* cand_c, int64_t n_cand, float* t_after,
              float* delta, float* share, uint8_t* regime, void* stream) {
  if (n_batches < 0 || n_cand < 0)
    return fail(LLMV_EINVAL, "negative sizes (n_batches=%lld, n_cand=%lld)",
                (long long)n_batches, (long long)n_cand);
  if (!coeffs) return fail(LLMV_EINVAL, "coeffs is NULL");
  for (int i = 0; i < 4 * NC; ++i)
    if (!std::isfinite(coeffs[i])) return fail(LLMV_EINVAL, "coeffs[%d] is not finite", i);
  AdmitParams<NC> A{};
  int rc = NC == 7 ? shape_constants_ext(shape, A.S) : shape_constants(shape, A.S);
  if (rc) return rc;
  for (int i = 0; i < 4 * NC; ++i) A.th[i] = (double)coeffs[i];
  if (n_cand == 0) return LLMV_OK;
  if (!cand_batch || !cand_p || !cand_c)
    return fail(LLMV_EINVAL, "candidate arrays must not be NULL");
  if (n_batches > 0 && (!sums || !phase)) return fail(LLMV_EINVAL, "sums or phase is NULL");
  const int64_t blocks = (n_cand + kWG - 1) / kWG;
  if (blocks > 0x7fffffff) return fail(LLMV_EINVAL, "n_cand=%lld too large", (long long)n_cand);
  hipLaunchKernelGGL(k_admit<NC>, dim3((unsigned)blocks), dim3(kWG), 0, (hipStream_t)stream, sums,
                     phase, n_batches, A, cand_batch, cand_p, cand_c, n_cand, t_after, delta,
                     share, regime);
  HIP_TRY(hipGetLastError(), "k_admit launch");
  return LLMV_OK;
}

// The what-if sweep under Eq. 1 (NC = 5) or the extended model (NC = 7).
template <int NC>
int sweep_run(const llmv_trace* trace, const llmv_shape* shapes, int32_t n_shapes,
              const float* coeffs, int32_t n_coeffs, int32_t n_tenants, double* out, void* ws,
              size_t ws_bytes, hipStream_t st) {
  constexpr bool EXT = NC == 7;
  int rc = check_trace(trace, true);
  if (rc) return rc;
  if (n_shapes < 1 || (!shapes && n_shapes != 1))
    return fail(LLMV_EINVAL, "n_shapes=%d (NULL shapes needs n_shapes == 1)", n_shapes);
  if (n_coeffs < 1 || !coeffs) return fail(LLMV_EINVAL, "n_coeffs=%d or coeffs NULL", n_coeffs);
  if (!lds_hist(n_tenants))
    return fail(LLMV_EINVAL, "n_tenants=%d outside [1, %d] for the sweep", n_tenants, kHistLdsMax);
  if (!out) return fail(LLMV_EINVAL, "out is NULL");
  for (int64_t i = 0; i < (int64_t)n_coeffs * 4 * NC; ++i)
    if (!std::isfinite(coeffs[i])) return fail(LLMV_EINVAL, "coeffs[%lld] is not finite", (long long)i);
  double S[64][6];  // S0..S3 (and S5, S6)
  if (n_shapes > 64) return fail(LLMV_EINVAL, "n_shapes=%d > 64", n_shapes);
  for (int s = 0; s < n_shapes; ++s) {
    const llmv_shape* sh = shapes ? &shapes[s] : nullptr;
    rc = EXT ? shape_constants_ext(sh, S[s]) : shape_constants(sh, S[s]);
    if (rc) return rc;
  }
  int cus = 0;
  rc = device_cus(&cus);
  if (rc) return rc;
  const int64_t nB = trace->n_batches, N = trace->n_requests;
  // One pass over the groups per G consecutive settings (shape-major, as in
  // out); each pass keeps G tenant histograms in LDS.
  const int G = sweep_group(n_tenants);
  const Layout L = layout(N, n_tenants, G);
  const GroupLayout GL = group_layout(L.total, nB, N, EXT, n_tenants, G);
  rc = check_ws(ws, ws_bytes, GL.total);
  if (rc) return rc;
  char* base = (char*)ws;
  const int64_t n_var = (int64_t)n_shapes * n_coeffs;
  if (N == 0) {  // no requests: every tenant sum is zero
    const int64_t n_out = n_var * n_tenants;
    int64_t blocks = (n_out + kWG - 1) / kWG;
    if (blocks > 1024) blocks = 1024;
    hipLaunchKernelGGL(k_zero_f64, dim3((unsigned)blocks), dim3(kWG), 0, st, out, n_out);
    HIP_TRY(hipGetLastError(), "k_zero_f64 launch");
    return LLMV_OK;
  }
  const size_t dyn = (size_t)G * (size_t)(n_tenants + kHotSlots) * sizeof(double);
  const SweepKernel<NC> kern = pick_sweep<NC>(G);
  const int64_t grid = grid_for(N, cus, blocks_per_cu(kern, dyn, kSweepWG));
  unsigned long long* claims = (unsigned long long*)(base + L.claims);

  // the most frequent tenants get replicated histogram entries
  unsigned long long* counts = (unsigned long long*)(base + L.counts);
  int32_t* hot = (int32_t*)(base + L.hot);
  hipLaunchKernelGGL(k_zero_u64, dim3(16), dim3(kWG), 0, st, counts, (int64_t)n_tenants);
  HIP_TRY(hipGetLastError(), "k_zero_u64 launch");
  int64_t blocks = (N + (int64_t)kWG * 64 - 1) / ((int64_t)kWG * 64);
  blocks = blocks < 1 ? 1 : (blocks > 2048 ? 2048 : blocks);
  hipLaunchKernelGGL(k_tenant_count, dim3((unsigned)blocks), dim3(kWG),
                     (size_t)n_tenants * sizeof(unsigned int), st, trace->tenant, N, n_tenants,
                     counts);
  HIP_TRY(hipGetLastError(), "k_tenant_count launch");
  hipLaunchKernelGGL(k_hot_tenants, dim3(1), dim3(kWG), 0, st, (const unsigned long long*)counts,
                     n_tenants, hot);
  HIP_TRY(hipGetLastError(), "k_hot_tenants launch");

  // the groups: counts and exact batch sums per slice, slice offsets, then
  // the groups themselves
  const int64_t nS = (N + kSlice - 1) / kSlice;
  int64_t* first = (int64_t*)(base + GL.first);
  int64_t* scnt = (int64_t*)(base + GL.scnt);
  int64_t* soff = (int64_t*)(base + GL.soff);
  int64_t* gofs = (int64_t*)(base + GL.gofs);
  unsigned long long* bsum = (unsigned long long*)(base + GL.bsum);
  int64_t* tsum = (int64_t*)(base + GL.tsum);
  uint32_t* gw = (uint32_t*)(base + GL.gw);
  v4f* gf = (v4f*)(base + GL.gf);
  float* gr = EXT ? (float*)(base + GL.gr) : nullptr;
  ChunkMap sm{};  // equal slices, none claimed
  sm.s1 = kSlice;
  sm.s2 = 1;
  sm.n_static = nS;
  sm.n_chunks = nS;
  sm.F = nS * kSlice;
  rc = partition(trace, sm, first, claims, st);
  if (rc) return rc;
  hipLaunchKernelGGL(k_zero_u64, dim3(256), dim3(kWG), 0, st, bsum, (EXT ? 5 : 4) * nB);
  HIP_TRY(hipGetLastError(), "k_zero_u64 launch");
  int64_t bgrid = (nS + kWaves - 1) / kWaves;
  const int64_t bcap = (int64_t)cus * blocks_per_cu(k_group_build<true, EXT>, 0);
  if (bgrid > bcap) bgrid = bcap;
  hipLaunchKernelGGL((k_group_build<false, EXT>), dim3((unsigned)bgrid), dim3(kWG), 0, st,
                     trace->offsets, trace->p, trace->c, trace->tenant, nB, N, (const int64_t*)first,
                     nS, scnt, bsum, (const int64_t*)nullptr, (int64_t*)nullptr, (uint32_t*)nullptr,
                     (v4f*)nullptr, (float*)nullptr);
  HIP_TRY(hipGetLastError(), "k_group_build launch");
  const int64_t nt = (nS + kScanTile - 1) / kScanTile;  // >= 1
  hipLaunchKernelGGL(k_scan_tiles, dim3((unsigned)nt), dim3(kScanWG), 0, st, (const int64_t*)scnt, nS,
                     tsum);
  HIP_TRY(hipGetLastError(), "k_scan_tiles launch");
  hipLaunchKernelGGL(k_scan_top, dim3(1), dim3(kScanWG), 0, st, tsum, nt);
  HIP_TRY(hipGetLastError(), "k_scan_top launch");
  hipLaunchKernelGGL(k_scan_apply, dim3((unsigned)nt), dim3(kScanWG), 0, st, (const int64_t*)scnt, nS,
                     (const int64_t*)tsum, soff);
  HIP_TRY(hipGetLastError(), "k_scan_apply launch");
  hipLaunchKernelGGL((k_group_build<true, EXT>), dim3((unsigned)bgrid), dim3(kWG), 0, st,
                     trace->offsets, trace->p, trace->c, trace->tenant, nB, N, (const int64_t*)first,
                     nS, (int64_t*)nullptr, (unsigned long long*)nullptr, (const int64_t*)soff, gofs,
                     gw, gf, gr);
  HIP_TRY(hipGetLastError(), "k_group_build launch");

  // the passes: the chunks of k_tiles over the batches; every launch takes
  // exactly n_chunks claims (one per chunk it runs, the static ones
  // included), so launch i starts at claim i * n_chunks
  const ChunkMap cm = chunk_map(N, grid * kSweepWaves, false, kCapNarrow);  // one static chunk per wave
  int64_t* wg_first = (int64_t*)(base + L.wg_first);
  rc = partition(trace, cm, wg_first, claims, st);
  if (rc) return rc;
  GroupSweep Q{};
  Q.off = trace->offsets;
  Q.gofs = gofs;
  Q.bsum = bsum;
  Q.gw = gw;
  Q.gf = gf;
  Q.gr = gr;
  Q.nB = nB;
  Q.wg_first = wg_first;
  Q.claims = claims;
  Q.n_chunks = cm.n_chunks;
  Q.partials = (double*)(base + L.partials);
  Q.n_tenants = n_tenants;
  Q.hot = hot;
  // pass i writes partials bufs[i % 2] and folds pass i - 1's from the
  // other buffer (when its sums fit the fold's mapping); the last pass's, or
  // every pass's otherwise, go to k_tenant_reduce
  double* bufs[2] = {(double*)(base + L.partials), (double*)(base + GL.part2)};
  const bool fold = grid <= (int64_t)kFoldGroups * kFoldRows &&
                    (int64_t)G * n_tenants <= (int64_t)kFoldPer * grid;
  int64_t launch = 0;
  int64_t pv0 = 0;  // the previous pass's first setting
  int32_t pn = 0;   // and its settings
  for (int64_t v0 = 0; v0 < n_var; v0 += G, ++launch) {
    VarTableOf<NC> V{};
    V.n = (int32_t)(n_var - v0 < G ? n_var - v0 : G);
    for (int g = 0; g < V.n; ++g) {
      const int64_t v = v0 + g;
      const int s = (int)(v / n_coeffs);
      const int64_t j = v % n_coeffs;
      for (int k = 0; k < NC - 1; ++k) V.S[g][k] = S[s][k];
      for (int i = 0; i < 4 * NC; ++i) V.th[g][i] = (double)coeffs[j * 4 * NC + i];
      for (int r = 0; r < 4; ++r) {
        for (int k = 1; k < 4; ++k) V.K[g][r][k - 1] = (float)(V.th[g][r * NC + k] * S[s][k]);
        if (EXT) V.K[g][r][3] = (float)(V.th[g][r * NC + 5] * S[s][4]);
      }
    }
    Q.claim_base = (uint64_t)launch * (uint64_t)cm.n_chunks;
    Q.partials = fold ? bufs[launch & 1] : bufs[0];
    Q.prev = fold && launch > 0 ? bufs[(launch - 1) & 1] : nullptr;
    Q.prev_out = out + pv0 * n_tenants;
    Q.prev_n = pn;
    hipLaunchKernelGGL(kern, dim3((unsigned)grid), dim3(kSweepWG), dyn, st, Q, V);
    HIP_TRY(hipGetLastError(), "k_sweep_groups launch");
    const bool last = v0 + G >= n_var;
    if (!fold || last) {
      const int n_hist = V.n * n_tenants;
      hipLaunchKernelGGL(k_tenant_reduce,
                         dim3((unsigned)((n_hist + kTenantChunk - 1) / kTenantChunk)),
                         dim3(64 * kReduceWaves), 0, st, (const double*)Q.partials, (int)grid,
                         n_hist, out + v0 * n_tenants);
      HIP_TRY(hipGetLastError(), "k_tenant_reduce launch");
    }
    pv0 = v0;
    pn = V.n;
  }
  return LLMV_OK;
}

// The batches of llmv_attribute_host (data checked, tenant sums cleared):
// exact sums, Eq. 1 (model.hpp), shares and tenant sums in request order.
#define LLMV_HOST_BATCHES(NAME, ATTR)                                                          \
  ATTR void NAME(const int64_t* off, const int32_t* p, const int32_t* c, const int32_t* t,     \
                 int64_t nB, const double* th, const double* S, float* latency,                \
                 uint8_t* regime, float* share, double* tenant_sums) {                         \
    for (int64_t b = 0; b < nB; ++b) {                                                         \
      const int64_t lo = off[b], hi = off[b + 1], n = hi - lo;                                 \
      if (n == 0) {                                                                            \
        if (latency) latency[b] = 0.0f;                                                        \
        if (regime) regime[b] = 255;                                                           \
        continue;                                                                              \
      }                                                                                        \
      uint64_t Ps = 0, Cs = 0, Qs = 0;                                                         \
      bool zero_context = false;                                                               \
      for (int64_t i = lo; i < hi; ++i) {                                                      \
        const uint64_t pi = (uint32_t)p[i], ci = (uint32_t)c[i];                               \
        Ps += pi;                                                                              \
        Cs += ci;                                                                              \
        Qs += pi * pi;                                                                         \
        zero_context |= ci == 0;                                                               \
      }                                                                                        \
      /* decode iff every request processes one token over a nonzero context */                \
      const bool prefill = zero_context || Ps != (uint64_t)n;                                  \
      double tB, k[4];                                                                         \
      const int reg = eq1_batch(th, S, n, Ps, Cs, Qs, prefill, &tB, k);                        \
      if (latency) latency[b] = (float)tB;                                                     \
      if (regime) regime[b] = (uint8_t)reg;                                                    \
      if (!share && !tenant_sums) continue;                                                    \
      const float K[4] = {(float)k[0], (float)k[1], (float)k[2], (float)k[3]};                 \
      for (int64_t i = lo; i < hi; ++i) {                                                      \
        const float sh = share_of(K, p[i], c[i]);                                              \
        if (share) share[i] = sh;                                                              \
        if (tenant_sums) tenant_sums[t[i]] += (double)sh;                                      \
      }                                                                                        \
    }                                                                                          \
  }
LLMV_HOST_BATCHES(host_batches, )
LLMV_HOST_BATCHES(host_batches_fma, __attribute__((target("fma"))))
#undef LLMV_HOST_BATCHES

}  // namespace

extern "C" {

const char* llmv_last_error(void) { return g_err; }

int llmv_set_kernel_events(void* before, void* after) {
  if ((before == nullptr) != (after == nullptr))
    return fail(LLMV_EINVAL, "set both events or neither");
  g_ev_before = (hipEvent_t)before;
  g_ev_after = (hipEvent_t)after;
  return LLMV_OK;
}

int llmv_shape_constants(const llmv_shape* shape, double S[4]) {
  if (!S) return fail(LLMV_EINVAL, "S is NULL");
  return shape_constants(shape, S);
}

size_t llmv_workspace_size(int64_t n_batches, int64_t n_requests, int32_t n_tenants) {
  (void)n_batches;
  const int64_t n = n_requests > 0 ? n_requests : 0;
  return layout(n, n_tenants > 0 ? n_tenants : 0).total;
}

static size_t sweep_ws(int64_t n_batches, int64_t n_requests, int32_t n_tenants, bool ext) {
  const int64_t nB = n_batches > 0 ? n_batches : 0;
  const int64_t n = n_requests > 0 ? n_requests : 0;
  const int32_t T = n_tenants > 0 ? n_tenants : 0;
  const int rows = lds_hist(T) ? sweep_group(T) : 1;
  const Layout L = layout(n, T, rows);
  return group_layout(L.total, nB, n, ext, T, rows).total;
}

size_t llmv_sweep_workspace_size(int64_t n_batches, int64_t n_requests, int32_t n_tenants) {
  return sweep_ws(n_batches, n_requests, n_tenants, false);
}

size_t llmv_sweep_workspace_size_ext(int64_t n_batches, int64_t n_requests, int32_t n_tenants) {
  return sweep_ws(n_batches, n_requests, n_tenants, true);
}

int llmv_attribute(const llmv_trace* trace, const llmv_shape* shape, const float coeffs[20],
                   float* latency, uint8_t* regime, float* share, int32_t n_tenants,
                   double* tenant_sums, void* ws, size_t ws_bytes, void* stream) {
  Params P{};
  int rc = attribute_params(trace, shape, coeffs, 20, latency, regime, share, n_tenants,
                            tenant_sums, P);
  if (rc) return rc;
  for (int i = 0; i < 20; ++i) P.th[i] = (double)coeffs[i];
  if (!latency && !regime && !share && !tenant_sums) return LLMV_OK;  // nothing requested
  if (step_fits(trace, tenant_sums != nullptr, n_tenants))
    return run_step(P, tenant_sums != nullptr, (hipStream_t)stream);
  return run_tiles(MODE_ATTR, trace, P, NoVars{}, n_tenants, tenant_sums != nullptr,
                   share != nullptr, ws, ws_bytes, (hipStream_t)stream);
}

int llmv_attribute_noalloc(const llmv_trace* trace, const llmv_shape* shape,
                           const float coeffs[20], float* latency, uint8_t* regime, float* share,
                           int32_t n_tenants, double* tenant_sums, void* stream) {
  Params P{};
  int rc = attribute_params(trace, shape, coeffs, 20, latency, regime, share, n_tenants,
                            tenant_sums, P);
  if (rc) return rc;
  for (int i = 0; i < 20; ++i) P.th[i] = (double)coeffs[i];
  if (!latency && !regime && !share && !tenant_sums) return LLMV_OK;  // nothing requested
  if (step_fits(trace, tenant_sums != nullptr, n_tenants))  // no scratch needed
    return run_step(P, tenant_sums != nullptr, (hipStream_t)stream);
  const size_t need = layout(trace->n_requests, tenant_sums ? n_tenants : 0).total;
  if (need > LLMV_NOALLOC_SCRATCH_BYTES)
    return fail(LLMV_EINVAL,
                "llmv_attribute_noalloc: this trace needs %zu bytes of scratch "
                "(n_requests=%lld, n_tenants=%d); the static scratch holds %zu",
                need, (long long)trace->n_requests, (int)n_tenants,
                (size_t)LLMV_NOALLOC_SCRATCH_BYTES);
  void* ws = nullptr;
  rc = scratch_address(&ws);
  if (rc) return rc;
  return run_tiles(MODE_ATTR, trace, P, NoVars{}, n_tenants, tenant_sums != nullptr,
                   share != nullptr, ws, LLMV_NOALLOC_SCRATCH_BYTES, (hipStream_t)stream);
}

int llmv_shape_constants_ext(const llmv_shape* shape, double S[6]) {
  if (!S) return fail(LLMV_EINVAL, "S is NULL");
  return shape_constants_ext(shape, S);
}

int llmv_attribute_ext(const llmv_trace* trace, const llmv_shape* shape, const float coeffs[28],
                       float* latency, uint8_t* regime, float* share, int32_t n_tenants,
                       double* tenant_sums, void* ws, size_t ws_bytes, void* stream) {
  Params P{};
  int rc = attribute_params(trace, shape, coeffs, 28, latency, regime, share, n_tenants,
                            tenant_sums, P);
  if (rc) return rc;
  double S[6];
  rc = shape_constants_ext(shape, S);
  if (rc) return rc;
  ExtModel E{};
  E.S5 = S[4];
  E.S6 = S[5];
  for (int i = 0; i < 28; ++i) E.th[i] = (double)coeffs[i];
  if (!latency && !regime && !share && !tenant_sums) return LLMV_OK;  // nothing requested
  return run_tiles(MODE_EXT, trace, P, E, n_tenants, tenant_sums != nullptr, share != nullptr,
                   ws, ws_bytes, (hipStream_t)stream);
}

int llmv_attribute_sweep(const llmv_trace* trace, const llmv_shape* shapes, int32_t n_shapes,
                         const float* coeffs, int32_t n_coeffs, int32_t n_tenants, double* out,
                         void* ws, size_t ws_bytes, void* stream) {
  return sweep_run<5>(trace, shapes, n_shapes, coeffs, n_coeffs, n_tenants, out, ws, ws_bytes,
                      (hipStream_t)stream);
}

int llmv_attribute_sweep_ext(const llmv_trace* trace, const llmv_shape* shapes, int32_t n_shapes,
                             const float* coeffs, int32_t n_coeffs, int32_t n_tenants, double* out,
                             void* ws, size_t ws_bytes, void* stream) {
  return sweep_run<7>(trace, shapes, n_shapes, coeffs, n_coeffs, n_tenants, out, ws, ws_bytes,
                      (hipStream_t)stream);
}

int llmv_batch_sums(const llmv_trace* trace, int64_t* sums, uint8_t* phase, void* ws,
                    size_t ws_bytes, void* stream) {
  int rc = check_trace(trace, false);
  if (rc) return rc;
  Params P{};
  rc = shape_constants(nullptr, P.S);
  if (rc) return rc;
  P.off = trace->offsets;
  P.p = trace->p;
  P.c = trace->c;
  P.nB = trace->n_batches;
  P.N = trace->n_requests;
  P.bsums = sums;
  P.bphase = phase;
  if (!sums && !phase) return LLMV_OK;
  return run_tiles(MODE_FEAT, trace, P, NoVars{}, 0, false, false, ws, ws_bytes,
                   (hipStream_t)stream);
}

int llmv_batch_sums_ext(const llmv_trace* trace, int64_t* sums, uint8_t* phase, void* ws,
                        size_t ws_bytes, void* stream) {
  int rc = check_trace(trace, false);
  if (rc) return rc;
  Params P{};
  rc = shape_constants(nullptr, P.S);
  if (rc) return rc;
  P.off = trace->offsets;
  P.p = trace->p;
  P.c = trace->c;
  P.nB = trace->n_batches;
  P.N = trace->n_requests;
  P.bsums = sums;
  P.bphase = phase;
  if (!sums && !phase) return LLMV_OK;
  return run_tiles(MODE_SUMS, trace, P, NoVars{}, 0, false, false, ws, ws_bytes,
                   (hipStream_t)stream);
}

int llmv_admit(const int64_t* sums, const uint8_t* phase, int64_t n_batches,
               const llmv_shape* shape, const float coeffs[20], const int64_t* cand_batch,
               const int32_t* cand_p, const int32_t* cand_c, int64_t n_cand, float* t_after,
               float* delta, float* share, uint8_t* regime, void* stream) {
  return admit_run<5>(sums, phase, n_batches, shape, coeffs, cand_batch, cand_p, cand_c, n_cand,
                      t_after, delta, share, regime, stream);
}

int llmv_admit_ext(const int64_t* sums, const uint8_t* phase, int64_t n_batches,
                   const llmv_shape* shape, const float coeffs[28], const int64_t* cand_batch,
                   const int32_t* cand_p, const int32_t* cand_c, int64_t n_cand, float* t_after,
                   float* delta, float* share, uint8_t* regime, void* stream) {
  return admit_run<7>(sums, phase, n_batches, shape, coeffs, cand_batch, cand_p, cand_c, n_cand,
                      t_after, delta, share, regime, stream);
}

int llmv_features(const llmv_trace* trace, const llmv_shape* shape, float* x_req,
                  double* x_batch, void* ws, size_t ws_bytes, void* stream) {
  int rc = check_trace(trace, false);
  if (rc) return rc;
  Params P{};
  rc = shape_constants(shape, P.S);
  if (rc) return rc;
  P.off = trace->offsets;
  P.p = trace->p;
  P.c = trace->c;
  P.nB = trace->n_batches;
  P.N = trace->n_requests;
  P.x_req = x_req;
  P.x_batch = x_batch;
  if (!x_req && !x_batch) return LLMV_OK;
  return run_tiles(MODE_FEAT, trace, P, NoVars{}, 0, false, false, ws, ws_bytes,
                   (hipStream_t)stream);
}

int llmv_tenant_sums(const int32_t* tenant, const float* share, int64_t n, int32_t n_tenants,
                     double* tenant_sums, void* ws, size_t ws_bytes, void* stream) {
  if (n < 0) return fail(LLMV_EINVAL, "n=%lld is negative", (long long)n);
  if (n_tenants <= 0 || n_tenants > LLMV_TENANTS_MAX)
    return fail(LLMV_EINVAL, "n_tenants=%d outside [1, 2^24]", n_tenants);
  if (!tenant_sums) return fail(LLMV_EINVAL, "tenant_sums is NULL");
  if (n > 0 && (!tenant || !share)) return fail(LLMV_EINVAL, "tenant or share is NULL");
  hipStream_t s = (hipStream_t)stream;
  int cus = 0;
  int rc = device_cus(&cus);
  if (rc) return rc;
  const Layout L = layout(n, n_tenants);
  rc = check_ws(ws, ws_bytes, L.total);
  if (rc) return rc;
  char* base = (char*)ws;
  const int n_chunks = (n_tenants + kTenantChunk - 1) / kTenantChunk;
  const bool lds = lds_hist(n_tenants);
  const int64_t grid =
      lds ? grid_for(n, cus, blocks_per_cu(k_tenant_hist<HIST_LDS>, (size_t)n_tenants * sizeof(double)))
          : grid_for(n, cus, blocks_per_cu(k_tenant_hist<HIST_GLOBAL>, kCacheLds));
  if (!lds) {
    // the atomics path accumulates into the output: clear it first
    hipLaunchKernelGGL(k_zero_f64, dim3(16), dim3(kWG), 0, s, tenant_sums, (int64_t)n_tenants);
    HIP_TRY(hipGetLastError(), "k_zero_f64 launch");
  }
  if (lds) {
    double* partials = (double*)(base + L.partials);
    hipLaunchKernelGGL(k_tenant_hist<HIST_LDS>, dim3((unsigned)grid), dim3(kWG),
                       (size_t)n_tenants * sizeof(double), s, tenant, share, n, n_tenants,
                       partials, tenant_sums);
    HIP_TRY(hipGetLastError(), "k_tenant_hist launch");
    hipLaunchKernelGGL(k_tenant_reduce, dim3((unsigned)n_chunks), dim3(64 * kReduceWaves), 0, s,
                       (const double*)partials, (int)grid, (int)n_tenants, tenant_sums);
    HIP_TRY(hipGetLastError(), "k_tenant_reduce launch");
  } else {
    hipLaunchKernelGGL(k_tenant_hist<HIST_GLOBAL>, dim3((unsigned)grid), dim3(kWG), kCacheLds, s, tenant,
                       share, n, n_tenants, (double*)nullptr, tenant_sums);
    HIP_TRY(hipGetLastError(), "k_tenant_hist launch");
  }
  return LLMV_OK;
}

int llmv_attribute_host(const llmv_trace* trace, const llmv_shape* shape, const float coeffs[20],
                        float* latency, uint8_t* regime, float* share, int32_t n_tenants,
                        double* tenant_sums) {
  const bool want_tenant = tenant_sums != nullptr;
  if (!trace) return fail(LLMV_EINVAL, "trace is NULL");
  const int64_t nB = trace->n_batches, N = trace->n_requests;
  if (nB < 0 || N < 0)
    return fail(LLMV_EINVAL, "negative sizes (n_batches=%lld, n_requests=%lld)", (long long)nB,
                (long long)N);
  if (!trace->offsets) return fail(LLMV_EINVAL, "trace offsets is NULL");
  if (N > 0 && (!trace->p || !trace->c)) return fail(LLMV_EINVAL, "trace p or c is NULL");
  if (want_tenant && (n_tenants <= 0 || n_tenants > LLMV_TENANTS_MAX))
    return fail(LLMV_EINVAL, "n_tenants=%d outside [1, 2^24]", n_tenants);
  if (want_tenant && N > 0 && !trace->tenant)
    return fail(LLMV_EINVAL, "tenant sums requested but trace tenant is NULL");
  if (!coeffs) return fail(LLMV_EINVAL, "coeffs is NULL");
  double th[20], S[4];
  for (int i = 0; i < 20; ++i) {
    if (!std::isfinite(coeffs[i])) return fail(LLMV_EINVAL, "coeffs[%d] is not finite", i);
    th[i] = (double)coeffs[i];
  }
  int rc = shape_constants(shape, S);
  if (rc) return rc;
  // host data: checked before any output is written (a tenant id out of
  // range would write out of bounds)
  const int64_t* off = trace->offsets;
  const int32_t *p = trace->p, *c = trace->c, *t = trace->tenant;
  if (off[0] != 0 || off[nB] != N) return fail(LLMV_ERANGE, "offsets[0] != 0 or offsets[nB] != N");
  for (int64_t b = 0; b < nB; ++b)
    if (off[b + 1] < off[b] || off[b + 1] - off[b] > LLMV_BATCH_MAX)
      return fail(LLMV_ERANGE, "batch %lld: size outside [0, 2^22]", (long long)b);
  for (int64_t i = 0; i < N; ++i) {
    if (p[i] < 1 || p[i] > LLMV_P_MAX || c[i] < 0)
      return fail(LLMV_ERANGE, "request %lld: p or c outside the limits", (long long)i);
    if (want_tenant && (t[i] < 0 || t[i] >= n_tenants))
      return fail(LLMV_ERANGE, "request %lld: tenant outside [0, n_tenants)", (long long)i);
  }
  if (want_tenant)
    for (int32_t u = 0; u < n_tenants; ++u) tenant_sums[u] = 0.0;
  // the shares' fused multiply-adds in hardware where the CPU has them (the
  // library function otherwise; both round once)
  if (__builtin_cpu_supports("fma"))
    host_batches_fma(off, p, c, t, nB, th, S, latency, regime, share, tenant_sums);
  else
    host_batches(off, p, c, t, nB, th, S, latency, regime, share, tenant_sums);
  return LLMV_OK;
}

int llmv_validate(const llmv_trace* trace, int32_t n_tenants, void* ws, size_t ws_bytes,
                  void* stream) {
  int rc = check_trace(trace, false);
  if (rc) return rc;
  if (trace->tenant && (n_tenants <= 0 || n_tenants > LLMV_TENANTS_MAX))
    return fail(LLMV_EINVAL, "n_tenants=%d outside [1, 2^24]", n_tenants);
  hipStream_t s = (hipStream_t)stream;
  const Layout L = layout(trace->n_requests, 0);
  rc = check_ws(ws, ws_bytes, L.flag + sizeof(int));
  if (rc) return rc;
  int* flag = (int*)((char*)ws + L.flag);
  hipLaunchKernelGGL(k_zero_i32, dim3(1), dim3(64), 0, s, flag, 1);
  HIP_TRY(hipGetLastError(), "k_zero_i32 launch");
  const int64_t work = trace->n_requests > trace->n_batches ? trace->n_requests : trace->n_batches;
  int64_t blocks = (work + kWG - 1) / kWG;
  if (blocks > 8192) blocks = 8192;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(k_validate, dim3((unsigned)blocks), dim3(kWG), 0, s, trace->offsets,
                     trace->n_batches, trace->n_requests, trace->p, trace->c, trace->tenant,
                     n_tenants, (int)LLMV_BATCH_MAX, (int)LLMV_P_MAX, flag);
  HIP_TRY(hipGetLastError(), "k_validate launch");
  int h = 0;
  HIP_TRY(hipMemcpyAsync(&h, flag, sizeof(int), hipMemcpyDeviceToHost, s), "hipMemcpyAsync");
  HIP_TRY(hipStreamSynchronize(s), "hipStreamSynchronize");
  if (h) return fail(LLMV_ERANGE, "trace data outside the limits");
  return LLMV_OK;
}

}  // extern "C"
