// groups.hpp -- gfx950 kernels of the what-if sweep: the tenant sums of one
// trace under many (shape, coefficient) settings (Sec. 1, what-if planning;
// Eq. 1 and Sec. 2 "Problem formulation" for each setting).
//
// Within a batch every request's share is k0 + k1*p + k2*c + k3*p^2 with the
// batch's constants (Eq. 1 under the chosen segment, beta split equally, the
// a4 term per request), so the shares of one tenant's requests in one batch
// sum to k0*n + k1*P + k2*C + k3*Q over that group's count n and sums P, C,
// Q.  The sweep forms these (batch, tenant) groups once per call and then,
// per setting, adds one term per group instead of one per request.  Under
// the extended model (NC = 7: the a5 term on p*c, the a6 term per request)
// a share gains k5*p*c and k0 gains a6*S6, so a group also carries R = its
// sum of p*c and adds k5*R.
//
//  * k_group_build<false>: per slice of kSlice requests, the number of
//    groups, and the exact batch sums; k_scan_*: the slices' group offsets;
//    k_group_build<true>: the groups and each batch's first group.  One wave
//    per slice; a wave-private LDS hash table keyed by tenant collects the
//    group sums and is emitted when it fills or the batch part ends (a tenant
//    emitted twice in one batch only costs an extra group: sums are linear).
//  * k_sweep_groups<NV, NC>: one pass of NV settings over the groups.  Wave
//    tiles are runs of whole batches (at most kGB batches, kGT group slots);
//    lane j evaluates batch j of the tile under every setting into a per-wave
//    LDS table of (k0, k1, k2, k3) (and k5); lane-local runs of kGV groups then add
//    their group sums into per-setting fp64 LDS tenant histograms, flushed to
//    [grid][NV][n_tenants] partials that k_tenant_reduce folds.
#pragma once

#include "kernels.hpp"

namespace llmv {

// ------------------------------------------------------------ settings

// The settings of one pass: shape constants and coefficients
// (theta[phase][segment][k], NC terms per set, as in Params or ExtModel) of
// each, and the batch-independent share constants k1..k3 = fp32(theta_a1*S1,
// theta_a2*S2, theta_a3*S3) and k5 = fp32(theta_a5*S5) of each regime
// (2*phase + segment), rounded from the same fp64 products as in MODE_ATTR
// and MODE_EXT.
constexpr int kSweepG = 8;
template <int NC>
struct VarTableOf {
  static_assert(NC == 5 || NC == 7, "Eq. 1 or the extended model");
  int32_t n;                    // settings in this pass, 1..kSweepG
  double S[kSweepG][NC - 1];    // S0..S3 (and S5, S6)
  double th[kSweepG][4 * NC];
  float K[kSweepG][4][4];       // [setting][regime][k1, k2, k3, k5 (NC = 7)]
};
using VarTable = VarTableOf<5>;
// Under tenant skew many lanes of one LDS atomic hit the same histogram
// entry and serialize.  Each of the kHot most frequent tenants gets kHotRep
// histogram entries per setting (lane l adds into entry l % kHotRep), folded
// at the end.
constexpr int kHot = 4;
constexpr int kHotRep = 4;
constexpr int kHotSlots = kHot * kHotRep;

// One batch under every setting: k0 of setting g (fp32, rounded from fp64
// as in MODE_ATTR / MODE_EXT) into k0[g]; returns the segments (bit g).
// Rsum (sum p*c) is read only under the extended model.
template <int NV, int NC>
__device__ __forceinline__ uint32_t sweep_batch(const VarTableOf<NC>& V, int64_t n, uint64_t Psum,
                                                uint64_t Csum, uint64_t Qsum, uint64_t Rsum,
                                                bool prefill, float* k0) {
  (void)Rsum;
  const int phase = prefill ? 0 : 1;
  uint32_t segs = 0;
  for (int g = 0; g < NV; ++g) {
    const double* S = V.S[g];
    const double* thm = V.th[g] + (phase * 2 + 0) * NC;
    const double* thc = V.th[g] + (phase * 2 + 1) * NC;
    bool comp;
    if constexpr (NC == 5) {
      const double X[5] = {S[0], S[1] * (double)Psum, S[2] * (double)Csum, S[3] * (double)Qsum,
                           (double)n * (double)n};
      // Roofline max of the two segments; ties stay memory-bound.
      comp = eq1(thc, X) > eq1(thm, X);
    } else {
      const double X[7] = {S[0], S[1] * (double)Psum, S[2] * (double)Csum, S[3] * (double)Qsum,
                           (double)n * (double)n, S[4] * (double)Rsum, S[5] * (double)n};
      comp = eq7(thc, X) > eq7(thm, X);
    }
    const double* th = comp ? thc : thm;
    segs |= (uint32_t)comp << g;
    if constexpr (NC == 5)
      k0[g] = (float)(th[0] * (S[0] / (double)n) + th[4] * (double)n);
    else
      k0[g] = (float)(th[0] * (S[0] / (double)n) + th[4] * (double)n + th[6] * S[5]);
  }
  return segs;
}

// ------------------------------------------------------ hot tenants

// counts[u] += number of requests of tenant u (counts cleared beforehand);
// a per-workgroup LDS histogram, then one global atomic per tenant.
__global__ __launch_bounds__(kWG) void k_tenant_count(const int32_t* __restrict__ tenant,
                                                      int64_t n, int32_t T,
                                                      unsigned long long* __restrict__ counts) {
  extern __shared__ unsigned int s_cnt[];
  for (int u = threadIdx.x; u < T; u += kWG) s_cnt[u] = 0u;
  __syncthreads();
  const int64_t stride = (int64_t)gridDim.x * kWG;
  for (int64_t i = (int64_t)blockIdx.x * kWG + threadIdx.x; i < n; i += stride)
    atomicAdd(&s_cnt[tenant[i]], 1u);
  __syncthreads();
  for (int u = threadIdx.x; u < T; u += kWG)
    if (s_cnt[u]) atomicAdd(&counts[u], (unsigned long long)s_cnt[u]);
}

// hot[0..kHot) = the most frequent tenants in decreasing count (ties: the
// smaller id first); -1 where fewer tenants have requests.  One workgroup.
__global__ __launch_bounds__(kWG) void k_hot_tenants(const unsigned long long* __restrict__ counts,
                                                     int32_t T, int32_t* __restrict__ hot) {
  __shared__ unsigned long long s_best[kWG / 64];
  __shared__ int32_t s_hot[kHot];
  const int tid = threadIdx.x, lane = tid & 63;
  for (int h = 0; h < kHot; ++h) {
    // key: count (saturated to 32 bits) above the complement of the id
    unsigned long long best = 0;
    for (int u = tid; u < T; u += kWG) {
      bool taken = false;
      for (int j = 0; j < h; ++j) taken |= (s_hot[j] == u);
      const unsigned long long c = counts[u] < 0xffffffffull ? counts[u] : 0xffffffffull;
      const unsigned long long key = (c << 32) | (unsigned long long)(0xffffffffu - (uint32_t)u);
      if (!taken && c > 0 && key > best) best = key;
    }
    for (int m = 32; m >= 1; m >>= 1) {
      const unsigned long long o = __shfl_xor(best, m, 64);
      best = o > best ? o : best;
    }
    if (lane == 0) s_best[tid >> 6] = best;
    __syncthreads();
    if (tid == 0) {
      unsigned long long b = 0;
      for (int w = 0; w < kWG / 64; ++w) b = s_best[w] > b ? s_best[w] : b;
      s_hot[h] = b ? (int32_t)(0xffffffffu - (uint32_t)(b & 0xffffffffull)) : -1;
    }
    __syncthreads();
  }
  if (tid < kHot) hot[tid] = s_hot[tid];
}

// ------------------------------------------------------------ group build

constexpr int kGrpSlots = 256;             // hash slots per wave
constexpr int kGrpFlush = kGrpSlots / 2;   // emit once more slots than this are taken
constexpr uint32_t kGrpEmpty = 0xffffffffu;
constexpr int kGrpTenantBits = 12;         // tenant ids of a sweep are below 4096
constexpr uint32_t kGrpTenantMask = (1u << kGrpTenantBits) - 1u;
constexpr uint32_t kGrpBatchMask = (1u << (32 - kGrpTenantBits)) - 1u;
constexpr int64_t kSlice = 2048;           // requests per build slice
static_assert(kHistLdsMax <= (1 << kGrpTenantBits), "sweep tenant ids fit the group word");
static_assert(kGrpFlush + 64 < kGrpSlots, "a round always finds a free slot");

template <bool EXT>
struct GroupTable {  // one wave's
  uint32_t key[kGrpSlots];
  uint32_t n[kGrpSlots];
  unsigned long long p[kGrpSlots], c[kGrpSlots], q[kGrpSlots];
  unsigned long long r[EXT ? kGrpSlots : 1];  // sum p*c (EXT)
};

__device__ __forceinline__ uint32_t grp_hash(uint32_t t) {
  static_assert(kGrpSlots == 256, "8-bit hash");
  return (t * 2654435761u) >> 24;  // Fibonacci hashing
}

// The requests are cut into slices of kSlice; wave w builds slices w, w + W,
// ...  A slice emits the groups of every batch part inside it in request
// order, so all groups are in request order and a batch's groups are
// contiguous even when slices split it.  first[k] = the first batch starting
// at or after request k*kSlice (k_partition over equal chunks).
// WRITE = false: slice_cnt[k] = groups of slice k; bsum[j*nB + b] (zeroed
// beforehand) += (sum p, sum c, sum p^2, count of c == 0, and with EXT
// sum p*c) of the part of batch b in the slice.  WRITE = true: the groups
// from slice_off[k] on, gw = ((b mod 2^20) << 12) | tenant, gf = (n, P, C, Q)
// and with EXT gr = R (sum p*c), rounded to fp32, and gofs[b] for every
// batch starting in the slice (gofs[nB] by the last).  Both passes emit the
// same groups: the emission points depend only on the data.
template <bool WRITE, bool EXT>
__global__ __launch_bounds__(kWG) void k_group_build(
    const int64_t* __restrict__ off, const int32_t* __restrict__ p, const int32_t* __restrict__ c,
    const int32_t* __restrict__ tenant, int64_t nB, int64_t N, const int64_t* __restrict__ first,
    int64_t nS, int64_t* __restrict__ slice_cnt, unsigned long long* __restrict__ bsum,
    const int64_t* __restrict__ slice_off, int64_t* __restrict__ gofs, uint32_t* __restrict__ gw,
    v4f* __restrict__ gf, float* __restrict__ gr) {
  __shared__ GroupTable<EXT> s_tab[kWaves];
  const int lane = threadIdx.x & 63;
  GroupTable<EXT>& H = s_tab[threadIdx.x >> 6];
  for (int s = lane; s < kGrpSlots; s += 64) {
    H.key[s] = kGrpEmpty;
    H.n[s] = 0;
    H.p[s] = 0;
    H.c[s] = 0;
    H.q[s] = 0;
    if (EXT) H.r[s] = 0;
  }
  wave_lds_sync();
  const int64_t waves = (int64_t)gridDim.x * kWaves;
  for (int64_t k = (int64_t)blockIdx.x * kWaves + (threadIdx.x >> 6); k < nS; k += waves) {
    const int64_t r0 = k * kSlice, r1 = min(N, r0 + kSlice);
    const bool last = k == nS - 1;
    int64_t b = uni(first[k]);
    if (b > 0 && (b == nB || uni(off[b]) > r0)) --b;  // the batch holding request r0
    int64_t out = WRITE ? uni(slice_off[k]) : 0;      // index of the next group
    for (; b < nB; ++b) {
      const int64_t bo0 = uni(off[b]), bo1 = uni(off[b + 1]);
      if (bo0 >= r1 && !last) break;  // the last slice also takes the empty batches at N
      if (WRITE && bo0 >= r0 && lane == 0) gofs[b] = out;
      const int64_t lo = max(bo0, r0), hi = min(bo1, r1);
      int32_t taken = 0;
      uint64_t sp = 0, sc = 0, sq = 0, sz = 0, sr = 0;
      for (int64_t base = lo; base < hi; base += 64) {
        const int64_t i = base + lane;
        bool fresh = false;
        if (i < hi) {
          const uint32_t pi = (uint32_t)p[i], ci = (uint32_t)c[i], ti = (uint32_t)tenant[i];
          const uint64_t pp = (uint64_t)pi * pi;
          const uint64_t pc = (uint64_t)pi * ci;
          if (!WRITE) {
            sp += pi;
            sc += ci;
            sz += ci == 0 ? 1u : 0u;
            sq += pp;
            if (EXT) sr += pc;
          }
          uint32_t h = grp_hash(ti);
          while (true) {  // ends: fewer than kGrpSlots keys are ever held
            const uint32_t old = atomicCAS(&H.key[h], kGrpEmpty, ti);
            if (old == kGrpEmpty) {
              fresh = true;
              break;
            }
            if (old == ti) break;
            h = (h + 1) & (kGrpSlots - 1);
          }
          if (WRITE) {
            atomicAdd(&H.n[h], 1u);
            atomicAdd(&H.p[h], (unsigned long long)pi);
            atomicAdd(&H.c[h], (unsigned long long)ci);
            atomicAdd(&H.q[h], (unsigned long long)pp);
            if (EXT) atomicAdd(&H.r[h], (unsigned long long)pc);
          }
        }
        taken += __builtin_popcountll(__ballot(fresh));
        wave_lds_sync();
        if (taken > kGrpFlush || base + 64 >= hi) {
          // emit the held groups in slot order, clearing their slots
#pragma unroll
          for (int j = 0; j < kGrpSlots / 64; ++j) {
            const int s = j * 64 + lane;
            const uint32_t key = H.key[s];
            const bool used = key != kGrpEmpty;
            const uint64_t m = __ballot(used);
            if (used) {
              if (WRITE) {
                const int64_t at = out + __builtin_popcountll(m & ((1ull << lane) - 1ull));
                gw[at] = (((uint32_t)b & kGrpBatchMask) << kGrpTenantBits) | key;
                gf[at] = (v4f){(float)H.n[s], (float)H.p[s], (float)H.c[s], (float)H.q[s]};
                if (EXT) {
                  gr[at] = (float)H.r[s];
                  H.r[s] = 0;
                }
                H.n[s] = 0;
                H.p[s] = 0;
                H.c[s] = 0;
                H.q[s] = 0;
              }
              H.key[s] = kGrpEmpty;
            }
            out += __builtin_popcountll(m);
          }
          taken = 0;
          wave_lds_sync();
        }
      }
      if (!WRITE) {
        sp = wave_sum(sp);
        sc = wave_sum(sc);
        sq = wave_sum(sq);
        sz = wave_sum(sz);
        if (EXT) sr = wave_sum(sr);
        if (lane == 0) {
          if (bo0 >= r0 && bo1 <= r1) {  // the whole batch
            bsum[b] = sp;
            bsum[nB + b] = sc;
            bsum[2 * nB + b] = sq;
            bsum[3 * nB + b] = sz;
            if (EXT) bsum[4 * nB + b] = sr;
          } else {
            atomicAdd(&bsum[b], (unsigned long long)sp);
            atomicAdd(&bsum[nB + b], (unsigned long long)sc);
            atomicAdd(&bsum[2 * nB + b], (unsigned long long)sq);
            atomicAdd(&bsum[3 * nB + b], (unsigned long long)sz);
            if (EXT) atomicAdd(&bsum[4 * nB + b], (unsigned long long)sr);
          }
        }
      }
    }
    if (!WRITE && lane == 0) slice_cnt[k] = out;
    if (WRITE && last && lane == 0) gofs[nB] = out;
  }
}

// ------------------------------------------------------------ offsets scan

constexpr int kScanWG = 1024;
constexpr int kScanPer = 8;
constexpr int64_t kScanTile = (int64_t)kScanWG * kScanPer;

// Exclusive scan of one value per thread over the workgroup; *total gets
// the sum.  Every thread of the workgroup calls it.
__device__ __forceinline__ int64_t block_excl_scan(int64_t v, int64_t* total) {
  __shared__ int64_t s_w[kScanWG / 64];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  int64_t x = v;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const int64_t y = __shfl_up(x, d, 64);
    if (lane >= d) x += y;
  }
  if (lane == 63) s_w[w] = x;
  __syncthreads();
  int64_t before = 0, tot = 0;
  for (int k = 0; k < kScanWG / 64; ++k) {
    const int64_t t = s_w[k];
    before += k < w ? t : 0;
    tot += t;
  }
  __syncthreads();
  *total = tot;
  return before + x - v;
}

// tile_sum[t] = sum of x over tile t (kScanTile elements).
__global__ __launch_bounds__(kScanWG) void k_scan_tiles(const int64_t* __restrict__ x, int64_t n,
                                                         int64_t* __restrict__ tile_sum) {
  const int64_t i0 = (int64_t)blockIdx.x * kScanTile + (int64_t)threadIdx.x * kScanPer;
  int64_t s = 0;
  for (int k = 0; k < kScanPer; ++k) s += i0 + k < n ? x[i0 + k] : 0;
  int64_t tot = 0;
  block_excl_scan(s, &tot);
  if (threadIdx.x == 0) tile_sum[blockIdx.x] = tot;
}

// One workgroup: exclusive scan of the nt tile sums, in place.
__global__ __launch_bounds__(kScanWG) void k_scan_top(int64_t* __restrict__ t, int64_t nt) {
  int64_t carry = 0;
  for (int64_t base = 0; base < nt; base += kScanTile) {
    const int64_t i0 = base + (int64_t)threadIdx.x * kScanPer;
    int64_t v[kScanPer], s = 0;
    for (int k = 0; k < kScanPer; ++k) {
      v[k] = i0 + k < nt ? t[i0 + k] : 0;
      s += v[k];
    }
    int64_t tot = 0;
    int64_t e = block_excl_scan(s, &tot) + carry;
    for (int k = 0; k < kScanPer; ++k) {
      if (i0 + k < nt) t[i0 + k] = e;
      e += v[k];
    }
    carry += tot;
  }
}

// y[i] = sum of x[0..i) for i <= n (y has n + 1 entries); tile_off from
// k_scan_tiles and k_scan_top.
__global__ __launch_bounds__(kScanWG) void k_scan_apply(const int64_t* __restrict__ x, int64_t n,
                                                         const int64_t* __restrict__ tile_off,
                                                         int64_t* __restrict__ y) {
  const int64_t i0 = (int64_t)blockIdx.x * kScanTile + (int64_t)threadIdx.x * kScanPer;
  int64_t v[kScanPer], s = 0;
  for (int k = 0; k < kScanPer; ++k) {
    v[k] = i0 + k < n ? x[i0 + k] : 0;
    s += v[k];
  }
  int64_t tot = 0;
  int64_t e = block_excl_scan(s, &tot) + tile_off[blockIdx.x];
  for (int k = 0; k < kScanPer; ++k) {
    if (i0 + k < n) y[i0 + k] = e;
    e += v[k];
    if (i0 + k == n - 1) y[n] = e;
  }
  if (n == 0 && blockIdx.x == 0 && threadIdx.x == 0) y[0] = 0;
}

// ------------------------------------------------------------ sweep pass

constexpr int kGV = 16;                    // group slots per lane of a sweep tile
constexpr int kGT = 64 * kGV;              // group slots per sweep tile
// batches per sweep tile: the per-wave constant tables of 8 settings then
// leave room for two workgroups per CU beside 8 histograms of 1040 entries
template <int NC> constexpr int kGBof = NC == 5 ? 28 : 22;
static_assert(kGV % 4 == 0 && kGBof<5> < 64 && kGBof<7> < 64, "sweep tile shape");

struct GroupSweep {
  const int64_t* off;               // request offsets [nB + 1]
  const int64_t* gofs;              // group offsets [nB + 1]
  const unsigned long long* bsum;   // [4][nB]: sum p, sum c, sum p^2, count of c == 0;
                                    // [5][nB] with sum p*c (extended model)
  const uint32_t* gw;               // [groups + kGT] ((b mod 2^20) << 12) | tenant
  const v4f* gf;                    // [groups + kGT] (n, P, C, Q)
  const float* gr;                  // [groups + kGT] R = sum p*c (extended model)
  int64_t nB;
  const int64_t* wg_first;          // chunk table over batches (k_partition)
  unsigned long long* claims;
  int64_t n_chunks;
  uint64_t claim_base;
  double* partials;                 // [grid][V.n][n_tenants]
  int32_t n_tenants;
  const int32_t* hot;               // [kHot]
  // the previous pass's partials ([gridDim.x][prev_n][n_tenants], the other
  // buffer), folded into its output rows by this pass (null: none)
  const double* prev;
  double* prev_out;
  int32_t prev_n;
};

// Fold of the previous pass inside a pass: workgroup w owns entries
// [w*kFoldPer, (w+1)*kFoldPer) of the prev_n*n_tenants sums; thread t holds
// entry t % kFoldPer and rows t/kFoldPer + kFoldGroups*k, k < kFoldRows, loaded
// at the start of the pass and added after its own work (rows in a fixed
// order).  Used when prev_n*n_tenants <= kFoldPer*gridDim.x and gridDim.x <=
// kFoldGroups*kFoldRows.
constexpr int kFoldPer = 32;
constexpr int kFoldGroups = 16;  // kSweepWG / kFoldPer
constexpr int kFoldRows = 16;

// Threads per sweep workgroup: eight waves share one set of NV tenant
// histograms (one workgroup per compute unit), so a pass writes half as many
// partial rows as with four-wave workgroups.
constexpr int kSweepWG = 512;
constexpr int kSweepWaves = kSweepWG / 64;
static_assert(kSweepWG == 16 * 32, "the fold's thread mapping");

// NV: histogram rows, i.e. settings per pass, >= V.n; NC: 5 (Eq. 1) or 7
// (the extended model).  Work: the chunks of k_tiles (one static chunk per
// wave, then claimed ones).  LDS per workgroup: NV * (n_tenants + kHotSlots)
// doubles (dynamic) plus the per-wave tables.
template <int NV, int NC>
__global__ __launch_bounds__(kSweepWG) void k_sweep_groups(const GroupSweep P, const VarTableOf<NC> V) {
  constexpr bool EXT = NC == 7;
  constexpr int kGB = kGBof<NC>;
  constexpr int KC = EXT ? 4 : 3;                    // batch-independent constants
#ifndef LLMV_SWEEP_PRE
#define LLMV_SWEEP_PRE 1
#endif
  constexpr bool PRE = LLMV_SWEEP_PRE && !(EXT && NV == 4);  // registers: no spills
  extern __shared__ double s_hist[];                 // [NV][n_tenants + kHotSlots]
  __shared__ v4f s_kt[kSweepWaves][NV][kGB];              // per wave: (k0, k1, k2, k3)
  __shared__ float s_kt5[kSweepWaves][EXT ? NV : 1][EXT ? kGB : 1];  // per wave: k5
  __shared__ float s_K[NV * 4 * KC];                 // [setting][regime][k1..k3 (, k5)]
  __shared__ double s_fold[kSweepWG];                // the fold's row groups
  const int tid = threadIdx.x, lane = tid & 63;
  // [setting][batch of the tile]: lanes of one read that hold different
  // batches fall in different banks
  v4f(*kt)[kGB] = s_kt[tid >> 6];
  float(*kt5)[EXT ? kGB : 1] = s_kt5[tid >> 6];
  const int32_t T = P.n_tenants, TS = T + kHotSlots;
  int32_t hot[kHot];
#pragma unroll
  for (int h = 0; h < kHot; ++h) hot[h] = uni(P.hot[h]);
  for (int i = tid; i < NV * 4 * KC; i += kSweepWG)
    s_K[i] = V.K[i / (4 * KC)][(i / KC) % 4][i % KC];
  // the previous pass's partials of this workgroup's entries, loaded now and
  // folded after this pass's own work
  const int64_t fe = (int64_t)blockIdx.x * kFoldPer + tid % kFoldPer;
  const int frg = tid / kFoldPer;
  const int64_t fE = (int64_t)P.prev_n * T;
  double fr[kFoldRows];
#pragma unroll
  for (int k = 0; k < kFoldRows; ++k) {
    const int row = frg + kFoldGroups * k;
    fr[k] = (P.prev && fe < fE && row < (int)gridDim.x) ? P.prev[(int64_t)row * fE + fe] : 0.0;
  }
  for (int u = tid; u < NV * TS; u += kSweepWG) s_hist[u] = 0.0;
  __syncthreads();

  const int64_t workers = (int64_t)gridDim.x * kSweepWaves;
  int64_t chunk = (int64_t)blockIdx.x * kSweepWaves + (tid >> 6);
  while (chunk < P.n_chunks) {
    // claim the next chunk now: the value is first read once this one is done
    unsigned long long claim = ~0ull;
    if (P.n_chunks > workers && lane == 0) claim = atomicAdd(P.claims, 1ull);
    const int64_t bw0 = uni(P.wg_first[chunk]), bw1 = uni(P.wg_first[chunk + 1]);
    int64_t b = bw0;
    while (b < bw1) {
      // ---- tile: the longest run of whole batches from b within kGT group
      // slots from a 4-aligned base, at most kGB batches; a batch with more
      // groups alone, in several rounds
      const int64_t lim = min((int64_t)kGB, bw1 - b);
      const int64_t gv = lane <= lim ? P.gofs[b + lane] : 0;  // lane j: gofs[b + j]
      const int64_t g0 = uni(readlane_i64(gv, 0));
      const int64_t ga = g0 & ~(int64_t)3;
      const uint64_t fits = __ballot(lane >= 1 && lane <= lim && gv - ga <= kGT);
      int32_t count = uni((int32_t)__builtin_popcountll(fits));  // a prefix of lanes
      if (count == 0) count = 1;
      const int64_t g1 = uni(readlane_i64(gv, count));

      // ---- lane j: batch b + j under every setting
      if (lane < count) {
        const int64_t bb = b + lane;
        const int64_t n = P.off[bb + 1] - P.off[bb];
        if (n > 0) {
          const uint64_t sp = P.bsum[bb], sc = P.bsum[P.nB + bb], sq = P.bsum[2 * P.nB + bb];
          const uint64_t sz = P.bsum[3 * P.nB + bb];
          const uint64_t sr = EXT ? P.bsum[4 * P.nB + bb] : 0;
          // decode iff every request processes one token over a nonzero context
          const bool prefill = (sp != (uint64_t)n) || (sz != 0);
          float k0[kSweepG];
          const uint32_t sg = sweep_batch<NV, NC>(V, n, sp, sc, sq, sr, prefill, k0);
          const int ph = prefill ? 0 : 1;
#pragma unroll
          for (int g = 0; g < NV; ++g) {
            const int r = 2 * ph + (int)((sg >> g) & 1u);
            const float* kr = &s_K[(g * 4 + r) * KC];
            kt[g][lane] = (v4f){k0[g], kr[0], kr[1], kr[2]};
            if (EXT) kt5[g][lane] = kr[KC - 1];
          }
        }
      }
      wave_lds_sync();

      // ---- groups: lane-local runs of kGV slots; a lane reloads its
      // constants when its batch changes
      for (int64_t base = ga; base < g1; base += kGT) {
        const int64_t x = base + (int64_t)lane * kGV;
        uint32_t wv[kGV];
        v4f fv[kGV];
        float rv[EXT ? kGV : 1];
        // (x is a multiple of 4; the group arrays hold kGT slots past the last group)
#pragma unroll
        for (int v = 0; v < kGV / 4; ++v) {
          const v4i a = *(const v4i*)(P.gw + x + 4 * v);
          wv[4 * v] = (uint32_t)a.x;
          wv[4 * v + 1] = (uint32_t)a.y;
          wv[4 * v + 2] = (uint32_t)a.z;
          wv[4 * v + 3] = (uint32_t)a.w;
        }
#pragma unroll
        for (int q = 0; q < kGV; ++q) fv[q] = P.gf[x + q];
        if constexpr (EXT) {
#pragma unroll
          for (int v = 0; v < kGV / 4; ++v) {
            const v4f a = *(const v4f*)(P.gr + x + 4 * v);
            rv[4 * v] = a.x;
            rv[4 * v + 1] = a.y;
            rv[4 * v + 2] = a.z;
            rv[4 * v + 3] = a.w;
          }
        }
        uint32_t kcur = 0xffffffffu;
        v4f K[NV];
        float K5[EXT ? NV : 1];
        // PRE: the constants of the batch of the lane's first slot and of
        // the batch after it are read before the first atomic: a read
        // between the atomics waits for every atomic before it (LDS
        // operations of a wave complete in order)
        v4f KB[PRE ? NV : 1];
        float KB5[PRE && EXT ? NV : 1];
        uint32_t kbi = 0xffffffffu;
        if constexpr (PRE) {
          uint32_t l0 = ((wv[0] >> kGrpTenantBits) - (uint32_t)b) & kGrpBatchMask;
          l0 = min(l0, (uint32_t)count - 1u);  // slots before the tile's first group: any batch
          kcur = l0;
#pragma unroll
          for (int g = 0; g < NV; ++g) {
            K[g] = kt[g][l0];
            if (EXT) K5[g] = kt5[g][l0];
          }
          if (l0 + 1u < (uint32_t)count) {
            kbi = l0 + 1u;
#pragma unroll
            for (int g = 0; g < NV; ++g) {
              KB[g] = kt[g][kbi];
              if (EXT) KB5[g] = kt5[g][kbi];
            }
          }
        }
#pragma unroll
        for (int q = 0; q < kGV; ++q) {
          if (x + q >= g0 && x + q < g1) {
            const uint32_t w = wv[q];
            const uint32_t lb = ((w >> kGrpTenantBits) - (uint32_t)b) & kGrpBatchMask;
            const int32_t t = (int32_t)(w & kGrpTenantMask);
            int32_t e = t;
#pragma unroll
            for (int h = 0; h < kHot; ++h)
              if (t == hot[h]) e = T + h * kHotRep + (lane & (kHotRep - 1));
            if (lb != kcur) {
              kcur = lb;
              if (PRE && lb == kbi) {
#pragma unroll
                for (int g = 0; g < NV; ++g) {
                  K[g] = KB[g];
                  if (EXT) K5[g] = KB5[g];
                }
              } else {
#pragma unroll
                for (int g = 0; g < NV; ++g) {
                  K[g] = kt[g][lb];
                  if (EXT) K5[g] = kt5[g][lb];
                }
              }
            }
            const v4f f = fv[q];
            // all NV rows: rows past V.n are scratch, never flushed
#pragma unroll
            for (int g = 0; g < NV; ++g) {
              float t = fmaf(K[g].w, f.w, fmaf(K[g].z, f.z, fmaf(K[g].y, f.y, K[g].x * f.x)));
              if constexpr (EXT) t = fmaf(K5[g], rv[q], t);
              atomicAdd(s_hist + g * TS + e, (double)t);
            }
          }
        }
      }
      wave_lds_sync();
      b += count;
    }
    // claim k of this launch names chunk workers + k; past the last chunk, stop
    const uint64_t k = readlane_u64((uint64_t)claim, 0) - P.claim_base;
    chunk = k < (uint64_t)(P.n_chunks - workers) ? workers + (int64_t)k : P.n_chunks;
  }

  // fold the hot tenants' replicas (fixed order), then flush n_tenants
  // entries per setting
  __syncthreads();
  for (int i = tid; i < V.n * kHot; i += kSweepWG) {
    const int g = i / kHot, h = i % kHot;
    if (hot[h] >= 0) {
      double acc = s_hist[g * TS + hot[h]];
      for (int r = 0; r < kHotRep; ++r) acc += s_hist[g * TS + T + h * kHotRep + r];
      s_hist[g * TS + hot[h]] = acc;
    }
  }
  __syncthreads();
  double* dst = P.partials + (int64_t)blockIdx.x * V.n * T;
  for (int i = tid; i < V.n * T; i += kSweepWG) dst[i] = s_hist[(i / T) * TS + i % T];

  // the fold: each thread's rows in order, then the row groups in order
  if (P.prev) {
    double acc = fr[0];
#pragma unroll
    for (int k = 1; k < kFoldRows; ++k) acc += fr[k];
    s_fold[frg * kFoldPer + tid % kFoldPer] = acc;
    __syncthreads();
    if (frg == 0 && fe < fE) {
      double t = s_fold[tid];
      for (int g = 1; g < kFoldGroups; ++g) t += s_fold[g * kFoldPer + tid];
      P.prev_out[fe] = t;
    }
  }
}

}  // namespace llmv
