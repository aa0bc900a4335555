// kernels.hpp -- gfx950 kernels for batched LLMVisor latency attribution.
//
// The method (LLMVisor Sec. 2.1, Eq. 1; Sec. 2 "Problem formulation"):
// per batch, exact sums P = sum p, C = sum c, Q = sum p^2 and the batch phase;
// Eq. 1 with the phase's two coefficient sets (memory-bound, compute-bound);
// the larger one is the batch latency; each request's share is its own terms
// of the chosen set; tenant usage is the sum of its requests' shares.
//
// Work decomposition (memory-bound ragged reduction, no dense contraction):
//  * k_partition: splits the batch list into contiguous chunks by request
//    count: one large chunk per wave worker, taken statically, and many
//    small ones that workers claim from a counter as they finish (guided
//    self-scheduling, so no wave waits on a slower one at the end).
//  * k_tiles: persistent workgroups of four independent wave workers.  A wave
//    walks each of its chunks in wave tiles: runs of whole batches whose
//    requests fit in 64*kVec slots (lane l holds kVec consecutive requests), so every request is
//    read from HBM once, held in registers while its batch totals are formed,
//    and its share written once.  Batch totals are lane-local run sums added
//    into per-batch LDS accumulators; batch membership comes from an LDS
//    bitmask of batch starts and popcounts.  A batch larger than a tile is
//    listed: for k_long, whose waves walk such batches one each (held whole
//    in registers when it spans two tiles), or, under Eq. 1 attribution with
//    more than kListMin requests, with its segments for k_big_sums and the
//    segment part of k_long, which spread it over the whole grid.
//  * Tenant sums accumulate in an fp64 LDS histogram per workgroup, flushed
//    once to a [grid][n_tenants] partial array that k_tenant_reduce folds in
//    a fixed order.
// The what-if sweep (many coefficient settings over one trace) has kernels
// of its own in groups.hpp.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "model.hpp"

namespace llmv {

constexpr int kWG = 256;                     // threads per workgroup
constexpr int kWaves = kWG / 64;             // wave64
// Consecutive requests held per lane (a tile kernel instance takes one of
// the two: kVecOf below); a wave tile holds 64 times as many.
constexpr int kVecNarrow = 24;
constexpr int kVecWide = 28;
constexpr int kCapNarrow = 64 * kVecNarrow;  // request slots per narrow wave tile
constexpr int kHistLdsMax = 4096;                // tenants held in an LDS histogram
constexpr int kMaxGrid = 1024;                   // persistent workgroups, upper bound (256 CUs x 4)
constexpr int kTenantChunk = 16;                 // tenants per k_tenant_reduce block
// Work split of the tile kernel (build-time settings, for measurement)
#ifndef LLMV_STATIC_EIGHTHS
#define LLMV_STATIC_EIGHTHS 7  // requests in static chunks, in eighths
#endif
#ifndef LLMV_DYN_PER_WORKER
#define LLMV_DYN_PER_WORKER 4  // claimed chunks per wave worker, at most
#endif
#ifndef LLMV_MIN_CHUNK_TILES
#define LLMV_MIN_CHUNK_TILES 2  // tiles per claimed chunk, at least
#endif
#ifndef LLMV_PIECE_TILES
#define LLMV_PIECE_TILES 8  // tiles per static piece
#endif
constexpr int kStaticEighths = LLMV_STATIC_EIGHTHS;
constexpr int kDynPerWorker = LLMV_DYN_PER_WORKER;
// For wave tiles of `cap` request slots:
constexpr int64_t min_chunk(int64_t cap) { return LLMV_MIN_CHUNK_TILES * cap; }  // requests per claimed chunk, at least
constexpr int64_t min_dyn_share(int64_t cap) { return 32 * cap; }  // per worker, for claimed chunks
constexpr int64_t piece(int64_t cap) { return LLMV_PIECE_TILES * cap; }       // requests per static piece

// Chunks of the tile kernel's work.  Chunk w < n_static (static) starts at
// request w*s1; chunk n_static + j (claimed) starts at request F + j*s2,
// F = n_static*s1.  A chunk holds the batches whose start offset lies in
// [its start, the next chunk's start).  Wave worker w takes the static
// chunks w, w + W, ... (W workers, n_static >= W), then claims.
struct ChunkMap {
  int64_t s1, s2, F, n_static, n_chunks;
  // Number of chunks that start at or before request x (x >= 0).
  __host__ __device__ int64_t count_le(int64_t x) const {
    if (x < F) return x / s1 + 1;
    const int64_t j = (x - F) / s2 + 1, m = n_chunks - n_static;
    return n_static + (j < m ? j : m);
  }
};

// Counters of a launch (claims[]): the chunk claims of the tile kernel in
// kClaimGroups groups (wave worker w claims the dynamic chunks n_static +
// (w mod kClaimGroups) + k*kClaimGroups, k = 0, 1, ..., from counter w mod
// kClaimGroups, so that claims spread over several addresses), the listed
// batches with their segments, and the long batches.
constexpr int kClaimGroups = 8;
constexpr int kSegCounter = kClaimGroups;
constexpr int kLongCounter = kClaimGroups + 1;
constexpr int kCounters = kClaimGroups + 2;

// MODE_ATTR: latency, regime, share, tenant sums of one (shape, theta).
// MODE_FEAT: the feature rows.  MODE_EXT: the outputs of MODE_ATTR under the
// extended model (Eq. 1 plus a cross term a5*S5*sum p*c and a per-request
// term a6*S6*|B|).  MODE_SUMS: the exact batch sums with the extended
// model's sum p*c, and the phase (no per-request outputs).
enum { MODE_ATTR = 0, MODE_FEAT = 1, MODE_EXT = 2, MODE_SUMS = 3 };
// modes that form the batch sums of p*c
template <int MODE> constexpr bool kCrossSum = MODE == MODE_EXT || MODE == MODE_SUMS;
template <int MODE> constexpr bool kAttrMode = MODE == MODE_ATTR || MODE == MODE_EXT;

// Native vectors: 16-byte global loads / stores (dwordx4).
typedef int32_t v4i __attribute__((ext_vector_type(4)));
typedef float v4f __attribute__((ext_vector_type(4)));
enum { HIST_NONE = 0, HIST_LDS = 1, HIST_GLOBAL = 2 };

// Lane slots of a tile kernel instance: the wide tile where it is faster
// (attribution under Eq. 1 or the extended model without the tenant cache:
// 28 slots, about 2% on the heavy-tailed trace; the feature rows and batch
// sums, about 1%); the narrow one for the tenant cache, where the wide
// tile's registers (up to 255 VGPRs) cost more than its longer tiles gain.
__host__ __device__ constexpr bool wide_tile(int mode, int hist) {
  return (hist != HIST_GLOBAL && (mode == MODE_ATTR || mode == MODE_EXT)) ||
         mode == MODE_FEAT || mode == MODE_SUMS;
}
template <int MODE, int HIST>
constexpr int kVecOf = wide_tile(MODE, HIST) ? kVecWide : kVecNarrow;
__host__ __device__ constexpr int64_t tile_cap(int mode, int hist) {
  return 64 * (wide_tile(mode, hist) ? kVecWide : kVecNarrow);
}

// A batch listed for the segment kernels: its index and exact sums (sum p,
// sum c, sum p^2, count of c == 0), accumulated by k_big_sums.
struct BigEntry {
  int64_t b;
  unsigned long long s[4];
};

struct Params {
  const int64_t* off;
  const int32_t* p;
  const int32_t* c;
  const int32_t* tenant;
  int64_t nB, N;
  const int64_t* wg_first;  // [n_chunks+1] first batch of each chunk
  unsigned long long* claims;  // the launch's counters (kCounters)
  uint64_t claim_base;      // counter value when this launch starts
  int64_t n_chunks;
  int64_t n_static;         // chunks taken statically, round-robin (>= the wave workers)
  int32_t split_by_count;   // one workgroup, no chunk table: wave w takes batches
                            // [w*nB/4, (w+1)*nB/4) (small traces, one launch)
  float* latency;           // [nB] or null
  uint8_t* regime;          // [nB] or null
  float* share;             // [N] or null
  double* partials;         // [grid][n_tenants] (HIST_LDS)
  double* tenant_sums;      // [n_tenants] (HIST_GLOBAL: the tenant cache's output)
  float* x_req;             // [5][N] (MODE_FEAT) or null
  double* x_batch;          // [5][nB] (MODE_FEAT) or null
  int64_t* bsums;           // [4][nB] (|B|, sum p, sum c, sum p^2) (MODE_FEAT), with
                            // sum p*c as a fifth row (MODE_SUMS), or null
  uint8_t* bphase;          // [nB] phase, 255 for an empty batch (MODE_FEAT) or null
  // MODE_ATTR, multi-workgroup launches: a batch of more than kListMin
  // requests is not walked by the wave that meets it but listed, with its
  // segments of kBigSeg requests, for k_big_sums and k_long (null: such a
  // batch goes to the long list).  Both counts are in claims[kSegCounter]
  // (cleared by k_partition).
  struct BigEntry* big_list;  // listed batches and their exact sums
  uint64_t* big_seg;          // segments: (list index << 32) | segment within the batch
  // The other batches larger than a wave tile, listed by the wave that meets
  // them for k_long (count at *long_count = claims[kLongCounter]).
  int64_t* long_list;
  unsigned long long* long_count;
  int32_t n_tenants;
  int32_t hist_rep;         // MODE_ATTR, HIST_LDS: histogram replicas (1, 2 or 4)
  double S[4];              // shape constants
  double th[20];            // theta[phase][segment][k]
};

struct NoVars {};
// The extended model of a MODE_EXT launch: the two extra shape constants
// and the coefficients theta[phase][segment][k], k = 0..6 (beta, a1..a6).
struct ExtModel {
  double S5, S6;
  double th[28];
};
template <int MODE> struct VarsOf { using type = NoVars; };
template <> struct VarsOf<MODE_EXT> { using type = ExtModel; };

// ---------------------------------------------------------------- wave ops

// v_mov_b32_dpp with `old` = 0: lanes whose DPP source is out of range, or
// whose row is masked off, read 0.
template <int CTRL, int ROW_MASK>
__device__ __forceinline__ uint32_t dpp_u32(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, CTRL, ROW_MASK, 0xf, false);
}

template <int CTRL, int ROW_MASK>
__device__ __forceinline__ uint64_t dpp_u64(uint64_t v) {
  const uint32_t lo = dpp_u32<CTRL, ROW_MASK>((uint32_t)v);
  const uint32_t hi = dpp_u32<CTRL, ROW_MASK>((uint32_t)(v >> 32));
  return ((uint64_t)hi << 32) | lo;
}

// Inclusive prefix sum over the 64 lanes of a wave (integer, modulo 2^64):
// row_shr 1/2/4/8 scan each 16-lane row, row_bcast15 and row_bcast31 carry
// row totals into the rows above.
__device__ __forceinline__ uint64_t wave_incl_scan(uint64_t x) {
  x += dpp_u64<0x111, 0xf>(x);  // row_shr:1
  x += dpp_u64<0x112, 0xf>(x);  // row_shr:2
  x += dpp_u64<0x114, 0xf>(x);  // row_shr:4
  x += dpp_u64<0x118, 0xf>(x);  // row_shr:8
  x += dpp_u64<0x142, 0xa>(x);  // row_bcast:15 into rows 1 and 3
  x += dpp_u64<0x143, 0xc>(x);  // row_bcast:31 into rows 2 and 3
  return x;
}

__device__ __forceinline__ uint64_t readlane_u64(uint64_t v, int lane) {
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)v, lane);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(v >> 32), lane);
  return ((uint64_t)hi << 32) | lo;
}

__device__ __forceinline__ uint64_t wave_sum_u64(uint64_t x) {
  for (int m = 32; m >= 1; m >>= 1) x += __shfl_xor(x, m, 64);
  return x;
}

// ------------------------------------------------------------- the model

// Per-batch evaluation from exact integer sums.  Writes the batch outputs
// and the per-request share constants k[0..3]:
//   share_i = k0 + k1*p_i + k2*c_i + k3*p_i^2,
//   k0 = theta_beta*S0/n + theta_a4*n, k1 = theta_a1*S1, k2 = theta_a2*S2,
//   k3 = theta_a3*S3   (MODE_ATTR)
// or the per-request feature constants (S0/n, n) (MODE_FEAT).
template <int MODE>
__device__ __forceinline__ void batch_model(const Params& P, int64_t bg, int64_t n,
                                            uint64_t Psum, uint64_t Csum, uint64_t Qsum,
                                            bool prefill, double* k) {
  const double X[5] = {P.S[0], P.S[1] * (double)Psum, P.S[2] * (double)Csum,
                       P.S[3] * (double)Qsum, (double)n * (double)n};
  if (MODE == MODE_FEAT) {
    if (P.x_batch)
      for (int q = 0; q < 5; ++q) P.x_batch[q * P.nB + bg] = X[q];
    if (P.bsums) {
      P.bsums[0 * P.nB + bg] = n;
      P.bsums[1 * P.nB + bg] = (int64_t)Psum;
      P.bsums[2 * P.nB + bg] = (int64_t)Csum;
      P.bsums[3 * P.nB + bg] = (int64_t)Qsum;
    }
    if (P.bphase) P.bphase[bg] = prefill ? 0 : 1;
    k[0] = P.S[0] / (double)n;
    k[1] = (double)n;
    return;
  }
  double t;
  const int regime = eq1_batch(P.th, P.S, n, Psum, Csum, Qsum, prefill, &t, k);
  if (P.latency) P.latency[bg] = (float)t;
  if (P.regime) P.regime[bg] = (uint8_t)regime;
}

// Eq. 1 plus the two extra terms, added in order k = 0..6.
__device__ __forceinline__ double eq7(const double* th, const double X[7]) {
  double acc = th[0] * X[0];
#pragma unroll
  for (int k = 1; k < 7; ++k) acc = acc + th[k] * X[k];
  return acc;
}

// batch_model under the extended model: Rsum = sum p*c.  The share
// constants gain k0 += theta_a6*S6 and k4 = theta_a5*S5 (the coefficient of
// p*c):  share_i = k0 + k1*p_i + k2*c_i + k3*p_i^2 + k4*p_i*c_i.
__device__ __forceinline__ void ext_model(const Params& P, const ExtModel& E, int64_t bg,
                                          int64_t n, uint64_t Psum, uint64_t Csum, uint64_t Qsum,
                                          uint64_t Rsum, bool prefill, double* k, double* k4) {
  const double X[7] = {P.S[0], P.S[1] * (double)Psum, P.S[2] * (double)Csum,
                       P.S[3] * (double)Qsum, (double)n * (double)n, E.S5 * (double)Rsum,
                       E.S6 * (double)n};
  const int phase = prefill ? 0 : 1;
  const double* thm = E.th + (phase * 2 + 0) * 7;
  const double* thc = E.th + (phase * 2 + 1) * 7;
  const double tm = eq7(thm, X);
  const double tc = eq7(thc, X);
  // Roofline max of the two segments; ties stay memory-bound.
  const int seg = (tc > tm) ? 1 : 0;
  if (P.latency) P.latency[bg] = (float)(seg ? tc : tm);
  if (P.regime) P.regime[bg] = (uint8_t)(2 * phase + seg);
  const double* th = seg ? thc : thm;
  k[0] = th[0] * (P.S[0] / (double)n) + th[4] * (double)n + th[6] * E.S6;
  k[1] = th[1] * P.S[1];
  k[2] = th[2] * P.S[2];
  k[3] = th[3] * P.S[3];
  *k4 = th[5] * E.S5;
}

// MODE_SUMS: the exact sums of a nonempty batch and its phase.
__device__ __forceinline__ void sums_out(const Params& P, int64_t bg, int64_t n, uint64_t Psum,
                                         uint64_t Csum, uint64_t Qsum, uint64_t Rsum,
                                         bool prefill) {
  if (P.bsums) {
    P.bsums[0 * P.nB + bg] = n;
    P.bsums[1 * P.nB + bg] = (int64_t)Psum;
    P.bsums[2 * P.nB + bg] = (int64_t)Csum;
    P.bsums[3 * P.nB + bg] = (int64_t)Qsum;
    P.bsums[4 * P.nB + bg] = (int64_t)Rsum;
  }
  if (P.bphase) P.bphase[bg] = prefill ? 0 : 1;
}

template <int MODE>
__device__ __forceinline__ void empty_batch(const Params& P, int64_t bg) {
  if (MODE == MODE_FEAT || MODE == MODE_SUMS) {
    if (P.x_batch)
      for (int q = 0; q < 5; ++q) P.x_batch[q * P.nB + bg] = 0.0;
    if (P.bsums)
      for (int q = 0; q < (MODE == MODE_SUMS ? 5 : 4); ++q) P.bsums[q * P.nB + bg] = 0;
    if (P.bphase) P.bphase[bg] = 255;
  } else {
    if (P.latency) P.latency[bg] = 0.0f;
    if (P.regime) P.regime[bg] = 255;
  }
}

// ---------------------------------------------------------- tenant cache
//
// Tenant sums for more tenants than an LDS histogram holds (HIST_GLOBAL):
// each workgroup keeps a 4-way set-associative table of kCacheSlots (tenant,
// fp64 sum) slots in LDS.  A tenant's bucket is a hash of its id; one 16-byte
// LDS read gives the bucket's four tags.  A tenant claims a free way of its
// bucket (compare-and-swap of the tag: tags only ever change from empty to a
// tenant, so a stale read is harmless) on its second sight in the workgroup,
// which a 64K-bit filter of hashed tenant ids records, so that tenants seen
// once do not take the ways frequent tenants need; one that finds its bucket
// full, or is seen for the first time, adds into the output with a global
// atomic.
// At the end each workgroup adds its slots into the output (cleared before
// the launch).  Under a skewed tenant mix the frequent tenants are seen first
// and stay in LDS, so the global atomics go to rare tenants and seldom
// collide.
constexpr int kCacheLog2 = 11;
constexpr int kCacheSlots = 1 << kCacheLog2;
constexpr int kSeenWords = 2048;  // 64K bits
constexpr size_t kCacheLds =
    kCacheSlots * (sizeof(double) + sizeof(int32_t)) + kSeenWords * sizeof(uint32_t);

__device__ __forceinline__ int32_t* cache_tags(double* base) {
  return (int32_t*)(base + kCacheSlots);
}

__device__ __forceinline__ uint32_t* cache_seen(double* base) {
  return (uint32_t*)(cache_tags(base) + kCacheSlots);
}

__device__ __forceinline__ void cache_init(double* base) {
  int32_t* tag = cache_tags(base);
  uint32_t* seen = cache_seen(base);
  for (int i = threadIdx.x; i < kCacheSlots; i += blockDim.x) {
    base[i] = 0.0;
    tag[i] = -1;
  }
  for (int i = threadIdx.x; i < kSeenWords; i += blockDim.x) seen[i] = 0u;
}

__device__ __forceinline__ void cache_add(double* base, int32_t t, double v, double* out) {
  int32_t* tag = cache_tags(base);
  const uint32_t bk = ((uint32_t)t * 2654435761u) >> (32 - (kCacheLog2 - 2));
  int32_t* tb = tag + 4 * bk;
  const v4i tg = *(const v4i*)tb;
  int w = tg.x == t ? 0 : (tg.y == t ? 1 : (tg.z == t ? 2 : (tg.w == t ? 3 : -1)));
  if (w < 0 && (tg.x < 0 || tg.y < 0 || tg.z < 0 || tg.w < 0)) {
    // a free way: claim it on the tenant's second sight
    const uint32_t hs = ((uint32_t)t * 0x85ebca6bu) >> 16;
    const uint32_t bit = 1u << (hs & 31u);
    if (atomicOr(cache_seen(base) + (hs >> 5), bit) & bit) {
      const int32_t ways[4] = {tg.x, tg.y, tg.z, tg.w};
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        if (w < 0 && ways[j] < 0) {
          const int32_t old = atomicCAS(tb + j, -1, t);
          if (old < 0 || old == t) w = j;
        }
      }
    }
  }
  if (w >= 0)
    atomicAdd(base + 4 * bk + w, v);
  else
    unsafeAtomicAdd(out + t, v);
}

// After the workgroup's last add (the caller synchronises first).
__device__ __forceinline__ void cache_flush(double* base, double* out) {
  const int32_t* tag = cache_tags(base);
  for (int i = threadIdx.x; i < kCacheSlots; i += blockDim.x) {
    const int32_t t = tag[i];
    if (t >= 0) unsafeAtomicAdd(out + t, base[i]);
  }
}

// Per-request epilogue: the share (+ tenant histogram) or the feature row.
// Shares: k0 + k1*p + k2*c + k3*p^2 (+ k4*p*c under the extended model, k[4])
// in fp32 from the batch's constants (themselves evaluated in fp64),
// relative error a few fp32 ulp.
template <int MODE, int HIST, bool SHARE>
__device__ __forceinline__ float request_out(const Params& P, const float* k, const double* kd,
                                             int32_t p, int32_t c, double* s_hist, int32_t t,
                                             int64_t i) {
  if (MODE == MODE_FEAT) {
    if (P.x_req) {
      const double pd = (double)p;
      const int64_t N = P.N;
      P.x_req[0 * N + i] = (float)kd[0];
      P.x_req[1 * N + i] = (float)(P.S[1] * pd);
      P.x_req[2 * N + i] = (float)(P.S[2] * (double)c);
      P.x_req[3 * N + i] = (float)(P.S[3] * (pd * pd));
      P.x_req[4 * N + i] = (float)kd[1];
    }
    return 0.0f;
  }
  float s = share_of(k, p, c);
  if constexpr (MODE == MODE_EXT) s = fmaf(k[4], (float)p * (float)c, s);
  if (HIST == HIST_LDS) atomicAdd(s_hist + t, (double)s);
  if (HIST == HIST_GLOBAL) cache_add(s_hist, t, (double)s, P.tenant_sums);
  return s;
}

// ------------------------------------------------------------ partition

// wg_first[w] = first batch whose start offset is >= the start of chunk w
// (w < n_chunks), wg_first[n_chunks] = nB; clears the launch's counters
// (claims[0 .. kCounters-1]).
__global__ void k_partition(const int64_t* __restrict__ off, int64_t nB, const ChunkMap cm,
                            int64_t* __restrict__ wg_first, unsigned long long* claims) {
  const int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t b = gid; b <= nB; b += stride) {
    const int64_t wlo = (b == 0) ? 0 : cm.count_le(off[b - 1]);
    const int64_t whi = (b == nB) ? cm.n_chunks - 1 : min(cm.n_chunks - 1, cm.count_le(off[b]) - 1);
    for (int64_t w = wlo; w <= whi; ++w) wg_first[w] = b;
  }
  if (gid == 0) {
    wg_first[cm.n_chunks] = nB;
    for (int i = 0; i < kCounters; ++i) claims[i] = 0ull;
  }
}

__global__ void k_zero_f64(double* __restrict__ x, int64_t n) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) x[i] = 0.0;
}

// ------------------------------------------------------------ wave tiles
//
// Every wave is an independent worker over its own contiguous range of
// batches (no workgroup barriers inside the loop); the four waves of a
// workgroup share only the LDS tenant histogram.  A wave tile is a run of
// whole batches whose requests fit in kTile slots from a 16-byte aligned
// base.  The tile is held in registers as kRounds rounds of 64*kVec slots:
// in round r lane l holds slots 64*kVec*r + kVec*l .. 64*kVec*r + kVec*l +
// kVec-1.

constexpr int kRounds = 1;
constexpr int kTileBatches = 63;                // batches per wave tile (64 offsets)

// The wave tile of VEC slots per lane.
template <int VEC>
struct TileShape {
  static_assert(VEC % 4 == 0 && VEC <= 28, "lane slots: multiple of 4, bits fit a word pair");
  static constexpr int kRoundSlots = 64 * VEC;
  static constexpr int kTile = kRounds * kRoundSlots;  // request slots per wave tile
  static constexpr int kTileMaskWords = kTile / 32;    // batch-start bitmask words
  // Lane pitch of the share stage, in floats: an odd number of 16-byte
  // units, so that the 16-byte stage writes of 16 consecutive lanes fall in
  // distinct groups of four of the 64 LDS banks (28 needs no padding; 24 is
  // padded to 28).
  static constexpr int kStagePitch = (VEC / 4) % 2 ? VEC : VEC + 4;
};
// The tile constants of VEC as local names.
#define LLMV_TILE_CONSTANTS(VEC)                                          \
  constexpr int kVec = (VEC);                                             \
  constexpr int kRoundSlots = TileShape<(VEC)>::kRoundSlots;              \
  constexpr int kTile = TileShape<(VEC)>::kTile;                          \
  constexpr int kTileMaskWords = TileShape<(VEC)>::kTileMaskWords;        \
  constexpr int kStagePitch = TileShape<(VEC)>::kStagePitch;              \
  (void)kVec; (void)kRoundSlots; (void)kTile; (void)kTileMaskWords; (void)kStagePitch

// Within one wave tile the sum of c and the count of c == 0 share a word:
// a tile holds fewer than 2^16 requests, each c < 2^31, so sum c < 2^47
// stays below the count's bits.  (long_batch keeps them apart: a batch
// larger than a tile may reach 2^22 requests and sum c up to 2^53.)
constexpr uint64_t kZeroUnit = 1ull << 48;      // count of c == 0, above the c sum
constexpr uint64_t kCMask = kZeroUnit - 1;
static_assert(64 * kVecWide < (1 << 16) && 64ull * kVecWide * 0x7fffffffull < kZeroUnit,
              "a wave tile's zero count and sum of c fit their fields");

struct BatchAcc {
  uint64_t p;   // sum p
  uint64_t cz;  // sum c (bits 0..47) | count of c == 0 (bits 48..63)
  uint64_t q;   // sum p^2
};

// LDS private to one wave.
template <int VEC>
struct WaveLds {
  uint32_t mask[TileShape<VEC>::kTileMaskWords + 2];  // bit x: a nonempty batch starts at slot x
  BatchAcc acc[kTileBatches];         // per nonempty batch of the tile
  double k[kTileBatches][4];          // per nonempty batch: share / feature constants
};

// Orders LDS accesses between the lanes of one wave (a wave's LDS accesses
// complete in order; this keeps the compiler from moving them across).
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

__device__ __forceinline__ int64_t readlane_i64(int64_t v, int lane) {
  return (int64_t)readlane_u64((uint64_t)v, lane);
}

// Wave-uniform values held in scalar registers.
__device__ __forceinline__ int32_t uni(int32_t v) { return __builtin_amdgcn_readfirstlane(v); }
__device__ __forceinline__ int64_t uni(int64_t v) {
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)v);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)((uint64_t)v >> 32));
  return (int64_t)(((uint64_t)hi << 32) | lo);
}

__device__ __forceinline__ float uni_f32(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_readfirstlane(__builtin_bit_cast(int, v)));
}
__device__ __forceinline__ double uni_f64(double v) {
  return __builtin_bit_cast(double, (uint64_t)uni((int64_t)__builtin_bit_cast(uint64_t, v)));
}

// The sum over the 64 lanes (integer, modulo 2^64), wave-uniform.  DPP
// steps (no LDS): a shuffle would go through the LDS and wait behind the
// wave's LDS atomics.
__device__ __forceinline__ uint64_t wave_sum(uint64_t x) {
  return readlane_u64(wave_incl_scan(x), 63);
}

__device__ __forceinline__ uint32_t wave_incl_scan_u32(uint32_t x) {
  x += dpp_u32<0x111, 0xf>(x);
  x += dpp_u32<0x112, 0xf>(x);
  x += dpp_u32<0x114, 0xf>(x);
  x += dpp_u32<0x118, 0xf>(x);
  x += dpp_u32<0x142, 0xa>(x);
  x += dpp_u32<0x143, 0xc>(x);
  return x;
}

// Loads slots x .. x+kVec-1 (x a multiple of 4, x >= 0) of p, c (and
// tenant); slots at or past N read as 0.
template <int VEC, bool TENANT>
__device__ __forceinline__ void load_slots(const Params& P, int64_t x, int32_t* pv, int32_t* cv,
                                       int32_t* tv) {
  LLMV_TILE_CONSTANTS(VEC);
  if (x + kVec <= P.N) {
#pragma unroll
    for (int g = 0; g < kVec / 4; ++g) {
      const v4i a = *(const v4i*)(P.p + x + 4 * g);
      const v4i d = *(const v4i*)(P.c + x + 4 * g);
      pv[4 * g] = a.x; pv[4 * g + 1] = a.y; pv[4 * g + 2] = a.z; pv[4 * g + 3] = a.w;
      cv[4 * g] = d.x; cv[4 * g + 1] = d.y; cv[4 * g + 2] = d.z; cv[4 * g + 3] = d.w;
      if (TENANT) {
        const v4i t = *(const v4i*)(P.tenant + x + 4 * g);
        tv[4 * g] = t.x; tv[4 * g + 1] = t.y; tv[4 * g + 2] = t.z; tv[4 * g + 3] = t.w;
      }
    }
  } else {
#pragma unroll
    for (int q = 0; q < kVec; ++q) {
      const bool in = x + q < P.N;
      pv[q] = in ? P.p[x + q] : 0;
      cv[q] = in ? P.c[x + q] : 0;
      if (TENANT) tv[q] = in ? P.tenant[x + q] : 0;
    }
  }
}

// Writes one round of shares staged lane-major in the wave's LDS stage
// (lane l: slots s0 + kVec*l .. s0 + kVec*l + kVec-1, pitch kStagePitch) so
// that every global store instruction writes 1 KB of consecutive shares.
// Only slots in [xf, L) are written.  BATCH: every group's stage read is
// issued before the first store, so that the reads wait once (a wave's LDS
// operations complete in order, behind the round's tenant-sum atomics)
// instead of once per store; it holds the round's shares in 28 more
// registers, which the tile kernel affords and k_long (at its register
// limit) does not.
template <int VEC, bool BATCH>
__device__ __forceinline__ void store_round(const Params& P, float* stage, int64_t ra, int32_t s0,
                                            int32_t xf, int32_t L) {
  LLMV_TILE_CONSTANTS(VEC);
  const int lane = threadIdx.x & 63;
  wave_lds_sync();
  // the round's shares of this lane's store groups: read all at once (BATCH)
  // or each before its store
  v4f val[BATCH ? kVec / 4 : 1];
  if constexpr (BATCH) {
#pragma unroll
    for (int g = 0; g < kVec / 4; ++g) {
      const int32_t e = 256 * g + 4 * lane;
      val[g] = *(const v4f*)&stage[(e / kVec) * kStagePitch + (e % kVec)];
    }
  }
#pragma unroll
  for (int g = 0; g < kVec / 4; ++g) {
    if (256 * g >= L - s0) break;          // no slot of the round left (wave-uniform)
    const int32_t e = 256 * g + 4 * lane;  // slot within the round
    const int32_t x = s0 + e;              // slot within the tile
    const v4f v = BATCH ? val[BATCH ? g : 0] : *(const v4f*)&stage[(e / kVec) * kStagePitch + (e % kVec)];
    if (x >= xf && x + 4 <= L) {
      __builtin_nontemporal_store(v, (v4f*)(P.share + ra + x));  // not re-read
    } else {
#pragma unroll
      for (int q = 0; q < 4; ++q)
        if (x + q >= xf && x + q < L) P.share[ra + x + q] = v[q];
    }
  }
  wave_lds_sync();
}

// Buffer resource over n int32 elements from base (both wave-uniform,
// n < 2^29): a load of an element at or past n returns 0 and reads no
// memory.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t elem_rsrc(const int32_t* base, int64_t n) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<int32_t*>(base), (short)0, (int)(n * 4),
                                           0x00020000);
}
constexpr int kNT = 2;  // cache policy of a buffer access: streamed (non-temporal)
template <int AUX = 0>
__device__ __forceinline__ v4i load4(__amdgpu_buffer_rsrc_t r, int32_t elem) {
  return (v4i)__builtin_amdgcn_raw_buffer_load_b128(r, 4 * elem, 0, AUX);
}

// Slots x .. x+VEC-1 (x = VEC * lane) of one round of a long batch: p, c
// (and tenant) through buffers over the round's m slots, so that slots past
// the batch read as 0 without a memory access.
// NG: the groups of 4 slots loaded (the rest are zero), all of them unless a
// round is known to hold at most 4*NG slots.
template <int VEC, bool TENANT, int NG = VEC / 4>
__device__ __forceinline__ void load_round(const Params& P, int64_t o, int64_t m, int32_t x,
                                           int32_t* pv, int32_t* cv, int32_t* tv) {
  const auto bp = elem_rsrc(P.p + o, m), bc = elem_rsrc(P.c + o, m);
#pragma unroll
  for (int g = 0; g < VEC / 4; ++g) {
    const v4i z = {0, 0, 0, 0};
    const v4i a = g < NG ? load4(bp, x + 4 * g) : z, d = g < NG ? load4(bc, x + 4 * g) : z;
    pv[4 * g] = a.x; pv[4 * g + 1] = a.y; pv[4 * g + 2] = a.z; pv[4 * g + 3] = a.w;
    cv[4 * g] = d.x; cv[4 * g + 1] = d.y; cv[4 * g + 2] = d.z; cv[4 * g + 3] = d.w;
  }
  if (TENANT) {
    const auto bt = elem_rsrc(P.tenant + o, m);
#pragma unroll
    for (int g = 0; g < VEC / 4; ++g) {
      const v4i t = g < NG ? load4(bt, x + 4 * g) : (v4i){0, 0, 0, 0};
      tv[4 * g] = t.x; tv[4 * g + 1] = t.y; tv[4 * g + 2] = t.z; tv[4 * g + 3] = t.w;
    }
  }
}

// One batch too large for a wave tile (k_long), walked by one wave in
// rounds of kRoundSlots slots from ra (its first request rounded down to 4).
// A batch of two rounds is held whole in registers: its requests are read
// once, as in a tile.  A longer one keeps its first round in registers and
// streams the others twice: for the exact sums, then for the per-request
// outputs.  wk, wk4: the wave's LDS words for the batch constants.
template <int MODE, int HIST, bool SHARE>
__device__ __forceinline__ void long_batch(const Params& P, const typename VarsOf<MODE>::type& V, double* wk,
                           double* wk4, float* stage, int64_t bg, int64_t rs, int64_t re,
                           double* s_hist) {
  constexpr int VEC = kVecOf<MODE, HIST>;
  LLMV_TILE_CONSTANTS(VEC);
  constexpr bool OUT = MODE != MODE_SUMS;  // per-request outputs
  constexpr bool TEN = OUT && HIST != HIST_NONE;
  constexpr bool STAGE = kAttrMode<MODE> && SHARE;
  const int lane = threadIdx.x & 63;
  const int64_t ra = uni(rs & ~(int64_t)3);
  const int32_t xf = uni((int32_t)(rs - ra));  // first slot of the batch
  const int32_t L = uni((int32_t)(re - ra));   // slots up to its end (> kRoundSlots)
  const int32_t nr = (L + kRoundSlots - 1) / kRoundSlots;  // rounds, at least 2
  const int32_t x0 = lane * kVec;
  // slots of round r: [r*kRoundSlots, min((r+1)*kRoundSlots, L)), from request o(r)
  auto o_of = [&](int32_t r) { return ra + (int64_t)r * kRoundSlots; };
  auto m_of = [&](int32_t r) { return (int64_t)min(kRoundSlots, L - r * kRoundSlots); };

  // Sums over up to 2^22 requests: sum c reaches 2^53, so the tile's packed
  // (sum c, zero count) word does not apply; a zero context is a flag.
  uint64_t sp = 0, sc = 0, sq = 0, sr = 0;
  bool zc = false;  // this lane saw a request with c == 0
  // this lane's slots of round r that hold requests of the batch, as a bit mask
  auto vmask = [&](int32_t r) {
    const int32_t s = r * kRoundSlots + x0;
    const int32_t a = max(xf - s, 0), z = min(L - s, kVec);
    return z > a ? ((1u << (z - a)) - 1u) << a : 0u;
  };
  auto add = [&](const int32_t* pv, const int32_t* cv, int32_t r) {
    const uint32_t v = vmask(r);
#pragma unroll
    for (int q = 0; q < kVec; ++q) {
      if ((v >> q) & 1u) {
        const uint32_t p = (uint32_t)pv[q], c = (uint32_t)cv[q];
        sp += p;
        sc += c;
        zc |= c == 0;
        sq += (uint64_t)p * p;
        if constexpr (kCrossSum<MODE>) sr += (uint64_t)p * c;
      }
    }
  };
  // the batch model on lane 0; every lane gets the share constants
  double kd[4] = {0.0, 0.0, 0.0, 0.0};
  float k[5] = {0.0f, 0.0f, 0.0f, 0.0f, 0.0f};
  auto model = [&]() {
    sp = wave_sum(sp);
    sc = wave_sum(sc);
    sq = wave_sum(sq);
    if constexpr (kCrossSum<MODE>) sr = wave_sum(sr);
    const int64_t n = re - rs;
    // decode iff every request processes one token over a nonzero context
    const bool prefill = (sp != (uint64_t)n) || (__ballot(zc) != 0);
    if (lane == 0) {
      if constexpr (MODE == MODE_SUMS)
        sums_out(P, bg, n, sp, sc, sq, sr, prefill);
      else if constexpr (MODE == MODE_EXT)
        ext_model(P, V, bg, n, sp, sc, sq, sr, prefill, wk, wk4);
      else
        batch_model<MODE>(P, bg, n, sp, sc, sq, prefill, wk);
    }
    if constexpr (OUT) {
      // the constants are wave-uniform: held in scalar registers
      wave_lds_sync();
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        kd[q] = uni_f64(wk[q]);
        k[q] = uni_f32((float)kd[q]);
      }
      if constexpr (MODE == MODE_EXT) k[4] = uni_f32((float)wk4[0]);
    }
  };
  auto out = [&](const int32_t* pv, const int32_t* cv, const int32_t* tv, int32_t r) {
    const int32_t s = r * kRoundSlots + x0;
    const uint32_t v = vmask(r);
    const int32_t m = (int32_t)m_of(r);
#pragma unroll
    for (int g = 0; g < kVec / 4; ++g) {
      if (4 * g >= m) break;  // no lane holds a slot of this group (wave-uniform)
      float sv[4];
#pragma unroll
      for (int qq = 0; qq < 4; ++qq) {
        const int q = 4 * g + qq;
        sv[qq] = 0.0f;
        if ((v >> q) & 1u)
          sv[qq] = request_out<MODE, HIST, SHARE>(P, k, kd, pv[q], cv[q], s_hist, tv[q], ra + s + q);
      }
      if (STAGE) *(v4f*)&stage[lane * kStagePitch + 4 * g] = (v4f){sv[0], sv[1], sv[2], sv[3]};
    }
    if (STAGE) store_round<VEC, false>(P, stage, ra, r * kRoundSlots, xf, L);
  };

  int32_t p0[kVec], c0[kVec], t0[kVec];
  load_round<VEC, TEN>(P, o_of(0), m_of(0), x0, p0, c0, t0);
  if (nr == 2) {
    int32_t p1[kVec], c1[kVec], t1[kVec];
    // a second round of at most 4 slots (a batch just over a tile) sits in
    // lane 0's first group: one load per array instead of VEC/4 (not with
    // the tenant cache, where the second path would spill)
    if (HIST != HIST_GLOBAL && m_of(1) <= 4)
      load_round<VEC, TEN, 1>(P, o_of(1), m_of(1), x0, p1, c1, t1);
    else
      load_round<VEC, TEN>(P, o_of(1), m_of(1), x0, p1, c1, t1);
    add(p0, c0, 0);
    add(p1, c1, 1);
    model();
    if constexpr (OUT) {
      out(p0, c0, t0, 0);
      out(p1, c1, t1, 1);
    }
  } else {
    {
      int32_t pa[kVec], ca[kVec], ta[kVec];
      load_round<VEC, false>(P, o_of(1), m_of(1), x0, pa, ca, ta);
      add(p0, c0, 0);
      add(pa, ca, 1);
    }
#pragma unroll 1
    for (int32_t r = 2; r < nr; ++r) {
      int32_t pa[kVec], ca[kVec], ta[kVec];
      load_round<VEC, false>(P, o_of(r), m_of(r), x0, pa, ca, ta);
      add(pa, ca, r);
    }
    model();
    if constexpr (OUT) {
      out(p0, c0, t0, 0);
#pragma unroll 1
      for (int32_t r = 1; r < nr; ++r) {
        int32_t pa[kVec], ca[kVec], ta[kVec];
        load_round<VEC, TEN>(P, o_of(r), m_of(r), x0, pa, ca, ta);
        out(pa, ca, ta, r);
      }
    }
  }
  wave_lds_sync();
}

// ------------------------------------------------------ long batches, listed

constexpr int kBigWG = kWG;                             // threads per segment workgroup
constexpr int kBigPer = 32;                             // requests per thread per pass
constexpr int64_t kBigSub = (int64_t)kBigWG * kBigPer;  // requests per workgroup pass
constexpr int64_t kBigSeg = 4 * kBigSub;                // requests per segment
constexpr int kBigGrid = 512;                           // k_big_sums workgroups
#ifndef LLMV_LIST_MIN
#define LLMV_LIST_MIN (64 * 64 * kVecWide)
#endif
// Eq. 1 attribution spreads the batches of more than kListMin requests (64
// wide tiles) over the grid in segments; shorter ones are walked by one
// k_long wave each.
constexpr int64_t kListMin = LLMV_LIST_MIN;
static_assert(kListMin >= 64 * kVecWide, "a listed batch is larger than any wave tile");

// The batches listed for the segment kernels and their segments share one
// counter (claims[kSegCounter]): the batch count above bit kSegBits, the
// segment count below.
constexpr int kSegBits = 40;
constexpr uint64_t kSegMask = (1ull << kSegBits) - 1;

// Lists the batches b .. b+adv-1, each larger than a wave tile (lane j < adv
// holds offsets[b+j] in wv, lane j+1 the batch's end).  Under Eq. 1
// attribution with the segment lists set (SEG), those of more than kListMin
// requests go to big_list with their segments (segment j of a batch holds
// its requests in [ra + j*kBigSeg, ra + (j+1)*kBigSeg), ra = its first
// request rounded down to 4; the entry's sums start at zero), with one
// atomic for the run.  The others are appended to the wave's LDS buffer
// lbuf (n_long entries, at most kLongBuf), flushed to the long list by
// flush() when the run would not fit.
constexpr int kLongBuf = 4 * kTileBatches;  // int64 entries in a wave's share-constant area
template <bool SEG, typename F>
__device__ __forceinline__ void list_run(const Params& P, int64_t b, int64_t wv, int32_t adv,
                                         int64_t* lbuf, int32_t& n_long, F&& flush) {
  const int lane = threadIdx.x & 63;
  const int64_t rs = wv, re = __shfl(wv, min(lane + 1, 63), 64);
  const bool in = lane < adv;
  const bool big = SEG && in && P.big_list != nullptr && re - rs > kListMin;
  const bool lng = in && !big;
  const uint64_t below = (1ull << lane) - 1ull;
  const uint64_t ml = __ballot(lng);
  if (ml) {
    const int32_t cnt = __builtin_popcountll(ml);
    if (n_long + cnt > kLongBuf) flush();
    if (lng) lbuf[n_long + __builtin_popcountll(ml & below)] = b + lane;
    n_long += cnt;
  }
  if constexpr (SEG) {
    const uint64_t mb = __ballot(big);
    if (mb) {
      const uint32_t q = big ? (uint32_t)((re - (rs & ~(int64_t)3) + kBigSeg - 1) / kBigSeg) : 0u;
      const uint32_t qs = wave_incl_scan_u32(q);
      const uint64_t Q = (uint32_t)__builtin_amdgcn_readlane((int)qs, 63);
      unsigned long long at = 0;
      if (lane == 0)
        at = atomicAdd(P.claims + kSegCounter,
                       ((unsigned long long)__builtin_popcountll(mb) << kSegBits) | Q);
      at = readlane_u64(at, 0);
      if (big) {
        const uint64_t k = (at >> kSegBits) + __builtin_popcountll(mb & below);
        P.big_list[k] = BigEntry{b + lane, {0ull, 0ull, 0ull, 0ull}};
        const uint64_t first = (at & kSegMask) + qs - q;
        for (uint32_t j = 0; j < q; ++j) P.big_seg[first + j] = (k << 32) | j;
      }
    }
  }
}

// V: the extended model (MODE_EXT), an empty struct otherwise.  The LDS
// tenant histogram (HIST_LDS) holds hist_rep replicas of n_tenants entries:
// lane l adds into replica l % hist_rep, so that lanes of one atomic that
// share a frequent tenant spread over hist_rep entries.
template <int MODE, int HIST, bool SHARE>
__global__ __launch_bounds__(kWG) void k_tiles(const Params P,
                                               const typename VarsOf<MODE>::type V) {
  constexpr int VEC = kVecOf<MODE, HIST>;
  LLMV_TILE_CONSTANTS(VEC);
  extern __shared__ double s_hist[];  // [hist_rep][n_tenants] when HIST_LDS
  __shared__ WaveLds<VEC> s_wave[kWaves];
  constexpr bool STAGE = kAttrMode<MODE> && SHARE;
  constexpr bool EXT = MODE == MODE_EXT;
  constexpr bool RSUM = kCrossSum<MODE>;
  // extended model, per wave: sum p*c and the share constant k4 of each batch
  __shared__ uint64_t s_rsum[RSUM ? kWaves * kTileBatches : 1];
  __shared__ double s_k4[EXT ? kWaves * kTileBatches : 1];
  __shared__ float s_stage[STAGE ? kWaves * 64 * kStagePitch : 1];  // shares, per wave
  constexpr bool TEN = HIST != HIST_NONE;
  // the share constants of a lane's first two batches read ahead (see the
  // per-request loop)
  constexpr bool PRE = kAttrMode<MODE>;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  WaveLds<VEC>& W = s_wave[tid >> 6];
  uint64_t* W_r = s_rsum + (RSUM ? (tid >> 6) * kTileBatches : 0);
  double* W_k4 = s_k4 + (EXT ? (tid >> 6) * kTileBatches : 0);
  float* stage = s_stage + (STAGE ? (tid >> 6) * 64 * kStagePitch : 0);
  const int32_t x0 = lane * kVec;  // first slot of this lane in a round
  const int32_t n_hist = P.hist_rep * P.n_tenants;

  if (HIST == HIST_LDS)
    for (int u = tid; u < n_hist; u += kWG) s_hist[u] = 0.0;
  if (HIST == HIST_GLOBAL) cache_init(s_hist);
  // one workgroup, no k_partition: the count of listed batches starts here
  if (P.split_by_count && tid == 0) atomicExch(P.long_count, 0ull);
  // this lane's replica of the histogram
  double* s_hist_lane = s_hist;
  if (HIST == HIST_LDS) s_hist_lane = s_hist + (lane & (P.hist_rep - 1)) * P.n_tenants;
  __syncthreads();

  // Wave w runs the static chunks w, w + W, ..., then claimed ones.  The
  // next chunk's batch range and offsets window are loaded during the
  // current chunk's first tiles: a static one is known at once, a claimed
  // one once the claim issued at the start of the current chunk returns (a
  // claim is issued for the last static chunk and every claimed chunk, so a
  // launch takes W + n_chunks - n_static claims).
  const int64_t workers = (int64_t)gridDim.x * kWaves;
  const bool dyn = P.n_chunks > P.n_static;
  auto first_batch = [&](int64_t ch) {
    return P.split_by_count ? P.nB * ch / workers : uni(P.wg_first[ch]);
  };
  // offsets window: lane j holds offsets[x0 + j] for j <= min(kTileBatches, x1 - x0)
  auto window = [&](int64_t x0, int64_t x1) {
    return (x0 < x1 && lane <= min((int64_t)kTileBatches, x1 - x0)) ? P.off[x0 + lane] : (int64_t)0;
  };
  // claim k of this worker's group cg names chunk n_static + cg + k*kClaimGroups;
  // past the last chunk, stop
  const int cg = (int)(((int64_t)blockIdx.x * kWaves + (tid >> 6)) % kClaimGroups);
  auto claimed_chunk = [&](unsigned long long cl) {
    const uint64_t k = readlane_u64((uint64_t)cl, 0) - P.claim_base;
    if (!dyn || k >= (uint64_t)(P.n_chunks - P.n_static)) return P.n_chunks;
    const uint64_t c = (uint64_t)P.n_static + (uint64_t)cg + k * (uint64_t)kClaimGroups;
    return c < (uint64_t)P.n_chunks ? (int64_t)c : P.n_chunks;
  };
  auto claim_next = [&](int64_t ch) {
    unsigned long long cl = ~0ull;
    if (dyn && ch < P.n_chunks && ch + workers >= P.n_static && lane == 0)
      cl = atomicAdd(P.claims + cg, 1ull);
    return cl;
  };
  // batches larger than a tile, buffered in the wave's share-constant area
  // (free between tiles) and flushed to the long list with one atomic
  int64_t* lbuf = (int64_t*)&W.k[0][0];
  int32_t n_long = 0;
  auto flush_long = [&]() {
    unsigned long long at = 0;
    if (lane == 0) at = atomicAdd(P.long_count, (unsigned long long)n_long);
    at = readlane_u64(at, 0);
    wave_lds_sync();
    for (int32_t i = lane; i < n_long; i += 64) P.long_list[at + i] = lbuf[i];
    wave_lds_sync();
    n_long = 0;
  };
  int64_t chunk = (int64_t)blockIdx.x * kWaves + (tid >> 6);
  int64_t cb0 = 0, cb1 = 0, cwv = 0;  // the chunk's batch range and first window
  if (chunk < P.n_chunks) {
    cb0 = first_batch(chunk);
    cb1 = first_batch(chunk + 1);
    cwv = window(cb0, cb1);
  }
  unsigned long long claim = claim_next(chunk);
  while (chunk < P.n_chunks) {
    const int64_t bw0 = cb0, bw1 = cb1;
    int64_t b = bw0;
    int64_t wv = cwv;
    int64_t r0 = uni(readlane_i64(wv, 0));  // first request of batch b
    // the next chunk: 0 = not known yet, 1 = its range loaded, 2 = its window too
    int64_t next = P.n_chunks, nb0 = 0, nb1 = 0, nwin = 0;
    int known = 0;
    if (chunk + workers < P.n_static) {  // a static successor: known now
      next = chunk + workers;
      nb0 = first_batch(next);
      nb1 = first_batch(next + 1);
      known = 1;
    }

    while (b < bw1) {
      // ---- tile: the longest run of whole batches from b within kTile slots
      const int64_t lim = min((int64_t)kTileBatches, bw1 - b);
      const int64_t ra = r0 & ~(int64_t)3;
      const int64_t rel = wv - ra;
      const uint64_t fits = __ballot(lane >= 1 && lane <= lim && rel <= kTile);
      const int32_t count = uni((int32_t)__builtin_popcountll(fits));  // a prefix of lanes
      // batches consumed by this step: the tile's, or (count == 0) the run of
      // batches from b each larger than a tile (lane j < lim: batch b+j)
      int32_t adv = count;
      if (count == 0) {
        const int64_t end = __shfl(wv, min(lane + 1, 63), 64);
        const uint64_t alone = __ballot(lane < lim && end - (wv & ~(int64_t)3) > kTile);
        adv = uni((int32_t)__builtin_ctzll(~alone));  // at least 1: batch b is one
      }
      const int64_t e = b + adv;
      const int64_t r1 = uni(readlane_i64(wv, adv));

      // next window: lane j takes offsets[e + j] from lane j + adv, or loads it
      int64_t nwv;
      {
        const int64_t sh = __shfl(wv, min(lane + adv, 63), 64);
        const bool have = lane + adv <= lim;
        nwv = have ? sh
                   : ((e < bw1 && lane <= min((int64_t)kTileBatches, bw1 - e)) ? P.off[e + lane] : 0);
      }

      if (count == 0) {
        // batches b .. e-1, each larger than a tile: listed for k_long, or
        // (Eq. 1 attribution, more than kListMin requests) with their
        // segments for k_big_sums and k_long
        list_run<MODE == MODE_ATTR>(P, b, wv, adv, lbuf, n_long, flush_long);
      } else {
        if (n_long) flush_long();  // the tile needs the share-constant area
        const int32_t lo = (int32_t)min(rel, (int64_t)kTile + 1);  // batch start, rel. to ra
        const int32_t lo_next = __shfl_down(lo, 1, 64);
        const int32_t L = (int32_t)(r1 - ra);
        const int32_t xf = (int32_t)(r0 - ra);
        const bool ne = lane < count && lo_next > lo;  // batch b+lane is nonempty
        const uint64_t ne_ball = __ballot(ne);

        // ---- held requests
        int32_t pv[kRounds][kVec], cv[kRounds][kVec], tv[kRounds][kVec];
#pragma unroll
        for (int r = 0; r < kRounds; ++r) {
          if (r * kRoundSlots + x0 < L) {
            load_slots<VEC, TEN>(P, ra + r * kRoundSlots + x0, pv[r], cv[r], tv[r]);
          } else {
#pragma unroll
            for (int q = 0; q < kVec; ++q) pv[r][q] = cv[r][q] = tv[r][q] = 0;
          }
        }

        // ---- batch-start bitmask, accumulators
        if (lane < kTileMaskWords + 2) W.mask[lane] = 0u;
        if (lane < count) W.acc[lane] = BatchAcc{0, 0, 0};
        if (RSUM && lane < count) W_r[lane] = 0ull;
        wave_lds_sync();
        if (ne) atomicOr(&W.mask[lo >> 5], 1u << (lo & 31));
        wave_lds_sync();

        uint32_t bits[kRounds], ord0[kRounds], valid[kRounds];
        {
          uint32_t before = 0;  // starts in earlier rounds
#pragma unroll
          for (int r = 0; r < kRounds; ++r) {
            const int32_t s = r * kRoundSlots + x0;
            const uint64_t w2 = ((uint64_t)W.mask[(s >> 5) + 1] << 32) | W.mask[s >> 5];
            bits[r] = (uint32_t)(w2 >> (s & 31)) & ((1u << kVec) - 1u);
            const uint32_t h = __builtin_popcount(bits[r]);
            const uint32_t hs = wave_incl_scan_u32(h);
            ord0[r] = before + hs - h;  // nonempty batches starting before slot s
            before += (uint32_t)__builtin_amdgcn_readlane((int)hs, 63);
            const int32_t a = max(xf - s, 0), z = min(L - s, kVec);
            valid[r] = z > a ? (((1u << (z - a)) - 1u) << a) & ((1u << kVec) - 1u) : 0u;
          }
        }

        // ---- batch sums: lane-local runs, added into the batch accumulators
#pragma unroll
        for (int r = 0; r < kRounds; ++r) {
          // a run ends where a batch starts at the next slot, at the last valid
          // slot, or at the end of the lane's slots
          const uint32_t ends =
              ((bits[r] >> 1) | (1u << (kVec - 1)) | (valid[r] & ~(valid[r] >> 1))) & valid[r];
          uint32_t rp = 0;
          uint64_t rcz = 0, rq = 0, rr = 0;
#pragma unroll
          for (int q = 0; q < kVec; ++q) {
            if ((valid[r] >> q) & 1u) {
              const uint32_t p = (uint32_t)pv[r][q], c = (uint32_t)cv[r][q];
              rp += p;
              rcz += (uint64_t)c + (c == 0 ? kZeroUnit : 0ull);
              rq += (uint64_t)p * p;
              if constexpr (RSUM) rr += (uint64_t)p * c;
              if ((ends >> q) & 1u) {
                const uint32_t k = ord0[r] + __builtin_popcount(bits[r] & ((2u << q) - 1u)) - 1u;
                atomicAdd((unsigned long long*)&W.acc[k].p, (unsigned long long)rp);
                atomicAdd((unsigned long long*)&W.acc[k].cz, (unsigned long long)rcz);
                atomicAdd((unsigned long long*)&W.acc[k].q, (unsigned long long)rq);
                if constexpr (RSUM) atomicAdd((unsigned long long*)&W_r[k], (unsigned long long)rr);
                rp = 0;
                rcz = 0;
                rq = 0;
                rr = 0;
              }
            }
          }
        }
        wave_lds_sync();

        {
          // ---- per batch (lane j holds batch b+j): the model
          if (lane < count) {
            const int64_t bg = b + lane;
            if (!ne) {
              empty_batch<MODE>(P, bg);
            } else {
              const uint32_t k = __builtin_popcountll(ne_ball & ((1ull << lane) - 1ull));
              const BatchAcc a = W.acc[k];
              const int64_t n = (int64_t)lo_next - lo;
              // decode iff every request processes one token over a nonzero context
              const bool prefill = (a.p != (uint64_t)n) || ((a.cz >> 48) != 0);
              if constexpr (EXT)
                ext_model(P, V, bg, n, a.p, a.cz & kCMask, a.q, W_r[k], prefill, W.k[k], &W_k4[k]);
              else if constexpr (MODE == MODE_SUMS)
                sums_out(P, bg, n, a.p, a.cz & kCMask, a.q, W_r[k], prefill);
              else
                batch_model<MODE>(P, bg, n, a.p, a.cz & kCMask, a.q, prefill, W.k[k]);
            }
          }
          wave_lds_sync();

          // ---- per request: share (+ tenant) or features
  #pragma unroll
          for (int r = 0; r < kRounds; ++r) {
            if (MODE == MODE_SUMS || r * kRoundSlots >= L) break;  // wave-uniform
            const int64_t pos = ra + r * kRoundSlots + x0;
            uint32_t kcur = 0xffffffffu;
            float kk[5] = {0.0f, 0.0f, 0.0f, 0.0f, 0.0f};
            double kd[4] = {0.0, 0.0, 0.0, 0.0};
            // PRE: the share constants of the lane's first two batches are
            // read before its first tenant-sum atomic.  A read between the
            // atomics waits for every atomic before it (LDS operations of a
            // wave complete in order), so only a third batch in the lane's
            // slots reads the table inside the loop (1% on the heavy-tailed
            // trace).
            float kb[5] = {0.0f, 0.0f, 0.0f, 0.0f, 0.0f};
            uint32_t kbi = 0xffffffffu;
            if constexpr (PRE) {
              const uint32_t nne = (uint32_t)__builtin_popcountll(ne_ball);
              const uint32_t k0 = ord0[r] + (bits[r] & 1u) - 1u;  // the lane's first batch
              if (k0 < nne) {
                kcur = k0;
                kk[0] = (float)W.k[k0][0]; kk[1] = (float)W.k[k0][1];
                kk[2] = (float)W.k[k0][2]; kk[3] = (float)W.k[k0][3];
                if constexpr (EXT) kk[4] = (float)W_k4[k0];
              }
              if (k0 + 1u < nne) {
                kbi = k0 + 1u;
                kb[0] = (float)W.k[kbi][0]; kb[1] = (float)W.k[kbi][1];
                kb[2] = (float)W.k[kbi][2]; kb[3] = (float)W.k[kbi][3];
                if constexpr (EXT) kb[4] = (float)W_k4[kbi];
              }
            }
  #pragma unroll
            for (int g = 0; g < kVec / 4; ++g) {
              float sv[4];
  #pragma unroll
              for (int qq = 0; qq < 4; ++qq) {
                const int q = 4 * g + qq;
                sv[qq] = 0.0f;
                if ((valid[r] >> q) & 1u) {
                  const uint32_t k = ord0[r] + __builtin_popcount(bits[r] & ((2u << q) - 1u)) - 1u;
                  if (k != kcur) {
                    kcur = k;
                    if (PRE && k == kbi) {
#pragma unroll
                      for (int j = 0; j < 5; ++j) kk[j] = kb[j];
                    } else {
                      kd[0] = W.k[k][0]; kd[1] = W.k[k][1]; kd[2] = W.k[k][2]; kd[3] = W.k[k][3];
                      kk[0] = (float)kd[0]; kk[1] = (float)kd[1]; kk[2] = (float)kd[2]; kk[3] = (float)kd[3];
                      if constexpr (EXT) kk[4] = (float)W_k4[k];
                    }
                  }
                  sv[qq] = request_out<MODE, HIST, SHARE>(P, kk, kd, pv[r][q], cv[r][q], s_hist_lane,
                                                          tv[r][q], pos + q);
                }
              }
              if (kAttrMode<MODE> && SHARE)
                *(v4f*)&stage[lane * kStagePitch + 4 * g] = (v4f){sv[0], sv[1], sv[2], sv[3]};
            }
            if (kAttrMode<MODE> && SHARE) store_round<VEC, true>(P, stage, ra, r * kRoundSlots, xf, L);
          }
        }
        wave_lds_sync();
      }

      b = e;
      r0 = r1;
      wv = nwv;
      // one step toward the next chunk per tile
      if (known == 1) {
        if (next < P.n_chunks) nwin = window(nb0, nb1);
        known = 2;
      } else if (known == 0) {
        next = claimed_chunk(claim);
        if (next < P.n_chunks) {
          nb0 = first_batch(next);
          nb1 = first_batch(next + 1);
        }
        known = 1;
      }
    }
    if (known == 0) {
      next = claimed_chunk(claim);
      if (next < P.n_chunks) {
        nb0 = first_batch(next);
        nb1 = first_batch(next + 1);
      }
      known = 1;
    }
    if (known == 1 && next < P.n_chunks) nwin = window(nb0, nb1);
    chunk = next;
    cb0 = nb0;
    cb1 = nb1;
    cwv = nwin;
    claim = claim_next(chunk);
  }
  if (n_long) flush_long();

  if (HIST == HIST_LDS) {
    // fold the replicas in a fixed order
    __syncthreads();
    const int32_t T = P.n_tenants;
    double* dst = P.partials + (int64_t)blockIdx.x * T;
    for (int u = tid; u < T; u += kWG) {
      double acc = s_hist[u];
      for (int r = 1; r < P.hist_rep; ++r) acc += s_hist[r * T + u];
      dst[u] = acc;
    }
  } else if (HIST == HIST_GLOBAL) {
    __syncthreads();
    cache_flush(s_hist, P.tenant_sums);
  }
}

// ------------------------------------------------------ admission queries

// Shape constants (S0..S3, and S5, S6 for the extended model) and the
// coefficients theta[phase][segment][k] of NC terms per set (5: Eq. 1, 7: the
// extended model).
template <int NC>
struct AdmitParams {
  double S[6];
  double th[4 * NC];
};

template <int NC>
__device__ __forceinline__ double admit_eq(const double* th, const double* X) {
  if constexpr (NC == 7) return eq7(th, X);
  else return eq1(th, X);
}

// One admission query per thread (Sec. 1: admission control): candidate j
// (p_j, c_j) joins batch b_j, whose exact sums and phase are given.  B' =
// B + candidate has |B|+1 requests, the sums plus the candidate's terms, and
// is a prefill batch if B is one or the candidate is prefill-type (p > 1 or
// c = 0).  Outputs (each optional): f(B'), f(B') - f(B), the candidate's
// share in B' (its own terms under B''s segment, fp64, rounded once), and
// B''s regime.  A batch index outside [0, nB) gives NaN and regime 255.
// sums: [4][nB], for the extended model [5][nB] with sum p*c.
template <int NC>
__global__ __launch_bounds__(kWG) void k_admit(const int64_t* __restrict__ sums,
                                               const uint8_t* __restrict__ phase, int64_t nB,
                                               const AdmitParams<NC> A,
                                               const int64_t* __restrict__ cand_b,
                                               const int32_t* __restrict__ cand_p,
                                               const int32_t* __restrict__ cand_c, int64_t m,
                                               float* __restrict__ t_after,
                                               float* __restrict__ delta,
                                               float* __restrict__ share,
                                               uint8_t* __restrict__ regime) {
  static_assert(NC == 5 || NC == 7, "Eq. 1 or the extended model");
  const int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (j >= m) return;
  const int64_t b = cand_b[j];
  if (b < 0 || b >= nB) {
    const float nan = __builtin_nanf("");
    if (t_after) t_after[j] = nan;
    if (delta) delta[j] = nan;
    if (share) share[j] = nan;
    if (regime) regime[j] = 255;
    return;
  }
  const int64_t n = sums[b], Ps = sums[nB + b], Cs = sums[2 * nB + b], Qs = sums[3 * nB + b];
  const int64_t Rs = NC == 7 ? sums[4 * nB + b] : 0;
  const int64_t p = cand_p[j], c = cand_c[j];
  // f(B): 0 for an empty batch
  double t0 = 0.0;
  const bool pre0 = n > 0 && phase[b] == 0;
  if (n > 0) {
    const double X[7] = {A.S[0], A.S[1] * (double)Ps, A.S[2] * (double)Cs, A.S[3] * (double)Qs,
                         (double)n * (double)n, A.S[4] * (double)Rs, A.S[5] * (double)n};
    const double* thm = A.th + ((pre0 ? 0 : 1) * 2 + 0) * NC;
    const double* thc = A.th + ((pre0 ? 0 : 1) * 2 + 1) * NC;
    const double tm = admit_eq<NC>(thm, X), tc = admit_eq<NC>(thc, X);
    t0 = (tc > tm) ? tc : tm;
  }
  // f(B')
  const int64_t n1 = n + 1;
  const int ph1 = (pre0 || p > 1 || c == 0) ? 0 : 1;
  const double X1[7] = {A.S[0], A.S[1] * (double)(Ps + p), A.S[2] * (double)(Cs + c),
                        A.S[3] * (double)(Qs + p * p), (double)n1 * (double)n1,
                        A.S[4] * (double)(Rs + p * c), A.S[5] * (double)n1};
  const double* thm = A.th + (ph1 * 2 + 0) * NC;
  const double* thc = A.th + (ph1 * 2 + 1) * NC;
  const double tm = admit_eq<NC>(thm, X1), tc = admit_eq<NC>(thc, X1);
  // Roofline max of the two segments; ties stay memory-bound.
  const int seg = (tc > tm) ? 1 : 0;
  const double t1 = seg ? tc : tm;
  // the candidate's own terms in B'
  const double x[7] = {A.S[0] / (double)n1, A.S[1] * (double)p, A.S[2] * (double)c,
                       A.S[3] * (double)(p * p), (double)n1, A.S[4] * (double)(p * c), A.S[5]};
  const double f = admit_eq<NC>(seg ? thc : thm, x);
  if (t_after) t_after[j] = (float)t1;
  if (delta) delta[j] = (float)(t1 - t0);
  if (share) share[j] = (float)f;
  if (regime) regime[j] = (uint8_t)(2 * ph1 + seg);
}

__global__ void k_zero_u64(unsigned long long* __restrict__ x, int64_t n) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) x[i] = 0ull;
}

// ------------------------------------------------------ listed batches

// Exact sums of the listed batches: workgroup w takes segments w, w +
// gridDim.x, ..., sums its requests of each in passes of kBigSub, and adds
// the totals into the batch's entry with four 64-bit atomics (integer sums:
// the order of the adds does not change them).
__global__ __launch_bounds__(kBigWG) void k_big_sums(const Params P) {
  __shared__ unsigned long long s_red[kBigWG / 64][4];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const uint64_t n_seg = *(volatile unsigned long long*)(P.claims + kSegCounter) & kSegMask;
  for (uint64_t g = blockIdx.x; g < n_seg; g += gridDim.x) {
    const uint64_t e = P.big_seg[g];
    BigEntry* E = P.big_list + (e >> 32);
    const int64_t b = E->b;
    const int64_t rs = P.off[b], re = P.off[b + 1];
    const int64_t lo = (rs & ~(int64_t)3) + (int64_t)(uint32_t)e * kBigSeg;
    const int64_t hi = min(lo + kBigSeg, re);
    uint64_t sp = 0, sc = 0, sq = 0, nz = 0;
    for (int64_t base = lo; base < hi; base += kBigSub) {
      const int64_t m = min(kBigSub, hi - base);
      const auto bp = elem_rsrc(P.p + base, m), bc = elem_rsrc(P.c + base, m);
      v4i pv[kBigPer / 4], cv[kBigPer / 4];
#pragma unroll
      for (int u = 0; u < kBigPer / 4; ++u) {
        pv[u] = load4<kNT>(bp, 4 * (tid + kBigWG * u));
        cv[u] = load4<kNT>(bc, 4 * (tid + kBigWG * u));
      }
#pragma unroll
      for (int u = 0; u < kBigPer / 4; ++u) {
        const int64_t i0 = base + 4 * (tid + kBigWG * u);
        const int32_t pa[4] = {pv[u].x, pv[u].y, pv[u].z, pv[u].w};
        const int32_t ca[4] = {cv[u].x, cv[u].y, cv[u].z, cv[u].w};
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          if (i0 + j >= rs && i0 + j < hi) {
            const uint32_t p = (uint32_t)pa[j], c = (uint32_t)ca[j];
            sp += p;
            sc += c;
            sq += (uint64_t)p * p;
            nz += c == 0 ? 1u : 0u;
          }
        }
      }
    }
    sp = wave_sum(sp);
    sc = wave_sum(sc);
    sq = wave_sum(sq);
    nz = wave_sum(nz);
    if (lane == 0) {
      s_red[wave][0] = sp;
      s_red[wave][1] = sc;
      s_red[wave][2] = sq;
      s_red[wave][3] = nz;
    }
    __syncthreads();
    if (tid < 4) {
      unsigned long long v = 0;
      for (int w = 0; w < kBigWG / 64; ++w) v += s_red[w][tid];
      if (v) atomicAdd(&E->s[tid], v);
    }
    __syncthreads();  // s_red is rewritten for the next segment
  }
}

// The batches larger than a wave tile.  Each wave of a workgroup takes
// entries of the long list in turn (long_batch); then, under Eq. 1
// attribution, workgroup w takes segments w, w + gridDim.x, ... of the
// batches listed for k_big_sums: thread 0 evaluates the batch model from the
// entry's sums (the workgroup of segment 0 writes the latency and regime),
// and the segment's shares are written and added to the tenant histogram.
// HIST_LDS: at the end the workgroup adds its histogram into row (w mod
// rows) of the tile kernel's partials (written before this launch);
// HIST_GLOBAL: its tenant cache is flushed into the output.
// Two workgroups per compute unit: a batch of two tiles held whole fits in
// 256 VGPRs.
template <int MODE, int HIST, bool SHARE>
__global__ __launch_bounds__(kWG, 2) void k_long(const Params P, const typename VarsOf<MODE>::type V,
                                              int64_t rows) {
  constexpr int VEC = kVecOf<MODE, HIST>;
  LLMV_TILE_CONSTANTS(VEC);
  constexpr bool STAGE = kAttrMode<MODE> && SHARE;
  constexpr bool TEN = HIST != HIST_NONE;
  extern __shared__ double s_hist[];  // HIST_LDS: [hist_rep][n_tenants]; HIST_GLOBAL: the cache
  __shared__ double s_k[kWaves][4];
  __shared__ double s_k4[kWaves];
  __shared__ float s_stage[STAGE ? kWaves * 64 * kStagePitch : 1];
  __shared__ float s_K[4];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const uint64_t n_long = *(volatile unsigned long long*)P.long_count;
  uint64_t n_seg = 0;
  if (MODE == MODE_ATTR && P.big_list)
    n_seg = *(volatile unsigned long long*)(P.claims + kSegCounter) & kSegMask;
  if ((uint64_t)blockIdx.x * kWaves >= n_long && blockIdx.x >= n_seg) return;  // nothing here
  const int32_t T = P.n_tenants;
  if (HIST == HIST_LDS)
    for (int u = tid; u < P.hist_rep * T; u += kWG) s_hist[u] = 0.0;
  if (HIST == HIST_GLOBAL) cache_init(s_hist);
  double* s_hist_lane = s_hist;
  if (HIST == HIST_LDS) s_hist_lane = s_hist + (lane & (P.hist_rep - 1)) * T;
  __syncthreads();

  float* stage = s_stage + (STAGE ? wave * 64 * kStagePitch : 0);
  for (uint64_t k = (uint64_t)blockIdx.x * kWaves + wave; k < n_long;
       k += (uint64_t)gridDim.x * kWaves) {
    const int64_t b = uni(P.long_list[k]);
    const int64_t rs = uni(P.off[b]), re = uni(P.off[b + 1]);
    long_batch<MODE, HIST, SHARE>(P, V, s_k[wave], &s_k4[wave], stage, b, rs, re, s_hist_lane);
  }

  if constexpr (MODE == MODE_ATTR) {
    for (uint64_t g = blockIdx.x; g < n_seg; g += gridDim.x) {
      __syncthreads();  // s_K is free (every wave is past its last use)
      const uint64_t e = P.big_seg[g];
      const BigEntry* E = P.big_list + (e >> 32);
      const int64_t b = E->b;
      const int64_t rs = P.off[b], re = P.off[b + 1];
      const int64_t lo = (rs & ~(int64_t)3) + (int64_t)(uint32_t)e * kBigSeg;
      const int64_t hi = min(lo + kBigSeg, re);
      if (tid == 0) {
        const int64_t n = re - rs;
        const uint64_t Ps = E->s[0], Cs = E->s[1], Qs = E->s[2], Zs = E->s[3];
        // decode iff every request processes one token over a nonzero context
        const bool prefill = (Ps != (uint64_t)n) || (Zs != 0);
        double kd[4];
        if ((uint32_t)e == 0) {
          batch_model<MODE_ATTR>(P, b, n, Ps, Cs, Qs, prefill, kd);
        } else {
          double t;
          eq1_batch(P.th, P.S, n, Ps, Cs, Qs, prefill, &t, kd);
        }
        for (int q = 0; q < 4; ++q) s_K[q] = (float)kd[q];
      }
      __syncthreads();
      if (!SHARE && !TEN) continue;
      const float K[4] = {s_K[0], s_K[1], s_K[2], s_K[3]};
      for (int64_t base = lo; base < hi; base += kBigSub) {
        const int64_t m = min(kBigSub, hi - base);
        const auto bp = elem_rsrc(P.p + base, m), bc = elem_rsrc(P.c + base, m);
        const auto bt = elem_rsrc(TEN ? P.tenant + base : P.p + base, m);
        v4i pv[kBigPer / 4], cv[kBigPer / 4], tv[kBigPer / 4];
#pragma unroll
        for (int u = 0; u < kBigPer / 4; ++u) {
          pv[u] = load4<kNT>(bp, 4 * (tid + kBigWG * u));
          cv[u] = load4<kNT>(bc, 4 * (tid + kBigWG * u));
          if (TEN) tv[u] = load4<kNT>(bt, 4 * (tid + kBigWG * u));
        }
#pragma unroll
        for (int u = 0; u < kBigPer / 4; ++u) {
          const int64_t i0 = base + 4 * (tid + kBigWG * u);
          const int32_t pa[4] = {pv[u].x, pv[u].y, pv[u].z, pv[u].w};
          const int32_t ca[4] = {cv[u].x, cv[u].y, cv[u].z, cv[u].w};
          const int32_t ta[4] = {TEN ? tv[u].x : 0, TEN ? tv[u].y : 0, TEN ? tv[u].z : 0,
                                 TEN ? tv[u].w : 0};
          float sv[4];
          uint32_t valid = 0;
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            sv[j] = 0.0f;
            if (i0 + j >= rs && i0 + j < hi) {
              valid |= 1u << j;
              sv[j] = share_of(K, pa[j], ca[j]);
              if (HIST == HIST_LDS) atomicAdd(s_hist_lane + ta[j], (double)sv[j]);
              if (HIST == HIST_GLOBAL) cache_add(s_hist, ta[j], (double)sv[j], P.tenant_sums);
            }
          }
          if (SHARE) {
            if (valid == 0xFu) {
              __builtin_nontemporal_store((v4f){sv[0], sv[1], sv[2], sv[3]}, (v4f*)(P.share + i0));
            } else {
#pragma unroll
              for (int j = 0; j < 4; ++j)
                if ((valid >> j) & 1u) P.share[i0 + j] = sv[j];
            }
          }
        }
      }
    }
  }

  if (HIST == HIST_LDS) {
    // the replicas folded, the nonzero entries added with fp64 atomics
    __syncthreads();
    double* row = P.partials + (int64_t)(blockIdx.x % rows) * T;
    for (int u = tid; u < T; u += kWG) {
      double acc = s_hist[u];
      for (int r = 1; r < P.hist_rep; ++r) acc += s_hist[r * T + u];
      if (acc != 0.0) unsafeAtomicAdd(row + u, acc);
    }
  } else if (HIST == HIST_GLOBAL) {
    __syncthreads();
    cache_flush(s_hist, P.tenant_sums);
  }
}

// ------------------------------------------------------ tenant reductions

// out[u] = sum over rows w of part[w][u], folded in a fixed order.  One
// block of kReduceWaves waves per kTenantChunk tenants; lane l of a wave
// takes tenant l % kTenantChunk and row offset l / kTenantChunk, so one load
// instruction reads kReduceRows rows of 128 contiguous bytes.  Wave v sums
// rows v*kReduceRows + l / kTenantChunk + k*kReduceStep (k = 0, 1, ...) into
// eight independent partial sums (up to 8*kReduceStep rows in one round of
// loads); the row offsets are then added by lane shuffles and the waves'
// sums in wave order.
constexpr int kReduceWaves = 16;
constexpr int kReduceRows = 64 / kTenantChunk;                 // rows per wave load
constexpr int kReduceStep = kReduceWaves * kReduceRows;        // rows per block load
static_assert(64 % kTenantChunk == 0 && kTenantChunk * 8 == 128, "128-byte row segments");

__global__ __launch_bounds__(64 * kReduceWaves) void k_tenant_reduce(
    const double* __restrict__ part, int rows, int T, double* __restrict__ out) {
  __shared__ double red[kReduceWaves][kTenantChunk];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int j = lane % kTenantChunk, rs = lane / kTenantChunk;
  const int u = blockIdx.x * kTenantChunk + j;
  double acc = 0.0;
  if (u < T) {
    double a8[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    int w = wave * kReduceRows + rs;
    for (; w + 7 * kReduceStep < rows; w += 8 * kReduceStep) {
#pragma unroll
      for (int i = 0; i < 8; ++i) a8[i] += part[(int64_t)(w + i * kReduceStep) * T + u];
    }
#pragma unroll
    for (int i = 0; i < 8; ++i)
      if (w + i * kReduceStep < rows) a8[i] += part[(int64_t)(w + i * kReduceStep) * T + u];
#pragma unroll
    for (int i = 0; i < 8; ++i) acc += a8[i];
  }
  // the row offsets of one tenant: lanes j, j + 16, j + 32, j + 48
  static_assert(kReduceRows == 4, "two shuffle steps");
  acc += __shfl_xor(acc, 16, 64);
  acc += __shfl_xor(acc, 32, 64);
  if (rs == 0) red[wave][j] = acc;
  __syncthreads();
  if (wave == 0 && rs == 0 && u < T) {
    double t = red[0][j];
    for (int v = 1; v < kReduceWaves; ++v) t += red[v][j];
    out[u] = t;
  }
}

// Standalone tenant sums of given fp32 shares: a grid-stride pass per
// workgroup over a contiguous slice into an LDS histogram (or global atomics).
template <int HIST>
__global__ __launch_bounds__(kWG) void k_tenant_hist(const int32_t* __restrict__ tenant,
                                                     const float* __restrict__ share,
                                                     int64_t n, int32_t T,
                                                     double* __restrict__ partials,
                                                     double* __restrict__ out) {
  extern __shared__ double s_hist[];
  if (HIST == HIST_LDS)
    for (int u = threadIdx.x; u < T; u += kWG) s_hist[u] = 0.0;
  else
    cache_init(s_hist);
  __syncthreads();
  const int64_t per = (n + gridDim.x - 1) / gridDim.x;
  const int64_t lo = per * blockIdx.x, hi = min(n, lo + per);
  for (int64_t i = lo + threadIdx.x; i < hi; i += kWG) {
    const double v = (double)share[i];
    if (HIST == HIST_LDS) atomicAdd(s_hist + tenant[i], v);
    else cache_add(s_hist, tenant[i], v, out);
  }
  __syncthreads();
  if (HIST == HIST_LDS) {
    for (int u = threadIdx.x; u < T; u += kWG) partials[(int64_t)blockIdx.x * T + u] = s_hist[u];
  } else {
    cache_flush(s_hist, out);
  }
}

// --------------------------------------------------------------- validate

__global__ void k_validate(const int64_t* __restrict__ off, int64_t nB, int64_t N,
                           const int32_t* __restrict__ p, const int32_t* __restrict__ c,
                           const int32_t* __restrict__ t, int32_t T, int batch_max,
                           int p_max, int* __restrict__ flag) {
  const int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  int bad = 0;
  if (gid == 0 && (off[0] != 0 || off[nB] != N)) bad = 1;
  for (int64_t b = gid; b < nB; b += stride) {
    const int64_t d = off[b + 1] - off[b];
    if (d < 0 || d > batch_max) bad = 1;
  }
  for (int64_t i = gid; i < N; i += stride) {
    if (p[i] < 1 || p[i] > p_max || c[i] < 0) bad = 1;
    if (t && (t[i] < 0 || t[i] >= T)) bad = 1;
  }
  if (bad) atomicOr(flag, 1);
}

__global__ void k_zero_i32(int* __restrict__ v, int n) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) v[i] = 0;
}

}  // namespace llmv
