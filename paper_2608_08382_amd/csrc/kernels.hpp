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
//    handled by the wave in two passes.
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
#ifndef LLMV_STATIC_EIGHTHS
#define LLMV_STATIC_EIGHTHS 6
#endif
#ifndef LLMV_DYN_PER_WORKER
#define LLMV_DYN_PER_WORKER 8
#endif
constexpr int kStaticEighths = LLMV_STATIC_EIGHTHS;  // requests in static chunks, in eighths
constexpr int kDynPerWorker = LLMV_DYN_PER_WORKER;   // claimed chunks per wave worker, at most
// For wave tiles of `cap` request slots:
constexpr int64_t min_chunk(int64_t cap) { return 4 * cap; }       // requests per claimed chunk, at least
constexpr int64_t min_dyn_share(int64_t cap) { return 32 * cap; }  // per worker, for claimed chunks
constexpr int64_t piece(int64_t cap) { return 16 * cap; }          // requests per static piece

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
// (Eq. 1 attribution without the tenant cache: 28 slots, about 2% on the
// heavy-tailed trace; the feature rows and batch sums, about 1%); the narrow
// one for the extended model and the tenant cache, where the wide tile's
// registers (up to 255 VGPRs) cost more than its longer tiles gain.
__host__ __device__ constexpr bool wide_tile(int mode, int hist) {
  return (mode == MODE_ATTR && hist != HIST_GLOBAL) || mode == MODE_FEAT || mode == MODE_SUMS;
}
template <int MODE, int HIST>
constexpr int kVecOf = wide_tile(MODE, HIST) ? kVecWide : kVecNarrow;
__host__ __device__ constexpr int64_t tile_cap(int mode, int hist) {
  return 64 * (wide_tile(mode, hist) ? kVecWide : kVecNarrow);
}

struct Params {
  const int64_t* off;
  const int32_t* p;
  const int32_t* c;
  const int32_t* tenant;
  int64_t nB, N;
  const int64_t* wg_first;  // [n_chunks+1] first batch of each chunk
  unsigned long long* claims;  // chunk claim counter
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
// (w < n_chunks), wg_first[n_chunks] = nB; clears the claim counter.
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
    *claims = 0ull;
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
// stays below the count's bits.  (big_batch keeps them apart: a batch
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

__device__ __forceinline__ uint64_t wave_sum(uint64_t x) {
  for (int m = 32; m >= 1; m >>= 1) x += __shfl_xor(x, m, 64);
  return x;
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
// Only slots in [xf, L) are written.
template <int VEC>
__device__ __forceinline__ void store_round(const Params& P, float* stage, int64_t ra, int32_t s0,
                                            int32_t xf, int32_t L) {
  LLMV_TILE_CONSTANTS(VEC);
  const int lane = threadIdx.x & 63;
  wave_lds_sync();
#pragma unroll
  for (int g = 0; g < kVec / 4; ++g) {
    const int32_t e = 256 * g + 4 * lane;  // slot within the round
    const int32_t x = s0 + e;              // slot within the tile
    const float* src = &stage[(e / kVec) * kStagePitch + (e % kVec)];
    if (x >= xf && x + 4 <= L) {
      __builtin_nontemporal_store(*(const v4f*)src, (v4f*)(P.share + ra + x));  // not re-read
    } else {
#pragma unroll
      for (int q = 0; q < 4; ++q)
        if (x + q >= xf && x + q < L) P.share[ra + x + q] = src[q];
    }
  }
  wave_lds_sync();
}

// One batch too large for a wave tile: two passes over its requests by the
// whole wave (the second pass mostly hits in L2).
template <int MODE, int HIST, bool SHARE>
__device__ void big_batch(const Params& P, const typename VarsOf<MODE>::type& V,
                          WaveLds<kVecOf<MODE, HIST>>& W, double* wk4, float* stage, int64_t bg,
                          int64_t rs, int64_t re, double* s_hist) {
  constexpr int VEC = kVecOf<MODE, HIST>;
  LLMV_TILE_CONSTANTS(VEC);
  const int lane = threadIdx.x & 63;
  const int64_t ra = rs & ~(int64_t)3;
  // Sums over up to 2^22 requests: sum c reaches 2^53, so the tile path's
  // packed (sum c, zero count) word does not apply; a zero context is
  // recorded as a flag of its own.
  uint64_t sp = 0, sc = 0, sq = 0, sr = 0;
  bool zc = false;  // this lane saw a request with c == 0
  int32_t pv[kVec], cv[kVec], tv[kVec];
  for (int64_t base = ra; base < re; base += kRoundSlots) {
    const int64_t x = base + lane * kVec;
    load_slots<VEC, false>(P, x, pv, cv, tv);
#pragma unroll
    for (int q = 0; q < kVec; ++q) {
      if (x + q >= rs && x + q < re) {
        const uint32_t p = (uint32_t)pv[q], c = (uint32_t)cv[q];
        sp += p;
        sc += c;
        zc |= c == 0;
        sq += (uint64_t)p * p;
        if constexpr (kCrossSum<MODE>) sr += (uint64_t)p * c;
      }
    }
  }
  sp = wave_sum(sp);
  sc = wave_sum(sc);
  sq = wave_sum(sq);
  if constexpr (kCrossSum<MODE>) sr = wave_sum(sr);
  const int64_t n = re - rs;
  // decode iff every request processes one token over a nonzero context
  const bool prefill = (sp != (uint64_t)n) || (__ballot(zc) != 0);
  if constexpr (MODE == MODE_SUMS) {
    if (lane == 0) sums_out(P, bg, n, sp, sc, sq, sr, prefill);
    return;
  }
  if (lane == 0) {
    if constexpr (MODE == MODE_EXT)
      ext_model(P, V, bg, n, sp, sc, sq, sr, prefill, W.k[0], wk4);
    else
      batch_model<MODE>(P, bg, n, sp, sc, sq, prefill, W.k[0]);
  }
  wave_lds_sync();
  const double kd[4] = {W.k[0][0], W.k[0][1], W.k[0][2], W.k[0][3]};
  const float k[5] = {(float)kd[0], (float)kd[1], (float)kd[2], (float)kd[3],
                      MODE == MODE_EXT ? (float)wk4[0] : 0.0f};
  for (int64_t base = ra; base < re; base += kRoundSlots) {
    const int64_t x = base + lane * kVec;
    load_slots<VEC, HIST != HIST_NONE>(P, x, pv, cv, tv);
#pragma unroll
    for (int g = 0; g < kVec / 4; ++g) {
      float sv[4];
#pragma unroll
      for (int qq = 0; qq < 4; ++qq) {
        const int q = 4 * g + qq;
        sv[qq] = 0.0f;
        if (x + q >= rs && x + q < re)
          sv[qq] = request_out<MODE, HIST, SHARE>(P, k, kd, pv[q], cv[q], s_hist, tv[q], x + q);
      }
      if (kAttrMode<MODE> && SHARE)
        *(v4f*)&stage[lane * kStagePitch + 4 * g] = (v4f){sv[0], sv[1], sv[2], sv[3]};
    }
    if (kAttrMode<MODE> && SHARE)
      store_round<VEC>(P, stage, ra, (int32_t)(base - ra), (int32_t)(rs - ra), (int32_t)(re - ra));
  }
  wave_lds_sync();
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
  // claim k of this launch names chunk n_static + k; past the last chunk, stop
  auto claimed_chunk = [&](unsigned long long cl) {
    const uint64_t k = readlane_u64((uint64_t)cl, 0) - P.claim_base;
    return (dyn && k < (uint64_t)(P.n_chunks - P.n_static)) ? P.n_static + (int64_t)k : P.n_chunks;
  };
  auto claim_next = [&](int64_t ch) {
    unsigned long long cl = ~0ull;
    if (dyn && ch < P.n_chunks && ch + workers >= P.n_static && lane == 0)
      cl = atomicAdd(P.claims, 1ull);
    return cl;
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
      const int32_t adv = count > 0 ? count : 1;  // batches consumed by this step
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
        big_batch<MODE, HIST, SHARE>(P, V, W, W_k4, stage, b, r0, r1, s_hist_lane);
      } else {
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
                    kd[0] = W.k[k][0]; kd[1] = W.k[k][1]; kd[2] = W.k[k][2]; kd[3] = W.k[k][3];
                    kk[0] = (float)kd[0]; kk[1] = (float)kd[1]; kk[2] = (float)kd[2]; kk[3] = (float)kd[3];
                    if constexpr (EXT) kk[4] = (float)W_k4[k];
                  }
                  sv[qq] = request_out<MODE, HIST, SHARE>(P, kk, kd, pv[r][q], cv[r][q], s_hist_lane,
                                                          tv[r][q], pos + q);
                }
              }
              if (kAttrMode<MODE> && SHARE)
                *(v4f*)&stage[lane * kStagePitch + 4 * g] = (v4f){sv[0], sv[1], sv[2], sv[3]};
            }
            if (kAttrMode<MODE> && SHARE) store_round<VEC>(P, stage, ra, r * kRoundSlots, xf, L);
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
