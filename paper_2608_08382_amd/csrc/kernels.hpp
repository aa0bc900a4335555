// kernels.hpp -- gfx950 kernels for batched LLMVisor latency attribution.
//
// The method (LLMVisor Sec. 2.1, Eq. 1; Sec. 2 "Problem formulation"):
// per batch, exact sums P = sum p, C = sum c, Q = sum p^2 and the batch phase;
// Eq. 1 with the phase's two coefficient sets (memory-bound, compute-bound);
// the larger one is the batch latency; each request's share is its own terms
// of the chosen set; tenant usage is the sum of its requests' shares.
//
// Work decomposition (memory-bound ragged reduction, no dense contraction):
//  * k_partition: splits the batch list into one contiguous range per
//    persistent workgroup, balanced by request count.
//  * k_tiles: each workgroup walks its range in tiles.  A tile is a run of
//    whole batches whose requests fit in kCap slots (greedy), so every
//    request is read from HBM once, held in registers while its batch totals
//    are formed, and its share written once.  Batch totals come from
//    prefix sums: a wave-level DPP scan per 256-request round, carried across
//    rounds and waves; the prefix at a batch's first request is subtracted
//    from the prefix at its last.  Batches that do not fit in a tile go
//    through a slower two-pass path inside the same workgroup.
//  * Tenant sums accumulate in an fp64 LDS histogram per workgroup, flushed
//    once to a [grid][n_tenants] partial array that k_tenant_reduce folds in
//    a fixed order.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace llmv {

constexpr int kWG = 256;                     // threads per workgroup
constexpr int kWaves = kWG / 64;             // wave64
constexpr int kVec = 16;                     // consecutive requests held per lane
constexpr int kWaveSpan = 64 * kVec;         // 1024 requests per wave
constexpr int kCap = kWaveSpan * kWaves;     // 4096 request slots per tile
constexpr int kMaskWords = kCap / 32;        // batch-start bitmask of a tile
constexpr int kWindow = 256;                 // offsets examined per tile
constexpr int kMaxTileBatches = kWindow - 1; // 255 batches per tile
constexpr int kHistLdsMax = 4096;                // tenants held in an LDS histogram
constexpr int kMaxGrid = 2048;                   // persistent workgroups, upper bound
constexpr int kReduceSplit = 16;                 // row blocks in k_tenant_reduce
constexpr int kTenantChunk = 64;                 // tenants per k_tenant_reduce block

enum { MODE_ATTR = 0, MODE_FEAT = 1 };

// Native vectors: 16-byte global loads / stores (dwordx4).
typedef int32_t v4i __attribute__((ext_vector_type(4)));
typedef float v4f __attribute__((ext_vector_type(4)));
enum { HIST_NONE = 0, HIST_LDS = 1, HIST_GLOBAL = 2 };

struct Params {
  const int64_t* off;
  const int32_t* p;
  const int32_t* c;
  const int32_t* tenant;
  int64_t nB, N;
  const int64_t* wg_first;  // [grid+1] first batch of each workgroup
  float* latency;           // [nB] or null
  uint8_t* regime;          // [nB] or null
  float* share;             // [N] or null
  double* partials;         // [grid][n_tenants] (HIST_LDS)
  double* tenant_sums;      // [n_tenants] (HIST_GLOBAL: atomics target)
  float* x_req;             // [5][N] (MODE_FEAT) or null
  double* x_batch;          // [5][nB] (MODE_FEAT) or null
  int32_t n_tenants;
  double S[4];              // shape constants
  double th[20];            // theta[phase][segment][k]
};

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

// Eq. 1 with one coefficient set, terms added in order k = 0..4.
__device__ __forceinline__ double eq1(const double* th, const double X[5]) {
  double acc = th[0] * X[0];
  acc = acc + th[1] * X[1];
  acc = acc + th[2] * X[2];
  acc = acc + th[3] * X[3];
  acc = acc + th[4] * X[4];
  return acc;
}

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
    k[0] = P.S[0] / (double)n;
    k[1] = (double)n;
    return;
  }
  const int phase = prefill ? 0 : 1;
  const double* thm = P.th + (phase * 2 + 0) * 5;
  const double* thc = P.th + (phase * 2 + 1) * 5;
  const double tm = eq1(thm, X);
  const double tc = eq1(thc, X);
  // Roofline max of the two segments; ties stay memory-bound.
  const int seg = (tc > tm) ? 1 : 0;
  if (P.latency) P.latency[bg] = (float)(seg ? tc : tm);
  if (P.regime) P.regime[bg] = (uint8_t)(2 * phase + seg);
  const double* th = seg ? thc : thm;
  k[0] = th[0] * (P.S[0] / (double)n) + th[4] * (double)n;
  k[1] = th[1] * P.S[1];
  k[2] = th[2] * P.S[2];
  k[3] = th[3] * P.S[3];
}

template <int MODE>
__device__ __forceinline__ void empty_batch(const Params& P, int64_t bg) {
  if (MODE == MODE_FEAT) {
    if (P.x_batch)
      for (int q = 0; q < 5; ++q) P.x_batch[q * P.nB + bg] = 0.0;
  } else {
    if (P.latency) P.latency[bg] = 0.0f;
    if (P.regime) P.regime[bg] = 255;
  }
}

// Per-request epilogue: share (+ tenant histogram) or the feature row.
template <int MODE, int HIST, bool SHARE>
__device__ __forceinline__ double request_out(const Params& P, const double* k, int32_t p,
                                              int32_t c, double* s_hist, int32_t t,
                                              int64_t i, bool store_scalar) {
  const double pd = (double)p;
  if (MODE == MODE_FEAT) {
    if (P.x_req) {
      const int64_t N = P.N;
      P.x_req[0 * N + i] = (float)k[0];
      P.x_req[1 * N + i] = (float)(P.S[1] * pd);
      P.x_req[2 * N + i] = (float)(P.S[2] * (double)c);
      P.x_req[3 * N + i] = (float)(P.S[3] * (pd * pd));
      P.x_req[4 * N + i] = (float)k[1];
    }
    return 0.0;
  }
  const double s = k[0] + k[1] * pd + k[2] * (double)c + k[3] * (pd * pd);
  if (SHARE && store_scalar) P.share[i] = (float)s;
  if (HIST == HIST_LDS) atomicAdd(s_hist + t, s);
  if (HIST == HIST_GLOBAL) unsafeAtomicAdd(P.tenant_sums + t, s);
  return s;
}

// ------------------------------------------------------------ partition

// wg_first[w] = first batch whose start offset is >= w*step (w < grid),
// wg_first[grid] = nB.  Also clears the reduction counters and, for the
// global-atomics tenant path, the tenant sums.
__global__ void k_partition(const int64_t* __restrict__ off, int64_t nB, int64_t step,
                            int grid, int64_t* __restrict__ wg_first,
                            uint32_t* __restrict__ cnt, int n_cnt,
                            double* __restrict__ zero_buf, int64_t n_zero) {
  const int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t b = gid; b <= nB; b += stride) {
    const int64_t wlo = (b == 0) ? 0 : off[b - 1] / step + 1;
    const int64_t whi = (b == nB) ? (int64_t)grid - 1
                                  : min((int64_t)grid - 1, off[b] / step);
    for (int64_t w = wlo; w <= whi; ++w) wg_first[w] = b;
  }
  if (gid == 0) wg_first[grid] = nB;
  for (int64_t i = gid; i < n_cnt; i += stride) cnt[i] = 0;
  for (int64_t i = gid; i < n_zero; i += stride) zero_buf[i] = 0.0;
}

// ------------------------------------------------------------ big batches

struct BigRed {
  uint64_t p, c, q, pre;
};

// One batch too large for a tile, processed by the whole workgroup in two
// passes over its requests (the second pass mostly hits in L2).
template <int MODE, int HIST, bool SHARE>
__device__ void big_batch(const Params& P, int64_t bg, int64_t rs, int64_t re,
                          double* s_hist, double (*s_k)[4], BigRed* s_red) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  uint64_t sp = 0, sc = 0, sq = 0, pre = 0;
  for (int64_t i = rs + tid; i < re; i += kWG) {
    const int32_t p = P.p[i], c = P.c[i];
    sp += (uint64_t)p;
    sc += (uint64_t)c;
    sq += (uint64_t)((int64_t)p * p);
    pre += (p > 1 || c == 0) ? 1 : 0;
  }
  sp = wave_sum_u64(sp);
  sc = wave_sum_u64(sc);
  sq = wave_sum_u64(sq);
  pre = wave_sum_u64(pre);
  if (lane == 0) s_red[wave] = BigRed{sp, sc, sq, pre};
  __syncthreads();
  if (tid == 0) {
    BigRed t{0, 0, 0, 0};
    for (int w = 0; w < kWaves; ++w) {
      t.p += s_red[w].p;
      t.c += s_red[w].c;
      t.q += s_red[w].q;
      t.pre += s_red[w].pre;
    }
    batch_model<MODE>(P, bg, re - rs, t.p, t.c, t.q, t.pre > 0, s_k[0]);
  }
  __syncthreads();
  const double k[4] = {s_k[0][0], s_k[0][1], s_k[0][2], s_k[0][3]};
  for (int64_t i = rs + tid; i < re; i += kWG) {
    const int32_t t = (HIST != HIST_NONE) ? P.tenant[i] : 0;
    request_out<MODE, HIST, SHARE>(P, k, P.p[i], P.c[i], s_hist, t, i, true);
  }
  __syncthreads();
}

// ----------------------------------------------------------------- tiles

// Running prefix of one request position, relative to the start of its
// lane's run of kVec requests.  id = lane + 64*wave locates the lane base.
struct LanePref {
  uint32_t p;   // sum p
  uint32_t id;
  uint64_t cz;  // sum c (bits 0..47) | count of c == 0 (bits 48..63)
  uint64_t q;   // sum p^2
};

struct Sums {
  uint64_t p, cz, q;
};

constexpr uint64_t kZeroUnit = 1ull << 48;
constexpr uint64_t kCMask = kZeroUnit - 1;

__device__ __forceinline__ uint32_t lds_popc_below(const uint32_t* mask, int pos) {
  // set bits of the tile bitmask at positions < pos, pos < 32 of its word
  return __builtin_popcount(mask[pos >> 5] & ((1u << (pos & 31)) - 1u));
}

template <int MODE, int HIST, bool SHARE>
__global__ __launch_bounds__(kWG) void k_tiles(const Params P) {
  extern __shared__ double s_hist[];       // [n_tenants] when HIST_LDS
  __shared__ int32_t s_lo[kWindow];        // batch starts relative to the tile base
  __shared__ uint32_t s_mask[kMaskWords + 1];  // bit x: a nonempty batch starts at x
  __shared__ uint64_t s_ball[kWaves];      // nonempty flags of the window's batches
  __shared__ LanePref s_xs[kWindow];       // prefix before each batch's first request
  __shared__ LanePref s_xe[kWindow];       // prefix through each batch's last request
  __shared__ Sums s_lb[kWG];               // exclusive prefix of each lane within its wave
  __shared__ Sums s_wt[kWaves];            // wave totals
  __shared__ double s_k[kWindow][4];       // per nonempty batch: share / feature constants
  __shared__ BigRed s_red[kWaves];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int64_t N = P.N;
  const int32_t x0 = wave * kWaveSpan + lane * kVec;  // first slot of this lane

  if (HIST == HIST_LDS)
    for (int u = tid; u < P.n_tenants; u += kWG) s_hist[u] = 0.0;

  const int64_t bw0 = P.wg_first[blockIdx.x];
  const int64_t bw1 = P.wg_first[blockIdx.x + 1];
  int64_t b = bw0;
  int64_t r0 = 0;  // first request of batch b
  int64_t wv = 0;  // offsets[b + tid] (window)
  if (b < bw1) {
    r0 = P.off[b];
    if (tid <= min((int64_t)kMaxTileBatches, bw1 - b)) wv = P.off[b + tid];
  }
  __syncthreads();

  while (b < bw1) {
    // ---- A: window -> s_lo; batches b .. b+count-1 end within kCap slots
    const int64_t lim = min((int64_t)kMaxTileBatches, bw1 - b);
    const int64_t ra = r0 & ~(int64_t)3;  // 16-byte aligned tile base
    int pred = 0;
    if (tid <= lim) {
      const int64_t rel = wv - ra;
      s_lo[tid] = (int32_t)min(rel, (int64_t)kCap + 1);
      pred = (tid >= 1 && rel <= kCap) ? 1 : 0;
    }
    if (tid <= kMaskWords) s_mask[tid] = 0u;
    const int count = __syncthreads_count(pred);

    if (count == 0) {
      const int64_t re = P.off[b + 1];
      big_batch<MODE, HIST, SHARE>(P, b, r0, re, s_hist, s_k, s_red);
      b += 1;
      r0 = re;
      if (b < bw1 && tid <= min((int64_t)kMaxTileBatches, bw1 - b)) wv = P.off[b + tid];
      continue;
    }

    const int64_t e = b + count;
    const int32_t L = s_lo[count];  // tile end relative to ra
    const int32_t xf = s_lo[0];     // first tile request relative to ra (0..3)
    const int64_t r1 = ra + L;

    // ---- B: batch-start bits, nonempty ballots; loads of this lane's slots
    bool ne = false;
    if (tid < count) {
      const int32_t lo = s_lo[tid];
      ne = s_lo[tid + 1] > lo;
      if (ne) atomicOr(&s_mask[lo >> 5], 1u << (lo & 31));
    }
    const uint64_t ball = __ballot(ne);
    if (lane == 0) s_ball[wave] = ball;

    int64_t nwv = 0;  // window of the next tile, in flight meanwhile
    if (e < bw1 && tid <= min((int64_t)kMaxTileBatches, bw1 - e)) nwv = P.off[e + tid];

    int32_t pv[kVec], cv[kVec], tv[kVec];
#pragma unroll
    for (int q = 0; q < kVec; ++q) pv[q] = cv[q] = tv[q] = 0;
    if (x0 < L) {
      const int32_t* pb = P.p + ra;
      const int32_t* cb = P.c + ra;
      const int32_t* tb = P.tenant + ra;
      if (ra + x0 + kVec <= N) {
#pragma unroll
        for (int g = 0; g < kVec / 4; ++g) {
          const v4i a = *(const v4i*)(pb + x0 + 4 * g);
          const v4i d = *(const v4i*)(cb + x0 + 4 * g);
          pv[4 * g] = a.x; pv[4 * g + 1] = a.y; pv[4 * g + 2] = a.z; pv[4 * g + 3] = a.w;
          cv[4 * g] = d.x; cv[4 * g + 1] = d.y; cv[4 * g + 2] = d.z; cv[4 * g + 3] = d.w;
          if (HIST != HIST_NONE) {
            const v4i t = *(const v4i*)(tb + x0 + 4 * g);
            tv[4 * g] = t.x; tv[4 * g + 1] = t.y; tv[4 * g + 2] = t.z; tv[4 * g + 3] = t.w;
          }
        }
      } else {
#pragma unroll
        for (int q = 0; q < kVec; ++q) {
          if (ra + x0 + q < N) {
            pv[q] = pb[x0 + q];
            cv[q] = cb[x0 + q];
            if (HIST != HIST_NONE) tv[q] = tb[x0 + q];
          }
        }
      }
    }
    __syncthreads();

    // ---- C: ordinal of each held request's batch among the tile's
    // nonempty batches, from the batch-start bitmask
    const uint32_t w0 = s_mask[x0 >> 5];
    const uint32_t bits = (w0 >> (x0 & 16)) & 0xffffu;  // starts at x0 .. x0+15
    const uint32_t next_bit = (s_mask[(x0 + kVec) >> 5] >> ((x0 + kVec) & 31)) & 1u;
    uint32_t wave_base = 0;  // starts in the slots of earlier waves
    if (wave > 0) {
      uint32_t cnt = 0;
      if (lane < 32 * wave) cnt += __builtin_popcount(s_mask[lane]);
      if (lane + 64 < 32 * wave) cnt += __builtin_popcount(s_mask[lane + 64]);
      for (int m = 32; m >= 1; m >>= 1) cnt += __shfl_xor(cnt, m, 64);
      wave_base = cnt;
    }
    const uint32_t h = __builtin_popcount(bits);
    uint32_t hs = h;  // inclusive wave scan of the lanes' start counts
    hs += dpp_u32<0x111, 0xf>(hs);
    hs += dpp_u32<0x112, 0xf>(hs);
    hs += dpp_u32<0x114, 0xf>(hs);
    hs += dpp_u32<0x118, 0xf>(hs);
    hs += dpp_u32<0x142, 0xa>(hs);
    hs += dpp_u32<0x143, 0xc>(hs);
    const uint32_t ord0 = wave_base + hs - h;  // starts before x0

    // ---- D: one pass over the lane's requests: lane-relative prefixes at
    // batch starts and ends, lane totals
    uint32_t ords[kVec / 4];  // 8-bit ordinal per held request
    uint32_t valid = 0;
    uint32_t ap = 0;
    uint64_t acz = 0, aq = 0;
    {
      uint32_t ord = ord0;
#pragma unroll
      for (int q = 0; q < kVec; ++q) {
        const int32_t x = x0 + q;
        const bool v = (x >= xf) && (x < L);
        const uint32_t st = (bits >> q) & 1u;
        const uint32_t en = ((q + 1 < kVec ? (bits >> (q + 1)) : next_bit) & 1u) | (x + 1 == L);
        ord += st;
        const uint32_t k = ord - 1u;
        if (q % 4 == 0) ords[q / 4] = 0;
        ords[q / 4] |= (k & 0xffu) << (8 * (q % 4));
        if (v) {
          valid |= 1u << q;
          const uint32_t p = (uint32_t)pv[q];
          const uint32_t c = (uint32_t)cv[q];
          if (st) s_xs[k] = LanePref{ap, (uint32_t)tid, acz, aq};
          ap += p;
          acz += (uint64_t)c + (c == 0 ? kZeroUnit : 0ull);
          aq += (uint64_t)p * p;
          if (en) s_xe[k] = LanePref{ap, (uint32_t)tid, acz, aq};
        }
      }
    }
    {
      const uint64_t sp = wave_incl_scan((uint64_t)ap);
      const uint64_t scz = wave_incl_scan(acz);
      const uint64_t sq = wave_incl_scan(aq);
      s_lb[tid] = Sums{sp - ap, scz - acz, sq - aq};
      if (lane == 63) s_wt[wave] = Sums{sp, scz, sq};
    }
    __syncthreads();

    // ---- E: per batch: totals from prefix differences, then the model
    if (tid < count) {
      const int j = tid;
      const int64_t bg = b + j;
      if (!ne) {
        empty_batch<MODE>(P, bg);
      } else {
        uint32_t k = __builtin_popcountll(s_ball[wave] & ((1ull << lane) - 1ull));
        for (int w = 0; w < wave; ++w) k += __builtin_popcountll(s_ball[w]);
        const LanePref xs = s_xs[k], xe = s_xe[k];
        const Sums ls = s_lb[xs.id], le = s_lb[xe.id];
        uint64_t p0 = xs.p + ls.p, cz0 = xs.cz + ls.cz, q0 = xs.q + ls.q;
        uint64_t p1 = xe.p + le.p, cz1 = xe.cz + le.cz, q1 = xe.q + le.q;
        for (uint32_t w = 0; w < (uint32_t)kWaves; ++w) {
          const Sums t = s_wt[w];
          if (w < (xs.id >> 6)) { p0 += t.p; cz0 += t.cz; q0 += t.q; }
          if (w < (xe.id >> 6)) { p1 += t.p; cz1 += t.cz; q1 += t.q; }
        }
        const int64_t n = (int64_t)s_lo[j + 1] - s_lo[j];
        const uint64_t Ps = p1 - p0, CZ = cz1 - cz0, Qs = q1 - q0;
        // decode iff every request processes one token over a nonzero context
        const bool prefill = (Ps != (uint64_t)n) || ((CZ >> 48) != 0);
        batch_model<MODE>(P, bg, n, Ps, CZ & kCMask, Qs, prefill, s_k[k]);
      }
    }
    __syncthreads();

    // ---- F: per request: share (+ tenant) or features
    if (valid) {
      const int64_t pos = ra + x0;
      uint32_t kcur = 0xffffffffu;
      double kk[4] = {0.0, 0.0, 0.0, 0.0};
      const bool full = valid == 0xffffu;
#pragma unroll
      for (int g = 0; g < kVec / 4; ++g) {
        float sv[4];
#pragma unroll
        for (int qq = 0; qq < 4; ++qq) {
          const int q = 4 * g + qq;
          sv[qq] = 0.0f;
          if ((valid >> q) & 1u) {
            const uint32_t k = (ords[g] >> (8 * qq)) & 0xffu;
            if (k != kcur) {
              kcur = k;
              kk[0] = s_k[k][0]; kk[1] = s_k[k][1]; kk[2] = s_k[k][2]; kk[3] = s_k[k][3];
            }
            sv[qq] = (float)request_out<MODE, HIST, SHARE>(P, kk, pv[q], cv[q], s_hist, tv[q],
                                                           pos + q, !full);
          }
        }
        if (MODE == MODE_ATTR && SHARE && full) {
          // ordinary (write-back) stores: the four 16-byte stores of a lane
          // land in the same lines, which L2 merges before writing them out
          const v4f v = {sv[0], sv[1], sv[2], sv[3]};
          *(v4f*)(P.share + pos + 4 * g) = v;
        }
      }
    }

    b = e;
    r0 = r1;
    wv = nwv;
  }

  if (HIST == HIST_LDS) {
    __syncthreads();
    double* dst = P.partials + (int64_t)blockIdx.x * P.n_tenants;
    for (int u = tid; u < P.n_tenants; u += kWG) dst[u] = s_hist[u];
  }
}

// ------------------------------------------------------ tenant reductions

// out[u] = sum over rows w of part[w][u], rows folded in a fixed order:
// block (s, x) sums rows of slice s for tenants x*64.., writes part2, and the
// last block of column x (counter, reset on the way out) adds the slices in
// order s = 0..S-1.
__global__ __launch_bounds__(kWG) void k_tenant_reduce(const double* __restrict__ part,
                                                       int rows, int T,
                                                       double* __restrict__ part2,
                                                       uint32_t* __restrict__ cnt,
                                                       double* __restrict__ out) {
  __shared__ double red[kWaves][kTenantChunk];
  __shared__ int last;
  const int S = gridDim.x, s = blockIdx.x, x = blockIdx.y;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int u = x * kTenantChunk + lane;
  const int w0 = (int)((int64_t)s * rows / S), w1 = (int)((int64_t)(s + 1) * rows / S);
  double acc = 0.0;
  if (u < T)
    for (int w = w0 + wave; w < w1; w += kWaves) acc += part[(int64_t)w * T + u];
  red[wave][lane] = acc;
  __syncthreads();
  if (wave == 0) {
    double v = red[0][lane];
    for (int w = 1; w < kWaves; ++w) v += red[w][lane];
    part2[((int64_t)x * S + s) * kTenantChunk + lane] = v;
  }
  __threadfence();
  __syncthreads();
  if (threadIdx.x == 0) last = (atomicAdd(cnt + x, 1u) == (uint32_t)(S - 1));
  __syncthreads();
  if (last) {
    __threadfence();
    if (wave == 0 && u < T) {
      double v = 0.0;
      for (int k = 0; k < S; ++k)
        v += __builtin_nontemporal_load(part2 + ((int64_t)x * S + k) * kTenantChunk + lane);
      out[u] = v;
    }
    if (threadIdx.x == 0) cnt[x] = 0;
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
  __syncthreads();
  const int64_t per = (n + gridDim.x - 1) / gridDim.x;
  const int64_t lo = per * blockIdx.x, hi = min(n, lo + per);
  for (int64_t i = lo + threadIdx.x; i < hi; i += kWG) {
    const double v = (double)share[i];
    if (HIST == HIST_LDS) atomicAdd(s_hist + tenant[i], v);
    else unsafeAtomicAdd(out + tenant[i], v);
  }
  if (HIST == HIST_LDS) {
    __syncthreads();
    for (int u = threadIdx.x; u < T; u += kWG) partials[(int64_t)blockIdx.x * T + u] = s_hist[u];
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
