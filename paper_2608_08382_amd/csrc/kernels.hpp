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

constexpr int kWG = 256;                         // threads per workgroup
constexpr int kWaves = kWG / 64;                 // wave64
constexpr int kVec = 4;                          // consecutive requests per lane per round
constexpr int kRounds = 3;                       // rounds held in registers per wave
constexpr int kRoundSpan = 64 * kVec;            // 256 requests per wave-round
constexpr int kWaveSpan = kRoundSpan * kRounds;  // 768
constexpr int kCap = kWaveSpan * kWaves;         // 3072 request slots per tile
constexpr int kWindow = 256;                     // offsets examined per tile
constexpr int kMaxTileBatches = kWindow - 1;     // 255 batches per tile
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
  if (SHARE && store_scalar) __builtin_nontemporal_store((float)s, P.share + i);
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

struct Pref {
  uint64_t pc;  // sum p (low 32 bits) | count of prefill-like requests (high)
  uint64_t c;
  uint64_t q;
  uint32_t w;   // wave whose running prefix this is relative to
  uint32_t pad;
};

template <int MODE, int HIST, bool SHARE>
__global__ __launch_bounds__(kWG) void k_tiles(const Params P) {
  extern __shared__ double s_hist[];  // [n_tenants] when HIST_LDS
  __shared__ int32_t s_lo[kWindow];   // batch starts relative to the tile base
  __shared__ Pref s_xs[kWindow];      // prefix before each batch's first request
  __shared__ Pref s_xe[kWindow];      // prefix through each batch's last request
  __shared__ double s_k[kWindow][4];  // per-batch share / feature constants
  __shared__ uint64_t s_wt[kWaves][3];
  __shared__ BigRed s_red[kWaves];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int64_t N = P.N;

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
    const int64_t lim = min((int64_t)kMaxTileBatches, bw1 - b);
    const int64_t ra = r0 & ~(int64_t)(kVec - 1);  // 16-byte aligned tile base
    int pred = 0;
    if (tid <= lim) {
      const int64_t rel = wv - ra;
      s_lo[tid] = (int32_t)min(rel, (int64_t)kCap + 1);
      pred = (tid >= 1 && rel <= kCap) ? 1 : 0;
    }
    // Batches b .. b+count-1 end within kCap slots of the tile base.
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

    // Window of the next tile, in flight while this one is processed.
    int64_t nwv = 0;
    if (e < bw1 && tid <= min((int64_t)kMaxTileBatches, bw1 - e)) nwv = P.off[e + tid];

    // ---- load: lane holds positions x0..x0+3 of each round (x rel. to ra)
    int32_t pv[kRounds][kVec], cv[kRounds][kVec], tv[kRounds][kVec];
#pragma unroll
    for (int k = 0; k < kRounds; ++k) {
      const int32_t x0 = wave * kWaveSpan + k * kRoundSpan + lane * kVec;
      const int64_t pos = ra + x0;
#pragma unroll
      for (int q = 0; q < kVec; ++q) pv[k][q] = cv[k][q] = tv[k][q] = 0;
      if (x0 < L) {
        if (pos + kVec <= N) {
          const v4i a = __builtin_nontemporal_load((const v4i*)(P.p + pos));
          const v4i d = __builtin_nontemporal_load((const v4i*)(P.c + pos));
          pv[k][0] = a.x; pv[k][1] = a.y; pv[k][2] = a.z; pv[k][3] = a.w;
          cv[k][0] = d.x; cv[k][1] = d.y; cv[k][2] = d.z; cv[k][3] = d.w;
          if (HIST != HIST_NONE) {
            const v4i t = __builtin_nontemporal_load((const v4i*)(P.tenant + pos));
            tv[k][0] = t.x; tv[k][1] = t.y; tv[k][2] = t.z; tv[k][3] = t.w;
          }
        } else {
#pragma unroll
          for (int q = 0; q < kVec; ++q) {
            if (pos + q < N) {
              pv[k][q] = P.p[pos + q];
              cv[k][q] = P.c[pos + q];
              if (HIST != HIST_NONE) tv[k][q] = P.tenant[pos + q];
            }
          }
        }
      }
    }

    // ---- batch id of each held request (binary search in s_lo), while the
    // loads are in flight.  bits: valid 0-3, first-of-batch 4-7, last 8-11.
    uint32_t bids[kRounds], flags[kRounds];
#pragma unroll
    for (int k = 0; k < kRounds; ++k) {
      const int32_t x0 = wave * kWaveSpan + k * kRoundSpan + lane * kVec;
      const int32_t xs = max(x0, xf);
      int lo_i = 0, hi_i = count;
      while (hi_i - lo_i > 1) {
        const int mid = (lo_i + hi_i) >> 1;
        if (s_lo[mid] <= xs) lo_i = mid;
        else hi_i = mid;
      }
      int j = lo_i;
      int32_t cur = s_lo[j], nxt = s_lo[j + 1];
      uint32_t bp = 0, fl = 0;
#pragma unroll
      for (int q = 0; q < kVec; ++q) {
        const int32_t x = x0 + q;
        const bool valid = (x >= xf) && (x < L);
        if (valid) {
          while (nxt <= x) {
            ++j;
            cur = nxt;
            nxt = s_lo[j + 1];
          }
          fl |= 1u << q;
          if (x == cur) fl |= 1u << (4 + q);
          if (x + 1 == nxt) fl |= 1u << (8 + q);
        }
        bp |= (uint32_t)j << (8 * q);
      }
      bids[k] = bp;
      flags[k] = fl;
    }

    // ---- prefix sums: in-lane, wave (DPP), carried across rounds
    uint64_t carry_pc = 0, carry_c = 0, carry_q = 0;
#pragma unroll
    for (int k = 0; k < kRounds; ++k) {
      uint64_t ipc[kVec], ic[kVec], iq[kVec];
      uint64_t apc = 0, ac = 0, aq = 0;
#pragma unroll
      for (int q = 0; q < kVec; ++q) {
        const bool valid = (flags[k] >> q) & 1u;
        const int32_t p = pv[k][q], c = cv[k][q];
        const uint64_t xpc = valid ? ((uint64_t)(uint32_t)p |
                                      ((uint64_t)((p > 1 || c == 0) ? 1 : 0) << 32))
                                   : 0;
        const uint64_t xc = valid ? (uint64_t)(uint32_t)c : 0;
        const uint64_t xq = valid ? (uint64_t)((int64_t)p * p) : 0;
        apc += xpc;
        ac += xc;
        aq += xq;
        ipc[q] = apc;
        ic[q] = ac;
        iq[q] = aq;
      }
      const uint64_t spc = wave_incl_scan(apc);
      const uint64_t sc = wave_incl_scan(ac);
      const uint64_t sq = wave_incl_scan(aq);
      const uint64_t bpc = carry_pc + spc - apc;  // prefix before this lane
      const uint64_t bc = carry_c + sc - ac;
      const uint64_t bq = carry_q + sq - aq;
      if (flags[k] & 0xff0u) {
#pragma unroll
        for (int q = 0; q < kVec; ++q) {
          const uint32_t j = (bids[k] >> (8 * q)) & 0xffu;
          const uint64_t prev_pc = q ? ipc[q - 1] : 0, prev_c = q ? ic[q - 1] : 0,
                         prev_q = q ? iq[q - 1] : 0;
          if ((flags[k] >> (4 + q)) & 1u)
            s_xs[j] = Pref{bpc + prev_pc, bc + prev_c, bq + prev_q, (uint32_t)wave, 0};
          if ((flags[k] >> (8 + q)) & 1u)
            s_xe[j] = Pref{bpc + ipc[q], bc + ic[q], bq + iq[q], (uint32_t)wave, 0};
        }
      }
      carry_pc += readlane_u64(spc, 63);
      carry_c += readlane_u64(sc, 63);
      carry_q += readlane_u64(sq, 63);
    }
    if (lane == 0) {
      s_wt[wave][0] = carry_pc;
      s_wt[wave][1] = carry_c;
      s_wt[wave][2] = carry_q;
    }
    __syncthreads();

    // ---- per batch: totals from prefix differences, then the model
    if (tid < count) {
      const int j = tid;
      const int64_t n = (int64_t)s_lo[j + 1] - s_lo[j];
      const int64_t bg = b + j;
      if (n == 0) {
        empty_batch<MODE>(P, bg);
      } else {
        const Pref xs = s_xs[j], xe = s_xe[j];
        uint64_t st_pc = xs.pc, st_c = xs.c, st_q = xs.q;
        uint64_t en_pc = xe.pc, en_c = xe.c, en_q = xe.q;
        for (uint32_t w = 0; w < (uint32_t)kWaves; ++w) {
          if (w < xs.w) { st_pc += s_wt[w][0]; st_c += s_wt[w][1]; st_q += s_wt[w][2]; }
          if (w < xe.w) { en_pc += s_wt[w][0]; en_c += s_wt[w][1]; en_q += s_wt[w][2]; }
        }
        const uint64_t dpc = en_pc - st_pc;
        batch_model<MODE>(P, bg, n, dpc & 0xffffffffull, en_c - st_c, en_q - st_q,
                          (dpc >> 32) != 0, s_k[j]);
      }
    }
    __syncthreads();

    // ---- per request: share (+ tenant) or features
#pragma unroll
    for (int k = 0; k < kRounds; ++k) {
      const uint32_t fl = flags[k];
      if (!(fl & 0xfu)) continue;
      const int32_t x0 = wave * kWaveSpan + k * kRoundSpan + lane * kVec;
      const int64_t pos = ra + x0;
      const bool full = (fl & 0xfu) == 0xfu;
      float sv[kVec];
#pragma unroll
      for (int q = 0; q < kVec; ++q) {
        sv[q] = 0.0f;
        if ((fl >> q) & 1u) {
          const uint32_t j = (bids[k] >> (8 * q)) & 0xffu;
          const double kk[4] = {s_k[j][0], s_k[j][1], s_k[j][2], s_k[j][3]};
          sv[q] = (float)request_out<MODE, HIST, SHARE>(P, kk, pv[k][q], cv[k][q], s_hist,
                                                        tv[k][q], pos + q, !full);
        }
      }
      if (MODE == MODE_ATTR && SHARE && full) {
        const v4f v = {sv[0], sv[1], sv[2], sv[3]};
        __builtin_nontemporal_store(v, (v4f*)(P.share + pos));
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
