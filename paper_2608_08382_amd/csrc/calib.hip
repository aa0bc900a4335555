// calib.hip -- STREAM-style bandwidth calibration for the attribution
// path's access mix (measurement context only; not part of the attribution
// library's C ABI).
//
// The attribution step reads three int32 arrays (p, c, tenant) and writes
// one fp32 array (the shares): 12 B read and 4 B written per request.  These
// kernels move exactly those bytes with the simplest access pattern there
// is -- every wave instruction touches 1 KB of consecutive memory, a
// grid-stride loop, nothing held across iterations -- so their rate is what
// a plain streaming kernel reaches on this device for the same mix.  Each
// access kind is timed with plain and with non-temporal loads and stores.
//
//   mode 0: read 12 B per element (three int32 arrays)
//   mode 1: write 4 B per element (one fp32 array)
//   mode 2: read 12 B and write 4 B per element (the attribution mix)
//   mode 3: the mix in wave tiles: each wave loads a tile of 256*G elements
//           of each input (group g: lane l takes elements 256g + 4l .. + 3),
//           then stores it; tiles are dealt to waves round-robin in chunks
//           of `chunk` tiles (G = unroll: 2, 4 or 7)
//   flags bit 0: non-temporal loads; bit 1: non-temporal stores
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

typedef int32_t v4i __attribute__((ext_vector_type(4)));
typedef float v4f __attribute__((ext_vector_type(4)));

template <bool NT>
__device__ __forceinline__ v4i ld(const v4i* p) {
  if constexpr (NT) return __builtin_nontemporal_load(p);
  else return *p;
}

template <bool NT>
__device__ __forceinline__ void st(v4f* p, v4f v) {
  if constexpr (NT) __builtin_nontemporal_store(v, p);
  else *p = v;
}

// U vec4 elements per thread per iteration, loads issued before use.
template <int MODE, bool NTL, bool NTS, int U>
__global__ __launch_bounds__(256) void k_stream(const v4i* __restrict__ a, const v4i* __restrict__ b,
                                                const v4i* __restrict__ t, v4f* __restrict__ s,
                                                int64_t n4, int32_t* __restrict__ sink) {
  const int64_t stride = (int64_t)gridDim.x * 256;
  int32_t acc = 0;
  for (int64_t i0 = (int64_t)blockIdx.x * 256 * U + threadIdx.x; i0 < n4; i0 += stride * U) {
    v4i x[U], y[U], z[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int64_t i = i0 + (int64_t)u * 256;
      if (MODE != 1 && i < n4) {
        x[u] = ld<NTL>(a + i);
        y[u] = ld<NTL>(b + i);
        z[u] = ld<NTL>(t + i);
      } else {
        x[u] = y[u] = z[u] = (v4i){(int)i, 1, 2, 3};
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int64_t i = i0 + (int64_t)u * 256;
      if (i >= n4) continue;
      const v4i w = x[u] + y[u] + z[u];
      if (MODE == 0) {
        acc ^= w.x ^ w.y ^ w.z ^ w.w;
      } else {
        st<NTS>(s + i, (v4f){(float)w.x, (float)w.y, (float)w.z, (float)w.w});
      }
    }
  }
  // keeps the read-only loads live; the value is never read
  if (MODE == 0 && acc == 0x7fffffff) sink[0] = acc;
}

// Wave tiles of 256*G elements, chunks of `chunk` tiles dealt round-robin
// over the waves; all loads of a tile are issued before its stores.
template <bool NTL, bool NTS, int G>
__global__ __launch_bounds__(256) void k_wave_tiles(const v4i* __restrict__ a,
                                                    const v4i* __restrict__ b,
                                                    const v4i* __restrict__ t,
                                                    v4f* __restrict__ s, int64_t n4, int chunk) {
  const int lane = threadIdx.x & 63;
  const int64_t waves = (int64_t)gridDim.x * 4, w = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int64_t tile4 = 64 * G;
  const int64_t ntiles = (n4 + tile4 - 1) / tile4;
  const int64_t nchunks = (ntiles + chunk - 1) / chunk;
  for (int64_t ch = w; ch < nchunks; ch += waves) {
    for (int64_t k = ch * chunk; k < ch * chunk + chunk && k < ntiles; ++k) {
      v4i x[G], y[G], z[G];
#pragma unroll
      for (int g = 0; g < G; ++g) {
        const int64_t i = k * tile4 + 64 * g + lane;
        x[g] = y[g] = z[g] = (v4i){0, 0, 0, 0};
        if (i < n4) {
          x[g] = ld<NTL>(a + i);
          y[g] = ld<NTL>(b + i);
          z[g] = ld<NTL>(t + i);
        }
      }
#pragma unroll
      for (int g = 0; g < G; ++g) {
        const int64_t i = k * tile4 + 64 * g + lane;
        const v4i v = x[g] + y[g] + z[g];
        if (i < n4) st<NTS>(s + i, (v4f){(float)v.x, (float)v.y, (float)v.z, (float)v.w});
      }
    }
  }
}

template <int G>
void* pick_tiles(int flags) {
  switch (flags & 3) {
    case 0: return (void*)k_wave_tiles<false, false, G>;
    case 1: return (void*)k_wave_tiles<true, false, G>;
    case 2: return (void*)k_wave_tiles<false, true, G>;
    default: return (void*)k_wave_tiles<true, true, G>;
  }
}

template <int MODE, int U>
void* pick(int flags) {
  switch (flags & 3) {
    case 0: return (void*)k_stream<MODE, false, false, U>;
    case 1: return (void*)k_stream<MODE, true, false, U>;
    case 2: return (void*)k_stream<MODE, false, true, U>;
    default: return (void*)k_stream<MODE, true, true, U>;
  }
}

template <int MODE>
void* pick_u(int flags, int u) {
  if (u == 1) return pick<MODE, 1>(flags);
  if (u == 2) return pick<MODE, 2>(flags);
  if (u == 4) return pick<MODE, 4>(flags);
  return nullptr;
}

}  // namespace

extern "C" {

// Runs one calibration kernel over n4 16-byte elements per array (the
// caller's device buffers, 16-byte aligned; a, b, t are read, s written).
// grid: workgroups of 256 threads.  unroll: 1, 2 or 4 elements per thread
// per iteration (modes 0-2).  Returns 0, or -1 on a bad argument or launch
// error.
// mode 3 (wave tiles): unroll is G (2, 4 or 7) and chunk the tiles per chunk.
int llmv_calib_stream(int mode, int flags, int unroll, int grid, const void* a, const void* b,
                      const void* t, void* s, int64_t n4, void* sink, void* stream, int chunk) {
  if (mode < 0 || mode > 3 || grid < 1 || n4 < 0 || !sink) return -1;
  if (mode != 1 && (!a || !b || !t)) return -1;
  if (mode != 0 && !s) return -1;
  hipStream_t st = (hipStream_t)stream;
  if (mode == 3) {
    if (chunk < 1) return -1;
    void* k = unroll == 2 ? pick_tiles<2>(flags)
              : (unroll == 4 ? pick_tiles<4>(flags) : (unroll == 7 ? pick_tiles<7>(flags) : nullptr));
    if (!k) return -1;
    void* args[] = {(void*)&a, (void*)&b, (void*)&t, (void*)&s, (void*)&n4, (void*)&chunk};
    if (hipLaunchKernel(k, dim3(grid), dim3(256), args, 0, st) != hipSuccess) return -1;
    return hipGetLastError() == hipSuccess ? 0 : -1;
  }
  if (unroll != 1 && unroll != 2 && unroll != 4) return -1;
  void* k = mode == 0 ? pick_u<0>(flags, unroll)
            : (mode == 1 ? pick_u<1>(flags, unroll) : pick_u<2>(flags, unroll));
  if (!k) return -1;
  void* args[] = {(void*)&a, (void*)&b, (void*)&t, (void*)&s, (void*)&n4, (void*)&sink};
  if (hipLaunchKernel(k, dim3(grid), dim3(256), args, 0, st) != hipSuccess) return -1;
  return hipGetLastError() == hipSuccess ? 0 : -1;
}

}  // extern "C"
