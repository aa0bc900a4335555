/*
 * tracegen.c -- seeded synthetic traces of co-batched LLM scheduling steps.
 *
 * Inputs only: this file draws batch sizes, prompt/context lengths and tenant
 * ids.  It contains none of the attribution arithmetic.
 *
 * Random numbers: counter-based SplitMix64 (G. Steele, D. Lea, C. Flood,
 * "Fast splittable pseudorandom number generators", OOPSLA 2014).  The value
 * for (seed, stream, index) is the SplitMix64 output function applied to
 * key(seed, stream) + (index + 1) * golden_gamma, i.e. the (index+1)-th
 * output of a SplitMix64 sequence started at that key.  Every draw therefore
 * depends only on its (seed, stream, index), never on thread count or order.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>

#define GOLDEN 0x9E3779B97F4A7C15ULL

enum {
  STREAM_SIZE = 1,   /* batch size, indexed by batch            */
  STREAM_PHASE = 2,  /* batch phase, indexed by batch           */
  STREAM_C = 4,      /* uniform context lengths, by request     */
  STREAM_TENANT = 5, /* tenant ids, by request                  */
  STREAM_CHUNK = 6,  /* prefill chunks, by batch*16 + slot      */
  STREAM_PNORM = 7,  /* normals for prompt lengths, by request  */
  STREAM_CNORM = 8   /* normals for context lengths, by request */
};

enum { KIND_TINY_MIXED = 1, KIND_DECODE_ONLY = 2, KIND_CHUNKED_PREFILL = 3,
       KIND_HEAVY_TAILED = 4, KIND_SWEEP_MIXED = 5 };

static inline uint64_t mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
  return z ^ (z >> 31);
}

static inline uint64_t key_of(uint64_t seed, uint64_t stream) {
  return mix64(seed * GOLDEN + mix64(stream + 1));
}

static inline uint64_t draw(uint64_t key, uint64_t idx) {
  return mix64(key + (idx + 1) * GOLDEN);
}

/* U in [0, 1) with 53 random bits. */
static inline double unif(uint64_t key, uint64_t idx) {
  return (double)(draw(key, idx) >> 11) * 0x1.0p-53;
}

/* Integer uniform on [a, b]. */
static inline int64_t unif_int(uint64_t key, uint64_t idx, int64_t a, int64_t b) {
  int64_t v = a + (int64_t)floor(unif(key, idx) * (double)(b - a + 1));
  return v > b ? b : v;
}

/* N(0,1), Box-Muller from the uniforms at 2*idx and 2*idx+1. */
static inline double normal(uint64_t key, uint64_t idx) {
  const double u1 = 1.0 - unif(key, 2 * idx); /* (0, 1] */
  const double u2 = unif(key, 2 * idx + 1);
  return sqrt(-2.0 * log(u1)) * cos(6.283185307179586476925 * u2);
}

/* round(median * exp(sigma * Z)) clipped to [lo, hi]. */
static inline int32_t lognormal_int(uint64_t key, uint64_t idx, double median,
                                    double sigma, int64_t lo, int64_t hi) {
  const double v = median * exp(sigma * normal(key, idx));
  if (!(v < (double)hi)) return (int32_t)hi;
  int64_t r = llround(v);
  if (r < lo) r = lo;
  if (r > hi) r = hi;
  return (int32_t)r;
}

void tg_uniform(uint64_t seed, uint64_t stream, int64_t start, int64_t n, double *out) {
  const uint64_t k = key_of(seed, stream);
  for (int64_t i = 0; i < n; ++i) out[i] = unif(k, (uint64_t)(start + i));
}

void tg_normal(uint64_t seed, uint64_t stream, int64_t start, int64_t n, double *out) {
  const uint64_t k = key_of(seed, stream);
  for (int64_t i = 0; i < n; ++i) out[i] = normal(k, (uint64_t)(start + i));
}

/* Cumulative Zipf weights: cdf[k] = sum_{j<=k} (j+1)^-s. */
static double *zipf_table(int32_t n_items, double s) {
  double *cdf = (double *)malloc(sizeof(double) * (size_t)n_items);
  if (!cdf) return NULL;
  double acc = 0.0;
  for (int32_t k = 0; k < n_items; ++k) {
    acc += pow((double)(k + 1), -s);
    cdf[k] = acc;
  }
  return cdf;
}

/* Smallest k with cdf[k] > u * total. */
static inline int32_t zipf_pick(const double *cdf, int32_t n_items, double u) {
  const double target = u * cdf[n_items - 1];
  int32_t lo = 0, hi = n_items - 1;
  while (lo < hi) {
    const int32_t mid = lo + (hi - lo) / 2;
    if (cdf[mid] > target) hi = mid;
    else lo = mid + 1;
  }
  return lo;
}

int tg_zipf(uint64_t seed, uint64_t stream, int64_t start, int64_t n, int32_t n_items,
            double s, int32_t *out) {
  if (n_items <= 0) return -1;
  double *cdf = zipf_table(n_items, s);
  if (!cdf) return -1;
  const uint64_t k = key_of(seed, stream);
  for (int64_t i = 0; i < n; ++i) out[i] = zipf_pick(cdf, n_items, unif(k, (uint64_t)(start + i)));
  free(cdf);
  return 0;
}

/* ---- chunked-prefill batch layout (shared by both passes) ---- */
#define CP_BUDGET 8192
#define CP_MAX_SEQS 256

typedef struct {
  int k_eff;
  int32_t len[4], prefix[4];
  int64_t n_dec;
} cp_batch;

static void cp_layout(uint64_t kchunk, int64_t b, cp_batch *o) {
  const int k = (int)unif_int(kchunk, (uint64_t)(b * 16), 0, 4);
  int64_t budget = CP_BUDGET;
  o->k_eff = 0;
  for (int j = 0; j < k; ++j) {
    int64_t len = unif_int(kchunk, (uint64_t)(b * 16 + 1 + 2 * j), 64, 4096);
    const int64_t pre = unif_int(kchunk, (uint64_t)(b * 16 + 2 + 2 * j), 0, 16384);
    if (len > budget) len = budget;
    if (len == 0) break;
    o->len[o->k_eff] = (int32_t)len;
    o->prefix[o->k_eff] = (int32_t)pre;
    o->k_eff++;
    budget -= len;
  }
  int64_t nd = CP_MAX_SEQS - o->k_eff;
  if (nd > budget) nd = budget;
  o->n_dec = nd;
}

/* Batch sizes for the recipe `kind`. */
int tg_sizes(int kind, uint64_t seed, int64_t nB, int64_t *sizes) {
  const uint64_t ks = key_of(seed, STREAM_SIZE), kc = key_of(seed, STREAM_CHUNK);
  switch (kind) {
    case KIND_TINY_MIXED:
#pragma omp parallel for schedule(static)
      for (int64_t b = 0; b < nB; ++b) sizes[b] = unif_int(ks, (uint64_t)b, 1, 32);
      return 0;
    case KIND_DECODE_ONLY:
    case KIND_SWEEP_MIXED:
#pragma omp parallel for schedule(static)
      for (int64_t b = 0; b < nB; ++b) sizes[b] = unif_int(ks, (uint64_t)b, 1, 256);
      return 0;
    case KIND_CHUNKED_PREFILL:
#pragma omp parallel for schedule(static)
      for (int64_t b = 0; b < nB; ++b) {
        cp_batch o;
        cp_layout(kc, b, &o);
        sizes[b] = o.k_eff + o.n_dec;
      }
      return 0;
    case KIND_HEAVY_TAILED:
      /* Lomax (Pareto type II), alpha 1.5, scale 86, shifted to start at 1
       * and clipped at 1024: n = min(1024, 1 + floor(86 * (V^(-1/1.5) - 1))),
       * V uniform on (0, 1]. */
#pragma omp parallel for schedule(static)
      for (int64_t b = 0; b < nB; ++b) {
        const double v = 1.0 - unif(ks, (uint64_t)b);
        const double x = 86.0 * (pow(v, -1.0 / 1.5) - 1.0);
        sizes[b] = x >= 1023.0 ? 1024 : 1 + (int64_t)floor(x);
      }
      return 0;
    default:
      return -1;
  }
}

/* Per-request fields for the recipe `kind`, given the offsets that
 * tg_sizes' sizes produce. */
int tg_fill(int kind, uint64_t seed, int64_t nB, const int64_t *off, int32_t *p,
            int32_t *c, int32_t *t, int32_t n_tenants) {
  if (n_tenants <= 0) return -1;
  const uint64_t kph = key_of(seed, STREAM_PHASE), kcu = key_of(seed, STREAM_C),
                 kt = key_of(seed, STREAM_TENANT), kch = key_of(seed, STREAM_CHUNK),
                 kpn = key_of(seed, STREAM_PNORM), kcn = key_of(seed, STREAM_CNORM);
  double *cdf = NULL;
  double zipf_s = 0.0;
  if (kind == KIND_DECODE_ONLY) zipf_s = 1.1;
  if (kind == KIND_HEAVY_TAILED || kind == KIND_SWEEP_MIXED) zipf_s = 1.2;
  if (zipf_s > 0.0) {
    cdf = zipf_table(n_tenants, zipf_s);
    if (!cdf) return -1;
  }
  int bad = 0;
#pragma omp parallel for schedule(dynamic, 256) reduction(| : bad)
  for (int64_t b = 0; b < nB; ++b) {
    const int64_t lo = off[b], hi = off[b + 1];
    switch (kind) {
      case KIND_TINY_MIXED:
      case KIND_SWEEP_MIXED: {
        const int prefill = unif(kph, (uint64_t)b) < 0.3;
        for (int64_t i = lo; i < hi; ++i) {
          if (prefill) {
            p[i] = lognormal_int(kpn, (uint64_t)i, 512.0, 1.0, 16, 8192);
            c[i] = 0;
          } else {
            p[i] = 1;
            c[i] = (int32_t)unif_int(kcu, (uint64_t)i, 128, 8192);
          }
        }
        break;
      }
      case KIND_DECODE_ONLY:
        for (int64_t i = lo; i < hi; ++i) {
          p[i] = 1;
          c[i] = lognormal_int(kcn, (uint64_t)i, 2048.0, 1.2, 1, 32768);
        }
        break;
      case KIND_CHUNKED_PREFILL: {
        cp_batch o;
        cp_layout(kch, b, &o);
        if (o.k_eff + o.n_dec != hi - lo) {
          bad = 1;
          break;
        }
        for (int j = 0; j < o.k_eff; ++j) {
          p[lo + j] = o.len[j];
          c[lo + j] = o.prefix[j];
        }
        for (int64_t i = lo + o.k_eff; i < hi; ++i) {
          p[i] = 1;
          c[i] = lognormal_int(kcn, (uint64_t)i, 1024.0, 1.2, 1, 32768);
        }
        break;
      }
      case KIND_HEAVY_TAILED: {
        const int prefill = unif(kph, (uint64_t)b) < 0.2;
        for (int64_t i = lo; i < hi; ++i) {
          if (prefill) {
            p[i] = lognormal_int(kpn, (uint64_t)i, 256.0, 1.0, 1, 16384);
            c[i] = 0;
          } else {
            p[i] = 1;
            c[i] = (int32_t)unif_int(kcu, (uint64_t)i, 1, 131072);
          }
        }
        break;
      }
      default:
        bad = 1;
    }
    for (int64_t i = lo; i < hi; ++i)
      t[i] = cdf ? zipf_pick(cdf, n_tenants, unif(kt, (uint64_t)i))
                 : (int32_t)unif_int(kt, (uint64_t)i, 0, n_tenants - 1);
  }
  free(cdf);
  return bad ? -1 : 0;
}
