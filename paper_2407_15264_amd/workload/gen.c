/*
 * Seeded synthetic workload generators for the feature-gather cache.
 *
 * This file produces INPUTS only: an R-MAT graph in CSR form, the per-node
 * in-degree used as the static score, GraphSAGE-style request streams, and
 * N(0,1) feature rows.  It holds none of the cache method's arithmetic and is
 * used both by the CPU oracle's tests and by the GPU path's tests and bench.
 *
 * Every random draw comes from a counter-based SplitMix64 stream (Steele, Lea
 * and Flood, "Fast splittable pseudorandom number generators", OOPSLA 2014):
 * output k of the stream keyed by K is mix(K + (k+1)*GAMMA), so any draw can be
 * computed independently of the others and results do not depend on thread
 * count or scheduling.
 *
 *   R-MAT: Chakrabarti, Zhan and Faloutsos, SDM 2004 -- per edge and per level
 *   one uniform chooses a quadrant with probabilities (a, b, c, d); no noise,
 *   no relabelling, self loops and multi-edges kept.  For N not a power of two
 *   the scale is ceil(log2 N) and attempts with an endpoint >= N are rejected
 *   until E edges are accepted (attempt order is the counter order).
 *
 *   Sampler (GraphSAGE uniform neighbour sampling, paper Sec. 2.1): hop h takes
 *   each frontier node v in ascending order and draws min(f_h, outdeg v)
 *   distinct adjacency positions with Floyd's algorithm (Bentley & Floyd,
 *   CACM 1987); the next frontier is the sorted unique set of the samples.
 *   The request list of one minibatch is seeds ++ samples of hop 0 ++ hop 1 ...
 *   (raw, with duplicates).  Seeds are consecutive chunks of a seeded
 *   Fisher-Yates permutation of [0, N).
 *
 *   Features: Box-Muller (Box and Muller, Ann. Math. Statist. 1958) in binary32,
 *   both outputs of each pair used.  Row v, pair j (elements 2j and 2j+1) takes
 *   draw r = output (v * ceil(dim/2) + j) of the stream keyed by the feature
 *   seed; its top 24 bits give u1 = (hi24 + 1) / 2^24 in (0, 1], the next 24
 *   bits an angle w / 2^24 of a full turn; the pair is (rho cos theta, rho sin
 *   theta) with rho = sqrt(-2 ln u1).  The logarithm and the circular
 *   functions are this file's own polynomials (see nrm_pair): any
 *   approximation serves a synthetic input as long as it is fixed, and these
 *   vectorize, which the library calls do not (a 200 GB table is filled in
 *   seconds per core-minute instead of hours).  fp16 rows are the fp32 values
 *   rounded to binary16 with round-to-nearest-even.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <omp.h>

#define GAMMA 0x9e3779b97f4a7c15ULL

static inline uint64_t sm_mix(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ULL;
  z = (z ^ (z >> 27)) * 0x94d049bb133111ebULL;
  return z ^ (z >> 31);
}
/* output k (0-based) of the SplitMix64 stream seeded with `key` */
static inline uint64_t sm_at(uint64_t key, uint64_t k) { return sm_mix(key + (k + 1) * GAMMA); }
/* derive an independent stream key from a parent key and a label */
static inline uint64_t sm_key(uint64_t parent, uint64_t label) { return sm_at(sm_mix(parent ^ 0x5851f42d4c957f2dULL), label); }
static inline double u01(uint64_t r) { return (double)(r >> 11) * (1.0 / 9007199254740992.0); }
/* uniform integer in [0, m) from the high 32 bits (m < 2^32) */
static inline uint64_t below(uint64_t r, uint64_t m) { return ((r >> 32) * m) >> 32; }

/* exported for the generator's own tests */
uint64_t wl_splitmix_at(uint64_t key, uint64_t k) { return sm_at(key, k); }

enum { LABEL_RMAT = 1, LABEL_PERM = 2, LABEL_SAMPLE = 3, LABEL_FEAT = 4 };

/* ------------------------------------------------------------------ R-MAT */
static inline int rmat_attempt(uint64_t key, uint64_t k, int scale, double a, double ab, double abc,
                               uint64_t n, uint32_t *s_out, uint32_t *d_out) {
  uint64_t s = 0, d = 0;
  for (int l = 0; l < scale; ++l) {
    double u = u01(sm_at(key, k * 64 + (uint64_t)l));
    int bs, bd;
    if (u < a) { bs = 0; bd = 0; }
    else if (u < ab) { bs = 0; bd = 1; }
    else if (u < abc) { bs = 1; bd = 0; }
    else { bs = 1; bd = 1; }
    s = (s << 1) | (uint64_t)bs;
    d = (d << 1) | (uint64_t)bd;
  }
  if (s >= n || d >= n) return 0;
  *s_out = (uint32_t)s;
  *d_out = (uint32_t)d;
  return 1;
}

/*
 * Generate an R-MAT graph with n nodes and e edges and build its CSR by source
 * (adjacency lists sorted ascending).  offsets has n+1 entries, adj e entries,
 * indeg n entries.  Returns 0 on success, -1 on allocation failure.
 */
int wl_rmat_csr(uint64_t n, uint64_t e, double a, double b, double c, uint64_t seed,
                int64_t *offsets, uint32_t *adj, uint32_t *indeg) {
  int scale = 0;
  while ((1ULL << scale) < n) ++scale;
  uint64_t key = sm_key(seed, LABEL_RMAT);
  double ab = a + b, abc = a + b + c;
  uint32_t *src = (uint32_t *)malloc(e * sizeof(uint32_t));
  uint32_t *dst = (uint32_t *)malloc(e * sizeof(uint32_t));
  if (!src || !dst) { free(src); free(dst); return -1; }

  /* Rounds of NCH chunks of CH consecutive attempts: each chunk keeps its
     accepted edges in attempt order, then they are placed after those of the
     earlier chunks until e edges are accepted. */
  const uint64_t CH = 1ULL << 16;  /* attempts per chunk */
  const int NCH = 256;             /* chunks per round */
  uint64_t *cnt = (uint64_t *)malloc(NCH * sizeof(uint64_t));
  uint32_t *kept = (uint32_t *)malloc((uint64_t)NCH * CH * 2 * sizeof(uint32_t));
  if (!cnt || !kept) { free(cnt); free(kept); free(src); free(dst); return -1; }
  uint64_t got = 0, base = 0;
  while (got < e) {
#pragma omp parallel for schedule(dynamic, 1)
    for (int ci = 0; ci < NCH; ++ci) {
      uint64_t k0 = base + (uint64_t)ci * CH, m = 0;
      uint32_t *kc = kept + (uint64_t)ci * CH * 2;
      for (uint64_t k = k0; k < k0 + CH; ++k)
        m += (uint64_t)rmat_attempt(key, k, scale, a, ab, abc, n, &kc[2 * m], &kc[2 * m + 1]);
      cnt[ci] = m;
    }
    uint64_t pos[256];
    uint64_t acc = got;
    for (int ci = 0; ci < NCH; ++ci) { pos[ci] = acc; acc += cnt[ci]; }
#pragma omp parallel for schedule(dynamic, 1)
    for (int ci = 0; ci < NCH; ++ci) {
      const uint32_t *kc = kept + (uint64_t)ci * CH * 2;
      for (uint64_t i = 0, p = pos[ci]; i < cnt[ci] && p < e; ++i, ++p) { src[p] = kc[2 * i]; dst[p] = kc[2 * i + 1]; }
    }
    got = acc < e ? acc : e;
    base += (uint64_t)NCH * CH;
  }
  free(kept);
  free(cnt);

  /* CSR by source: count, exclusive prefix, place, then sort each list */
  uint32_t *deg = (uint32_t *)calloc(n, sizeof(uint32_t));
  memset(indeg, 0, n * sizeof(uint32_t));
#pragma omp parallel for
  for (uint64_t i = 0; i < e; ++i) {
    __atomic_fetch_add(&deg[src[i]], 1u, __ATOMIC_RELAXED);
    __atomic_fetch_add(&indeg[dst[i]], 1u, __ATOMIC_RELAXED);
  }
  offsets[0] = 0;
  for (uint64_t v = 0; v < n; ++v) offsets[v + 1] = offsets[v] + deg[v];
  memset(deg, 0, n * sizeof(uint32_t));
#pragma omp parallel for
  for (uint64_t i = 0; i < e; ++i) {
    uint32_t s = src[i];
    uint32_t slot = __atomic_fetch_add(&deg[s], 1u, __ATOMIC_RELAXED);
    adj[offsets[s] + slot] = dst[i];
  }
  free(src);
  free(dst);
  free(deg);
#pragma omp parallel for schedule(dynamic, 4096)
  for (uint64_t v = 0; v < n; ++v) {
    /* insertion sort for short lists, shell-like gaps otherwise (lists are
       arbitrary multisets, so sorting makes the layout deterministic) */
    uint32_t *l = adj + offsets[v];
    int64_t m = offsets[v + 1] - offsets[v];
    static const int64_t gaps[] = {701, 301, 132, 57, 23, 10, 4, 1};
    for (int gi = 0; gi < 8; ++gi) {
      int64_t g = gaps[gi];
      for (int64_t i = g; i < m; ++i) {
        uint32_t x = l[i];
        int64_t j = i;
        while (j >= g && l[j - g] > x) { l[j] = l[j - g]; j -= g; }
        l[j] = x;
      }
    }
  }
  return 0;
}

/* ---------------------------------------------------------- permutation */
/* First m entries of a seeded Fisher-Yates permutation of [0, n). */
int wl_perm_prefix(uint64_t n, uint64_t m, uint64_t seed, int64_t *out) {
  uint32_t *p = (uint32_t *)malloc(n * sizeof(uint32_t));
  if (!p) return -1;
  for (uint64_t i = 0; i < n; ++i) p[i] = (uint32_t)i;
  uint64_t key = sm_key(seed, LABEL_PERM);
  for (uint64_t i = 0; i < m && i < n; ++i) {
    uint64_t j = i + below(sm_at(key, i), n - i);
    uint32_t t = p[i]; p[i] = p[j]; p[j] = t;
    out[i] = p[i];
  }
  free(p);
  return 0;
}

/* ---------------------------------------------------------------- sampler */
static int cmp_i64(const void *x, const void *y) {
  int64_t a = *(const int64_t *)x, b = *(const int64_t *)y;
  return (a > b) - (a < b);
}

typedef struct { int64_t *v; uint64_t n, cap; } vec_t;
static int vpush(vec_t *q, int64_t x) {
  if (q->n == q->cap) {
    uint64_t nc = q->cap ? q->cap * 2 : 1024;
    int64_t *nv = (int64_t *)realloc(q->v, nc * sizeof(int64_t));
    if (!nv) return -1;
    q->v = nv; q->cap = nc;
  }
  q->v[q->n++] = x;
  return 0;
}

/* Sample one minibatch: writes the raw request list into *res (malloc'd). */
static int sample_one(const int64_t *off, const uint32_t *adj, const int64_t *seeds, uint64_t nseeds,
                      const uint32_t *fanout, int hops, uint64_t key_batch, vec_t *res) {
  vec_t fr = {0, 0, 0};
  for (uint64_t i = 0; i < nseeds; ++i) { if (vpush(res, seeds[i]) || vpush(&fr, seeds[i])) return -1; }
  qsort(fr.v, fr.n, sizeof(int64_t), cmp_i64);
  { uint64_t w = 0; for (uint64_t i = 0; i < fr.n; ++i) if (w == 0 || fr.v[w - 1] != fr.v[i]) fr.v[w++] = fr.v[i]; fr.n = w; }
  for (int h = 0; h < hops; ++h) {
    vec_t nx = {0, 0, 0};
    uint64_t key_hop = sm_key(key_batch, (uint64_t)h);
    for (uint64_t i = 0; i < fr.n; ++i) {
      int64_t v = fr.v[i];
      uint64_t deg = (uint64_t)(off[v + 1] - off[v]);
      uint64_t k = fanout[h] < deg ? fanout[h] : deg;
      if (k == 0) continue;
      uint64_t key_v = sm_key(key_hop, (uint64_t)v);
      uint64_t pos[64];
      uint64_t m = 0;
      if (k == deg) {
        for (uint64_t j = 0; j < deg; ++j) pos[m++] = j;
      } else {
        uint64_t draw = 0;
        for (uint64_t j = deg - k; j < deg; ++j) {
          uint64_t r = below(sm_at(key_v, draw++), j + 1);
          int seen = 0;
          for (uint64_t q = 0; q < m; ++q) if (pos[q] == r) { seen = 1; break; }
          pos[m++] = seen ? j : r;
        }
        for (uint64_t x = 1; x < m; ++x) {  /* ascending position order */
          uint64_t y = pos[x]; int64_t z = (int64_t)x - 1;
          while (z >= 0 && pos[z] > y) { pos[z + 1] = pos[z]; --z; }
          pos[z + 1] = y;
        }
      }
      for (uint64_t q = 0; q < m; ++q) {
        int64_t u = (int64_t)adj[off[v] + (int64_t)pos[q]];
        if (vpush(res, u) || vpush(&nx, u)) return -1;
      }
    }
    free(fr.v);
    qsort(nx.v, nx.n, sizeof(int64_t), cmp_i64);
    uint64_t w = 0;
    for (uint64_t i = 0; i < nx.n; ++i) if (w == 0 || nx.v[w - 1] != nx.v[i]) nx.v[w++] = nx.v[i];
    nx.n = w;
    fr = nx;
  }
  free(fr.v);
  return 0;
}

/*
 * Sample minibatches [b0, b1).  perm holds at least b1*batch_size seed IDs.
 * Pass out == NULL to obtain only the lengths (lens[b-b0]); then call again
 * with out sized to their sum.  fanout has `hops` entries (each <= 64).
 */
int wl_sample(const int64_t *off, const uint32_t *adj, const int64_t *perm, uint64_t batch_size,
              const uint32_t *fanout, int hops, uint64_t seed, uint64_t b0, uint64_t b1,
              uint64_t *lens, int64_t *out) {
  uint64_t nb = b1 - b0;
  for (int h = 0; h < hops; ++h) if (fanout[h] > 64) return -2;
  vec_t *res = (vec_t *)calloc(nb, sizeof(vec_t));
  if (!res) return -1;
  int err = 0;
  uint64_t key = sm_key(seed, LABEL_SAMPLE);
#pragma omp parallel for schedule(dynamic, 1) reduction(| : err)
  for (uint64_t i = 0; i < nb; ++i) {
    uint64_t b = b0 + i;
    err |= sample_one(off, adj, perm + b * batch_size, batch_size, fanout, hops, sm_key(key, b), &res[i]) ? 1 : 0;
  }
  if (!err) {
    uint64_t acc = 0;
    for (uint64_t i = 0; i < nb; ++i) { lens[i] = res[i].n; acc += res[i].n; }
    if (out) {
      uint64_t p = 0;
      for (uint64_t i = 0; i < nb; ++i) { memcpy(out + p, res[i].v, res[i].n * sizeof(int64_t)); p += res[i].n; }
    }
  }
  for (uint64_t i = 0; i < nb; ++i) free(res[i].v);
  free(res);
  return err ? -1 : 0;
}

/* --------------------------------------------------------------- features */
static inline float f_of(uint32_t b) { float f; memcpy(&f, &b, 4); return f; }
static inline uint32_t b_of(float f) { uint32_t b; memcpy(&b, &f, 4); return b; }

/* binary32 -> binary16, round to nearest even, for finite |f| < 65504 (the
   features stay far below it).  Below 2^-14 the result is subnormal: adding
   0.5 (whose unit in the last place is 2^-24, fp16's subnormal step) rounds
   |f| to a multiple of 2^-24 in the float adder, and the sum's low mantissa
   bits are the subnormal's.  Otherwise the exponent is rebiased by 15 - 127
   and the 13 dropped mantissa bits are rounded half to even by adding
   0xfff plus the lowest kept bit before the shift (a carry into the exponent
   is the correct result).  Branch-free, so loops over rows vectorize. */
static inline uint16_t f32_to_f16_rne(float f) {
  const uint32_t x = b_of(f), sign = (x >> 16) & 0x8000u, ax = x & 0x7fffffffu;
  const uint32_t sub = b_of(f_of(ax) + 0.5f) - 0x3f000000u;
  const uint32_t nrm = (ax + 0xc8000fffu + ((ax >> 13) & 1u)) >> 13; /* 0xc8000000 = (15 - 127) << 23 */
  const uint32_t is_sub = 0u - (uint32_t)(ax < 0x38800000u);
  return (uint16_t)(sign | (sub & is_sub) | (nrm & ~is_sub));
}

/* One Box-Muller pair from a 64-bit draw r, in binary32 throughout.
     ln u1:  u1 = m * 2^e with m in [sqrt(1/2), sqrt(2)); ln m = 2 atanh(s),
             s = (m - 1)/(m + 1) (|s| <= 0.172), by its odd series to s^9.
     angle:  w in [0, 2^24) is a fraction w / 2^24 of a turn; q = w / 2^22
             rounded to the nearest integer names the quadrant and
             phi = (w - q 2^22) (pi/2) / 2^22 in [-pi/4, pi/4] the rest;
             sin phi and cos phi by their Taylor series to phi^9 and phi^10,
             then rotated by q quarter turns.
   Truncation errors are below 2e-9, under the binary32 rounding. */
static inline void nrm_pair(uint64_t r, float *x0, float *x1) {
  const float u1 = (float)((uint32_t)(r >> 40) + 1u) * (1.0f / 16777216.0f);
  uint32_t ub = b_of(u1);
  int32_t e = (int32_t)(ub >> 23) - 127;
  uint32_t mb = (ub & 0x007fffffu) | 0x3f800000u;   /* mantissa in [1, 2) */
  const uint32_t big = mb > 0x3fb504f3u;             /* above sqrt(2): halve it */
  mb -= big << 23;
  e += (int32_t)big;
  const float m = f_of(mb), s = (m - 1.0f) / (m + 1.0f), s2 = s * s;
  const float lnm = 2.0f * s * (1.0f + s2 * (1.0f / 3.0f + s2 * (1.0f / 5.0f + s2 * (1.0f / 7.0f + s2 * (1.0f / 9.0f)))));
  const float ln_u1 = (float)e * 0.69314718055994531f + lnm;
  const float rho = sqrtf(-2.0f * ln_u1);

  const int32_t w = (int32_t)((r >> 16) & 0xffffffu);
  const int32_t q = (w + (1 << 21)) >> 22;           /* 0..4 */
  const float phi = (float)(w - (q << 22)) * (1.5707963267948966f / 4194304.0f);
  const float p2 = phi * phi;
  const float sn = phi * (1.0f + p2 * (-1.0f / 6.0f + p2 * (1.0f / 120.0f + p2 * (-1.0f / 5040.0f +
                                                                                 p2 * (1.0f / 362880.0f)))));
  const float cs = 1.0f + p2 * (-0.5f + p2 * (1.0f / 24.0f + p2 * (-1.0f / 720.0f + p2 * (1.0f / 40320.0f +
                                                                                      p2 * (-1.0f / 3628800.0f)))));
  const int32_t qq = q & 3;
  const float c = qq == 0 ? cs : qq == 1 ? -sn : qq == 2 ? -cs : sn;
  const float sv = qq == 0 ? sn : qq == 1 ? cs : qq == 2 ? -sn : -cs;
  *x0 = rho * c;
  *x1 = rho * sv;
}

/* Fill rows [v0, v1) of a feature table; elt_bytes is 4 (fp32) or 2 (fp16).
   `out` points at row v0.  Every row depends only on (seed, v, dim). */
void wl_features(uint64_t dim, int elt_bytes, uint64_t seed, uint64_t v0, uint64_t v1, void *out) {
  const uint64_t key = sm_key(seed, LABEL_FEAT);
  const uint64_t pairs = (dim + 1) / 2;
#pragma omp parallel
  {
    float *tmp = (float *)malloc(2 * pairs * sizeof(float));
#pragma omp for schedule(static)
    for (uint64_t v = v0; v < v1; ++v) {
      const uint64_t c0 = v * pairs;
      for (uint64_t j = 0; j < pairs; ++j) nrm_pair(sm_at(key, c0 + j), &tmp[2 * j], &tmp[2 * j + 1]);
      if (elt_bytes == 4) {
        memcpy((float *)out + (v - v0) * dim, tmp, dim * sizeof(float));
      } else {
        uint16_t *o = (uint16_t *)out + (v - v0) * dim;
        for (uint64_t k = 0; k < dim; ++k) o[k] = f32_to_f16_rne(tmp[k]);
      }
    }
    free(tmp);
  }
}

/* exported for the generator's own tests: the binary16 rounding */
void wl_f32_to_f16(const float *in, uint16_t *out, uint64_t n) {
  for (uint64_t i = 0; i < n; ++i) out[i] = f32_to_f16_rne(in[i]);
}
