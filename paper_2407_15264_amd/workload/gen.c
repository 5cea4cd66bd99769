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
 *   Features: x[v][k] = sqrt(-2 ln u1) cos(2 pi u2) (Box-Muller) with u1, u2
 *   from the stream keyed by the feature seed at counters 2(v*dim+k) and
 *   2(v*dim+k)+1; rounded to fp32, and for fp16 further rounded from fp32 to
 *   binary16 with round-to-nearest-even.
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

  const uint64_t CH = 1ULL << 16;  /* attempts per chunk */
  const int NCH = 256;             /* chunks per round */
  uint64_t *cnt = (uint64_t *)malloc(NCH * sizeof(uint64_t));
  uint64_t got = 0, base = 0;
  while (got < e) {
#pragma omp parallel for schedule(dynamic, 1)
    for (int ci = 0; ci < NCH; ++ci) {
      uint64_t k0 = base + (uint64_t)ci * CH, m = 0;
      uint32_t s, d;
      for (uint64_t k = k0; k < k0 + CH; ++k) m += (uint64_t)rmat_attempt(key, k, scale, a, ab, abc, n, &s, &d);
      cnt[ci] = m;
    }
    uint64_t pos[256];
    uint64_t acc = got;
    for (int ci = 0; ci < NCH; ++ci) { pos[ci] = acc; acc += cnt[ci]; }
#pragma omp parallel for schedule(dynamic, 1)
    for (int ci = 0; ci < NCH; ++ci) {
      uint64_t p = pos[ci];
      if (p >= e) continue;
      uint64_t k0 = base + (uint64_t)ci * CH;
      uint32_t s, d;
      for (uint64_t k = k0; k < k0 + CH && p < e; ++k)
        if (rmat_attempt(key, k, scale, a, ab, abc, n, &s, &d)) { src[p] = s; dst[p] = d; ++p; }
    }
    got = acc < e ? acc : e;
    base += (uint64_t)NCH * CH;
  }
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
static inline uint16_t f32_to_f16_rne(float f) {
  uint32_t x;
  memcpy(&x, &f, 4);
  uint32_t sign = (x >> 16) & 0x8000u;
  uint32_t ex = (x >> 23) & 0xffu;
  uint32_t man = x & 0x7fffffu;
  if (ex == 0xffu) return (uint16_t)(sign | 0x7c00u | (man ? 0x200u : 0));
  int32_t e = (int32_t)ex - 127 + 15;
  if (e >= 31) return (uint16_t)(sign | 0x7c00u);
  if (e <= 0) {
    if (e < -10) return (uint16_t)sign;
    man |= 0x800000u;
    uint32_t shift = (uint32_t)(14 - e);
    uint32_t h = man >> shift;
    uint32_t rem = man & ((1u << shift) - 1), half = 1u << (shift - 1);
    if (rem > half || (rem == half && (h & 1u))) ++h;
    return (uint16_t)(sign | h);
  }
  uint32_t h = ((uint32_t)e << 10) | (man >> 13);
  uint32_t rem = man & 0x1fffu;
  if (rem > 0x1000u || (rem == 0x1000u && (h & 1u))) ++h;
  return (uint16_t)(sign | h);
}

/* Fill rows [v0, v1) of a feature table; elt_bytes is 4 (fp32) or 2 (fp16).
   `out` points at row v0. */
void wl_features(uint64_t dim, int elt_bytes, uint64_t seed, uint64_t v0, uint64_t v1, void *out) {
  uint64_t key = sm_key(seed, LABEL_FEAT);
  const double two_pi = 6.283185307179586476925286766559;
#pragma omp parallel for schedule(static)
  for (uint64_t v = v0; v < v1; ++v) {
    for (uint64_t k = 0; k < dim; ++k) {
      uint64_t c = 2 * (v * dim + k);
      double u1 = u01(sm_at(key, c)) + (1.0 / 9007199254740992.0); /* (0, 1] */
      double u2 = u01(sm_at(key, c + 1));
      float x = (float)(sqrt(-2.0 * log(u1)) * cos(two_pi * u2));
      if (elt_bytes == 4) ((float *)out)[(v - v0) * dim + k] = x;
      else ((uint16_t *)out)[(v - v0) * dim + k] = f32_to_f16_rne(x);
    }
  }
}
