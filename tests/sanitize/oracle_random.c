/* Random driver of the C oracle (every policy, victim form and update period,
   rare out-of-range IDs, the static-score PageRank), built with the address and
   undefined-behaviour sanitizers by tests/test_sanitizers.py. */
#include <stdio.h>
#include <stdlib.h>
#include <string.h>
#include "oracle.h"
static uint64_t st = 88172645463325252ull;
static uint64_t rnd(void) { st ^= st << 13; st ^= st >> 7; st ^= st << 17; return st; }
int main(int argc, char **argv) {
  int cases = argc > 1 ? atoi(argv[1]) : 2000;
  for (int cs = 0; cs < cases; ++cs) {
    uint64_t N = 1 + rnd() % 300, S = 1 + rnd() % 9, ways = 1 + rnd() % 8, L = rnd() % 10, V = rnd() % 40;
    uint32_t pol = rnd() % 4, vm = rnd() % 2, U = 1 + rnd() % 5, R = 16 * (1 + rnd() % 3);
    if (vm && V && V < L + 1) V = L + 1;
    uint32_t *stat = malloc(N * 4);
    unsigned char *store = malloc(N * R);
    for (uint64_t i = 0; i < N; ++i) stat[i] = rnd() % 7;
    for (uint64_t i = 0; i < N * R; ++i) store[i] = (unsigned char)rnd();
    orc_cache *c = NULL;
    if (orc_create(N, R, store, stat, S, (uint32_t)ways, V, (uint32_t)L, (uint32_t)(rnd() % 3), pol, vm, U, &c)) {
      printf("create failed\n");
      return 1;
    }
    int nb = 1 + rnd() % 30;
    int64_t ids[200];
    for (uint64_t j = 0; j <= L; ++j) {
      uint64_t n = rnd() % 60;
      for (uint64_t i = 0; i < n; ++i) ids[i] = (int64_t)(rnd() % N);
      orc_advance(c, ids, n);
    }
    for (int b = 0; b < nb; ++b) {
      uint64_t n = rnd() % 200;
      for (uint64_t i = 0; i < n; ++i) ids[i] = (int64_t)(rnd() % (N + (rnd() % 50 == 0)));  /* rare bad ID */
      unsigned char *out = malloc((n ? n : 1) * R);
      int64_t uq[200], inv[200];
      uint8_t oc[200];
      uint64_t U2 = 0;
      orc_gather(c, ids, n, out, uq, inv, oc, &U2);
      free(out);
      uint64_t m = rnd() % 60;
      for (uint64_t i = 0; i < m; ++i) ids[i] = (int64_t)(rnd() % N);
      orc_advance(c, ids, m);
      orc_counts last, tot;
      orc_stats(c, &last, &tot);
    }
    uint32_t *tags = malloc(S * ways * 4), *rt = malloc((V ? V : 1) * 4);
    uint64_t tail, t;
    orc_export_state(c, tags, rt, &tail, &t);
    free(tags); free(rt);
    orc_destroy(c);
    /* pagerank on a random graph */
    uint64_t E = rnd() % (4 * N + 1);
    int64_t *off = malloc((N + 1) * 8);
    uint32_t *adj = malloc((E ? E : 1) * 4);
    off[0] = 0;
    for (uint64_t u = 0; u < N; ++u) off[u + 1] = off[u] + (u + 1 == N ? (int64_t)(E - (uint64_t)off[u]) : (int64_t)(rnd() % (E / N + 2) > E - (uint64_t)off[u] ? 0 : rnd() % (E / N + 2)));
    if ((uint64_t)off[N] != E) off[N] = (int64_t)E;
    for (uint64_t e = 0; e < E; ++e) adj[e] = (uint32_t)(rnd() % N);
    double *rk = malloc(N * 8);
    uint32_t *sc = malloc(N * 4);
    if (orc_pagerank(N, off, adj, 0.85, (uint32_t)(rnd() % 20), rk) == ORC_OK) orc_rank_scores(N, rk, sc);
    free(off); free(adj); free(rk); free(sc);
    free(stat); free(store);
  }
  printf("sanitized oracle run ok: %d cases\n", cases);
  return 0;
}
