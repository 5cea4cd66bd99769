/*
 * CPU ORACLE for the static score -- TEST INFRASTRUCTURE ONLY.
 *
 * The static information of the hybrid policy (Sec. 4.2; the evaluation's
 * static policy, Sec. 5) is a normalized reverse PageRank.  Reading used here
 * (listed in the design notes): the graph is the sampling adjacency in CSR
 * form, where node u lists the neighbours it samples, which is the reverse of
 * the direction in which features flow in message passing.  The walk moves
 * from u to one of its CSR entries chosen uniformly (a repeated entry counts
 * each time) with probability d and jumps to a uniformly chosen node
 * otherwise; a node with no entries always jumps.  Its PageRank is approached
 * by K power iterations from the uniform vector:
 *
 *   r'(v) = (1 - d)/N + d * ( sum over CSR entries u->v of r(u)/deg(u)
 *                             + (sum over nodes w with deg(w) = 0 of r(w)) / N )
 *
 * The score is the rank normalized by the largest rank and quantized to 32
 * bits: floor(r(v) / max r * (2^32 - 1)).
 *
 * Plain sequential double-precision loops in the order of the formula.
 */
#include "oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>

int orc_pagerank(uint64_t N, const int64_t *offsets, const uint32_t *adj, double d, uint32_t K, double *rank) {
  if (N == 0 || !offsets || !rank || !(d >= 0.0 && d < 1.0)) return ORC_E_INVAL;
  if (offsets[0] != 0) return ORC_E_INVAL;
  for (uint64_t u = 0; u < N; ++u)
    if (offsets[u + 1] < offsets[u]) return ORC_E_INVAL;
  const int64_t E = offsets[N];
  if (E > 0 && !adj) return ORC_E_INVAL;
  for (int64_t e = 0; e < E; ++e)
    if (adj[e] >= N) return ORC_E_RANGE;
  double *next = (double *)malloc(N * sizeof(double));
  if (!next) return ORC_E_NOMEM;
  for (uint64_t v = 0; v < N; ++v) rank[v] = 1.0 / (double)N;
  for (uint32_t k = 0; k < K; ++k) {
    double dangling = 0.0;
    for (uint64_t v = 0; v < N; ++v) next[v] = 0.0;
    for (uint64_t u = 0; u < N; ++u) {
      const int64_t deg = offsets[u + 1] - offsets[u];
      if (deg == 0) {
        dangling += rank[u];
        continue;
      }
      const double share = rank[u] / (double)deg;
      for (int64_t e = offsets[u]; e < offsets[u + 1]; ++e) next[adj[e]] += share;
    }
    for (uint64_t v = 0; v < N; ++v) rank[v] = (1.0 - d) / (double)N + d * (next[v] + dangling / (double)N);
  }
  free(next);
  return ORC_OK;
}

int orc_rank_scores(uint64_t N, const double *rank, uint32_t *score) {
  if (N == 0 || !rank || !score) return ORC_E_INVAL;
  double mx = 0.0;
  for (uint64_t v = 0; v < N; ++v)
    if (rank[v] > mx) mx = rank[v];
  if (!(mx > 0.0)) return ORC_E_INVAL;
  for (uint64_t v = 0; v < N; ++v) score[v] = (uint32_t)floor(rank[v] / mx * 4294967295.0);
  return ORC_OK;
}
