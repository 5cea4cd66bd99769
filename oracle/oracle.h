/*
 * CPU ORACLE for the LSM-GNN feature-gather cache -- TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow, sequential definition of what the GPU library computes.  Only
 * the test suite, the smoke check and the benchmark's CPU-baseline leg may
 * load it; the GPU product path never calls it and shares no code with it.
 *
 * Paper: Kim et al., "LSM-GNN: Large-scale Storage-based Multi-GPU GNN Training
 * by Optimizing Data Transfer Scheme" (arXiv 2407.15264).
 *   - software cache, set associative, serving the sampled-node list: Sec. 4
 *     (system design overview) and Sec. 4.1
 *   - window of upcoming minibatches and next-reuse information: Sec. 4.2
 *   - hybrid eviction with four priority levels and static tie-break: Sec. 4.2
 *   - victim buffer (PVP) enqueue of lines that carry reuse information, and
 *     the swap of the two lowest levels when it is enabled: Sec. 4.3.1, 4.3.2
 *
 * Status codes carry the same numbers as the GPU library's, but are declared
 * here independently.
 */
#ifndef LSMGNN_ORACLE_H
#define LSMGNN_ORACLE_H
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
  ORC_OK = 0,
  ORC_E_INVAL = 1,
  ORC_E_RANGE = 2,
  ORC_E_WINDOW = 3,
  ORC_E_NOMEM = 4
};

/* per-unique outcome codes */
enum { ORC_HIT = 0, ORC_VICTIM_HIT = 1, ORC_MISS = 2 };

/* eviction policies compared in the paper's evaluation (Sec. 5, impact of the
   cache eviction policy): hybrid (Sec. 4.2), static information only, dynamic
   information only, round-robin */
enum { ORC_POLICY_HYBRID = 0, ORC_POLICY_STATIC = 1, ORC_POLICY_DYNAMIC = 2, ORC_POLICY_ROUND_ROBIN = 3 };

/* victim buffer forms: one FIFO ring, or per-reuse-iteration queues with
   prefetch (Sec. 4.3.1) */
enum { ORC_VICTIM_FIFO = 0, ORC_VICTIM_QUEUES = 1 };

typedef struct orc_cache orc_cache;

typedef struct {
  uint64_t batch, requests, unique, hits, victim_hits, misses, evictions, enqueued, dropped;
  /* the same outcomes counted per raw request (a repeated ID counts each time) */
  uint64_t request_hits, request_victim_hits;
} orc_counts;

/* set index of node x in a cache of num_sets sets */
uint64_t orc_set_of(uint64_t x, uint64_t num_sets);

/* store may be NULL: gather then skips row copies (metadata-only runs) */
int orc_create(uint64_t num_nodes, uint32_t row_bytes, const void *store, const uint32_t *static_score,
               uint64_t num_sets, uint32_t ways, uint64_t victim_rows, uint32_t lookahead,
               uint32_t near_threshold, uint32_t policy, uint32_t victim_mode, uint32_t refresh_period,
               orc_cache **out);
void orc_destroy(orc_cache *c);
int orc_advance(orc_cache *c, const int64_t *ids, uint64_t n);
/* out (U rows), uniq (U), inv (n), outcome (U) may each be NULL */
int orc_gather(orc_cache *c, const int64_t *ids, uint64_t n, void *out, int64_t *uniq, int64_t *inv,
               uint8_t *outcome, uint64_t *n_unique);
int orc_stats(const orc_cache *c, orc_counts *last, orc_counts *total);
/* tags: num_sets*ways entries, ring_tags: victim_rows entries (either may be NULL) */
int orc_export_state(const orc_cache *c, uint32_t *tags, uint32_t *ring_tags, uint64_t *ring_tail, uint64_t *t);

/* Static score (pagerank.c): K power iterations of the PageRank of the walk
   along CSR entries (offsets[N+1], adj[offsets[N]]) with damping d, from the
   uniform vector, dangling mass spread uniformly; rank[N] receives it.
   orc_rank_scores: floor(rank / max rank * (2^32 - 1)). */
int orc_pagerank(uint64_t N, const int64_t *offsets, const uint32_t *adj, double d, uint32_t K, double *rank);
int orc_rank_scores(uint64_t N, const double *rank, uint32_t *score);
uint32_t orc_near_threshold(const orc_cache *c);

#ifdef __cplusplus
}
#endif
#endif
