/*
 * CPU ORACLE for the LSM-GNN feature-gather cache -- TEST INFRASTRUCTURE ONLY.
 * Plain sequential C; every step follows the definition in the order the
 * paper's design section gives it (citations per function).  No blocking, no
 * parallelism, no shared code with the GPU library.
 *
 * Readings of points the paper leaves open (each is listed in the design notes
 * of the repository):
 *   - requests are deduplicated and served in ascending node-ID order;
 *   - the output holds one row per unique ID, ascending, plus an inverse index;
 *   - set(x) = fastrange(high 32 bits of SplitMix64(x), S): the output of a
 *     SplitMix64 generator seeded with x, reduced with Lemire's multiply-shift;
 *   - reuse "dynamic value" is read as the distance d from the current gather to
 *     the next announced use; d <= T is the kept "near" level, T < d <= L the
 *     "far" level; T defaults to max(1, floor(L/8));
 *   - the dynamic information (each resident line's next reuse iteration) is
 *     updated before every U-th gather (U = 1 by default: exact at every
 *     gather), from the lists announced by then; a line inserted since the
 *     last update has none ("recently inserted"), and a recorded reuse
 *     iteration that has passed counts as recently used, the same level;
 *   - ties at equal level and equal static score go to the lowest way index,
 *     and empty ways are always filled first, lowest index first;
 *   - the victim buffer is one FIFO ring of V entries that overwrites its
 *     oldest entry; lines in the far or near level are enqueued, others are
 *     dropped; a victim hit removes the entry and refills the line through the
 *     normal fill path; V > 0 turns on the swapped (PVP) level order.
 * The victim buffer may instead take the form of Sec. 4.3.1's per-iteration
 * queues (victim_mode ORC_VICTIM_QUEUES): queue j holds lines evicted with
 * next reuse iteration j, at most C = V / (L + 1) of them in eviction order
 * (a line finding its queue full is dropped); while minibatch t is gathered,
 * a requested node that queue t holds is a victim hit (its row having been
 * prefetched, Sec. 4.3), and after the gather queue t is emptied.  Queues are
 * kept in L + 1 slots, slot j mod (L + 1).
 * The other policies of the evaluation (Sec. 5) choose the victim among the
 * full set's lines differently and keep everything else: static-only evicts
 * the lowest static score; dynamic-only evicts the line whose next announced
 * use is furthest away (no announced use first); round-robin evicts the way a
 * per-set pointer names and then advances the pointer.  Ties go to the lowest
 * way index in every policy.
 */
#include "oracle.h"

#include <stdlib.h>
#include <string.h>

#define EMPTY 0xffffffffu

/* dynamic classes of a resident line */
enum { CLS_N = 0, CLS_F = 1, CLS_R = 2, CLS_C = 3 };

typedef struct {
  int64_t *ids; /* sorted, unique */
  uint64_t n;
} ann_list;

struct orc_cache {
  uint64_t num_nodes, num_sets, victim_rows;
  uint32_t row_bytes, ways, lookahead, near_thr, policy, vmode, period;
  uint64_t t_upd;    /* gather index of the last update of the dynamic information */
  uint32_t upd;      /* number of updates so far */
  uint32_t *seen;    /* [num_nodes] the update at which `first` was last written */
  int64_t *first;    /* [num_nodes] at that update, the node's first announced use in the window */
  uint64_t qcap, nslots; /* queue mode: rows per queue, queue slots */
  uint64_t *qcnt;        /* [nslots] entries in each queue */
  uint32_t *qbits;       /* [num_nodes] bit k: the node has an entry in slot k */
  uint32_t *rr;      /* [num_sets] round-robin pointer (next way to evict) */
  const unsigned char *store;
  uint32_t *stat;    /* static score per node (copied) */
  uint32_t *tag;     /* [num_sets][ways] */
  int64_t *ins;      /* [num_sets][ways] gather index at insertion */
  uint32_t *vtag;    /* [victim_rows] ring entries, or queue slot k's entries at k * qcap */
  int64_t *where;    /* [num_nodes] ring slot holding the node, or -1 */
  uint64_t tail;     /* total enqueues ever */
  ann_list *ann;     /* announced batches, index j */
  uint64_t n_ann, cap_ann;
  uint64_t t;        /* completed gathers */
  orc_counts last, total;
};

/* SplitMix64 (Steele, Lea, Flood 2014): first output of the generator whose
   state is x, then Lemire's fastrange on its high 32 bits. */
uint64_t orc_set_of(uint64_t x, uint64_t num_sets) {
  uint64_t z = x + 0x9e3779b97f4a7c15ULL;
  z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ULL;
  z = (z ^ (z >> 27)) * 0x94d049bb133111ebULL;
  z = z ^ (z >> 31);
  return ((z >> 32) * num_sets) >> 32;
}

static int cmp_i64(const void *a, const void *b) {
  int64_t x = *(const int64_t *)a, y = *(const int64_t *)b;
  return (x > y) - (x < y);
}

/* sorted unique copy of ids */
static int64_t *sorted_unique(const int64_t *ids, uint64_t n, uint64_t *m) {
  int64_t *u = (int64_t *)malloc((n ? n : 1) * sizeof(int64_t));
  if (!u) return NULL;
  memcpy(u, ids, n * sizeof(int64_t));
  qsort(u, n, sizeof(int64_t), cmp_i64);
  uint64_t w = 0;
  for (uint64_t i = 0; i < n; ++i)
    if (w == 0 || u[w - 1] != u[i]) u[w++] = u[i];
  *m = w;
  return u;
}

int orc_create(uint64_t num_nodes, uint32_t row_bytes, const void *store, const uint32_t *static_score,
               uint64_t num_sets, uint32_t ways, uint64_t victim_rows, uint32_t lookahead,
               uint32_t near_threshold, uint32_t policy, uint32_t victim_mode, uint32_t refresh_period,
               orc_cache **out) {
  if (!out || !static_score) return ORC_E_INVAL;
  *out = NULL;
  if (num_nodes == 0 || num_nodes > 0xffffffffULL || row_bytes == 0 || row_bytes % 16 != 0 ||
      num_sets == 0 || num_sets > 0xffffffffULL || ways == 0 || lookahead > 31 || policy > ORC_POLICY_ROUND_ROBIN ||
      victim_mode > ORC_VICTIM_QUEUES)
    return ORC_E_INVAL;
  /* queue mode needs room for at least one entry per queue */
  if (victim_mode == ORC_VICTIM_QUEUES && victim_rows && victim_rows < (uint64_t)lookahead + 1) return ORC_E_INVAL;
  orc_cache *c = (orc_cache *)calloc(1, sizeof(orc_cache));
  if (!c) return ORC_E_NOMEM;
  c->num_nodes = num_nodes;
  c->num_sets = num_sets;
  c->victim_rows = victim_rows;
  c->row_bytes = row_bytes;
  c->ways = ways;
  c->lookahead = lookahead;
  c->policy = policy;
  c->vmode = victim_mode;
  c->period = refresh_period ? refresh_period : 1;
  c->nslots = (uint64_t)lookahead + 1;
  c->qcap = victim_mode == ORC_VICTIM_QUEUES ? victim_rows / c->nslots : 0;
  /* Sec. 4.2: the default threshold is one eighth of the window; at least 1 */
  c->near_thr = near_threshold ? near_threshold : (lookahead / 8 > 1 ? lookahead / 8 : 1);
  c->store = (const unsigned char *)store;
  c->stat = (uint32_t *)malloc(num_nodes * sizeof(uint32_t));
  c->tag = (uint32_t *)malloc(num_sets * ways * sizeof(uint32_t));
  c->ins = (int64_t *)malloc(num_sets * ways * sizeof(int64_t));
  c->vtag = (uint32_t *)malloc((victim_rows ? victim_rows : 1) * sizeof(uint32_t));
  c->where = (int64_t *)malloc(num_nodes * sizeof(int64_t));
  c->rr = (uint32_t *)calloc(num_sets, sizeof(uint32_t));
  c->qcnt = (uint64_t *)calloc(c->nslots, sizeof(uint64_t));
  c->qbits = (uint32_t *)calloc(num_nodes, sizeof(uint32_t));
  c->seen = (uint32_t *)calloc(num_nodes, sizeof(uint32_t));
  c->first = (int64_t *)malloc(num_nodes * sizeof(int64_t));
  if (!c->stat || !c->tag || !c->ins || !c->vtag || !c->where || !c->rr || !c->qcnt || !c->qbits || !c->seen ||
      !c->first) {
    orc_destroy(c);
    return ORC_E_NOMEM;
  }
  memcpy(c->stat, static_score, num_nodes * sizeof(uint32_t));
  for (uint64_t i = 0; i < num_sets * ways; ++i) { c->tag[i] = EMPTY; c->ins[i] = -1; }
  for (uint64_t k = 0; k < victim_rows; ++k) c->vtag[k] = EMPTY;
  for (uint64_t v = 0; v < num_nodes; ++v) c->where[v] = -1;
  *out = c;
  return ORC_OK;
}

void orc_destroy(orc_cache *c) {
  if (!c) return;
  for (uint64_t j = 0; j < c->n_ann; ++j) free(c->ann[j].ids);
  free(c->ann);
  free(c->stat); free(c->tag); free(c->ins); free(c->vtag); free(c->where); free(c->rr);
  free(c->qcnt); free(c->qbits); free(c->seen); free(c->first);
  free(c);
}

uint32_t orc_near_threshold(const orc_cache *c) { return c->near_thr; }

/* Window buffering (Sec. 4, overview; Sec. 4.2): the k-th call announces the
   sampled list of minibatch k.  At most L minibatches beyond the current one
   may be known ahead. */
int orc_advance(orc_cache *c, const int64_t *ids, uint64_t n) {
  if (!c || (n && !ids)) return ORC_E_INVAL;
  uint64_t j = c->n_ann;
  if (j > c->t + c->lookahead) return ORC_E_WINDOW;
  for (uint64_t i = 0; i < n; ++i)
    if (ids[i] < 0 || (uint64_t)ids[i] >= c->num_nodes) return ORC_E_RANGE;
  if (c->n_ann == c->cap_ann) {
    uint64_t nc = c->cap_ann ? 2 * c->cap_ann : 64;
    ann_list *na = (ann_list *)realloc(c->ann, nc * sizeof(ann_list));
    if (!na) return ORC_E_NOMEM;
    c->ann = na;
    c->cap_ann = nc;
  }
  ann_list l = {NULL, 0};
  if (j > c->t) { /* a list for a minibatch already being served is never consulted */
    l.ids = sorted_unique(ids, n, &l.n);
    if (!l.ids) return ORC_E_NOMEM;
  }
  c->ann[c->n_ann++] = l;
  return ORC_OK;
}

/* The update of the dynamic information (Sec. 4.2), run before every U-th
   gather: every resident line's next reuse iteration from the announced lists
   of the next L minibatches.  Kept per node (the first of those lists that
   names it, found by walking the lists in order), which is what each resident
   line records: a line inserted later has no record (it counts as recently
   inserted), so a per-node value frozen at the update is all a line reads. */
static void update_reuse(orc_cache *c) {
  c->t_upd = c->t;
  ++c->upd;
  for (uint64_t j = c->t + 1; j <= c->t + c->lookahead && j < c->n_ann; ++j)
    for (uint64_t k = 0; k < c->ann[j].n; ++k) {
      uint32_t x = (uint32_t)c->ann[j].ids[k];
      if (c->seen[x] != c->upd) {
        c->seen[x] = c->upd;
        c->first[x] = (int64_t)j;
      }
    }
}

/* The next reuse iteration recorded for the line in way w of set s at the
   last update, or -1 (none) */
static int64_t recorded_reuse(const orc_cache *c, uint64_t i) {
  uint32_t x = c->tag[i];
  return (x != EMPTY && c->seen[x] == c->upd) ? c->first[x] : -1;
}

/* Dynamic information (Sec. 4.2): the class of the line in way w of set s while
   gather t is served.  A line inserted since the last update has no reuse
   information ("recently inserted"); so is treated a line whose recorded
   reuse iteration has passed.  Otherwise, with d the distance to the recorded
   reuse iteration: none -> no reuse; d <= T -> near; T < d -> far. */
static int line_class(const orc_cache *c, uint64_t s, uint32_t w) {
  uint64_t i = s * c->ways + w;
  if (c->ins[i] >= (int64_t)c->t_upd) return CLS_R;
  int64_t r = recorded_reuse(c, i);
  if (r < 0) return CLS_N;
  if (r <= (int64_t)c->t) return CLS_R;
  return (uint64_t)(r - (int64_t)c->t) <= c->near_thr ? CLS_C : CLS_F;
}

/* The dynamic-only policy's view (Sec. 5): the distance to the line's recorded
   reuse iteration, or 0 (no expected reuse) when it has none, it has passed,
   or the line was inserted since the last update. */
static uint64_t line_distance(const orc_cache *c, uint64_t s, uint32_t w) {
  uint64_t i = s * c->ways + w;
  int64_t r = recorded_reuse(c, i);
  if (c->ins[i] >= (int64_t)c->t_upd || r <= (int64_t)c->t) return 0;
  return (uint64_t)(r - (int64_t)c->t);
}

/* Eviction priority, lowest level evicted first.  Hybrid order (Sec. 4.2):
   no reuse < far < recently inserted < near.  With the victim buffer enabled the
   two lowest levels swap (Sec. 4.3.2): far < no reuse < recent < near. */
static int level_of(const orc_cache *c, int cls) {
  if (c->victim_rows > 0) {
    switch (cls) {
      case CLS_F: return 0;
      case CLS_N: return 1;
      case CLS_R: return 2;
      default: return 3;
    }
  }
  switch (cls) {
    case CLS_N: return 0;
    case CLS_F: return 1;
    case CLS_R: return 2;
    default: return 3;
  }
}

static void ring_put(orc_cache *c, uint64_t k, uint32_t v) {
  if (c->vtag[k] != EMPTY) c->where[c->vtag[k]] = -1;
  c->vtag[k] = v;
  if (v != EMPTY) c->where[v] = (int64_t)k;
}

/* Feature aggregation of one minibatch through the cache (Sec. 4 overview,
   Sec. 4.2, Sec. 4.3.1). */
int orc_gather(orc_cache *c, const int64_t *ids, uint64_t n, void *out, int64_t *uniq_out, int64_t *inv,
               uint8_t *outcome, uint64_t *n_unique) {
  if (!c || (n && !ids)) return ORC_E_INVAL;
  for (uint64_t i = 0; i < n; ++i)
    if (ids[i] < 0 || (uint64_t)ids[i] >= c->num_nodes) return ORC_E_RANGE;

  uint64_t U = 0;
  int64_t *uniq = sorted_unique(ids, n, &U);
  if (!uniq) return ORC_E_NOMEM;
  uint8_t *oc = (uint8_t *)malloc(U ? U : 1); /* each unique ID's outcome */
  if (!oc) {
    free(uniq);
    return ORC_E_NOMEM;
  }
  if (c->t % c->period == 0) update_reuse(c);
  orc_counts st;
  memset(&st, 0, sizeof st);
  st.batch = c->t;
  st.requests = n;
  st.unique = U;

  for (uint64_t u = 0; u < U; ++u) {
    uint32_t x = (uint32_t)uniq[u];
    uint64_t s = orc_set_of(x, c->num_sets);
    uint32_t *tag = c->tag + s * c->ways;
    int64_t *ins = c->ins + s * c->ways;
    int hit = 0;
    for (uint32_t w = 0; w < c->ways; ++w)
      if (tag[w] == x) hit = 1;
    if (hit) {
      ++st.hits;
      oc[u] = ORC_HIT;
    } else {
      /* the victim buffer is probed for the line before storage (Sec. 4.3);
         in queue mode only the current iteration's queue holds rows */
      if (c->vmode == ORC_VICTIM_QUEUES && c->qcap && ((c->qbits[x] >> (c->t % c->nslots)) & 1u)) {
        ++st.victim_hits;
        oc[u] = ORC_VICTIM_HIT;
      } else if (c->vmode == ORC_VICTIM_FIFO && c->victim_rows && c->where[x] >= 0) {
        ++st.victim_hits;
        ring_put(c, (uint64_t)c->where[x], EMPTY);
        oc[u] = ORC_VICTIM_HIT;
      } else {
        ++st.misses;
        oc[u] = ORC_MISS;
      }
      /* choose the way: an empty way first; in a full set the policy's
         victim (Sec. 4.2 for the hybrid; Sec. 5 for the others) */
      uint32_t pick = c->ways;
      for (uint32_t w = 0; w < c->ways && pick == c->ways; ++w)
        if (tag[w] == EMPTY) pick = w;
      if (pick == c->ways) {
        if (c->policy == ORC_POLICY_HYBRID) {
          /* the lowest level, then the lowest static score, then the lowest way */
          int best_lvl = 99;
          uint32_t best_stat = 0;
          for (uint32_t w = 0; w < c->ways; ++w) {
            int lvl = level_of(c, line_class(c, s, w));
            uint32_t sv = c->stat[tag[w]];
            if (lvl < best_lvl || (lvl == best_lvl && sv < best_stat)) {
              best_lvl = lvl;
              best_stat = sv;
              pick = w;
            }
          }
        } else if (c->policy == ORC_POLICY_STATIC) {
          /* the lowest static score, then the lowest way */
          for (uint32_t w = 0; w < c->ways; ++w)
            if (pick == c->ways || c->stat[tag[w]] < c->stat[tag[pick]]) pick = w;
        } else if (c->policy == ORC_POLICY_DYNAMIC) {
          /* no announced use first, then the furthest next use, then the lowest way */
          uint64_t best = 0;
          for (uint32_t w = 0; w < c->ways; ++w) {
            uint64_t d = line_distance(c, s, w);
            uint64_t far = d ? d : c->lookahead + 1;
            if (pick == c->ways || far > best) {
              best = far;
              pick = w;
            }
          }
        } else {
          /* round-robin: the way the set's pointer names; the pointer advances */
          pick = c->rr[s];
          c->rr[s] = (c->rr[s] + 1) % c->ways;
        }
        /* evict: a line with reuse information goes to the victim buffer,
           others are discarded (Sec. 4.3.1) */
        uint32_t z = tag[pick];
        int cls = line_class(c, s, pick);
        ++st.evictions;
        if (c->vmode == ORC_VICTIM_QUEUES && c->qcap && (cls == CLS_F || cls == CLS_C)) {
          /* the queue of the line's next reuse iteration, unless it is full */
          uint64_t slot = (uint64_t)recorded_reuse(c, s * c->ways + pick) % c->nslots;
          if (c->qcnt[slot] < c->qcap) {
            c->vtag[slot * c->qcap + c->qcnt[slot]] = z;
            ++c->qcnt[slot];
            c->qbits[z] |= 1u << slot;
            ++c->tail;
            ++st.enqueued;
          } else {
            ++st.dropped;
          }
        } else if (c->vmode == ORC_VICTIM_FIFO && c->victim_rows && (cls == CLS_F || cls == CLS_C)) {
          ring_put(c, c->tail % c->victim_rows, z);
          ++c->tail;
          ++st.enqueued;
        } else {
          ++st.dropped;
        }
      }
      tag[pick] = x;
      ins[pick] = (int64_t)c->t;
    }
    /* every served row is the stored row of its node, whatever path served it */
    if (out && c->store)
      memcpy((unsigned char *)out + u * c->row_bytes, c->store + (uint64_t)x * c->row_bytes, c->row_bytes);
  }

  if (uniq_out) memcpy(uniq_out, uniq, U * sizeof(int64_t));
  if (outcome) memcpy(outcome, oc, U);
  /* each request takes its unique ID's outcome */
  for (uint64_t i = 0; i < n; ++i) {
    int64_t *p = (int64_t *)bsearch(&ids[i], uniq, U, sizeof(int64_t), cmp_i64);
    if (inv) inv[i] = p - uniq;
    if (oc[p - uniq] == ORC_HIT) ++st.request_hits;
    if (oc[p - uniq] == ORC_VICTIM_HIT) ++st.request_victim_hits;
  }
  free(oc);
  free(uniq);
  if (n_unique) *n_unique = U;

  /* queue mode: the current iteration's queue has been served */
  if (c->vmode == ORC_VICTIM_QUEUES && c->qcap) {
    uint64_t slot = c->t % c->nslots;
    for (uint64_t p = 0; p < c->qcnt[slot]; ++p) {
      c->qbits[c->vtag[slot * c->qcap + p]] &= ~(1u << slot);
      c->vtag[slot * c->qcap + p] = EMPTY;
    }
    c->qcnt[slot] = 0;
  }
  /* lists of minibatches up to t are never consulted again */
  if (c->t < c->n_ann) {
    free(c->ann[c->t].ids);
    c->ann[c->t].ids = NULL;
    c->ann[c->t].n = 0;
  }
  c->last = st;
  c->total.batch = st.batch + 1;
  c->total.requests += st.requests;
  c->total.unique += st.unique;
  c->total.hits += st.hits;
  c->total.victim_hits += st.victim_hits;
  c->total.misses += st.misses;
  c->total.evictions += st.evictions;
  c->total.enqueued += st.enqueued;
  c->total.dropped += st.dropped;
  c->total.request_hits += st.request_hits;
  c->total.request_victim_hits += st.request_victim_hits;
  ++c->t;
  return ORC_OK;
}

int orc_stats(const orc_cache *c, orc_counts *last, orc_counts *total) {
  if (!c) return ORC_E_INVAL;
  if (last) *last = c->last;
  if (total) *total = c->total;
  return ORC_OK;
}

int orc_export_state(const orc_cache *c, uint32_t *tags, uint32_t *ring_tags, uint64_t *ring_tail, uint64_t *t) {
  if (!c) return ORC_E_INVAL;
  if (tags) memcpy(tags, c->tag, c->num_sets * c->ways * sizeof(uint32_t));
  if (ring_tags && c->victim_rows) memcpy(ring_tags, c->vtag, c->victim_rows * sizeof(uint32_t));
  if (ring_tail) *ring_tail = c->tail;
  if (t) *t = c->t;
  return ORC_OK;
}
