/*
 * lsmgnn.h -- C ABI of the MI355X (gfx950) feature-gather cache.
 *
 * The library serves the per-minibatch node-feature gather of storage-based GNN
 * training through a GPU-resident, 8-way set-associative software cache in HBM,
 * with the hybrid eviction policy and the victim buffer of LSM-GNN (Kim et al.,
 * arXiv 2407.15264):
 *   - the software cache holding recently used feature rows, with misses served
 *     from the backing feature store (Sec. 4, system design overview);
 *   - the window of sampled-node lists of upcoming minibatches that supplies
 *     the dynamic (next-reuse) information (Sec. 4 overview, Sec. 4.2);
 *   - the hybrid eviction policy: four levels from the dynamic information, the
 *     lowest static score evicted first within a level (Sec. 4.2);
 *   - the victim buffer in host memory that keeps evicted lines carrying reuse
 *     information, with the two lowest levels swapped when it is enabled
 *     (Sec. 4.3.1, 4.3.2).
 * Storage (SSDs in the paper) is a host-resident, pinned backing feature table.
 *
 * Semantics, fixed where the paper is silent (for the default configuration;
 * lsmgnn_config.policy, .victim_mode and .refresh_period select the
 * alternatives the paper's evaluation compares, documented with them below):
 *   - a gather deduplicates its IDs and serves them in ascending ID order; the
 *     output holds one row per unique ID, ascending, plus an inverse index;
 *   - set(x) = ((hi32(splitmix64(x)) * num_sets) >> 32), where splitmix64(x) is
 *     the first output of a SplitMix64 generator with state x;
 *   - a line's class while gather t runs: "recent" if inserted during gather t;
 *     otherwise with d the distance to its next announced use in (t, t+L]:
 *     none -> "no reuse", d <= T -> "near", T < d <= L -> "far";
 *   - eviction: an empty way first (lowest index); else the minimum of
 *     (level, static score, way) with levels far < none < recent < near when the
 *     victim ring is on (V > 0) and none < far < recent < near when it is off;
 *   - an evicted line of class far or near enters the victim ring (a FIFO of V
 *     entries that overwrites its oldest entry); others are dropped;
 *   - a request missing in the cache but present in the ring is a victim hit:
 *     the entry is removed and the line is refilled like any miss.
 * Every gathered row is bit-identical to the backing-store row of its node.
 *
 * Threading: one cache object must not be used from two threads at once.
 * Streams: a hipStream_t passed as void* (NULL = the null stream).  Each call
 * first waits for the work already queued on that stream; lsmgnn_gather and
 * lsmgnn_advance return once their work is complete, lsmgnn_gather_async once
 * its unique count is known (see there).
 */
#ifndef LSMGNN_H
#define LSMGNN_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct lsmgnn_cache lsmgnn_cache; /* opaque, owned by the library */

typedef enum {
  LSMGNN_OK = 0,
  LSMGNN_E_INVAL = 1,  /* bad argument or configuration */
  LSMGNN_E_RANGE = 2,  /* a node ID outside [0, num_nodes) */
  LSMGNN_E_WINDOW = 3, /* advance would announce a minibatch beyond t + L */
  LSMGNN_E_NOMEM = 4,  /* device or pinned host allocation failed */
  LSMGNN_E_DEVICE = 5, /* a HIP runtime call failed */
  LSMGNN_E_STATE = 6   /* the object is unusable after an earlier device error */
} lsmgnn_status;

/* per-unique-ID outcome codes written by lsmgnn_gather */
enum { LSMGNN_HIT = 0, LSMGNN_VICTIM_HIT = 1, LSMGNN_MISS = 2 };

/* lsmgnn_config.flags */
#define LSMGNN_FLAG_PAGEABLE_STORE 1u /* host_store is ordinary (pageable) host memory */

/* lsmgnn_config.policy: how a full set chooses the line to evict.  The hybrid
   order is the method's (Sec. 4.2, with the level swap of Sec. 4.3.2 when the
   victim ring is on); the other three are the alternatives its evaluation
   compares against (Sec. 5, impact of the cache eviction policy).  Only the
   choice changes: empty ways are taken first (lowest index), an evicted line
   goes to the victim ring iff its next announced use lies within the window
   and it was not inserted by the current gather, and ties go to the lowest
   way index. */
#define LSMGNN_POLICY_HYBRID 0u      /* lowest level, then lowest static score */
#define LSMGNN_POLICY_STATIC 1u      /* lowest static score */
#define LSMGNN_POLICY_DYNAMIC 2u     /* no announced use, else the furthest next use */
#define LSMGNN_POLICY_ROUND_ROBIN 3u /* a per-set pointer (from way 0) that advances by one per eviction */

/* lsmgnn_config.victim_mode: the form of the victim buffer (victim_rows > 0).
   FIFO: one ring of victim_rows entries that overwrites its oldest; a node
   with a live entry is a victim hit whenever it is requested, and its row is
   read from the victim buffer during that gather: over the host link from the
   pinned ring, or, for an entry the previous gather made, from the evicted
   rows that gather staged in HBM for its ring write (lsmgnn_counts
   victim_rows_*).
   QUEUES: the per-reuse-iteration queues of Sec. 4.3.1: an evicted line whose
   next announced use is minibatch j goes to the queue of iteration j at the
   position its counter gives (ascending request ID within a gather), unless
   the queue already holds C = victim_rows / (lookahead + 1) entries (then it
   is dropped).  After gather t is queued, the library copies queue t+1 into
   a prefetch buffer in HBM on its host-link stream (while the caller works on
   minibatch t, Sec. 4.3); gather t+1 serves the nodes queue t+1 holds from
   there (victim hits) and then empties it.  Requires victim_rows = 0 or
   lookahead + 1 <= victim_rows with C < 2^31; uses 2 C extra rows of HBM. */
#define LSMGNN_VICTIM_FIFO 0u
#define LSMGNN_VICTIM_QUEUES 1u

typedef struct {
  uint64_t num_nodes;   /* IDs are int64 in [0, num_nodes); 1 <= num_nodes <= 2^32 - 1 */
  uint64_t row_bytes;   /* bytes per feature row; a positive multiple of 16 */
  uint64_t num_sets;    /* S >= 1 sets of 8 ways; S * 8 * row_bytes bytes of HBM */
  uint64_t victim_rows; /* V rows of pinned host victim ring; 0 disables it */
  uint64_t max_batch;   /* largest n accepted by gather and advance (>= 1) */
  uint32_t lookahead;   /* L in [0, 31]: minibatches announced ahead */
  uint32_t near_threshold; /* T; 0 selects max(1, L / 8) (one eighth of the window) */
  int32_t device;       /* HIP device ordinal */
  uint32_t flags;       /* 0 or LSMGNN_FLAG_PAGEABLE_STORE; other bits must be 0 */
  uint32_t host_threads; /* pageable store: host threads copying rows (0 selects 8) */
  uint32_t policy;      /* LSMGNN_POLICY_*; other values are rejected */
  uint32_t victim_mode; /* LSMGNN_VICTIM_*; other values are rejected */
  /* Update period U of the dynamic information (Sec. 4.2); 0 selects 1.  U = 1:
     every gather sees each resident line's exact next use among the next
     lookahead minibatches.  U > 1: before every U-th gather (gather index a
     multiple of U) each resident line records its next reuse iteration from
     the lists announced by then; until the next update, a line inserted since
     then, or whose recorded iteration has come, ranks as recently inserted,
     and the others by the distance to the recorded iteration.  Costs one pass
     over the S * 8 lines per update instead of one window lookup per
     eviction candidate. */
  uint32_t refresh_period;
  /* Backing store: num_nodes * row_bytes bytes of host memory, row v at offset
     v * row_bytes.  Borrowed: the caller keeps it alive and unchanged while
     the cache exists; the library only reads it.
     Without flags it must be PINNED memory (from lsmgnn_host_alloc,
     hipHostMalloc or a pinned torch tensor): the GPU reads miss rows from it
     directly.  With LSMGNN_FLAG_PAGEABLE_STORE it may be ordinary memory, for
     stores larger than the pinned memory a process may hold: after a
     gather's metadata, host threads copy the rows of its misses and victim
     hits into a pinned bounce buffer (max_batch rows per gather in flight)
     that the GPU then reads.  Same results; lsmgnn_gather_async then returns
     once those rows are copied. */
  const void *host_store;
  /* Static score per node (host, num_nodes entries); copied at create. */
  const uint32_t *static_score;
} lsmgnn_config;

typedef struct {
  uint64_t batch;       /* gather index t of the last gather (total: gathers done) */
  uint64_t requests;    /* raw IDs */
  uint64_t unique;      /* unique IDs = hits + victim_hits + misses */
  uint64_t hits;        /* served from the HBM cache */
  uint64_t victim_hits; /* served from the victim ring */
  uint64_t misses;      /* served from the backing store */
  uint64_t evictions;   /* = enqueued + dropped */
  uint64_t enqueued;    /* evicted lines written to the victim ring */
  uint64_t dropped;     /* evicted lines discarded */
  /* the outcomes counted per raw request (a repeated ID counts each time):
     request misses = requests - request_hits - request_victim_hits */
  uint64_t request_hits;
  uint64_t request_victim_hits;
  /* where the victim hits' rows were read (they sum to victim_hits); all come
     from the victim buffer, none from the backing store:
       ring       FIFO: the pinned host ring (entries of gathers up to t-2);
       staged     FIFO: entries of the previous gather, from its evicted rows
                  staged in HBM for the ring write (which may still be running);
       cache      FIFO: lines evicted earlier in the same gather, from the
                  cache row the evicting fill took (not yet overwritten);
       prefetched queues: the HBM buffer the queue was prefetched into. */
  uint64_t victim_rows_ring;
  uint64_t victim_rows_staged;
  uint64_t victim_rows_cache;
  uint64_t victim_rows_prefetched;
} lsmgnn_counts;

/* Accumulated device time of the data movement (filled only while profiling
   is on; see lsmgnn_set_profiling).  Bytes are algorithmic: rows moved times
   row_bytes, per direction.  The enqueue figures time the ring write (the
   runtime copy of the staged evicted rows), not the staging kernel.  A
   gather's host fetch is two launches (the misses known at batch start, then
   the remaining host rows), both counted; its time excludes the wait between
   them. */
typedef struct {
  double hbm_copy_ms;   uint64_t hbm_copy_launches;   uint64_t hbm_copy_rows;   /* cache -> out */
  double host_fetch_ms; uint64_t host_fetch_launches; uint64_t host_fetch_rows; /* store/ring -> out */
  double enqueue_ms;    uint64_t enqueue_launches;    uint64_t enqueue_rows;    /* staging -> ring */
  double fill_ms;       uint64_t fill_launches;       uint64_t fill_rows;       /* out -> cache */
  double host_copy_ms;  uint64_t host_copy_rows;      /* pageable store: host threads' row copies (wall time) */
  double prefetch_ms;   uint64_t prefetch_launches;   uint64_t prefetch_rows;   /* victim queue -> HBM buffer */
  double gather_ms;     uint64_t gathers;             /* whole gather, first to last kernel */
} lsmgnn_profile;

/* Create a cache on cfg->device.  Allocates the HBM cache (S*8 rows), its
   metadata, per-node arrays (about 21 bytes per node), scratch and staging
   rows sized for max_batch, and the pinned victim ring (V rows).  On
   failure *out is NULL and nothing stays allocated. */
lsmgnn_status lsmgnn_cache_create(const lsmgnn_config *cfg, lsmgnn_cache **out);
void lsmgnn_cache_destroy(lsmgnn_cache *c);

/* Announce the sampled-node list of the next minibatch (the k-th call announces
   minibatch k).  ids: device pointer to n int64 IDs (duplicates allowed).
   E_WINDOW if k > t + L (t = gathers done); E_RANGE if an ID is out of range;
   E_INVAL if n > max_batch.  An announcement for k <= t is accepted and unused.
   On error nothing changes.  Synchronises `stream`. */
lsmgnn_status lsmgnn_advance(lsmgnn_cache *c, const int64_t *ids, uint64_t n, void *stream);

/* Gather one minibatch (gather index t, then t += 1).
     ids        device, n int64 node IDs (duplicates allowed)
     out        device, >= n * row_bytes bytes; row u = feature row of unique_ids[u]
     unique_ids device, >= n int64; ascending unique IDs
     inverse    device, n int64 or NULL; unique_ids[inverse[i]] == ids[i]
     outcome    device, >= n uint8 or NULL; LSMGNN_HIT / _VICTIM_HIT / _MISS per unique ID
     n_unique   host; number of unique IDs
   E_RANGE (nothing changes) if an ID is out of range; E_INVAL if n > max_batch
   or a required pointer is NULL.  Synchronises `stream`. */
lsmgnn_status lsmgnn_gather(lsmgnn_cache *c, const int64_t *ids, uint64_t n, void *out,
                            int64_t *unique_ids, int64_t *inverse, uint8_t *outcome,
                            uint64_t *n_unique, void *stream);

/* Pipelined gather, for loops that overlap consecutive minibatches (the
   sampler running ahead of training, Sec. 4.3.2).  Gathers ids like
   lsmgnn_gather and then, if next_ids is not NULL, announces the next_n IDs at
   next_ids (device int64) like lsmgnn_advance: the call is equivalent to that
   pair of calls, but checks both ID lists with one wait for the dedup result.
   next_ids == NULL announces nothing (next_n must be 0); an empty minibatch is
   announced with any non-NULL next_ids and next_n == 0 (nothing is read).
   Returns as soon as *n_unique is known, with *ticket identifying the gather.
   The gather's outputs (out, unique_ids, inverse, outcome) are complete once
   the caller has called lsmgnn_gather_wait(c, ticket, s) and then synchronised
   s (or run work on s after it).  Until then the caller must not read, reuse
   or free those buffers, nor change ids or next_ids.  The metadata of the next
   gather runs while this one still moves rows; at most two gathers are in
   flight and later calls wait for the oldest.  Waits for the work already
   queued on `stream` before reading ids.
   Errors: E_WINDOW if the announcement would be beyond the window once this
   gather is done (k > t + 1 + L); E_RANGE if an ID of either list is out of
   range; E_INVAL as for lsmgnn_gather, or if next_n > max_batch.  On any
   error neither the gather nor the announcement happens. */
lsmgnn_status lsmgnn_gather_async(lsmgnn_cache *c, const int64_t *ids, uint64_t n, const int64_t *next_ids,
                                  uint64_t next_n, void *out, int64_t *unique_ids, int64_t *inverse,
                                  uint8_t *outcome, uint64_t *n_unique, uint64_t *ticket, void *stream);

/* Make `stream` wait (on the device, without blocking the host) until the
   gather `ticket` has completed.  E_INVAL for a ticket never issued. */
lsmgnn_status lsmgnn_gather_wait(lsmgnn_cache *c, uint64_t ticket, void *stream);

/* Block the host until every queued gather and announcement has completed. */
lsmgnn_status lsmgnn_sync(lsmgnn_cache *c);

/* Counters of the last completed gather and totals over all gathers (either
   may be NULL).  Waits for queued gathers first. */
lsmgnn_status lsmgnn_stats(lsmgnn_cache *c, lsmgnn_counts *last, lsmgnn_counts *total);

/* Copy the policy state to host memory (each pointer may be NULL):
   tags num_sets*8 uint32 (0xFFFFFFFF = empty way), ring_tags victim_rows uint32
   (0xFFFFFFFF = empty entry), ring_tail = entries ever enqueued, t = gathers done. */
lsmgnn_status lsmgnn_export_state(lsmgnn_cache *c, uint32_t *tags, uint32_t *ring_tags,
                                  uint64_t *ring_tail, uint64_t *t);

/* Turn per-kernel event timing of the data-movement kernels on (1) or off (0);
   turning it on clears the accumulated profile. */
lsmgnn_status lsmgnn_set_profiling(lsmgnn_cache *c, int on);
lsmgnn_status lsmgnn_get_profile(lsmgnn_cache *c, lsmgnn_profile *out);

/* Pinned, device-mapped host memory for a backing store (exact size, unlike
   caching allocators that round up).  Free with lsmgnn_host_free. */
lsmgnn_status lsmgnn_host_alloc(uint64_t bytes, void **ptr);
void lsmgnn_host_free(void *ptr);

/* Calibration copy: bytes (a multiple of 16) from src to dst, both 16-byte
   aligned, each either device memory or pinned host memory, with the 128-bit
   access pattern of the gather's row copies (device to device: the HBM-side
   copies' tiles with the non-temporal hint; across the link: the host
   fetch's grid-strided vectors).  Used to measure the
   host-link and HBM ceilings the gather is compared against.  Synchronises
   `stream`. */
lsmgnn_status lsmgnn_copy_bytes(void *dst, const void *src, uint64_t bytes, void *stream);

/* Rows in request order: out[i] <- rows[inverse[i]] for i < n, row_bytes each
   (a positive multiple of 16).  rows is a gather's output (one row per unique
   ID) and inverse its inverse index; together they give every requested
   position its feature row, as a minibatch consumer indexes them (the paper's
   prefetched rows go to their positions in the minibatch, Sec. 4.3.2).  All
   pointers are DEVICE memory; rows and out 16-byte aligned, inverse 8-byte
   aligned; every inverse[i] must index a row of `rows` (a gather's inverse
   does).  Queued on `stream` after the work already there (the gather's
   output is ready once the caller's stream has waited for it); returns
   without waiting.  Errors: E_INVAL (NULL pointer with n > 0, bad row_bytes
   or alignment), E_DEVICE. */
lsmgnn_status lsmgnn_expand(const void *rows, const int64_t *inverse, uint64_t n, uint64_t row_bytes, void *out,
                            void *stream);

/* Static score from the graph: the normalized reverse PageRank that Sec. 4.2
   names as the hybrid policy's static information (and the evaluation's static
   policy uses, Sec. 5), as an alternative to the in-degree.
   offsets (num_nodes + 1 int64) and adj (offsets[num_nodes] uint32, may be
   NULL when there are no entries): the sampling adjacency in CSR form, node u
   listing the neighbours it samples; DEVICE memory on `device`, read only.
   The walk moves to a uniformly chosen CSR entry of the current node with
   probability `damping` (a repeated entry counts each time) and jumps to a
   uniformly chosen node otherwise; a node without entries always jumps.
   `iterations` power iterations start from the uniform vector.
   scores (num_nodes uint32, device): floor(rank / max rank * (2^32 - 1)).
   rank (num_nodes double, device) receives the ranks, or may be NULL.
   Ranks agree with a sequential evaluation to rounding (the per-node sums are
   accumulated with atomics in varying order), so a score may differ by one
   where its rank lies within rounding of a quantization step.
   Work memory of 4 bytes per entry plus 24 bytes per node is allocated and
   freed inside; the call is ordered after the work queued on `stream` and
   returns once the scores are written.
   Errors: E_INVAL (num_nodes 0 or above 2^32 - 1, damping outside [0, 1), NULL
   offsets/scores, or NULL adj with entries); E_RANGE (offsets not starting at 0
   or decreasing, or an entry >= num_nodes; nothing written); E_NOMEM; E_DEVICE. */
lsmgnn_status lsmgnn_pagerank_scores(const int64_t *offsets, const uint32_t *adj, uint64_t num_nodes,
                                     double damping, uint32_t iterations, uint32_t *scores, double *rank,
                                     int device, void *stream);

/* ---------------------------------------------------------- GPU sampler
   The raw request lists of GraphSAGE minibatches (uniform neighbour sampling
   with a fixed fanout per hop, Sec. 2.1), produced on the GPU as the system
   overview's GPU-side sampler does (Sec. 4), so that lsmgnn_gather_async and
   its announcement take them straight from device memory.  For minibatch b:
     frontier_0 = the seeds, sorted, duplicates removed;
     hop h: each frontier node v, ascending, draws k = min(fanout[h], deg v)
       distinct adjacency positions with Floyd's algorithm and lists them
       ascending; its samples are adj[offsets[v] + position] in that order;
       frontier_{h+1} = the hop's samples, sorted, duplicates removed;
     list = seeds (in the given order) ++ hop 0's samples ++ hop 1's ++ ...
   Draws come from counter-based SplitMix64 streams: key_b =
   derive(derive(seed, 3), b) with derive(p, l) = output l of the stream keyed
   by mix(p ^ 0x5851f42d4c957f2d), where output k of the stream keyed by K is
   mix(K + (k + 1) * 0x9e3779b97f4a7c15) and mix is SplitMix64's finalizer;
   hop h uses derive(key_b, h), node v in it derive(key_hop, v), and Floyd's
   j-th draw for v is output j of that stream reduced to [0, m) as
   ((r >> 32) * m) >> 32.  The list depends only on the graph, the seeds, the
   fanouts, `seed` and b.

   lsmgnn_sampler_create: offsets (num_nodes + 1 int64) and adj
   (offsets[num_nodes] uint32) in device-accessible memory on `device` (HBM,
   or pinned host memory through its device address), read only, borrowed:
   they must outlive the sampler.  1 <= hops <= 8, every fanout[h] <= 64
   (copied).  The graph is checked once (offsets from 0, non-decreasing, every
   degree below 2^32, every entry < num_nodes).  Work memory in HBM: about 9
   bytes per node (two frontier arrays, a byte map rounded up to 16 KiB, the
   per-tile sums).
   Errors: E_INVAL (NULL pointers, num_nodes 0 or above 2^32 - 1, hops or a
   fanout out of range); E_RANGE (a malformed graph); E_NOMEM; E_DEVICE.

   lsmgnn_sample: seeds (n_seeds int64, device) in [0, num_nodes); out
   (out_cap int64, device) receives the list.  Ordered after the work queued
   on `stream`; returns once *n_out (the list's length) is known, with the
   list written.  Calls of one sampler share its work memory: one at a time,
   or queued on one stream.
   Errors: E_RANGE (a seed outside [0, num_nodes): *n_out is set, the list is
   not valid); E_INVAL (NULL pointers, or a list longer than out_cap: *n_out
   is the length needed and only the first out_cap entries were written);
   E_DEVICE. */
typedef struct lsmgnn_sampler lsmgnn_sampler; /* opaque, owned by the library */
lsmgnn_status lsmgnn_sampler_create(const int64_t *offsets, const uint32_t *adj, uint64_t num_nodes,
                                    const uint32_t *fanout, uint32_t hops, uint64_t seed, int device,
                                    lsmgnn_sampler **out);
/* Waits for all work queued on the sampler's device, then frees it. */
void lsmgnn_sampler_destroy(lsmgnn_sampler *s);
lsmgnn_status lsmgnn_sample(lsmgnn_sampler *s, const int64_t *seeds, uint64_t n_seeds, uint64_t batch, int64_t *out,
                            uint64_t out_cap, uint64_t *n_out, void *stream);
/* lsmgnn_sample_async: the same sampling, queued on `stream` without waiting
   for it (a data-loading stream can then sample minibatches ahead of the
   gathers).  When the stream has run the call, result_host[0] holds the
   list's length and result_host[1] its status (LSMGNN_OK, LSMGNN_E_RANGE for a
   seed outside [0, num_nodes), LSMGNN_E_INVAL for a list longer than
   out_cap); result_host is two uint64 in pinned host memory (lsmgnn_host_alloc),
   to be read after the caller has synchronized with the stream.  Calls of one
   sampler share its work memory: queue them on one stream.  Returns E_INVAL
   for NULL pointers, E_DEVICE if queueing failed, else LSMGNN_OK. */
lsmgnn_status lsmgnn_sample_async(lsmgnn_sampler *s, const int64_t *seeds, uint64_t n_seeds, uint64_t batch,
                                  int64_t *out, uint64_t out_cap, uint64_t *result_host, void *stream);

/* Typed graphs (the heterogeneous workloads: one cache per node type): a
   request list of global node IDs split into one list per type, in request
   order, each ID replaced by its index within its type.
   ids (n int64, device); node_type (num_nodes uint8, device, each < num_types);
   local (num_nodes uint32, device): each node's index within its type;
   outs: num_types device pointers (host array), each to out_cap int64;
   work: device memory of at least lsmgnn_split_work_bytes(n, num_types) bytes,
   the caller's (no allocation inside); result_host: num_types + 1 uint64 in
   pinned host memory.  Queued on `stream`, returns at once; once the stream
   has run it, result_host[t] is type t's list length and result_host[num_types]
   the status (LSMGNN_OK; LSMGNN_E_RANGE for an ID outside [0, num_nodes) or a
   type >= num_types; LSMGNN_E_INVAL for a list longer than out_cap, of which
   the first out_cap entries were written).  1 <= num_types <= 16.
   Returns E_INVAL for bad arguments (work too small included), E_DEVICE if
   queueing failed, else LSMGNN_OK. */
uint64_t lsmgnn_split_work_bytes(uint64_t n, uint32_t num_types);
lsmgnn_status lsmgnn_split_by_type_async(const int64_t *ids, uint64_t n, uint64_t num_nodes, const uint8_t *node_type,
                                         const uint32_t *local, uint32_t num_types, int64_t *const *outs,
                                         uint64_t out_cap, void *work, uint64_t work_bytes, uint64_t *result_host,
                                         void *stream);

/* For callers that cannot allocate device memory (code under HIP graph
   capture, serving loops, harnesses that forbid hipMalloc): the same split as
   lsmgnn_split_by_type_async, with the same arguments, results and status
   words, but without `work`: its work memory is a device array inside the
   library, LSMGNN_SPLIT_SCRATCH_BYTES bytes on each device it runs on, held
   until the process ends.  The call allocates nothing (the array's address is
   looked up on the first call on each device).  E_INVAL also when
   lsmgnn_split_work_bytes(n, num_types) exceeds that size: n up to 2^24
   requests with 16 types (2^26 with 4).  Every call on a device uses the
   same array: calls that may overlap on one device (on different streams,
   or from several threads) race and must be ordered by the caller; queued on
   one stream they are ordered.  E_DEVICE if the stream's device cannot be
   found or the array's address not looked up. */
#define LSMGNN_SPLIT_SCRATCH_BYTES (256ull + (1ull << 24) / 256 * 16 * 4)
lsmgnn_status lsmgnn_split_by_type_noalloc_async(const int64_t *ids, uint64_t n, uint64_t num_nodes,
                                                 const uint8_t *node_type, const uint32_t *local, uint32_t num_types,
                                                 int64_t *const *outs, uint64_t out_cap, uint64_t *result_host,
                                                 void *stream);

/* Set index the cache uses for node x (host-side helper, for tests). */
uint64_t lsmgnn_set_of(uint64_t x, uint64_t num_sets);

const char *lsmgnn_strerror(lsmgnn_status s);

#ifdef __cplusplus
}
#endif
#endif /* LSMGNN_H */
