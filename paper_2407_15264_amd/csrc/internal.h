// Internal declarations shared by the gfx950 kernels and the host runtime of
// the feature-gather cache.  Not part of the public C ABI (include/lsmgnn.h).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace lsm {

constexpr uint32_t kWays = 8;
constexpr uint32_t kEmpty = 0xffffffffu;
constexpr int kBlock = 256;          // threads per block for every kernel
constexpr int kBytesPerThread = 64;  // dedup map bytes per thread
constexpr int kWordsPerThread = kBytesPerThread / 4;
constexpr int kChunkBytes = kBlock * kBytesPerThread;  // dedup map bytes (nodes) per block
constexpr int kScanPerThread = 8;    // flags per thread in the enqueue scan
constexpr int kScanChunk = kBlock * kScanPerThread;
constexpr int kMaxQueues = 32;       // victim-queue slots: L + 1 <= 32
constexpr uint32_t kSmallSet = 64;   // sets with more unique IDs in a batch are sorted by a block each

// dynamic classes of a resident line while a gather runs
enum : uint32_t { kClsNone = 0, kClsFar = 1, kClsRecent = 2, kClsNear = 3 };
// per-unique kinds from the set walk
enum : uint8_t { kKindHit = 0, kKindFill = 1 };
// per-unique flags: bit 0 the evicted line goes to the victim buffer; bits 1-5
// its next reuse distance (queue mode)
enum : uint8_t { kFlagEnqueue = 1 };
constexpr int kFlagDistShift = 1;
// per-unique row source: top two bits select the place, the rest index it
constexpr uint64_t kSrcHbm = 0ull << 62;    // cache slot in HBM
constexpr uint64_t kSrcStore = 1ull << 62;  // backing-store row (pinned host)
constexpr uint64_t kSrcRing = 2ull << 62;   // victim-ring row (pinned host)
constexpr uint64_t kSrcIndex = (1ull << 62) - 1;
// an HBM row index that names no row (the hit copy's list entry of a unique ID
// whose row comes over the host link); cache create keeps the row count below it
constexpr uint32_t kNoRow = 0xffffffffu;

// One set = one 128-byte record (one L2 line): the 8 resident node IDs, their
// static scores, the gather index at which each was inserted, and (round-robin
// policy only) the complement of the next way to evict, so that the all-ones
// initial record means way 0.
struct alignas(128) SetRec {
  uint32_t tag[kWays];
  uint32_t stat[kWays];
  uint32_t ins[kWays];
  uint32_t rr_inv;
  uint32_t pad[kWays - 1];
};

// victim-buffer forms (values of lsmgnn_config.victim_mode)
enum : uint32_t { kVictimFifo = 0, kVictimQueues = 1 };

// eviction policies (values of lsmgnn_config.policy)
enum : uint32_t { kPolicyHybrid = 0, kPolicyStatic = 1, kPolicyDynamic = 2, kPolicyRoundRobin = 3 };
static_assert(sizeof(SetRec) == 128, "set record must be one 128-byte line");

// Per-block partial counts: each block of a counting kernel stores its sums
// with plain stores and the last kernel of the call adds them up (no atomics
// on one shared line, which serialize across the GPU).
enum StatSlot : int {
  kStHits, kStFills, kStEvictions, kStEnqueued, kStDropped, kStFinal,  // set walk
  kStVictimHits, kStMisses, kStHbm, kStHost,                           // resolve
  kStEnqCopy,                                                          // enqueue finalize
  kStReqHits, kStReqVictimHits,                                        // per-request outcomes
  kStVhRing, kStVhStaged, kStVhSame,                                   // victim hits by row source
  kStEarly,                                                            // misses listed before the walk
  kNumStat
};
constexpr unsigned kMaxGrid = 8192;  // grid cap of every grid-stride kernel
struct StatGrids {
  uint32_t g[kNumStat];  // blocks that wrote each slot in this call (0 = none)
};

// Device counters of one call; zero at create, published and re-zeroed by the
// last kernel of every call.
struct Counters {
  uint32_t err;         // nonzero once any ID was out of range
  uint32_t n_unique;
  uint32_t n_touched;   // distinct sets touched by the batch
  uint32_t seg_cursor;
  uint32_t hits, fills, evictions, enqueued, dropped, victim_hits, misses;
  uint32_t n_hbm, n_host, n_enq_copy, n_fill;  // rows per data kernel
  uint32_t enq_total;
  uint32_t req_hits, req_victim_hits;  // outcomes counted per raw request
  // FIFO victim hits by where their rows were read: the pinned ring, the
  // previous gather's staged evicted rows (HBM), the cache row of a line
  // evicted earlier in the same gather
  uint32_t vh_ring, vh_staged, vh_same;
  uint32_t n_big;       // touched sets with more than kSmallSet unique IDs
  // victim queues (queue mode): enqueue candidates that found their queue
  // full, and per queue slot the entries before this gather and those it placed
  uint32_t q_overflow;
  uint32_t q_before[kMaxQueues];
  uint32_t q_placed[kMaxQueues];
  uint32_t pad[11];
};

// Dedup result of a gather, written by the chunk scan to pinned host memory:
// the host reads the unique count and the error flag from it.
struct DedupResult {
  uint32_t err;
  uint32_t n_unique;
  uint32_t pad[2];
};

// The gather's gate in device memory: the error flag and unique count (set by
// the chunk scan) and the lengths of the row-copy lists (appended by the
// resolve and enqueue kernels).  The row copies run on other streams after the
// metadata kernels have reset the call counters, so they read it from here.
struct Gate {
  uint32_t err;
  uint32_t n_unique;
  uint32_t n_host;   // host-fetch list: entries after the first n_early (appended by the resolve)
  uint32_t n_fill;   // fill list
  uint32_t n_stage;  // staging list
  // queue mode, written by the gather's last metadata kernel for the prefetch
  // of the next gather's queue: its entries, how many of them earlier gathers
  // placed (their rows are in the host queue), and where this gather staged
  // the rest
  uint32_t q_count, q_before, q_stage_off;
  // host-fetch list entries [0, n_early): misses known from the batch-start
  // state, listed right after the dedup and fetched before the set walk ends
  uint32_t n_early;
  uint32_t pad[3];
};

// A row-copy list: entry i moves row src[i] of its source to row dst[i] of its
// destination (dense, in arbitrary order).  The hit copy's list is the
// exception: one entry per unique ID, to output row i, dst unused.
struct RowList {
  uint32_t *src;
  uint32_t *dst;
};

// Per-call scratch, every array sized for max_batch entries unless noted.
// The row-copy lists, the gate and the staging rows are read by the row copies
// of a gather while the next gather's metadata kernels run, so the runtime
// keeps two of them and alternates by gather parity.
struct Scratch {
  uint32_t *uniq;       // ascending unique IDs
  uint32_t *uset;       // set of uniq[u]
  uint32_t *arrival;    // arrival order of u within its set
  uint32_t *touched;    // touched set list (arbitrary order)
  uint32_t *seg_off;    // segment offset of touched[i]
  uint32_t *seg;        // u grouped by set, arrival order
  uint32_t *seg_u;      // u grouped by set, ascending within the set
  uint32_t *seg_x;      // uniq[seg_u[.]]
  uint32_t *seg_st;     // static score of seg_x[.]
  uint32_t *big;        // [max_batch / (kSmallSet + 1) + 1] touched-set indices of sets with more than kSmallSet IDs
  uint8_t *kind;
  uint8_t *flags;
  uint8_t *oc;          // outcome of u (LSMGNN_HIT / _VICTIM_HIT / _MISS)
  uint8_t *dead;        // enqueue entry whose line was victim-hit in the same batch
  uint8_t *early;       // 1: u's row is fetched by the early host fetch (a miss known at batch start)
  uint32_t *slot;       // cache slot (set*8+way) hit or filled by u
  uint32_t *evicted;    // node evicted by u's fill, or kEmpty
  uint32_t *enq_before; // enqueues by unique IDs below u in this batch
  uint32_t *scan_part;  // ceil(max_batch / kScanChunk) + 2 partial sums
  uint64_t *this_q;     // 1 + ring sequence of u's own enqueue in this batch, or 0
  uint32_t *this_enq;   // the unique index that enqueued u in this batch
  uint32_t *fill_dst;   // 1 + cache slot that out row u refills (the way's final fill), or 0
  uint32_t *stat_part;  // [kNumStat][kMaxGrid] per-block partial counts
  Gate *gate;           // [1]
  uint32_t *host_list;  // host fetch: out rows whose rows come from pinned host memory
  uint64_t *host_src;   //   and the source code (kSrc*) of each
  RowList hbm;          // hit copy, one entry per unique ID: source row (kNoRow: none) -> out row u
  RowList fill;         // final occupants: out row -> cache slot
  RowList stage;        // surviving enqueues: cache slot -> staging row
  uint8_t *staging;     // [min(max_batch, V)][R] evicted rows in ring order, for the ring write (in DevState::rows)
  uint8_t *bounce;      // pageable store only: [max_batch][R] pinned, the host-fetch rows in list order
  uint32_t *qpart;      // queue mode: [kMaxQueues][ceil(max_batch / kBlock)] per-block enqueue counts
};

struct DevState {
  SetRec *sets;          // [S]
  uint8_t *rows;         // [S*8][R] cache data
  uint32_t *mask;        // [N] announced-batch bits (bit j mod 32)
  uint32_t *stat;        // [N] static score
  uint64_t *vpos;        // [N] FIFO: 1 + sequence of the node's latest ring entry, or 0;
                         //     queues: (1 + reuse iteration) << 32 | position of its latest entry
  uint32_t *ring_tag;    // [V] FIFO ring entries, or queue slot k's entries at k * C
  uint8_t *ring_rows;    // [V][R] pinned host, device-visible address (ring or queue rows)
  const uint8_t *store;  // [N][R] pinned host, device-visible address
  uint8_t *present;      // [nchunks * kChunkBytes] dedup byte map (all zero between calls)
  uint32_t *chunk_sums;  // [nchunks]
  uint32_t *set_count;   // [S] (all zero between calls)
  uint32_t *set_idx;     // [S]
  uint32_t *uidx;        // [N] unique index of the node in the current batch
                         //     (meaningful only where uniq[uidx[x]] == x)
  uint64_t *tail;        // [2] ring entries ever enqueued (the FIFO tail), and
                         //     the tail before the last gather's enqueues
  uint64_t N, R, S, V;
  uint64_t nchunks;
  uint32_t L, T;
  uint32_t policy;
  uint32_t qmode;        // kVictimQueues: per-reuse-iteration queues instead of the ring
  uint64_t C;            // queue mode: rows per queue, V / (L + 1)
  uint32_t *qcount;      // queue mode: [L + 1] entries in each queue slot
  uint32_t U;            // update period of the dynamic information (1: exact at every gather)
  uint32_t host_grid;    // blocks of the host fetch (0: the default), chosen per gather by the runtime
  uint32_t *lreuse;      // U > 1: [S*8] 1 + next reuse iteration recorded at the last update, or 0
  // Rows of `rows` after the S*8 cache lines: in queue mode the two prefetch
  // buffers (C rows each, by gather parity); then, with a victim buffer, the
  // two staging buffers (stage_rows each, by gather parity) holding each
  // gather's evicted rows in ring (or queue) order until they are written to
  // pinned host memory.  The hit copy reads both through row indices.
  uint64_t stage_row0;   // row index of parity 0's staging buffer
  uint64_t stage_rows;   // rows per staging buffer: min(max_batch, V)
};

// kHostEarly / kHostToOut: the host fetch of the host-fetch list's first
// n_early entries, and of the rest
enum class CopyMode { kHbmToOut, kHostToOut, kCacheToStage, kOutToCache, kHostEarly };

// What the last kernel of a gather does for the victim queues: empty the
// served slot `cur` and record in the gate what the prefetch of slot `next`
// needs.  qcount == nullptr: nothing (ring mode, announcements).
struct QueueFinish {
  uint32_t *qcount = nullptr;
  Gate *gate = nullptr;
  uint32_t cur = 0, next = 0;
};

// The announcement made with a gather, set by the gather's last kernel
// (ids == nullptr: none): the IDs, the minibatch's window bit, the window
// words and the list's window slot.
struct AnnounceArgs {
  const int64_t *ids = nullptr;
  uint32_t n = 0, bit = 0;
  uint32_t *mask = nullptr;
  int64_t *slot_ids = nullptr;
  const Gate *gate = nullptr;
};

// ----- launchers (gather_kernels.hip) -----
void launch_finish(Counters *cn, Counters *host, const uint32_t *stat_part, const StatGrids &grids,
                   uint64_t *tail, const QueueFinish &qf, const AnnounceArgs &ann, hipStream_t s);
// ann_ids/ann_n: the list announced with this gather (validated here), or NULL/0
void launch_dedup(const DevState &d, const int64_t *ids, uint64_t n, const int64_t *ann_ids, uint64_t ann_n,
                  const int64_t *clear_ids, uint64_t clear_n, uint32_t clear_bit, Scratch &sc, int64_t *unique_out,
                  Counters *cn, DedupResult *dd, hipStream_t s);
void launch_group_by_set(const DevState &d, const int64_t *ids, uint64_t n, int64_t *inverse, Scratch &sc,
                         Counters *cn, hipStream_t s);
void launch_set_walk(const DevState &d, uint64_t n, uint32_t t, Scratch &sc, Counters *cn, StatGrids &grids,
                     hipStream_t s);
// U > 1, before every U-th gather's set walk: record every resident line's next reuse iteration
void launch_refresh(const DevState &d, uint32_t t, const Counters *cn, hipStream_t s);
// t: the gather's index (queue mode serves queue t from prefetch buffer t & 1)
// sequence numbers of the batch's enqueues, then the resolve: outcomes, the
// hit-copy, host-fetch and fill lists
void launch_ring_resolve(const DevState &d, uint64_t n, uint64_t t, Scratch &sc, uint8_t *outcome, Counters *cn,
                         StatGrids &grids, hipStream_t s);
// after the resolve: the enqueues' ring (or queue) entries and the staging
// list, and the outcome counts per raw request (each request takes its
// unique ID's outcome)
void launch_ring_enqueue(const DevState &d, const int64_t *ids, uint64_t n, uint64_t t, Scratch &sc, Counters *cn,
                         StatGrids &grids, hipStream_t s);
// Queue mode: copy the queue of gather t+1 (slot `slot`) into prefetch buffer
// `par`: entries placed by gathers up to t-1 from the pinned host queue, those
// placed by gather t from its staging rows; sizes from gather t's gate.
void launch_prefetch(const DevState &d, const Gate *gate, const uint8_t *staging, uint32_t slot, uint32_t par,
                     hipStream_t s);
// out[i] <- rows[inv[i]] for i < n (R bytes each)
void launch_expand(const uint8_t *rows, const int64_t *inv, uint64_t n, uint64_t R, uint8_t *out, hipStream_t s);
// n bounds the gather's unique count (the copies read the exact one from the gate)
void launch_copy(CopyMode mode, const DevState &d, uint64_t n, const Scratch &sc, uint8_t *out, hipStream_t s);
void launch_window_set(const int64_t *ids, uint64_t n, uint64_t N, uint32_t bit, uint32_t *mask, int64_t *slot_ids,
                       bool record, uint32_t *err, hipStream_t s);
void launch_window_rollback(const int64_t *ids, uint64_t n, uint64_t N, uint32_t bit, uint32_t *mask,
                            hipStream_t s);
void launch_copy_plain(const void *src, void *dst, uint64_t bytes, bool device_to_device, hipStream_t s);
// pageable store: a host-fetch list length in the gate (0 for a rejected gather) to pinned host memory
void launch_publish_count(const Gate *gate, const uint32_t *count, uint32_t *dst, hipStream_t s);
// right after the dedup: list the misses known from the batch-start state
// (no way of the set holds the ID and the victim buffer has no entry for it)
// as the first entries of the host-fetch list
void launch_early(const DevState &d, uint64_t n, uint64_t t, Scratch &sc, Counters *cn, StatGrids &grids,
                  hipStream_t s);
// uidx[uniq[u]] = u for the gather's unique IDs (n bounds their count)
void launch_unique_index(const DevState &d, uint64_t n, const Scratch &sc, const Counters *cn, hipStream_t s);

// host twin of the device set-index function
uint64_t set_of_host(uint64_t x, uint64_t num_sets);

}  // namespace lsm
