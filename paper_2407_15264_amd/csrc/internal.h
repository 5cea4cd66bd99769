// Internal declarations shared by the gfx950 kernels and the host runtime of
// the feature-gather cache.  Not part of the public C ABI (include/lsmgnn.h).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace lsm {

constexpr uint32_t kWays = 8;
constexpr uint32_t kEmpty = 0xffffffffu;
constexpr int kBlock = 256;          // threads per block for every kernel
constexpr int kWordsPerThread = 8;   // dedup bitmap words per thread
constexpr int kChunkWords = kBlock * kWordsPerThread;  // bitmap words per block
constexpr int kScanPerThread = 8;    // flags per thread in the enqueue scan
constexpr int kScanChunk = kBlock * kScanPerThread;

// dynamic classes of a resident line while a gather runs
enum : uint32_t { kClsNone = 0, kClsFar = 1, kClsRecent = 2, kClsNear = 3 };
// per-unique kinds from the set walk
enum : uint8_t { kKindHit = 0, kKindFill = 1 };
// per-unique flags
enum : uint8_t { kFlagEnqueue = 1, kFlagFinal = 2 };
// host-fetch source code: bit 63 set = victim-ring row, else backing-store row
constexpr uint64_t kSrcRing = 1ull << 63;

// One set = one 128-byte record (one L2 line): the 8 resident node IDs, their
// static scores and the gather index at which each was inserted.
struct alignas(128) SetRec {
  uint32_t tag[kWays];
  uint32_t stat[kWays];
  uint32_t ins[kWays];
  uint32_t pad[kWays];
};
static_assert(sizeof(SetRec) == 128, "set record must be one 128-byte line");

// Device counters of one call; zeroed by the first kernel of each call.
struct Counters {
  uint32_t err;         // nonzero once any ID was out of range
  uint32_t n_unique;
  uint32_t n_touched;   // distinct sets touched by the batch
  uint32_t seg_cursor;
  uint32_t hits, fills, evictions, enqueued, dropped, victim_hits, misses;
  uint32_t n_hbm, n_host, n_enq_copy, n_fill;
  uint32_t enq_total;
  uint32_t pad[16];
};

// Per-call scratch, every array sized for max_batch entries unless noted.
struct Scratch {
  uint32_t *uniq;       // ascending unique IDs
  uint32_t *uset;       // set of uniq[u]
  uint32_t *ustat;      // static score of uniq[u]
  uint32_t *arrival;    // arrival order of u within its set
  uint32_t *touched;    // touched set list (arbitrary order)
  uint32_t *seg_off;    // segment offset of touched[i]
  uint32_t *seg;        // u grouped by set, arrival order
  uint32_t *sorted;     // u grouped by set, ascending within the set
  uint8_t *kind;
  uint8_t *flags;
  uint8_t *dead;        // enqueue entry whose line was victim-hit in the same batch
  uint32_t *slot;       // cache slot (set*8+way) hit or filled by u
  uint32_t *evicted;    // node evicted by u's fill, or kEmpty
  uint32_t *enq_before; // enqueues by unique IDs below u in this batch
  uint32_t *scan_part;  // ceil(max_batch / kScanChunk) + 1 partial sums
  uint64_t *this_q;     // 1 + ring sequence of u's own enqueue in this batch, or 0
  uint32_t *this_enq;   // the unique index that enqueued u in this batch
  // work lists: (a, b) pairs
  uint32_t *hbm_a; uint64_t *hbm_b;    // out row u  <- cache slot
  uint32_t *host_a; uint64_t *host_b;  // out row u  <- store row / ring row
  uint32_t *enq_a; uint64_t *enq_b;    // cache slot -> ring row
  uint32_t *fill_a; uint64_t *fill_b;  // cache slot <- out row u
};

struct DevState {
  SetRec *sets;          // [S]
  uint8_t *rows;         // [S*8][R] cache data
  uint32_t *mask;        // [N] announced-batch bits (bit j mod 32)
  uint32_t *stat;        // [N] static score
  uint64_t *vpos;        // [N] 1 + sequence of the node's latest ring entry, or 0
  uint32_t *ring_tag;    // [V]
  uint8_t *ring_rows;    // [V][R] pinned host, device-visible address
  const uint8_t *store;  // [N][R] pinned host, device-visible address
  uint32_t *bitmap;      // [nchunks * kChunkWords] dedup bitmap (all zero between calls)
  uint32_t *word_rank;   // [same] unique IDs before each nonzero word
  uint32_t *chunk_sums;  // [nchunks]
  uint32_t *set_count;   // [S] (all zero between calls)
  uint32_t *set_idx;     // [S]
  uint64_t N, R, S, V;
  uint64_t nchunks;
  uint32_t L, T;
};

enum class CopyMode { kHbmToOut, kHostToOut, kCacheToRing, kOutToCache };

// ----- launchers (gather_kernels.hip) -----
void launch_begin(Counters *cn, hipStream_t s);
void launch_validate(const int64_t *ids, uint64_t n, uint64_t N, Counters *cn, hipStream_t s);
void launch_dedup(const DevState &d, const int64_t *ids, uint64_t n, Scratch &sc, int64_t *unique_out,
                  int64_t *inverse, Counters *cn, hipStream_t s);
void launch_group_by_set(const DevState &d, uint64_t n, Scratch &sc, Counters *cn, hipStream_t s);
void launch_set_walk(const DevState &d, uint64_t n, uint32_t t, Scratch &sc, Counters *cn, hipStream_t s);
void launch_ring_resolve(const DevState &d, uint64_t n, uint64_t tail0, Scratch &sc, uint8_t *outcome,
                         Counters *cn, hipStream_t s);
void launch_copy(CopyMode mode, const DevState &d, uint64_t max_rows, const uint32_t *a, const uint64_t *b,
                 const uint32_t *count, uint8_t *out, Counters *cn, hipStream_t s);
void launch_window_set(const int64_t *ids, uint64_t n, uint32_t bit, uint32_t *mask, int64_t *slot_ids,
                       Counters *cn, hipStream_t s);
void launch_window_clear(const int64_t *slot_ids, uint64_t n, uint32_t bit, uint32_t *mask, Counters *cn,
                         hipStream_t s);

// host twin of the device set-index function
uint64_t set_of_host(uint64_t x, uint64_t num_sets);

}  // namespace lsm
