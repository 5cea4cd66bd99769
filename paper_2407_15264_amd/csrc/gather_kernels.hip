// gfx950 kernels of the feature-gather cache (LSM-GNN, arXiv 2407.15264).
//
// One gather runs as a short pipeline of stream-ordered kernels.  Every count
// that depends on the batch (unique IDs, touched sets, work-list lengths, the
// ring tail) stays in device memory, so the host queues the whole pipeline
// before it learns anything about the batch.  Each kernel reads the error flag
// first (Counters::err, or the gather's gate in the row copies) and does
// nothing once an out-of-range ID was seen, so an invalid batch changes no state.
//
//   dedup       byte map over node IDs marked with plain stores, per-chunk
//               popcount, chunk scan, ascending compaction that records each
//               node's unique index; the inverse index is one lookup
//   group       per-set counts with atomics, segment allocation, placement and
//               ranking so each touched set sees its IDs in ascending order
//   set walk    one lane per touched set walks its IDs in ascending order over
//               the 8 ways held in registers: tag probe, then on a fill the
//               empty way or the minimum (level, static score, way) victim
//               (Sec. 4.2 levels; Sec. 4.3.2 swap when the victim ring is on)
//   ring        exclusive scan of enqueue flags gives FIFO sequence numbers in
//               ascending-ID order; victim hits are resolved arithmetically:
//               an entry with sequence q is still in the ring at x's turn iff
//               q + V >= tail0 + (enqueues before x)  (Sec. 4.3.1)
//   data        row copies with 128-bit loads/stores: hits HBM->out, misses
//               and victim hits pinned host->out (a dense list, small grid),
//               enqueued rows HBM->staging in ring order (a runtime copy then
//               writes them to the pinned ring), then fills out->HBM for each
//               way's final occupant
#include "internal.h"

namespace lsm {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// ---------------------------------------------------------------- helpers
// set index: SplitMix64 output for state x (Steele, Lea, Flood 2014), reduced
// with Lemire's multiply-shift on its high 32 bits
__host__ __device__ __forceinline__ uint32_t set_index(uint64_t x, uint64_t S) {
  uint64_t z = x + 0x9e3779b97f4a7c15ull;
  z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ull;
  z = (z ^ (z >> 27)) * 0x94d049bb133111ebull;
  z ^= z >> 31;
  return (uint32_t)(((z >> 32) * S) >> 32);
}

uint64_t set_of_host(uint64_t x, uint64_t num_sets) { return set_index(x, num_sets); }

// Block-wide exclusive scan of one value per thread (kBlock threads).
__device__ __forceinline__ uint32_t block_exclusive_scan(uint32_t v, uint32_t &total) {
  __shared__ uint32_t wsum[kBlock / 64];
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  uint32_t x = v;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const uint32_t y = __shfl_up(x, d);
    if (lane >= d) x += y;
  }
  if (lane == 63) wsum[wid] = x;
  __syncthreads();
  uint32_t base = 0, tot = 0;
#pragma unroll
  for (int w = 0; w < kBlock / 64; ++w) {
    const uint32_t sw = wsum[w];
    base += (w < wid) ? sw : 0u;
    tot += sw;
  }
  __syncthreads();
  total = tot;
  return base + x - v;
}

__device__ __forceinline__ uint32_t block_sum(uint32_t v) {
  uint32_t tot;
  (void)block_exclusive_scan(v, tot);
  return tot;
}

// A gather's gate as the dedup leaves it: the error flag and the unique count,
// every list empty.
__device__ __forceinline__ Gate gate_with(uint32_t err, uint32_t n_unique) {
  Gate g{};
  g.err = err;
  g.n_unique = n_unique;
  return g;
}

static inline unsigned grid_for(uint64_t work, uint64_t per_block, unsigned cap) {
  uint64_t b = (work + per_block - 1) / per_block;
  if (b < 1) b = 1;
  if (b > cap) b = cap;
  return (unsigned)b;
}

// ------------------------------------------------------------------ finish
// Last kernel of every call: add up the per-block partial counts, publish all
// counters to pinned host memory, advance the ring tail by the call's enqueues
// (keeping the previous tail) and zero the device counters for the next call
// (they start zeroed at create).
//
// With an announcement (ann.ids != NULL) the launch has more blocks, which all
// also set the announced minibatch's bit for each of its IDs and record its
// list, unless the gather's gate holds an error: the announced bits are first
// read by the next gather's set walk.  Only that bit of a node's window word
// changes in this kernel (duplicates write the same value), so a plain
// read-modify-write is exact.
__device__ __forceinline__ void announce(const AnnounceArgs &a) {
  if (a.gate->err) return;
  const uint32_t b = 1u << a.bit;
  for (uint32_t i = blockIdx.x * kBlock + threadIdx.x; i < a.n; i += gridDim.x * kBlock) {
    const int64_t x = a.ids[i];
    a.slot_ids[i] = x;
    const uint32_t m = a.mask[x];
    if (!(m & b)) a.mask[x] = m | b;
  }
}

__global__ __launch_bounds__(kBlock) void k_finish(Counters *cn, Counters *host, const uint32_t *part,
                                                   StatGrids grids, uint64_t *tail, QueueFinish qf,
                                                   AnnounceArgs ann) {
  if (ann.ids) announce(ann);
  if (blockIdx.x != 0) return;
  __shared__ uint32_t red[kNumStat][kBlock / 64];
  __shared__ uint32_t sums[kNumStat];
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  // Each pass loads one partial of every slot before adding any: the loads
  // are independent, so a pass costs one memory round trip (several µs while
  // host-link reads are in flight beside this kernel) instead of one per slot.
  uint32_t gmax = 0;
#pragma unroll
  for (int st = 0; st < kNumStat; ++st) gmax = grids.g[st] > gmax ? grids.g[st] : gmax;
  uint32_t v[kNumStat];
#pragma unroll
  for (int st = 0; st < kNumStat; ++st) v[st] = 0;
  for (uint32_t b = threadIdx.x; b < gmax; b += kBlock) {
    uint32_t a[kNumStat];
#pragma unroll
    for (int st = 0; st < kNumStat; ++st) a[st] = b < grids.g[st] ? part[st * kMaxGrid + b] : 0u;
#pragma unroll
    for (int st = 0; st < kNumStat; ++st) v[st] += a[st];
  }
#pragma unroll
  for (int st = 0; st < kNumStat; ++st) {
    uint32_t x = v[st];
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) x += __shfl_xor(x, o);
    if (lane == 0) red[st][wid] = x;
  }
  __syncthreads();
  // the counters are staged in LDS and copied word by word by the whole block
  // (a private copy would live in scratch memory: its queue arrays are indexed
  // at run time)
  constexpr uint32_t kWords = sizeof(Counters) / 4;
  static_assert(sizeof(Counters) % 4 == 0 && kWords <= kBlock, "counters are copied one word per thread");
  __shared__ Counters c;
  if (threadIdx.x < kWords) reinterpret_cast<uint32_t *>(&c)[threadIdx.x] = reinterpret_cast<const uint32_t *>(cn)[threadIdx.x];
  if (threadIdx.x < kNumStat) {
    uint32_t v = 0;
#pragma unroll
    for (int w = 0; w < kBlock / 64; ++w) v += red[threadIdx.x][w];
    sums[threadIdx.x] = v;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    c.hits = sums[kStHits];
    c.fills = sums[kStFills];
    c.evictions = sums[kStEvictions];
    c.enqueued = sums[kStEnqueued];
    c.dropped = sums[kStDropped];
    c.n_fill = sums[kStFinal];
    c.victim_hits = sums[kStVictimHits];
    c.misses = sums[kStMisses];
    c.n_hbm = sums[kStHbm];
    c.n_host = sums[kStHost] + sums[kStEarly];  // both parts of the host-fetch list
    c.n_enq_copy = sums[kStEnqCopy];
    c.req_hits = sums[kStReqHits];
    c.req_victim_hits = sums[kStReqVictimHits];
    c.vh_ring = sums[kStVhRing];
    c.vh_staged = sums[kStVhStaged];
    c.vh_same = sums[kStVhSame];
    // queue mode: candidates that found their queue full were dropped
    c.enqueued -= c.q_overflow;
    c.dropped += c.q_overflow;
    if (tail && !c.err) {  // a rejected gather leaves both tails alone
      tail[1] = tail[0];
      tail[0] += c.enq_total;
    }
    if (qf.qcount && !c.err) {
      // the served queue is empty from now on; the next gather's queue holds
      // qcount[next] entries, the last q_placed[next] of them staged by this
      // gather after the rows it staged for the lower slots
      qf.qcount[qf.cur] = 0;
      uint32_t off = 0;
      for (uint32_t k = 0; k < qf.next; ++k) off += c.q_placed[k];
      const uint32_t cnt = qf.qcount[qf.next];
      qf.gate->q_count = cnt;
      qf.gate->q_before = cnt - c.q_placed[qf.next];
      qf.gate->q_stage_off = off;
    }
  }
  __syncthreads();
  if (threadIdx.x < kWords) {
    reinterpret_cast<uint32_t *>(host)[threadIdx.x] = reinterpret_cast<const uint32_t *>(&c)[threadIdx.x];
    reinterpret_cast<uint32_t *>(cn)[threadIdx.x] = 0u;
  }
}

void launch_finish(Counters *cn, Counters *host, const uint32_t *stat_part, const StatGrids &grids,
                   uint64_t *tail, const QueueFinish &qf, const AnnounceArgs &ann, hipStream_t s) {
  const unsigned g = ann.ids ? grid_for(ann.n, kBlock, kMaxGrid) : 1u;
  hipLaunchKernelGGL(k_finish, dim3(g), dim3(kBlock), 0, s, cn, host, stat_part, grids, tail, qf, ann);
}

// ------------------------------------------------------------------- dedup
// A byte per node marks the batch's requests.  Plain byte stores need no
// atomics: every writer of a byte writes the same value, and bytes of
// different nodes never interfere.  A bit per node would make the popcount
// and compaction passes read N/8 bytes instead of N, but its marks need
// atomic ORs, and repeated IDs of hub nodes queue on one word: measured on
// the MI355X, the byte map gives 478 GB/s on the 100M-node workload (the
// largest N here, 100 MB per pass) against 428-437 with the bitmap.
//
// Validate and mark.  Out-of-range IDs set Counters::err; valid ones are still
// marked, and the compaction kernel then clears the map instead of compacting
// it, so a rejected batch leaves no trace.  The list announced with the gather
// (if any) is validated here too; its bits are set only after the gather has
// been accepted.  The same kernel clears the window bit of the minibatch being
// gathered: that list is never consulted again, whether or not this call
// succeeds.  Only that bit of a node's window word changes in this kernel, so a
// plain read-modify-write is exact.
__global__ void k_mark(const int64_t *ids, uint32_t n, const int64_t *ann_ids, uint32_t ann_n, uint64_t N,
                       uint8_t *present, const int64_t *clear_ids, uint32_t clear_n, uint32_t clear_bit,
                       uint32_t *mask, Counters *cn) {
  bool bad = false;
  for (uint32_t i = blockIdx.x * kBlock + threadIdx.x; i < n; i += gridDim.x * kBlock) {
    const int64_t x = ids[i];
    if (x < 0 || (uint64_t)x >= N) {
      bad = true;
    } else {
      present[x] = 1;
    }
  }
  for (uint32_t i = blockIdx.x * kBlock + threadIdx.x; i < ann_n; i += gridDim.x * kBlock) {
    const int64_t x = ann_ids[i];
    bad |= x < 0 || (uint64_t)x >= N;
  }
  if (__ballot(bad) && __lane_id() == 0) atomicOr(&cn->err, 1u);
  const uint32_t cb = 1u << clear_bit;
  for (uint32_t i = blockIdx.x * kBlock + threadIdx.x; i < clear_n; i += gridDim.x * kBlock) {
    const int64_t x = clear_ids[i];
    const uint32_t m = mask[x];
    if (m & cb) mask[x] = m & ~cb;
  }
}

// Each thread owns kBytesPerThread consecutive bytes of the map (four 128-bit
// loads); marked bytes hold exactly 1, so a popcount of a word counts them.
__device__ __forceinline__ void load_words(const uint8_t *present, uint32_t (&w)[kWordsPerThread]) {
  const u32x4 *p = reinterpret_cast<const u32x4 *>(present + ((size_t)blockIdx.x * kBlock + threadIdx.x) *
                                                                 kBytesPerThread);
#pragma unroll
  for (int k = 0; k < kWordsPerThread / 4; ++k) {
    const u32x4 a = p[k];
    w[4 * k] = a.x; w[4 * k + 1] = a.y; w[4 * k + 2] = a.z; w[4 * k + 3] = a.w;
  }
}

__global__ __launch_bounds__(kBlock) void k_chunk_popc(const uint8_t *present, uint32_t *chunk_sums,
                                                       const Counters *cn) {
  if (cn->err) return;
  uint32_t w[kWordsPerThread];
  load_words(present, w);
  uint32_t c = 0;
#pragma unroll
  for (int k = 0; k < kWordsPerThread; ++k) c += __popc(w[k]);
  const uint32_t tot = block_sum(c);
  if (threadIdx.x == 0) chunk_sums[blockIdx.x] = tot;
}

__global__ __launch_bounds__(kBlock) void k_chunk_scan(uint32_t *chunk_sums, uint32_t nchunks, Counters *cn,
                                                       DedupResult *dd, Gate *gate) {
  const uint32_t err = cn->err;
  if (err) {
    if (threadIdx.x == 0) {
      *gate = gate_with(err, 0);
      *dd = DedupResult{err, 0, {0, 0}};
    }
    return;
  }
  uint32_t carry = 0;
  for (uint32_t base = 0; base < nchunks; base += kBlock) {
    const uint32_t i = base + threadIdx.x;
    const uint32_t v = i < nchunks ? chunk_sums[i] : 0u;
    uint32_t tot;
    const uint32_t ex = block_exclusive_scan(v, tot);
    if (i < nchunks) chunk_sums[i] = carry + ex;
    carry += tot;
  }
  if (threadIdx.x == 0) {
    cn->n_unique = carry;
    *gate = gate_with(0, carry);
    *dd = DedupResult{0, carry, {0, 0}};
  }
}

// The compaction: each node of the chunk with its bit set, ascending, gets the
// next unique index.  kFused: the chunk's first index is the sum of the
// earlier chunks' counts, added up by the block itself (few chunks: this
// saves the separate one-block scan), and the last chunk's block publishes
// the unique count; otherwise chunk_off holds the scanned offsets.  Each
// node's own unique index is written later (k_unique_index).
template <bool kFused>
__global__ __launch_bounds__(kBlock) void k_compact(uint8_t *present, const uint32_t *chunk_off, uint32_t *uniq,
                                                    int64_t *uniq_out, Counters *cn, uint32_t nchunks,
                                                    DedupResult *dd, Gate *gate) {
  uint32_t w[kWordsPerThread];
  load_words(present, w);
  const size_t b0 = ((size_t)blockIdx.x * kBlock + threadIdx.x) * kBytesPerThread;  // first byte of this thread
  const uint32_t err = cn->err;
  if (err) {  // rejected batch: undo the marks
#pragma unroll
    for (int k = 0; k < kWordsPerThread; ++k)
      if (w[k]) reinterpret_cast<uint32_t *>(present + b0)[k] = 0;
    if (kFused && blockIdx.x == 0 && threadIdx.x == 0) {
      *gate = gate_with(err, 0);
      *dd = DedupResult{err, 0, {0, 0}};
    }
    return;
  }
  uint32_t c = 0;
#pragma unroll
  for (int k = 0; k < kWordsPerThread; ++k) c += __popc(w[k]);
  uint32_t tot;
  const uint32_t ex = block_exclusive_scan(c, tot);
  uint32_t first;
  if constexpr (kFused) {
    uint32_t v = 0;
    for (uint32_t j = threadIdx.x; j < blockIdx.x; j += kBlock) v += chunk_off[j];
    first = block_sum(v);
    if (blockIdx.x == nchunks - 1 && threadIdx.x == 0) {
      const uint32_t total = first + tot;
      cn->n_unique = total;
      *gate = gate_with(0, total);
      *dd = DedupResult{0, total, {0, 0}};
    }
  } else {
    first = chunk_off[blockIdx.x];
  }
  if (tot == 0) return;
  uint32_t pos = first + ex;
#pragma unroll
  for (int k = 0; k < kWordsPerThread; ++k) {
    uint32_t word = w[k];
    while (word) {  // marked bytes ascending: bit 8j is set for byte j of word k
      const uint32_t x = (uint32_t)(b0 + 4 * k + (__builtin_ctz(word) >> 3));
      uniq[pos] = x;
      uniq_out[pos] = (int64_t)x;
      ++pos;
      word &= word - 1u;
    }
  }
}

constexpr uint32_t kFusedScanMax = 2048;  // at most this many partial sums are added up by each block

void launch_dedup(const DevState &d, const int64_t *ids, uint64_t n, const int64_t *ann_ids, uint64_t ann_n,
                  const int64_t *clear_ids, uint64_t clear_n, uint32_t clear_bit, Scratch &sc, int64_t *unique_out,
                  Counters *cn, DedupResult *dd, hipStream_t s) {
  uint64_t work = n > clear_n ? n : clear_n;
  work = work > ann_n ? work : ann_n;
  const unsigned g = grid_for(work, kBlock, kMaxGrid);
  hipLaunchKernelGGL(k_mark, dim3(g), dim3(kBlock), 0, s, ids, (uint32_t)n, ann_ids, (uint32_t)ann_n, d.N,
                     d.present, clear_ids, (uint32_t)clear_n, clear_bit, d.mask, cn);
  hipLaunchKernelGGL(k_chunk_popc, dim3((unsigned)d.nchunks), dim3(kBlock), 0, s, d.present, d.chunk_sums, cn);
  if (d.nchunks <= kFusedScanMax) {
    hipLaunchKernelGGL(k_compact<true>, dim3((unsigned)d.nchunks), dim3(kBlock), 0, s, d.present, d.chunk_sums,
                       sc.uniq, unique_out, cn, (uint32_t)d.nchunks, dd, sc.gate);
  } else {
    hipLaunchKernelGGL(k_chunk_scan, dim3(1), dim3(kBlock), 0, s, d.chunk_sums, (uint32_t)d.nchunks, cn, dd,
                       sc.gate);
    hipLaunchKernelGGL(k_compact<false>, dim3((unsigned)d.nchunks), dim3(kBlock), 0, s, d.present, d.chunk_sums,
                       sc.uniq, unique_out, cn, (uint32_t)d.nchunks, dd, sc.gate);
  }
}

// Each unique ID's index, uidx[uniq[u]] = u, read by the inverse index and the
// per-request counts.  Kept out of the compaction: these scattered 4-byte
// writes (one per unique ID over an N-entry array) cost the compaction most
// of its time beside the host-link reads, and the early-miss list, which
// needs only the unique list, need not wait for them.
__global__ __launch_bounds__(kBlock) void k_unique_index(const uint32_t *uniq, uint32_t *uidx, const Counters *cn) {
  if (cn->err) return;
  const uint32_t U = cn->n_unique;
  for (uint32_t u = blockIdx.x * kBlock + threadIdx.x; u < U; u += gridDim.x * kBlock) uidx[uniq[u]] = u;
}

void launch_unique_index(const DevState &d, uint64_t n, const Scratch &sc, const Counters *cn, hipStream_t s) {
  hipLaunchKernelGGL(k_unique_index, dim3(grid_for(n, kBlock, kMaxGrid)), dim3(kBlock), 0, s, sc.uniq, d.uidx, cn);
}

// ------------------------------------------------------------ group by set
// Every thread of the block must call this; returns the list index for
// threads with pred set (one atomic per block).
__device__ __forceinline__ uint32_t block_append(bool pred, uint32_t *counter) {
  __shared__ uint32_t base;
  uint32_t tot;
  const uint32_t ex = block_exclusive_scan(pred ? 1u : 0u, tot);
  if (threadIdx.x == 0 && tot) base = atomicAdd(counter, tot);
  __syncthreads();
  const uint32_t r = base + ex;
  __syncthreads();
  return r;
}

// Sum of a per-thread counter over the block, stored as this block's partial.
__device__ __forceinline__ void block_count(uint32_t v, uint32_t *part, int slot) {
  const uint32_t tot = block_sum(v);
  if (threadIdx.x == 0) part[slot * kMaxGrid + blockIdx.x] = tot;
}

// Inverse index of every request (the compaction recorded each node's unique
// index), then per-set counts of the unique IDs.
__global__ __launch_bounds__(kBlock) void k_inverse_claim(const DevState d, Scratch sc, const int64_t *ids,
                                                          uint32_t n, int64_t *inv, Counters *cn) {
  if (cn->err) return;
  if (inv) {
    for (uint32_t i = blockIdx.x * kBlock + threadIdx.x; i < n; i += gridDim.x * kBlock) {
      inv[i] = (int64_t)d.uidx[ids[i]];
    }
  }
  const uint32_t U = cn->n_unique;
  for (uint32_t base = blockIdx.x * kBlock; base < U; base += gridDim.x * kBlock) {
    const uint32_t u = base + threadIdx.x;
    bool claim = false;
    uint32_t s = 0;
    if (u < U) {
      const uint32_t x = sc.uniq[u];
      s = set_index(x, d.S);
      sc.uset[u] = s;
      const uint32_t old = atomicAdd(&d.set_count[s], 1u);
      sc.arrival[u] = old;
      claim = (old == 0);
      sc.flags[u] = 0;
      sc.dead[u] = 0;
      sc.this_q[u] = 0;
      sc.fill_dst[u] = 0;
      d.present[x] = 0;  // the map's last reader (the compaction) is done
    }
    const uint32_t i = block_append(claim, &cn->n_touched);
    if (claim) {
      sc.touched[i] = s;
      d.set_idx[s] = i;
    }
  }
}

__global__ __launch_bounds__(kBlock) void k_seg_alloc(const DevState d, Scratch sc, Counters *cn) {
  if (cn->err) return;
  const uint32_t T = cn->n_touched;
  __shared__ uint32_t boff;
  for (uint32_t base = blockIdx.x * kBlock; base < T; base += gridDim.x * kBlock) {
    const uint32_t i = base + threadIdx.x;
    const uint32_t c = i < T ? d.set_count[sc.touched[i]] : 0u;
    uint32_t tot;
    const uint32_t ex = block_exclusive_scan(c, tot);
    if (threadIdx.x == 0) boff = atomicAdd(&cn->seg_cursor, tot);
    __syncthreads();
    if (i < T) sc.seg_off[i] = boff + ex;
    __syncthreads();
    // sets with more than kSmallSet IDs are ordered by k_big_sort
    const bool big = c > kSmallSet;
    const uint32_t j = block_append(big, &cn->n_big);
    if (big) sc.big[j] = i;
  }
}

__global__ void k_place(const DevState d, Scratch sc, const Counters *cn) {
  if (cn->err) return;
  const uint32_t U = cn->n_unique;
  for (uint32_t u = blockIdx.x * kBlock + threadIdx.x; u < U; u += gridDim.x * kBlock)
    sc.seg[sc.seg_off[d.set_idx[sc.uset[u]]] + sc.arrival[u]] = u;
}

// Rank of u among the IDs of its set (all smaller unique indices come first)
// in a set of at most kSmallSet IDs, by counting (at most kSmallSet loads);
// lays out (u, ID, static score) contiguously per set for the walk.
__global__ void k_rank(const DevState d, Scratch sc, const Counters *cn) {
  if (cn->err) return;
  const uint32_t U = cn->n_unique;
  for (uint32_t u = blockIdx.x * kBlock + threadIdx.x; u < U; u += gridDim.x * kBlock) {
    const uint32_t s = sc.uset[u];
    const uint32_t off = sc.seg_off[d.set_idx[s]];
    const uint32_t k = d.set_count[s];
    if (k > kSmallSet) continue;
    uint32_t r = 0;
    if (k > 1)
      for (uint32_t j = 0; j < k; ++j) r += sc.seg[off + j] < u ? 1u : 0u;
    const uint32_t x = sc.uniq[u];
    sc.seg_u[off + r] = u;
    sc.seg_x[off + r] = x;
    sc.seg_st[off + r] = d.stat[x];
  }
}

// A set with more than kSmallSet IDs: one block sorts its segment (distinct
// unique indices, in arrival order) ascending with an LSD radix sort over
// 8-bit digits of the index, in O(k) per pass, ping-ponging between seg and
// seg_u.  Each pass: digit histogram in LDS, exclusive scan, then the scatter
// in index order, 256 entries at a time: an entry's place among the chunk's
// entries with the same digit comes from eight ballots per wave (the lanes
// whose digit matches) and the counts of the lower waves.
__global__ __launch_bounds__(kBlock) void k_big_sort(const DevState d, Scratch sc, const Counters *cn) {
  if (cn->err) return;
  const uint32_t nbig = cn->n_big;
  const uint32_t U = cn->n_unique;
  const uint32_t bits = U > 1 ? 32u - (uint32_t)__builtin_clz(U - 1u) : 1u;
  const uint32_t passes = (bits + 7u) / 8u;
  __shared__ uint32_t base[256];
  __shared__ uint32_t wcnt[kBlock / 64][256];
  const uint32_t lane = threadIdx.x & 63u, wid = threadIdx.x >> 6;
  const uint64_t lt = lane ? (~0ull >> (64u - lane)) : 0ull;
  for (uint32_t b = blockIdx.x; b < nbig; b += gridDim.x) {
    const uint32_t i = sc.big[b];
    const uint32_t off = sc.seg_off[i];
    const uint32_t k = d.set_count[sc.touched[i]];
    uint32_t *src = sc.seg + off, *dst = sc.seg_u + off;
    for (uint32_t p = 0; p < passes; ++p) {
      const uint32_t shift = 8u * p;
      base[threadIdx.x] = 0;
      __syncthreads();
      for (uint32_t j = threadIdx.x; j < k; j += kBlock) atomicAdd(&base[(src[j] >> shift) & 255u], 1u);
      __syncthreads();
      uint32_t tot;
      const uint32_t ex = block_exclusive_scan(base[threadIdx.x], tot);
      __syncthreads();
      base[threadIdx.x] = ex;
      for (uint32_t c0 = 0; c0 < k; c0 += kBlock) {
#pragma unroll
        for (int w = 0; w < kBlock / 64; ++w) wcnt[w][threadIdx.x] = 0;
        __syncthreads();
        const uint32_t j = c0 + threadIdx.x;
        const bool valid = j < k;
        const uint32_t v = valid ? src[j] : 0u;
        const uint32_t dg = (v >> shift) & 255u;
        uint64_t m = __ballot(valid);
#pragma unroll
        for (int bit = 0; bit < 8; ++bit) {
          const bool on = (dg >> bit) & 1u;
          const uint64_t bb = __ballot(valid && on);
          m &= on ? bb : ~bb;
        }
        if (valid && (m & lt) == 0) wcnt[wid][dg] = (uint32_t)__popcll(m);
        __syncthreads();
        if (valid) {
          uint32_t r = base[dg] + (uint32_t)__popcll(m & lt);
          for (uint32_t w = 0; w < wid; ++w) r += wcnt[w][dg];
          dst[r] = v;
        }
        __syncthreads();
        uint32_t add = 0;
#pragma unroll
        for (int w = 0; w < kBlock / 64; ++w) add += wcnt[w][threadIdx.x];
        base[threadIdx.x] += add;
      }
      __syncthreads();
      uint32_t *tmp = src;
      src = dst;
      dst = tmp;
    }
    // the sorted indices are in src; lay out (u, ID, static score)
    for (uint32_t j = threadIdx.x; j < k; j += kBlock) {
      const uint32_t u = src[j];
      const uint32_t x = sc.uniq[u];
      sc.seg_u[off + j] = u;
      sc.seg_x[off + j] = x;
      sc.seg_st[off + j] = d.stat[x];
    }
    __syncthreads();
  }
}

void launch_group_by_set(const DevState &d, const int64_t *ids, uint64_t n, int64_t *inverse, Scratch &sc,
                         Counters *cn, hipStream_t s) {
  const unsigned g = grid_for(n, kBlock, kMaxGrid);
  hipLaunchKernelGGL(k_inverse_claim, dim3(g), dim3(kBlock), 0, s, d, sc, ids, (uint32_t)n, inverse, cn);
  hipLaunchKernelGGL(k_seg_alloc, dim3(g), dim3(kBlock), 0, s, d, sc, cn);
  hipLaunchKernelGGL(k_place, dim3(g), dim3(kBlock), 0, s, d, sc, cn);
  hipLaunchKernelGGL(k_rank, dim3(g), dim3(kBlock), 0, s, d, sc, cn);
  // sets of more than kSmallSet IDs exist only if n does
  if (n > kSmallSet)
    hipLaunchKernelGGL(k_big_sort, dim3(grid_for(n / (kSmallSet + 1), 1, 256)), dim3(kBlock), 0, s, d, sc, cn);
}

// ---------------------------------------------------------------- set walk
// Class of a resident line from its announced-batch bits: bit (j mod 32) is
// set while minibatch j is announced and not yet served.  The next use after
// gather t is the lowest set bit after rotating bit (t+1) to position 0.
__device__ __forceinline__ uint32_t class_from_bits(uint32_t m, uint32_t t, uint32_t L, uint32_t T) {
  const uint32_t rel = __builtin_amdgcn_alignbit(m, m, (t + 1u) & 31u) & ((1u << L) - 1u);
  if (rel == 0) return kClsNone;
  return (uint32_t)__builtin_ctz(rel) + 1u <= T ? kClsNear : kClsFar;
}

// Distance from gather t to the line's next announced use (1..L), or 0 when
// none of the next L minibatches names it.
__device__ __forceinline__ uint32_t dist_from_bits(uint32_t m, uint32_t t, uint32_t L) {
  const uint32_t rel = __builtin_amdgcn_alignbit(m, m, (t + 1u) & 31u) & ((1u << L) - 1u);
  return rel ? (uint32_t)__builtin_ctz(rel) + 1u : 0u;
}

// The update of the dynamic information (Sec. 4.2) with an update period U >
// 1, before every U-th gather: each resident line records 1 + its next reuse
// iteration from the announced-batch bits (0: none).  Skipped when the
// gather's IDs were rejected; the retry of the same gather runs it.
__global__ __launch_bounds__(kBlock) void k_refresh(const DevState d, uint32_t t, const Counters *cn) {
  if (cn->err) return;
  const uint64_t lines = d.S * kWays;
  for (uint64_t i = (uint64_t)blockIdx.x * kBlock + threadIdx.x; i < lines; i += (uint64_t)gridDim.x * kBlock) {
    const uint32_t tag = d.sets[i / kWays].tag[i % kWays];
    uint32_t r = 0;
    if (tag != kEmpty) {
      const uint32_t dist = dist_from_bits(d.mask[tag], t, d.L);
      r = dist ? t + dist + 1u : 0u;
    }
    d.lreuse[i] = r;
  }
}

void launch_refresh(const DevState &d, uint32_t t, const Counters *cn, hipStream_t s) {
  hipLaunchKernelGGL(k_refresh, dim3(grid_for(d.S * kWays, kBlock, kMaxGrid)), dim3(kBlock), 0, s, d, t, cn);
}

// Class and next-reuse distance of a batch-start resident from the
// information recorded at the last update (update period U > 1): inserted at
// or after that update, or its recorded reuse has come -> recently inserted
// (distance 0); none recorded -> no reuse; else near or far by the distance.
__device__ __forceinline__ void class_from_record(uint32_t rec, uint32_t ins, uint32_t t, uint32_t t_upd, uint32_t T,
                                                  uint32_t &cls, uint32_t &dist) {
  dist = 0;
  if (ins >= t_upd) {
    cls = kClsRecent;
  } else if (rec == 0) {
    cls = kClsNone;
  } else if (rec - 1u <= t) {
    cls = kClsRecent;
  } else {
    dist = rec - 1u - t;
    cls = dist <= T ? kClsNear : kClsFar;
  }
}

// eviction level, lowest evicted first: none < far < recent < near, or with
// the victim ring on, far < none < recent < near
__device__ __forceinline__ uint32_t level_of(uint32_t cls, bool ring_on) {
  return (ring_on && cls <= kClsFar) ? (cls ^ 1u) : cls;
}

// Minimum of a 64-bit key over the 8 lanes of a set's lane group.
__device__ __forceinline__ uint64_t group_min(uint64_t v) {
#pragma unroll
  for (int o = 1; o < (int)kWays; o <<= 1) {
    const uint32_t lo = __shfl_xor((uint32_t)v, o, kWays);
    const uint32_t hi = __shfl_xor((uint32_t)(v >> 32), o, kWays);
    const uint64_t w = ((uint64_t)hi << 32) | lo;
    v = w < v ? w : v;
  }
  return v;
}

// One set per group of 8 lanes, lane w owning way w.  The group walks the
// set's IDs in ascending order (the per-set order of the definition); each
// step is a ballot for the tag probe, a ballot for an empty way, and on a full
// set the policy's victim: for the hybrid order (Sec. 4.2) a 3-step shuffle
// minimum of (level, static score, way); for the evaluation's ablations
// (Sec. 5) the minimum of (static score, way), of (no announced use first,
// then the furthest next use; way), or the set's round-robin pointer.
template <int P>
__global__ __launch_bounds__(kBlock) void k_set_walk(const DevState d, Scratch sc, uint32_t t, Counters *cn) {
  if (cn->err) return;
  const uint32_t Tn = cn->n_touched;
  const bool ring_on = d.V > 0;
  const uint32_t recent_lvl = level_of(kClsRecent, ring_on);
  const uint32_t lane = threadIdx.x & 63u;
  const uint32_t w = lane & (kWays - 1);   // the way this lane owns
  const uint32_t gsh = lane & ~(kWays - 1);  // first lane of the group in the wave
  const bool lead = w == 0;
  uint32_t c_hit = 0, c_fill = 0, c_evict = 0, c_enq = 0, c_drop = 0, c_final = 0;
  const uint32_t groups = gridDim.x * (kBlock / kWays);
  for (uint32_t i = blockIdx.x * (kBlock / kWays) + (threadIdx.x / kWays); i < Tn; i += groups) {
    const uint32_t s = sc.touched[i];
    const uint32_t off = sc.seg_off[i];
    const uint32_t k = d.set_count[s];
    SetRec *rec = d.sets + s;
    uint32_t tag = rec->tag[w], st = rec->stat[w], ins = rec->ins[w];
    uint32_t cls = kClsNone, lvl = 0, dist = 0;
    bool known = false;  // class (and next-use distance) of this way for this gather computed
    uint32_t rr = 0;     // round-robin pointer (the record holds its complement)
    if constexpr (P == kPolicyRoundRobin) rr = ~rec->rr_inv & (kWays - 1);
    const uint32_t rr0 = rr;
    int32_t last = -1;   // unique index of this way's last fill
    bool dirty = false;
    uint32_t pu = 0, px = 0, ps = 0;  // entry (j & ~7) + w of the segment, loaded 8 at a time
    for (uint32_t j = 0; j < k; ++j) {
      if ((j & (kWays - 1)) == 0 && j + w < k) {
        pu = sc.seg_u[off + j + w];
        px = sc.seg_x[off + j + w];
        ps = sc.seg_st[off + j + w];
      }
      const int src = (int)(j & (kWays - 1));
      const uint32_t u = __shfl(pu, src, kWays);
      const uint32_t x = __shfl(px, src, kWays);
      const uint32_t xs = __shfl(ps, src, kWays);
      const uint32_t hitm = (uint32_t)(__ballot(tag == x) >> gsh) & 0xffu;
      if (hitm) {
        if (lead) {
          sc.kind[u] = kKindHit;
          sc.slot[u] = s * kWays + (uint32_t)__builtin_ctz(hitm);
          ++c_hit;
        }
        continue;
      }
      dirty = true;
      const uint32_t emptym = (uint32_t)(__ballot(tag == kEmpty) >> gsh) & 0xffu;
      uint32_t pick, z = kEmpty;
      uint8_t f = 0;
      if (emptym) {
        pick = (uint32_t)__builtin_ctz(emptym);
      } else {
        if (!known) {  // batch-start resident
          if (d.U > 1) {  // from the information recorded at the last update
            class_from_record(d.lreuse[s * kWays + w], ins, t, t - t % d.U, d.T, cls, dist);
          } else {        // exact: from its announced-use bits
            const uint32_t m = d.mask[tag];
            cls = (ins == t) ? kClsRecent : class_from_bits(m, t, d.L, d.T);
            if (P == kPolicyDynamic || d.qmode) dist = dist_from_bits(m, t, d.L);
          }
          lvl = level_of(cls, ring_on);
          known = true;
        }
        if constexpr (P == kPolicyHybrid) {
          pick = (uint32_t)(group_min(((uint64_t)lvl << 35) | ((uint64_t)st << 3) | w) & 7u);
        } else if constexpr (P == kPolicyStatic) {
          pick = (uint32_t)(group_min(((uint64_t)st << 3) | w) & 7u);
        } else if constexpr (P == kPolicyDynamic) {
          pick = (uint32_t)(group_min((uint64_t)((dist ? 32u - dist : 0u) << 3) | w) & 7u);
        } else {
          pick = rr;
          rr = (rr + 1u) & (kWays - 1);
        }
        z = __shfl(tag, (int)pick, kWays);
        const uint32_t pc = __shfl(cls, (int)pick, kWays);
        const uint32_t pd = __shfl(dist, (int)pick, kWays);
        if (lead) {
          ++c_evict;
          if (ring_on && (pc == kClsFar || pc == kClsNear)) {
            f = (uint8_t)(kFlagEnqueue | (pd << kFlagDistShift));
            ++c_enq;
          } else {
            ++c_drop;
          }
        }
      }
      if (lead) {
        ++c_fill;
        sc.kind[u] = kKindFill;
        sc.slot[u] = s * kWays + pick;
        sc.evicted[u] = z;
        sc.flags[u] = f;
      }
      if (w == pick) {
        tag = x;
        st = xs;
        ins = t;
        cls = kClsRecent;
        lvl = recent_lvl;
        dist = 0;  // a line inserted by this gather has no dynamic information yet
        known = true;
        last = (int32_t)u;
      }
    }
    if (last >= 0) {  // the way's final occupant refills the cache row
      sc.fill_dst[last] = s * kWays + w + 1;
      ++c_final;
    }
    if (dirty) {
      rec->tag[w] = tag;
      rec->stat[w] = st;
      rec->ins[w] = ins;
    }
    if constexpr (P == kPolicyRoundRobin)
      if (lead && rr != rr0) rec->rr_inv = ~rr;
    if (lead) d.set_count[s] = 0;
  }
  block_count(c_hit, sc.stat_part, kStHits);
  block_count(c_fill, sc.stat_part, kStFills);
  block_count(c_evict, sc.stat_part, kStEvictions);
  block_count(c_enq, sc.stat_part, kStEnqueued);
  block_count(c_drop, sc.stat_part, kStDropped);
  block_count(c_final, sc.stat_part, kStFinal);
}

#ifndef LSM_WALK_GRID
#define LSM_WALK_GRID 4096  // set-walk blocks of 32 lane groups: enough sets in flight to hide the record loads
#endif
void launch_set_walk(const DevState &d, uint64_t n, uint32_t t, Scratch &sc, Counters *cn, StatGrids &grids,
                     hipStream_t s) {
  const unsigned g = grid_for(n * kWays, kBlock, LSM_WALK_GRID);
  switch (d.policy) {
    case kPolicyStatic:
      hipLaunchKernelGGL(k_set_walk<kPolicyStatic>, dim3(g), dim3(kBlock), 0, s, d, sc, t, cn);
      break;
    case kPolicyDynamic:
      hipLaunchKernelGGL(k_set_walk<kPolicyDynamic>, dim3(g), dim3(kBlock), 0, s, d, sc, t, cn);
      break;
    case kPolicyRoundRobin:
      hipLaunchKernelGGL(k_set_walk<kPolicyRoundRobin>, dim3(g), dim3(kBlock), 0, s, d, sc, t, cn);
      break;
    default:
      hipLaunchKernelGGL(k_set_walk<kPolicyHybrid>, dim3(g), dim3(kBlock), 0, s, d, sc, t, cn);
  }
  for (int st = kStHits; st <= kStFinal; ++st) grids.g[st] = g;
}

// ---------------------------------------------------------- ring sequences
__global__ __launch_bounds__(kBlock) void k_scan_partial(const uint8_t *flags, uint32_t *part, const Counters *cn) {
  if (cn->err) return;
  const uint32_t U = cn->n_unique;
  const uint32_t nb = (U + kScanChunk - 1) / kScanChunk;
  for (uint32_t b = blockIdx.x; b < nb; b += gridDim.x) {
    const uint32_t base = b * kScanChunk + threadIdx.x * kScanPerThread;
    uint32_t c = 0;
#pragma unroll
    for (int k = 0; k < kScanPerThread; ++k)
      if (base + k < U) c += flags[base + k] & kFlagEnqueue;
    const uint32_t tot = block_sum(c);
    if (threadIdx.x == 0) part[b] = tot;
  }
}

__global__ __launch_bounds__(kBlock) void k_scan_top(uint32_t *part, Counters *cn) {
  if (cn->err) return;
  const uint32_t U = cn->n_unique;
  const uint32_t nb = (U + kScanChunk - 1) / kScanChunk;
  uint32_t carry = 0;
  for (uint32_t base = 0; base < nb; base += kBlock) {
    const uint32_t i = base + threadIdx.x;
    const uint32_t v = i < nb ? part[i] : 0u;
    uint32_t tot;
    const uint32_t ex = block_exclusive_scan(v, tot);
    if (i < nb) part[i] = carry + ex;
    carry += tot;
  }
  if (threadIdx.x == 0) cn->enq_total = carry;
}

// Exclusive scan of the enqueue flags in ascending-ID order gives each
// enqueue its ring sequence number.  An enqueued line requested later in the
// same batch is told where its entry went.
// kFused: the chunk's offset is the sum of the earlier chunks' partial counts,
// added up by the block itself, and the last chunk's block records the total
// (few chunks: this saves the one-block scan); otherwise scan_part holds the
// scanned offsets.
template <bool kFused>
__global__ __launch_bounds__(kBlock) void k_scan_final(const DevState d, Scratch sc, Counters *cn) {
  if (cn->err) return;
  const uint32_t U = cn->n_unique;
  const uint64_t tail0 = d.tail[0];
  const uint32_t nb = (U + kScanChunk - 1) / kScanChunk;
  for (uint32_t b = blockIdx.x; b < nb; b += gridDim.x) {
    const uint32_t base = b * kScanChunk + threadIdx.x * kScanPerThread;
    uint32_t f[kScanPerThread];
    uint32_t c = 0;
#pragma unroll
    for (int k = 0; k < kScanPerThread; ++k) {
      f[k] = (base + k < U) ? (sc.flags[base + k] & kFlagEnqueue) : 0u;
      c += f[k];
    }
    uint32_t tot;
    const uint32_t ex = block_exclusive_scan(c, tot);
    uint32_t off;
    if constexpr (kFused) {
      uint32_t v = 0;
      for (uint32_t j = threadIdx.x; j < b; j += kBlock) v += sc.scan_part[j];
      off = block_sum(v);
      if (b == nb - 1 && threadIdx.x == 0) cn->enq_total = off + tot;
    } else {
      off = sc.scan_part[b];
    }
    uint32_t run = off + ex;
#pragma unroll
    for (int k = 0; k < kScanPerThread; ++k) {
      const uint32_t u = base + k;
      if (u < U) {
        sc.enq_before[u] = run;
        if (f[k]) {
          const uint32_t z = sc.evicted[u];
          const uint32_t v = d.uidx[z];  // stale unless z is requested in this batch
          if (v < U && v > u && sc.uniq[v] == z) {
            sc.this_q[v] = tail0 + run + 1;
            sc.this_enq[v] = u;
          }
        }
      }
      run += f[k];
    }
  }
}

// ------------------------------------------------------------ victim queues
// Queue mode (Sec. 4.3.1): an enqueue candidate u goes to the queue of its
// line's next reuse iteration j = t + distance (slot j mod (L+1)) at the
// position the queue's counter gives in ascending-u order, or is dropped when
// that position is C or more.  Per-block counts per slot, one block's scan of
// them per slot, then each candidate's rank among its block's candidates for
// the same slot (one ballot per slot).
__device__ __forceinline__ bool q_candidate(const Scratch &sc, uint32_t u, uint32_t U, uint64_t t, uint32_t slots,
                                            uint32_t &key) {
  if (u >= U || sc.kind[u] != kKindFill) return false;
  const uint32_t f = sc.flags[u];
  if (!(f & kFlagEnqueue)) return false;
  key = (uint32_t)((t + (f >> kFlagDistShift)) % slots);
  return true;
}

__global__ __launch_bounds__(kBlock) void k_qcount(const DevState d, Scratch sc, uint64_t t, const Counters *cn) {
  if (cn->err) return;
  const uint32_t U = cn->n_unique;
  const uint32_t slots = d.L + 1;
  const uint32_t nb = (U + kBlock - 1) / kBlock;
  __shared__ uint32_t cnt[kMaxQueues];
  for (uint32_t b = blockIdx.x; b < nb; b += gridDim.x) {
    if (threadIdx.x < kMaxQueues) cnt[threadIdx.x] = 0;
    __syncthreads();
    uint32_t key = 0;
    if (q_candidate(sc, b * kBlock + threadIdx.x, U, t, slots, key)) atomicAdd(&cnt[key], 1u);
    __syncthreads();
    if (threadIdx.x < slots) sc.qpart[(uint64_t)threadIdx.x * nb + b] = cnt[threadIdx.x];
    __syncthreads();
  }
}

// One block: per slot, the exclusive scan of the per-block counts, then the
// slot's placements (up to C entries in all) and the counters the finish and
// the host read.  The queue counters advance here; the placement kernel reads
// the values from before this gather from the call's counters.
__global__ __launch_bounds__(kBlock) void k_qtop(const DevState d, Scratch sc, Counters *cn) {
  if (cn->err) return;
  const uint32_t U = cn->n_unique;
  const uint32_t slots = d.L + 1;
  const uint32_t nb = (U + kBlock - 1) / kBlock;
  __shared__ uint32_t tot[kMaxQueues];
  for (uint32_t k = 0; k < slots; ++k) {
    uint32_t carry = 0;
    uint32_t *row = sc.qpart + (uint64_t)k * nb;
    for (uint32_t base = 0; base < nb; base += kBlock) {
      const uint32_t i = base + threadIdx.x;
      const uint32_t v = i < nb ? row[i] : 0u;
      uint32_t blk;
      const uint32_t ex = block_exclusive_scan(v, blk);
      if (i < nb) row[i] = carry + ex;
      carry += blk;
    }
    if (threadIdx.x == 0) tot[k] = carry;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t placed_all = 0, over = 0;
    for (uint32_t k = 0; k < slots; ++k) {
      const uint32_t before = d.qcount[k];
      const uint32_t room = (uint32_t)d.C - before;
      const uint32_t placed = tot[k] < room ? tot[k] : room;
      cn->q_before[k] = before;
      cn->q_placed[k] = placed;
      d.qcount[k] = before + placed;
      placed_all += placed;
      over += tot[k] - placed;
    }
    cn->enq_total = placed_all;
    cn->q_overflow = over;
  }
}

// Position of every candidate: the slot's entries before this gather, the
// candidates of lower blocks and those of lower lanes of this block.  A placed
// entry records its tag and its node's latest entry, and lists its row for
// staging: the gather's placements are staged slot by slot, in position order.
// Runs after the resolve kernel, which reads the nodes' entries from before
// this gather.
__global__ __launch_bounds__(kBlock) void k_qplace(const DevState d, Scratch sc, uint64_t t, Counters *cn) {
  if (cn->err) return;
  const uint32_t U = cn->n_unique;
  const uint32_t slots = d.L + 1;
  const uint32_t nb = (U + kBlock - 1) / kBlock;
  const uint32_t lane = threadIdx.x & 63u, wid = threadIdx.x >> 6;
  __shared__ uint32_t wcnt[kBlock / 64][kMaxQueues];
  __shared__ uint32_t off[kMaxQueues];
  if (threadIdx.x == 0) {
    uint32_t o = 0;
    for (uint32_t k = 0; k < slots; ++k) {
      off[k] = o;
      o += cn->q_placed[k];
    }
  }
  __syncthreads();
  uint32_t c_copy = 0;
  for (uint32_t b = blockIdx.x; b < nb; b += gridDim.x) {
    const uint32_t u = b * kBlock + threadIdx.x;
    uint32_t key = 0;
    const bool cand = q_candidate(sc, u, U, t, slots, key);
    uint32_t rank = 0;
    for (uint32_t k = 0; k < slots; ++k) {
      const uint64_t m = __ballot(cand && key == k);
      if (cand && key == k) rank = (uint32_t)__popcll(m & ((1ull << lane) - 1ull));
      if (lane == 0) wcnt[wid][k] = (uint32_t)__popcll(m);
    }
    __syncthreads();
    bool stage = false;
    uint32_t pos = 0;
    if (cand) {
      for (uint32_t w = 0; w < wid; ++w) rank += wcnt[w][key];
      const uint32_t before = cn->q_before[key];
      const uint64_t p = (uint64_t)before + sc.qpart[(uint64_t)key * nb + b] + rank;
      if (p < d.C) {
        const uint32_t z = sc.evicted[u];
        const uint64_t j = t + (sc.flags[u] >> kFlagDistShift);
        d.ring_tag[key * d.C + p] = z;
        d.vpos[z] = ((j + 1) << 32) | p;
        pos = off[key] + (uint32_t)(p - before);
        stage = true;
        ++c_copy;
      }
    }
    const uint32_t i = block_append(stage, &sc.gate->n_stage);
    if (stage) {
      sc.stage.src[i] = sc.slot[u];
      sc.stage.dst[i] = pos;
    }
  }
  block_count(c_copy, sc.stat_part, kStEnqCopy);
}

// Misses known from the batch-start state, listed right after the dedup so
// that their rows start crossing the link while the rest of the metadata
// runs: a unique ID x that no way of its set holds at batch start is filled
// at its turn (only x itself inserts x), and with no entry for it in the
// victim buffer (FIFO: no ring entry naming x; queues: no entry in the queue
// of this iteration) the fill is a miss, whatever the walk decides.  The
// resolve, which finds the same outcome, leaves these out of its list.
__global__ __launch_bounds__(kBlock) void k_early(const DevState d, Scratch sc, uint64_t t, const Counters *cn) {
  if (cn->err) return;
  const uint32_t U = cn->n_unique;
  uint32_t c_early = 0;
  for (uint32_t base = blockIdx.x * kBlock; base < U; base += gridDim.x * kBlock) {
    const uint32_t u = base + threadIdx.x;
    bool early = false;
    uint32_t x = 0;
    if (u < U) {
      x = sc.uniq[u];
      const u32x4 *tp = reinterpret_cast<const u32x4 *>(d.sets[set_index(x, d.S)].tag);
      const u32x4 a = tp[0], b = tp[1];
      const bool resident = a.x == x || a.y == x || a.z == x || a.w == x || b.x == x || b.y == x || b.z == x ||
                            b.w == x;
      if (!resident) {
        bool entry = false;
        if (d.V) {
          const uint64_t vp = d.vpos[x];
          if (d.qmode)
            entry = (vp >> 32) == t + 1;
          else if (vp)
            entry = d.ring_tag[(vp - 1) % d.V] == x;
        }
        early = !entry;
      }
      sc.early[u] = early ? 1 : 0;
      c_early += early;
    }
    const uint32_t i = block_append(early, &sc.gate->n_early);
    if (early) {
      sc.host_list[i] = u;
      sc.host_src[i] = kSrcStore | x;
    }
  }
  block_count(c_early, sc.stat_part, kStEarly);
}

void launch_early(const DevState &d, uint64_t n, uint64_t t, Scratch &sc, Counters *cn, StatGrids &grids,
                  hipStream_t s) {
  const unsigned g = grid_for(n, kBlock, kMaxGrid);
  hipLaunchKernelGGL(k_early, dim3(g), dim3(kBlock), 0, s, d, sc, t, cn);
  grids.g[kStEarly] = g;
}

// Victim-ring probe of every fill and the row source of every unique ID.  Builds
// the gather's row-copy lists: the rest of the host fetch's (rows from pinned
// host memory, after the early misses; dense, in arbitrary order), the hit
// copy's (one entry per unique ID: its HBM row, or none) and the fills' (each
// way's final occupant; dense, in arbitrary order).
__global__ __launch_bounds__(kBlock) void k_resolve(const DevState d, Scratch sc, uint64_t t, uint8_t *outcome,
                                                    Counters *cn) {
  if (cn->err) return;
  const uint32_t U = cn->n_unique;
  const uint64_t tail0 = d.tail[0], tail_prev = d.tail[1];
  const uint64_t tail_end = tail0 + cn->enq_total;
  // the previous gather's surviving entries, [q_lo_prev, tail0), were staged
  // in that order in its staging buffer
  const uint64_t q_lo_prev = tail0 - ((tail0 - tail_prev) < d.V ? (tail0 - tail_prev) : d.V);
  const uint64_t stage_prev = d.stage_row0 + ((t + 1u) & 1u) * d.stage_rows;
  const uint32_t n_early = sc.gate->n_early;  // the list's first entries, written by k_early
  uint32_t c_vhit = 0, c_miss = 0, c_hbm = 0, c_host = 0, c_vring = 0, c_vstaged = 0, c_vsame = 0;
  for (uint32_t base = blockIdx.x * kBlock; base < U; base += gridDim.x * kBlock) {
    const uint32_t u = base + threadIdx.x;
    bool from_host = false, from_hbm = false, refill = false;
    uint64_t code = 0;
    uint32_t fd = 0;
    if (u < U) {
      const uint8_t kind = sc.kind[u];
      uint8_t oc = 0;  // LSMGNN_HIT
      if (kind == kKindHit) {
        code = kSrcHbm | sc.slot[u];
        ++c_hbm;
      } else if (sc.early[u]) {  // a miss already listed (its row is on its way)
        ++c_miss;
        oc = 2;  // LSMGNN_MISS
        code = kSrcStore;
      } else if (d.qmode) {
        // queue mode: a victim hit iff the node's latest entry is in the queue
        // of this iteration, whose rows were prefetched into buffer t & 1
        const uint32_t x = sc.uniq[u];
        const uint64_t vp = d.V ? d.vpos[x] : 0;
        if ((vp >> 32) == t + 1) {
          ++c_vhit;
          oc = 1;  // LSMGNN_VICTIM_HIT
          code = kSrcHbm | (d.S * kWays + (t & 1) * d.C + (vp & 0xffffffffu));
          ++c_hbm;
        } else {
          ++c_miss;
          oc = 2;  // LSMGNN_MISS
          code = kSrcStore | x;
          ++c_host;
        }
      } else {
        const uint32_t x = sc.uniq[u];
        uint64_t q = 0;
        bool valid = false, same_batch = false;
        const uint64_t tq = sc.this_q[u];
        if (tq) {
          q = tq - 1;
          valid = true;
          same_batch = true;
        } else if (d.V) {
          const uint64_t vp = d.vpos[x];
          if (vp) {
            q = vp - 1;
            valid = d.ring_tag[q % d.V] == x;
          }
        }
        const bool live = valid && q + d.V >= tail0 + sc.enq_before[u];
        if (live) {
          ++c_vhit;
          oc = 1;  // LSMGNN_VICTIM_HIT
          if (same_batch) {
            // evicted earlier in this batch: its row is still in the cache slot
            // the evicting fill took, which no copy has overwritten yet
            const uint32_t e = sc.this_enq[u];
            code = kSrcHbm | sc.slot[e];
            sc.dead[e] = 1;
            ++c_hbm;
            ++c_vsame;
          } else {
            // The entry leaves the ring: removed now, unless an enqueue of this
            // batch takes its slot anyway.  Its row is the victim buffer's:
            //  - an entry of the previous gather is read from that gather's
            //    staging rows in HBM (its ring write may still be running);
            //  - an older one from the pinned ring.  The ring rows it is read
            //    from are overwritten only by this gather's ring write, which
            //    the runtime queues after this gather's host fetch.
            if (q + d.V >= tail_end) d.ring_tag[q % d.V] = kEmpty;
            if (q >= tail_prev) {
              code = kSrcHbm | (stage_prev + (q - q_lo_prev));
              ++c_hbm;
              ++c_vstaged;
            } else {
              code = kSrcRing | (q % d.V);
              ++c_host;
              ++c_vring;
            }
          }
        } else {
          ++c_miss;
          oc = 2;  // LSMGNN_MISS
          code = kSrcStore | x;
          ++c_host;
        }
      }
      from_host = (code & ~kSrcIndex) != kSrcHbm && !sc.early[u];
      from_hbm = (code & ~kSrcIndex) == kSrcHbm;
      fd = sc.fill_dst[u];
      refill = fd != 0;
      sc.oc[u] = oc;
      if (outcome) outcome[u] = oc;
      // the hit copy's list is indexed by unique index (its destination row),
      // so the copy writes the output rows in order
      sc.hbm.src[u] = from_hbm ? (uint32_t)(code & kSrcIndex) : kNoRow;
    }
    const uint32_t ih = n_early + block_append(from_host, &sc.gate->n_host);
    if (from_host) {
      sc.host_list[ih] = u;
      sc.host_src[ih] = code;
    }
    const uint32_t ifl = block_append(refill, &sc.gate->n_fill);
    if (refill) {
      sc.fill.src[ifl] = u;
      sc.fill.dst[ifl] = fd - 1;
    }
  }
  block_count(c_vhit, sc.stat_part, kStVictimHits);
  block_count(c_miss, sc.stat_part, kStMisses);
  block_count(c_hbm, sc.stat_part, kStHbm);
  block_count(c_host, sc.stat_part, kStHost);
  block_count(c_vring, sc.stat_part, kStVhRing);
  block_count(c_vstaged, sc.stat_part, kStVhStaged);
  block_count(c_vsame, sc.stat_part, kStVhSame);
}

// Outcomes per raw request: each request takes its unique ID's outcome (the
// compaction recorded every requested node's unique index).
__device__ __forceinline__ void request_counts(const DevState &d, const Scratch &sc, const int64_t *ids,
                                               uint32_t n) {
  uint32_t c_hit = 0, c_vhit = 0;
  for (uint32_t i = blockIdx.x * kBlock + threadIdx.x; i < n; i += gridDim.x * kBlock) {
    const uint8_t o = sc.oc[d.uidx[ids[i]]];
    c_hit += o == 0;   // LSMGNN_HIT
    c_vhit += o == 1;  // LSMGNN_VICTIM_HIT
  }
  block_count(c_hit, sc.stat_part, kStReqHits);
  block_count(c_vhit, sc.stat_part, kStReqVictimHits);
}

__global__ __launch_bounds__(kBlock) void k_request_counts(const DevState d, Scratch sc, const int64_t *ids,
                                                           uint32_t n, const Counters *cn) {
  if (cn->err) return;
  request_counts(d, sc, ids, n);
}


// Ring bookkeeping for this batch's enqueues; lists the row copies of the
// entries that are still in the ring at the end of the batch.  Those entries
// have the sequence numbers [q_lo, tail_end), q_lo = tail_end - min(E, V) for E
// enqueues, and their rows are staged in that order (entries removed again in
// this batch leave a hole that nothing reads).
__global__ __launch_bounds__(kBlock) void k_enq_finalize(const DevState d, Scratch sc, const int64_t *ids, uint32_t n,
                                                         Counters *cn) {
  if (cn->err) return;
  const uint32_t U = cn->n_unique;
  const uint64_t tail0 = d.tail[0];
  const uint64_t E = cn->enq_total;
  const uint64_t tail_end = tail0 + E;
  const uint64_t q_lo = tail_end - (E < d.V ? E : d.V);
  uint32_t c_copy = 0;
  for (uint32_t base = blockIdx.x * kBlock; base < U; base += gridDim.x * kBlock) {
    const uint32_t u = base + threadIdx.x;
    bool stage = false;
    uint32_t pos = 0;
    if (u < U && sc.kind[u] == kKindFill && (sc.flags[u] & kFlagEnqueue)) {
      const uint64_t q = tail0 + sc.enq_before[u];
      const uint32_t z = sc.evicted[u];
      d.vpos[z] = q + 1;
      if (q + d.V >= tail_end) {
        if (sc.dead[u]) {
          d.ring_tag[q % d.V] = kEmpty;
        } else {
          d.ring_tag[q % d.V] = z;
          stage = true;
          pos = (uint32_t)(q - q_lo);
          ++c_copy;
        }
      }
    }
    const uint32_t i = block_append(stage, &sc.gate->n_stage);
    if (stage) {
      sc.stage.src[i] = sc.slot[u];
      sc.stage.dst[i] = pos;
    }
  }
  block_count(c_copy, sc.stat_part, kStEnqCopy);
  // the per-request outcome counts, in the same launch
  request_counts(d, sc, ids, n);
}

void launch_ring_resolve(const DevState &d, uint64_t n, uint64_t t, Scratch &sc, uint8_t *outcome, Counters *cn,
                         StatGrids &grids, hipStream_t s) {
  const unsigned g = grid_for(n, kBlock, kMaxGrid);
  const unsigned gs = grid_for(n, kScanChunk, kMaxGrid);
  const bool ring = d.V && !d.qmode;
  const bool queues = d.V && d.qmode && d.L > 0;  // with L = 0 no line has a reuse iteration
  if (ring) {
    hipLaunchKernelGGL(k_scan_partial, dim3(gs), dim3(kBlock), 0, s, sc.flags, sc.scan_part, cn);
    if ((n + kScanChunk - 1) / kScanChunk <= kFusedScanMax) {
      hipLaunchKernelGGL(k_scan_final<true>, dim3(gs), dim3(kBlock), 0, s, d, sc, cn);
    } else {
      hipLaunchKernelGGL(k_scan_top, dim3(1), dim3(kBlock), 0, s, sc.scan_part, cn);
      hipLaunchKernelGGL(k_scan_final<false>, dim3(gs), dim3(kBlock), 0, s, d, sc, cn);
    }
  }
  if (queues) {
    hipLaunchKernelGGL(k_qcount, dim3(g), dim3(kBlock), 0, s, d, sc, t, cn);
    hipLaunchKernelGGL(k_qtop, dim3(1), dim3(kBlock), 0, s, d, sc, cn);
  }
  hipLaunchKernelGGL(k_resolve, dim3(g), dim3(kBlock), 0, s, d, sc, t, outcome, cn);
  for (int st = kStVictimHits; st <= kStHost; ++st) grids.g[st] = g;
  for (int st = kStVhRing; st <= kStVhSame; ++st) grids.g[st] = g;
}

void launch_ring_enqueue(const DevState &d, const int64_t *ids, uint64_t n, uint64_t t, Scratch &sc, Counters *cn,
                         StatGrids &grids, hipStream_t s) {
  const unsigned g = grid_for(n, kBlock, kMaxGrid);
  const bool ring = d.V && !d.qmode;
  const bool queues = d.V && d.qmode && d.L > 0;
  if (ring) {  // with the per-request counts
    hipLaunchKernelGGL(k_enq_finalize, dim3(g), dim3(kBlock), 0, s, d, sc, ids, (uint32_t)n, cn);
    grids.g[kStEnqCopy] = g;
  } else {
    if (queues) {
      hipLaunchKernelGGL(k_qplace, dim3(g), dim3(kBlock), 0, s, d, sc, t, cn);
      grids.g[kStEnqCopy] = g;
    }
    hipLaunchKernelGGL(k_request_counts, dim3(g), dim3(kBlock), 0, s, d, sc, ids, (uint32_t)n, cn);
  }
  grids.g[kStReqHits] = g;
  grids.g[kStReqVictimHits] = g;
}

// -------------------------------------------------------------- row copies
// Work item w = (unique index e, 16-byte vector v): consecutive lanes take
// consecutive vectors of one row, so a wave moves whole rows with 128-bit
// accesses, and each lane keeps kUnroll vectors in flight before storing.
// The HBM-side modes read the per-unique descriptor and skip rows they do not
// own; the host fetch walks the dense host-fetch list instead.  Counts come
// from the gather's gate; a rejected gather moves nothing.
constexpr int kUnroll = 4;

// Copy of a row list: item w = (list entry i, 16-byte vector v).  Each block
// takes a tile of kListUnroll * kBlock consecutive items (whole rows, their
// 16-byte vectors on consecutive lanes), the tiles striding over the grid;
// loads and stores carry the non-temporal hint (every row moves once).
// Measured on the MI355X against grid-strided items without the hint:
// 5.7-6.0 against 4.9-5.2 TB/s for 1-2 KiB random rows.  The mode only names
// the instance (hit copy, staging, fills) so that profiles tell them apart.
constexpr int kListUnroll = 2;
//
// The hit copy's list (M = kHbmToOut) is dense by destination: entry i moves
// to output row i, from row sidx[i] unless that is kNoRow (the unique ID's
// row comes over the host link).  Writing the output rows in order measured
// 6.0 TB/s against 5.2-5.4 for the same rows listed in per-block runs of
// arbitrary order (600 K random 2 KiB rows from a 96 GiB region).
template <CopyMode M, bool kPow2>
__global__ __launch_bounds__(kBlock) void k_list_copy(const uint8_t *src, const uint32_t *sidx, uint8_t *dst,
                                                      const uint32_t *didx, const Gate *gate, const uint32_t *count,
                                                      uint64_t R, uint32_t nvec, uint32_t vshift) {
  constexpr bool kDense = M == CopyMode::kHbmToOut;
  if (gate->err) return;
  const uint64_t total = (uint64_t)*count * nvec;
  constexpr uint64_t tile = (uint64_t)kListUnroll * kBlock;
  for (uint64_t base = (uint64_t)blockIdx.x * tile; base < total; base += (uint64_t)gridDim.x * tile) {
    u32x4 v[kListUnroll];
    uint8_t *dp[kListUnroll];
#pragma unroll
    for (int k = 0; k < kListUnroll; ++k) {
      const uint64_t w = base + (uint64_t)k * kBlock + threadIdx.x;
      dp[k] = nullptr;
      if (w < total) {
        const uint32_t i = kPow2 ? (uint32_t)(w >> vshift) : (uint32_t)(w / nvec);
        const uint64_t byte = (w - (uint64_t)i * nvec) * 16u;
        const uint32_t si = sidx[i];
        if (!kDense || si != kNoRow) {
          v[k] = __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(src + (uint64_t)si * R + byte));
          dp[k] = dst + (uint64_t)(kDense ? i : didx[i]) * R + byte;
        }
      }
    }
#pragma unroll
    for (int k = 0; k < kListUnroll; ++k)
      if (dp[k]) __builtin_nontemporal_store(v[k], reinterpret_cast<u32x4 *>(dp[k]));
  }
}

// Host fetch: item w = (host-list entry i, 16-byte vector v).  The list entry
// is the same for all lanes of a row (broadcast loads), and the entries of the
// next pass are loaded while this pass's host reads are in flight, so the
// reads never wait behind a dependent HBM load.  With a pageable store the
// host has already copied entry i's row to bounce row i.
#ifndef LSM_HOST_UNROLL
#define LSM_HOST_UNROLL 4
#endif
//
// The list has two parts: its first n_early entries (misses known at batch
// start, `late` false) and the n_host entries after them (the resolve's,
// `late` true); each launch moves one part.
template <bool kPow2>
__global__ __launch_bounds__(kBlock) void k_host_fetch(const DevState d, Scratch sc, uint8_t *out, uint32_t nvec,
                                                       uint32_t vshift, int late) {
  constexpr int kU = LSM_HOST_UNROLL;
  const Gate g = *sc.gate;
  if (g.err) return;
  const uint64_t R = d.R;
  const uint32_t first = late ? g.n_early : 0u;
  const uint64_t total = (uint64_t)(late ? g.n_host : g.n_early) * nvec;
  const uint64_t stride = (uint64_t)gridDim.x * kBlock;
  const uint32_t *list = sc.host_list + first;
  const uint64_t *src = sc.host_src + first;
  const u32x4 *bounce = sc.bounce ? reinterpret_cast<const u32x4 *>(sc.bounce) + (uint64_t)first * nvec : nullptr;
  auto entry = [&](uint64_t w, uint32_t &e, uint64_t &code) {
    if (w < total) {
      const uint32_t i = kPow2 ? (uint32_t)(w >> vshift) : (uint32_t)(w / nvec);
      e = list[i];
      code = src[i];
    }
  };
  uint32_t e[kU];
  uint64_t code[kU];
  uint64_t w0 = (uint64_t)blockIdx.x * kBlock + threadIdx.x;
#pragma unroll
  for (int k = 0; k < kU; ++k) entry(w0 + k * stride, e[k], code[k]);
  for (; w0 < total; w0 += stride * kU) {
    u32x4 v[kU];
    uint8_t *dst[kU];
#pragma unroll
    for (int k = 0; k < kU; ++k) {
      const uint64_t w = w0 + k * stride;
      dst[k] = nullptr;
      if (w < total) {
        const uint64_t byte = (kPow2 ? (w & (nvec - 1)) : (w % nvec)) * 16u;
        // bounce row i holds entry i: vector w is the w-th of the buffer
        const u32x4 *sp =
            bounce ? bounce + w
                   : reinterpret_cast<const u32x4 *>(
                            ((code[k] & ~kSrcIndex) == kSrcRing ? d.ring_rows : d.store) + (code[k] & kSrcIndex) * R +
                            byte);
        v[k] = *sp;
        dst[k] = out + (uint64_t)e[k] * R + byte;
      }
    }
    const uint64_t w1 = w0 + stride * kU;
#pragma unroll
    for (int k = 0; k < kU; ++k) entry(w1 + k * stride, e[k], code[k]);
    // the output rows are written once and read next by other kernels: the
    // non-temporal hint keeps them from displacing what the kernels beside
    // this one hold in L2 (measured: never slower, up to 3.5 % faster on the
    // 100M-node workload)
#pragma unroll
    for (int k = 0; k < kU; ++k)
      if (dst[k]) __builtin_nontemporal_store(v[k], reinterpret_cast<u32x4 *>(dst[k]));
  }
}

// Grid caps.  Every outstanding host-link read queues in front of the memory
// requests of the kernels that run beside it (the next gather's metadata, the
// hit copy, the fills, the ring write), so the host fetch keeps only about
// 640 KB in flight (40 blocks x 256 lanes x 4 x 16 B): enough to cover the
// link's latency, not more.  A sweep of block counts and unroll depths on
// the full pipeline chose it.  The runtime picks another grid per gather
// (DevState::host_grid): fewer blocks when more traffic shares the host or
// the link, more when the fetch reads a pageable store's contiguous bounce
// rows.
#ifndef LSM_HOST_GRID
#define LSM_HOST_GRID 40
#endif
#ifndef LSM_HBM_GRID
#define LSM_HBM_GRID 65536  // the HBM-side copies: the largest grid of the measured sweep
#endif

template <CopyMode M>
static void launch_list(const uint8_t *src, const RowList &l, uint8_t *dst, const Gate *gate, const uint32_t *count,
                        uint64_t n, uint64_t R, hipStream_t s) {
  const uint32_t nvec = (uint32_t)(R / 16);
  const unsigned g = grid_for(n * nvec, (uint64_t)kBlock * kListUnroll, LSM_HBM_GRID);
  if ((nvec & (nvec - 1)) == 0)
    hipLaunchKernelGGL((k_list_copy<M, true>), dim3(g), dim3(kBlock), 0, s, src, l.src, dst, l.dst, gate, count, R,
                       nvec, (uint32_t)__builtin_ctz(nvec));
  else
    hipLaunchKernelGGL((k_list_copy<M, false>), dim3(g), dim3(kBlock), 0, s, src, l.src, dst, l.dst, gate, count, R,
                       nvec, 0u);
}

void launch_copy(CopyMode mode, const DevState &d, uint64_t n, const Scratch &sc, uint8_t *out, hipStream_t s) {
  const uint32_t nvec = (uint32_t)(d.R / 16);
  const bool pow2 = (nvec & (nvec - 1)) == 0;
  const uint32_t vshift = pow2 ? (uint32_t)__builtin_ctz(nvec) : 0u;
  if (mode == CopyMode::kHostToOut || mode == CopyMode::kHostEarly) {
    const unsigned g = grid_for(n * nvec, (uint64_t)kBlock * kUnroll, d.host_grid ? d.host_grid : LSM_HOST_GRID);
    const int late = mode == CopyMode::kHostToOut;
    if (pow2)
      hipLaunchKernelGGL((k_host_fetch<true>), dim3(g), dim3(kBlock), 0, s, d, sc, out, nvec, vshift, late);
    else
      hipLaunchKernelGGL((k_host_fetch<false>), dim3(g), dim3(kBlock), 0, s, d, sc, out, nvec, vshift, late);
    return;
  }
  switch (mode) {
    case CopyMode::kHbmToOut:
      launch_list<CopyMode::kHbmToOut>(d.rows, sc.hbm, out, sc.gate, &sc.gate->n_unique, n, d.R, s);
      break;
    case CopyMode::kCacheToStage:
      launch_list<CopyMode::kCacheToStage>(d.rows, sc.stage, sc.staging, sc.gate, &sc.gate->n_stage, n, d.R, s);
      break;
    default:
      launch_list<CopyMode::kOutToCache>(out, sc.fill, d.rows, sc.gate, &sc.gate->n_fill, n, d.R, s);
      break;
  }
}

// Queue mode: the queue of the next gather into its prefetch buffer.  Rows of
// entries placed by earlier gathers cross the host link (a small grid, like
// the host fetch); those placed by the gather just issued are still in its
// staging rows in HBM.
__global__ __launch_bounds__(kBlock) void k_prefetch(const DevState d, const Gate *gate, const uint8_t *staging,
                                                     uint32_t slot, uint32_t par, uint32_t nvec) {
  const uint32_t cnt = gate->q_count, before = gate->q_before, off = gate->q_stage_off;
  const uint64_t R = d.R;
  const uint64_t total = (uint64_t)cnt * nvec;
  const uint64_t stride = (uint64_t)gridDim.x * kBlock;
  uint8_t *pf = d.rows + (d.S * kWays + (uint64_t)par * d.C) * R;
  const uint8_t *q = d.ring_rows + (uint64_t)slot * d.C * R;
  for (uint64_t w0 = (uint64_t)blockIdx.x * kBlock + threadIdx.x; w0 < total; w0 += stride * kUnroll) {
    u32x4 v[kUnroll];
    uint8_t *dp[kUnroll];
#pragma unroll
    for (int k = 0; k < kUnroll; ++k) {
      const uint64_t w = w0 + k * stride;
      dp[k] = nullptr;
      if (w < total) {
        const uint64_t i = w / nvec;
        const uint64_t byte = (w - i * nvec) * 16u;
        const uint8_t *src = i < before ? q + i * R + byte : staging + (off + (i - before)) * R + byte;
        v[k] = *reinterpret_cast<const u32x4 *>(src);
        dp[k] = pf + i * R + byte;
      }
    }
#pragma unroll
    for (int k = 0; k < kUnroll; ++k)
      if (dp[k]) *reinterpret_cast<u32x4 *>(dp[k]) = v[k];
  }
}

void launch_prefetch(const DevState &d, const Gate *gate, const uint8_t *staging, uint32_t slot, uint32_t par,
                     hipStream_t s) {
  hipLaunchKernelGGL(k_prefetch, dim3(LSM_HOST_GRID), dim3(kBlock), 0, s, d, gate, staging, slot, par,
                     (uint32_t)(d.R / 16));
}

// ------------------------------------------------------------ calibration
// Plain contiguous copy with the same 128-bit access pattern and unrolling as
// the row copies; used to measure the host-link and HBM ceilings and to scale
// hardware byte counters against a copy of known size.
__global__ __launch_bounds__(kBlock) void k_copy_plain(const u32x4 *src, u32x4 *dst, uint64_t nvec) {
  const uint64_t stride = (uint64_t)gridDim.x * kBlock;
  for (uint64_t w0 = (uint64_t)blockIdx.x * kBlock + threadIdx.x; w0 < nvec; w0 += stride * kUnroll) {
    u32x4 v[kUnroll];
#pragma unroll
    for (int k = 0; k < kUnroll; ++k) {
      const uint64_t w = w0 + k * stride;
      if (w < nvec) v[k] = src[w];
    }
#pragma unroll
    for (int k = 0; k < kUnroll; ++k) {
      const uint64_t w = w0 + k * stride;
      if (w < nvec) dst[w] = v[k];
    }
  }
}

__global__ void k_publish_count(const Gate *gate, const uint32_t *count, uint32_t *dst) {
  if (threadIdx.x == 0) *dst = gate->err ? 0u : *count;
}

void launch_publish_count(const Gate *gate, const uint32_t *count, uint32_t *dst, hipStream_t s) {
  hipLaunchKernelGGL(k_publish_count, dim3(1), dim3(64), 0, s, gate, count, dst);
}

// Device-to-device: tiles of 4 * kBlock vectors per block with the
// non-temporal hint, the copy pattern of the row lists.
__global__ __launch_bounds__(kBlock) void k_copy_tiles(const u32x4 *src, u32x4 *dst, uint64_t nvec) {
  constexpr uint64_t tile = 4 * (uint64_t)kBlock;
  for (uint64_t base = (uint64_t)blockIdx.x * tile; base < nvec; base += (uint64_t)gridDim.x * tile) {
    u32x4 v[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const uint64_t w = base + (uint64_t)k * kBlock + threadIdx.x;
      if (w < nvec) v[k] = __builtin_nontemporal_load(src + w);
    }
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const uint64_t w = base + (uint64_t)k * kBlock + threadIdx.x;
      if (w < nvec) __builtin_nontemporal_store(v[k], dst + w);
    }
  }
}

void launch_copy_plain(const void *src, void *dst, uint64_t bytes, bool device_to_device, hipStream_t s) {
  const uint64_t nvec = bytes / 16;
  if (device_to_device)
    hipLaunchKernelGGL(k_copy_tiles, dim3(grid_for(nvec, 4 * (uint64_t)kBlock, 262144)), dim3(kBlock), 0, s,
                       static_cast<const u32x4 *>(src), static_cast<u32x4 *>(dst), nvec);
  else
    hipLaunchKernelGGL(k_copy_plain, dim3(grid_for(nvec, (uint64_t)kBlock * kUnroll, 4096)), dim3(kBlock), 0, s,
                       static_cast<const u32x4 *>(src), static_cast<u32x4 *>(dst), nvec);
}

// ------------------------------------------------------------------ window
// Announce: validate the IDs and, when the list is recorded, copy it into its
// window slot and set the minibatch's bit for every ID.  Only that bit of a
// node's window word changes in this kernel (duplicates write the same value),
// so a plain read-modify-write is exact.
__global__ void k_window_set(const int64_t *ids, uint32_t n, uint64_t N, uint32_t bit, uint32_t *mask,
                             int64_t *slot_ids, int record, uint32_t *err) {
  bool bad = false;
  const uint32_t b = 1u << bit;
  for (uint32_t i = blockIdx.x * kBlock + threadIdx.x; i < n; i += gridDim.x * kBlock) {
    const int64_t x = ids[i];
    if (x < 0 || (uint64_t)x >= N) {
      bad = true;
    } else if (record) {
      slot_ids[i] = x;
      const uint32_t m = mask[x];
      if (!(m & b)) mask[x] = m | b;
    }
  }
  if (__ballot(bad) && __lane_id() == 0) *err = 1u;  // every writer stores the same value
}

// After a rejected announcement (the host launches it only then): clear the
// bit again (it was clear before, since the minibatch that last used this bit
// position has been gathered).
__global__ void k_window_rollback(const int64_t *ids, uint32_t n, uint64_t N, uint32_t bit, uint32_t *mask) {
  for (uint32_t i = blockIdx.x * kBlock + threadIdx.x; i < n; i += gridDim.x * kBlock) {
    const int64_t x = ids[i];
    if (x >= 0 && (uint64_t)x < N) {
      const uint32_t m = mask[x];
      if (m & (1u << bit)) mask[x] = m & ~(1u << bit);
    }
  }
}

void launch_window_set(const int64_t *ids, uint64_t n, uint64_t N, uint32_t bit, uint32_t *mask, int64_t *slot_ids,
                       bool record, uint32_t *err, hipStream_t s) {
  const unsigned g = grid_for(n, kBlock, kMaxGrid);
  hipLaunchKernelGGL(k_window_set, dim3(g), dim3(kBlock), 0, s, ids, (uint32_t)n, N, bit, mask, slot_ids,
                     record ? 1 : 0, err);
}

void launch_window_rollback(const int64_t *ids, uint64_t n, uint64_t N, uint32_t bit, uint32_t *mask,
                            hipStream_t s) {
  const unsigned g = grid_for(n, kBlock, kMaxGrid);
  hipLaunchKernelGGL(k_window_rollback, dim3(g), dim3(kBlock), 0, s, ids, (uint32_t)n, N, bit, mask);
}

// Announcement made together with a gather: the gather's mark kernel has
// validated the IDs, and its gate says whether the call was accepted.  Records
// the list in its window slot and sets the minibatch's bit for every ID (only
// that bit changes in this kernel, so a plain read-modify-write is exact).
// ------------------------------------------------------ request order
// Per-position output: row i of `out` <- row inv[i] of `rows` (the unique-row
// output of a gather), for the n requests in their original order.  Item w =
// (request i, 16-byte vector v); the inverse entry is a broadcast load.
template <bool kPow2>
__global__ __launch_bounds__(kBlock) void k_expand(const uint8_t *rows, const int64_t *inv, uint64_t n, uint64_t R,
                                                   uint32_t nvec, uint32_t vshift, uint8_t *out) {
  const uint64_t total = n * nvec;
  const uint64_t stride = (uint64_t)gridDim.x * kBlock;
  for (uint64_t w0 = (uint64_t)blockIdx.x * kBlock + threadIdx.x; w0 < total; w0 += stride * kUnroll) {
    u32x4 v[kUnroll];
    uint8_t *dp[kUnroll];
#pragma unroll
    for (int k = 0; k < kUnroll; ++k) {
      const uint64_t w = w0 + k * stride;
      dp[k] = nullptr;
      if (w < total) {
        const uint64_t i = kPow2 ? (w >> vshift) : (w / nvec);
        const uint64_t byte = (w - i * nvec) * 16u;
        v[k] = *reinterpret_cast<const u32x4 *>(rows + (uint64_t)inv[i] * R + byte);
        dp[k] = out + i * R + byte;
      }
    }
#pragma unroll
    for (int k = 0; k < kUnroll; ++k)
      if (dp[k]) *reinterpret_cast<u32x4 *>(dp[k]) = v[k];
  }
}

void launch_expand(const uint8_t *rows, const int64_t *inv, uint64_t n, uint64_t R, uint8_t *out, hipStream_t s) {
  const uint32_t nvec = (uint32_t)(R / 16);
  const unsigned g = grid_for(n * nvec, (uint64_t)kBlock * kListUnroll, LSM_HBM_GRID);
  if ((nvec & (nvec - 1)) == 0)
    hipLaunchKernelGGL(k_expand<true>, dim3(g), dim3(kBlock), 0, s, rows, inv, n, R, nvec,
                       (uint32_t)__builtin_ctz(nvec), out);
  else
    hipLaunchKernelGGL(k_expand<false>, dim3(g), dim3(kBlock), 0, s, rows, inv, n, R, nvec, 0u, out);
}

}  // namespace lsm
