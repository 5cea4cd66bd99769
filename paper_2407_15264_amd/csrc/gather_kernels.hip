// gfx950 kernels of the feature-gather cache (LSM-GNN, arXiv 2407.15264).
//
// One gather runs as a short pipeline of stream-ordered kernels.  Every count
// that depends on the batch (unique IDs, touched sets, work-list lengths) stays
// in device memory, so the host launches the whole pipeline without waiting and
// synchronises once at the end.  Each kernel reads Counters::err first and does
// nothing once an out-of-range ID was seen, so an invalid batch changes no state.
//
//   dedup       bitmap over node IDs: mark, per-chunk popcount, chunk scan,
//               ascending compaction (ballot-free: one thread per 8 words),
//               inverse index by rank = prefix + popcount below the bit
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
//               and victim hits pinned host->out, enqueues HBM->pinned ring,
//               then fills out->HBM for each way's final occupant
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

__device__ __forceinline__ uint32_t lanes_below(uint64_t m) {
  return __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
}

// Wave-aggregated append: every lane of the wave must call this.  Returns the
// list index for lanes with pred set (one atomic per wave).
__device__ __forceinline__ uint32_t wave_append(bool pred, uint32_t *counter) {
  const uint64_t m = __ballot(pred);
  uint32_t base = 0;
  if (m) {
    const int leader = __ffsll((unsigned long long)m) - 1;
    if ((int)__lane_id() == leader) base = atomicAdd(counter, (uint32_t)__popcll(m));
    base = __shfl(base, leader);
  }
  return base + lanes_below(m);
}

__device__ __forceinline__ uint32_t wave_sum(uint32_t v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

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

static inline unsigned grid_for(uint64_t work, uint64_t per_block, unsigned cap) {
  uint64_t b = (work + per_block - 1) / per_block;
  if (b < 1) b = 1;
  if (b > cap) b = cap;
  return (unsigned)b;
}
constexpr unsigned kMaxGrid = 8192;

// ------------------------------------------------------------------- begin
__global__ void k_begin(Counters *cn) {
  uint32_t *p = reinterpret_cast<uint32_t *>(cn);
  for (unsigned i = threadIdx.x; i < sizeof(Counters) / 4; i += blockDim.x) p[i] = 0;
}

void launch_begin(Counters *cn, hipStream_t s) { hipLaunchKernelGGL(k_begin, dim3(1), dim3(64), 0, s, cn); }

// ---------------------------------------------------------------- validate
__global__ void k_validate(const int64_t *ids, uint32_t n, uint64_t N, Counters *cn) {
  bool bad = false;
  for (uint32_t i = blockIdx.x * kBlock + threadIdx.x; i < n; i += gridDim.x * kBlock) {
    const int64_t x = ids[i];
    bad |= (x < 0) | ((uint64_t)x >= N);
  }
  if (__ballot(bad) && __lane_id() == 0) atomicOr(&cn->err, 1u);
}

void launch_validate(const int64_t *ids, uint64_t n, uint64_t N, Counters *cn, hipStream_t s) {
  hipLaunchKernelGGL(k_validate, dim3(grid_for(n, kBlock, kMaxGrid)), dim3(kBlock), 0, s, ids, (uint32_t)n, N, cn);
}

// ------------------------------------------------------------------- dedup
__global__ void k_mark(const int64_t *ids, uint32_t n, uint32_t *bitmap, const Counters *cn) {
  if (cn->err) return;
  for (uint32_t i = blockIdx.x * kBlock + threadIdx.x; i < n; i += gridDim.x * kBlock) {
    const uint32_t x = (uint32_t)ids[i];
    atomicOr(&bitmap[x >> 5], 1u << (x & 31u));
  }
}

__device__ __forceinline__ void load_words(const uint32_t *bitmap, uint32_t (&w)[kWordsPerThread]) {
  const u32x4 *p = reinterpret_cast<const u32x4 *>(bitmap + (size_t)blockIdx.x * kChunkWords +
                                                    threadIdx.x * kWordsPerThread);
  const u32x4 a = p[0], b = p[1];
  w[0] = a.x; w[1] = a.y; w[2] = a.z; w[3] = a.w;
  w[4] = b.x; w[5] = b.y; w[6] = b.z; w[7] = b.w;
}

__global__ __launch_bounds__(kBlock) void k_chunk_popc(const uint32_t *bitmap, uint32_t *chunk_sums,
                                                       const Counters *cn) {
  if (cn->err) return;
  uint32_t w[kWordsPerThread];
  load_words(bitmap, w);
  uint32_t c = 0;
#pragma unroll
  for (int k = 0; k < kWordsPerThread; ++k) c += __popc(w[k]);
  const uint32_t tot = block_sum(c);
  if (threadIdx.x == 0) chunk_sums[blockIdx.x] = tot;
}

__global__ __launch_bounds__(kBlock) void k_chunk_scan(uint32_t *chunk_sums, uint32_t nchunks, Counters *cn) {
  if (cn->err) return;
  uint32_t carry = 0;
  for (uint32_t base = 0; base < nchunks; base += kBlock) {
    const uint32_t i = base + threadIdx.x;
    const uint32_t v = i < nchunks ? chunk_sums[i] : 0u;
    uint32_t tot;
    const uint32_t ex = block_exclusive_scan(v, tot);
    if (i < nchunks) chunk_sums[i] = carry + ex;
    carry += tot;
  }
  if (threadIdx.x == 0) cn->n_unique = carry;
}

__global__ __launch_bounds__(kBlock) void k_compact(const uint32_t *bitmap, const uint32_t *chunk_off,
                                                    uint32_t *word_rank, uint32_t *uniq, int64_t *uniq_out,
                                                    const Counters *cn) {
  if (cn->err) return;
  uint32_t w[kWordsPerThread];
  load_words(bitmap, w);
  uint32_t c = 0;
#pragma unroll
  for (int k = 0; k < kWordsPerThread; ++k) c += __popc(w[k]);
  uint32_t tot;
  const uint32_t ex = block_exclusive_scan(c, tot);
  if (tot == 0) return;
  uint32_t pos = chunk_off[blockIdx.x] + ex;
  const size_t w0 = (size_t)blockIdx.x * kChunkWords + threadIdx.x * kWordsPerThread;
#pragma unroll
  for (int k = 0; k < kWordsPerThread; ++k) {
    uint32_t word = w[k];
    if (word) {
      word_rank[w0 + k] = pos;
      const uint32_t idbase = (uint32_t)((w0 + k) * 32u);
      while (word) {
        const uint32_t x = idbase + (uint32_t)__builtin_ctz(word);
        uniq[pos] = x;
        uniq_out[pos] = (int64_t)x;
        ++pos;
        word &= word - 1u;
      }
    }
  }
}

__global__ void k_inverse(const int64_t *ids, uint32_t n, const uint32_t *bitmap, const uint32_t *word_rank,
                          int64_t *inv, const Counters *cn) {
  if (cn->err) return;
  for (uint32_t i = blockIdx.x * kBlock + threadIdx.x; i < n; i += gridDim.x * kBlock) {
    const uint32_t x = (uint32_t)ids[i];
    const uint32_t wi = x >> 5, b = x & 31u;
    inv[i] = (int64_t)(word_rank[wi] + __popc(bitmap[wi] & ((1u << b) - 1u)));
  }
}

void launch_dedup(const DevState &d, const int64_t *ids, uint64_t n, Scratch &sc, int64_t *unique_out,
                  int64_t *inverse, Counters *cn, hipStream_t s) {
  const unsigned g = grid_for(n, kBlock, kMaxGrid);
  hipLaunchKernelGGL(k_mark, dim3(g), dim3(kBlock), 0, s, ids, (uint32_t)n, d.bitmap, cn);
  hipLaunchKernelGGL(k_chunk_popc, dim3((unsigned)d.nchunks), dim3(kBlock), 0, s, d.bitmap, d.chunk_sums, cn);
  hipLaunchKernelGGL(k_chunk_scan, dim3(1), dim3(kBlock), 0, s, d.chunk_sums, (uint32_t)d.nchunks, cn);
  hipLaunchKernelGGL(k_compact, dim3((unsigned)d.nchunks), dim3(kBlock), 0, s, d.bitmap, d.chunk_sums,
                     d.word_rank, sc.uniq, unique_out, cn);
  if (inverse)
    hipLaunchKernelGGL(k_inverse, dim3(g), dim3(kBlock), 0, s, ids, (uint32_t)n, d.bitmap, d.word_rank, inverse,
                       cn);
}

// ------------------------------------------------------------ group by set
__global__ __launch_bounds__(kBlock) void k_claim(const DevState d, Scratch sc, Counters *cn) {
  if (cn->err) return;
  const uint32_t U = cn->n_unique;
  const uint32_t lane = threadIdx.x & 63u;
  for (uint32_t base = blockIdx.x * kBlock + (threadIdx.x - lane); base < U; base += gridDim.x * kBlock) {
    const uint32_t u = base + lane;
    bool claim = false;
    uint32_t s = 0;
    if (u < U) {
      const uint32_t x = sc.uniq[u];
      s = set_index(x, d.S);
      sc.uset[u] = s;
      sc.ustat[u] = d.stat[x];
      const uint32_t old = atomicAdd(&d.set_count[s], 1u);
      sc.arrival[u] = old;
      claim = (old == 0);
      sc.flags[u] = 0;
      sc.dead[u] = 0;
      sc.this_q[u] = 0;
      d.bitmap[x >> 5] = 0;  // every marked word holds only IDs of this batch
    }
    const uint32_t i = wave_append(claim, &cn->n_touched);
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
  }
}

__global__ void k_place(const DevState d, Scratch sc, const Counters *cn) {
  if (cn->err) return;
  const uint32_t U = cn->n_unique;
  for (uint32_t u = blockIdx.x * kBlock + threadIdx.x; u < U; u += gridDim.x * kBlock)
    sc.seg[sc.seg_off[d.set_idx[sc.uset[u]]] + sc.arrival[u]] = u;
}

__global__ void k_rank(const DevState d, Scratch sc, const Counters *cn) {
  if (cn->err) return;
  const uint32_t U = cn->n_unique;
  for (uint32_t u = blockIdx.x * kBlock + threadIdx.x; u < U; u += gridDim.x * kBlock) {
    const uint32_t s = sc.uset[u];
    const uint32_t off = sc.seg_off[d.set_idx[s]];
    const uint32_t k = d.set_count[s];
    uint32_t r = 0;
    if (k > 1)
      for (uint32_t j = 0; j < k; ++j) r += sc.seg[off + j] < u ? 1u : 0u;
    sc.sorted[off + r] = u;
  }
}

void launch_group_by_set(const DevState &d, uint64_t n, Scratch &sc, Counters *cn, hipStream_t s) {
  const unsigned g = grid_for(n, kBlock, kMaxGrid);
  hipLaunchKernelGGL(k_claim, dim3(g), dim3(kBlock), 0, s, d, sc, cn);
  hipLaunchKernelGGL(k_seg_alloc, dim3(g), dim3(kBlock), 0, s, d, sc, cn);
  hipLaunchKernelGGL(k_place, dim3(g), dim3(kBlock), 0, s, d, sc, cn);
  hipLaunchKernelGGL(k_rank, dim3(g), dim3(kBlock), 0, s, d, sc, cn);
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

// eviction level, lowest evicted first: none < far < recent < near, or with
// the victim ring on, far < none < recent < near
__device__ __forceinline__ uint32_t level_of(uint32_t cls, bool ring_on) {
  return (ring_on && cls <= kClsFar) ? (cls ^ 1u) : cls;
}

template <typename T>
__device__ __forceinline__ T pick_of(const T (&a)[kWays], int w) {
  T r = a[0];
#pragma unroll
  for (int q = 1; q < (int)kWays; ++q)
    if (q == w) r = a[q];
  return r;
}

__global__ __launch_bounds__(kBlock) void k_set_walk(const DevState d, Scratch sc, uint32_t t, Counters *cn) {
  if (cn->err) return;
  const uint32_t Tn = cn->n_touched;
  const bool ring_on = d.V > 0;
  const uint32_t recent_lvl = level_of(kClsRecent, ring_on);
  uint32_t c_hit = 0, c_fill = 0, c_evict = 0, c_enq = 0, c_drop = 0;
  for (uint32_t i = blockIdx.x * kBlock + threadIdx.x; i < Tn; i += gridDim.x * kBlock) {
    const uint32_t s = sc.touched[i];
    const uint32_t off = sc.seg_off[i];
    const uint32_t k = d.set_count[s];
    d.set_count[s] = 0;
    u32x4 *rp = reinterpret_cast<u32x4 *>(d.sets + s);
    const u32x4 t0 = rp[0], t1 = rp[1], s0 = rp[2], s1 = rp[3], i0 = rp[4], i1 = rp[5];
    uint32_t tag[kWays] = {t0.x, t0.y, t0.z, t0.w, t1.x, t1.y, t1.z, t1.w};
    uint32_t st[kWays] = {s0.x, s0.y, s0.z, s0.w, s1.x, s1.y, s1.z, s1.w};
    uint32_t ins[kWays] = {i0.x, i0.y, i0.z, i0.w, i1.x, i1.y, i1.z, i1.w};
    uint32_t cls[kWays], lvl[kWays];
    int32_t last[kWays];
#pragma unroll
    for (int w = 0; w < (int)kWays; ++w) { cls[w] = kClsNone; lvl[w] = 0; last[w] = -1; }
    uint32_t known = 0;  // ways whose class for this gather is known
    bool dirty = false;
    for (uint32_t j = 0; j < k; ++j) {
      const uint32_t u = sc.sorted[off + j];
      const uint32_t x = sc.uniq[u];
      int hw = -1;
#pragma unroll
      for (int w = 0; w < (int)kWays; ++w)
        if (tag[w] == x) hw = w;
      if (hw >= 0) {
        sc.kind[u] = kKindHit;
        sc.slot[u] = s * kWays + (uint32_t)hw;
        ++c_hit;
        continue;
      }
      ++c_fill;
      dirty = true;
      int pick = -1;
#pragma unroll
      for (int w = (int)kWays - 1; w >= 0; --w)
        if (tag[w] == kEmpty) pick = w;
      uint32_t z = kEmpty;
      uint8_t f = 0;
      if (pick < 0) {
        // classes of batch-start residents, computed once per gather
#pragma unroll
        for (int w = 0; w < (int)kWays; ++w) {
          if (!((known >> w) & 1u)) {
            const uint32_t c = (ins[w] == t) ? kClsRecent : class_from_bits(d.mask[tag[w]], t, d.L, d.T);
            cls[w] = c;
            lvl[w] = level_of(c, ring_on);
          }
        }
        known = (1u << kWays) - 1u;
        pick = 0;
        uint32_t bl = lvl[0], bs = st[0];
#pragma unroll
        for (int w = 1; w < (int)kWays; ++w) {
          if (lvl[w] < bl || (lvl[w] == bl && st[w] < bs)) {
            pick = w;
            bl = lvl[w];
            bs = st[w];
          }
        }
        z = pick_of(tag, pick);
        const uint32_t pc = pick_of(cls, pick);
        ++c_evict;
        if (ring_on && (pc == kClsFar || pc == kClsNear)) {
          f = kFlagEnqueue;
          ++c_enq;
        } else {
          ++c_drop;
        }
      }
      sc.kind[u] = kKindFill;
      sc.slot[u] = s * kWays + (uint32_t)pick;
      sc.evicted[u] = z;
      sc.flags[u] = f;
      const uint32_t nst = sc.ustat[u];
#pragma unroll
      for (int w = 0; w < (int)kWays; ++w) {
        if (w == pick) {
          tag[w] = x;
          st[w] = nst;
          ins[w] = t;
          cls[w] = kClsRecent;
          lvl[w] = recent_lvl;
          last[w] = (int32_t)u;
        }
      }
      known |= 1u << pick;
    }
#pragma unroll
    for (int w = 0; w < (int)kWays; ++w)
      if (last[w] >= 0) sc.flags[last[w]] |= kFlagFinal;
    if (dirty) {
      rp[0] = u32x4{tag[0], tag[1], tag[2], tag[3]};
      rp[1] = u32x4{tag[4], tag[5], tag[6], tag[7]};
      rp[2] = u32x4{st[0], st[1], st[2], st[3]};
      rp[3] = u32x4{st[4], st[5], st[6], st[7]};
      rp[4] = u32x4{ins[0], ins[1], ins[2], ins[3]};
      rp[5] = u32x4{ins[4], ins[5], ins[6], ins[7]};
    }
  }
  c_hit = wave_sum(c_hit);
  c_fill = wave_sum(c_fill);
  c_evict = wave_sum(c_evict);
  c_enq = wave_sum(c_enq);
  c_drop = wave_sum(c_drop);
  if (__lane_id() == 0) {
    if (c_hit) atomicAdd(&cn->hits, c_hit);
    if (c_fill) atomicAdd(&cn->fills, c_fill);
    if (c_evict) atomicAdd(&cn->evictions, c_evict);
    if (c_enq) atomicAdd(&cn->enqueued, c_enq);
    if (c_drop) atomicAdd(&cn->dropped, c_drop);
  }
}

void launch_set_walk(const DevState &d, uint64_t n, uint32_t t, Scratch &sc, Counters *cn, hipStream_t s) {
  hipLaunchKernelGGL(k_set_walk, dim3(grid_for(n, kBlock, kMaxGrid)), dim3(kBlock), 0, s, d, sc, t, cn);
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

__global__ __launch_bounds__(kBlock) void k_scan_final(const uint8_t *flags, const uint32_t *part,
                                                       uint32_t *enq_before, const Counters *cn) {
  if (cn->err) return;
  const uint32_t U = cn->n_unique;
  const uint32_t nb = (U + kScanChunk - 1) / kScanChunk;
  for (uint32_t b = blockIdx.x; b < nb; b += gridDim.x) {
    const uint32_t base = b * kScanChunk + threadIdx.x * kScanPerThread;
    uint32_t f[kScanPerThread];
    uint32_t c = 0;
#pragma unroll
    for (int k = 0; k < kScanPerThread; ++k) {
      f[k] = (base + k < U) ? (flags[base + k] & kFlagEnqueue) : 0u;
      c += f[k];
    }
    uint32_t tot;
    uint32_t run = part[b] + block_exclusive_scan(c, tot);
#pragma unroll
    for (int k = 0; k < kScanPerThread; ++k) {
      if (base + k < U) enq_before[base + k] = run;
      run += f[k];
    }
  }
}

// For each enqueue of this batch whose line is requested later in the same
// batch, tell that line where its entry went.
__global__ void k_enq_map(Scratch sc, uint64_t tail0, const Counters *cn) {
  if (cn->err) return;
  const uint32_t U = cn->n_unique;
  for (uint32_t u = blockIdx.x * kBlock + threadIdx.x; u < U; u += gridDim.x * kBlock) {
    if (sc.kind[u] != kKindFill || !(sc.flags[u] & kFlagEnqueue)) continue;
    const uint32_t z = sc.evicted[u];
    uint32_t lo = 0, hi = U;
    while (lo < hi) {
      const uint32_t mid = (lo + hi) >> 1;
      if (sc.uniq[mid] < z) lo = mid + 1; else hi = mid;
    }
    if (lo < U && lo > u && sc.uniq[lo] == z) {
      sc.this_q[lo] = tail0 + sc.enq_before[u] + 1;
      sc.this_enq[lo] = u;
    }
  }
}

__global__ __launch_bounds__(kBlock) void k_resolve(const DevState d, Scratch sc, uint64_t tail0, uint8_t *outcome,
                                                    Counters *cn) {
  if (cn->err) return;
  const uint32_t U = cn->n_unique;
  const uint64_t tail_end = tail0 + cn->enq_total;
  const uint32_t lane = threadIdx.x & 63u;
  uint32_t c_vhit = 0, c_miss = 0;
  for (uint32_t base = blockIdx.x * kBlock + (threadIdx.x - lane); base < U; base += gridDim.x * kBlock) {
    const uint32_t u = base + lane;
    bool to_hbm = false, to_host = false, to_fill = false;
    uint64_t hbm_src = 0, host_src = 0;
    if (u < U) {
      const uint8_t kind = sc.kind[u];
      uint8_t oc = 0;  // LSMGNN_HIT
      if (kind == kKindHit) {
        to_hbm = true;
        hbm_src = sc.slot[u];
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
            // evicted earlier in this batch: its row is still in the cache
            // slot the evicting fill took, which no copy has overwritten yet
            const uint32_t e = sc.this_enq[u];
            to_hbm = true;
            hbm_src = sc.slot[e];
            sc.dead[e] = 1;
          } else {
            to_host = true;
            host_src = kSrcRing | (q % d.V);
            // no entry of this batch reuses the slot: remove the entry now
            if (q + d.V >= tail_end) d.ring_tag[q % d.V] = kEmpty;
          }
        } else {
          ++c_miss;
          oc = 2;  // LSMGNN_MISS
          to_host = true;
          host_src = x;
        }
        to_fill = (sc.flags[u] & kFlagFinal) != 0;
      }
      if (outcome) outcome[u] = oc;
    }
    const uint32_t ih = wave_append(to_hbm, &cn->n_hbm);
    if (to_hbm) { sc.hbm_a[ih] = u; sc.hbm_b[ih] = hbm_src; }
    const uint32_t io = wave_append(to_host, &cn->n_host);
    if (to_host) { sc.host_a[io] = u; sc.host_b[io] = host_src; }
    const uint32_t iff = wave_append(to_fill, &cn->n_fill);
    if (to_fill) { sc.fill_a[iff] = sc.slot[u]; sc.fill_b[iff] = u; }
  }
  c_vhit = wave_sum(c_vhit);
  c_miss = wave_sum(c_miss);
  if (__lane_id() == 0) {
    if (c_vhit) atomicAdd(&cn->victim_hits, c_vhit);
    if (c_miss) atomicAdd(&cn->misses, c_miss);
  }
}

// Ring bookkeeping for this batch's enqueues; queue the row copies of the
// entries that are still in the ring at the end of the batch.
__global__ __launch_bounds__(kBlock) void k_enq_finalize(const DevState d, Scratch sc, uint64_t tail0,
                                                         Counters *cn) {
  if (cn->err) return;
  const uint32_t U = cn->n_unique;
  const uint64_t tail_end = tail0 + cn->enq_total;
  const uint32_t lane = threadIdx.x & 63u;
  for (uint32_t base = blockIdx.x * kBlock + (threadIdx.x - lane); base < U; base += gridDim.x * kBlock) {
    const uint32_t u = base + lane;
    bool copy = false;
    uint64_t ring_slot = 0;
    if (u < U && sc.kind[u] == kKindFill && (sc.flags[u] & kFlagEnqueue)) {
      const uint64_t q = tail0 + sc.enq_before[u];
      const uint32_t z = sc.evicted[u];
      d.vpos[z] = q + 1;
      if (q + d.V >= tail_end) {
        ring_slot = q % d.V;
        if (sc.dead[u]) {
          d.ring_tag[ring_slot] = kEmpty;
        } else {
          d.ring_tag[ring_slot] = z;
          copy = true;
        }
      }
    }
    const uint32_t ie = wave_append(copy, &cn->n_enq_copy);
    if (copy) { sc.enq_a[ie] = sc.slot[u]; sc.enq_b[ie] = ring_slot; }
  }
}

void launch_ring_resolve(const DevState &d, uint64_t n, uint64_t tail0, Scratch &sc, uint8_t *outcome,
                         Counters *cn, hipStream_t s) {
  const unsigned g = grid_for(n, kBlock, kMaxGrid);
  const unsigned gs = grid_for(n, kScanChunk, kMaxGrid);
  if (d.V) {
    hipLaunchKernelGGL(k_scan_partial, dim3(gs), dim3(kBlock), 0, s, sc.flags, sc.scan_part, cn);
    hipLaunchKernelGGL(k_scan_top, dim3(1), dim3(kBlock), 0, s, sc.scan_part, cn);
    hipLaunchKernelGGL(k_scan_final, dim3(gs), dim3(kBlock), 0, s, sc.flags, sc.scan_part, sc.enq_before, cn);
    hipLaunchKernelGGL(k_enq_map, dim3(g), dim3(kBlock), 0, s, sc, tail0, cn);
  }
  hipLaunchKernelGGL(k_resolve, dim3(g), dim3(kBlock), 0, s, d, sc, tail0, outcome, cn);
  if (d.V) hipLaunchKernelGGL(k_enq_finalize, dim3(g), dim3(kBlock), 0, s, d, sc, tail0, cn);
}

// -------------------------------------------------------------- row copies
// Work item w = (entry e, 16-byte vector v) with consecutive lanes on
// consecutive vectors of one row, so each wave moves whole rows with 128-bit
// accesses; every lane keeps kUnroll vectors in flight before storing.
constexpr int kUnroll = 4;

template <CopyMode M, bool kPow2>
__global__ __launch_bounds__(kBlock) void k_copy(const DevState d, const uint32_t *a, const uint64_t *b,
                                                 const uint32_t *count, uint8_t *out, uint32_t nvec,
                                                 uint32_t vshift, const Counters *cn) {
  if (cn->err) return;
  const uint64_t total = (uint64_t)(*count) * nvec;
  const uint64_t stride = (uint64_t)gridDim.x * kBlock;
  const uint64_t R = d.R;
  for (uint64_t w0 = (uint64_t)blockIdx.x * kBlock + threadIdx.x; w0 < total; w0 += stride * kUnroll) {
    u32x4 v[kUnroll];
    uint8_t *dst[kUnroll];
#pragma unroll
    for (int k = 0; k < kUnroll; ++k) {
      const uint64_t w = w0 + k * stride;
      dst[k] = nullptr;
      if (w < total) {
        const uint32_t e = kPow2 ? (uint32_t)(w >> vshift) : (uint32_t)(w / nvec);
        const uint64_t byte = (w - (uint64_t)e * nvec) * 16u;
        const uint8_t *src;
        uint8_t *dp;
        if constexpr (M == CopyMode::kHbmToOut) {
          src = d.rows + b[e] * R;
          dp = out + (uint64_t)a[e] * R;
        } else if constexpr (M == CopyMode::kHostToOut) {
          const uint64_t code = b[e];
          src = (code & kSrcRing) ? d.ring_rows + (code & ~kSrcRing) * R : d.store + code * R;
          dp = out + (uint64_t)a[e] * R;
        } else if constexpr (M == CopyMode::kCacheToRing) {
          src = d.rows + (uint64_t)a[e] * R;
          dp = d.ring_rows + b[e] * R;
        } else {
          src = out + b[e] * R;
          dp = d.rows + (uint64_t)a[e] * R;
        }
        v[k] = *reinterpret_cast<const u32x4 *>(src + byte);
        dst[k] = dp + byte;
      }
    }
#pragma unroll
    for (int k = 0; k < kUnroll; ++k)
      if (dst[k]) *reinterpret_cast<u32x4 *>(dst[k]) = v[k];
  }
}

template <CopyMode M>
static void launch_copy_mode(const DevState &d, uint64_t max_rows, const uint32_t *a, const uint64_t *b,
                             const uint32_t *count, uint8_t *out, const Counters *cn, hipStream_t s) {
  const uint32_t nvec = (uint32_t)(d.R / 16);
  const bool pow2 = (nvec & (nvec - 1)) == 0;
  const uint32_t vshift = pow2 ? (uint32_t)__builtin_ctz(nvec) : 0u;
  const unsigned g = grid_for(max_rows * nvec, (uint64_t)kBlock * kUnroll, 4096);
  if (pow2)
    hipLaunchKernelGGL((k_copy<M, true>), dim3(g), dim3(kBlock), 0, s, d, a, b, count, out, nvec, vshift, cn);
  else
    hipLaunchKernelGGL((k_copy<M, false>), dim3(g), dim3(kBlock), 0, s, d, a, b, count, out, nvec, vshift, cn);
}

void launch_copy(CopyMode mode, const DevState &d, uint64_t max_rows, const uint32_t *a, const uint64_t *b,
                 const uint32_t *count, uint8_t *out, Counters *cn, hipStream_t s) {
  switch (mode) {
    case CopyMode::kHbmToOut: launch_copy_mode<CopyMode::kHbmToOut>(d, max_rows, a, b, count, out, cn, s); break;
    case CopyMode::kHostToOut: launch_copy_mode<CopyMode::kHostToOut>(d, max_rows, a, b, count, out, cn, s); break;
    case CopyMode::kCacheToRing: launch_copy_mode<CopyMode::kCacheToRing>(d, max_rows, a, b, count, out, cn, s); break;
    case CopyMode::kOutToCache: launch_copy_mode<CopyMode::kOutToCache>(d, max_rows, a, b, count, out, cn, s); break;
  }
}

// ------------------------------------------------------------------ window
__global__ void k_window_set(const int64_t *ids, uint32_t n, uint32_t bit, uint32_t *mask, int64_t *slot_ids,
                             const Counters *cn) {
  if (cn->err) return;
  for (uint32_t i = blockIdx.x * kBlock + threadIdx.x; i < n; i += gridDim.x * kBlock) {
    const int64_t x = ids[i];
    slot_ids[i] = x;
    atomicOr(&mask[x], 1u << bit);
  }
}

__global__ void k_window_clear(const int64_t *slot_ids, uint32_t n, uint32_t bit, uint32_t *mask,
                               const Counters *cn) {
  if (cn->err) return;
  for (uint32_t i = blockIdx.x * kBlock + threadIdx.x; i < n; i += gridDim.x * kBlock)
    atomicAnd(&mask[slot_ids[i]], ~(1u << bit));
}

void launch_window_set(const int64_t *ids, uint64_t n, uint32_t bit, uint32_t *mask, int64_t *slot_ids,
                       Counters *cn, hipStream_t s) {
  hipLaunchKernelGGL(k_window_set, dim3(grid_for(n, kBlock, kMaxGrid)), dim3(kBlock), 0, s, ids, (uint32_t)n, bit,
                     mask, slot_ids, cn);
}

void launch_window_clear(const int64_t *slot_ids, uint64_t n, uint32_t bit, uint32_t *mask, Counters *cn,
                         hipStream_t s) {
  hipLaunchKernelGGL(k_window_clear, dim3(grid_for(n, kBlock, kMaxGrid)), dim3(kBlock), 0, s, slot_ids,
                     (uint32_t)n, bit, mask, cn);
}

}  // namespace lsm
