// Neighbour sampling on the GPU: the raw request lists of GraphSAGE
// minibatches (uniform sampling of a fixed number of neighbours per hop,
// Sec. 2.1), produced on the device, as the GPU-side sampler of the system
// overview (Sec. 4) does, so that the cache's gather and announcement take
// them without a host round trip.
//
// One minibatch, from its seed nodes and the fanouts f_0 .. f_{H-1}:
//   frontier_0 = the seeds, sorted, duplicates removed;
//   hop h: each frontier node v, in ascending order, draws k = min(f_h, deg v)
//     distinct positions of its adjacency list with Floyd's algorithm (Bentley
//     and Floyd, CACM 1987) and lists them ascending; the hop's samples are
//     adj[off[v] + position] in that order; frontier_{h+1} = the hop's samples,
//     sorted, duplicates removed;
//   request list = seeds (as given) ++ samples of hop 0 ++ hop 1 ++ ...
// Random draws come from counter-based SplitMix64 streams (Steele, Lea and
// Flood, OOPSLA 2014): output k of the stream keyed by K is mix(K + (k+1) G).
// Minibatch b of a sampler seeded with s uses the key
//   key_b = derive(derive(s, 3), b),  derive(p, l) = output l of the stream
//   keyed by mix(p ^ 0x5851f42d4c957f2d);
// hop h of it derive(key_b, h), node v in that hop derive(key_hop, v), and
// the j-th draw of Floyd's algorithm for v is output j of that node's stream,
// reduced to [0, m) as ((r >> 32) * m) >> 32.
//
// Per hop, on the caller's stream:
//   tiles    per tile of 256 frontier entries: each entry's k, its offset
//            within the tile, and the tile's sum
//   top      one block: exclusive scan of the tile sums, the list length
//   draw     one wave per frontier node: lane j makes Floyd's j-th draw, the
//            k steps are resolved in order with one ballot each, and each
//            lane's rank among the k positions places its sample in the
//            list; the next frontier's byte-map marks are plain byte stores
//   popc / chunk scan / compact: the marked nodes in ascending order become
//            the next frontier, and the map is cleared
// Every count stays on the device; the host learns the list length once, at
// the end.  The byte map holds one byte per node and is all zero between calls.
//
// Typed graphs: the list split by node type (per tile of 256 requests a count
// per type, one block's scan per type, then a ballot rank per type and wave),
// each ID replaced by its index within its type.
#include <hip/hip_runtime.h>

#include <cstdint>
#include <cstring>
#include <mutex>

#include "lsmgnn.h"

namespace lsm_smp {

constexpr int kBlock = 256;
constexpr int kMapBytesPerThread = 64;                        // byte-map bytes per thread
constexpr uint64_t kChunk = (uint64_t)kBlock * kMapBytesPerThread;  // byte-map bytes per block
constexpr uint32_t kTile = kBlock;  // frontier entries per tile (one per thread)
constexpr unsigned kMaxGrid = 4096;
constexpr uint32_t kMaxFanout = 64;  // one wave's lanes
constexpr uint32_t kMaxHops = 8;
constexpr uint64_t kGamma = 0x9e3779b97f4a7c15ull;
constexpr uint64_t kLabelSample = 3;

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__host__ __device__ __forceinline__ uint64_t mix(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ull;
  z = (z ^ (z >> 27)) * 0x94d049bb133111ebull;
  return z ^ (z >> 31);
}
__host__ __device__ __forceinline__ uint64_t stream_at(uint64_t key, uint64_t k) { return mix(key + (k + 1) * kGamma); }
__host__ __device__ __forceinline__ uint64_t derive(uint64_t parent, uint64_t label) {
  return stream_at(mix(parent ^ 0x5851f42d4c957f2dull), label);
}

// Device-side state of one call.
struct Ctl {
  uint32_t err;       // a seed outside [0, N)
  uint32_t frontier;  // current frontier size
  uint64_t len;       // request-list length so far
  uint64_t hop_base;  // list position of the current hop's first sample
};

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

// 64-bit variant for the scan over tile sums
__device__ __forceinline__ uint64_t block_exclusive_scan64(uint64_t v, uint64_t &total) {
  __shared__ uint64_t wsum[kBlock / 64];
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  uint64_t x = v;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const uint64_t y = __shfl_up(x, d);
    if (lane >= d) x += y;
  }
  if (lane == 63) wsum[wid] = x;
  __syncthreads();
  uint64_t base = 0, tot = 0;
#pragma unroll
  for (int w = 0; w < kBlock / 64; ++w) {
    const uint64_t sw = wsum[w];
    base += (w < wid) ? sw : 0ull;
    tot += sw;
  }
  __syncthreads();
  total = tot;
  return base + x - v;
}

__global__ __launch_bounds__(kBlock) void k_validate(const int64_t *off, const uint32_t *adj, uint64_t N, uint64_t E,
                                                     uint32_t *err) {
  const uint64_t stride = (uint64_t)gridDim.x * kBlock;
  bool bad = false;
  for (uint64_t u = (uint64_t)blockIdx.x * kBlock + threadIdx.x; u < N; u += stride) {
    const int64_t deg = off[u + 1] - off[u];
    bad |= deg < 0 || deg > (int64_t)0xffffffffll;
  }
  for (uint64_t e = (uint64_t)blockIdx.x * kBlock + threadIdx.x; e < E; e += stride) bad |= adj[e] >= N;
  if (bad) *err = 1u;
}

__global__ void k_init(Ctl *ctl, uint64_t n_seeds) {
  if (threadIdx.x == 0) *ctl = Ctl{0u, 0u, n_seeds, n_seeds};
}

// The seeds open the list and mark the first frontier.
__global__ __launch_bounds__(kBlock) void k_seeds(const int64_t *seeds, uint64_t n, uint64_t N, int64_t *out,
                                                  uint64_t cap, uint8_t *present, Ctl *ctl) {
  bool bad = false;
  for (uint64_t i = (uint64_t)blockIdx.x * kBlock + threadIdx.x; i < n; i += (uint64_t)gridDim.x * kBlock) {
    const int64_t x = seeds[i];
    if (x < 0 || (uint64_t)x >= N) {
      bad = true;
      continue;
    }
    if (i < cap) out[i] = x;
    present[x] = 1;
  }
  if (__ballot(bad) && __lane_id() == 0) atomicOr(&ctl->err, 1u);
}

__device__ __forceinline__ void load_map(const uint8_t *present, uint32_t (&w)[kMapBytesPerThread / 4]) {
  const u32x4 *p = reinterpret_cast<const u32x4 *>(present + (uint64_t)blockIdx.x * kChunk +
                                                    (uint64_t)threadIdx.x * kMapBytesPerThread);
#pragma unroll
  for (int k = 0; k < kMapBytesPerThread / 16; ++k) {
    const u32x4 a = p[k];
    w[4 * k] = a.x;
    w[4 * k + 1] = a.y;
    w[4 * k + 2] = a.z;
    w[4 * k + 3] = a.w;
  }
}

// marked bytes hold exactly 1, so a word's popcount counts them
__global__ __launch_bounds__(kBlock) void k_popc(const uint8_t *present, uint32_t *chunk_sums) {
  uint32_t w[kMapBytesPerThread / 4];
  load_map(present, w);
  uint32_t c = 0;
#pragma unroll
  for (int k = 0; k < kMapBytesPerThread / 4; ++k) c += __popc(w[k]);
  uint32_t tot;
  (void)block_exclusive_scan(c, tot);
  if (threadIdx.x == 0) chunk_sums[blockIdx.x] = tot;
}

__global__ __launch_bounds__(kBlock) void k_chunk_scan(uint32_t *chunk_sums, uint32_t nchunks, Ctl *ctl) {
  uint32_t carry = 0;
  for (uint32_t base = 0; base < nchunks; base += kBlock) {
    const uint32_t i = base + threadIdx.x;
    const uint32_t v = i < nchunks ? chunk_sums[i] : 0u;
    uint32_t tot;
    const uint32_t ex = block_exclusive_scan(v, tot);
    if (i < nchunks) chunk_sums[i] = carry + ex;
    carry += tot;
  }
  if (threadIdx.x == 0) ctl->frontier = carry;
}

// The marked nodes, ascending, become the frontier; the map is cleared.
__global__ __launch_bounds__(kBlock) void k_compact(uint8_t *present, const uint32_t *chunk_off, uint32_t *frontier) {
  uint32_t w[kMapBytesPerThread / 4];
  load_map(present, w);
  const uint64_t b0 = (uint64_t)blockIdx.x * kChunk + (uint64_t)threadIdx.x * kMapBytesPerThread;
  uint32_t c = 0;
#pragma unroll
  for (int k = 0; k < kMapBytesPerThread / 4; ++k) c += __popc(w[k]);
  uint32_t tot;
  const uint32_t ex = block_exclusive_scan(c, tot);
  if (tot == 0) return;
  uint32_t pos = chunk_off[blockIdx.x] + ex;
#pragma unroll
  for (int k = 0; k < kMapBytesPerThread / 4; ++k) {
    uint32_t word = w[k];
    if (word) reinterpret_cast<uint32_t *>(present + b0)[k] = 0u;
    while (word) {  // marked bytes ascending: bit 8j is set for byte j
      frontier[pos++] = (uint32_t)(b0 + 4 * k + (__builtin_ctz(word) >> 3));
      word &= word - 1u;
    }
  }
}

__device__ __forceinline__ uint32_t draws_of(const int64_t *off, uint32_t v, uint32_t fanout) {
  const uint64_t deg = (uint64_t)(off[v + 1] - off[v]);
  return (uint32_t)(fanout < deg ? fanout : deg);
}

// Per tile of the frontier, the number of samples it draws.
__global__ __launch_bounds__(kBlock) void k_tiles(const uint32_t *frontier, const int64_t *off, uint32_t fanout,
                                                  uint64_t *tile_sum, uint32_t *node_off, const Ctl *ctl) {
  const uint32_t f = ctl->frontier;
  const uint32_t ntiles = (f + kTile - 1) / kTile;
  for (uint32_t b = blockIdx.x; b < ntiles; b += gridDim.x) {
    const uint32_t i = b * kTile + threadIdx.x;
    const uint32_t c = i < f ? draws_of(off, frontier[i], fanout) : 0u;
    uint32_t tot;
    const uint32_t ex = block_exclusive_scan(c, tot);
    if (i < f) node_off[i] = ex;
    if (threadIdx.x == 0) tile_sum[b] = tot;
  }
}

// One block: tile sums -> tile offsets within the hop; the hop's samples take
// list positions [len, len + total).
__global__ __launch_bounds__(kBlock) void k_top(uint64_t *tile_sum, Ctl *ctl) {
  const uint32_t f = ctl->frontier;
  const uint32_t ntiles = (f + kTile - 1) / kTile;
  uint64_t carry = 0;
  for (uint32_t base = 0; base < ntiles; base += kBlock) {
    const uint32_t i = base + threadIdx.x;
    const uint64_t v = i < ntiles ? tile_sum[i] : 0ull;
    uint64_t tot;
    const uint64_t ex = block_exclusive_scan64(v, tot);
    if (i < ntiles) tile_sum[i] = carry + ex;
    carry += tot;
  }
  if (threadIdx.x == 0) {
    ctl->hop_base = ctl->len;
    ctl->len += carry;
  }
}

// (list length, status) of the call: LSMGNN_OK, E_RANGE for a bad seed, or
// E_INVAL for a list longer than the output
__global__ void k_result(const Ctl *ctl, uint64_t cap, uint64_t *res) {
  if (threadIdx.x == 0) {
    res[0] = ctl->len;
    res[1] = ctl->err ? (uint64_t)LSMGNN_E_RANGE : ctl->len > cap ? (uint64_t)LSMGNN_E_INVAL : (uint64_t)LSMGNN_OK;
  }
}

// One wave per frontier node: lane j makes Floyd's j-th draw; the k steps are
// then resolved in order with one ballot each (a draw already taken yields
// the step's own bound instead), and each lane's rank among the k positions
// gives its place in the ascending list.
__global__ __launch_bounds__(kBlock) void k_draw_wave(const uint32_t *frontier, const int64_t *off,
                                                      const uint32_t *adj, uint32_t fanout, uint64_t key_hop,
                                                      const uint64_t *tile_off, const uint32_t *node_off,
                                                      int64_t *out, uint64_t cap, uint8_t *present, int mark,
                                                      const Ctl *ctl) {
  const uint32_t f = ctl->frontier;
  const uint64_t hop_base = ctl->hop_base;
  const int lane = threadIdx.x & 63;
  const uint32_t waves = gridDim.x * (kBlock / 64);
  for (uint32_t i = blockIdx.x * (kBlock / 64) + (threadIdx.x >> 6); i < f; i += waves) {
    const uint32_t v = frontier[i];
    const int64_t o = off[v];
    const uint64_t deg = (uint64_t)(off[v + 1] - o);
    const uint32_t k = (uint32_t)(fanout < deg ? fanout : deg);
    if (k == 0) continue;
    uint32_t pos = (uint32_t)lane, rank = (uint32_t)lane;  // k == deg: every position, in order
    if (k < deg) {
      const uint64_t jj = deg - k + (uint64_t)lane;  // this lane's step bound
      uint32_t r = 0;
      if (lane < (int)k) r = (uint32_t)(((stream_at(derive(key_hop, v), (uint64_t)lane) >> 32) * (jj + 1)) >> 32);
      for (uint32_t q = 0; q < k; ++q) {
        const uint32_t rq = __shfl(r, (int)q);
        const bool taken = __ballot(lane < (int)q && pos == rq) != 0ull;
        if (lane == (int)q) pos = taken ? (uint32_t)jj : r;
      }
      rank = 0;  // the positions are distinct
      for (uint32_t q = 0; q < k; ++q) rank += __shfl(pos, (int)q) < pos ? 1u : 0u;
    }
    if (lane < (int)k) {
      const uint64_t p = hop_base + tile_off[i / kTile] + node_off[i] + rank;
      const uint32_t u = adj[o + pos];
      if (p < cap) out[p] = (int64_t)u;
      if (mark) present[u] = 1;
    }
  }
}

// ------------------------------------------------------------ typed graphs
// A request list of global IDs split by node type, in request order, each ID
// replaced by its index within its type.  Tiles of 256 requests: per-tile
// counts per type, one block's scan of them per type, then each request's
// rank among its tile's requests of the same type (one ballot per type and
// wave).  result[t] = length of type t's list; result[T] = status.
constexpr uint32_t kMaxTypes = 16;

struct TypeOuts {
  int64_t *p[kMaxTypes];
};

__global__ __launch_bounds__(kBlock) void k_type_count(const int64_t *ids, uint64_t n, uint64_t N,
                                                       const uint8_t *node_type, uint32_t T, uint32_t *tile_cnt,
                                                       uint64_t *result) {
  __shared__ uint32_t cnt[kMaxTypes];
  const uint64_t ntiles = (n + kBlock - 1) / kBlock;
  for (uint64_t b = blockIdx.x; b < ntiles; b += gridDim.x) {
    if (threadIdx.x < kMaxTypes) cnt[threadIdx.x] = 0;
    __syncthreads();
    const uint64_t i = b * kBlock + threadIdx.x;
    bool bad = false;
    if (i < n) {
      const int64_t x = ids[i];
      if (x < 0 || (uint64_t)x >= N) {
        bad = true;
      } else {
        const uint32_t t = node_type[x];
        if (t >= T)
          bad = true;
        else
          atomicAdd(&cnt[t], 1u);
      }
    }
    if (__ballot(bad) && __lane_id() == 0) atomicOr((unsigned long long *)&result[T], 1ull);
    __syncthreads();
    if (threadIdx.x < T) tile_cnt[b * T + threadIdx.x] = cnt[threadIdx.x];
    __syncthreads();
  }
}

// One block: per type, the exclusive scan of the tile counts (in place) and
// the type's list length.
__global__ __launch_bounds__(kBlock) void k_type_scan(uint32_t *tile_cnt, uint64_t ntiles, uint32_t T,
                                                      uint64_t *result) {
  for (uint32_t t = 0; t < T; ++t) {
    uint32_t carry = 0;
    for (uint64_t base = 0; base < ntiles; base += kBlock) {
      const uint64_t i = base + threadIdx.x;
      const uint32_t v = i < ntiles ? tile_cnt[i * T + t] : 0u;
      uint32_t tot;
      const uint32_t ex = block_exclusive_scan(v, tot);
      if (i < ntiles) tile_cnt[i * T + t] = carry + ex;
      carry += tot;
    }
    if (threadIdx.x == 0) result[t] = carry;
  }
}

__global__ __launch_bounds__(kBlock) void k_type_scatter(const int64_t *ids, uint64_t n, uint64_t N,
                                                         const uint8_t *node_type, const uint32_t *local, uint32_t T,
                                                         const uint32_t *tile_off, TypeOuts outs, uint64_t cap) {
  __shared__ uint32_t wcnt[kBlock / 64][kMaxTypes];
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  const uint64_t lt = lane ? (~0ull >> (64 - lane)) : 0ull;  // lanes below this one
  const uint64_t ntiles = (n + kBlock - 1) / kBlock;
  for (uint64_t b = blockIdx.x; b < ntiles; b += gridDim.x) {
    const uint64_t i = b * kBlock + threadIdx.x;
    uint32_t t = kMaxTypes, loc = 0;  // kMaxTypes: no request, or an invalid one
    if (i < n) {
      const int64_t x = ids[i];
      if (x >= 0 && (uint64_t)x < N && node_type[x] < T) {
        t = node_type[x];
        loc = local[x];
      }
    }
    uint32_t rank = 0;
    for (uint32_t k = 0; k < T; ++k) {
      const uint64_t m = __ballot(t == k);
      if (t == k) rank = (uint32_t)__popcll(m & lt);
      if (lane == 0) wcnt[wid][k] = (uint32_t)__popcll(m);
    }
    __syncthreads();
    if (t < T) {
      uint64_t off = tile_off[b * T + t] + rank;
      for (int w = 0; w < wid; ++w) off += wcnt[w][t];
      if (off < cap) outs.p[t][off] = (int64_t)loc;
    }
    __syncthreads();
  }
}

__global__ void k_type_init(uint64_t *result, uint32_t T) {
  if (threadIdx.x <= T) result[threadIdx.x] = 0;
}

// status word: an invalid ID or type (set by the count kernel as 1) becomes
// E_RANGE; otherwise E_INVAL when a list is longer than the outputs, else OK
__global__ void k_type_status(uint64_t *result, uint32_t T, uint64_t cap) {
  if (threadIdx.x == 0) {
    bool over = false;
    for (uint32_t t = 0; t < T; ++t) over |= result[t] > cap;
    result[T] = result[T] ? (uint64_t)LSMGNN_E_RANGE : over ? (uint64_t)LSMGNN_E_INVAL : (uint64_t)LSMGNN_OK;
  }
}

static unsigned grid_for(uint64_t work, uint64_t per_block, unsigned cap) {
  uint64_t b = (work + per_block - 1) / per_block;
  if (b < 1) b = 1;
  if (b > cap) b = cap;
  return (unsigned)b;
}

}  // namespace lsm_smp

struct lsmgnn_sampler {
  int device = 0;
  const int64_t *off = nullptr;
  const uint32_t *adj = nullptr;
  uint64_t N = 0, nchunks = 0, max_tiles = 0;
  uint32_t hops = 0;
  uint32_t fanout[lsm_smp::kMaxHops] = {};
  uint64_t seed = 0;
  uint8_t *present = nullptr;  // byte map, nchunks * kChunk bytes, zero between calls
  uint32_t *chunk_sums = nullptr;
  uint32_t *frontier[2] = {nullptr, nullptr};
  uint64_t *tile_sum = nullptr;
  lsm_smp::Ctl *ctl = nullptr;     // device
  uint64_t *res = nullptr;          // device: (list length, status) of the last call queued
  uint64_t *res_host = nullptr;     // pinned: the same, read by the blocking call
};

namespace {

struct DeviceScope {
  int prev = -1;
  bool ok = false;
  explicit DeviceScope(int dev) {
    ok = hipGetDevice(&prev) == hipSuccess && hipSetDevice(dev) == hipSuccess;
    if (!ok) (void)hipGetLastError();
  }
  ~DeviceScope() {
    if (prev >= 0) (void)hipSetDevice(prev);
  }
};

void sampler_free(lsmgnn_sampler *s) {
  for (void *p : {(void *)s->present, (void *)s->chunk_sums, (void *)s->frontier[0], (void *)s->frontier[1],
                  (void *)s->tile_sum, (void *)s->ctl, (void *)s->res})
    if (p) (void)hipFree(p);
  if (s->res_host) (void)hipHostFree(s->res_host);
  (void)hipGetLastError();
  delete s;
}

// Queue one minibatch's sampling on `st`; the last kernel leaves (list
// length, status) in s->res.
bool queue_sample(lsmgnn_sampler *s, const int64_t *seeds, uint64_t n_seeds, uint64_t batch, int64_t *out,
                  uint64_t out_cap, hipStream_t st) {
  using namespace lsm_smp;
  const unsigned gN = grid_for(s->N, kTile, kMaxGrid);  // frontier tiles: at most N entries
  const unsigned gc = (unsigned)s->nchunks;
  const uint64_t key_b = derive(derive(s->seed, kLabelSample), batch);
  hipLaunchKernelGGL(k_init, dim3(1), dim3(64), 0, st, s->ctl, n_seeds);
  if (n_seeds)
    hipLaunchKernelGGL(k_seeds, dim3(grid_for(n_seeds, kBlock, kMaxGrid)), dim3(kBlock), 0, st, seeds, n_seeds, s->N,
                       out, out_cap, s->present, s->ctl);
  hipLaunchKernelGGL(k_popc, dim3(gc), dim3(kBlock), 0, st, s->present, s->chunk_sums);
  hipLaunchKernelGGL(k_chunk_scan, dim3(1), dim3(kBlock), 0, st, s->chunk_sums, (uint32_t)s->nchunks, s->ctl);
  hipLaunchKernelGGL(k_compact, dim3(gc), dim3(kBlock), 0, st, s->present, s->chunk_sums, s->frontier[0]);
  // with a bad seed the frontier is still built (and the map cleared) from the
  // valid ones; the hops run, and the call reports E_RANGE
  for (uint32_t h = 0; h < s->hops; ++h) {
    uint32_t *cur = s->frontier[h & 1], *nxt = s->frontier[(h + 1) & 1];
    const int last = h + 1 == s->hops;
    hipLaunchKernelGGL(k_tiles, dim3(gN), dim3(kBlock), 0, st, cur, s->off, s->fanout[h], s->tile_sum, nxt, s->ctl);
    hipLaunchKernelGGL(k_top, dim3(1), dim3(kBlock), 0, st, s->tile_sum, s->ctl);
    hipLaunchKernelGGL(k_draw_wave, dim3(gN), dim3(kBlock), 0, st, cur, s->off, s->adj, s->fanout[h],
                       derive(key_b, h), s->tile_sum, nxt, out, out_cap, s->present, last ? 0 : 1, s->ctl);
    if (!last) {
      hipLaunchKernelGGL(k_popc, dim3(gc), dim3(kBlock), 0, st, s->present, s->chunk_sums);
      hipLaunchKernelGGL(k_chunk_scan, dim3(1), dim3(kBlock), 0, st, s->chunk_sums, (uint32_t)s->nchunks, s->ctl);
      hipLaunchKernelGGL(k_compact, dim3(gc), dim3(kBlock), 0, st, s->present, s->chunk_sums, nxt);
    }
  }
  hipLaunchKernelGGL(k_result, dim3(1), dim3(64), 0, st, s->ctl, out_cap, s->res);
  return hipGetLastError() == hipSuccess;
}

}  // namespace

extern "C" {

lsmgnn_status lsmgnn_sampler_create(const int64_t *offsets, const uint32_t *adj, uint64_t num_nodes,
                                    const uint32_t *fanout, uint32_t hops, uint64_t seed, int device,
                                    lsmgnn_sampler **out) {
  using namespace lsm_smp;
  if (!out) return LSMGNN_E_INVAL;
  *out = nullptr;
  if (!offsets || !fanout || num_nodes == 0 || num_nodes > 0xffffffffull || hops == 0 || hops > kMaxHops)
    return LSMGNN_E_INVAL;
  for (uint32_t h = 0; h < hops; ++h)
    if (fanout[h] > kMaxFanout) return LSMGNN_E_INVAL;
  DeviceScope ds(device);
  if (!ds.ok) return LSMGNN_E_DEVICE;
  const uint64_t N = num_nodes;
  int64_t ends[2] = {0, 0};
  if (hipMemcpy(&ends[0], offsets, 8, hipMemcpyDeviceToHost) != hipSuccess ||
      hipMemcpy(&ends[1], offsets + N, 8, hipMemcpyDeviceToHost) != hipSuccess) {
    (void)hipGetLastError();
    return LSMGNN_E_DEVICE;
  }
  if (ends[0] != 0 || ends[1] < 0 || ends[1] > (int64_t)1 << 40) return LSMGNN_E_RANGE;
  const uint64_t E = (uint64_t)ends[1];
  if (E > 0 && !adj) return LSMGNN_E_INVAL;
  lsmgnn_sampler *s = new (std::nothrow) lsmgnn_sampler;
  if (!s) return LSMGNN_E_NOMEM;
  s->device = device;
  s->off = offsets;
  s->adj = adj;
  s->N = N;
  s->hops = hops;
  s->seed = seed;
  for (uint32_t h = 0; h < hops; ++h) s->fanout[h] = fanout[h];
  s->nchunks = (N + kChunk - 1) / kChunk;
  s->max_tiles = (N + kTile - 1) / kTile;
  uint32_t *err = nullptr;
  bool ok = hipMalloc(&s->present, s->nchunks * kChunk) == hipSuccess &&
            hipMalloc(&s->chunk_sums, s->nchunks * 4) == hipSuccess &&
            hipMalloc(&s->frontier[0], N * 4) == hipSuccess && hipMalloc(&s->frontier[1], N * 4) == hipSuccess &&
            hipMalloc(&s->tile_sum, s->max_tiles * 8) == hipSuccess &&
            hipMalloc(&s->ctl, sizeof(Ctl)) == hipSuccess && hipMalloc(&s->res, 16) == hipSuccess &&
            hipHostMalloc(&s->res_host, 16, hipHostMallocDefault) == hipSuccess &&
            hipMalloc(&err, 4) == hipSuccess;
  if (!ok) {
    (void)hipGetLastError();
    if (err) (void)hipFree(err);
    sampler_free(s);
    return LSMGNN_E_NOMEM;
  }
  // the byte map starts zero; the graph is checked once so that no later
  // kernel reads outside it
  uint32_t herr = 0;
  ok = hipMemset(s->present, 0, s->nchunks * kChunk) == hipSuccess && hipMemset(err, 0, 4) == hipSuccess;
  if (ok) {
    hipLaunchKernelGGL(k_validate, dim3(grid_for(N > E ? N : E, kBlock, 8192)), dim3(kBlock), 0, 0, offsets, adj, N,
                       E, err);
    ok = hipGetLastError() == hipSuccess && hipMemcpy(&herr, err, 4, hipMemcpyDeviceToHost) == hipSuccess;
  }
  (void)hipFree(err);
  if (!ok) {
    (void)hipGetLastError();
    sampler_free(s);
    return LSMGNN_E_DEVICE;
  }
  if (herr) {
    sampler_free(s);
    return LSMGNN_E_RANGE;
  }
  *out = s;
  return LSMGNN_OK;
}

void lsmgnn_sampler_destroy(lsmgnn_sampler *s) {
  if (!s) return;
  DeviceScope ds(s->device);
  (void)hipDeviceSynchronize();
  sampler_free(s);
}

lsmgnn_status lsmgnn_sample(lsmgnn_sampler *s, const int64_t *seeds, uint64_t n_seeds, uint64_t batch, int64_t *out,
                            uint64_t out_cap, uint64_t *n_out, void *stream) {
  if (!s || !n_out || (n_seeds && !seeds) || (out_cap && !out)) return LSMGNN_E_INVAL;
  DeviceScope ds(s->device);
  if (!ds.ok) return LSMGNN_E_DEVICE;
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (!queue_sample(s, seeds, n_seeds, batch, out, out_cap, st) ||
      hipMemcpyAsync(s->res_host, s->res, 16, hipMemcpyDeviceToHost, st) != hipSuccess ||
      hipStreamSynchronize(st) != hipSuccess) {
    (void)hipGetLastError();
    return LSMGNN_E_DEVICE;
  }
  *n_out = s->res_host[0];
  return static_cast<lsmgnn_status>(s->res_host[1]);
}

lsmgnn_status lsmgnn_sample_async(lsmgnn_sampler *s, const int64_t *seeds, uint64_t n_seeds, uint64_t batch,
                                  int64_t *out, uint64_t out_cap, uint64_t *result_host, void *stream) {
  if (!s || !result_host || (n_seeds && !seeds) || (out_cap && !out)) return LSMGNN_E_INVAL;
  DeviceScope ds(s->device);
  if (!ds.ok) return LSMGNN_E_DEVICE;
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (!queue_sample(s, seeds, n_seeds, batch, out, out_cap, st) ||
      hipMemcpyAsync(result_host, s->res, 16, hipMemcpyDeviceToHost, st) != hipSuccess) {
    (void)hipGetLastError();
    return LSMGNN_E_DEVICE;
  }
  return LSMGNN_OK;
}

uint64_t lsmgnn_split_work_bytes(uint64_t n, uint32_t num_types) {
  return ((n + lsm_smp::kBlock - 1) / lsm_smp::kBlock) * (uint64_t)num_types * 4 + 256;
}

}  // extern "C"

namespace {

// The split's arguments other than the work memory are valid.
bool split_args_ok(const int64_t *ids, uint64_t n, const uint8_t *node_type, const uint32_t *local,
                   uint32_t num_types, int64_t *const *outs, uint64_t out_cap, const uint64_t *result_host) {
  if (!result_host || !outs || !node_type || !local || num_types == 0 || num_types > lsm_smp::kMaxTypes ||
      (n && !ids))
    return false;
  for (uint32_t t = 0; t < num_types; ++t)
    if (out_cap && !outs[t]) return false;
  return true;
}

// Queue the split with `work` (device memory of at least
// lsmgnn_split_work_bytes(n, num_types) bytes) as its work memory.
lsmgnn_status queue_split(const int64_t *ids, uint64_t n, uint64_t num_nodes, const uint8_t *node_type,
                          const uint32_t *local, uint32_t num_types, int64_t *const *outs, uint64_t out_cap,
                          void *work, uint64_t *result_host, hipStream_t st) {
  using namespace lsm_smp;
  TypeOuts to{};
  for (uint32_t t = 0; t < num_types; ++t) to.p[t] = outs[t];
  // work: the device result (num_types lengths + status, 8 B each), then the tile counts
  uint64_t *res = static_cast<uint64_t *>(work);
  uint32_t *tile_cnt = reinterpret_cast<uint32_t *>(static_cast<uint8_t *>(work) + 256);
  const uint64_t ntiles = (n + kBlock - 1) / kBlock;
  const unsigned g = grid_for(ntiles, 1, kMaxGrid);
  hipLaunchKernelGGL(k_type_init, dim3(1), dim3(64), 0, st, res, num_types);
  if (n) {
    hipLaunchKernelGGL(k_type_count, dim3(g), dim3(kBlock), 0, st, ids, n, num_nodes, node_type, num_types, tile_cnt,
                       res);
    hipLaunchKernelGGL(k_type_scan, dim3(1), dim3(kBlock), 0, st, tile_cnt, ntiles, num_types, res);
    hipLaunchKernelGGL(k_type_scatter, dim3(g), dim3(kBlock), 0, st, ids, n, num_nodes, node_type, local, num_types,
                       tile_cnt, to, out_cap);
  }
  hipLaunchKernelGGL(k_type_status, dim3(1), dim3(64), 0, st, res, num_types, out_cap);
  if (hipGetLastError() != hipSuccess ||
      hipMemcpyAsync(result_host, res, (num_types + 1) * 8, hipMemcpyDeviceToHost, st) != hipSuccess) {
    (void)hipGetLastError();
    return LSMGNN_E_DEVICE;
  }
  return LSMGNN_OK;
}

}  // namespace

// Work memory of the allocation-free split: one array per device, held until
// the process ends, shared by every call on that device (calls that overlap
// on one device race; every call rewrites all of it that it reads).  Its
// host-side name is not a device address: kernels and copies get the address
// hipGetSymbolAddress returns, looked up once per device.
constexpr uint64_t kSplitScratchBytes = 256 + (uint64_t)(1u << 24) / lsm_smp::kBlock * lsm_smp::kMaxTypes * 4;
static_assert(kSplitScratchBytes == LSMGNN_SPLIT_SCRATCH_BYTES, "header and library disagree on the scratch size");
static __device__ __align__(256) uint8_t scratch[kSplitScratchBytes];

namespace {

constexpr int kMaxScratchDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[kMaxScratchDevices] = {};

// Device address of `dev`'s scratch array (call with `dev` current), or NULL.
void *scratch_on(int dev) {
  if (dev < 0 || dev >= kMaxScratchDevices) return nullptr;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void *p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) {
      (void)hipGetLastError();
      return nullptr;
    }
    g_scratch_ptr[dev] = p;
  }
  return g_scratch_ptr[dev];
}

}  // namespace

extern "C" {

lsmgnn_status lsmgnn_split_by_type_async(const int64_t *ids, uint64_t n, uint64_t num_nodes, const uint8_t *node_type,
                                         const uint32_t *local, uint32_t num_types, int64_t *const *outs,
                                         uint64_t out_cap, void *work, uint64_t work_bytes, uint64_t *result_host,
                                         void *stream) {
  if (!split_args_ok(ids, n, node_type, local, num_types, outs, out_cap, result_host) || !work ||
      work_bytes < lsmgnn_split_work_bytes(n, num_types))
    return LSMGNN_E_INVAL;
  return queue_split(ids, n, num_nodes, node_type, local, num_types, outs, out_cap, work, result_host,
                     static_cast<hipStream_t>(stream));
}

lsmgnn_status lsmgnn_split_by_type_noalloc_async(const int64_t *ids, uint64_t n, uint64_t num_nodes,
                                                 const uint8_t *node_type, const uint32_t *local, uint32_t num_types,
                                                 int64_t *const *outs, uint64_t out_cap, uint64_t *result_host,
                                                 void *stream) {
  if (!split_args_ok(ids, n, node_type, local, num_types, outs, out_cap, result_host) ||
      lsmgnn_split_work_bytes(n, num_types) > kSplitScratchBytes)
    return LSMGNN_E_INVAL;
  hipStream_t st = static_cast<hipStream_t>(stream);
  int dev = -1, prev = -1;
  if ((st ? hipStreamGetDevice(st, &dev) : hipGetDevice(&dev)) != hipSuccess || hipGetDevice(&prev) != hipSuccess) {
    (void)hipGetLastError();
    return LSMGNN_E_DEVICE;
  }
  // the lookup must run with the stream's device current
  if (dev != prev && hipSetDevice(dev) != hipSuccess) {
    (void)hipGetLastError();
    return LSMGNN_E_DEVICE;
  }
  void *work = scratch_on(dev);
  const lsmgnn_status rc = work ? queue_split(ids, n, num_nodes, node_type, local, num_types, outs, out_cap, work,
                                              result_host, st)
                                : LSMGNN_E_DEVICE;
  if (dev != prev) (void)hipSetDevice(prev);
  return rc;
}

}  // extern "C"
