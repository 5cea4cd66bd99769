// Host runtime of the feature-gather cache: the C ABI of include/lsmgnn.h.
//
// Owns every allocation (HBM cache and metadata, per-node arrays, scratch,
// pinned victim ring), validates arguments before anything changes, and
// launches the gfx950 pipeline of gather_kernels.hip on the caller's stream.
#include <hip/hip_runtime.h>

#include <cstdint>
#include <cstdio>
#include <cstring>
#include <new>
#include <vector>

#include "internal.h"
#include "lsmgnn.h"

using lsm::Counters;
using lsm::CopyMode;
using lsm::DevState;
using lsm::Scratch;

namespace {

constexpr int kMaxSlots = 32;  // window slots: L + 1 <= 32

struct DeviceGuard {
  int prev = -1;
  bool ok = false;
  explicit DeviceGuard(int dev) {
    ok = hipGetDevice(&prev) == hipSuccess && hipSetDevice(dev) == hipSuccess;
  }
  ~DeviceGuard() {
    if (ok && prev >= 0) (void)hipSetDevice(prev);
  }
};

enum { kEvHbm0, kEvHbm1, kEvEnq0, kEvEnq1, kEvHost0, kEvHost1, kEvFill0, kEvFill1, kEvAll0, kEvAll1, kNumEv };

}  // namespace

struct lsmgnn_cache {
  int device = 0;
  DevState d{};
  Scratch sc{};
  uint64_t max_batch = 0;
  int64_t *win_ids = nullptr;  // (L+1) slots of max_batch IDs
  int64_t win_batch[kMaxSlots];
  uint64_t win_len[kMaxSlots];
  Counters *cn = nullptr;       // device
  Counters *cn_host = nullptr;  // pinned host mirror, written by the last kernel of each call
  Counters *cn_host_dev = nullptr;
  uint64_t t = 0, n_adv = 0, tail = 0;
  lsmgnn_counts last{}, total{};
  bool broken = false;
  std::vector<void *> dev_allocs;
  void *ring_host = nullptr;
  hipStream_t side = nullptr;           // host-fetch stream (default priority)
  hipEvent_t ev_meta = nullptr, ev_host = nullptr;
  int prof = 0;
  hipEvent_t ev[kNumEv] = {};
  lsmgnn_profile acc{};
};

namespace {

void release(lsmgnn_cache *c) {
  for (void *p : c->dev_allocs) (void)hipFree(p);
  c->dev_allocs.clear();
  if (c->ring_host) (void)hipHostFree(c->ring_host);
  if (c->cn_host) (void)hipHostFree(c->cn_host);
  for (auto &e : c->ev)
    if (e) (void)hipEventDestroy(e);
  if (c->ev_meta) (void)hipEventDestroy(c->ev_meta);
  if (c->ev_host) (void)hipEventDestroy(c->ev_host);
  if (c->side) (void)hipStreamDestroy(c->side);
}

template <typename T>
bool dev_alloc(lsmgnn_cache *c, T **p, uint64_t count) {
  void *q = nullptr;
  if (hipMalloc(&q, (count ? count : 1) * sizeof(T)) != hipSuccess) {
    (void)hipGetLastError();
    return false;
  }
  c->dev_allocs.push_back(q);
  *p = static_cast<T *>(q);
  return true;
}

lsmgnn_status fail_device(lsmgnn_cache *c) {
  c->broken = true;
  return LSMGNN_E_DEVICE;
}

}  // namespace

extern "C" {

const char *lsmgnn_strerror(lsmgnn_status s) {
  switch (s) {
    case LSMGNN_OK: return "ok";
    case LSMGNN_E_INVAL: return "invalid argument or configuration";
    case LSMGNN_E_RANGE: return "node ID out of range";
    case LSMGNN_E_WINDOW: return "announcement beyond the lookahead window";
    case LSMGNN_E_NOMEM: return "out of device or pinned host memory";
    case LSMGNN_E_DEVICE: return "HIP runtime error";
    case LSMGNN_E_STATE: return "cache unusable after an earlier device error";
  }
  return "unknown status";
}

uint64_t lsmgnn_set_of(uint64_t x, uint64_t num_sets) { return lsm::set_of_host(x, num_sets); }

lsmgnn_status lsmgnn_host_alloc(uint64_t bytes, void **ptr) {
  if (!ptr || bytes == 0) return LSMGNN_E_INVAL;
  *ptr = nullptr;
  if (hipHostMalloc(ptr, bytes, hipHostMallocMapped | hipHostMallocPortable) != hipSuccess) {
    (void)hipGetLastError();
    *ptr = nullptr;
    return LSMGNN_E_NOMEM;
  }
  return LSMGNN_OK;
}

void lsmgnn_host_free(void *ptr) {
  if (ptr) (void)hipHostFree(ptr);
}

lsmgnn_status lsmgnn_cache_create(const lsmgnn_config *cfg, lsmgnn_cache **out) {
  if (!out) return LSMGNN_E_INVAL;
  *out = nullptr;
  if (!cfg || !cfg->host_store || !cfg->static_score) return LSMGNN_E_INVAL;
  if (reinterpret_cast<uintptr_t>(cfg->host_store) & 15u) return LSMGNN_E_INVAL;
  const uint64_t N = cfg->num_nodes, R = cfg->row_bytes, S = cfg->num_sets, V = cfg->victim_rows;
  if (N == 0 || N > 0xffffffffull || R == 0 || R % 16 != 0 || S == 0 || S > (0xffffffffull / lsm::kWays) ||
      cfg->lookahead > 31 || cfg->max_batch == 0 || cfg->max_batch > (1ull << 31) || cfg->flags != 0 ||
      V > (1ull << 40))
    return LSMGNN_E_INVAL;
  // byte sizes must not overflow 64 bits
  if (R > (1ull << 40) || S * lsm::kWays > (~0ull / R) || (V && V > (~0ull / R))) return LSMGNN_E_INVAL;

  int ndev = 0;
  if (hipGetDeviceCount(&ndev) != hipSuccess || cfg->device < 0 || cfg->device >= ndev) {
    (void)hipGetLastError();
    return LSMGNN_E_INVAL;
  }
  DeviceGuard guard(cfg->device);
  if (!guard.ok) return LSMGNN_E_DEVICE;

  // the backing store must be pinned host memory the device can address
  void *store_dev = nullptr;
  if (hipHostGetDevicePointer(&store_dev, const_cast<void *>(cfg->host_store), 0) != hipSuccess || !store_dev) {
    (void)hipGetLastError();
    return LSMGNN_E_INVAL;
  }

  auto *c = new (std::nothrow) lsmgnn_cache();
  if (!c) return LSMGNN_E_NOMEM;
  c->device = cfg->device;
  c->max_batch = cfg->max_batch;
  for (int i = 0; i < kMaxSlots; ++i) {
    c->win_batch[i] = -1;
    c->win_len[i] = 0;
  }
  DevState &d = c->d;
  d.N = N;
  d.R = R;
  d.S = S;
  d.V = V;
  d.L = cfg->lookahead;
  d.T = cfg->near_threshold ? cfg->near_threshold : (cfg->lookahead / 8 > 1 ? cfg->lookahead / 8 : 1);
  d.store = static_cast<const uint8_t *>(store_dev);
  const uint64_t nwords = (N + 31) / 32;
  d.nchunks = (nwords + lsm::kChunkWords - 1) / lsm::kChunkWords;
  const uint64_t bitmap_words = d.nchunks * lsm::kChunkWords;
  const uint64_t B = cfg->max_batch;
  Scratch &sc = c->sc;

  bool ok = dev_alloc(c, &d.sets, S) && dev_alloc(c, &d.rows, S * lsm::kWays * R) && dev_alloc(c, &d.mask, N) &&
            dev_alloc(c, &d.stat, N) && dev_alloc(c, &d.bitmap, bitmap_words) &&
            dev_alloc(c, &d.word_rank, bitmap_words) && dev_alloc(c, &d.chunk_sums, d.nchunks) &&
            dev_alloc(c, &d.set_count, S) && dev_alloc(c, &d.set_idx, S) && dev_alloc(c, &d.uidx, N) &&
            (V == 0 || (dev_alloc(c, &d.vpos, N) && dev_alloc(c, &d.ring_tag, V))) &&
            dev_alloc(c, &c->win_ids, (uint64_t)(d.L + 1) * B) && dev_alloc(c, &c->cn, 1) &&
            dev_alloc(c, &sc.uniq, B) && dev_alloc(c, &sc.uset, B) && dev_alloc(c, &sc.arrival, B) &&
            dev_alloc(c, &sc.touched, B) && dev_alloc(c, &sc.seg_off, B) && dev_alloc(c, &sc.seg, B) &&
            dev_alloc(c, &sc.seg_u, B) && dev_alloc(c, &sc.seg_x, B) && dev_alloc(c, &sc.seg_st, B) &&
            dev_alloc(c, &sc.kind, B) && dev_alloc(c, &sc.flags, B) && dev_alloc(c, &sc.dead, B) &&
            dev_alloc(c, &sc.slot, B) && dev_alloc(c, &sc.evicted, B) && dev_alloc(c, &sc.enq_before, B) &&
            dev_alloc(c, &sc.scan_part, B / lsm::kScanChunk + 2) && dev_alloc(c, &sc.this_q, B) &&
            dev_alloc(c, &sc.this_enq, B) && dev_alloc(c, &sc.src, B) && dev_alloc(c, &sc.ring_dst, B) &&
            dev_alloc(c, &sc.fill_dst, B) && dev_alloc(c, &sc.stat_part, (uint64_t)lsm::kNumStat * lsm::kMaxGrid);
  if (ok && hipHostMalloc(reinterpret_cast<void **>(&c->cn_host), sizeof(Counters), hipHostMallocMapped) !=
                hipSuccess) {
    (void)hipGetLastError();
    c->cn_host = nullptr;
    ok = false;
  }
  if (ok && hipHostGetDevicePointer(reinterpret_cast<void **>(&c->cn_host_dev), c->cn_host, 0) != hipSuccess) {
    (void)hipGetLastError();
    ok = false;
  }
  if (ok && V) {
    if (hipHostMalloc(&c->ring_host, V * R, hipHostMallocMapped | hipHostMallocPortable) != hipSuccess) {
      (void)hipGetLastError();
      c->ring_host = nullptr;
      ok = false;
    } else {
      void *rd = nullptr;
      if (hipHostGetDevicePointer(&rd, c->ring_host, 0) != hipSuccess) {
        (void)hipGetLastError();
        ok = false;
      }
      d.ring_rows = static_cast<uint8_t *>(rd);
    }
  }
  if (!ok) {
    release(c);
    delete c;
    return LSMGNN_E_NOMEM;
  }
  for (auto &e : c->ev)
    if (hipEventCreate(&e) != hipSuccess) ok = false;
  ok = ok && hipStreamCreateWithFlags(&c->side, hipStreamNonBlocking) == hipSuccess &&
       hipEventCreateWithFlags(&c->ev_meta, hipEventDisableTiming) == hipSuccess &&
       hipEventCreateWithFlags(&c->ev_host, hipEventDisableTiming) == hipSuccess;
  // initial state: all ways empty, nothing announced, ring empty
  ok = ok && hipMemset(d.sets, 0xff, S * sizeof(lsm::SetRec)) == hipSuccess &&
       hipMemset(d.mask, 0, N * 4) == hipSuccess && hipMemset(d.bitmap, 0, bitmap_words * 4) == hipSuccess &&
       hipMemset(d.set_count, 0, S * 4) == hipSuccess && hipMemset(c->cn, 0, sizeof(Counters)) == hipSuccess &&
       hipMemcpy(d.stat, cfg->static_score, N * 4, hipMemcpyHostToDevice) == hipSuccess &&
       (V == 0 || (hipMemset(d.vpos, 0, N * 8) == hipSuccess && hipMemset(d.ring_tag, 0xff, V * 4) == hipSuccess)) &&
       hipDeviceSynchronize() == hipSuccess;
  if (!ok) {
    (void)hipGetLastError();
    release(c);
    delete c;
    return LSMGNN_E_DEVICE;
  }
  *out = c;
  return LSMGNN_OK;
}

void lsmgnn_cache_destroy(lsmgnn_cache *c) {
  if (!c) return;
  {
    DeviceGuard guard(c->device);
    (void)hipDeviceSynchronize();
    release(c);
  }
  delete c;
}

lsmgnn_status lsmgnn_advance(lsmgnn_cache *c, const int64_t *ids, uint64_t n, void *stream) {
  if (!c) return LSMGNN_E_INVAL;
  if (c->broken) return LSMGNN_E_STATE;
  if (n > c->max_batch || (n && !ids) || (reinterpret_cast<uintptr_t>(ids) & 7u)) return LSMGNN_E_INVAL;
  const uint64_t j = c->n_adv;
  if (j > c->t + c->d.L) return LSMGNN_E_WINDOW;
  DeviceGuard guard(c->device);
  if (!guard.ok) return LSMGNN_E_DEVICE;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const bool record = j > c->t && c->d.L > 0 && n > 0;  // lists for j <= t are never consulted
  const int slot = (int)(j % (c->d.L + 1));
  if (n)
    lsm::launch_window_set(ids, n, c->d.N, (uint32_t)(j & 31u), c->d.mask,
                           c->win_ids + (uint64_t)slot * c->max_batch, record, c->cn, s);
  lsm::launch_finish(c->cn, c->cn_host_dev, c->sc.stat_part, lsm::StatGrids{}, s);
  if (hipGetLastError() != hipSuccess || hipStreamSynchronize(s) != hipSuccess) {
    (void)hipGetLastError();
    return fail_device(c);
  }
  if (c->cn_host->err) return LSMGNN_E_RANGE;
  if (record) {
    c->win_batch[slot] = (int64_t)j;
    c->win_len[slot] = n;
  }
  c->n_adv = j + 1;
  return LSMGNN_OK;
}

lsmgnn_status lsmgnn_gather(lsmgnn_cache *c, const int64_t *ids, uint64_t n, void *out, int64_t *unique_ids,
                            int64_t *inverse, uint8_t *outcome, uint64_t *n_unique, void *stream) {
  if (!c) return LSMGNN_E_INVAL;
  if (c->broken) return LSMGNN_E_STATE;
  if (!n_unique || n > c->max_batch || (n && (!ids || !out || !unique_ids))) return LSMGNN_E_INVAL;
  // rows move as 16-byte vectors; ID arrays as 8-byte words
  if ((reinterpret_cast<uintptr_t>(out) & 15u) || (reinterpret_cast<uintptr_t>(ids) & 7u) ||
      (reinterpret_cast<uintptr_t>(unique_ids) & 7u) || (reinterpret_cast<uintptr_t>(inverse) & 7u))
    return LSMGNN_E_INVAL;
  DeviceGuard guard(c->device);
  if (!guard.ok) return LSMGNN_E_DEVICE;
  hipStream_t s = static_cast<hipStream_t>(stream);
  DevState &d = c->d;
  Scratch &sc = c->sc;
  const uint32_t t = (uint32_t)c->t;
  const bool prof = c->prof != 0;
  auto rec = [&](int e) {
    if (prof) (void)hipEventRecord(c->ev[e], s);
  };
  uint8_t *outp = static_cast<uint8_t *>(out);

  // the window list of the minibatch being gathered is cleared by the first
  // kernel (it is never consulted again)
  const int slot = (int)(c->t % (d.L + 1));
  const bool clear = d.L > 0 && c->win_batch[slot] == (int64_t)c->t;
  const int64_t *clear_ids = clear ? c->win_ids + (uint64_t)slot * c->max_batch : nullptr;
  const uint64_t clear_n = clear ? c->win_len[slot] : 0;

  lsm::StatGrids grids{};
  rec(kEvAll0);
  if (n || clear_n) lsm::launch_dedup(d, ids, n, clear_ids, clear_n, (uint32_t)(c->t & 31u), sc, unique_ids, c->cn, s);
  if (n) {
    lsm::launch_group_by_set(d, ids, n, inverse, sc, c->cn, s);
    lsm::launch_set_walk(d, n, t, sc, c->cn, grids, s);
    lsm::launch_ring_resolve(d, n, c->tail, sc, outcome, c->cn, grids, s);
    // Data movement.  Every read of a batch-start row precedes every write to
    // the same place: cache rows are read by the hit copy and the enqueue copy
    // before fills overwrite them.  The host fetch (PCIe ingress) runs on the
    // side stream concurrently with the hit copy and the enqueue copy (PCIe
    // egress); it never reads a ring slot an enqueue of this batch rewrites.
    (void)hipEventRecord(c->ev_meta, s);
    (void)hipStreamWaitEvent(c->side, c->ev_meta, 0);
    if (prof) (void)hipEventRecord(c->ev[kEvHost0], c->side);
    lsm::launch_copy(CopyMode::kHostToOut, d, n, sc, outp, c->cn, c->side);
    if (prof) (void)hipEventRecord(c->ev[kEvHost1], c->side);
    (void)hipEventRecord(c->ev_host, c->side);
    if (d.V) {
      rec(kEvEnq0);
      lsm::launch_copy(CopyMode::kCacheToRing, d, n, sc, outp, c->cn, s);
      rec(kEvEnq1);
    }
    rec(kEvHbm0);
    lsm::launch_copy(CopyMode::kHbmToOut, d, n, sc, outp, c->cn, s);
    rec(kEvHbm1);
    (void)hipStreamWaitEvent(s, c->ev_host, 0);
    rec(kEvFill0);
    lsm::launch_copy(CopyMode::kOutToCache, d, n, sc, outp, c->cn, s);
    rec(kEvFill1);
  }
  lsm::launch_finish(c->cn, c->cn_host_dev, sc.stat_part, grids, s);
  rec(kEvAll1);
  if (hipGetLastError() != hipSuccess || hipStreamSynchronize(s) != hipSuccess) {
    (void)hipGetLastError();
    return fail_device(c);
  }
  const Counters &h = *c->cn_host;
  if (h.err) return LSMGNN_E_RANGE;

  if (prof) {
    float ms = 0;
    auto el = [&](int a, int b) {
      float v = 0;
      return hipEventElapsedTime(&v, c->ev[a], c->ev[b]) == hipSuccess ? (double)v : 0.0;
    };
    c->acc.gather_ms += el(kEvAll0, kEvAll1);
    c->acc.gathers += 1;
    if (n) {
      c->acc.hbm_copy_ms += el(kEvHbm0, kEvHbm1);
      c->acc.hbm_copy_launches += 1;
      c->acc.hbm_copy_rows += h.n_hbm;
      if (d.V) {
        c->acc.enqueue_ms += el(kEvEnq0, kEvEnq1);
        c->acc.enqueue_launches += 1;
        c->acc.enqueue_rows += h.n_enq_copy;
      }
      c->acc.host_fetch_ms += el(kEvHost0, kEvHost1);
      c->acc.host_fetch_launches += 1;
      c->acc.host_fetch_rows += h.n_host;
      c->acc.fill_ms += el(kEvFill0, kEvFill1);
      c->acc.fill_launches += 1;
      c->acc.fill_rows += h.n_fill;
    }
    (void)ms;
  }

  *n_unique = h.n_unique;
  lsmgnn_counts st{};
  st.batch = c->t;
  st.requests = n;
  st.unique = h.n_unique;
  st.hits = h.hits;
  st.victim_hits = h.victim_hits;
  st.misses = h.misses;
  st.evictions = h.evictions;
  st.enqueued = h.enqueued;
  st.dropped = h.dropped;
  c->last = st;
  c->total.batch = c->t + 1;
  c->total.requests += st.requests;
  c->total.unique += st.unique;
  c->total.hits += st.hits;
  c->total.victim_hits += st.victim_hits;
  c->total.misses += st.misses;
  c->total.evictions += st.evictions;
  c->total.enqueued += st.enqueued;
  c->total.dropped += st.dropped;
  c->tail += h.enq_total;
  if (clear) c->win_batch[slot] = -1;
  c->t += 1;
  return LSMGNN_OK;
}

lsmgnn_status lsmgnn_stats(const lsmgnn_cache *c, lsmgnn_counts *last, lsmgnn_counts *total) {
  if (!c) return LSMGNN_E_INVAL;
  if (last) *last = c->last;
  if (total) *total = c->total;
  return LSMGNN_OK;
}

lsmgnn_status lsmgnn_export_state(const lsmgnn_cache *c, uint32_t *tags, uint32_t *ring_tags, uint64_t *ring_tail,
                                  uint64_t *t) {
  if (!c) return LSMGNN_E_INVAL;
  if (c->broken) return LSMGNN_E_STATE;
  DeviceGuard guard(c->device);
  if (!guard.ok) return LSMGNN_E_DEVICE;
  if (tags) {
    std::vector<lsm::SetRec> recs;
    try {
      recs.resize(c->d.S);
    } catch (...) {
      return LSMGNN_E_NOMEM;
    }
    if (hipMemcpy(recs.data(), c->d.sets, c->d.S * sizeof(lsm::SetRec), hipMemcpyDeviceToHost) != hipSuccess) {
      (void)hipGetLastError();
      return LSMGNN_E_DEVICE;
    }
    for (uint64_t s = 0; s < c->d.S; ++s) std::memcpy(tags + s * lsm::kWays, recs[s].tag, sizeof(recs[s].tag));
  }
  if (ring_tags && c->d.V) {
    if (hipMemcpy(ring_tags, c->d.ring_tag, c->d.V * 4, hipMemcpyDeviceToHost) != hipSuccess) {
      (void)hipGetLastError();
      return LSMGNN_E_DEVICE;
    }
  }
  if (ring_tail) *ring_tail = c->tail;
  if (t) *t = c->t;
  return LSMGNN_OK;
}

lsmgnn_status lsmgnn_copy_bytes(void *dst, const void *src, uint64_t bytes, void *stream) {
  if (!dst || !src || bytes % 16 != 0 || (reinterpret_cast<uintptr_t>(dst) & 15u) ||
      (reinterpret_cast<uintptr_t>(src) & 15u))
    return LSMGNN_E_INVAL;
  if (bytes == 0) return LSMGNN_OK;
  // pinned host memory is addressed through its device mapping
  auto dev_view = [](const void *p) -> const void * {
    hipPointerAttribute_t a{};
    if (hipPointerGetAttributes(&a, p) != hipSuccess) {
      (void)hipGetLastError();
      return nullptr;
    }
    if (a.type == hipMemoryTypeHost) {
      void *dp = nullptr;
      if (hipHostGetDevicePointer(&dp, const_cast<void *>(p), 0) != hipSuccess) {
        (void)hipGetLastError();
        return nullptr;
      }
      return dp;
    }
    return (a.type == hipMemoryTypeDevice) ? p : nullptr;
  };
  const void *s_dev = dev_view(src);
  void *d_dev = const_cast<void *>(dev_view(dst));
  if (!s_dev || !d_dev) return LSMGNN_E_INVAL;
  hipStream_t s = static_cast<hipStream_t>(stream);
  lsm::launch_copy_plain(s_dev, d_dev, bytes, s);
  if (hipGetLastError() != hipSuccess || hipStreamSynchronize(s) != hipSuccess) {
    (void)hipGetLastError();
    return LSMGNN_E_DEVICE;
  }
  return LSMGNN_OK;
}

lsmgnn_status lsmgnn_set_profiling(lsmgnn_cache *c, int on) {
  if (!c) return LSMGNN_E_INVAL;
  c->prof = on ? 1 : 0;
  if (on) c->acc = lsmgnn_profile{};
  return LSMGNN_OK;
}

lsmgnn_status lsmgnn_get_profile(const lsmgnn_cache *c, lsmgnn_profile *out) {
  if (!c || !out) return LSMGNN_E_INVAL;
  *out = c->acc;
  return LSMGNN_OK;
}

}  // extern "C"
