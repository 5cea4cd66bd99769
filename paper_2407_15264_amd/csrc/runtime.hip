// Host runtime of the feature-gather cache: the C ABI of include/lsmgnn.h.
//
// Owns every allocation (HBM cache and metadata, per-node arrays, scratch,
// pinned victim ring), validates arguments before anything changes, and
// launches the gfx950 kernels of gather_kernels.hip.
//
// Streams.  A gather runs on three internal streams, all at default priority,
// shared by every cache on the device (three in all, so that with the caller's
// stream each gets its own hardware queue under HIP's default of four per
// process; streams that share a queue run in order with each other, and the
// caches of a heterogeneous graph, one per node type, would otherwise
// multiply them).  Each cache orders its own work with its own events; on a
// shared stream the work of different caches only interleaves:
//   meta  - dedup, set grouping, set walk, ring resolution, counters, then
//           staging of the enqueued rows and the hit copy
//   host  - the host fetch (misses and victim hits, PCIe ingress), back to
//           back from gather to gather
//   dma   - the staged rows to the pinned victim ring as a runtime copy
//           (hipMemcpyAsync: a DMA engine, or the runtime's own copy kernel,
//           as the runtime decides; either stalls the kernels beside it far
//           less than a copy kernel of ours writing over the host link), and
//           after each ring write the fills of the next gather
// The host queues all of a gather's kernels at once (every batch-dependent
// size, and the ring tail, stay in device memory) and then waits only for the
// dedup result, to report the unique count or reject the batch; a rejected
// batch's kernels are already queued and do nothing.  A runtime copy needs its
// size on the host, so gather t's ring write is queued once its counters are
// known: by the next call's dedup wait, or by any call that synchronises.
// The metadata of gather t+1 depends only on the metadata of gather t, so it
// runs while gather t's host fetch moves rows.  The data copies of a gather
// read the row-copy lists, the gate and the staging rows that its metadata
// wrote; two copies of them alternate by gather parity, so gather t's metadata
// first waits for gather t-2's fills, and its staging for gather t-2's ring
// write.  Other cross-gather hazards:
//   - cache rows: gather t's staging and hit copy wait for gather t-1's fills;
//     gather t's fills wait for its host fetch, staging and hit copy;
//   - ring rows: gather t reads ring rows only of entries enqueued by gathers
//     up to t-2 (entries of gather t-1 are read by the hit copy from gather
//     t-1's staging rows, which gather t+1's staging overwrites after gather
//     t's hit copy on the in-order meta stream), so its host fetch waits for
//     gather t-2's ring write; gather t's ring write overwrites slots that
//     gathers t-1 and t may read: it is queued on the dma stream behind gather
//     t's fills, which wait for gather t's host fetch (and gather t-1's), and
//     with a pageable store only after the host threads copied gather t's rows.
// Every call first makes the meta stream wait for the work already queued on
// the caller's stream (the IDs and the output buffers).
#include <emmintrin.h>
#include <hip/hip_runtime.h>
#include <xmmintrin.h>

#include <chrono>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <new>
#include <vector>

#include "host_pool.h"
#include "internal.h"
#include "lsmgnn.h"

using lsm::Counters;
using lsm::CopyMode;
using lsm::DedupResult;
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

// The host fetch is two launches: kEvHost0..kEvHostMid brackets the first
// (the misses known at batch start), kEvHostLate..kEvHost1 the second.
enum { kEvHbm0, kEvHbm1, kEvEnq0, kEvEnq1, kEvHost0, kEvHostMid, kEvHostLate, kEvHost1, kEvFill0, kEvFill1, kEvAll0,
       kEvAll1, kEvPf0, kEvPf1, kNumEv };

// One gather in flight; two of these alternate by gather parity.
struct Flight {
  Scratch sc{};                // metadata scratch (shared) + this parity's row-copy lists and gate
  Counters *hc = nullptr;      // pinned: counters published by the gather's last metadata kernel
  Counters *hc_dev = nullptr;
  hipEvent_t meta_done = nullptr, finish_done = nullptr, stage_done = nullptr, hit_done = nullptr, host_done = nullptr,
             data_done = nullptr, dma_done = nullptr;
  hipEvent_t pf_done = nullptr;  // queue mode: this parity's prefetch buffer holds the gather's queue
  bool pf_ready = false;         // pf_done has been recorded for the gather that uses this parity next
  uint32_t *hlist_host = nullptr;  // pageable store: host views of sc.host_list, sc.host_src, sc.bounce
  uint64_t *hsrc_host = nullptr;
  uint8_t *bounce_host = nullptr;
  bool used = false;           // events of this slot have been recorded at least once
  // The gather's data work (staging, hit copy, fills): its size, output and
  // whether it is timed; with `data_deferred` its hit copy and fills are not
  // queued yet (a pipelined gather's are queued by the next call, after that
  // call's metadata, or by any call that waits for the gather).
  uint64_t data_n = 0;
  uint8_t *data_out = nullptr;
  bool data_prof = false;
  bool data_deferred = false;
  hipEvent_t early_done = nullptr;  // the host-fetch list's early part (misses known at batch start) is written
  hipEvent_t list_done = nullptr;   // pageable store: the host-fetch list's rest is written
  uint32_t *hcount_host = nullptr, *hcount_dev = nullptr;  // pageable store: the two parts' lengths (pinned)
  bool stats_pending = false;  // counters not yet added to the totals
  bool dma_pending = false;    // staged rows not yet queued for the ring
  bool dma_used = false;       // dma_done has been recorded at least once
  uint64_t dma_seq = 0, fill_seq = 0;  // positions of the ring write and the fill among the cache's dma submissions
  bool fill_host = false;              // the fills ran on the host-link stream (blocking gather), not the dma one
  uint64_t t = 0, requests = 0;
  uint64_t enq_total = 0, tail_end = 0;  // enqueues of the gather, ring tail after it
  uint32_t q_before[lsm::kMaxQueues] = {}, q_placed[lsm::kMaxQueues] = {};  // queue mode, per slot
};

// Timing events of one gather.  Four sets rotate by gather index: when gather
// t is queued, gather t-4's events are complete (gather t-2's dedup, already
// waited for, ran after gather t-4's rows had moved), so reading them never
// blocks.
constexpr int kPerfSets = 4;
struct PerfSet {
  hipEvent_t e[kNumEv] = {};
  bool pending = false;  // events recorded for gather t and not yet read
  bool counted = false;  // row counts of gather t copied in
  bool ring = false;     // the ring write was timed
  bool pf = false;       // the prefetch this gather issued for the next one was timed
  uint64_t t = 0, requests = 0;
  uint32_t n_hbm = 0, n_host = 0, n_enq = 0, n_fill = 0, n_pf = 0;
};

// The per-device stream triple, created with the first cache on a device and
// destroyed with the last.
constexpr int kMaxDevices = 64;
struct StreamSet {
  hipStream_t meta = nullptr, host = nullptr, dma = nullptr;
  int refs = 0;
};
std::mutex g_streams_mu;
StreamSet g_streams[kMaxDevices];

// Call with the device current.
bool acquire_streams(int dev, StreamSet &out) {
  std::lock_guard<std::mutex> lock(g_streams_mu);
  StreamSet &ss = g_streams[dev];
  if (ss.refs == 0) {
    bool ok = true;
    for (hipStream_t *st : {&ss.meta, &ss.host, &ss.dma})
      ok = ok && hipStreamCreateWithFlags(st, hipStreamNonBlocking) == hipSuccess;
    if (!ok) {
      (void)hipGetLastError();
      for (hipStream_t *st : {&ss.meta, &ss.host, &ss.dma}) {
        if (*st) (void)hipStreamDestroy(*st);
        *st = nullptr;
      }
      return false;
    }
  }
  ++ss.refs;
  out = ss;
  return true;
}

// Caches sharing the device's streams.
int caches_on_device(int dev) {
  std::lock_guard<std::mutex> lock(g_streams_mu);
  return g_streams[dev].refs;
}

void release_streams(int dev) {
  std::lock_guard<std::mutex> lock(g_streams_mu);
  StreamSet &ss = g_streams[dev];
  if (ss.refs <= 0) return;
  if (--ss.refs == 0) {
    for (hipStream_t *st : {&ss.meta, &ss.host, &ss.dma}) {
      if (*st) (void)hipStreamDestroy(*st);
      *st = nullptr;
    }
  }
}

}  // namespace

struct lsmgnn_cache {
  int device = 0;
  DevState d{};
  uint64_t max_batch = 0;
  int64_t *win_ids = nullptr;  // (L+1) slots of max_batch IDs
  int64_t win_batch[kMaxSlots];
  uint64_t win_len[kMaxSlots];
  Counters *cn = nullptr;      // counters of the metadata kernels (meta stream only)
  // a separate announcement's error flag (pinned), set by the window kernel
  uint32_t *adv_err = nullptr, *adv_err_dev = nullptr;
  DedupResult *dd = nullptr, *dd_dev = nullptr;
  Flight fl[2];
  PerfSet ps[kPerfSets];
  hipStream_t meta = nullptr, host = nullptr, dma = nullptr;  // the device's shared streams
  bool has_streams = false;
  uint8_t *ring_host = nullptr;  // pinned victim ring rows, host address
  bool pageable = false;         // the backing store is pageable: host threads copy its rows
  const uint8_t *store_host = nullptr;
  lsm::HostPool *pool = nullptr;
  hipEvent_t ev_in = nullptr, ev_dedup = nullptr, ev_adv = nullptr;
  hipEvent_t ev_q = nullptr;  // queue mode: the queue writes queued so far have landed
  uint64_t t = 0;  // gathers issued
  // Submissions of this cache to the in-order dma stream are numbered; the
  // meta stream has waited for one recorded right after submission
  // meta_dma_seen, so everything the cache submitted there up to it is done.
  // A later wait on anything at or below it would only add a queue packet.
  uint64_t dma_subs = 0, meta_dma_seen = 0;
  uint64_t n_adv = 0, tail = 0;
  lsmgnn_counts last{}, total{};
  bool broken = false;
  std::vector<void *> dev_allocs;
  std::vector<void *> host_allocs;
  int prof = 0;
  lsmgnn_profile acc{};
};

namespace {

void release(lsmgnn_cache *c) {
  delete c->pool;
  c->pool = nullptr;
  for (void *p : c->dev_allocs) (void)hipFree(p);
  c->dev_allocs.clear();
  for (void *p : c->host_allocs) (void)hipHostFree(p);
  c->host_allocs.clear();
  for (Flight &f : c->fl)
    for (hipEvent_t e : {f.meta_done, f.finish_done, f.stage_done, f.hit_done, f.host_done, f.data_done, f.dma_done,
                         f.pf_done, f.early_done, f.list_done})
      if (e) (void)hipEventDestroy(e);
  for (PerfSet &p : c->ps)
    for (hipEvent_t e : p.e)
      if (e) (void)hipEventDestroy(e);
  for (hipEvent_t e : {c->ev_in, c->ev_dedup, c->ev_adv, c->ev_q})
    if (e) (void)hipEventDestroy(e);
  if (c->has_streams) release_streams(c->device);
  c->has_streams = false;
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

// Pinned, device-mapped host memory; *dev receives its device-side address.
template <typename T>
bool host_alloc(lsmgnn_cache *c, T **p, T **dev, uint64_t bytes, bool zero) {
  void *q = nullptr, *qd = nullptr;
  if (hipHostMalloc(&q, bytes, hipHostMallocMapped | hipHostMallocPortable) != hipSuccess) {
    (void)hipGetLastError();
    return false;
  }
  c->host_allocs.push_back(q);
  if (hipHostGetDevicePointer(&qd, q, 0) != hipSuccess) {
    (void)hipGetLastError();
    return false;
  }
  if (zero) std::memset(q, 0, bytes);
  *p = static_cast<T *>(q);
  *dev = static_cast<T *>(qd);
  return true;
}

lsmgnn_status fail_device(lsmgnn_cache *c) {
  (void)hipGetLastError();
  c->broken = true;
  return LSMGNN_E_DEVICE;
}

// Add a finished gather's counters to the totals (its counter kernel must be
// complete).  Gathers are accounted in issue order.
void harvest_stats(lsmgnn_cache *c, Flight &f) {
  if (!f.stats_pending) return;
  const Counters &h = *f.hc;
  lsmgnn_counts st{};
  st.batch = f.t;
  st.requests = f.requests;
  st.unique = h.n_unique;
  st.hits = h.hits;
  st.victim_hits = h.victim_hits;
  st.misses = h.misses;
  st.evictions = h.evictions;
  st.enqueued = h.enqueued;
  st.dropped = h.dropped;
  st.request_hits = h.req_hits;
  st.request_victim_hits = h.req_victim_hits;
  st.victim_rows_ring = h.vh_ring;
  st.victim_rows_staged = h.vh_staged;
  st.victim_rows_cache = h.vh_same;
  st.victim_rows_prefetched = c->d.qmode ? h.victim_hits : 0;
  c->last = st;
  c->total.batch = f.t + 1;
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
  c->total.victim_rows_ring += st.victim_rows_ring;
  c->total.victim_rows_staged += st.victim_rows_staged;
  c->total.victim_rows_cache += st.victim_rows_cache;
  c->total.victim_rows_prefetched += st.victim_rows_prefetched;
  c->tail += h.enq_total;
  f.enq_total = h.enq_total;
  f.tail_end = c->tail;
  f.dma_pending = c->d.V > 0 && h.enq_total > 0;
  if (c->d.qmode)
    for (int k = 0; k < lsm::kMaxQueues; ++k) {
      f.q_before[k] = h.q_before[k];
      f.q_placed[k] = h.q_placed[k];
    }
  PerfSet &p = c->ps[f.t % kPerfSets];
  if (p.pending && p.t == f.t) {
    p.n_hbm = h.n_hbm;
    p.n_host = h.n_host;
    p.n_enq = h.n_enq_copy;
    p.n_fill = h.n_fill;
    if (c->d.qmode) {  // the prefetch this gather issued moved the next queue's entries
      const uint32_t nx = (uint32_t)((f.t + 1) % (c->d.L + 1));
      p.n_pf = h.q_before[nx] + h.q_placed[nx];
    }
    p.counted = true;
  }
  f.stats_pending = false;
}

// Make the meta stream wait for an event recorded on the dma stream right
// after this cache's submission number `seq` there, unless it already waited
// for a later one.
void meta_wait_dma(lsmgnn_cache *c, hipEvent_t e, uint64_t seq) {
  if (seq <= c->meta_dma_seen) return;
  (void)hipStreamWaitEvent(c->meta, e, 0);
  c->meta_dma_seen = seq;
}

// Order the meta stream after the work queued so far on the caller's stream
// s.  If that work is already complete there is nothing to wait for, and the
// first kernel need not wait for a marker on another queue.
bool after_caller(lsmgnn_cache *c, hipStream_t s) {
  if (hipGetLastError() != hipSuccess) return false;  // an earlier call failed
  const hipError_t q = hipStreamQuery(s);
  if (q == hipSuccess) return true;
  (void)hipGetLastError();  // the query's hipErrorNotReady is no failure
  if (q != hipErrorNotReady) return false;
  return hipEventRecord(c->ev_in, s) == hipSuccess && hipStreamWaitEvent(c->meta, c->ev_in, 0) == hipSuccess;
}

// Make the meta stream wait for gather G's fills.
void meta_wait_fills(lsmgnn_cache *c, const Flight &G) {
  if (G.fill_host)
    (void)hipStreamWaitEvent(c->meta, G.data_done, 0);
  else
    meta_wait_dma(c, G.data_done, G.fill_seq);
}

// Queue a harvested gather's ring write: its E enqueues have the sequence
// numbers [tail_end - E, tail_end), of which the last min(E, V) survive; they
// were staged in that order and land in at most two contiguous ring pieces.
//
// Queue mode: the placements were staged slot by slot; slot k's go to its
// positions [q_before[k], q_before[k] + q_placed[k]).
//
// `after` (optional): an event the write also waits for.  The write that the
// next gather's call queues waits for that gather's metadata up to its
// host-fetch list: the write's host-link traffic then runs beside that
// gather's host fetch (the link's other direction) instead of slowing the
// metadata kernels, whose memory requests queue behind it.
void issue_dma(lsmgnn_cache *c, Flight &f, hipEvent_t after = nullptr) {
  if (!f.dma_pending) return;
  f.dma_pending = false;
  const uint64_t V = c->d.V, R = c->d.R;
  PerfSet &p = c->ps[f.t % kPerfSets];
  const bool prof = p.pending && p.t == f.t;
  (void)hipStreamWaitEvent(c->dma, f.stage_done, 0);
  // the gather's own host fetch may read ring rows this write overwrites
  // (victim hits on older entries in slots its enqueues take); a blocking
  // gather's fills follow its host fetch on the host-link stream
  (void)hipStreamWaitEvent(c->dma, f.fill_host ? f.data_done : f.host_done, 0);
  if (after) (void)hipStreamWaitEvent(c->dma, after, 0);
  if (prof) (void)hipEventRecord(p.e[kEvEnq0], c->dma);
  if (c->d.qmode) {
    uint64_t off = 0;
    for (uint32_t k = 0; k <= c->d.L; ++k) {
      const uint64_t m = f.q_placed[k];
      if (m)
        (void)hipMemcpyAsync(c->ring_host + (k * c->d.C + f.q_before[k]) * R, f.sc.staging + off * R, m * R,
                             hipMemcpyDeviceToHost, c->dma);
      off += m;
    }
  } else {
    const uint64_t rows = f.enq_total < V ? f.enq_total : V;
    const uint64_t p0 = (f.tail_end - rows) % V;
    const uint64_t first = rows < V - p0 ? rows : V - p0;
    (void)hipMemcpyAsync(c->ring_host + p0 * R, f.sc.staging, first * R, hipMemcpyDeviceToHost, c->dma);
    if (rows > first)
      (void)hipMemcpyAsync(c->ring_host, f.sc.staging + first * R, (rows - first) * R, hipMemcpyDeviceToHost,
                           c->dma);
  }
  if (prof) {
    (void)hipEventRecord(p.e[kEvEnq1], c->dma);
    p.ring = true;
  }
  (void)hipEventRecord(f.dma_done, c->dma);
  f.dma_used = true;
  f.dma_seq = ++c->dma_subs;
}

// Pageable store: copy the rows of the gather's host-fetch list entries
// [first, first + n) (misses and victim hits) into its pinned bounce buffer,
// row i for list entry i, on the pool's threads.  The list and the source
// codes were written by the early-miss and resolve kernels into pinned memory.
//
// Each thread reads the source rows a few entries ahead (software prefetch:
// the rows are scattered over the store, and one row at a time per thread
// leaves the memory system mostly idle) and writes the bounce rows with
// non-temporal stores: the GPU reads them over the link, so the CPU caches
// need not hold them, and a streaming store does not first read the line.
// Bounce rows are 16-byte aligned (row_bytes is a multiple of 16).
void copy_host_rows(lsmgnn_cache *c, Flight &f, uint64_t first, uint64_t n, bool prof) {
  const uint64_t R = c->d.R;
  const uint64_t *src = f.hsrc_host + first;
  uint8_t *bounce = f.bounce_host + first * R;
  const uint8_t *store = c->store_host, *ring = c->ring_host;
  const auto t0 = std::chrono::steady_clock::now();
  constexpr uint64_t kAhead = 16;  // rows in flight per thread (measured: 16 > 8 > 4)
  c->pool->run(n, 256, [&](uint64_t i0, uint64_t i1) {
    auto row = [&](uint64_t i) {
      const uint64_t code = src[i];
      return ((code & ~lsm::kSrcIndex) == lsm::kSrcRing ? ring : store) + (code & lsm::kSrcIndex) * R;
    };
    auto prefetch = [&](uint64_t i) {
      const char *p = reinterpret_cast<const char *>(row(i));
      for (uint64_t off = 0; off < R; off += 64) _mm_prefetch(p + off, _MM_HINT_T0);
    };
    for (uint64_t i = i0; i < i1 && i < i0 + kAhead; ++i) prefetch(i);
    for (uint64_t i = i0; i < i1; ++i) {
      if (i + kAhead < i1) prefetch(i + kAhead);
      const __m128i *s = reinterpret_cast<const __m128i *>(row(i));
      __m128i *d = reinterpret_cast<__m128i *>(bounce + i * R);
      for (uint64_t k = 0; k < R / 16; ++k) _mm_stream_si128(d + k, _mm_loadu_si128(s + k));
    }
    _mm_sfence();  // the streaming stores are visible before the chunk counts as done
  });
  if (prof) {
    c->acc.host_copy_ms += std::chrono::duration<double, std::milli>(std::chrono::steady_clock::now() - t0).count();
    c->acc.host_copy_rows += n;
  }
}

// Read a finished gather's kernel timings (its rows must have moved and its
// counters must have been harvested).
void harvest_profile(lsmgnn_cache *c, PerfSet &p) {
  if (!p.pending || !p.counted) return;
  auto el = [&](int a, int b) {
    float v = 0;
    return hipEventElapsedTime(&v, p.e[a], p.e[b]) == hipSuccess ? (double)v : 0.0;
  };
  if (p.ring) (void)hipEventSynchronize(p.e[kEvEnq1]);  // queued three gathers ago: long done
  c->acc.gather_ms += el(kEvAll0, kEvAll1);
  c->acc.gathers += 1;
  if (p.requests) {
    c->acc.hbm_copy_ms += el(kEvHbm0, kEvHbm1);
    c->acc.hbm_copy_launches += 1;
    c->acc.hbm_copy_rows += p.n_hbm;
    if (p.ring) {
      c->acc.enqueue_ms += el(kEvEnq0, kEvEnq1);
      c->acc.enqueue_launches += 1;
      c->acc.enqueue_rows += p.n_enq;
    }
    c->acc.host_fetch_ms += el(kEvHost0, kEvHostMid) + el(kEvHostLate, kEvHost1);  // not the wait between them
    c->acc.host_fetch_launches += 2;
    c->acc.host_fetch_rows += p.n_host;
    c->acc.fill_ms += el(kEvFill0, kEvFill1);
    c->acc.fill_launches += 1;
    c->acc.fill_rows += p.n_fill;
  }
  if (p.pf) {
    (void)hipEventSynchronize(p.e[kEvPf1]);
    c->acc.prefetch_ms += el(kEvPf0, kEvPf1);
    c->acc.prefetch_launches += 1;
    c->acc.prefetch_rows += p.n_pf;
  }
  (void)hipGetLastError();
  p.pending = false;
}

// Staging of gather g (flight G) on the meta stream: its evicted rows that
// survive in the victim buffer, copied to its staging rows, once gather g-1's
// fills (the cache rows) and gather g-2's ring write (the staging rows of
// parity g) have landed.
void queue_stage(lsmgnn_cache *c, uint64_t g) {
  DevState &d = c->d;
  Flight &G = c->fl[g & 1], &P = c->fl[(g + 1) & 1];
  if (P.used) meta_wait_fills(c, P);
  if (G.dma_used) meta_wait_dma(c, G.dma_done, G.dma_seq);
  if (G.data_n && d.V) lsm::launch_copy(CopyMode::kCacheToStage, d, G.data_n, G.sc, G.data_out, c->meta);
  (void)hipEventRecord(G.stage_done, c->meta);
  G.used = true;
}

// Hit copy of gather g on the meta stream, after its staging (in stream order,
// so also after gather g-1's fills).  It also reads gather g-1's staging rows
// (victim hits on its entries), which gather g+1's staging overwrites later
// on the same stream.
void queue_hit(lsmgnn_cache *c, uint64_t g) {
  DevState &d = c->d;
  Flight &G = c->fl[g & 1];
  PerfSet &ps = c->ps[g % kPerfSets];
  const bool queues = d.qmode && d.V && d.L > 0;
  // queue mode: the hit copy also moves the victim hits, from the prefetch
  // buffer that the previous call filled
  if (queues && G.pf_ready) (void)hipStreamWaitEvent(c->meta, G.pf_done, 0);
  if (G.data_prof) (void)hipEventRecord(ps.e[kEvHbm0], c->meta);
  if (G.data_n) lsm::launch_copy(CopyMode::kHbmToOut, d, G.data_n, G.sc, G.data_out, c->meta);
  if (G.data_prof) (void)hipEventRecord(ps.e[kEvHbm1], c->meta);
  (void)hipEventRecord(G.hit_done, c->meta);
}

// Fills of gather g, once its host fetch, staging and hit copy are done.
// Pipelined gathers queue them on the dma stream, behind the ring writes
// queued there so far, so that the next host fetch need not wait for them.
// A blocking gather (`on_host`) queues them on the host-link stream right
// behind its own host fetch: its caller waits for them, and on the dma stream
// they would wait for the previous gather's ring write, which runs beside the
// host fetch and often ends after it.
void queue_fills(lsmgnn_cache *c, uint64_t g, bool on_host) {
  Flight &G = c->fl[g & 1];
  PerfSet &ps = c->ps[g % kPerfSets];
  const hipStream_t st = on_host ? c->host : c->dma;
  if (!on_host) (void)hipStreamWaitEvent(st, G.host_done, 0);
  (void)hipStreamWaitEvent(st, G.hit_done, 0);  // after the staging on the meta stream
  if (G.data_prof) (void)hipEventRecord(ps.e[kEvFill0], st);
  if (G.data_n) lsm::launch_copy(CopyMode::kOutToCache, c->d, G.data_n, G.sc, G.data_out, st);
  if (G.data_prof) {
    (void)hipEventRecord(ps.e[kEvFill1], st);
    (void)hipEventRecord(ps.e[kEvAll1], st);
  }
  (void)hipEventRecord(G.data_done, st);
  G.fill_host = on_host;
  G.fill_seq = on_host ? 0 : ++c->dma_subs;
}

// Queue the latest gather's hit copy and fills if they were deferred.
void flush_deferred(lsmgnn_cache *c) {
  if (c->t == 0) return;
  const uint64_t g = c->t - 1;
  Flight &G = c->fl[g & 1];
  if (!G.data_deferred) return;
  G.data_deferred = false;
  queue_hit(c, g);
  queue_fills(c, g, false);
}

// Wait for every queued kernel and copy, then account everything in issue
// order.
lsmgnn_status sync_all(lsmgnn_cache *c) {
  flush_deferred(c);
  if (hipStreamSynchronize(c->meta) != hipSuccess) return fail_device(c);
  Flight &older = c->fl[c->t & 1], &newer = c->fl[(c->t + 1) & 1];
  harvest_stats(c, older);
  issue_dma(c, older);
  harvest_stats(c, newer);
  issue_dma(c, newer);
  if (hipGetLastError() != hipSuccess) return fail_device(c);
  for (hipStream_t s : {c->host, c->dma})
    if (hipStreamSynchronize(s) != hipSuccess) return fail_device(c);
  for (uint64_t k = kPerfSets; k > 0; --k) harvest_profile(c, c->ps[(c->t + k) % kPerfSets]);
  return LSMGNN_OK;
}

// The announcement made together with a gather, if any.
struct Announce {
  bool on = false;
  const int64_t *ids = nullptr;
  uint64_t n = 0;
};

// Queue one gather (and the announcement after it).  Returns once its unique
// count is known; its metadata and row movement may still be running on the
// three streams.  *issued receives the gather index.
//
// With `defer` (pipelined gathers) the gather's hit copy and fills are queued
// by the next call, after that call's metadata: the next gather's metadata
// then need not wait behind this gather's hit copy.  Nothing the next
// metadata does touches what they read or write: it writes the other
// parity's lists and gate, and changes tags, not cache rows.  The staging
// stays in this call, ahead of the next metadata, since this gather's ring
// write waits for it and the host fetch two gathers on waits for that.
lsmgnn_status issue_gather(lsmgnn_cache *c, const int64_t *ids, uint64_t n, const Announce &an, void *out,
                           int64_t *unique_ids, int64_t *inverse, uint8_t *outcome, uint64_t *n_unique,
                           hipStream_t s, uint64_t *issued, bool defer) {
  DevState &d = c->d;
  const uint64_t t = c->t;
  // the announcement is the k-th, made once t+1 gathers are done
  const uint64_t k = c->n_adv;
  if (an.on && k > t + 1 + d.L) return LSMGNN_E_WINDOW;
  const bool record = an.on && k > t + 1 && d.L > 0 && an.n > 0;  // lists for k <= t+1 are never consulted
  const int kslot = (int)(k % (d.L + 1));
  Flight &f = c->fl[t & 1];
  Flight &pf = c->fl[(t + 1) & 1];  // gather t-1
  PerfSet &ps = c->ps[t % kPerfSets];
  harvest_profile(c, ps);  // gather t-4's events are complete
  issue_dma(c, f);         // gather t-2's ring write (normally queued by gather t-1's call)
  const bool prof = c->prof != 0;
  const bool queues = d.qmode && d.V && d.L > 0;  // per-iteration victim queues with prefetch
  // The host fetch's grid: 40 blocks when this cache has the link and the
  // host's memory to itself; 48 when its store is pageable (the GPU then reads
  // contiguous bounce rows); 32 when other caches' host fetches, ring writes
  // and copies share the device.  Measured: one pinned cache gains 8-11 % from
  // 40 blocks over 32; several caches lose 2-5 % with 40; a pageable store on
  // the 100M-node workload gives 487 GB/s with 32 blocks, 494 with 40, 498-500
  // with 48, 502 with 56 and 444 with 64 (more reads in flight stall the hit
  // copy beside them: 0.71 of the HBM peak with 32 blocks, 0.66 with 48).
  d.host_grid = caches_on_device(c->device) > 1 ? 32u : c->pageable ? 48u : 0u;
  auto rec = [&](int e, hipStream_t st) {
    if (prof) (void)hipEventRecord(ps.e[e], st);
  };
  uint8_t *outp = static_cast<uint8_t *>(out);
  const bool blocking = !defer;  // the caller waits for this gather's rows
  if (queues) defer = false;  // the prefetch of the next queue follows this gather's staging

  // inputs are ready once the caller's queued work is; this parity's arrays
  // are free once gather t-2's rows have moved
  if (!after_caller(c, s)) return fail_device(c);
  if (f.used) meta_wait_fills(c, f);

  // the window list of the minibatch being gathered is never consulted again:
  // the first kernel clears its bits
  const int slot = (int)(t % (d.L + 1));
  const bool clear = d.L > 0 && c->win_batch[slot] == (int64_t)t;
  const int64_t *clear_ids = clear ? c->win_ids + (uint64_t)slot * c->max_batch : nullptr;
  const uint64_t clear_n = clear ? c->win_len[slot] : 0;

  // host fetch (PCIe ingress), right after gather t-1's on the same stream,
  // in two parts: the misses known at batch start once they are listed, the
  // rest once the resolve has listed it (and the ring write of gather t-2,
  // whose rows the victim hits may read, has landed).  Each part is queued as
  // soon as the event it waits for is, so that the host's submission of the
  // metadata kernels does not hold it back; with a pageable store each part is
  // queued once the host has copied its rows.
  auto host_fetch_early = [&]() {
    if (n) (void)hipStreamWaitEvent(c->host, f.early_done, 0);
    rec(kEvHost0, c->host);
    if (n) lsm::launch_copy(CopyMode::kHostEarly, d, n, f.sc, outp, c->host);
    rec(kEvHostMid, c->host);
  };
  auto host_fetch_late = [&]() {
    (void)hipStreamWaitEvent(c->host, f.meta_done, 0);
    if (!c->pageable && f.dma_used) (void)hipStreamWaitEvent(c->host, f.dma_done, 0);
    rec(kEvHostLate, c->host);
    if (n) lsm::launch_copy(CopyMode::kHostToOut, d, n, f.sc, outp, c->host);
    rec(kEvHost1, c->host);
    // a blocking gather's fills follow on this stream, and its ring write
    // waits for them instead: one packet fewer between the fetch and the fills
    if (!blocking) (void)hipEventRecord(f.host_done, c->host);
  };

  rec(kEvAll0, c->meta);
  const uint64_t ann_n = an.on ? an.n : 0;
  const bool dedup = n || clear_n || ann_n;
  if (dedup)
    lsm::launch_dedup(d, ids, n, ann_n ? an.ids : nullptr, ann_n, clear_ids, clear_n, (uint32_t)(t & 31u), f.sc,
                      unique_ids, c->cn, c->dd_dev, c->meta);
  (void)hipEventRecord(c->ev_dedup, c->meta);
  // the update of the dynamic information (every U-th gather) reads the window
  // bits the dedup updated; the early-miss list neither reads what it writes
  // nor needs it, so it runs after that list
  const bool refresh = d.U > 1 && t % d.U == 0;
  lsm::StatGrids grids{};
  if (n) {
    // the misses known at batch start first: their rows cross the link while
    // the rest of the metadata runs (pageable store: the host threads copy
    // them meanwhile)
    lsm::launch_early(d, n, t, f.sc, c->cn, grids, c->meta);
    if (c->pageable) lsm::launch_publish_count(f.sc.gate, &f.sc.gate->n_early, f.hcount_dev, c->meta);
    (void)hipEventRecord(f.early_done, c->meta);
    if (!c->pageable) host_fetch_early();
    lsm::launch_unique_index(d, n, f.sc, c->cn, c->meta);
    if (refresh) lsm::launch_refresh(d, (uint32_t)t, c->cn, c->meta);
    lsm::launch_group_by_set(d, ids, n, inverse, f.sc, c->cn, c->meta);
    lsm::launch_set_walk(d, n, (uint32_t)t, f.sc, c->cn, grids, c->meta);
    lsm::launch_ring_resolve(d, n, t, f.sc, outcome, c->cn, grids, c->meta);
    if (c->pageable) {
      lsm::launch_publish_count(f.sc.gate, &f.sc.gate->n_host, f.hcount_dev + 1, c->meta);
      (void)hipEventRecord(f.list_done, c->meta);
    }
  } else if (refresh) {
    lsm::launch_refresh(d, (uint32_t)t, c->cn, c->meta);
  }
  // the host fetch needs only the resolve's list; the rest of the metadata
  // runs beside it
  (void)hipEventRecord(f.meta_done, c->meta);
  if (!c->pageable) {
    if (!n) host_fetch_early();  // no rows: only its events
    host_fetch_late();
  }
  if (n) {
    lsm::launch_ring_enqueue(d, ids, n, t, f.sc, c->cn, grids, c->meta);
  }
  lsm::QueueFinish qf;
  if (queues) {
    qf.qcount = d.qcount;
    qf.gate = f.sc.gate;
    qf.cur = (uint32_t)(t % (d.L + 1));
    qf.next = (uint32_t)((t + 1) % (d.L + 1));
  }
  // the announced bits are first read by the next gather's set walk
  lsm::AnnounceArgs ann;
  if (record) {
    ann.ids = an.ids;
    ann.n = (uint32_t)an.n;
    ann.bit = (uint32_t)(k & 31u);
    ann.mask = d.mask;
    ann.slot_ids = c->win_ids + (uint64_t)kslot * c->max_batch;
    ann.gate = f.sc.gate;
  }
  lsm::launch_finish(c->cn, f.hc_dev, f.sc.stat_part, grids, d.tail, qf, ann, c->meta);
  (void)hipEventRecord(f.finish_done, c->meta);

  // gather t-1's deferred hit copy and fills, now behind this gather's
  // metadata
  flush_deferred(c);
  // this gather's data work: its size and output (the lists are in f.sc)
  f.data_n = n;
  f.data_out = outp;
  f.data_prof = prof;
  // staging (and unless deferred the hit copy) once gather t-1's fills have
  // landed; the ring write (PCIe egress) is queued later on the dma stream
  queue_stage(c, t);
  if (!defer) queue_hit(c, t);
  ps.pending = false;
  if (hipGetLastError() != hipSuccess) return fail_device(c);

  // the GPU runs on while the host waits for the dedup result (with a pageable
  // store: for the early part of the host-fetch list); the meta stream is in
  // order, so gather t-1's counters are published by then and its ring write
  // can be queued
  const bool pageable_lists = c->pageable && n;
  if (hipEventSynchronize(pageable_lists ? f.early_done : c->ev_dedup) != hipSuccess) return fail_device(c);
  harvest_stats(c, pf);
  issue_dma(c, pf, n ? f.meta_done : nullptr);
  if (queues) (void)hipEventRecord(c->ev_q, c->dma);  // every queue write up to gather t-1's
  if (c->pageable) {
    const bool rows = n && !(dedup && c->dd->err);
    const uint64_t n_early = rows ? f.hcount_host[0] : 0;
    if (rows) copy_host_rows(c, f, 0, n_early, prof);  // store rows only
    host_fetch_early();
    if (rows) {
      if (hipEventSynchronize(f.list_done) != hipSuccess) return fail_device(c);
      // ring rows are read only for entries of gathers up to t-2, whose ring
      // writes must have landed
      if (f.dma_used && hipEventSynchronize(f.dma_done) != hipSuccess) return fail_device(c);
      copy_host_rows(c, f, n_early, f.hcount_host[1], prof);
    }
    host_fetch_late();
  }

  // fills after the host fetch, the staging and the hit copy
  if (!defer) queue_fills(c, t, blocking);
  if (hipGetLastError() != hipSuccess) return fail_device(c);
  const uint32_t err = dedup ? c->dd->err : 0u;
  const uint32_t U = dedup ? c->dd->n_unique : 0u;
  if (err) return LSMGNN_E_RANGE;  // every queued kernel of the batch is a no-op
  f.data_deferred = defer;

  f.stats_pending = true;
  f.t = t;
  f.requests = n;
  if (prof) {
    ps.pending = true;
    ps.counted = false;
    ps.t = t;
    ps.requests = n;
    ps.ring = false;
    ps.pf = false;
  }
  if (queues) {
    // prefetch of the next gather's queue, on the host-link stream after this
    // gather's host fetch: while the caller consumes this minibatch.  Its rows
    // are in the host queue (written by the queue writes up to gather t-1's)
    // or in this gather's staging rows; its buffer was last read by gather
    // t-1's hit copy, which precedes this gather's staging.
    Flight &nf = c->fl[(t + 1) & 1];
    (void)hipStreamWaitEvent(c->host, f.stage_done, 0);
    (void)hipStreamWaitEvent(c->host, c->ev_q, 0);
    if (prof) (void)hipEventRecord(ps.e[kEvPf0], c->host);
    lsm::launch_prefetch(d, f.sc.gate, f.sc.staging, (uint32_t)((t + 1) % (d.L + 1)), (uint32_t)((t + 1) & 1),
                         c->host);
    if (prof) {
      (void)hipEventRecord(ps.e[kEvPf1], c->host);
      ps.pf = true;
    }
    (void)hipEventRecord(nf.pf_done, c->host);
    nf.pf_ready = true;
    if (hipGetLastError() != hipSuccess) return fail_device(c);
  }
  if (clear) c->win_batch[slot] = -1;
  if (record) {
    c->win_batch[kslot] = (int64_t)k;
    c->win_len[kslot] = an.n;
  }
  if (an.on) c->n_adv = k + 1;
  c->t = t + 1;
  *n_unique = U;
  if (issued) *issued = t;
  return LSMGNN_OK;
}

lsmgnn_status check_gather_args(const lsmgnn_cache *c, const int64_t *ids, uint64_t n, const void *out,
                                const int64_t *unique_ids, const int64_t *inverse, const uint64_t *n_unique) {
  if (!c) return LSMGNN_E_INVAL;
  if (c->broken) return LSMGNN_E_STATE;
  if (!n_unique || n > c->max_batch || (n && (!ids || !out || !unique_ids))) return LSMGNN_E_INVAL;
  // rows move as 16-byte vectors; ID arrays as 8-byte words
  if ((reinterpret_cast<uintptr_t>(out) & 15u) || (reinterpret_cast<uintptr_t>(ids) & 7u) ||
      (reinterpret_cast<uintptr_t>(unique_ids) & 7u) || (reinterpret_cast<uintptr_t>(inverse) & 7u))
    return LSMGNN_E_INVAL;
  return LSMGNN_OK;
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
  const bool pageable = (cfg->flags & LSMGNN_FLAG_PAGEABLE_STORE) != 0;
  const uint64_t N = cfg->num_nodes, R = cfg->row_bytes, S = cfg->num_sets, V = cfg->victim_rows;
  if (N == 0 || N > 0xffffffffull || R == 0 || R % 16 != 0 || S == 0 || S > (0xffffffffull / lsm::kWays) ||
      cfg->lookahead > 31 || cfg->max_batch == 0 || cfg->max_batch > (1ull << 31) ||
      (cfg->flags & ~LSMGNN_FLAG_PAGEABLE_STORE) != 0 || cfg->host_threads > 256 || cfg->policy > LSMGNN_POLICY_ROUND_ROBIN ||
      cfg->victim_mode > LSMGNN_VICTIM_QUEUES || V > (1ull << 40))
    return LSMGNN_E_INVAL;
  // the queues need a row each at least
  const bool qmode = cfg->victim_mode == LSMGNN_VICTIM_QUEUES;
  if (qmode && V && (V < (uint64_t)cfg->lookahead + 1 || V / ((uint64_t)cfg->lookahead + 1) > 0x7fffffffull))
    return LSMGNN_E_INVAL;
  // byte sizes must not overflow 64 bits
  if (R > (1ull << 40) || S * lsm::kWays > (~0ull / R) || (V && V > (~0ull / R))) return LSMGNN_E_INVAL;

  int ndev = 0;
  if (hipGetDeviceCount(&ndev) != hipSuccess || cfg->device < 0 || cfg->device >= ndev ||
      cfg->device >= kMaxDevices) {
    (void)hipGetLastError();
    return LSMGNN_E_INVAL;
  }
  DeviceGuard guard(cfg->device);
  if (!guard.ok) return LSMGNN_E_DEVICE;

  // without the pageable flag the backing store must be pinned host memory
  // the device can address
  void *store_dev = nullptr;
  if (!pageable &&
      (hipHostGetDevicePointer(&store_dev, const_cast<void *>(cfg->host_store), 0) != hipSuccess || !store_dev)) {
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
  d.policy = cfg->policy;
  d.qmode = qmode ? lsm::kVictimQueues : lsm::kVictimFifo;
  d.C = qmode ? V / ((uint64_t)d.L + 1) : 0;
  d.U = cfg->refresh_period ? cfg->refresh_period : 1;
  const bool queues = qmode && V && d.L > 0;  // queues that can hold entries, and their prefetch buffers
  d.store = static_cast<const uint8_t *>(store_dev);  // null for a pageable store
  c->pageable = pageable;
  c->store_host = static_cast<const uint8_t *>(cfg->host_store);
  d.nchunks = (N + lsm::kChunkBytes - 1) / lsm::kChunkBytes;
  const uint64_t map_bytes = d.nchunks * lsm::kChunkBytes;
  const uint64_t B = cfg->max_batch;
  Scratch sc{};

  // rows: the cache lines, then (queue mode) the two prefetch buffers, then
  // (with a victim buffer) the two staging buffers
  d.stage_row0 = S * lsm::kWays + (queues ? 2 * d.C : 0);
  d.stage_rows = V ? (B < V ? B : V) : 0;
  const uint64_t total_rows = d.stage_row0 + 2 * d.stage_rows;
  // the row copies index these rows with 32 bits (all ones: no row)
  if (total_rows >= 0xffffffffull || total_rows > ~0ull / R) {
    delete c;
    return LSMGNN_E_INVAL;
  }
  bool ok = dev_alloc(c, &d.sets, S) && dev_alloc(c, &d.rows, total_rows * R) &&
            dev_alloc(c, &d.mask, N) &&
            dev_alloc(c, &d.stat, N) && dev_alloc(c, &d.present, map_bytes) &&
            dev_alloc(c, &d.chunk_sums, d.nchunks) &&
            dev_alloc(c, &d.set_count, S) && dev_alloc(c, &d.set_idx, S) && dev_alloc(c, &d.uidx, N) &&
            dev_alloc(c, &d.tail, 2) &&
            (V == 0 || (dev_alloc(c, &d.vpos, N) && dev_alloc(c, &d.ring_tag, V))) &&
            (d.U == 1 || dev_alloc(c, &d.lreuse, S * lsm::kWays)) &&
            (!queues || (dev_alloc(c, &d.qcount, (uint64_t)d.L + 1) &&
                         dev_alloc(c, &sc.qpart, (uint64_t)lsm::kMaxQueues * (B / lsm::kBlock + 1)))) &&
            dev_alloc(c, &c->win_ids, (uint64_t)(d.L + 1) * B) && dev_alloc(c, &c->cn, 1) &&
            dev_alloc(c, &sc.uniq, B) && dev_alloc(c, &sc.uset, B) &&
            dev_alloc(c, &sc.arrival, B) && dev_alloc(c, &sc.touched, B) && dev_alloc(c, &sc.seg_off, B) &&
            dev_alloc(c, &sc.seg, B) && dev_alloc(c, &sc.seg_u, B) && dev_alloc(c, &sc.seg_x, B) &&
            dev_alloc(c, &sc.seg_st, B) && dev_alloc(c, &sc.big, B / (lsm::kSmallSet + 1) + 1) && dev_alloc(c, &sc.kind, B) && dev_alloc(c, &sc.flags, B) &&
            dev_alloc(c, &sc.oc, B) &&
            dev_alloc(c, &sc.dead, B) && dev_alloc(c, &sc.early, B) && dev_alloc(c, &sc.evicted, B) && dev_alloc(c, &sc.enq_before, B) &&
            dev_alloc(c, &sc.scan_part, B / lsm::kScanChunk + 2) && dev_alloc(c, &sc.this_q, B) &&
            dev_alloc(c, &sc.this_enq, B) && dev_alloc(c, &sc.slot, B) && dev_alloc(c, &sc.fill_dst, B) &&
            dev_alloc(c, &sc.stat_part, (uint64_t)lsm::kNumStat * lsm::kMaxGrid) &&
            host_alloc(c, &c->dd, &c->dd_dev, sizeof(DedupResult), true) &&
            host_alloc(c, &c->adv_err, &c->adv_err_dev, sizeof(uint32_t), true);
  for (Flight &f : c->fl) {
    f.sc = sc;
    ok = ok && dev_alloc(c, &f.sc.gate, 1) &&
         (pageable || (dev_alloc(c, &f.sc.host_list, B) && dev_alloc(c, &f.sc.host_src, B))) &&
         dev_alloc(c, &f.sc.hbm.src, B) && dev_alloc(c, &f.sc.fill.src, B) &&
         dev_alloc(c, &f.sc.fill.dst, B) && dev_alloc(c, &f.sc.stage.src, B) && dev_alloc(c, &f.sc.stage.dst, B) &&
         host_alloc(c, &f.hc, &f.hc_dev, sizeof(Counters), true);
    if (ok && V) f.sc.staging = d.rows + (d.stage_row0 + (uint64_t)(&f - c->fl) * d.stage_rows) * R;
    if (ok && pageable) {
      // the host reads the host-fetch list and fills the bounce rows
      ok = host_alloc(c, &f.hcount_host, &f.hcount_dev, 2 * sizeof(uint32_t), true) &&
           host_alloc(c, &f.hlist_host, &f.sc.host_list, B * sizeof(uint32_t), false) &&
           host_alloc(c, &f.hsrc_host, &f.sc.host_src, B * sizeof(uint64_t), false) &&
           host_alloc(c, &f.bounce_host, &f.sc.bounce, B * R, false);
    }
  }
  if (ok && V) ok = host_alloc(c, &c->ring_host, &d.ring_rows, V * R, false);
  if (ok && pageable) {
    const unsigned threads = cfg->host_threads ? cfg->host_threads : 8;
    try {
      c->pool = new lsm::HostPool(threads - 1);
    } catch (...) {
      c->pool = nullptr;
    }
    ok = c->pool != nullptr;
  }
  if (!ok) {
    release(c);
    delete c;
    return LSMGNN_E_NOMEM;
  }
  {
    StreamSet ss;
    c->has_streams = acquire_streams(c->device, ss);
    ok = ok && c->has_streams;
    c->meta = ss.meta;
    c->host = ss.host;
    c->dma = ss.dma;
  }
  for (hipEvent_t *e : {&c->ev_in, &c->ev_dedup, &c->ev_adv, &c->ev_q})
    ok = ok && hipEventCreateWithFlags(e, hipEventDisableTiming) == hipSuccess;
  for (Flight &f : c->fl)
    for (hipEvent_t *e : {&f.meta_done, &f.finish_done, &f.stage_done, &f.hit_done, &f.host_done, &f.data_done,
                          &f.dma_done,
                          &f.pf_done, &f.early_done, &f.list_done})
      ok = ok && hipEventCreateWithFlags(e, hipEventDisableTiming) == hipSuccess;
  for (PerfSet &p : c->ps)
    for (hipEvent_t &e : p.e) ok = ok && hipEventCreate(&e) == hipSuccess;
  // initial state: all ways empty, nothing announced, ring empty, counters zero
  ok = ok && hipMemset(d.sets, 0xff, S * sizeof(lsm::SetRec)) == hipSuccess &&
       hipMemset(d.mask, 0, N * 4) == hipSuccess && hipMemset(d.present, 0, map_bytes) == hipSuccess &&
       hipMemset(d.set_count, 0, S * 4) == hipSuccess && hipMemset(d.tail, 0, 16) == hipSuccess &&
       hipMemset(c->cn, 0, sizeof(Counters)) == hipSuccess &&
       hipMemcpy(d.stat, cfg->static_score, N * 4, hipMemcpyHostToDevice) == hipSuccess &&
       (V == 0 || (hipMemset(d.vpos, 0, N * 8) == hipSuccess && hipMemset(d.ring_tag, 0xff, V * 4) == hipSuccess)) &&
       (!queues || hipMemset(d.qcount, 0, ((uint64_t)d.L + 1) * 4) == hipSuccess) &&
       (d.U == 1 || hipMemset(d.lreuse, 0, S * lsm::kWays * 4) == hipSuccess) &&
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
    (void)sync_all(c);  // queues any pending ring write, then waits for everything
    for (hipStream_t s : {c->meta, c->host, c->dma})
      if (s) (void)hipStreamSynchronize(s);
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
  if (!after_caller(c, s)) return fail_device(c);
  const uint32_t bit = (uint32_t)(j & 31u);
  volatile uint32_t *err = c->adv_err;  // the window kernel sets it on an out-of-range ID
  *err = 0u;
  if (n)
    lsm::launch_window_set(ids, n, c->d.N, bit, c->d.mask, c->win_ids + (uint64_t)slot * c->max_batch, record,
                           c->adv_err_dev, c->meta);
  if (hipEventRecord(c->ev_adv, c->meta) != hipSuccess || hipGetLastError() != hipSuccess ||
      hipEventSynchronize(c->ev_adv) != hipSuccess)
    return fail_device(c);
  if (*err) {
    // the valid IDs of a recorded list had their bit set: clear it again
    if (record) {
      lsm::launch_window_rollback(ids, n, c->d.N, bit, c->d.mask, c->meta);
      if (hipGetLastError() != hipSuccess || hipStreamSynchronize(c->meta) != hipSuccess) return fail_device(c);
    }
    return LSMGNN_E_RANGE;
  }
  if (record) {
    c->win_batch[slot] = (int64_t)j;
    c->win_len[slot] = n;
  }
  c->n_adv = j + 1;
  return LSMGNN_OK;
}

lsmgnn_status lsmgnn_gather(lsmgnn_cache *c, const int64_t *ids, uint64_t n, void *out, int64_t *unique_ids,
                            int64_t *inverse, uint8_t *outcome, uint64_t *n_unique, void *stream) {
  lsmgnn_status st = check_gather_args(c, ids, n, out, unique_ids, inverse, n_unique);
  if (st != LSMGNN_OK) return st;
  DeviceGuard guard(c->device);
  if (!guard.ok) return LSMGNN_E_DEVICE;
  hipStream_t s = static_cast<hipStream_t>(stream);
  uint64_t t = 0;
  st = issue_gather(c, ids, n, Announce{}, out, unique_ids, inverse, outcome, n_unique, s, &t, false);
  if (st != LSMGNN_OK) return st;
  Flight &f = c->fl[t & 1];
  // every output is written once the fills are done (they follow the host
  // fetch, the hit copy and, on the meta stream, all the metadata); later work
  // on the caller's stream is ordered after them
  if (hipEventSynchronize(f.data_done) != hipSuccess || hipEventSynchronize(f.finish_done) != hipSuccess ||
      hipStreamWaitEvent(s, f.data_done, 0) != hipSuccess)
    return fail_device(c);
  harvest_stats(c, f);  // its ring write is queued by the next call (after that gather's metadata) or a sync
  return LSMGNN_OK;
}

lsmgnn_status lsmgnn_gather_async(lsmgnn_cache *c, const int64_t *ids, uint64_t n, const int64_t *next_ids,
                                  uint64_t next_n, void *out, int64_t *unique_ids, int64_t *inverse,
                                  uint8_t *outcome, uint64_t *n_unique, uint64_t *ticket, void *stream) {
  lsmgnn_status st = check_gather_args(c, ids, n, out, unique_ids, inverse, n_unique);
  if (st != LSMGNN_OK) return st;
  if (!ticket || (!next_ids && next_n) || next_n > c->max_batch || (reinterpret_cast<uintptr_t>(next_ids) & 7u))
    return LSMGNN_E_INVAL;
  Announce an;
  an.on = next_ids != nullptr;
  an.ids = next_ids;
  an.n = next_n;
  DeviceGuard guard(c->device);
  if (!guard.ok) return LSMGNN_E_DEVICE;
  return issue_gather(c, ids, n, an, out, unique_ids, inverse, outcome, n_unique,
                      static_cast<hipStream_t>(stream), ticket, true);
}

lsmgnn_status lsmgnn_gather_wait(lsmgnn_cache *c, uint64_t ticket, void *stream) {
  if (!c) return LSMGNN_E_INVAL;
  if (c->broken) return LSMGNN_E_STATE;
  if (ticket >= c->t) return LSMGNN_E_INVAL;
  DeviceGuard guard(c->device);
  if (!guard.ok) return LSMGNN_E_DEVICE;
  flush_deferred(c);  // the latest gather's data work may not be queued yet
  // the slot may hold a later gather by now: waiting for that one is conservative
  if (hipStreamWaitEvent(static_cast<hipStream_t>(stream), c->fl[ticket & 1].data_done, 0) != hipSuccess)
    return fail_device(c);
  return LSMGNN_OK;
}

lsmgnn_status lsmgnn_sync(lsmgnn_cache *c) {
  if (!c) return LSMGNN_E_INVAL;
  if (c->broken) return LSMGNN_E_STATE;
  DeviceGuard guard(c->device);
  if (!guard.ok) return LSMGNN_E_DEVICE;
  return sync_all(c);
}

lsmgnn_status lsmgnn_stats(lsmgnn_cache *c, lsmgnn_counts *last, lsmgnn_counts *total) {
  lsmgnn_status st = lsmgnn_sync(c);
  if (st != LSMGNN_OK) return st;
  if (last) *last = c->last;
  if (total) *total = c->total;
  return LSMGNN_OK;
}

lsmgnn_status lsmgnn_export_state(lsmgnn_cache *c, uint32_t *tags, uint32_t *ring_tags, uint64_t *ring_tail,
                                  uint64_t *t) {
  lsmgnn_status st = lsmgnn_sync(c);
  if (st != LSMGNN_OK) return st;
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
    if (c->d.qmode) {
      // queue slot k holds qcount[k] entries from position 0; the rest is empty
      uint32_t cnt[lsm::kMaxQueues] = {};
      if (c->d.qcount &&
          hipMemcpy(cnt, c->d.qcount, ((uint64_t)c->d.L + 1) * 4, hipMemcpyDeviceToHost) != hipSuccess) {
        (void)hipGetLastError();
        return LSMGNN_E_DEVICE;
      }
      const uint64_t C = c->d.C;
      for (uint64_t i = 0; i < c->d.V; ++i) {
        const uint64_t k = i / C, pos = i % C;
        if (k > c->d.L || pos >= cnt[k]) ring_tags[i] = lsm::kEmpty;
      }
    }
  }
  if (ring_tail) *ring_tail = c->tail;
  if (t) *t = c->t;
  return LSMGNN_OK;
}

lsmgnn_status lsmgnn_expand(const void *rows, const int64_t *inverse, uint64_t n, uint64_t row_bytes, void *out,
                            void *stream) {
  if (n == 0) return LSMGNN_OK;
  if (!rows || !inverse || !out || row_bytes == 0 || row_bytes % 16 != 0 || n > (1ull << 40) ||
      (reinterpret_cast<uintptr_t>(rows) & 15u) || (reinterpret_cast<uintptr_t>(out) & 15u) ||
      (reinterpret_cast<uintptr_t>(inverse) & 7u))
    return LSMGNN_E_INVAL;
  lsm::launch_expand(static_cast<const uint8_t *>(rows), inverse, n, row_bytes, static_cast<uint8_t *>(out),
                     static_cast<hipStream_t>(stream));
  if (hipGetLastError() != hipSuccess) return LSMGNN_E_DEVICE;
  return LSMGNN_OK;
}

lsmgnn_status lsmgnn_copy_bytes(void *dst, const void *src, uint64_t bytes, void *stream) {
  if (!dst || !src || bytes % 16 != 0 || (reinterpret_cast<uintptr_t>(dst) & 15u) ||
      (reinterpret_cast<uintptr_t>(src) & 15u))
    return LSMGNN_E_INVAL;
  if (bytes == 0) return LSMGNN_OK;
  // pinned host memory is addressed through its device mapping
  int on_device = 0;
  auto dev_view = [&on_device](const void *p) -> const void * {
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
    on_device += a.type == hipMemoryTypeDevice;
    return (a.type == hipMemoryTypeDevice) ? p : nullptr;
  };
  const void *s_dev = dev_view(src);
  void *d_dev = const_cast<void *>(dev_view(dst));
  if (!s_dev || !d_dev) return LSMGNN_E_INVAL;
  hipStream_t s = static_cast<hipStream_t>(stream);
  lsm::launch_copy_plain(s_dev, d_dev, bytes, on_device == 2, s);
  if (hipGetLastError() != hipSuccess || hipStreamSynchronize(s) != hipSuccess) {
    (void)hipGetLastError();
    return LSMGNN_E_DEVICE;
  }
  return LSMGNN_OK;
}

lsmgnn_status lsmgnn_set_profiling(lsmgnn_cache *c, int on) {
  lsmgnn_status st = lsmgnn_sync(c);
  if (st != LSMGNN_OK) return st;
  c->prof = on ? 1 : 0;
  if (on) c->acc = lsmgnn_profile{};
  return LSMGNN_OK;
}

lsmgnn_status lsmgnn_get_profile(lsmgnn_cache *c, lsmgnn_profile *out) {
  if (!out) return LSMGNN_E_INVAL;
  lsmgnn_status st = lsmgnn_sync(c);
  if (st != LSMGNN_OK) return st;
  *out = c->acc;
  return LSMGNN_OK;
}

}  // extern "C"
