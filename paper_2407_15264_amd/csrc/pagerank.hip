// Static score on the GPU: the normalized reverse PageRank that the hybrid
// policy's static information is built from (Sec. 4.2; the static policy of
// Sec. 5).
//
// The graph is the sampling adjacency in CSR form: node u lists the neighbours
// it samples, the reverse of the direction features flow in message passing.
// The walk moves from u to a uniformly chosen CSR entry of u with probability
// d (a repeated entry counts each time) and jumps to a uniformly chosen node
// otherwise; a node with no entries always jumps.  K power iterations from the
// uniform vector:
//
//   r'(v) = (1 - d)/N + d * (sum over entries u->v of r(u)/deg(u) + D/N),
//   D = total rank of the nodes without entries,
//
// then score(v) = floor(r(v) / max r * (2^32 - 1)).
//
//   sources   one pass writes each entry's source node (the push needs it)
//   share     r(u)/deg(u) per node; per-block partial sums of D
//   push      one thread per entry adds its source's share to its target with
//             a hardware float64 atomic (the order of the additions varies
//             from run to run: results agree to rounding, not bit for bit)
//   update    r(v) from the pushed sums
//   scores    the maximum rank (a 64-bit integer maximum over the bit patterns
//             of non-negative doubles, exact in any order), then the scores
//
// Every pass is bound by HBM bandwidth or by the atomics' throughput; this is
// a one-time preprocessing step, not part of the per-minibatch gather.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>

#include "lsmgnn.h"

namespace lsm_pr {

constexpr int kBlock = 256;
constexpr unsigned kMaxGrid = 8192;

static unsigned grid_for(uint64_t work, unsigned cap) {
  uint64_t b = (work + kBlock - 1) / kBlock;
  if (b < 1) b = 1;
  if (b > cap) b = cap;
  return (unsigned)b;
}

__device__ __forceinline__ double block_sum(double v) {
  __shared__ double part[kBlock / 64];
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  if (lane == 0) part[wid] = v;
  __syncthreads();
  double t = 0.0;
  if (threadIdx.x == 0)
    for (int w = 0; w < kBlock / 64; ++w) t += part[w];
  return t;  // meaningful in thread 0
}

// offsets non-decreasing from 0, every entry < N; a failure sets *err
__global__ __launch_bounds__(kBlock) void k_validate(const int64_t *off, const uint32_t *adj, uint64_t N, uint64_t E,
                                                     uint32_t *err) {
  const uint64_t stride = (uint64_t)gridDim.x * kBlock;
  bool bad = false;
  for (uint64_t u = (uint64_t)blockIdx.x * kBlock + threadIdx.x; u < N; u += stride)
    bad |= off[u + 1] < off[u];
  for (uint64_t e = (uint64_t)blockIdx.x * kBlock + threadIdx.x; e < E; e += stride) bad |= adj[e] >= N;
  if (bad) *err = 1u;
}

__global__ __launch_bounds__(kBlock) void k_sources(const int64_t *off, uint64_t N, uint32_t *src) {
  const uint64_t stride = (uint64_t)gridDim.x * kBlock;
  for (uint64_t u = (uint64_t)blockIdx.x * kBlock + threadIdx.x; u < N; u += stride)
    for (int64_t e = off[u]; e < off[u + 1]; ++e) src[e] = (uint32_t)u;
}

__global__ __launch_bounds__(kBlock) void k_init(double *r, double *next, uint64_t N) {
  const uint64_t stride = (uint64_t)gridDim.x * kBlock;
  for (uint64_t v = (uint64_t)blockIdx.x * kBlock + threadIdx.x; v < N; v += stride) {
    r[v] = 1.0 / (double)N;
    next[v] = 0.0;
  }
}

__global__ __launch_bounds__(kBlock) void k_share(const int64_t *off, const double *r, double *share, uint64_t N,
                                                  double *dpart) {
  const uint64_t stride = (uint64_t)gridDim.x * kBlock;
  double dang = 0.0;
  for (uint64_t u = (uint64_t)blockIdx.x * kBlock + threadIdx.x; u < N; u += stride) {
    const int64_t deg = off[u + 1] - off[u];
    if (deg == 0) {
      dang += r[u];
      share[u] = 0.0;
    } else {
      share[u] = r[u] / (double)deg;
    }
  }
  const double t = block_sum(dang);
  if (threadIdx.x == 0) dpart[blockIdx.x] = t;
}

__global__ __launch_bounds__(kBlock) void k_push(const uint32_t *src, const uint32_t *adj, const double *share,
                                                 double *next, uint64_t E) {
  const uint64_t stride = (uint64_t)gridDim.x * kBlock;
  for (uint64_t e = (uint64_t)blockIdx.x * kBlock + threadIdx.x; e < E; e += stride) {
    const double s = share[src[e]];
    if (s != 0.0) unsafeAtomicAdd(next + adj[e], s);
  }
}

// r(v) from the pushed sums; clears them for the next iteration
__global__ __launch_bounds__(kBlock) void k_update(double *r, double *next, uint64_t N, double d, const double *dpart,
                                                   unsigned nparts) {
  __shared__ double D;
  if (threadIdx.x == 0) {
    double t = 0.0;
    for (unsigned b = 0; b < nparts; ++b) t += dpart[b];
    D = t;
  }
  __syncthreads();
  const double base = (1.0 - d) / (double)N;
  const double jump = D / (double)N;
  const uint64_t stride = (uint64_t)gridDim.x * kBlock;
  for (uint64_t v = (uint64_t)blockIdx.x * kBlock + threadIdx.x; v < N; v += stride) {
    r[v] = base + d * (next[v] + jump);
    next[v] = 0.0;
  }
}

// maximum rank: non-negative doubles order like their bit patterns
__global__ __launch_bounds__(kBlock) void k_max(const double *r, uint64_t N, unsigned long long *mx) {
  const uint64_t stride = (uint64_t)gridDim.x * kBlock;
  unsigned long long m = 0;
  for (uint64_t v = (uint64_t)blockIdx.x * kBlock + threadIdx.x; v < N; v += stride) {
    const unsigned long long b = (unsigned long long)__double_as_longlong(r[v]);
    m = b > m ? b : m;
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const unsigned long long w = __shfl_xor(m, o);
    m = w > m ? w : m;
  }
  if ((threadIdx.x & 63) == 0) atomicMax(mx, m);
}

__global__ __launch_bounds__(kBlock) void k_scores(const double *r, uint64_t N, const unsigned long long *mx,
                                                   uint32_t *score) {
  const double m = __longlong_as_double((long long)*mx);
  const uint64_t stride = (uint64_t)gridDim.x * kBlock;
  for (uint64_t v = (uint64_t)blockIdx.x * kBlock + threadIdx.x; v < N; v += stride)
    score[v] = (uint32_t)floor(r[v] / m * 4294967295.0);
}

}  // namespace lsm_pr

extern "C" lsmgnn_status lsmgnn_pagerank_scores(const int64_t *offsets, const uint32_t *adj, uint64_t num_nodes,
                                                double damping, uint32_t iterations, uint32_t *scores, double *rank,
                                                int device, void *stream) {
  using namespace lsm_pr;
  if (!offsets || !scores || num_nodes == 0 || num_nodes > 0xffffffffull || !(damping >= 0.0 && damping < 1.0))
    return LSMGNN_E_INVAL;
  int prev = -1;
  if (hipGetDevice(&prev) != hipSuccess || hipSetDevice(device) != hipSuccess) {
    (void)hipGetLastError();
    return LSMGNN_E_DEVICE;
  }
  hipStream_t s = static_cast<hipStream_t>(stream);
  const uint64_t N = num_nodes;
  lsmgnn_status st = LSMGNN_OK;
  int64_t ends[2] = {0, 0};
  uint32_t *src = nullptr, *err = nullptr;
  double *r = rank, *r_own = nullptr, *next = nullptr, *share = nullptr, *dpart = nullptr;
  unsigned long long *mx = nullptr;
  uint32_t herr = 0;
  uint64_t E = 0;
  const unsigned gN = grid_for(N, kMaxGrid);
  // the edge count and the first offset, read once the caller's work is done
  if (hipMemcpyAsync(&ends[0], offsets, 8, hipMemcpyDeviceToHost, s) != hipSuccess ||
      hipMemcpyAsync(&ends[1], offsets + N, 8, hipMemcpyDeviceToHost, s) != hipSuccess ||
      hipStreamSynchronize(s) != hipSuccess) {
    st = LSMGNN_E_DEVICE;
    goto done;
  }
  if (ends[0] != 0 || ends[1] < 0 || ends[1] > (int64_t)1 << 40) {
    st = LSMGNN_E_RANGE;
    goto done;
  }
  E = (uint64_t)ends[1];
  if (E > 0 && !adj) {
    st = LSMGNN_E_INVAL;
    goto done;
  }
  if ((E && hipMalloc(&src, E * 4) != hipSuccess) || hipMalloc(&err, 4) != hipSuccess ||
      (!r && hipMalloc(&r_own, N * 8) != hipSuccess) || hipMalloc(&next, N * 8) != hipSuccess ||
      hipMalloc(&share, N * 8) != hipSuccess || hipMalloc(&dpart, kMaxGrid * 8) != hipSuccess ||
      hipMalloc(&mx, 8) != hipSuccess) {
    (void)hipGetLastError();
    st = LSMGNN_E_NOMEM;
    goto done;
  }
  if (!r) r = r_own;
  if (hipMemsetAsync(err, 0, 4, s) != hipSuccess || hipMemsetAsync(mx, 0, 8, s) != hipSuccess) {
    st = LSMGNN_E_DEVICE;
    goto done;
  }
  hipLaunchKernelGGL(k_validate, dim3(grid_for(N > E ? N : E, kMaxGrid)), dim3(kBlock), 0, s, offsets, adj, N, E, err);
  if (hipMemcpyAsync(&herr, err, 4, hipMemcpyDeviceToHost, s) != hipSuccess || hipStreamSynchronize(s) != hipSuccess) {
    st = LSMGNN_E_DEVICE;
    goto done;
  }
  if (herr) {
    st = LSMGNN_E_RANGE;
    goto done;
  }
  if (E) hipLaunchKernelGGL(k_sources, dim3(gN), dim3(kBlock), 0, s, offsets, N, src);
  hipLaunchKernelGGL(k_init, dim3(gN), dim3(kBlock), 0, s, r, next, N);
  for (uint32_t k = 0; k < iterations; ++k) {
    hipLaunchKernelGGL(k_share, dim3(gN), dim3(kBlock), 0, s, offsets, r, share, N, dpart);
    if (E) hipLaunchKernelGGL(k_push, dim3(grid_for(E, kMaxGrid)), dim3(kBlock), 0, s, src, adj, share, next, E);
    hipLaunchKernelGGL(k_update, dim3(gN), dim3(kBlock), 0, s, r, next, N, damping, dpart, gN);
  }
  hipLaunchKernelGGL(k_max, dim3(gN), dim3(kBlock), 0, s, r, N, mx);
  hipLaunchKernelGGL(k_scores, dim3(gN), dim3(kBlock), 0, s, r, N, mx, scores);
  if (hipGetLastError() != hipSuccess || hipStreamSynchronize(s) != hipSuccess) st = LSMGNN_E_DEVICE;
done:
  (void)hipStreamSynchronize(s);
  for (void *p : {(void *)src, (void *)err, (void *)r_own, (void *)next, (void *)share, (void *)dpart, (void *)mx})
    if (p) (void)hipFree(p);
  (void)hipGetLastError();
  if (prev >= 0) (void)hipSetDevice(prev);
  return st;
}
