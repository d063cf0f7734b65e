// Weakly-connected components of the thresholded edge graph: the step after
// the edge classifier in the track-finding pipeline (paper section 2.1: the
// GNN edge scores are passed to WCC; section 2.3: the custom backend returns
// one integer label per space point).
//
// Min-label hooking with pointer jumping.  Every node starts as its own
// parent.  A hook round walks all kept edges (score > threshold), finds the
// two roots and lowers the parent of the larger root to the smaller one with
// an integer atomicMin; a compress round points every node at its root.
// Parents only ever decrease (parent[v] <= v), so every root is the smallest
// id of its tree, and once a hook round finds no edge joining two different
// roots the labels are the smallest node id of each component -- a unique
// answer, independent of the order in which the GPU ran the updates.
#include "gnn_internal.h"

namespace gnn {
namespace {

__device__ __forceinline__ int32_t clampi(int32_t v, int32_t n) {
  return v < 0 ? 0 : (v >= n ? n - 1 : v);
}

// Follows parent links to a root.  Links read here may be older than the
// newest atomicMin of another thread: they are still valid unions with
// parent <= node, so the walk ends, and any mismatch is corrected in a later
// round (every round revisits every edge).
__device__ __forceinline__ int32_t load_parent(const int32_t *parent, int32_t v) {
  return __hip_atomic_load(parent + v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Path halving on the way: each visited node is pointed at its grandparent
// with atomicMin, so links only ever decrease (a smaller link written by a
// concurrent hook is never overwritten) and the chains that concurrent
// hooks build in a large component stay short.
__device__ __forceinline__ int32_t find_root(int32_t *parent, int32_t v) {
  int32_t p = load_parent(parent, v);
  while (p != v) {
    const int32_t gp = load_parent(parent, p);
    if (gp == p) return p;
    if (gp < load_parent(parent, v)) atomicMin(&parent[v], gp);
    v = gp;
    p = load_parent(parent, v);
  }
  return v;
}

__global__ void wcc_init(int32_t *__restrict__ parent, int32_t n) {
  const int64_t v = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (v < n) parent[v] = (int32_t)v;
}

// `changed` is raised once per workgroup: one store per joining edge to a
// single word would serialise on its L2 channel (milliseconds in the first
// round, when most kept edges join two trees).  `prev` is the previous
// round's flag (nullptr in the first round): once a round has joined
// nothing the labels are final, and the rounds queued after it return at
// once, so several rounds can be queued between two host checks.
__global__ void wcc_hook(const int32_t *__restrict__ ei, const float *__restrict__ scores,
                         float threshold, int64_t n_edges, int32_t n_nodes, int32_t *parent,
                         const int32_t *prev, int32_t *__restrict__ changed) {
  if (prev && __hip_atomic_load(prev, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == 0) return;
  __shared__ int32_t joined;
  if (threadIdx.x == 0) joined = 0;
  __syncthreads();
  const int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (j < n_edges && (!scores || scores[j] > threshold)) {
    const int32_t ru = find_root(parent, clampi(ei[j], n_nodes));
    const int32_t rv = find_root(parent, clampi(ei[n_edges + j], n_nodes));
    if (ru != rv) {
      const int32_t hi = ru > rv ? ru : rv, lo = ru > rv ? rv : ru;
      // Many edges join the same pair of large trees: the atomic is issued
      // only when it would lower the link, so a root is not a hot spot.
      if (lo < load_parent(parent, hi)) atomicMin(&parent[hi], lo);
      joined = 1;  // every writer stores the same value
    }
  }
  __syncthreads();
  if (threadIdx.x == 0 && joined) *changed = 1;
}

// Skipped after a round that joined nothing (the links are roots already).
__global__ void wcc_compress(int32_t *parent, int32_t n, const int32_t *changed) {
  if (__hip_atomic_load(changed, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == 0) return;
  const int64_t v = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (v < n) parent[v] = find_root(parent, (int32_t)v);
}

inline unsigned blocks_for(int64_t n, int per) { return (unsigned)((n + per - 1) / per); }

}  // namespace

hipError_t wcc_launch_init(int32_t *labels, int32_t n, hipStream_t stream) {
  if (n > 0) wcc_init<<<blocks_for(n, 256), 256, 0, stream>>>(labels, n);
  return hipGetLastError();
}

hipError_t wcc_launch_round(const int32_t *edge_index, const float *scores, float threshold,
                            int64_t n_edges, int32_t n_nodes, int32_t *labels,
                            const int32_t *prev, int32_t *changed, hipStream_t stream) {
  if (n_edges > 0)
    wcc_hook<<<blocks_for(n_edges, 256), 256, 0, stream>>>(edge_index, scores, threshold,
                                                          n_edges, n_nodes, labels, prev,
                                                          changed);
  if (n_nodes > 0)
    wcc_compress<<<blocks_for(n_nodes, 256), 256, 0, stream>>>(labels, n_nodes, changed);
  return hipGetLastError();
}

}  // namespace gnn
