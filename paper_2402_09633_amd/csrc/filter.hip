// Edge filtering before the GNN (paper section 2.1: after the embedding
// step a Filtering MLP scores the candidate edges and applyFiltering keeps
// the edges above a fixed threshold).
//
// filter     one wave per 32 candidate edges: gather the raw features of
//             both endpoints, layer 1 ([x_src; x_dst], 2F -> H) on VALU,
//             LayerNorm/ReLU, layer 2 (H -> H) on the matrix cores,
//             LayerNorm/ReLU, H -> 1 head, sigmoid.  Layer 2 runs on the
//             fp16 matrix cores from split operands (SPLIT, as in split.hip:
//             f16x2 records of s W1 with s a power of two, the LayerNorm/ReLU
//             output as x1 + x2, three products per k-step, every partial
//             product accumulated in fp32; the LayerNorm then takes the bias
//             as s b1 and eps as eps s^2, which is the LayerNorm of W1 x + b1
//             exactly), or on the fp32 matrix cores when the handle found the
//             layer-1 LayerNorm output bound outside the fp16 range.
// compaction  keep = score > threshold, in input order: per-block counts,
//             one exclusive scan of the block counts, then a stable scatter
//             (wave ballots inside a block); the kept edges are written as a
//             contiguous [2][n_kept] edge_index, ready for gnn_infer.
#include "device_common.h"

namespace gnn {
namespace {

constexpr int FWAVES = 4;
constexpr int CTHREADS = 256;
constexpr int CITEMS = 4;
constexpr int CTILE = CTHREADS * CITEMS;

template <int MB, bool SPLIT>
__global__ __launch_bounds__(64 * FWAVES) void filter_mlp(FilterArgs a) {
  constexpr int H = 32 * MB;
  const int lane = threadIdx.x & 63, hh = lane >> 5, n = lane & 31;
  const int blk = xcd_remap(blockIdx.x, gridDim.x);
  const int64_t row0 = ((int64_t)blk * FWAVES + (threadIdx.x >> 6)) * 32;
  if (row0 >= a.n_edges) return;
  const int64_t row = row0 + n;
  const bool valid = row < a.n_edges;
  const int64_t r = valid ? row : a.n_edges - 1;
  const int64_t s = clamp_idx(a.edge_index[r], a.n_nodes);
  const int64_t d = clamp_idx(a.edge_index[a.n_edges + r], a.n_nodes);

  // layer 1 over [x_src; x_dst]; W0t is [2F][H]
  f16v acc[MB];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const f4 bb = *(const f4 *)(a.b0 + mb * 32 + 8 * q + 4 * hh);
#pragma unroll
      for (int t = 0; t < 4; ++t) acc[mb][4 * q + t] = bb[t];
    }
  for (int k = 0; k < 2 * a.F; ++k) {
    const float xk = k < a.F ? a.x[s * a.F + k] : a.x[d * a.F + (k - a.F)];
    const float *wk = a.w0t + k * H + 4 * hh;
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const f4 ww = *(const f4 *)(wk + mb * 32 + 8 * q);
#pragma unroll
        for (int t = 0; t < 4; ++t) acc[mb][4 * q + t] += ww[t] * xk;
      }
  }
  bias_ln_relu<MB>(acc, nullptr, a.g0, a.beta0, a.eps, hh, false);
  f16v acc2[MB];
  if constexpr (SPLIT) {
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc2[mb][v] = 0.f;
    const h8 *rec = (const h8 *)a.w1r + lane;
#pragma unroll
    for (int g = 0; g < 2 * MB; ++g) step_h<MB>(acc2, rec + g * 2 * MB * 64, acc_x<MB>(acc, g));
    bias_ln_relu<MB>(acc2, a.b1, a.g1, a.beta1, a.eps * a.s1 * a.s1, hh, true, a.s1);
  } else {
    gemm_acc_f32<MB, MB>(acc2, acc, (const f4 *)a.w1 + lane, 0);
    bias_ln_relu<MB>(acc2, a.b1, a.g1, a.beta1, a.eps, hh, true);
  }
  float part = 0.f;
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const f4 ww = *(const f4 *)(a.w2 + mb * 32 + 8 * q + 4 * hh);
#pragma unroll
      for (int t = 0; t < 4; ++t) part += acc2[mb][4 * q + t] * ww[t];
    }
  part += __shfl_xor(part, 32);
  if (valid && hh == 0) a.scores[row] = sigmoidf_stable(part + a.b2[0]);
}

// Kept edges per tile of CTILE consecutive candidates.
__global__ __launch_bounds__(CTHREADS) void compact_count(const float *__restrict__ scores,
                                                          int64_t n, float threshold,
                                                          int32_t *__restrict__ counts) {
  __shared__ int32_t part[CTHREADS / 64];
  const int64_t base = (int64_t)blockIdx.x * CTILE;
  int c = 0;
#pragma unroll
  for (int it = 0; it < CITEMS; ++it) {
    const int64_t i = base + (int64_t)it * CTHREADS + threadIdx.x;
    c += (i < n && scores[i] > threshold) ? 1 : 0;
  }
  for (int off = 32; off > 0; off >>= 1) c += __shfl_xor(c, off);
  if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = c;
  __syncthreads();
  if (threadIdx.x == 0) {
    int t = 0;
    for (int w = 0; w < CTHREADS / 64; ++w) t += part[w];
    counts[blockIdx.x] = t;
  }
}

// Exclusive scan of the tile counts in place; total -> *total.  One block.
__global__ __launch_bounds__(1024) void compact_scan(int32_t *__restrict__ counts, int32_t ntiles,
                                                     int32_t *__restrict__ total) {
  __shared__ int32_t part[1024];
  const int t = threadIdx.x;
  const int chunk = (ntiles + 1023) / 1024;
  const int beg = min(t * chunk, ntiles), end = min(beg + chunk, ntiles);
  int32_t s = 0;
  for (int i = beg; i < end; ++i) s += counts[i];
  part[t] = s;
  __syncthreads();
  for (int off = 1; off < 1024; off <<= 1) {
    const int32_t v = t >= off ? part[t - off] : 0;
    __syncthreads();
    part[t] += v;
    __syncthreads();
  }
  int32_t run = part[t] - s;
  for (int i = beg; i < end; ++i) {
    const int32_t v = counts[i];
    counts[i] = run;
    run += v;
  }
  if (t == 1023) *total = part[1023];
}

// Stable scatter of the kept edges: position = tile offset + kept items
// before this one in the tile (item order = (round, wave, lane)).
__global__ __launch_bounds__(CTHREADS) void compact_scatter(
    const float *__restrict__ scores, const int32_t *__restrict__ edge_index, int64_t n,
    float threshold, const int32_t *__restrict__ offs, const int32_t *__restrict__ total,
    int32_t *__restrict__ out) {
  __shared__ int32_t wcnt[CITEMS][CTHREADS / 64];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int64_t base = (int64_t)blockIdx.x * CTILE;
  const uint64_t lt = (1ull << lane) - 1ull;
  bool keep[CITEMS];
  int rank[CITEMS];
#pragma unroll
  for (int it = 0; it < CITEMS; ++it) {
    const int64_t i = base + (int64_t)it * CTHREADS + threadIdx.x;
    keep[it] = i < n && scores[i] > threshold;
    const uint64_t m = __ballot(keep[it]);
    rank[it] = __popcll(m & lt);
    if (lane == 0) wcnt[it][w] = __popcll(m);
  }
  __syncthreads();
  const int32_t tot = *total;
  int32_t run = offs[blockIdx.x];
#pragma unroll
  for (int it = 0; it < CITEMS; ++it) {
    int32_t before = run;
    for (int ww = 0; ww < w; ++ww) before += wcnt[it][ww];
    for (int ww = 0; ww < CTHREADS / 64; ++ww) run += wcnt[it][ww];
    if (keep[it]) {
      const int64_t i = base + (int64_t)it * CTHREADS + threadIdx.x;
      const int32_t pos = before + rank[it];
      if (pos < tot) {  // always true when the counts are consistent
        out[pos] = edge_index[i];
        out[(int64_t)tot + pos] = edge_index[n + i];
      }
    }
  }
}

inline unsigned blocks_for(int64_t n, int per) { return (unsigned)((n + per - 1) / per); }

}  // namespace

hipError_t launch_filter_scores(int hidden, const FilterArgs &a, hipStream_t stream) {
  const int64_t waves = (a.n_edges + 31) / 32;
  const int64_t blocks = (waves + FWAVES - 1) / FWAVES;
  if (blocks <= 0) return hipSuccess;
  if (blocks > INT32_MAX) return hipErrorInvalidValue;
  switch (hidden) {
    case 64:
      if (a.w1r) filter_mlp<2, true><<<(unsigned)blocks, 64 * FWAVES, 0, stream>>>(a);
      else filter_mlp<2, false><<<(unsigned)blocks, 64 * FWAVES, 0, stream>>>(a);
      break;
    case 128:
      if (a.w1r) filter_mlp<4, true><<<(unsigned)blocks, 64 * FWAVES, 0, stream>>>(a);
      else filter_mlp<4, false><<<(unsigned)blocks, 64 * FWAVES, 0, stream>>>(a);
      break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

size_t compact_tiles(int64_t n) { return (size_t)((n + CTILE - 1) / CTILE); }

hipError_t launch_compact(const float *scores, const int32_t *edge_index, int64_t n,
                          float threshold, int32_t *counts, int32_t *total, int32_t *out,
                          hipStream_t stream) {
  const int32_t ntiles = (int32_t)compact_tiles(n);
  if (ntiles == 0) return hipSuccess;
  compact_count<<<ntiles, CTHREADS, 0, stream>>>(scores, n, threshold, counts);
  compact_scan<<<1, 1024, 0, stream>>>(counts, ntiles, total);
  compact_scatter<<<ntiles, CTHREADS, 0, stream>>>(scores, edge_index, n, threshold, counts,
                                                   total, out);
  return hipGetLastError();
}

}  // namespace gnn
