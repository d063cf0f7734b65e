// Stable CSR construction on the GPU: an LSD radix sort of (key, edge id)
// pairs with 8-bit digits, then row pointers read off the sorted keys.
//
// The aggregation step sums messages into each destination (and each
// source) node; this file builds the destination-sorted and source-sorted
// edge lists it walks.  Stability makes every row list ascending in edge id,
// so the CSR equals the plain counting-sort definition word for word and the
// segmented sums run in a fixed order (bitwise run-to-run determinism).
// Only integer atomics on LDS counters are used.
//
// Sort layout: a block of 256 threads (4 waves) owns a tile of
// RS_TILE = 4 x 64 x RS_ITEMS consecutive items; wave w owns the w-th
// quarter, lane l item w*512 + it*64 + l in round it.  Stable order inside a
// tile is (wave, round, lane) = item order.
#include "gnn_internal.h"

namespace gnn {
namespace {

constexpr int RS_ITEMS = 8;
constexpr int RS_WAVES = 4;
constexpr int RS_THREADS = 64 * RS_WAVES;
constexpr int RS_TILE = RS_THREADS * RS_ITEMS;
constexpr int RS_RADIX = 256;

__device__ __forceinline__ uint32_t clamp_key(int32_t k, int32_t n) {
  return k < 0 ? 0u : (k >= n ? (uint32_t)(n - 1) : (uint32_t)k);
}

// The two sorts of one CSR build (by destination, by source) run side by
// side: blockIdx.y selects the sort, and each sort has its own slice of the
// scratch buffers.
struct SortSet {
  const int32_t *keys_i32[2];   // pass 0: raw indices (clamped here)
  const uint32_t *keys_in[2];   // later passes
  const uint32_t *vals_in[2];   // nullptr in pass 0: the value is the item index
  uint32_t *keys_out[2];
  uint32_t *vals_out[2];
  uint32_t *hist[2];            // [RS_RADIX][ntiles] counts, then offsets
  uint32_t *totals[2];          // [RS_RADIX] per-digit totals (zeroed beforehand)
};

__device__ __forceinline__ uint32_t load_key(const SortSet &S, int y, int64_t i, int32_t n_nodes) {
  return S.keys_i32[y] ? clamp_key(S.keys_i32[y][i], n_nodes) : S.keys_in[y][i];
}

__global__ __launch_bounds__(RS_THREADS) void rs_upsweep(SortSet S, int32_t n, int32_t n_nodes,
                                                         int shift, int32_t ntiles) {
  __shared__ uint32_t cnt[RS_RADIX];
  const int y = blockIdx.y;
  cnt[threadIdx.x] = 0;  // RS_THREADS == RS_RADIX
  __syncthreads();
  const int64_t base = (int64_t)blockIdx.x * RS_TILE;
#pragma unroll
  for (int it = 0; it < RS_ITEMS; ++it) {
    const int64_t i = base + (int64_t)it * RS_THREADS + threadIdx.x;
    if (i < n) atomicAdd(&cnt[(load_key(S, y, i, n_nodes) >> shift) & (RS_RADIX - 1)], 1u);
  }
  __syncthreads();
  const uint32_t c = cnt[threadIdx.x];
  S.hist[y][(int64_t)threadIdx.x * ntiles + blockIdx.x] = c;
  if (c) atomicAdd(&S.totals[y][threadIdx.x], c);
}

// Block d turns row d of the count matrix into exclusive offsets:
// offs[d][t] = (items with a smaller digit) + (items with digit d in earlier
// tiles).  Digit-major order is what makes the sort stable.
__global__ __launch_bounds__(RS_THREADS) void rs_scan_digit(SortSet S, int32_t ntiles) {
  __shared__ uint32_t part[RS_THREADS];
  __shared__ uint32_t carry;
  const int y = blockIdx.y, d = blockIdx.x, t = threadIdx.x;
  part[t] = t < d ? S.totals[y][t] : 0u;
  __syncthreads();
  for (int off = RS_THREADS / 2; off > 0; off >>= 1) {
    if (t < off) part[t] += part[t + off];
    __syncthreads();
  }
  if (t == 0) carry = part[0];
  __syncthreads();
  uint32_t *row = S.hist[y] + (int64_t)d * ntiles;
  for (int32_t c0 = 0; c0 < ntiles; c0 += RS_THREADS) {
    const int32_t i = c0 + t;
    const uint32_t v = i < ntiles ? row[i] : 0u;
    part[t] = v;
    __syncthreads();
    // Hillis-Steele inclusive scan of this chunk.
    for (int off = 1; off < RS_THREADS; off <<= 1) {
      const uint32_t u = t >= off ? part[t - off] : 0u;
      __syncthreads();
      part[t] += u;
      __syncthreads();
    }
    if (i < ntiles) row[i] = carry + part[t] - v;
    __syncthreads();
    if (t == RS_THREADS - 1) carry += part[t];
    __syncthreads();
  }
}

__global__ __launch_bounds__(RS_THREADS) void rs_scatter(SortSet S, int32_t n, int32_t n_nodes,
                                                         int shift, int32_t ntiles) {
  __shared__ uint32_t cnt[RS_WAVES][RS_RADIX];
  __shared__ uint32_t base[RS_WAVES][RS_RADIX];
  const int y = blockIdx.y;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  for (int i = 0; i < RS_WAVES; ++i) cnt[i][threadIdx.x] = 0;
  __syncthreads();

  const int64_t tile0 = (int64_t)blockIdx.x * RS_TILE + (int64_t)w * 64 * RS_ITEMS;
  const uint64_t lt = (1ull << lane) - 1ull;
  uint32_t key[RS_ITEMS], val[RS_ITEMS], pre[RS_ITEMS];
#pragma unroll
  for (int it = 0; it < RS_ITEMS; ++it) {
    const int64_t i = tile0 + (int64_t)it * 64 + lane;
    const bool ok = i < n;
    uint32_t k = 0, v = 0;
    if (ok) {
      k = load_key(S, y, i, n_nodes);
      v = S.vals_in[y] ? S.vals_in[y][i] : (uint32_t)i;
    }
    key[it] = k;
    val[it] = v;
    const uint32_t d = (k >> shift) & (RS_RADIX - 1);
    // Lanes of this round holding the same digit (8 ballots).
    uint64_t m = __ballot(ok);
#pragma unroll
    for (int b = 0; b < 8; ++b) {
      const uint64_t bal = __ballot((d >> b) & 1u);
      m &= ((d >> b) & 1u) ? bal : ~bal;
    }
    uint32_t before = 0;
    if (ok) before = cnt[w][d];
    pre[it] = before + (uint32_t)__popcll(m & lt);
    // The lowest lane of each digit group advances the wave's counter; all
    // lanes read the counter above before any lane writes it.
    if (ok && (m & lt) == 0) cnt[w][d] = before + (uint32_t)__popcll(m);
  }
  __syncthreads();
  {
    const int d = threadIdx.x;
    uint32_t run = S.hist[y][(int64_t)d * ntiles + blockIdx.x];
#pragma unroll
    for (int i = 0; i < RS_WAVES; ++i) {
      base[i][d] = run;
      run += cnt[i][d];
    }
  }
  __syncthreads();
#pragma unroll
  for (int it = 0; it < RS_ITEMS; ++it) {
    const int64_t i = tile0 + (int64_t)it * 64 + lane;
    if (i < n) {
      const uint32_t d = (key[it] >> shift) & (RS_RADIX - 1);
      const uint32_t pos = base[w][d] + pre[it];
      if (pos < (uint32_t)n) {  // always true when the ranks are consistent
        S.keys_out[y][pos] = key[it];
        S.vals_out[y][pos] = val[it];
      }
    }
  }
}

// row_ptr[v] = number of sorted keys < v (lower bound), v in [0, n_nodes];
// also copies the sorted values out as the permutation.
struct CsrOut {
  const uint32_t *skeys[2];
  const uint32_t *svals[2];
  int32_t *row_ptr[2];
  int32_t *perm[2];
};

__global__ void csr_finish(CsrOut O, int32_t n, int32_t n_nodes) {
  const int y = blockIdx.y;
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i <= n_nodes) {
    const uint32_t v = (uint32_t)i;
    const uint32_t *k = O.skeys[y];
    int32_t lo = 0, hi = n;
    while (lo < hi) {
      const int32_t mid = (int32_t)(((int64_t)lo + hi) >> 1);
      if (k[mid] < v) lo = mid + 1;
      else hi = mid;
    }
    O.row_ptr[y][i] = lo;
  }
  if (i < n) O.perm[y][i] = (int32_t)O.svals[y][i];
}

__global__ void validate_idx(const int32_t *__restrict__ ei, int64_t n, int32_t n_nodes,
                             int32_t *__restrict__ flag) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) {
    const int32_t v = ei[i];
    if (v < 0 || v >= n_nodes) *flag = 1;  // every writer stores the same value
  }
}

__global__ void fill_i32(int32_t *__restrict__ p, int64_t n, int32_t v) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = v;
}

__global__ void bf16_to_f32(const __bf16 *__restrict__ in, float *__restrict__ out, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) out[i] = (float)in[i];
}

// The edge list in source order (positions p of the source CSR) and the
// inverse of that order.
__global__ void edge_order_k(const int32_t *__restrict__ ei, const int32_t *__restrict__ perm_out,
                             int32_t n, int32_t n_nodes, int32_t *__restrict__ eis,
                             int32_t *__restrict__ inv) {
  const int64_t p = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (p >= n) return;
  const int32_t j = perm_out[p];
  eis[p] = (int32_t)clamp_key(ei[j], n_nodes);
  eis[n + p] = (int32_t)clamp_key(ei[n + j], n_nodes);
  inv[j] = (int32_t)p;
}

__global__ void compose_k(const int32_t *__restrict__ perm_in, const int32_t *__restrict__ inv,
                          int32_t n, int32_t *__restrict__ q_in) {
  const int64_t k = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (k < n) q_in[k] = inv[perm_in[k]];
}

template <typename T>
__global__ void scatter_rows_k(const T *__restrict__ src, const int32_t *__restrict__ idx,
                               float *__restrict__ dst, int64_t rows, int H) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= rows * H) return;
  const int64_t r = i / H, c = i % H;
  dst[(int64_t)idx[r] * H + c] = (float)src[i];
}

inline unsigned blocks_for(int64_t n, int per) { return (unsigned)((n + per - 1) / per); }

}  // namespace

size_t csr_hist_len(int64_t n_edges) {
  return (size_t)RS_RADIX * (size_t)((n_edges + RS_TILE - 1) / RS_TILE);
}

hipError_t build_csr(const int32_t *edge_index, int32_t n, int32_t n_nodes, int32_t *row_ptr_in,
                     int32_t *perm_in, int32_t *row_ptr_out, int32_t *perm_out,
                     const CsrScratch &s, hipStream_t stream) {
  // Number of 8-bit digits needed for keys in [0, n_nodes); at least one
  // pass so that the sorted arrays are always written.
  int bits = 0;
  while (bits < 31 && ((int64_t)1 << bits) < (int64_t)n_nodes) ++bits;
  const int passes = bits > 0 ? (bits + 7) / 8 : 1;
  const int32_t ntiles = (int32_t)((n + RS_TILE - 1) / RS_TILE);
  const size_t hl = csr_hist_len(n);
  const dim3 grid(ntiles, 2);

  // Sort 0: keys = destinations (row 1), sort 1: keys = sources (row 0).
  uint32_t *ka[2] = {s.keys_a, s.keys_a + n}, *kb[2] = {s.keys_b, s.keys_b + n};
  uint32_t *va[2] = {s.vals_a, s.vals_a + n}, *vb[2] = {s.vals_b, s.vals_b + n};
  fill_i32<<<blocks_for(2 * RS_RADIX * passes, 256), 256, 0, stream>>>(
      (int32_t *)s.totals, 2 * RS_RADIX * passes, 0);
  SortSet S{};
  S.keys_i32[0] = edge_index + n;
  S.keys_i32[1] = edge_index;
  for (int y = 0; y < 2; ++y) {
    S.hist[y] = s.hist + y * hl;
  }
  for (int p = 0; p < passes; ++p) {
    for (int y = 0; y < 2; ++y) {
      S.totals[y] = s.totals + (p * 2 + y) * RS_RADIX;
      S.keys_out[y] = (p & 1) ? kb[y] : ka[y];
      S.vals_out[y] = (p & 1) ? vb[y] : va[y];
    }
    const int shift = 8 * p;
    rs_upsweep<<<grid, RS_THREADS, 0, stream>>>(S, n, n_nodes, shift, ntiles);
    rs_scan_digit<<<dim3(RS_RADIX, 2), RS_THREADS, 0, stream>>>(S, ntiles);
    rs_scatter<<<grid, RS_THREADS, 0, stream>>>(S, n, n_nodes, shift, ntiles);
    for (int y = 0; y < 2; ++y) {
      S.keys_i32[y] = nullptr;
      S.keys_in[y] = S.keys_out[y];
      S.vals_in[y] = S.vals_out[y];
    }
  }
  CsrOut O{};
  for (int y = 0; y < 2; ++y) {
    O.skeys[y] = S.keys_in[y];
    O.svals[y] = S.vals_in[y];
  }
  O.row_ptr[0] = row_ptr_in;
  O.perm[0] = perm_in;
  O.row_ptr[1] = row_ptr_out;
  O.perm[1] = perm_out;
  const int64_t m = (int64_t)(n > n_nodes ? n : n_nodes) + 1;
  csr_finish<<<dim3(blocks_for(m, 256), 2), 256, 0, stream>>>(O, n, n_nodes);
  return hipGetLastError();
}

hipError_t launch_validate(const int32_t *edge_index, int64_t n_edges, int32_t n_nodes,
                           int32_t *flag, hipStream_t stream) {
  const int64_t n = 2 * n_edges;
  validate_idx<<<blocks_for(n, 256), 256, 0, stream>>>(edge_index, n, n_nodes, flag);
  return hipGetLastError();
}

hipError_t launch_fill_i32(int32_t *p, int64_t n, int32_t v, hipStream_t stream) {
  if (n > 0) fill_i32<<<blocks_for(n, 256), 256, 0, stream>>>(p, n, v);
  return hipGetLastError();
}

hipError_t launch_edge_order(const int32_t *edge_index, const int32_t *perm_out,
                             const int32_t *perm_in, int32_t n_edges, int32_t n_nodes,
                             int32_t *eis, int32_t *inv, int32_t *q_in, hipStream_t stream) {
  if (n_edges <= 0) return hipSuccess;
  edge_order_k<<<blocks_for(n_edges, 256), 256, 0, stream>>>(edge_index, perm_out, n_edges,
                                                            n_nodes, eis, inv);
  compose_k<<<blocks_for(n_edges, 256), 256, 0, stream>>>(perm_in, inv, n_edges, q_in);
  return hipGetLastError();
}

hipError_t launch_scatter_rows(Act act, const void *src, const int32_t *idx, float *dst,
                               int64_t rows, int H, hipStream_t stream) {
  const int64_t n = rows * H;
  if (n <= 0) return hipSuccess;
  if (act == Act::F32)
    scatter_rows_k<float><<<blocks_for(n, 256), 256, 0, stream>>>((const float *)src, idx, dst,
                                                                  rows, H);
  else
    scatter_rows_k<__bf16><<<blocks_for(n, 256), 256, 0, stream>>>((const __bf16 *)src, idx,
                                                                   dst, rows, H);
  return hipGetLastError();
}

hipError_t launch_bf16_to_f32(const void *in, float *out, int64_t n, hipStream_t stream) {
  if (n > 0)
    bf16_to_f32<<<blocks_for(n, 256), 256, 0, stream>>>((const __bf16 *)in, out, n);
  return hipGetLastError();
}

}  // namespace gnn
