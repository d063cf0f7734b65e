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

// Pass 0 reads int32 keys from edge_index (clamped); later passes read the
// previous pass's uint32 keys.
__global__ __launch_bounds__(RS_THREADS) void rs_upsweep(const int32_t *__restrict__ keys_i32,
                                                         const uint32_t *__restrict__ keys_u32,
                                                         int32_t n, int32_t n_nodes, int shift,
                                                         uint32_t *__restrict__ hist,
                                                         int32_t ntiles) {
  __shared__ uint32_t cnt[RS_RADIX];
  cnt[threadIdx.x] = 0;  // RS_THREADS == RS_RADIX
  __syncthreads();
  const int64_t base = (int64_t)blockIdx.x * RS_TILE;
#pragma unroll
  for (int it = 0; it < RS_ITEMS; ++it) {
    const int64_t i = base + (int64_t)it * RS_THREADS + threadIdx.x;
    if (i < n) {
      const uint32_t k = keys_i32 ? clamp_key(keys_i32[i], n_nodes) : keys_u32[i];
      atomicAdd(&cnt[(k >> shift) & (RS_RADIX - 1)], 1u);
    }
  }
  __syncthreads();
  hist[(int64_t)threadIdx.x * ntiles + blockIdx.x] = cnt[threadIdx.x];
}

// Exclusive scan, in place, of `len` counters (digit-major: all tiles of
// digit 0, then digit 1, ...).  One block; thread t scans a contiguous chunk.
__global__ __launch_bounds__(1024) void rs_scan(uint32_t *__restrict__ a, int32_t len) {
  __shared__ uint32_t part[1024];
  const int t = threadIdx.x;
  const int chunk = (len + 1023) / 1024;
  const int beg = min(t * chunk, len), end = min(beg + chunk, len);
  uint32_t s = 0;
  for (int i = beg; i < end; ++i) s += a[i];
  part[t] = s;
  __syncthreads();
  // Hillis-Steele inclusive scan over the 1024 partial sums.
  for (int off = 1; off < 1024; off <<= 1) {
    const uint32_t v = t >= off ? part[t - off] : 0u;
    __syncthreads();
    part[t] += v;
    __syncthreads();
  }
  uint32_t run = part[t] - s;
  for (int i = beg; i < end; ++i) {
    const uint32_t v = a[i];
    a[i] = run;
    run += v;
  }
}

__global__ __launch_bounds__(RS_THREADS) void rs_scatter(
    const int32_t *__restrict__ keys_i32, const uint32_t *__restrict__ keys_u32,
    const uint32_t *__restrict__ vals_in, int32_t n, int32_t n_nodes, int shift,
    const uint32_t *__restrict__ offs, int32_t ntiles, uint32_t *__restrict__ keys_out,
    uint32_t *__restrict__ vals_out) {
  __shared__ uint32_t cnt[RS_WAVES][RS_RADIX];
  __shared__ uint32_t base[RS_WAVES][RS_RADIX];
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
      k = keys_i32 ? clamp_key(keys_i32[i], n_nodes) : keys_u32[i];
      v = vals_in ? vals_in[i] : (uint32_t)i;
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
    uint32_t run = offs[(int64_t)d * ntiles + blockIdx.x];
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
        keys_out[pos] = key[it];
        vals_out[pos] = val[it];
      }
    }
  }
}

// row_ptr[v] = number of sorted keys < v, for v in [0, n_nodes].  Thread p
// (0 <= p <= n) writes every v with skeys[p-1] < v <= skeys[p].
__global__ void csr_rowptr(const uint32_t *__restrict__ skeys, int32_t n, int32_t n_nodes,
                           int32_t *__restrict__ row_ptr) {
  const int64_t p = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (p > n) return;
  const int64_t lo = p == 0 ? 0 : (int64_t)skeys[p - 1] + 1;
  const int64_t hi = p == n ? n_nodes : min((int64_t)skeys[p], (int64_t)n_nodes);
  for (int64_t v = lo; v <= hi; ++v) row_ptr[v] = (int32_t)p;
}

__global__ void copy_u32(const uint32_t *__restrict__ a, int32_t *__restrict__ b, int32_t n) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) b[i] = (int32_t)a[i];
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

inline unsigned blocks_for(int64_t n, int per) { return (unsigned)((n + per - 1) / per); }

}  // namespace

size_t csr_hist_len(int64_t n_edges) {
  return (size_t)RS_RADIX * (size_t)((n_edges + RS_TILE - 1) / RS_TILE);
}

hipError_t build_csr(const int32_t *keys, int32_t n, int32_t n_nodes, int32_t *row_ptr,
                     int32_t *perm, const CsrScratch &s, hipStream_t stream) {
  // Number of 8-bit digits needed for keys in [0, n_nodes).
  int bits = 0;
  while (bits < 31 && ((int64_t)1 << bits) < (int64_t)n_nodes) ++bits;
  const int passes = (bits + 7) / 8;
  const int32_t ntiles = (int32_t)((n + RS_TILE - 1) / RS_TILE);
  const int32_t len = RS_RADIX * ntiles;

  const uint32_t *kin = nullptr, *vin = nullptr;
  uint32_t *kout = s.keys_a, *vout = s.vals_a;
  for (int p = 0; p < passes; ++p) {
    const int shift = 8 * p;
    const int32_t *k32 = p == 0 ? keys : nullptr;
    rs_upsweep<<<ntiles, RS_THREADS, 0, stream>>>(k32, kin, n, n_nodes, shift, s.hist, ntiles);
    rs_scan<<<1, 1024, 0, stream>>>(s.hist, len);
    rs_scatter<<<ntiles, RS_THREADS, 0, stream>>>(k32, kin, vin, n, n_nodes, shift, s.hist,
                                                 ntiles, kout, vout);
    kin = kout;
    vin = vout;
    kout = (kout == s.keys_a) ? s.keys_b : s.keys_a;
    vout = (vout == s.vals_a) ? s.vals_b : s.vals_a;
  }
  if (passes == 0) {
    // n_nodes == 1: every key is 0 and the order is the identity.
    rs_upsweep<<<ntiles, RS_THREADS, 0, stream>>>(keys, nullptr, n, n_nodes, 0, s.hist, ntiles);
    rs_scan<<<1, 1024, 0, stream>>>(s.hist, len);
    rs_scatter<<<ntiles, RS_THREADS, 0, stream>>>(keys, nullptr, nullptr, n, n_nodes, 0, s.hist,
                                                 ntiles, s.keys_a, s.vals_a);
    kin = s.keys_a;
    vin = s.vals_a;
  }
  copy_u32<<<blocks_for(n, 256), 256, 0, stream>>>(vin, perm, n);
  csr_rowptr<<<blocks_for((int64_t)n + 1, 256), 256, 0, stream>>>(kin, n, n_nodes, row_ptr);
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

hipError_t launch_bf16_to_f32(const void *in, float *out, int64_t n, hipStream_t stream) {
  if (n > 0)
    bf16_to_f32<<<blocks_for(n, 256), 256, 0, stream>>>((const __bf16 *)in, out, n);
  return hipGetLastError();
}

}  // namespace gnn
