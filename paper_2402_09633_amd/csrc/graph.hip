// Graph construction, the first stage of the pipeline (paper section 2.1: an
// embedding network maps every space point into a latent space, and a
// fixed-radius nearest-neighbour search there proposes the candidate edges
// that the filter and the GNN then score).
//
// embed       one wave per 32 points: layer 1 (F -> H) on VALU, LayerNorm/
//             ReLU, layer 2 (H -> H) on the matrix cores through the
//             accumulator chain, LayerNorm/ReLU, then the D outputs as VALU
//             dot products (D <= 16).  Layer 2 takes the split fp16 products
//             of split.hip (SPLIT: f16x2 records of s W1, bias s b1, eps
//             eps s^2) when the first LayerNorm's output bound fits the fp16
//             range, the fp32 matrix cores otherwise.
// frnn        every pair i < j with d2(i, j) < r2, where d2 is evaluated in
//             fp32 as d = fmaf(t, t, d) over the coordinates in ascending
//             order (t = z_i[k] - z_j[k]).  Points are binned on a grid over
//             the first min(3, D) coordinates with cells no narrower than the
//             radius, so a pair within the radius sits in the same or
//             adjacent cells; cells are hashed into a power-of-two table that
//             is turned into buckets by the CSR builder (a stable sort of the
//             points by bucket).  A point scans the buckets of the 3^g
//             neighbouring cells, each bucket once, so hash collisions never
//             produce a pair twice.  A count pass, an exclusive scan and a fill pass write
//             the pairs grouped by i (within one i in cell-scan order), which
//             is deterministic.
#include "device_common.h"

namespace gnn {
namespace {

constexpr int EWAVES = 4;
constexpr int FTHREADS = 256;

template <int MB, bool SPLIT>
__global__ __launch_bounds__(64 * EWAVES) void embed_mlp(EmbedArgs a) {
  constexpr int H = 32 * MB;
  const int lane = threadIdx.x & 63, hh = lane >> 5, n = lane & 31;
  const int blk = xcd_remap(blockIdx.x, gridDim.x);
  const int64_t row0 = ((int64_t)blk * EWAVES + (threadIdx.x >> 6)) * 32;
  if (row0 >= a.n) return;
  const int64_t row = row0 + n;
  const bool valid = row < a.n;
  const int64_t r = valid ? row : a.n - 1;

  f16v acc[MB];
  small_k_layer<MB>(acc, a.x, a.F, (int)r, a.w0t, a.b0, hh);
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
  for (int d = 0; d < a.D; ++d) {
    const float *wd = a.w2 + (int64_t)d * H + 4 * hh;
    float part = 0.f;
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const f4 ww = *(const f4 *)(wd + mb * 32 + 8 * q);
#pragma unroll
        for (int t = 0; t < 4; ++t) part += acc2[mb][4 * q + t] * ww[t];
      }
    part += __shfl_xor(part, 32);
    if (valid && hh == 0) a.z[row * a.D + d] = part + a.b2[d];
  }
}

// Grid cell of a point along the first g coordinates (coordinates clamped so
// that the cell index fits comfortably in an int).
__device__ __forceinline__ void cell_of(const float *zp, int g, float inv_cell, int (&c)[3]) {
#pragma unroll
  for (int k = 0; k < 3; ++k) {
    float v = k < g ? floorf(zp[k] * inv_cell) : 0.f;
    v = fminf(fmaxf(v, -1.0e9f), 1.0e9f);
    c[k] = (int)v;
  }
}

__device__ __forceinline__ uint32_t cell_hash(const int (&c)[3], uint32_t mask) {
  return ((uint32_t)c[0] * 73856093u ^ (uint32_t)c[1] * 19349663u ^ (uint32_t)c[2] * 83492791u) &
         mask;
}

// Bucket keys, written twice ([2][n]) as the CSR builder's edge list.
__global__ __launch_bounds__(FTHREADS) void frnn_keys(FrnnArgs a, int32_t *__restrict__ keys) {
  const int64_t i = (int64_t)blockIdx.x * FTHREADS + threadIdx.x;
  if (i >= a.n) return;
  int c[3];
  cell_of(a.z + i * a.D, a.g, a.inv_cell, c);
  const int32_t k = (int32_t)cell_hash(c, a.mask);
  keys[i] = k;
  keys[a.n + i] = k;
}

// The points' coordinates in bucket order: zs[p] = z[perm[p]].
__global__ __launch_bounds__(FTHREADS) void frnn_gather(FrnnArgs a, float *__restrict__ zs) {
  const int64_t t = (int64_t)blockIdx.x * FTHREADS + threadIdx.x;
  if (t >= a.n * a.D) return;
  const int64_t p = t / a.D;
  zs[t] = a.z[(int64_t)a.perm[p] * a.D + (t - p * a.D)];
}

// FILL = false: count the pairs of every point; true: write them.  Thread
// p handles the point at bucket position p (neighbouring threads handle
// neighbouring points, whose candidates they share in the caches).  The
// neighbouring cells' buckets are scanned once each (a bucket that two
// cells share through the hash is skipped the second time), so every other
// point is tested at most once; a point of a colliding far cell simply fails
// the distance test.  Candidates are taken U at a time: their ids and
// coordinates are requested together before any distance is formed, so a
// bucket costs one round of cache latency per U candidates rather than two
// dependent ones per candidate (positions past the bucket's end repeat its
// last point and are not counted).  The dimension D is a template argument:
// the coordinate loads and the distance chain unroll, with 16-byte loads
// when D is a multiple of 4 (rows of zs then start on 16-byte boundaries).
template <bool FILL, int D>
__global__ __launch_bounds__(FTHREADS) void frnn_pairs(FrnnArgs a, const float *__restrict__ zs) {
  constexpr int U = 4;
  constexpr int DZ = D < 3 ? 3 : D;  // cell_of reads up to 3 coordinates
  const int64_t p = (int64_t)blockIdx.x * FTHREADS + threadIdx.x;
  if (p >= a.n) return;
  const int32_t i = a.perm[p];
  auto load_row = [&](int64_t q, float *dst) {
    const float *src = zs + q * D;
    if constexpr (D % 4 == 0) {
#pragma unroll
      for (int k = 0; k < D; k += 4) {
        const f4 v = *(const f4 *)(src + k);
        dst[k] = v[0];
        dst[k + 1] = v[1];
        dst[k + 2] = v[2];
        dst[k + 3] = v[3];
      }
    } else {
#pragma unroll
      for (int k = 0; k < D; ++k) dst[k] = src[k];
    }
  };
  float zi[DZ];
#pragma unroll
  for (int k = D; k < DZ; ++k) zi[k] = 0.f;
  load_row(p, zi);
  int ci[3];
  cell_of(zi, a.g, a.inv_cell, ci);
  int64_t o = FILL ? a.offs[i] : 0;
  int32_t cnt = 0;
  uint32_t seen[27];
  int ns = 0;
  const int r2d = a.g > 1 ? 1 : 0, r3d = a.g > 2 ? 1 : 0;
  for (int dz = -r3d; dz <= r3d; ++dz)
    for (int dy = -r2d; dy <= r2d; ++dy)
      for (int dx = -1; dx <= 1; ++dx) {
        const int nc[3] = {ci[0] + dx, ci[1] + dy, ci[2] + dz};
        const uint32_t key = cell_hash(nc, a.mask);
        bool dup = false;
        for (int u = 0; u < ns; ++u) dup |= seen[u] == key;
        if (dup) continue;
        seen[ns++] = key;
        const int32_t qb = a.rp[key], qe = a.rp[key + 1];
        for (int32_t q0 = qb; q0 < qe; q0 += U) {
          int32_t jj[U];
          float zz[U][D];
#pragma unroll
          for (int u = 0; u < U; ++u) {
            const int32_t q = q0 + u < qe ? q0 + u : qe - 1;
            jj[u] = a.perm[q];
            load_row(q, zz[u]);
          }
#pragma unroll
          for (int u = 0; u < U; ++u) {
            if (q0 + u >= qe || jj[u] <= i) continue;
            float acc = 0.f;
#pragma unroll
            for (int k = 0; k < D; ++k) {
              const float t = zi[k] - zz[u][k];
              acc = __builtin_fmaf(t, t, acc);
            }
            if (acc < a.r2) {
              if constexpr (FILL) {
                a.out[o] = i;
                a.out[a.total + o] = jj[u];
                ++o;
              } else {
                ++cnt;
              }
            }
          }
        }
      }
  if constexpr (!FILL) a.count[i] = cnt;
}

template <bool FILL>
hipError_t launch_pairs(const FrnnArgs &a, const float *zs, hipStream_t stream) {
  const unsigned blocks = (unsigned)((a.n + FTHREADS - 1) / FTHREADS);
  switch (a.D) {
#define GNN_FRNN_D(d) \
  case d: frnn_pairs<FILL, d><<<blocks, FTHREADS, 0, stream>>>(a, zs); break;
    GNN_FRNN_D(1) GNN_FRNN_D(2) GNN_FRNN_D(3) GNN_FRNN_D(4) GNN_FRNN_D(5) GNN_FRNN_D(6)
    GNN_FRNN_D(7) GNN_FRNN_D(8) GNN_FRNN_D(9) GNN_FRNN_D(10) GNN_FRNN_D(11) GNN_FRNN_D(12)
    GNN_FRNN_D(13) GNN_FRNN_D(14) GNN_FRNN_D(15) GNN_FRNN_D(16)
#undef GNN_FRNN_D
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

// Exclusive scan of the per-point counts into offs (int64), total -> *total:
// per-tile sums (tiles of 2048 counts), a scan of the tile sums, then each
// tile's own scan.  Thread t of a tile owns its 8 consecutive counts.
constexpr int ST = 256, SI = 8, STILE = ST * SI;

// Exclusive scan of v over the block; *sum gets the block total.
__device__ __forceinline__ int64_t block_excl_scan(int64_t v, int64_t *sum) {
  __shared__ int64_t part[ST];
  const int t = threadIdx.x;
  part[t] = v;
  __syncthreads();
  for (int off = 1; off < ST; off <<= 1) {
    const int64_t u = t >= off ? part[t - off] : 0;
    __syncthreads();
    part[t] += u;
    __syncthreads();
  }
  const int64_t incl = part[t];
  *sum = part[ST - 1];
  __syncthreads();
  return incl - v;
}

__global__ __launch_bounds__(ST) void scan_tiles(const int32_t *__restrict__ count, int64_t n,
                                                 int64_t *__restrict__ bsum) {
  const int64_t base = (int64_t)blockIdx.x * STILE + (int64_t)threadIdx.x * SI;
  int64_t s = 0;
#pragma unroll
  for (int k = 0; k < SI; ++k)
    if (base + k < n) s += count[base + k];
  int64_t tot;
  (void)block_excl_scan(s, &tot);
  if (threadIdx.x == 0) bsum[blockIdx.x] = tot;
}

// In place over the nb tile sums, ST at a time with a running carry.
__global__ __launch_bounds__(ST) void scan_sums(int64_t *__restrict__ bsum, int64_t nb,
                                                int64_t *__restrict__ total) {
  int64_t carry = 0;
  for (int64_t b0 = 0; b0 < nb; b0 += ST) {
    const int64_t i = b0 + threadIdx.x;
    const int64_t v = i < nb ? bsum[i] : 0;
    int64_t tot;
    const int64_t ex = block_excl_scan(v, &tot);
    if (i < nb) bsum[i] = carry + ex;
    carry += tot;
  }
  if (threadIdx.x == 0) *total = carry;
}

__global__ __launch_bounds__(ST) void scan_down(const int32_t *__restrict__ count, int64_t n,
                                                const int64_t *__restrict__ bsum,
                                                int64_t *__restrict__ offs) {
  const int64_t base = (int64_t)blockIdx.x * STILE + (int64_t)threadIdx.x * SI;
  int32_t c[SI];
  int64_t s = 0;
#pragma unroll
  for (int k = 0; k < SI; ++k) {
    c[k] = base + k < n ? count[base + k] : 0;
    s += c[k];
  }
  int64_t tot;
  int64_t run = bsum[blockIdx.x] + block_excl_scan(s, &tot);
#pragma unroll
  for (int k = 0; k < SI; ++k)
    if (base + k < n) {
      offs[base + k] = run;
      run += c[k];
    }
}

}  // namespace

hipError_t launch_embed(int hidden, const EmbedArgs &a, hipStream_t stream) {
  if (a.n <= 0) return hipSuccess;
  if (a.D < 1 || a.D > 16 || a.F < 1 || a.F > MAX_F) return hipErrorInvalidValue;
  const int64_t waves = (a.n + 31) / 32;
  const unsigned blocks = (unsigned)((waves + EWAVES - 1) / EWAVES);
  switch (hidden) {
    case 64:
      if (a.w1r) embed_mlp<2, true><<<blocks, 64 * EWAVES, 0, stream>>>(a);
      else embed_mlp<2, false><<<blocks, 64 * EWAVES, 0, stream>>>(a);
      break;
    case 128:
      if (a.w1r) embed_mlp<4, true><<<blocks, 64 * EWAVES, 0, stream>>>(a);
      else embed_mlp<4, false><<<blocks, 64 * EWAVES, 0, stream>>>(a);
      break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

size_t frnn_scan_blocks(int64_t n) { return (size_t)((n + STILE - 1) / STILE); }

hipError_t launch_frnn_keys(const FrnnArgs &a, int32_t *keys, hipStream_t stream) {
  if (a.n <= 0) return hipSuccess;
  frnn_keys<<<(unsigned)((a.n + FTHREADS - 1) / FTHREADS), FTHREADS, 0, stream>>>(a, keys);
  return hipGetLastError();
}

hipError_t launch_frnn_count(const FrnnArgs &a, float *zs, hipStream_t stream) {
  if (a.n <= 0) return hipSuccess;
  const int64_t nz = a.n * a.D;
  frnn_gather<<<(unsigned)((nz + FTHREADS - 1) / FTHREADS), FTHREADS, 0, stream>>>(a, zs);
  hipError_t e = launch_pairs<false>(a, zs, stream);
  if (e != hipSuccess) return e;
  const int64_t nb = (int64_t)frnn_scan_blocks(a.n);
  scan_tiles<<<(unsigned)nb, ST, 0, stream>>>(a.count, a.n, a.bsum);
  scan_sums<<<1, ST, 0, stream>>>(a.bsum, nb, a.total_dev);
  scan_down<<<(unsigned)nb, ST, 0, stream>>>(a.count, a.n, a.bsum, a.offs);
  return hipGetLastError();
}

hipError_t launch_frnn_fill(const FrnnArgs &a, const float *zs, hipStream_t stream) {
  if (a.n <= 0) return hipSuccess;
  return launch_pairs<true>(a, zs, stream);
}

}  // namespace gnn

// ---------------------------------------------------------------- host ---

#include <cmath>

#include "../../include/gnn.h"

namespace {

size_t align256(size_t n) { return (n + 255) & ~(size_t)255; }

}  // namespace

extern "C" int gnn_frnn(const float *z, int64_t n_nodes, int32_t dim, float r2,
                        int32_t *edge_index, int64_t max_pairs, int64_t *n_pairs,
                        hipStream_t stream) {
  using namespace gnn;
  if (!n_pairs) return set_error(GNN_E_INVALID_ARG, "n_pairs is NULL");
  *n_pairs = 0;
  if (n_nodes < 0 || n_nodes > INT32_MAX)
    return set_error(GNN_E_INVALID_ARG, "n_nodes outside 0..INT32_MAX");
  if (n_nodes >= CSR_MAX_ITEMS)
    return set_error(GNN_E_UNSUPPORTED, "the cell sort takes at most 2^30 - 1 points");
  if (dim < 1 || dim > 16) return set_error(GNN_E_INVALID_ARG, "dim outside 1..16");
  if (max_pairs < 0) return set_error(GNN_E_INVALID_ARG, "max_pairs is negative");
  if (n_nodes > 0 && !z) return set_error(GNN_E_INVALID_ARG, "z is NULL");
  if (std::isnan(r2)) return set_error(GNN_E_INVALID_ARG, "r2 is NaN");
  if (n_nodes < 2 || !(r2 > 0.f)) return GNN_OK;

  FrnnArgs a;
  a.z = z;
  a.n = n_nodes;
  a.D = dim;
  a.g = dim < 3 ? dim : 3;
  a.r2 = r2;
  // Cells a little wider than the radius: a pair that passes the fp32 test
  // differs by less than that along every coordinate.
  const double cell = 1.001 * std::sqrt((double)r2);
  a.inv_cell = std::isfinite(cell) && cell > 0.0 ? (float)(1.0 / cell) : 0.f;
  uint32_t m = 64;
  while ((int64_t)m < 2 * n_nodes && m < (1u << 30)) m <<= 1;
  a.mask = m - 1;

  const int64_t n = n_nodes;
  size_t off = 0;
  auto take = [&](size_t b) {
    const size_t o = off;
    off += align256(b > 0 ? b : 1);
    return o;
  };
  const size_t o_keys = take((size_t)2 * n * 4);
  const size_t o_rpi = take(((size_t)m + 1) * 4), o_pi = take((size_t)n * 4);
  const size_t o_rpo = take(((size_t)m + 1) * 4), o_po = take((size_t)n * 4);
  const size_t o_pa = take((size_t)2 * n * 8), o_pb = take((size_t)2 * n * 8);
  const size_t o_st = take(csr_scratch_bytes(n, m));
  const size_t o_cnt = take((size_t)n * 4), o_offs = take((size_t)n * 8), o_total = take(8);
  const size_t o_bsum = take(frnn_scan_blocks(n) * 8);
  const size_t o_zs = take((size_t)n * dim * 4);
  void *base = nullptr;
  if (hipMallocAsync(&base, off, stream) != hipSuccess) {
    (void)hipGetLastError();
    return set_error(GNN_E_OOM, "frnn workspace allocation failed");
  }
  unsigned char *b = (unsigned char *)base;
  int32_t *keys = (int32_t *)(b + o_keys);
  CsrScratch cs;
  cs.pairs_a = (uint2 *)(b + o_pa);
  cs.pairs_b = (uint2 *)(b + o_pb);
  cs.status = (uint32_t *)(b + o_st);
  a.rp = (const int32_t *)(b + o_rpi);
  a.perm = (const int32_t *)(b + o_pi);
  a.count = (int32_t *)(b + o_cnt);
  a.offs = (int64_t *)(b + o_offs);
  a.total_dev = (int64_t *)(b + o_total);
  a.bsum = (int64_t *)(b + o_bsum);

  int rc = GNN_OK;
  int64_t total = 0;
  hipError_t e = launch_frnn_keys(a, keys, stream);
  if (e == hipSuccess)
    e = build_csr(keys, (int32_t)n, (int32_t)m, (int32_t *)(b + o_rpi), (int32_t *)(b + o_pi),
                  (int32_t *)(b + o_rpo), (int32_t *)(b + o_po), cs, nullptr, nullptr, nullptr,
                  stream);
  float *zs = (float *)(b + o_zs);
  if (e == hipSuccess) e = launch_frnn_count(a, zs, stream);
  if (e == hipSuccess) e = hipMemcpyAsync(&total, a.total_dev, 8, hipMemcpyDeviceToHost, stream);
  if (e == hipSuccess) e = hipStreamSynchronize(stream);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    rc = set_error(GNN_E_HIP, hipGetErrorString(e));
  } else {
    *n_pairs = total;
    if (total > INT32_MAX) {
      rc = set_error(GNN_E_UNSUPPORTED, "more than INT32_MAX pairs");
    } else if (edge_index && total > max_pairs) {
      rc = set_error(GNN_E_INVALID_ARG, "edge_index holds fewer pairs than found (see n_pairs)");
    } else if (edge_index && total > 0) {
      a.total = total;
      a.out = edge_index;
      e = launch_frnn_fill(a, zs, stream);
      if (e != hipSuccess) rc = set_error(GNN_E_HIP, hipGetErrorString(e));
    }
  }
  if (hipFreeAsync(base, stream) != hipSuccess && rc == GNN_OK)
    rc = set_error(GNN_E_HIP, "frnn workspace release failed");
  return rc;
}
