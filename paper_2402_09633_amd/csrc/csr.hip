// Stable CSR construction on the GPU: an LSD radix sort of (key, edge id)
// pairs, then row pointers read off the sorted keys.
//
// The aggregation step sums messages into each destination (and each
// source) node; this file builds the destination-sorted and source-sorted
// edge lists it walks.  Stability makes every row list ascending in edge id,
// so the CSR equals the plain counting-sort definition word for word and the
// segmented sums run in a fixed order (bitwise run-to-run determinism).
// Counts are integer atomics; no floating point is involved.
//
// Digits are up to 10 bits wide: keys below 2^20 (a million nodes) take two
// passes, keys below 2^10 one.  Launches per build: one fill (clears the
// counters), one histogram of every pass's digits, one single-sweep launch
// per pass, and one that reads off the row pointers.  Both sorts (by
// destination, by source) share each launch.
//
// Sort layout: a block of 1024 threads (16 waves) owns a tile of
// OS_TILE = 16 x 64 x OS_ITEMS consecutive items; wave w owns the w-th
// sixteenth, lane l item w*64*OS_ITEMS + it*64 + l in round it.  Stable
// order inside a tile is (wave, round, lane) = item order.
#include "gnn_internal.h"

namespace gnn {
namespace {

constexpr int RS_MAX_BITS = 10;             // widest digit
constexpr int RS_RADIX = 1 << RS_MAX_BITS;  // counters per digit position
constexpr int RS_MAX_PASSES = 4;            // 31-bit keys: four 8-bit digits
// single-sweep pass: 16 waves (one thread per counter), OS_ITEMS items per lane
constexpr int OS_WAVES = 16;
constexpr int OS_THREADS = 64 * OS_WAVES;
#ifndef CSR_OS_ITEMS
#define CSR_OS_ITEMS 8
#endif
#ifndef CSR_OS_WINDOW
#define CSR_OS_WINDOW 8
#endif
constexpr int OS_ITEMS = CSR_OS_ITEMS, OS_TILE = OS_THREADS * OS_ITEMS;
static_assert(OS_THREADS == RS_RADIX, "one look-back thread per counter");

__device__ __forceinline__ uint32_t clamp_key(int32_t k, int32_t n) {
  return k < 0 ? 0u : (k >= n ? (uint32_t)(n - 1) : (uint32_t)k);
}

// The two sorts of one CSR build (by destination, by source) run side by
// side: blockIdx.y selects the sort, and each sort has its own slice of the
// scratch buffers.  Items travel between passes as (key, edge id) pairs in
// one 8-byte word: a tile's run of one digit is then twice as many bytes
// of contiguous output as with separate key and id arrays, which matters for
// the scattered stores (runs from several workgroups share a cache line).
struct SortSet {
  const int32_t *keys_i32[2];   // pass 0: raw indices (clamped here), id = index
  const uint2 *in[2];           // later passes
  uint2 *out[2];
};

// Digit totals of every pass at once (keys only depend on the input, not on
// the order an earlier pass leaves them in): totals[y][p][d] = number of keys
// of sort y whose digit p is d.  Each thread counts HS_ITEMS consecutive keys
// and adds runs of equal digits with one LDS atomic (edge lists often hold
// runs of equal node ids, whose high digits would otherwise all hit one LDS
// word); four LDS copies of the histogram spread the rest; per-block sums go
// to the totals with one integer atomic per nonzero digit.
constexpr int HS_THREADS = 1024, HS_ITEMS = 16, HS_TILE = HS_THREADS * HS_ITEMS, HS_COPIES = 4;

__global__ __launch_bounds__(HS_THREADS) void rs_hist(SortSet S, int32_t n, int32_t n_nodes,
                                                      int passes, int bits, uint32_t *totals) {
  __shared__ uint32_t h[HS_COPIES][RS_MAX_PASSES][RS_RADIX];
  const int y = blockIdx.y, cp = (threadIdx.x >> 6) & (HS_COPIES - 1);
  for (int i = threadIdx.x; i < HS_COPIES * RS_MAX_PASSES * RS_RADIX; i += HS_THREADS)
    (&h[0][0][0])[i] = 0;
  // Threads count 16 keys from a 16-byte boundary on (int4 loads); the
  // f < 4 keys before the first boundary are counted by thread 0 of block 0.
  const int32_t *src = S.keys_i32[y];
  const int f = (int)(((16u - ((uint32_t)(uintptr_t)src & 15u)) & 15u) >> 2);
  const int64_t i0 = f + (int64_t)blockIdx.x * HS_TILE + (int64_t)threadIdx.x * HS_ITEMS;
  const int nv = (int)(n - i0 < 0 ? 0 : (n - i0 < HS_ITEMS ? n - i0 : HS_ITEMS));
  uint32_t k[HS_ITEMS];
  if (nv == HS_ITEMS) {
#pragma unroll
    for (int q = 0; q < HS_ITEMS / 4; ++q) {
      const int4 v = *(const int4 *)(src + i0 + 4 * q);
      k[4 * q] = clamp_key(v.x, n_nodes);
      k[4 * q + 1] = clamp_key(v.y, n_nodes);
      k[4 * q + 2] = clamp_key(v.z, n_nodes);
      k[4 * q + 3] = clamp_key(v.w, n_nodes);
    }
  } else {
#pragma unroll
    for (int it = 0; it < HS_ITEMS; ++it) k[it] = it < nv ? clamp_key(src[i0 + it], n_nodes) : 0u;
  }
  __syncthreads();
  const uint32_t mask = (1u << bits) - 1u;
  if (nv > 0) {
    for (int p = 0; p < passes; ++p) {
      const int sh = bits * p;
      uint32_t cur = (k[0] >> sh) & mask, c = 1;
#pragma unroll
      for (int it = 1; it < HS_ITEMS; ++it) {
        if (it < nv) {
          const uint32_t d = (k[it] >> sh) & mask;
          if (d == cur) {
            ++c;
          } else {
            atomicAdd(&h[cp][p][cur], c);
            cur = d;
            c = 1;
          }
        }
      }
      atomicAdd(&h[cp][p][cur], c);
    }
  }
  if (blockIdx.x == 0 && threadIdx.x == 0)
    for (int i = 0; i < f && i < n; ++i) {
      const uint32_t kk = clamp_key(src[i], n_nodes);
      for (int p = 0; p < passes; ++p) atomicAdd(&h[cp][p][(kk >> (bits * p)) & mask], 1u);
    }
  __syncthreads();
  if (threadIdx.x <= mask)
    for (int p = 0; p < passes; ++p) {
      uint32_t c = 0;
#pragma unroll
      for (int i = 0; i < HS_COPIES; ++i) c += h[i][p][threadIdx.x];
      if (c) atomicAdd(&totals[(y * RS_MAX_PASSES + p) * RS_RADIX + threadIdx.x], c);
    }
}

// One pass of the stable LSD sort in a single launch.  Tile numbers are taken
// in launch order from a counter, so every tile a workgroup waits for belongs
// to a workgroup that is already running.  Per digit, a tile publishes its
// own count (AGG), then adds up its predecessors' published words backwards
// until one carries an inclusive prefix (INC), and publishes its own
// inclusive prefix.  Those words are 32-bit: the flag in the top two bits,
// the count below (items per build < 2^30), zeroed before the first pass.
// The look-back reads OS_WINDOW predecessors per round trip.  The wait is
// bounded; past the bound (never reached while every workgroup progresses)
// the pass records a failure in err and goes on.
struct OneSweep {
  uint32_t *status;         // [passes][2][ntiles][RS_RADIX]
  const uint32_t *totals;   // [2][RS_MAX_PASSES][RS_RADIX]
  uint32_t *ctr;            // [2][RS_MAX_PASSES] tile counters
  uint32_t *err;
  // last pass, source sort (y = 1), when eis is set: the edges in source
  // order (eis[0][p] = source, eis[1][p] = destination, clamped) and the
  // inverse of that order (inv[j] = p)
  const int32_t *dst_raw;
  int32_t *eis, *inv;
};
constexpr uint32_t RS_AGG = 1u << 30, RS_INC = 2u << 30, RS_COUNT = RS_AGG - 1u;
constexpr int OS_WINDOW = CSR_OS_WINDOW;

__global__ __launch_bounds__(OS_THREADS) void rs_onesweep(SortSet S, OneSweep O, int32_t n,
                                                          int32_t n_nodes, int pass, int bits,
                                                          int32_t ntiles, int last) {
  __shared__ uint32_t cnt[OS_WAVES][RS_RADIX];  // per-wave digit counts, then bases
  __shared__ uint32_t wsum[OS_WAVES];
  __shared__ int32_t tile_sh;
  const int y = blockIdx.y;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int shift = bits * pass;
  const uint32_t mask = (1u << bits) - 1u;
  if (tid == 0) tile_sh = (int32_t)atomicAdd(&O.ctr[y * RS_MAX_PASSES + pass], 1u);
  for (int i = tid; i < OS_WAVES * RS_RADIX; i += OS_THREADS) (&cnt[0][0])[i] = 0;
  // Exclusive prefix of the digit totals: thread d holds digit d; a scan in
  // each wave, then the sums of the waves before.
  const uint32_t dtot = (uint32_t)tid <= mask ? O.totals[(y * RS_MAX_PASSES + pass) * RS_RADIX + tid]
                                               : 0u;
  uint32_t dincl = dtot;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const uint32_t u = __shfl_up(dincl, off);
    if (lane >= off) dincl += u;
  }
  if (lane == 63) wsum[w] = dincl;
  __syncthreads();
  const int32_t tile = tile_sh;
  for (int i = 0; i < w; ++i) dincl += wsum[i];
  const uint32_t digit_base = dincl - dtot;

  // Stable ranks within the tile: (wave, round, lane) is item order.
  const int64_t tile0 = (int64_t)tile * OS_TILE + (int64_t)w * 64 * OS_ITEMS;
  const uint64_t lt = (1ull << lane) - 1ull;
  uint32_t key[OS_ITEMS], val[OS_ITEMS], pre[OS_ITEMS];
#pragma unroll
  for (int it = 0; it < OS_ITEMS; ++it) {
    const int64_t i = tile0 + (int64_t)it * 64 + lane;
    uint32_t k = 0, v = 0;
    if (i < n) {
      if (S.keys_i32[y]) {
        k = clamp_key(S.keys_i32[y][i], n_nodes);
        v = (uint32_t)i;
      } else {
        const uint2 q = S.in[y][i];
        k = q.x;
        v = q.y;
      }
    }
    key[it] = k;
    val[it] = v;
  }
  // The last source-sort pass also writes each edge's destination in source
  // order; its gather is issued here, ahead of the ranking, so that its
  // latency is hidden (and no wait for it queues behind the scatter stores).
  const bool order = last && y == 1 && O.eis;
  uint32_t dst[OS_ITEMS];
#pragma unroll
  for (int it = 0; it < OS_ITEMS; ++it) {
    dst[it] = 0;
    if (order && tile0 + (int64_t)it * 64 + lane < n)
      dst[it] = clamp_key(O.dst_raw[val[it]], n_nodes);
  }
#pragma unroll
  for (int it = 0; it < OS_ITEMS; ++it) {
    const bool ok = tile0 + (int64_t)it * 64 + lane < n;
    const uint32_t d = (key[it] >> shift) & mask;
    // Lanes of this round holding the same digit: bit l of x is set when
    // lane l differs from this lane in some bit of the digit (one ballot per
    // bit; bits above the digit width are zero everywhere and change
    // nothing).
    uint32_t xl = 0, xh = 0;
#pragma unroll
    for (int b = 0; b < RS_MAX_BITS; ++b) {
      const uint32_t ext = (uint32_t)((int32_t)(d << (31 - b)) >> 31);  // 0 or all ones
      const uint64_t bal = __ballot(ext != 0u);
      xl |= (uint32_t)bal ^ ext;
      xh |= (uint32_t)(bal >> 32) ^ ext;
    }
    const uint64_t m = ~(((uint64_t)xh << 32) | xl) & __ballot(ok);
    uint32_t before = 0;
    if (ok) before = cnt[w][d];
    pre[it] = before + (uint32_t)__popcll(m & lt);
    // The lowest lane of each digit group advances the wave's counter; all
    // lanes read the counter above before any lane writes it.
    if (ok && (m & lt) == 0) cnt[w][d] = before + (uint32_t)__popcll(m);
  }
  __syncthreads();

  // Look-back over the earlier tiles, thread d for digit d; then the
  // per-wave bases replace the counts.
  if ((uint32_t)tid <= mask) {
    uint32_t local = 0;
#pragma unroll
    for (int i = 0; i < OS_WAVES; ++i) local += cnt[i][tid];
    uint32_t *st = O.status + ((int64_t)(pass * 2 + y) * ntiles) * RS_RADIX + tid;
    uint32_t excl = 0;
    if (tile == 0) {
      __hip_atomic_store(st, RS_INC | local, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    } else {
      __hip_atomic_store(st + (int64_t)tile * RS_RADIX, RS_AGG | local, __ATOMIC_RELAXED,
                         __HIP_MEMORY_SCOPE_AGENT);
      int64_t j = tile - 1;  // the nearest predecessor not yet added
      uint32_t spins = 0;
      for (;;) {
        uint32_t v[OS_WINDOW];
#pragma unroll
        for (int k = 0; k < OS_WINDOW; ++k) {
          const int64_t t = j - k < 0 ? 0 : j - k;
          v[k] = __hip_atomic_load(st + t * RS_RADIX, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
        // Add words from the nearest one back, up to the first that is not
        // published yet or through the first inclusive one.  Tile 0 always
        // publishes an inclusive word, so the walk never passes it.
        bool live = true, done = false;
        int used = 0;
#pragma unroll
        for (int k = 0; k < OS_WINDOW; ++k) {
          const uint32_t f = v[k] & (RS_AGG | RS_INC);
          if (live) {
            if (f == 0) {
              live = false;
            } else {
              excl += v[k] & RS_COUNT;
              ++used;
              if (f & RS_INC) {
                live = false;
                done = true;
              }
            }
          }
        }
        if (done) break;
        j -= used;
        if (used == 0) {
          if (++spins > (1u << 20)) {
            atomicOr(O.err, 1u);
            break;
          }
          __builtin_amdgcn_s_sleep(1);
        } else {
          spins = 0;
        }
      }
      __hip_atomic_store(st + (int64_t)tile * RS_RADIX, RS_INC | (excl + local), __ATOMIC_RELAXED,
                         __HIP_MEMORY_SCOPE_AGENT);
    }
    uint32_t run = digit_base + excl;
#pragma unroll
    for (int i = 0; i < OS_WAVES; ++i) {
      const uint32_t c = cnt[i][tid];
      cnt[i][tid] = run;
      run += c;
    }
  }
  __syncthreads();
#pragma unroll
  for (int it = 0; it < OS_ITEMS; ++it) {
    const int64_t i = tile0 + (int64_t)it * 64 + lane;
    if (i < n) {
      const uint32_t d = (key[it] >> shift) & mask;
      const uint32_t pos = cnt[w][d] + pre[it];
      if (pos < (uint32_t)n) {  // always true when the ranks are consistent
        S.out[y][pos] = make_uint2(key[it], val[it]);
        if (order) {
          O.eis[pos] = (int32_t)key[it];
          O.eis[n + pos] = (int32_t)dst[it];
          O.inv[val[it]] = (int32_t)pos;
        }
      }
    }
  }
}

// row_ptr[v] = number of sorted keys < v, v in [0, n_nodes], for both sorts:
// sorted position i owns row_ptr[v] = i for k[i-1] < v <= k[i] (k[-1] = -1,
// k[n] = n_nodes), ranges that cover [0, n_nodes] once.  Nodes without edges
// make long ranges (a whole layer of a detector graph has no out-edges), so a
// block writes the ranges of its FIN_POS positions together: entry e of the
// block's concatenated ranges goes to the position whose prefix of range
// lengths brackets e (a binary search in LDS, skipped while e stays in the
// range of the thread's previous entry).  With q_in set, also the in-CSR
// over the source order: q_in[k] = inv[perm_in[k]].  The permutations
// themselves are copied out of the sorted pairs here, with coalesced stores.
constexpr int FIN_THREADS = 1024, FIN_PER = 4, FIN_POS = FIN_THREADS * FIN_PER;

struct CsrOut {
  const uint2 *sorted[2];
  int32_t *row_ptr[2];
  int32_t *perm[2];
  const int32_t *inv;
  int32_t *q_in;
};

__global__ __launch_bounds__(FIN_THREADS) void csr_finish(CsrOut O, int32_t n, int32_t n_nodes) {
  __shared__ uint32_t incl[FIN_POS];  // inclusive prefix of range lengths
  __shared__ uint32_t first[FIN_POS];
  __shared__ uint32_t wsum[FIN_THREADS / 64];
  const int y = blockIdx.y, tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int64_t i0 = (int64_t)blockIdx.x * FIN_POS, ib = i0 + (int64_t)tid * FIN_PER;
  const uint2 *srt = O.sorted[y];
  uint32_t kv[FIN_PER + 1];  // keys at ib - 1 .. ib + FIN_PER - 1 where in range
  kv[0] = ib >= 1 && ib - 1 < n ? srt[ib - 1].x : 0u;
#pragma unroll
  for (int j = 0; j < FIN_PER; ++j) {
    kv[j + 1] = 0u;
    if (ib + j < n) {
      const uint2 q = srt[ib + j];
      kv[j + 1] = q.x;
      O.perm[y][ib + j] = (int32_t)q.y;
    }
  }
  uint32_t lo[FIN_PER], len[FIN_PER], sum = 0;
#pragma unroll
  for (int j = 0; j < FIN_PER; ++j) {
    const int64_t i = ib + j;
    lo[j] = 0;
    len[j] = 0;
    if (i <= n) {
      lo[j] = i == 0 ? 0u : kv[j] + 1u;
      const uint32_t hi = i == n ? (uint32_t)n_nodes : kv[j + 1];
      len[j] = hi + 1u - lo[j];  // k is sorted, so hi + 1 >= lo
    }
    sum += len[j];
  }
  uint32_t s = sum;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const uint32_t u = __shfl_up(s, off);
    if (lane >= off) s += u;
  }
  if (lane == 63) wsum[w] = s;
  __syncthreads();
  for (int j = 0; j < w; ++j) s += wsum[j];
  s -= sum;
#pragma unroll
  for (int j = 0; j < FIN_PER; ++j) {
    s += len[j];
    incl[tid * FIN_PER + j] = s;
    first[tid * FIN_PER + j] = lo[j];
  }
  __syncthreads();
  const uint32_t total = incl[FIN_POS - 1];
  int32_t *rp = O.row_ptr[y];
  int a = 0;  // smallest t with incl[t] > e; e only grows
  for (uint32_t e = tid; e < total; e += FIN_THREADS) {
    if (incl[a] <= e) {
      int lo2 = a + 1, hi2 = FIN_POS - 1;
      while (lo2 < hi2) {
        const int mid = (lo2 + hi2) >> 1;
        if (incl[mid] > e) hi2 = mid;
        else lo2 = mid + 1;
      }
      a = lo2;
    }
    const uint32_t before = a == 0 ? 0u : incl[a - 1];
    rp[first[a] + (e - before)] = (int32_t)(i0 + a);
  }
  // q_in: the blocks of both sorts share the block's positions
  if (O.q_in)
#pragma unroll
    for (int j = 0; j < FIN_PER / 2; ++j) {
      const int64_t i = i0 + (int64_t)(2 * j + y) * FIN_THREADS + tid;
      if (i < n) O.q_in[i] = O.inv[O.sorted[0][i].y];
    }
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

namespace {

struct Digits {
  int passes, bits;
};

// Digit layout for keys in [0, n_nodes): the fewest passes of at most
// RS_MAX_BITS bits, the bits spread evenly over them; at least one pass of
// one bit so that the sorted arrays are always written.
Digits csr_digits(int64_t n_nodes) {
  int b = 0;
  while (b < 31 && ((int64_t)1 << b) < n_nodes) ++b;
  if (b == 0) b = 1;
  const int passes = (b + RS_MAX_BITS - 1) / RS_MAX_BITS;
  return {passes, (b + passes - 1) / passes};
}

int64_t csr_tiles(int64_t n_edges) { return (n_edges + OS_TILE - 1) / OS_TILE; }

// Scratch words after the look-back status: digit totals, tile counters and
// the error word.
constexpr size_t CSR_TAIL_WORDS = (size_t)2 * RS_MAX_PASSES * RS_RADIX + 2 * RS_MAX_PASSES + 8;

size_t csr_status_words(int64_t n_edges, int64_t n_nodes) {
  return (size_t)csr_digits(n_nodes).passes * 2 * RS_RADIX * (size_t)csr_tiles(n_edges);
}

}  // namespace

size_t csr_scratch_bytes(int64_t n_edges, int64_t n_nodes) {
  return (csr_status_words(n_edges, n_nodes) + CSR_TAIL_WORDS) * 4;
}

uint32_t *csr_err_word(const CsrScratch &s, int64_t n_edges, int64_t n_nodes) {
  return s.status + csr_status_words(n_edges, n_nodes) + 2 * RS_MAX_PASSES * RS_RADIX +
         2 * RS_MAX_PASSES;
}

hipError_t build_csr(const int32_t *edge_index, int32_t n, int32_t n_nodes, int32_t *row_ptr_in,
                     int32_t *perm_in, int32_t *row_ptr_out, int32_t *perm_out,
                     const CsrScratch &s, int32_t *eis, int32_t *inv, int32_t *q_in,
                     hipStream_t stream) {
  if (n < 0 || n >= CSR_MAX_ITEMS || n_nodes < 0) return hipErrorInvalidValue;
  const Digits dg = csr_digits(n_nodes);
  const int32_t ntiles = (int32_t)csr_tiles(n);
  // look-back words, digit totals, tile counters and the error word: one
  // region, zeroed by a fill kernel (also under stream capture)
  const size_t sw = csr_status_words(n, n_nodes);
  const int64_t words = (int64_t)(sw + CSR_TAIL_WORDS);
  if (const hipError_t e =
          launch(fill_i32, blocks_for(words, 256), 256, 0, stream, (int32_t *)s.status, words, 0))
    return e;
  uint32_t *totals = s.status + sw;

  SortSet S{};
  if (n > 0) {
    // Sort 0: keys = destinations (row 1), sort 1: keys = sources (row 0).
    uint2 *pa[2] = {s.pairs_a, s.pairs_a + n}, *pb[2] = {s.pairs_b, s.pairs_b + n};
    OneSweep O{};
    O.status = s.status;
    O.totals = totals;
    O.ctr = totals + 2 * RS_MAX_PASSES * RS_RADIX;
    O.err = O.ctr + 2 * RS_MAX_PASSES;
    O.dst_raw = edge_index + n;
    O.eis = eis;
    O.inv = inv;
    S.keys_i32[0] = edge_index + n;
    S.keys_i32[1] = edge_index;
    if (const hipError_t e = launch(rs_hist, dim3(blocks_for(n, HS_TILE), 2), HS_THREADS, 0,
                                    stream, S, n, n_nodes, dg.passes, dg.bits, totals))
      return e;
    for (int p = 0; p < dg.passes; ++p) {
      const bool last = p == dg.passes - 1;
      for (int y = 0; y < 2; ++y) S.out[y] = (p & 1) ? pb[y] : pa[y];
      if (const hipError_t e = launch(rs_onesweep, dim3(ntiles, 2), OS_THREADS, 0, stream, S, O,
                                      n, n_nodes, p, dg.bits, ntiles, last ? 1 : 0))
        return e;
      for (int y = 0; y < 2; ++y) {
        S.keys_i32[y] = nullptr;
        S.in[y] = S.out[y];
      }
    }
  }
  CsrOut C{};
  for (int y = 0; y < 2; ++y) C.sorted[y] = S.in[y];  // not read when n == 0
  C.row_ptr[0] = row_ptr_in;
  C.row_ptr[1] = row_ptr_out;
  C.perm[0] = perm_in;
  C.perm[1] = perm_out;
  C.inv = inv;
  C.q_in = eis ? q_in : nullptr;
  return launch(csr_finish, dim3(blocks_for((int64_t)n + 1, FIN_POS), 2), FIN_THREADS, 0, stream,
                C, n, n_nodes);
}

hipError_t launch_validate(const int32_t *edge_index, int64_t n_edges, int32_t n_nodes,
                           int32_t *flag, hipStream_t stream) {
  const int64_t n = 2 * n_edges;
  return launch(validate_idx, blocks_for(n, 256), 256, 0, stream, edge_index, n, n_nodes, flag);
}

hipError_t launch_fill_i32(int32_t *p, int64_t n, int32_t v, hipStream_t stream) {
  if (n <= 0) return hipSuccess;
  return launch(fill_i32, blocks_for(n, 256), 256, 0, stream, p, n, v);
}

hipError_t launch_scatter_rows(Act act, const void *src, const int32_t *idx, float *dst,
                               int64_t rows, int H, hipStream_t stream) {
  const int64_t n = rows * H;
  if (n <= 0) return hipSuccess;
  const unsigned nb = (unsigned)blocks_for(n, 256);
  if (act == Act::F32)
    return launch(scatter_rows_k<float>, nb, 256, 0, stream, (const float *)src, idx, dst, rows, H);
  if (act == Act::BF16)
    return launch(scatter_rows_k<__bf16>, nb, 256, 0, stream, (const __bf16 *)src, idx, dst, rows,
                  H);
  return launch(scatter_rows_k<_Float16>, nb, 256, 0, stream, (const _Float16 *)src, idx, dst,
                rows, H);
}

hipError_t launch_bf16_to_f32(const void *in, float *out, int64_t n, hipStream_t stream) {
  if (n <= 0) return hipSuccess;
  return launch(bf16_to_f32, blocks_for(n, 256), 256, 0, stream, (const __bf16 *)in, out, n);
}

}  // namespace gnn
