// Deterministic CSR segmented sums: message aggregation of the interaction
// network (paper section 2.1), agg_in(v) = sum of e_j over edges into v and
// agg_out(v) = sum over edges out of v.
//
// A group of H/4 (fp32) or H/8 (bf16) lanes owns one (node, direction) task
// and walks its CSR row in ascending position, each lane adding one 16-byte
// slice of every message row: each message row is read as one contiguous,
// fully coalesced 256/512-byte chunk, sums run in a fixed order (bitwise
// reproducible, no float atomics), and empty rows are written as zeros.
// The row ids of a task come in with one load and four rows are requested
// before any is added, so a typical node (a few messages) costs three
// dependent round trips: row bounds, row ids, rows.  The gather of 512-byte
// rows at scattered positions is bound by HBM at a lower rate than a
// streaming read.  Message rows are loaded and aggregates stored with the
// nontemporal hint (each row is touched once per launch): on the full
// event that took the fp32 launch from 0.158 to 0.138 ms, moving the same
// bytes.  Accumulation is fp32 in both storage modes.  Rows
// longer than LONG_ROW messages use Neumaier's compensated summation: a hub
// node can receive 10^5 messages, where a plain fp32 running sum drifts by
// ~10^-4 relative, while the compensated sum stays within a few ulps of the
// exact sum at any length.  Either way the order is fixed.
#include "gnn_internal.h"

namespace gnn {
namespace {

typedef float f4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf8 __attribute__((ext_vector_type(8)));

// Block sizes: small blocks schedule the short, uneven node tasks best
// (full event, against 256 threads: fp32 0.1248 -> 0.1236 ms with 128,
// bf16 0.0745 -> 0.0694 ms with 64).
constexpr int THREADS_F32 = 128;
constexpr int THREADS_BF16 = 64;

// Loads and stores of rows that this kernel touches once (nontemporal).
template <typename T>
__device__ __forceinline__ T ld_once(const T *p) {
  return __builtin_nontemporal_load(p);
}
template <typename T>
__device__ __forceinline__ void st_once(T *p, T v) {
  __builtin_nontemporal_store(v, p);
}
constexpr int LONG_ROW = 32;

// One step of Neumaier summation: s + c carries the running sum.  With
// COMP false it is a plain sum (c stays 0).
template <bool COMP>
__device__ __forceinline__ void nsum(float &s, float &c, float x) {
  if constexpr (COMP) {
    const float t = s + x;
    c += fabsf(s) >= fabsf(x) ? (s - t) + x : (x - t) + s;
    s = t;
  } else {
    s += x;
  }
}

// Value of x held by lane j of the calling lane's G-lane group (G divides 64).
template <int G>
__device__ __forceinline__ int32_t group_lane(int32_t x, int j) {
  const int src = ((int)threadIdx.x & 63 & ~(G - 1)) + j;
  return __builtin_amdgcn_ds_bpermute(src << 2, x);
}

// Sum of the message rows at CSR positions [p, pe) into (s, c), G lanes per
// row, each lane one 16-byte slice.  The row ids of up to G positions are
// fetched with one coalesced load (lane i holds position p + i) and handed
// round the group, then B rows are requested before any of them is added,
// so a node's whole row list is in flight after two round trips rather than
// one pair of dependent loads per message.  Rows are added in ascending
// position whatever B is.  A null perm means row id = position.
template <int H, int B, bool COMP, bool IDX>
__device__ __forceinline__ void row_sum_f32(const float *__restrict__ base,
                                            const int32_t *__restrict__ perm, int32_t p,
                                            int32_t pe, int sub, float (&s)[4], float (&c)[4]) {
  constexpr int G = H / 4;
  static_assert(G % B == 0, "batch must divide the group");
  for (; p < pe; p += G) {
    const int n = min(G, pe - p);
    int32_t my = 0;
    if constexpr (IDX) my = perm[p + min(sub, n - 1)];
    for (int j = 0; j < n; j += B) {
      // Every load is issued (positions past the end repeat the last row, a
      // cache hit), so the waits before the adds count loads exactly.
      f4 r[B];
#pragma unroll
      for (int u = 0; u < B; ++u) {
        int64_t q;
        if constexpr (IDX)
          q = group_lane<G>(my, min(j + u, n - 1));
        else
          q = p + min(j + u, n - 1);
        r[u] = ld_once((const f4 *)(base + q * H));
      }
#pragma unroll
      for (int u = 0; u < B; ++u)
        if (j + u < n)
#pragma unroll
          for (int k = 0; k < 4; ++k) nsum<COMP>(s[k], c[k], r[u][k]);
    }
  }
}

template <int H, int B, bool COMP, bool IDX, typename T>
__device__ __forceinline__ void row_sum_bf16(const T *__restrict__ base,
                                             const int32_t *__restrict__ perm, int32_t p,
                                             int32_t pe, int sub, float (&s)[8], float (&c)[8]) {
  typedef T t8 __attribute__((ext_vector_type(8)));
  constexpr int G = H / 8;
  static_assert(G % B == 0, "batch must divide the group");
  for (; p < pe; p += G) {
    const int n = min(G, pe - p);
    int32_t my = 0;
    if constexpr (IDX) my = perm[p + min(sub, n - 1)];
    for (int j = 0; j < n; j += B) {
      t8 r[B];
#pragma unroll
      for (int u = 0; u < B; ++u) {
        int64_t q;
        if constexpr (IDX)
          q = group_lane<G>(my, min(j + u, n - 1));
        else
          q = p + min(j + u, n - 1);
        r[u] = ld_once((const t8 *)(base + q * H));
      }
#pragma unroll
      for (int u = 0; u < B; ++u)
        if (j + u < n)
#pragma unroll
          for (int k = 0; k < 8; ++k) nsum<COMP>(s[k], c[k], (float)r[u][k]);
    }
  }
}

template <int H, int B = 4>
__device__ __forceinline__ void row_sum_f32(const float *base, const int32_t *perm, int32_t p,
                                            int32_t pe, int sub, float (&s)[4], float (&c)[4]) {
  const bool comp = pe - p > LONG_ROW;
  if (perm) {
    if (comp) row_sum_f32<H, B, true, true>(base, perm, p, pe, sub, s, c);
    else row_sum_f32<H, B, false, true>(base, perm, p, pe, sub, s, c);
  } else {
    if (comp) row_sum_f32<H, B, true, false>(base, perm, p, pe, sub, s, c);
    else row_sum_f32<H, B, false, false>(base, perm, p, pe, sub, s, c);
  }
}

template <int H, int B = 4, typename T>
__device__ __forceinline__ void row_sum_bf16(const T *base, const int32_t *perm, int32_t p,
                                             int32_t pe, int sub, float (&s)[8], float (&c)[8]) {
  const bool comp = pe - p > LONG_ROW;
  if (perm) {
    if (comp) row_sum_bf16<H, B, true, true, T>(base, perm, p, pe, sub, s, c);
    else row_sum_bf16<H, B, false, true, T>(base, perm, p, pe, sub, s, c);
  } else {
    if (comp) row_sum_bf16<H, B, true, false, T>(base, perm, p, pe, sub, s, c);
    else row_sum_bf16<H, B, false, false, T>(base, perm, p, pe, sub, s, c);
  }
}

template <int H>
__global__ __launch_bounds__(THREADS_F32) void segsum_f32(
    const float *__restrict__ e, const int32_t *__restrict__ rp_in,
    const int32_t *__restrict__ perm_in, const int32_t *__restrict__ rp_out,
    const int32_t *__restrict__ perm_out, float *__restrict__ agg_in,
    float *__restrict__ agg_out, int32_t n_nodes) {
  constexpr int LPR = H / 4;
  constexpr int TPB = THREADS_F32 / LPR;
  const int sub = threadIdx.x % LPR;
  const int64_t task = (int64_t)blockIdx.x * TPB + threadIdx.x / LPR;
  if (task >= 2 * (int64_t)n_nodes) return;
  const bool out = task >= n_nodes;
  const int64_t v = out ? task - n_nodes : task;
  const int32_t *rp = out ? rp_out : rp_in;
  const int32_t *perm = out ? perm_out : perm_in;
  float *dst = out ? agg_out : agg_in;
  int32_t p = rp[v];
  const int32_t pe = rp[v + 1];
  const float *base = e + 4 * sub;
  float s[4] = {0.f, 0.f, 0.f, 0.f}, c[4] = {0.f, 0.f, 0.f, 0.f};
  row_sum_f32<H>(base, perm, p, pe, sub, s, c);
  const f4 res = {s[0] + c[0], s[1] + c[1], s[2] + c[2], s[3] + c[3]};
  st_once((f4 *)(dst + v * H + 4 * sub), res);
}

// After a fused edge update (rows in source order), one task per node v:
// agg_in[v] as in segsum_f32; then agg_out[v] is completed when v's run of
// rows spans several 32-row units, from the pieces the edge update left
// (the tail piece of the first unit, the whole middle units, the head piece
// of the last unit, added in that order), zeroed when v has no out-edges,
// and otherwise left as the edge update wrote it.
template <int H>
__global__ __launch_bounds__(THREADS_F32) void segsum_fused_f32(
    const float *__restrict__ e, const int32_t *__restrict__ rp_in,
    const int32_t *__restrict__ perm_in, const int32_t *__restrict__ rp_out,
    const float *__restrict__ part, float *__restrict__ agg_in, float *__restrict__ agg_out,
    int32_t n_nodes) {
  constexpr int LPR = H / 4;
  constexpr int TPB = THREADS_F32 / LPR;
  const int sub = threadIdx.x % LPR;
  const int64_t v = (int64_t)blockIdx.x * TPB + threadIdx.x / LPR;
  if (v >= n_nodes) return;
  const int32_t a = rp_out[v], b = rp_out[v + 1];
  const int32_t pi = rp_in[v], pie = rp_in[v + 1];
  const int32_t u0 = a >> 5, u1 = (b - 1) >> 5;
  const bool spans = a < b && u1 > u0;
  const float *pc = part + 4 * sub;
  {
    float s[4] = {0.f, 0.f, 0.f, 0.f}, c[4] = {0.f, 0.f, 0.f, 0.f};
    row_sum_f32<H>(e + 4 * sub, perm_in, pi, pie, sub, s, c);
    st_once((f4 *)(agg_in + v * H + 4 * sub), f4{s[0] + c[0], s[1] + c[1], s[2] + c[2], s[3] + c[3]});
  }
  if (a < b && !spans) return;  // written by the edge update
  // Pieces only for the runs that span units (about one node in ten):
  // requesting two for every node, to overlap them with the row gathers,
  // cost 2% (fp32) and 13% (bf16) in extra piece traffic.
  float s[4] = {0.f, 0.f, 0.f, 0.f}, c[4] = {0.f, 0.f, 0.f, 0.f};
  if (spans) {
    const f4 t0 = *(const f4 *)(pc + (int64_t)(2 * u0 + 1) * H);
    const f4 t1 = *(const f4 *)(pc + (int64_t)(2 * u0 + 2) * H);
#pragma unroll
    for (int k = 0; k < 4; ++k) s[k] = t0[k];
    if (u1 - u0 > LONG_ROW) {
#pragma unroll
      for (int k = 0; k < 4; ++k) nsum<true>(s[k], c[k], t1[k]);
      for (int32_t u = u0 + 2; u <= u1; ++u) {
        const f4 r = *(const f4 *)(pc + (int64_t)(2 * u) * H);
#pragma unroll
        for (int k = 0; k < 4; ++k) nsum<true>(s[k], c[k], r[k]);
      }
    } else {
#pragma unroll
      for (int k = 0; k < 4; ++k) s[k] += t1[k];
      for (int32_t u = u0 + 2; u <= u1; ++u) {
        const f4 r = *(const f4 *)(pc + (int64_t)(2 * u) * H);
#pragma unroll
        for (int k = 0; k < 4; ++k) s[k] += r[k];
      }
    }
  }
  st_once((f4 *)(agg_out + v * H + 4 * sub), f4{s[0] + c[0], s[1] + c[1], s[2] + c[2], s[3] + c[3]});
}

// The same for 16-bit rows and bf16 aggregates (H/8 lanes per node, 8
// features each); the pieces are fp32, the sums fp32.  ET is the row type:
// bf16, or fp16 for the edge rows of the bf16 model with fp16 weights.
template <int H, typename ET>
__global__ __launch_bounds__(THREADS_BF16) void segsum_fused_bf16(
    const ET *__restrict__ e, const int32_t *__restrict__ rp_in,
    const int32_t *__restrict__ perm_in, const int32_t *__restrict__ rp_out,
    const float *__restrict__ part, __bf16 *__restrict__ agg_in, __bf16 *__restrict__ agg_out,
    int32_t n_nodes) {
  constexpr int LPR = H / 8;
  constexpr int TPB = THREADS_BF16 / LPR;
  const int sub = threadIdx.x % LPR;
  const int64_t v = (int64_t)blockIdx.x * TPB + threadIdx.x / LPR;
  if (v >= n_nodes) return;
  const int32_t a = rp_out[v], b = rp_out[v + 1];
  const int32_t pi = rp_in[v], pie = rp_in[v + 1];
  const int32_t u0 = a >> 5, u1 = (b - 1) >> 5;
  const bool spans = a < b && u1 > u0;
  const float *pc = part + 8 * sub;
  auto piece = [&](int64_t slot, float (&r)[8]) {
    const f4 lo = *(const f4 *)(pc + slot * H), hi = *(const f4 *)(pc + slot * H + 4);
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      r[k] = lo[k];
      r[4 + k] = hi[k];
    }
  };
  {
    float s[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    float c[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    row_sum_bf16<H>(e + 8 * sub, perm_in, pi, pie, sub, s, c);
    bf8 o;
#pragma unroll
    for (int k = 0; k < 8; ++k) o[k] = (__bf16)(s[k] + c[k]);
    st_once((bf8 *)(agg_in + v * H + 8 * sub), o);
  }
  if (a < b && !spans) return;  // written by the edge update
  float s[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  float c[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  if (spans) {  // pieces only for spanning runs, as in the fp32 kernel
    float t0[8], t1[8];
    piece(2 * (int64_t)u0 + 1, t0);
    piece(2 * (int64_t)u0 + 2, t1);
    const bool comp = u1 - u0 > LONG_ROW;
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      s[k] = t0[k];
      if (comp)
        nsum<true>(s[k], c[k], t1[k]);
      else
        s[k] += t1[k];
    }
    for (int32_t u = u0 + 2; u <= u1; ++u) {
      float r[8];
      piece(2 * (int64_t)u, r);
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        if (comp)
          nsum<true>(s[k], c[k], r[k]);
        else
          s[k] += r[k];
      }
    }
  }
  bf8 o;
#pragma unroll
  for (int k = 0; k < 8; ++k) o[k] = (__bf16)(s[k] + c[k]);
  st_once((bf8 *)(agg_out + v * H + 8 * sub), o);
}

template <int H>
__global__ __launch_bounds__(THREADS_BF16) void segsum_bf16(
    const __bf16 *__restrict__ e, const int32_t *__restrict__ rp_in,
    const int32_t *__restrict__ perm_in, const int32_t *__restrict__ rp_out,
    const int32_t *__restrict__ perm_out, __bf16 *__restrict__ agg_in,
    __bf16 *__restrict__ agg_out, int32_t n_nodes) {
  constexpr int LPR = H / 8;
  constexpr int TPB = THREADS_BF16 / LPR;
  const int sub = threadIdx.x % LPR;
  const int64_t task = (int64_t)blockIdx.x * TPB + threadIdx.x / LPR;
  if (task >= 2 * (int64_t)n_nodes) return;
  const bool out = task >= n_nodes;
  const int64_t v = out ? task - n_nodes : task;
  const int32_t *rp = out ? rp_out : rp_in;
  const int32_t *perm = out ? perm_out : perm_in;
  __bf16 *dst = out ? agg_out : agg_in;
  int32_t p = rp[v];
  const int32_t pe = rp[v + 1];
  const __bf16 *base = e + 8 * sub;
  float s[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  float c[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  row_sum_bf16<H>(base, perm, p, pe, sub, s, c);
  bf8 o;
#pragma unroll
  for (int k = 0; k < 8; ++k) o[k] = (__bf16)(s[k] + c[k]);
  st_once((bf8 *)(dst + v * H + 8 * sub), o);
}

template <int H>
hipError_t launch_h(Act act, const void *e, const int32_t *rp_in, const int32_t *perm_in,
                    const int32_t *rp_out, const int32_t *perm_out, void *agg_in, void *agg_out,
                    int32_t n_nodes, hipStream_t stream) {
  const int lpr = act == Act::F32 ? H / 4 : H / 8;
  const int threads = act == Act::F32 ? THREADS_F32 : THREADS_BF16;
  const int tpb = threads / lpr;
  const int64_t tasks = 2 * (int64_t)n_nodes;
  const unsigned blocks = (unsigned)((tasks + tpb - 1) / tpb);
  if (blocks == 0) return hipSuccess;
  if (act == Act::F32)
    return launch(segsum_f32<H>, blocks, THREADS_F32, 0, stream, (const float *)e, rp_in, perm_in,
                  rp_out, perm_out, (float *)agg_in, (float *)agg_out, n_nodes);
  return launch(segsum_bf16<H>, blocks, THREADS_BF16, 0, stream, (const __bf16 *)e, rp_in, perm_in,
                rp_out, perm_out, (__bf16 *)agg_in, (__bf16 *)agg_out, n_nodes);
}

template <int H>
hipError_t launch_fused_h(Act act, const void *e, const int32_t *rp_in, const int32_t *perm_in,
                          const int32_t *rp_out, const float *part, void *agg_in, void *agg_out,
                          int32_t n_nodes, int64_t n_edges, hipStream_t stream) {
  const int tpb = act == Act::F32 ? THREADS_F32 / (H / 4) : THREADS_BF16 / (H / 8);
  const int64_t tasks = n_nodes;
  const unsigned blocks = (unsigned)((tasks + tpb - 1) / tpb);
  if (blocks == 0) return hipSuccess;
  // the pieces come from an edge update over a non-empty edge list
  if (n_edges < 1 || n_edges > INT32_MAX) return hipErrorInvalidValue;
  if (act == Act::F32)
    return launch(segsum_fused_f32<H>, blocks, THREADS_F32, 0, stream, (const float *)e, rp_in,
                  perm_in, rp_out, part, (float *)agg_in, (float *)agg_out, n_nodes);
  if (act == Act::BF16)
    return launch(segsum_fused_bf16<H, __bf16>, blocks, THREADS_BF16, 0, stream, (const __bf16 *)e,
                  rp_in, perm_in, rp_out, part, (__bf16 *)agg_in, (__bf16 *)agg_out, n_nodes);
  return launch(segsum_fused_bf16<H, _Float16>, blocks, THREADS_BF16, 0, stream,
                (const _Float16 *)e, rp_in, perm_in, rp_out, part, (__bf16 *)agg_in,
                (__bf16 *)agg_out, n_nodes);
}

}  // namespace

hipError_t launch_segsum_fused(Act act, int hidden, const void *e, const int32_t *rp_in,
                               const int32_t *perm_in, const int32_t *rp_out,
                               const float *agg_part, void *agg_in, void *agg_out,
                               int32_t n_nodes, int64_t n_edges, hipStream_t stream) {
  switch (hidden) {
    case 64: return launch_fused_h<64>(act, e, rp_in, perm_in, rp_out, agg_part, agg_in, agg_out, n_nodes, n_edges, stream);
    case 128: return launch_fused_h<128>(act, e, rp_in, perm_in, rp_out, agg_part, agg_in, agg_out, n_nodes, n_edges, stream);
  }
  return hipErrorInvalidValue;
}

hipError_t launch_segsum(Act act, int hidden, const void *e, const int32_t *rp_in,
                         const int32_t *perm_in, const int32_t *rp_out, const int32_t *perm_out,
                         void *agg_in, void *agg_out, int32_t n_nodes, hipStream_t stream) {
  switch (hidden) {
    case 64: return launch_h<64>(act, e, rp_in, perm_in, rp_out, perm_out, agg_in, agg_out, n_nodes, stream);
    case 128: return launch_h<128>(act, e, rp_in, perm_in, rp_out, perm_out, agg_in, agg_out, n_nodes, stream);
  }
  return hipErrorInvalidValue;
}

}  // namespace gnn
