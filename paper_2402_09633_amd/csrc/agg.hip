// Deterministic CSR segmented sums: message aggregation of the interaction
// network (paper section 2.1), agg_in(v) = sum of e_j over edges into v and
// agg_out(v) = sum over edges out of v.
//
// A group of H/4 (fp32) or H/8 (bf16) lanes owns one (node, direction) task
// and walks its CSR row in ascending position, each lane adding one 16-byte
// slice of every message row: each message row is read as one contiguous,
// fully coalesced 256/512-byte chunk, sums run in a fixed order (bitwise
// reproducible, no float atomics), and empty rows are written as zeros.
// Four rows are loaded before they are added to keep several HBM requests
// in flight per lane.  Accumulation is fp32 in both storage modes.  Rows
// longer than LONG_ROW messages use Neumaier's compensated summation: a hub
// node can receive 10^5 messages, where a plain fp32 running sum drifts by
// ~10^-4 relative, while the compensated sum stays within a few ulps of the
// exact sum at any length.  Either way the order is fixed.
#include "gnn_internal.h"

namespace gnn {
namespace {

typedef float f4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf8 __attribute__((ext_vector_type(8)));

constexpr int THREADS = 256;
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

// Message row of CSR position p: perm[p], or p itself for a null perm
// (rows already in CSR order).
template <bool IDX>
__device__ __forceinline__ int64_t msg_row(const int32_t *__restrict__ perm, int32_t p) {
  if constexpr (IDX)
    return perm[p];
  else
    return p;
}

template <int H, bool COMP, bool IDX>
__device__ __forceinline__ void row_sum_f32(const float *__restrict__ base,
                                            const int32_t *__restrict__ perm, int32_t p,
                                            int32_t pe, float (&s)[4], float (&c)[4]) {
  for (; p + 4 <= pe; p += 4) {
    f4 r[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) r[u] = *(const f4 *)(base + msg_row<IDX>(perm, p + u) * H);
#pragma unroll
    for (int u = 0; u < 4; ++u)
#pragma unroll
      for (int k = 0; k < 4; ++k) nsum<COMP>(s[k], c[k], r[u][k]);
  }
  for (; p < pe; ++p) {
    const f4 r = *(const f4 *)(base + msg_row<IDX>(perm, p) * H);
#pragma unroll
    for (int k = 0; k < 4; ++k) nsum<COMP>(s[k], c[k], r[k]);
  }
}

template <int H, bool COMP, bool IDX>
__device__ __forceinline__ void row_sum_bf16(const __bf16 *__restrict__ base,
                                             const int32_t *__restrict__ perm, int32_t p,
                                             int32_t pe, float (&s)[8], float (&c)[8]) {
  for (; p + 4 <= pe; p += 4) {
    bf8 r[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) r[u] = *(const bf8 *)(base + msg_row<IDX>(perm, p + u) * H);
#pragma unroll
    for (int u = 0; u < 4; ++u)
#pragma unroll
      for (int k = 0; k < 8; ++k) nsum<COMP>(s[k], c[k], (float)r[u][k]);
  }
  for (; p < pe; ++p) {
    const bf8 r = *(const bf8 *)(base + msg_row<IDX>(perm, p) * H);
#pragma unroll
    for (int k = 0; k < 8; ++k) nsum<COMP>(s[k], c[k], (float)r[k]);
  }
}

template <int H>
__device__ __forceinline__ void row_sum_f32(const float *base, const int32_t *perm, int32_t p,
                                            int32_t pe, float (&s)[4], float (&c)[4]) {
  const bool comp = pe - p > LONG_ROW;
  if (perm) {
    if (comp) row_sum_f32<H, true, true>(base, perm, p, pe, s, c);
    else row_sum_f32<H, false, true>(base, perm, p, pe, s, c);
  } else {
    if (comp) row_sum_f32<H, true, false>(base, perm, p, pe, s, c);
    else row_sum_f32<H, false, false>(base, perm, p, pe, s, c);
  }
}

template <int H>
__device__ __forceinline__ void row_sum_bf16(const __bf16 *base, const int32_t *perm, int32_t p,
                                             int32_t pe, float (&s)[8], float (&c)[8]) {
  const bool comp = pe - p > LONG_ROW;
  if (perm) {
    if (comp) row_sum_bf16<H, true, true>(base, perm, p, pe, s, c);
    else row_sum_bf16<H, false, true>(base, perm, p, pe, s, c);
  } else {
    if (comp) row_sum_bf16<H, true, false>(base, perm, p, pe, s, c);
    else row_sum_bf16<H, false, false>(base, perm, p, pe, s, c);
  }
}

template <int H>
__global__ __launch_bounds__(THREADS) void segsum_f32(
    const float *__restrict__ e, const int32_t *__restrict__ rp_in,
    const int32_t *__restrict__ perm_in, const int32_t *__restrict__ rp_out,
    const int32_t *__restrict__ perm_out, float *__restrict__ agg_in,
    float *__restrict__ agg_out, int32_t n_nodes) {
  constexpr int LPR = H / 4;
  constexpr int TPB = THREADS / LPR;
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
  row_sum_f32<H>(base, perm, p, pe, s, c);
  const f4 res = {s[0] + c[0], s[1] + c[1], s[2] + c[2], s[3] + c[3]};
  *(f4 *)(dst + v * H + 4 * sub) = res;
}

// After a fused edge update (rows in source order), one task per node v:
// agg_in[v] as in segsum_f32; then agg_out[v] is completed when v's run of
// rows spans several 32-row units, from the pieces the edge update left
// (the tail piece of the first unit, the whole middle units, the head piece
// of the last unit, added in that order), zeroed when v has no out-edges,
// and otherwise left as the edge update wrote it.
template <int H>
__global__ __launch_bounds__(THREADS) void segsum_fused_f32(
    const float *__restrict__ e, const int32_t *__restrict__ rp_in,
    const int32_t *__restrict__ perm_in, const int32_t *__restrict__ rp_out,
    const float *__restrict__ part, float *__restrict__ agg_in, float *__restrict__ agg_out,
    int32_t n_nodes) {
  constexpr int LPR = H / 4;
  constexpr int TPB = THREADS / LPR;
  const int sub = threadIdx.x % LPR;
  const int64_t v = (int64_t)blockIdx.x * TPB + threadIdx.x / LPR;
  if (v >= n_nodes) return;
  const int32_t a = rp_out[v], b = rp_out[v + 1];
  {
    float s[4] = {0.f, 0.f, 0.f, 0.f}, c[4] = {0.f, 0.f, 0.f, 0.f};
    row_sum_f32<H>(e + 4 * sub, perm_in, rp_in[v], rp_in[v + 1], s, c);
    *(f4 *)(agg_in + v * H + 4 * sub) = f4{s[0] + c[0], s[1] + c[1], s[2] + c[2], s[3] + c[3]};
  }
  const int32_t u0 = a >> 5, u1 = (b - 1) >> 5;
  if (a < b && u0 == u1) return;  // written by the edge update
  float s[4] = {0.f, 0.f, 0.f, 0.f}, c[4] = {0.f, 0.f, 0.f, 0.f};
  if (a < b) {
    const float *pc = part + 4 * sub;
    const f4 t = *(const f4 *)(pc + (int64_t)(2 * u0 + 1) * H);
#pragma unroll
    for (int k = 0; k < 4; ++k) s[k] = t[k];
    if (u1 - u0 > LONG_ROW) {
      for (int32_t u = u0 + 1; u <= u1; ++u) {
        const f4 r = *(const f4 *)(pc + (int64_t)(2 * u) * H);
#pragma unroll
        for (int k = 0; k < 4; ++k) nsum<true>(s[k], c[k], r[k]);
      }
    } else {
      for (int32_t u = u0 + 1; u <= u1; ++u) {
        const f4 r = *(const f4 *)(pc + (int64_t)(2 * u) * H);
#pragma unroll
        for (int k = 0; k < 4; ++k) s[k] += r[k];
      }
    }
  }
  *(f4 *)(agg_out + v * H + 4 * sub) = f4{s[0] + c[0], s[1] + c[1], s[2] + c[2], s[3] + c[3]};
}

// The same for bf16 rows and aggregates (H/8 lanes per node, 8 features
// each); the pieces are fp32, the sums fp32, the stored aggregates bf16.
template <int H>
__global__ __launch_bounds__(THREADS) void segsum_fused_bf16(
    const __bf16 *__restrict__ e, const int32_t *__restrict__ rp_in,
    const int32_t *__restrict__ perm_in, const int32_t *__restrict__ rp_out,
    const float *__restrict__ part, __bf16 *__restrict__ agg_in, __bf16 *__restrict__ agg_out,
    int32_t n_nodes) {
  constexpr int LPR = H / 8;
  constexpr int TPB = THREADS / LPR;
  const int sub = threadIdx.x % LPR;
  const int64_t v = (int64_t)blockIdx.x * TPB + threadIdx.x / LPR;
  if (v >= n_nodes) return;
  const int32_t a = rp_out[v], b = rp_out[v + 1];
  {
    float s[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    float c[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    row_sum_bf16<H>(e + 8 * sub, perm_in, rp_in[v], rp_in[v + 1], s, c);
    bf8 o;
#pragma unroll
    for (int k = 0; k < 8; ++k) o[k] = (__bf16)(s[k] + c[k]);
    *(bf8 *)(agg_in + v * H + 8 * sub) = o;
  }
  const int32_t u0 = a >> 5, u1 = (b - 1) >> 5;
  if (a < b && u0 == u1) return;  // written by the edge update
  float s[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  float c[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  if (a < b) {
    const float *pc = part + 8 * sub;
    auto piece = [&](int64_t slot, float (&r)[8]) {
      const f4 lo = *(const f4 *)(pc + slot * H), hi = *(const f4 *)(pc + slot * H + 4);
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        r[k] = lo[k];
        r[4 + k] = hi[k];
      }
    };
    piece(2 * (int64_t)u0 + 1, s);
    const bool comp = u1 - u0 > LONG_ROW;
    for (int32_t u = u0 + 1; u <= u1; ++u) {
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
  *(bf8 *)(agg_out + v * H + 8 * sub) = o;
}

template <int H>
__global__ __launch_bounds__(THREADS) void segsum_bf16(
    const __bf16 *__restrict__ e, const int32_t *__restrict__ rp_in,
    const int32_t *__restrict__ perm_in, const int32_t *__restrict__ rp_out,
    const int32_t *__restrict__ perm_out, __bf16 *__restrict__ agg_in,
    __bf16 *__restrict__ agg_out, int32_t n_nodes) {
  constexpr int LPR = H / 8;
  constexpr int TPB = THREADS / LPR;
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
  row_sum_bf16<H>(base, perm, p, pe, s, c);
  bf8 o;
#pragma unroll
  for (int k = 0; k < 8; ++k) o[k] = (__bf16)(s[k] + c[k]);
  *(bf8 *)(dst + v * H + 8 * sub) = o;
}

template <int H>
hipError_t launch_h(Act act, const void *e, const int32_t *rp_in, const int32_t *perm_in,
                    const int32_t *rp_out, const int32_t *perm_out, void *agg_in, void *agg_out,
                    int32_t n_nodes, hipStream_t stream) {
  const int lpr = act == Act::F32 ? H / 4 : H / 8;
  const int tpb = THREADS / lpr;
  const int64_t tasks = 2 * (int64_t)n_nodes;
  const unsigned blocks = (unsigned)((tasks + tpb - 1) / tpb);
  if (blocks == 0) return hipSuccess;
  if (act == Act::F32)
    segsum_f32<H><<<blocks, THREADS, 0, stream>>>((const float *)e, rp_in, perm_in, rp_out,
                                                  perm_out, (float *)agg_in, (float *)agg_out,
                                                  n_nodes);
  else
    segsum_bf16<H><<<blocks, THREADS, 0, stream>>>((const __bf16 *)e, rp_in, perm_in, rp_out,
                                                   perm_out, (__bf16 *)agg_in, (__bf16 *)agg_out,
                                                   n_nodes);
  return hipGetLastError();
}

template <int H>
hipError_t launch_fused_h(Act act, const void *e, const int32_t *rp_in, const int32_t *perm_in,
                          const int32_t *rp_out, const float *part, void *agg_in, void *agg_out,
                          int32_t n_nodes, hipStream_t stream) {
  const int tpb = THREADS / (act == Act::F32 ? H / 4 : H / 8);
  const int64_t tasks = n_nodes;
  const unsigned blocks = (unsigned)((tasks + tpb - 1) / tpb);
  if (blocks == 0) return hipSuccess;
  if (act == Act::F32)
    segsum_fused_f32<H><<<blocks, THREADS, 0, stream>>>((const float *)e, rp_in, perm_in, rp_out,
                                                        part, (float *)agg_in, (float *)agg_out,
                                                        n_nodes);
  else
    segsum_fused_bf16<H><<<blocks, THREADS, 0, stream>>>((const __bf16 *)e, rp_in, perm_in,
                                                         rp_out, part, (__bf16 *)agg_in,
                                                         (__bf16 *)agg_out, n_nodes);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_segsum_fused(Act act, int hidden, const void *e, const int32_t *rp_in,
                               const int32_t *perm_in, const int32_t *rp_out,
                               const float *agg_part, void *agg_in, void *agg_out,
                               int32_t n_nodes, hipStream_t stream) {
  switch (hidden) {
    case 64: return launch_fused_h<64>(act, e, rp_in, perm_in, rp_out, agg_part, agg_in, agg_out, n_nodes, stream);
    case 128: return launch_fused_h<128>(act, e, rp_in, perm_in, rp_out, agg_part, agg_in, agg_out, n_nodes, stream);
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
