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
// in flight per lane.  Accumulation is fp32 in both storage modes.
#include "gnn_internal.h"

namespace gnn {
namespace {

typedef float f4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf8 __attribute__((ext_vector_type(8)));

constexpr int THREADS = 256;

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
  f4 acc = {0.f, 0.f, 0.f, 0.f};
  for (; p + 4 <= pe; p += 4) {
    const int64_t j0 = perm[p], j1 = perm[p + 1], j2 = perm[p + 2], j3 = perm[p + 3];
    const f4 r0 = *(const f4 *)(base + j0 * H);
    const f4 r1 = *(const f4 *)(base + j1 * H);
    const f4 r2 = *(const f4 *)(base + j2 * H);
    const f4 r3 = *(const f4 *)(base + j3 * H);
    acc += r0;
    acc += r1;
    acc += r2;
    acc += r3;
  }
  for (; p < pe; ++p) acc += *(const f4 *)(base + (int64_t)perm[p] * H);
  *(f4 *)(dst + v * H + 4 * sub) = acc;
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
  float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  for (; p + 4 <= pe; p += 4) {
    bf8 r[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) r[u] = *(const bf8 *)(base + (int64_t)perm[p + u] * H);
#pragma unroll
    for (int u = 0; u < 4; ++u)
#pragma unroll
      for (int k = 0; k < 8; ++k) acc[k] += (float)r[u][k];
  }
  for (; p < pe; ++p) {
    const bf8 r = *(const bf8 *)(base + (int64_t)perm[p] * H);
#pragma unroll
    for (int k = 0; k < 8; ++k) acc[k] += (float)r[k];
  }
  bf8 o;
#pragma unroll
  for (int k = 0; k < 8; ++k) o[k] = (__bf16)acc[k];
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

}  // namespace

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
