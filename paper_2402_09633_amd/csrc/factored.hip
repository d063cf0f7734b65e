// fp32 interaction-network kernels with the first Linear layer of every
// edge-side MLP regrouped at node level.
//
// The edge MLPs (edge encoder, edge update, classifier) start with
// W1 [h_src; h_dst; e] + b1.  Splitting W1 by column blocks,
//     W1 [h_src; h_dst; e] = (W_s h)[src] + (W_d h)[dst] + W_e e,
// so the node kernel that produces h also produces the projection rows
// P[v] = [W_s h_v ; W_d h_v] (2H floats per node, computed once per node
// instead of once per incident edge) and the edge kernel gathers
// P[src][0:H] and P[dst][H:2H] by index and adds W_e e.  This is the same
// layer evaluated in a different summation order (fp32 rounding aside), and
// it moves 2/3 of the first layer's products from E edges to N nodes.
//
// node_f32  one wave per 32 nodes: layer 1 (small-K VALU for the encoder, or
//           MFMA over [h; agg_in; agg_out]), LayerNorm/ReLU, layer 2, then one
//           or two projections [W_s; W_d] h' for the next edge consumer(s),
//           all chained through the accumulator layout (no LDS, no
//           transposes); weights stream from L2.
// edge_f32  persistent: each workgroup (8 waves) first copies W_e and W2
//           (fp32 MFMA fragments, up to 128 KB) into LDS once, then every
//           wave walks 32-edge units: gather P rows into the accumulators,
//           MFMA W_e e with A fragments from LDS, LayerNorm/ReLU, layer 2 from
//           LDS (or the classifier head + sigmoid), store.
#include "device_common.h"

namespace gnn {
namespace {

constexpr int NODE_WAVES = 4;
constexpr int EDGE_WAVES = 8;

// out[mb] (mb < MB) = sum over k < H of Wf[MB0 + mb][k] * act[k]; Wf holds
// fragments of an (MBT*32) x H matrix; act is in accumulator order.
template <int MB, int MBT>
__device__ __forceinline__ void gemm_acc_f32(f16v (&out)[MB], const f16v (&act)[MB],
                                             const f4 *__restrict__ wf, int mb0) {
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int v = 0; v < 16; ++v) out[mb][v] = 0.f;
  constexpr int G = MB * 4;
  f4 wb[2][MB];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) wb[0][mb] = wf[(mb0 + mb) * 64];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    const int cur = g & 1, nxt = cur ^ 1;
    if (g + 1 < G) {
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) wb[nxt][mb] = wf[((g + 1) * MBT + mb0 + mb) * 64];
    }
#pragma unroll
    for (int t = 0; t < 4; ++t)
#pragma unroll
      for (int mb = 0; mb < MB; ++mb)
        out[mb] = __builtin_amdgcn_mfma_f32_32x32x2f32(wb[cur][mb][t], act[g / 4][4 * (g % 4) + t],
                                                       out[mb], 0, 0, 0);
  }
}

// Layer 1 over the concatenation of three row sources with K = 3H; the B
// operand is prefetched two k-groups ahead, the weights one ahead.
template <int MB>
__device__ __forceinline__ void layer1_cat3_f32(f16v (&acc)[MB], const float *const (&rowp)[3],
                                                const f4 *__restrict__ wf) {
  constexpr int GPS = MB * 4;
  constexpr int G = 3 * GPS;
  f4 xb[3];
  f4 wb[2][MB];
  xb[0] = *(const f4 *)(rowp[0]);
  xb[1] = *(const f4 *)(rowp[0] + 8);
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) wb[0][mb] = wf[mb * 64];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    const int cur = g & 1, nxt = cur ^ 1;
    if (g + 2 < G) {
      const int s = (g + 2) / GPS, c = ((g + 2) % GPS) * 8;
      xb[(g + 2) % 3] = *(const f4 *)(rowp[s] + c);
    }
    if (g + 1 < G) {
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) wb[nxt][mb] = wf[((g + 1) * MB + mb) * 64];
    }
    const f4 x = xb[g % 3];
#pragma unroll
    for (int t = 0; t < 4; ++t)
#pragma unroll
      for (int mb = 0; mb < MB; ++mb)
        acc[mb] = __builtin_amdgcn_mfma_f32_32x32x2f32(wb[cur][mb][t], x[t], acc[mb], 0, 0, 0);
  }
}

template <int MB>
__device__ __forceinline__ void store_rows_f32(float *__restrict__ o, const f16v (&acc)[MB]) {
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const f4 val = {acc[mb][4 * q], acc[mb][4 * q + 1], acc[mb][4 * q + 2], acc[mb][4 * q + 3]};
      *(f4 *)(o + mb * 32 + 8 * q) = val;
    }
}

template <int MB, bool ENC, int NPROJ>
__global__ __launch_bounds__(64 * NODE_WAVES) void node_f32(NodeArgs a) {
  constexpr int H = 32 * MB;
  const int lane = threadIdx.x & 63, hh = lane >> 5, n = lane & 31;
  const int blk = xcd_remap(blockIdx.x, gridDim.x);
  const int64_t row0 = ((int64_t)blk * NODE_WAVES + (threadIdx.x >> 6)) * 32;
  if (row0 >= a.n_rows) return;
  const int64_t row = row0 + n;
  const bool valid = row < a.n_rows;
  const int64_t r = valid ? row : a.n_rows - 1;

  f16v acc[MB];
  if constexpr (ENC) {
    small_k_layer<MB>(acc, a.x, a.F, (int)r, (const float *)a.mlp.l0.w, a.mlp.l0.b, hh);
    bias_ln_relu<MB>(acc, nullptr, a.mlp.l0.g, a.mlp.l0.beta, a.eps, hh, false);
  } else {
    const float *rowp[3];
#pragma unroll
    for (int s = 0; s < 3; ++s) rowp[s] = a.src[s] + r * H + 4 * hh;
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[mb][v] = 0.f;
    layer1_cat3_f32<MB>(acc, rowp, (const f4 *)a.mlp.l0.w + lane);
    bias_ln_relu<MB>(acc, a.mlp.l0.b, a.mlp.l0.g, a.mlp.l0.beta, a.eps, hh, true);
  }
  f16v hv[MB];
  gemm_acc_f32<MB, MB>(hv, acc, (const f4 *)a.mlp.l1.w + lane, 0);
  bias_ln_relu<MB>(hv, a.mlp.l1.b, a.mlp.l1.g, a.mlp.l1.beta, a.eps, hh, true);
  if (valid && a.h_out) store_rows_f32<MB>(a.h_out + row * H + 4 * hh, hv);

#pragma unroll
  for (int p = 0; p < NPROJ; ++p) {
#pragma unroll
    for (int half = 0; half < 2; ++half) {
      f16v pv[MB];
      gemm_acc_f32<MB, 2 * MB>(pv, hv, (const f4 *)a.proj[p] + lane, half * MB);
      if (valid) store_rows_f32<MB>(a.p_out[p] + row * 2 * H + half * H + 4 * hh, pv);
    }
  }
}

template <int MB, int MODE>
__global__ __launch_bounds__(64 * EDGE_WAVES) void edge_f32(EdgeArgs a) {
  constexpr int H = 32 * MB;
  constexpr int NW = H * H / 4;  // float4 fragments of one H x H matrix
  constexpr bool HAS_E = MODE != (int)EdgeMode::Enc;
  constexpr bool HAS_L2 = MODE != (int)EdgeMode::Cls;
  __shared__ f4 lds[(HAS_E ? NW : 0) + (HAS_L2 ? NW : 0)];
  f4 *lw_e = lds;
  f4 *lw_2 = lds + (HAS_E ? NW : 0);
  for (int i = threadIdx.x; i < NW; i += 64 * EDGE_WAVES) {
    if constexpr (HAS_E) lw_e[i] = ((const f4 *)a.we)[i];
    if constexpr (HAS_L2) lw_2[i] = ((const f4 *)a.w2)[i];
  }
  __syncthreads();

  const int lane = threadIdx.x & 63, hh = lane >> 5, n = lane & 31;
  const int blk = xcd_remap(blockIdx.x, gridDim.x);
  const int64_t gw = (int64_t)blk * EDGE_WAVES + (threadIdx.x >> 6);
  const int64_t nw = (int64_t)gridDim.x * EDGE_WAVES;
  const int64_t units = (a.n_rows + 31) / 32;
  for (int64_t u = gw; u < units; u += nw) {
    // Keeps the LDS fragment reads inside the loop: hoisting them out of it
    // (they are loop-invariant) would pin every fragment in registers.
    asm volatile("" ::: "memory");
    const int64_t row = u * 32 + n;
    const bool valid = row < a.n_rows;
    const int64_t r = valid ? row : a.n_rows - 1;
    const int64_t s = clamp_idx(a.src_idx[r], a.n_nodes);
    const int64_t d = clamp_idx(a.dst_idx[r], a.n_nodes);

    // Layer 1 = P[src][0:H] + P[dst][H:2H] (+ W_e e) + b1.
    f16v acc[MB];
    {
      const float *ps = a.P + s * 2 * H + 4 * hh;
      const float *pd = a.P + d * 2 * H + H + 4 * hh;
#pragma unroll
      for (int mb = 0; mb < MB; ++mb)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int f = mb * 32 + 8 * q;
          const f4 x = *(const f4 *)(ps + f) + *(const f4 *)(pd + f);
#pragma unroll
          for (int t = 0; t < 4; ++t) acc[mb][4 * q + t] = x[t];
        }
    }
    if constexpr (HAS_E) {
      // e row streamed two k-groups ahead, A fragments from LDS one ahead
      constexpr int G = MB * 4;
      const float *ep = a.e_in + r * H + 4 * hh;
      const f4 *wf = lw_e + lane;
      f4 xb[3];
      f4 wb[2][MB];
      xb[0] = *(const f4 *)(ep);
      xb[1] = *(const f4 *)(ep + 8);
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) wb[0][mb] = wf[mb * 64];
#pragma unroll
      for (int g = 0; g < G; ++g) {
        const int cur = g & 1, nxt = cur ^ 1;
        if (g + 2 < G) xb[(g + 2) % 3] = *(const f4 *)(ep + 8 * (g + 2));
        if (g + 1 < G) {
#pragma unroll
          for (int mb = 0; mb < MB; ++mb) wb[nxt][mb] = wf[((g + 1) * MB + mb) * 64];
        }
        const f4 x = xb[g % 3];
#pragma unroll
        for (int t = 0; t < 4; ++t)
#pragma unroll
          for (int mb = 0; mb < MB; ++mb)
            acc[mb] = __builtin_amdgcn_mfma_f32_32x32x2f32(wb[cur][mb][t], x[t], acc[mb], 0, 0,
                                                           0);
      }
    }
    bias_ln_relu<MB>(acc, a.b1, a.g1, a.beta1, a.eps, hh, true);

    if constexpr (!HAS_L2) {
      float part = 0.f;
#pragma unroll
      for (int mb = 0; mb < MB; ++mb)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const f4 ww = *(const f4 *)(a.w2 + mb * 32 + 8 * q + 4 * hh);
#pragma unroll
          for (int t = 0; t < 4; ++t) part += acc[mb][4 * q + t] * ww[t];
        }
      part += __shfl_xor(part, 32);
      if (valid && hh == 0) {
        const float z = part + a.b2[0];
        if (a.out_logit) a.out_logit[row] = z;
        if (a.out_score) a.out_score[row] = sigmoidf_stable(z);
      }
    } else {
      f16v acc2[MB];
      gemm_acc_f32<MB, MB>(acc2, acc, lw_2 + lane, 0);
      bias_ln_relu<MB>(acc2, a.b2, a.g2, a.beta2, a.eps, hh, true);
      if (valid) store_rows_f32<MB>(a.e_out + row * H + 4 * hh, acc2);
    }
  }
}

template <int MB>
hipError_t node_h(bool enc, const NodeArgs &a, hipStream_t stream) {
  const int64_t waves = (a.n_rows + 31) / 32;
  const int64_t blocks = (waves + NODE_WAVES - 1) / NODE_WAVES;
  if (blocks <= 0) return hipSuccess;
  if (blocks > INT32_MAX) return hipErrorInvalidValue;
  const unsigned nb = (unsigned)blocks;
  if (enc) {
    if (a.nproj == 2)
      node_f32<MB, true, 2><<<nb, 64 * NODE_WAVES, 0, stream>>>(a);
    else
      node_f32<MB, true, 1><<<nb, 64 * NODE_WAVES, 0, stream>>>(a);
  } else {
    node_f32<MB, false, 1><<<nb, 64 * NODE_WAVES, 0, stream>>>(a);
  }
  return hipGetLastError();
}

template <int MB>
hipError_t edge_h(EdgeMode mode, const EdgeArgs &a, int grid, hipStream_t stream) {
  const int64_t units = (a.n_rows + 31) / 32;
  const int64_t need = (units + EDGE_WAVES - 1) / EDGE_WAVES;
  if (need <= 0) return hipSuccess;
  const unsigned nb = (unsigned)(need < grid ? need : grid);
  switch (mode) {
    case EdgeMode::Enc: edge_f32<MB, 0><<<nb, 64 * EDGE_WAVES, 0, stream>>>(a); break;
    case EdgeMode::Upd: edge_f32<MB, 1><<<nb, 64 * EDGE_WAVES, 0, stream>>>(a); break;
    case EdgeMode::Cls: edge_f32<MB, 2><<<nb, 64 * EDGE_WAVES, 0, stream>>>(a); break;
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_node_f32(bool enc, int hidden, const NodeArgs &a, hipStream_t stream) {
  if (a.F > MAX_F || a.nproj < 1 || a.nproj > 2 || (!enc && a.nproj != 1))
    return hipErrorInvalidValue;
  switch (hidden) {
    case 64: return node_h<2>(enc, a, stream);
    case 128: return node_h<4>(enc, a, stream);
  }
  return hipErrorInvalidValue;
}

// Workgroups that fit on the chip at once (persistent grid).
int edge_f32_grid(EdgeMode mode, int hidden, int n_cu) {
  const void *fn = nullptr;
  if (hidden == 64)
    fn = mode == EdgeMode::Enc   ? (const void *)edge_f32<2, 0>
         : mode == EdgeMode::Upd ? (const void *)edge_f32<2, 1>
                                 : (const void *)edge_f32<2, 2>;
  else
    fn = mode == EdgeMode::Enc   ? (const void *)edge_f32<4, 0>
         : mode == EdgeMode::Upd ? (const void *)edge_f32<4, 1>
                                 : (const void *)edge_f32<4, 2>;
  int per_cu = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, fn, 64 * EDGE_WAVES, 0) !=
          hipSuccess ||
      per_cu < 1)
    per_cu = 1;
  return per_cu * (n_cu > 0 ? n_cu : 1);
}

hipError_t launch_edge_f32(EdgeMode mode, int hidden, const EdgeArgs &a, int grid,
                           hipStream_t stream) {
  if (grid <= 0) return hipErrorInvalidValue;
  switch (hidden) {
    case 64: return edge_h<2>(mode, a, grid, stream);
    case 128: return edge_h<4>(mode, a, grid, stream);
  }
  return hipErrorInvalidValue;
}

}  // namespace gnn
