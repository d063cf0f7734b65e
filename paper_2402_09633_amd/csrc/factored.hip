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

// Layer 1 over the concatenation of three row sources with K = 3H.  A
// lane's half-row of each source (16 float4) is loaded in one burst, the
// next source's while the current one is multiplied, so an HBM miss is
// exposed at most once per node; the weights stream from L2 one k-group
// ahead.
template <int MB>
__device__ __forceinline__ void layer1_cat3_f32(f16v (&acc)[MB], const float *const (&rowp)[3],
                                                const f4 *__restrict__ wf) {
  constexpr int GPS = MB * 4;
  f4 xb[2][GPS];
#pragma unroll
  for (int g = 0; g < GPS; ++g) xb[0][g] = *(const f4 *)(rowp[0] + 8 * g);
  f4 wb[2][MB];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) wb[0][mb] = wf[mb * 64];
#pragma unroll
  for (int src = 0; src < 3; ++src) {
    const int cb = src & 1;
    if (src + 1 < 3) {
#pragma unroll
      for (int g = 0; g < GPS; ++g) xb[cb ^ 1][g] = *(const f4 *)(rowp[src + 1] + 8 * g);
    }
#pragma unroll
    for (int gl = 0; gl < GPS; ++gl) {
      const int g = src * GPS + gl;
      const int cur = g & 1, nxt = cur ^ 1;
      if (g + 1 < 3 * GPS) {
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) wb[nxt][mb] = wf[((g + 1) * MB + mb) * 64];
      }
#pragma unroll
      for (int t = 0; t < 4; ++t)
#pragma unroll
        for (int mb = 0; mb < MB; ++mb)
          acc[mb] = __builtin_amdgcn_mfma_f32_32x32x2f32(wb[cur][mb][t], xb[cb][gl][t], acc[mb],
                                                         0, 0, 0);
    }
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

// Node kernel: persistent workgroups of 8 waves, each wave 32 nodes of a
// 256-node tile.  All weights of the kernel form one fragment stream
// (layer 1 | layer 2 | projection halves), cut into 32 KB chunks of
// CH = 8 k-groups that the workgroup double-buffers through LDS: while the
// waves multiply chunk c out of one buffer, chunk c+1 is fetched from L2
// into registers and written to the other buffer; one barrier per chunk.
constexpr int CH = 8;

template <int MB>
struct WStream {
  const f4 *base;     // fragment stream in global memory
  int nchunks;        // chunks per tile
  f4 (*buf)[CH * MB * 64];
  int c = 0;          // chunk index within the tile (position in the stream)
  int k = 0;          // chunks consumed so far (selects the LDS buffer)
  f4 st[MB];          // staged next chunk (CH*MB*64 f4 / 512 threads = MB each)
  __device__ void fetch(int cc, int tid) {
#pragma unroll
    for (int i = 0; i < MB; ++i) st[i] = base[(size_t)cc * CH * MB * 64 + i * 512 + tid];
  }
  __device__ void commit(int b, int tid) {
#pragma unroll
    for (int i = 0; i < MB; ++i) buf[b][i * 512 + tid] = st[i];
  }
  // Start of a chunk: wait until it is in LDS, request the next one.
  __device__ const f4 *begin(int tid) {
    __syncthreads();
    fetch((c + 1) % nchunks, tid);
    return buf[k & 1];
  }
  // End of a chunk: publish the next one (read by others after the barrier)
  // into the other buffer.  The buffer alternates with every chunk consumed,
  // also across tiles when a tile has an odd number of chunks.
  __device__ void end(int tid) {
    commit((k + 1) & 1, tid);
    ++k;
    c = (c + 1) % nchunks;
  }
};

// One chunk of MFMAs: out[mb] += Wchunk x B, with B supplied per k-group.
template <int MB, typename BF>
__device__ __forceinline__ void chunk_mfma(f16v (&out)[MB], const f4 *w, int lane, BF bsrc) {
#pragma unroll
  for (int gl = 0; gl < CH; ++gl) {
    f4 wb[MB];
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) wb[mb] = w[(gl * MB + mb) * 64 + lane];
    const f4 x = bsrc(gl);
#pragma unroll
    for (int t = 0; t < 4; ++t)
#pragma unroll
      for (int mb = 0; mb < MB; ++mb)
        out[mb] = __builtin_amdgcn_mfma_f32_32x32x2f32(wb[mb][t], x[t], out[mb], 0, 0, 0);
  }
}

template <int MB>
__device__ __forceinline__ void zero_acc(f16v (&a)[MB]) {
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int v = 0; v < 16; ++v) a[mb][v] = 0.f;
}

// act[mb][v] in accumulator order as the B operand of k-group g0 + gl.
template <int MB>
__device__ __forceinline__ f4 acc_b(const f16v (&act)[MB], int g) {
  return f4{act[g / 4][4 * (g % 4)], act[g / 4][4 * (g % 4) + 1], act[g / 4][4 * (g % 4) + 2],
            act[g / 4][4 * (g % 4) + 3]};
}

template <int MB, bool ENC, int NPROJ>
__global__ __launch_bounds__(64 * EDGE_WAVES) void node_f32(NodeArgs a) {
  constexpr int H = 32 * MB;
  constexpr int GPS = MB * 4;  // k-groups per H-wide operand
  __shared__ f4 wbuf[2][CH * MB * 64];
  const int tid = threadIdx.x, lane = tid & 63, hh = lane >> 5, n = lane & 31;
  const int wave = tid >> 6;
  WStream<MB> ws{(const f4 *)a.wstream, a.nchunks, wbuf};
  ws.fetch(0, tid);
  ws.commit(0, tid);

  const int blk = xcd_remap(blockIdx.x, gridDim.x);
  const int64_t tiles = (a.n_rows + 32 * EDGE_WAVES - 1) / (32 * EDGE_WAVES);
  for (int64_t tile = blk; tile < tiles; tile += gridDim.x) {
    // Keeps the loop-invariant parameter loads inside the loop (hoisting
    // them would pin them in registers for the whole kernel).
    asm volatile("" ::: "memory");
    const int64_t row = tile * 32 * EDGE_WAVES + wave * 32 + n;
    const bool valid = row < a.n_rows;
    const int64_t r = valid ? row : a.n_rows - 1;

    f16v acc[MB];
    if constexpr (ENC) {
      small_k_layer<MB>(acc, a.x, a.F, (int)r, (const float *)a.mlp.l0.w, a.mlp.l0.b, hh);
      bias_ln_relu<MB>(acc, nullptr, a.mlp.l0.g, a.mlp.l0.beta, a.eps, hh, false);
    } else {
      zero_acc<MB>(acc);
      // The node rows are staged one chunk (8 k-groups) ahead.
      constexpr int PARTS = 3 * GPS / CH;
      auto part_ptr = [&](int j) {
        return a.src[(j * CH) / GPS] + r * H + 4 * hh + 8 * ((j * CH) % GPS);
      };
      f4 xb[2][CH];
#pragma unroll
      for (int g = 0; g < CH; ++g) xb[0][g] = *(const f4 *)(part_ptr(0) + 8 * g);
#pragma unroll
      for (int j = 0; j < PARTS; ++j) {
        if (j + 1 < PARTS) {
#pragma unroll
          for (int g = 0; g < CH; ++g) xb[(j + 1) & 1][g] = *(const f4 *)(part_ptr(j + 1) + 8 * g);
        }
        const f4 *w = ws.begin(tid);
        chunk_mfma<MB>(acc, w, lane, [&](int gl) { return xb[j & 1][gl]; });
        ws.end(tid);
      }
      bias_ln_relu<MB>(acc, a.mlp.l0.b, a.mlp.l0.g, a.mlp.l0.beta, a.eps, hh, true);
    }
    // layer 2
    f16v hv[MB];
    zero_acc<MB>(hv);
#pragma unroll
    for (int part = 0; part < GPS / CH; ++part) {
      const f4 *w = ws.begin(tid);
      chunk_mfma<MB>(hv, w, lane, [&](int gl) { return acc_b<MB>(acc, part * CH + gl); });
      ws.end(tid);
    }
    bias_ln_relu<MB>(hv, a.mlp.l1.b, a.mlp.l1.g, a.mlp.l1.beta, a.eps, hh, true);
    if (valid && a.h_out) store_rows_f32<MB>(a.h_out + row * H + 4 * hh, hv);
    // projections [W_s; W_d] h', one H-wide half at a time
#pragma unroll
    for (int p = 0; p < NPROJ; ++p)
#pragma unroll
      for (int half = 0; half < 2; ++half) {
        f16v pv[MB];
        zero_acc<MB>(pv);
#pragma unroll
        for (int part = 0; part < GPS / CH; ++part) {
          const f4 *w = ws.begin(tid);
          chunk_mfma<MB>(pv, w, lane, [&](int gl) { return acc_b<MB>(hv, part * CH + gl); });
          ws.end(tid);
        }
        if (valid) store_rows_f32<MB>(a.p_out[p] + row * 2 * H + half * H + 4 * hh, pv);
      }
  }
}

template <int MB, int MODE>
__global__ __launch_bounds__(64 * EDGE_WAVES) void edge_f32(EdgeArgs a) {
  constexpr int H = 32 * MB;
  constexpr int NW = H * H / 4;  // float4 fragments of one H x H matrix
  constexpr int G = MB * 4;      // 8-feature k-groups of one H-wide operand
  constexpr bool HAS_E = MODE != (int)EdgeMode::Enc;
  constexpr bool HAS_L2 = MODE != (int)EdgeMode::Cls;
  __shared__ f4 lds[(HAS_E ? NW : 0) + (HAS_L2 ? NW : 0)];
  __shared__ float prm[6 * H];  // b1, gamma1, beta1, b2, gamma2, beta2
  f4 *lw_e = lds;
  f4 *lw_2 = lds + (HAS_E ? NW : 0);
  for (int i = threadIdx.x; i < NW; i += 64 * EDGE_WAVES) {
    if constexpr (HAS_E) lw_e[i] = ((const f4 *)a.we)[i];
    if constexpr (HAS_L2) lw_2[i] = ((const f4 *)a.w2)[i];
  }
  for (int i = threadIdx.x; i < H; i += 64 * EDGE_WAVES) {
    prm[i] = a.b1[i];
    prm[H + i] = a.g1[i];
    prm[2 * H + i] = a.beta1[i];
    if constexpr (HAS_L2) {
      prm[3 * H + i] = a.b2[i];
      prm[4 * H + i] = a.g2[i];
      prm[5 * H + i] = a.beta2[i];
    } else {
      prm[3 * H + i] = a.w2[i];  // classifier head row
    }
  }
  __syncthreads();

  const int lane = threadIdx.x & 63, hh = lane >> 5, n = lane & 31;
  const int blk = xcd_remap(blockIdx.x, gridDim.x);
  const int64_t gw = (int64_t)blk * EDGE_WAVES + (threadIdx.x >> 6);
  const int64_t nw = (int64_t)gridDim.x * EDGE_WAVES;
  const int64_t units = (a.n_rows + 31) / 32;
  auto row_of = [&](int64_t u) {
    const int64_t row = u * 32 + n;
    return row < a.n_rows ? row : a.n_rows - 1;  // tail lanes recompute the last row
  };

  // The next unit's edge indices and e row are requested before the
  // current unit's stores: vector-memory completions are counted in issue
  // order, so a load issued after a store can only be waited for together
  // with that store.
  f4 ev[HAS_E ? G : 1];
  int32_t nsrc = 0, ndst = 0;
  if (gw < units) {
    const int64_t r0 = row_of(gw);
    nsrc = a.src_idx[r0];
    ndst = a.dst_idx[r0];
    if constexpr (HAS_E) {
      const float *ep = a.e_in + r0 * H + 4 * hh;
#pragma unroll
      for (int g = 0; g < G; ++g) ev[g] = *(const f4 *)(ep + 8 * g);
    }
  }
  for (int64_t u = gw; u < units; u += nw) {
    // Keeps the LDS fragment reads inside the loop: hoisting them out of it
    // (they are loop-invariant) would pin every fragment in registers.
    asm volatile("" ::: "memory");
    const int64_t row = u * 32 + n;
    const bool valid = row < a.n_rows;
    const int64_t s = clamp_idx(nsrc, a.n_nodes);
    const int64_t d = clamp_idx(ndst, a.n_nodes);

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
      const f4 *wf = lw_e + lane;
#pragma unroll
      for (int g = 0; g < G; ++g) {
        f4 wb[MB];
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) wb[mb] = wf[(g * MB + mb) * 64];
#pragma unroll
        for (int t = 0; t < 4; ++t)
#pragma unroll
          for (int mb = 0; mb < MB; ++mb)
            acc[mb] = __builtin_amdgcn_mfma_f32_32x32x2f32(wb[mb][t], ev[g][t], acc[mb], 0, 0,
                                                           0);
      }
    }
    {
      const int64_t un = u + nw;
      if (un < units) {
        const int64_t rn = row_of(un);
        nsrc = a.src_idx[rn];
        ndst = a.dst_idx[rn];
        if constexpr (HAS_E) {
          const float *ep = a.e_in + rn * H + 4 * hh;
#pragma unroll
          for (int g = 0; g < G; ++g) ev[g] = *(const f4 *)(ep + 8 * g);
        }
      }
    }
    ln_relu_lds<MB>(acc, prm, a.eps, hh);

    if constexpr (!HAS_L2) {
      float part = 0.f;
#pragma unroll
      for (int mb = 0; mb < MB; ++mb)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const f4 ww = *(const f4 *)(prm + 3 * H + mb * 32 + 8 * q + 4 * hh);
#pragma unroll
          for (int t = 0; t < 4; ++t) part += acc[mb][4 * q + t] * ww[t];
        }
      part += __shfl_xor(part, 32);
      if (valid && hh == 0) {
        const float z = part + a.b2[0];
        const int64_t o = a.out_idx ? a.out_idx[row] : row;
        if (a.out_logit) a.out_logit[o] = z;
        if (a.out_score) a.out_score[o] = sigmoidf_stable(z);
      }
    } else {
      f16v acc2[MB];
      {
        const f4 *wf = lw_2 + lane;
#pragma unroll
        for (int mb = 0; mb < MB; ++mb)
#pragma unroll
          for (int v = 0; v < 16; ++v) acc2[mb][v] = 0.f;
#pragma unroll
        for (int g = 0; g < G; ++g) {
          f4 wb[MB];
#pragma unroll
          for (int mb = 0; mb < MB; ++mb) wb[mb] = wf[(g * MB + mb) * 64];
#pragma unroll
          for (int t = 0; t < 4; ++t)
#pragma unroll
            for (int mb = 0; mb < MB; ++mb)
              acc2[mb] = __builtin_amdgcn_mfma_f32_32x32x2f32(wb[mb][t], acc[g / 4][4 * (g % 4) + t],
                                                              acc2[mb], 0, 0, 0);
        }
      }
      ln_relu_lds<MB>(acc2, prm + 3 * H, a.eps, hh);
      if (valid) store_rows_f32<MB>(a.e_out + row * H + 4 * hh, acc2);
    }
  }
}

template <int MB>
hipError_t node_h(bool enc, const NodeArgs &a, int grid, hipStream_t stream) {
  const int64_t tiles = (a.n_rows + 32 * EDGE_WAVES - 1) / (32 * EDGE_WAVES);
  if (tiles <= 0) return hipSuccess;
  const unsigned nb = (unsigned)(tiles < grid ? tiles : grid);
  if (!enc) return launch(node_f32<MB, false, 1>, nb, 64 * EDGE_WAVES, 0, stream, a);
  if (a.nproj == 2) return launch(node_f32<MB, true, 2>, nb, 64 * EDGE_WAVES, 0, stream, a);
  return launch(node_f32<MB, true, 1>, nb, 64 * EDGE_WAVES, 0, stream, a);
}

template <int MB>
hipError_t edge_h(EdgeMode mode, const EdgeArgs &a, int grid, hipStream_t stream) {
  const int64_t units = (a.n_rows + 31) / 32;
  const int64_t need = (units + EDGE_WAVES - 1) / EDGE_WAVES;
  if (need <= 0) return hipSuccess;
  const unsigned nb = (unsigned)(need < grid ? need : grid);
  switch (mode) {
    case EdgeMode::Enc: return launch(edge_f32<MB, 0>, nb, 64 * EDGE_WAVES, 0, stream, a);
    case EdgeMode::Upd: return launch(edge_f32<MB, 1>, nb, 64 * EDGE_WAVES, 0, stream, a);
    case EdgeMode::Cls: return launch(edge_f32<MB, 2>, nb, 64 * EDGE_WAVES, 0, stream, a);
    default: return hipErrorInvalidValue;  // no fused sums on the fp32 matrix cores
  }
}

}  // namespace

hipError_t launch_node_f32(bool enc, int hidden, const NodeArgs &a, int grid,
                           hipStream_t stream) {
  if (a.F > MAX_F || a.nproj < 1 || a.nproj > 2 || (!enc && a.nproj != 1) || grid <= 0)
    return hipErrorInvalidValue;
  const int gps = hidden / 8;
  const int expect = ((enc ? 0 : 3 * gps) + gps + 2 * a.nproj * gps) / CH;
  if (a.nchunks != expect || gps % CH) return hipErrorInvalidValue;
  switch (hidden) {
    case 64: return node_h<2>(enc, a, grid, stream);
    case 128: return node_h<4>(enc, a, grid, stream);
  }
  return hipErrorInvalidValue;
}

int node_f32_grid(int n_cu) { return n_cu > 0 ? n_cu : 1; }

// Fragments per chunk are laid out [k-group][m-block][lane] (f4), so the
// stream is the concatenation of the per-matrix fragment arrays.
int node_stream_chunk_f4(int hidden) { return CH * (hidden / 32) * 64; }

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
