// Fused gather + two-layer MLP kernels on the CDNA4 matrix cores.
//
// One kernel template serves every MLP of the interaction network (the edge
// classifier of paper section 2.1): node encoder, edge encoder, edge update,
// node update and edge classifier.  A wave owns 32 rows (edges or nodes) and
// all H output features:
//
//   layer 1  the rows of [src0[idx0[r]]; src1[idx1[r]]; src2[idx2[r]]] are
//            gathered straight from HBM/L2 into MFMA B-operand registers
//            (two lanes per row, 16 contiguous bytes each) and multiplied by
//            the weights; the concatenation is never materialised;
//   epilogue bias + LayerNorm + ReLU on the accumulators;
//   layer 2  a second MFMA product whose B operand is the layer-1 result
//            still in registers; bias + LayerNorm + ReLU, or, for the
//            classifier, an H->1 dot and a sigmoid.
//
// The products are computed transposed, Y^T = W X^T, so that weights are
// the MFMA A operand (M = output features) and rows the B operand
// (N = 32 rows).  In the 32x32 accumulator layout lane l holds, for row
// n = l % 32, the features 8*(v/4) + 4*(l/32) + v%4 (v = 0..15) of each
// 32-feature block.  Those are exactly the K slots the next product needs
// from this lane once K is enumerated in that order, so the layer-1 result
// feeds layer 2 without any data movement; the weight converter on the host
// stores every weight matrix in matching fragment order (see gnn_api.hip).
//
// fp32 uses v_mfma_f32_32x32x2_f32; bf16 uses v_mfma_f32_32x32x16_bf16 with
// bf16 activations, weights carried as hi + lo bf16 pairs, fp32
// accumulation, fp32 LayerNorm statistics and bf16 storage.
#include "device_common.h"

namespace gnn {
namespace {

// ---------------------------------------------------------------- fp32 ---

template <int MB, int NSRC>
__device__ __forceinline__ void layer1_f32(f16v (&acc)[MB], const float *const (&rowp)[3],
                                           const f4 *__restrict__ wf) {
  constexpr int GPS = MB * 4;  // 8-feature k-groups per source (H / 8)
  constexpr int G = NSRC * GPS;
  f4 xb[2];
  f4 wb[2][MB];
  xb[0] = *(const f4 *)(rowp[0]);
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) wb[0][mb] = wf[mb * 64];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    const int cur = g & 1, nxt = cur ^ 1;
    if (g + 1 < G) {
      const int s = (g + 1) / GPS, c = ((g + 1) % GPS) * 8;
      xb[nxt] = *(const f4 *)(rowp[s] + c);
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) wb[nxt][mb] = wf[((g + 1) * MB + mb) * 64];
    }
#pragma unroll
    for (int t = 0; t < 4; ++t)
#pragma unroll
      for (int mb = 0; mb < MB; ++mb)
        acc[mb] = __builtin_amdgcn_mfma_f32_32x32x2f32(wb[cur][mb][t], xb[cur][t], acc[mb], 0, 0,
                                                       0);
  }
}

// Layer 2: K = H, B operand = the layer-1 activations in accumulator order.
template <int MB>
__device__ __forceinline__ void layer2_f32(f16v (&out)[MB], const f16v (&act)[MB],
                                           const f4 *__restrict__ wf) {
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int v = 0; v < 16; ++v) out[mb][v] = 0.f;
  constexpr int G = MB * 4;
  f4 wb[2][MB];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) wb[0][mb] = wf[mb * 64];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    const int cur = g & 1, nxt = cur ^ 1;
    if (g + 1 < G) {
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) wb[nxt][mb] = wf[((g + 1) * MB + mb) * 64];
    }
#pragma unroll
    for (int t = 0; t < 4; ++t)
#pragma unroll
      for (int mb = 0; mb < MB; ++mb)
        out[mb] = __builtin_amdgcn_mfma_f32_32x32x2f32(wb[cur][mb][t], act[g / 4][4 * (g % 4) + t],
                                                       out[mb], 0, 0, 0);
  }
}

// KIND (a GmlpKind) only separates the instances so that profiles name the
// stage each launch belongs to.
template <int MB, int NSRC, bool SMALLK, bool CLS, int KIND>
__global__ __launch_bounds__(64 * WAVES_PER_BLOCK) void gmlp_f32(GmlpArgs a) {
  constexpr int H = 32 * MB;
  const int lane = threadIdx.x & 63, hh = lane >> 5, n = lane & 31;
  const int blk = xcd_remap(blockIdx.x, gridDim.x);
  const int64_t row0 = ((int64_t)blk * WAVES_PER_BLOCK + (threadIdx.x >> 6)) * ROWS_PER_WAVE;
  if (row0 >= a.n_rows) return;
  const int64_t row = row0 + n;
  const bool valid = row < a.n_rows;
  const int64_t r = valid ? row : a.n_rows - 1;  // tail lanes recompute the last row

  f16v acc[MB];
  if constexpr (SMALLK) {
    small_k_layer<MB>(acc, a.x, a.F, (int)r, (const float *)a.mlp.l0.w, a.mlp.l0.b, hh);
    bias_ln_relu<MB>(acc, nullptr, a.mlp.l0.g, a.mlp.l0.beta, a.eps, hh, false);
  } else {
    const float *rowp[3];
#pragma unroll
    for (int s = 0; s < 3; ++s) {
      if (s < NSRC) {
        const int64_t id = a.idx[s] ? clamp_idx(a.idx[s][r], a.n_nodes) : r;
        rowp[s] = (const float *)a.src[s] + id * H + 4 * hh;
      } else {
        rowp[s] = nullptr;
      }
    }
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[mb][v] = 0.f;
    layer1_f32<MB, NSRC>(acc, rowp, (const f4 *)a.mlp.l0.w + lane);
    bias_ln_relu<MB>(acc, a.mlp.l0.b, a.mlp.l0.g, a.mlp.l0.beta, a.eps, hh, true);
  }

  if constexpr (CLS) {
    const float *w2 = (const float *)a.mlp.l1.w;
    float part = 0.f;
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const f4 ww = *(const f4 *)(w2 + mb * 32 + 8 * q + 4 * hh);
#pragma unroll
        for (int t = 0; t < 4; ++t) part += acc[mb][4 * q + t] * ww[t];
      }
    part += __shfl_xor(part, 32);
    if (valid && hh == 0) {
      const float z = part + a.mlp.l1.b[0];
      if (a.out_logit) a.out_logit[row] = z;
      if (a.out_score) a.out_score[row] = sigmoidf_stable(z);
    }
  } else {
    f16v acc2[MB];
    layer2_f32<MB>(acc2, acc, (const f4 *)a.mlp.l1.w + lane);
    bias_ln_relu<MB>(acc2, a.mlp.l1.b, a.mlp.l1.g, a.mlp.l1.beta, a.eps, hh, true);
    if (valid) {
      float *o = (float *)a.out + row * H + 4 * hh;
#pragma unroll
      for (int mb = 0; mb < MB; ++mb)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const f4 val = {acc2[mb][4 * q], acc2[mb][4 * q + 1], acc2[mb][4 * q + 2],
                          acc2[mb][4 * q + 3]};
          *(f4 *)(o + mb * 32 + 8 * q) = val;
        }
    }
  }
}

// ---------------------------------------------------------------- bf16 ---

// bf16 products: every weight is the unevaluated sum hi + lo of two bf16
// values (two MFMAs per k-step, fp32 accumulation); the activation operand
// is bf16.
template <int MB, int NSRC>
__device__ __forceinline__ void layer1_bf16(f16v (&acc)[MB], const __bf16 *const (&rowp)[3],
                                            const bf8 *__restrict__ wf,
                                            const bf8 *__restrict__ wl) {
  constexpr int GPS = MB * 2;  // 16-feature k-steps per source (H / 16)
  constexpr int G = NSRC * GPS;
  bf8 xb[2];
  bf8 wb[2][MB], lb[2][MB];
  xb[0] = *(const bf8 *)(rowp[0]);
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) {
    wb[0][mb] = wf[mb * 64];
    lb[0][mb] = wl[mb * 64];
  }
#pragma unroll
  for (int g = 0; g < G; ++g) {
    const int cur = g & 1, nxt = cur ^ 1;
    if (g + 1 < G) {
      const int s = (g + 1) / GPS, c = ((g + 1) % GPS) * 16;
      xb[nxt] = *(const bf8 *)(rowp[s] + c);
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) {
        wb[nxt][mb] = wf[((g + 1) * MB + mb) * 64];
        lb[nxt][mb] = wl[((g + 1) * MB + mb) * 64];
      }
    }
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) {
      acc[mb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(lb[cur][mb], xb[cur], acc[mb], 0, 0, 0);
      acc[mb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(wb[cur][mb], xb[cur], acc[mb], 0, 0, 0);
    }
  }
}

template <int MB>
__device__ __forceinline__ void layer2_bf16(f16v (&out)[MB], const f16v (&act)[MB],
                                            const bf8 *__restrict__ wf,
                                            const bf8 *__restrict__ wl) {
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int v = 0; v < 16; ++v) out[mb][v] = 0.f;
  constexpr int G = MB * 2;
#pragma unroll
  for (int g = 0; g < G; ++g) {
    bf8 xb;
#pragma unroll
    for (int s = 0; s < 8; ++s) xb[s] = (__bf16)act[g / 2][8 * (g % 2) + s];
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) {
      out[mb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(wl[(g * MB + mb) * 64], xb, out[mb], 0,
                                                        0, 0);
      out[mb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(wf[(g * MB + mb) * 64], xb, out[mb], 0,
                                                        0, 0);
    }
  }
}

template <int MB, int NSRC, bool SMALLK, bool CLS, int KIND>
__global__ __launch_bounds__(64 * WAVES_PER_BLOCK) void gmlp_bf16(GmlpArgs a) {
  constexpr int H = 32 * MB;
  const int lane = threadIdx.x & 63, hh = lane >> 5, n = lane & 31;
  const int blk = xcd_remap(blockIdx.x, gridDim.x);
  const int64_t row0 = ((int64_t)blk * WAVES_PER_BLOCK + (threadIdx.x >> 6)) * ROWS_PER_WAVE;
  if (row0 >= a.n_rows) return;
  const int64_t row = row0 + n;
  const bool valid = row < a.n_rows;
  const int64_t r = valid ? row : a.n_rows - 1;

  f16v acc[MB];
  if constexpr (SMALLK) {
    small_k_layer<MB>(acc, a.x, a.F, (int)r, (const float *)a.mlp.l0.w, a.mlp.l0.b, hh);
    bias_ln_relu<MB>(acc, nullptr, a.mlp.l0.g, a.mlp.l0.beta, a.eps, hh, false);
  } else {
    const __bf16 *rowp[3];
#pragma unroll
    for (int s = 0; s < 3; ++s) {
      if (s < NSRC) {
        const int64_t id = a.idx[s] ? clamp_idx(a.idx[s][r], a.n_nodes) : r;
        rowp[s] = (const __bf16 *)a.src[s] + id * H + 8 * hh;
      } else {
        rowp[s] = nullptr;
      }
    }
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[mb][v] = 0.f;
    layer1_bf16<MB, NSRC>(acc, rowp, (const bf8 *)a.mlp.l0.w + lane,
                          (const bf8 *)a.mlp.l0.w_lo + lane);
    bias_ln_relu<MB>(acc, a.mlp.l0.b, a.mlp.l0.g, a.mlp.l0.beta, a.eps, hh, true);
  }

  if constexpr (CLS) {
    const float *w2 = (const float *)a.mlp.l1.w;
    float part = 0.f;
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const f4 ww = *(const f4 *)(w2 + mb * 32 + 8 * q + 4 * hh);
#pragma unroll
        for (int t = 0; t < 4; ++t) part += acc[mb][4 * q + t] * ww[t];
      }
    part += __shfl_xor(part, 32);
    if (valid && hh == 0) {
      const float z = part + a.mlp.l1.b[0];
      if (a.out_logit) a.out_logit[row] = z;
      if (a.out_score) a.out_score[row] = sigmoidf_stable(z);
    }
  } else {
    f16v acc2[MB];
    layer2_bf16<MB>(acc2, acc, (const bf8 *)a.mlp.l1.w + lane, (const bf8 *)a.mlp.l1.w_lo + lane);
    bias_ln_relu<MB>(acc2, a.mlp.l1.b, a.mlp.l1.g, a.mlp.l1.beta, a.eps, hh, true);
    if (valid) {
      __bf16 *o = (__bf16 *)a.out + row * H + 4 * hh;
#pragma unroll
      for (int mb = 0; mb < MB; ++mb)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          bf4 val;
#pragma unroll
          for (int t = 0; t < 4; ++t) val[t] = (__bf16)acc2[mb][4 * q + t];
          *(bf4 *)(o + mb * 32 + 8 * q) = val;
        }
    }
  }
}

template <int MB, int NSRC, bool SMALLK, bool CLS, int KIND>
hipError_t launch_one(Act act, const GmlpArgs &a, hipStream_t stream) {
  const int64_t waves = (a.n_rows + ROWS_PER_WAVE - 1) / ROWS_PER_WAVE;
  const int64_t blocks = (waves + WAVES_PER_BLOCK - 1) / WAVES_PER_BLOCK;
  if (blocks <= 0) return hipSuccess;
  if (blocks > INT32_MAX) return hipErrorInvalidValue;
  const unsigned nb = (unsigned)blocks;
  if (act == Act::F32)
    return launch(gmlp_f32<MB, NSRC, SMALLK, CLS, KIND>, nb, 64 * WAVES_PER_BLOCK, 0, stream, a);
  return launch(gmlp_bf16<MB, NSRC, SMALLK, CLS, KIND>, nb, 64 * WAVES_PER_BLOCK, 0, stream, a);
}

template <int MB>
hipError_t launch_kind(GmlpKind kind, Act act, const GmlpArgs &a, hipStream_t stream) {
  switch (kind) {
    case GmlpKind::NodeEnc: return launch_one<MB, 0, true, false, 0>(act, a, stream);
    case GmlpKind::EdgeEnc: return launch_one<MB, 2, false, false, 1>(act, a, stream);
    case GmlpKind::EdgeUpd: return launch_one<MB, 3, false, false, 2>(act, a, stream);
    case GmlpKind::NodeUpd: return launch_one<MB, 3, false, false, 3>(act, a, stream);
    case GmlpKind::Classifier: return launch_one<MB, 3, false, true, 4>(act, a, stream);
  }
  return hipErrorInvalidValue;
}

}  // namespace

hipError_t launch_gmlp(GmlpKind kind, Act act, int hidden, const GmlpArgs &a,
                       hipStream_t stream) {
  if (a.F > MAX_F) return hipErrorInvalidValue;
  switch (hidden) {
    case 64: return launch_kind<2>(kind, act, a, stream);
    case 128: return launch_kind<4>(kind, act, a, stream);
  }
  return hipErrorInvalidValue;
}

}  // namespace gnn
