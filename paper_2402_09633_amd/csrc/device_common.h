// Device helpers shared by the MLP kernel files (mlp.hip, factored.hip,
// split.hip):
// vector types, the XCD-aware block remap, index clamping, the stable
// sigmoid, the LayerNorm/ReLU epilogue on MFMA accumulators and the small-K
// first layer of the node encoder.
//
// Accumulator layout (v_mfma_*_32x32*): for a 32x32 block, lane l holds
// column n = l % 32 and rows 8*(v/4) + 4*(l/32) + v%4 for v = 0..15.  The
// kernels put output features on rows and graph rows (edges or nodes) on
// columns, so lane l holds half of the features of row n and lane l ^ 32 the
// other half.
#pragma once

#include "gnn_internal.h"

namespace gnn {
namespace {

typedef float f4 __attribute__((ext_vector_type(4)));
typedef float f16v __attribute__((ext_vector_type(16)));
typedef __bf16 bf8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf4 __attribute__((ext_vector_type(4)));

constexpr int WAVES_PER_BLOCK = 4;
constexpr int ROWS_PER_WAVE = 32;
constexpr int MAX_F = 16;

// Workgroups are dispatched round-robin over the 8 XCDs of the chip; give
// each XCD a contiguous range of row tiles so that neighbouring edges, which
// share gathered node rows, reuse one L2.
__device__ __forceinline__ int xcd_remap(int bid, int nblocks) {
  const int q = nblocks >> 3, rmd = nblocks & 7;
  const int r = bid & 7, k = bid >> 3;
  return r * q + min(r, rmd) + k;
}

__device__ __forceinline__ int clamp_idx(int32_t v, int32_t n) {
  return v < 0 ? 0 : (v >= n ? n - 1 : v);
}

__device__ __forceinline__ float sigmoidf_stable(float z) {
  if (z >= 0.f) return 1.f / (1.f + __expf(-z));
  const float ez = __expf(z);
  return ez / (1.f + ez);
}

// Bias + LayerNorm + ReLU over the H = 32*MB features of this lane's row,
// held half in this lane and half in lane ^ 32.  With add_bias false the
// bias is already in the accumulators.  Accumulators that hold s * y for a
// power-of-two s (split-precision products) pass bscale = s and eps * s^2:
// LayerNorm of s * (y + b) with eps s^2 equals LayerNorm of y + b with eps.
// 1 / sqrt(x) for the LayerNorm scale, x = variance + eps > 0: the hardware
// reciprocal square root (v_rsq_f32, about 1 ulp), in place of a square root
// followed by an IEEE division (two roundings and a dozen instructions).
__device__ __forceinline__ float ln_rstd(float x) { return __builtin_amdgcn_rsqf(x); }

template <int MB>
__device__ __forceinline__ void bias_ln_relu(f16v (&acc)[MB], const float *__restrict__ b,
                                             const float *__restrict__ g,
                                             const float *__restrict__ beta, float eps, int hh,
                                             bool add_bias, float bscale = 1.f) {
  constexpr float inv_h = 1.0f / (32 * MB);
  float s = 0.f;
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int f = mb * 32 + 8 * q + 4 * hh;
      const f4 bb = add_bias ? *(const f4 *)(b + f) : f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        acc[mb][4 * q + t] += bb[t] * bscale;
        s += acc[mb][4 * q + t];
      }
    }
  s += __shfl_xor(s, 32);
  const float mean = s * inv_h;
  float var = 0.f;
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const float d = acc[mb][v] - mean;
      var += d * d;
    }
  var += __shfl_xor(var, 32);
  const float rstd = ln_rstd(var * inv_h + eps);
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int f = mb * 32 + 8 * q + 4 * hh;
      const f4 gg = *(const f4 *)(g + f);
      const f4 bt = *(const f4 *)(beta + f);
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const float y = (acc[mb][4 * q + t] - mean) * rstd * gg[t] + bt[t];
        acc[mb][4 * q + t] = fmaxf(y, 0.f);
      }
    }
}

// LayerNorm epilogue with its parameters (b, gamma, beta; H floats each)
// read from LDS (the bias already multiplied by the accumulators' scale,
// eps by its square).  ADD_BIAS false: the bias is in the accumulators
// already (b is then not read).
template <int MB, bool ADD_BIAS = true>
__device__ __forceinline__ void ln_relu_lds(f16v (&acc)[MB], const float *prm, float eps, int hh) {
  constexpr int H = 32 * MB;
  constexpr float inv_h = 1.0f / H;
  float s = 0.f;
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      f4 bb = {0.f, 0.f, 0.f, 0.f};
      if constexpr (ADD_BIAS) bb = *(const f4 *)(prm + mb * 32 + 8 * q + 4 * hh);
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        if constexpr (ADD_BIAS) acc[mb][4 * q + t] += bb[t];
        s += acc[mb][4 * q + t];
      }
    }
  s += __shfl_xor(s, 32);
  const float mean = s * inv_h;
  // centred in place: the normalisation reuses x - mean (same roundings as
  // recomputing it, one subtraction fewer per value)
  float var = 0.f;
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      acc[mb][v] -= mean;
      var += acc[mb][v] * acc[mb][v];
    }
  var += __shfl_xor(var, 32);
  const float rstd = ln_rstd(var * inv_h + eps);
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int f = mb * 32 + 8 * q + 4 * hh;
      const f4 gg = *(const f4 *)(prm + H + f);
      const f4 bt = *(const f4 *)(prm + 2 * H + f);
#pragma unroll
      for (int t = 0; t < 4; ++t)
        acc[mb][4 * q + t] = fmaxf(acc[mb][4 * q + t] * rstd * gg[t] + bt[t], 0.f);
    }
}

// Layer 1 on VALU for a small input width F (node encoder): the accumulator
// slots are filled directly with W x + b.  Wt is W transposed, [F][H], so
// a lane reads its four consecutive features of one input as a float4.
template <int MB>
__device__ __forceinline__ void small_k_layer(f16v (&acc)[MB], const float *__restrict__ x,
                                              int F, int row, const float *__restrict__ Wt,
                                              const float *__restrict__ b, int hh) {
  constexpr int H = 32 * MB;
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const f4 bb = *(const f4 *)(b + mb * 32 + 8 * q + 4 * hh);
#pragma unroll
      for (int t = 0; t < 4; ++t) acc[mb][4 * q + t] = bb[t];
    }
  for (int k = 0; k < F; ++k) {
    const float xk = x[(int64_t)row * F + k];
    const float *wk = Wt + k * H + 4 * hh;
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const f4 ww = *(const f4 *)(wk + mb * 32 + 8 * q);
#pragma unroll
        for (int t = 0; t < 4; ++t) acc[mb][4 * q + t] += ww[t] * xk;
      }
  }
}

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


// ---- split-precision products (split.hip, filter.hip) ----
typedef _Float16 h8 __attribute__((ext_vector_type(8)));
typedef float f8 __attribute__((ext_vector_type(8)));

// x = x1 + x2 with x1 = fp16(x), x2 = fp16(x - x1), both rounded to nearest.
__device__ __forceinline__ void split2(const f8 &x, h8 &x1, h8 &x2) {
  x1 = __builtin_convertvector(x, h8);
  x2 = __builtin_convertvector(x - __builtin_convertvector(x1, f8), h8);
}

__device__ __forceinline__ f16v mma_h(const h8 &a, const h8 &b, const f16v &c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, c, 0, 0, 0);
}
// Weight records.  One record holds the A operands of one 16-wide k-step for
// all MB output blocks, laid out [mb][part][lane] (16 bytes per slot), so
// that lane l reads its parts of block mb at rec[(parts * mb + part) * 64].
//
// acc[mb] += (w1 + w2) (x1 + x2) over one k-step, x given split.
template <int MB>
__device__ __forceinline__ void step_h(f16v (&acc)[MB], const h8 *rec, const h8 &x1,
                                       const h8 &x2) {
  h8 w1[MB], w2[MB];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) {
    w1[mb] = rec[(2 * mb) * 64];
    w2[mb] = rec[(2 * mb + 1) * 64];
  }
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) acc[mb] = mma_h(w1[mb], x1, acc[mb]);
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) acc[mb] = mma_h(w2[mb], x1, acc[mb]);
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) acc[mb] = mma_h(w1[mb], x2, acc[mb]);
}

template <int MB>
__device__ __forceinline__ void step_h(f16v (&acc)[MB], const h8 *rec, const f8 &x) {
  h8 x1, x2;
  split2(x, x1, x2);
  step_h<MB>(acc, rec, x1, x2);
}

// The eight accumulator values a lane supplies as the B operand of k-step
// g = 2 mb + p when the operand is the previous layer's accumulators: the
// features 16 g + 8 (j / 4) + 4 hh + j % 4, j = 0..7.
template <int MB>
__device__ __forceinline__ f8 acc_x(const f16v (&a)[MB], int g) {
  const int mb = g / 2, o = 8 * (g % 2);
  return f8{a[mb][o], a[mb][o + 1], a[mb][o + 2], a[mb][o + 3],
            a[mb][o + 4], a[mb][o + 5], a[mb][o + 6], a[mb][o + 7]};
}

}  // namespace
}  // namespace gnn
