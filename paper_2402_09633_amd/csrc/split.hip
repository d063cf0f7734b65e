// fp32 interaction-network kernels whose matrix products run on the fp16 and
// bf16 matrix cores, with the first Linear layer of every edge-side MLP
// regrouped per node as in factored.hip.
//
// gfx950 multiplies fp16/bf16 16 times faster than fp32 on its matrix cores,
// so every fp32 product here is evaluated from an exact, or nearly exact,
// splitting of both operands into low-precision parts, with every partial
// product accumulated in fp32 (products of the parts are exact in fp32):
//
//  f16x2   x = x1 + x2, x1 = fp16(x), x2 = fp16(x - x1), both rounded to
//          nearest, so |x - x1 - x2| <= 2^-22 |x| (2^-25 absolute once x2 is
//          subnormal).  W is scaled first by a power of two s chosen on the
//          host so that max |s W| lies in [2^13, 2^14), split the same way,
//          and  s W x = w1 x1 + w2 x1 + w1 x2  up to the dropped w2 x2
//          (<= 2^-22 |sW||x|).  Three v_mfma_f32_32x32x16_f16 replace eight
//          v_mfma_f32_32x32x2_f32 per 16-wide k-step.  It is used where the
//          operand is a LayerNorm/ReLU output, bounded by
//          max_f |gamma_f| sqrt(H-1) + |beta_f|; the handle checks that bound
//          against the fp16 range when it is created.  The edge kernels keep
//          both of their H x H matrices in LDS in this form (2 x 64 KB).
//          The node MLP's first layer also takes the aggregates, sums over a
//          node's whole degree: there each node's input row is first
//          multiplied by a power of two (1 unless the degree times the
//          message bound leaves the fp16 range) and its product column
//          divided by it again.
//
// The same kernels serve the bf16 model (PREC = BF16): h, e and the
// aggregates are stored in bf16 and fed to the bf16 matrix cores as they are,
// every weight is a pair hi = bf16(W), lo = bf16(W - hi) (two products), the
// LayerNorm outputs are rounded to bf16 where they feed a product, and all
// sums are fp32.  The projections P are stored in fp16 there, multiplied by
// the consuming edge MLP's layer-1 scale (a power of two chosen on the host
// so that every |s P| stays below 2^15), in the permuted order of
// store_block16: their rounding (2^-11 relative) is four times finer than
// the bf16 rounding of h itself.
//
// An accumulator that holds s * y is never rescaled: the bias is added as
// s * b and LayerNorm runs with eps * s^2, which gives the LayerNorm of y + b
// exactly (s is a power of two).  The node kernel stores the projections
// P = [W_s h; W_d h] already multiplied by the scale of the consuming edge
// MLP's first layer, which is the scale its W_e part uses too.
#include <type_traits>

#include "device_common.h"


namespace gnn {
namespace {

typedef unsigned u4 __attribute__((ext_vector_type(4)));

constexpr int SW = 8;  // waves per workgroup (node kernels; edge kernels: edge_waves)

__device__ __forceinline__ f8 cat8(const f4 &a, const f4 &b) {
  return f8{a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
}

__device__ __forceinline__ f16v mma_b(const bf8 &a, const bf8 &b, const f16v &c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// The same k-step with the operands exchanged: the graph rows are the A
// operand and the weights the B operand (a record's lane slots hold W[f][k]
// for f = lane % 32, which is also the B-operand layout of W^T), so the
// accumulators hold the product transposed: lane l has feature 32 mb + l % 32
// of the rows 8 (v / 4) + 4 (l / 32) + v % 4, v = 0..15.
template <int MB>
__device__ __forceinline__ void step_ht(f16v (&acc)[MB], const h8 *rec, const f8 &x) {
  h8 x1, x2, w1[MB], w2[MB];
  split2(x, x1, x2);
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) {
    w1[mb] = rec[(2 * mb) * 64];
    w2[mb] = rec[(2 * mb + 1) * 64];
  }
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) acc[mb] = mma_h(x1, w1[mb], acc[mb]);
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) acc[mb] = mma_h(x1, w2[mb], acc[mb]);
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) acc[mb] = mma_h(x2, w1[mb], acc[mb]);
}

// Sum over the 32 lanes of this lane's half of the wave; every lane of the
// half receives the same value (each step adds two partial sums, and fp32
// addition is commutative).
template <int CTRL>
__device__ __forceinline__ float dpp_f(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v),
                                                               CTRL, 0xF, 0xF, false));
}
__device__ __forceinline__ float sum32(float v) {
  v += dpp_f<0xB1>(v);   // quad_perm [1,0,3,2]
  v += dpp_f<0x4E>(v);   // quad_perm [2,3,0,1]
  v += dpp_f<0x141>(v);  // row_half_mirror
  v += dpp_f<0x140>(v);  // row_mirror
  // swap the two 16-lane rows of each 32-lane group
  return v + __builtin_bit_cast(float, __builtin_amdgcn_ds_swizzle(__builtin_bit_cast(int, v),
                                                                   0x401F));
}

// Bias + LayerNorm + ReLU on transposed accumulators (step_ht): lane l holds
// feature 32 mb + n, n = l % 32, of 16 rows; a row's statistics are sums
// over the 32 lanes of its half of the wave.  prm as for ln_relu_lds.
template <int MB>
__device__ __forceinline__ void ln_relu_t(f16v (&t)[MB], const float *prm, float eps, int n) {
  constexpr int H = 32 * MB;
  constexpr float inv_h = 1.0f / H;
  float gg[MB], bt[MB];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) {
    const float bb = prm[32 * mb + n];
    gg[mb] = prm[H + 32 * mb + n];
    bt[mb] = prm[2 * H + 32 * mb + n];
#pragma unroll
    for (int v = 0; v < 16; ++v) t[mb][v] += bb;
  }
  // four rows at a time: their reductions overlap, with few live registers
#pragma unroll
  for (int v0 = 0; v0 < 16; v0 += 4) {
    float mean[4], rstd[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      float sv = 0.f;
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) sv += t[mb][v0 + j];
      mean[j] = sum32(sv) * inv_h;
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      float q = 0.f;
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) {
        t[mb][v0 + j] -= mean[j];  // centred in place, reused below
        q += t[mb][v0 + j] * t[mb][v0 + j];
      }
      rstd[j] = ln_rstd(sum32(q) * inv_h + eps);
    }
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
      for (int j = 0; j < 4; ++j)
        t[mb][v0 + j] = fmaxf(t[mb][v0 + j] * rstd[j] * gg[mb] + bt[mb], 0.f);
  }
}

// acc[mb] += (w_hi + w_lo) x over one k-step, x exact in bf16.
template <int MB>
__device__ __forceinline__ void step_hl(f16v (&acc)[MB], const bf8 *rec, const bf8 &x) {
  bf8 w1[MB], w2[MB];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) {
    w1[mb] = rec[(2 * mb) * 64];
    w2[mb] = rec[(2 * mb + 1) * 64];
  }
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) acc[mb] = mma_b(w1[mb], x, acc[mb]);
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) acc[mb] = mma_b(w2[mb], x, acc[mb]);
}

// step_hl with the operands exchanged (transposed accumulators, as step_ht).
template <int MB>
__device__ __forceinline__ void step_hlt(f16v (&acc)[MB], const bf8 *rec, const bf8 &x) {
  bf8 w1[MB], w2[MB];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) {
    w1[mb] = rec[(2 * mb) * 64];
    w2[mb] = rec[(2 * mb + 1) * 64];
  }
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) acc[mb] = mma_b(x, w1[mb], acc[mb]);
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) acc[mb] = mma_b(x, w2[mb], acc[mb]);
}

__device__ __forceinline__ bf8 to_bf16(const f8 &x) { return __builtin_convertvector(x, bf8); }

// a + b in fp32 for two fp16 values held in the low (HI = false) or high
// halves of 32-bit registers: one mixed-precision fma, a * 1 + b, whose fp16
// sources are converted exactly (instead of two conversions and an add).
template <bool HI>
__device__ __forceinline__ float add_f16(unsigned a, unsigned b) {
  float r;
  if constexpr (HI)
    asm("v_fma_mix_f32 %0, %1, 1.0, %2 op_sel:[1,0,1] op_sel_hi:[1,0,1]" : "=v"(r) : "v"(a), "v"(b));
  else
    asm("v_fma_mix_f32 %0, %1, 1.0, %2 op_sel_hi:[1,0,1]" : "=v"(r) : "v"(a), "v"(b));
  return r;
}

// Operand precision of the kernels below.
constexpr int SPLIT = 0;  // fp32 activations, split products
constexpr int BF16 = 1;   // bf16 activations, hi/lo bf16 weights
constexpr int F16W = 2;   // bf16 activations, fp16 weights (one product per weight)

// Waves per workgroup of the edge kernels.  With fp16 weights (one record
// part: 64 KB of LDS) the encoder and the update fit 168 registers, which
// leaves room for three waves per SIMD: full event, update 0.203 -> 0.180 ms,
// encoder 0.132 -> 0.129 ms; the classifier ran slower that way (0.097 ->
// 0.101 ms), as did the bf16 hi/lo encoder and classifier, so they keep two.
template <int PREC, int MODE>
constexpr int edge_waves() {
  return PREC == F16W && MODE != (int)EdgeMode::Cls ? 12 : SW;
}

// Parts per weight record: two (f16x2 or bf16 hi/lo) or one (fp16 weights).
template <int PREC>
constexpr int rec_parts() { return PREC == F16W ? 1 : 2; }

// acc[mb] += w x over one k-step, one fp16 weight part (F16W).
template <int MB>
__device__ __forceinline__ void step_f(f16v (&acc)[MB], const h8 *rec, const h8 &x) {
  h8 w[MB];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) w[mb] = rec[mb * 64];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) acc[mb] = mma_h(w[mb], x, acc[mb]);
}

// step_f with the operands exchanged (transposed accumulators, as step_ht).
template <int MB>
__device__ __forceinline__ void step_ft(f16v (&acc)[MB], const h8 *rec, const h8 &x) {
  h8 w[MB];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) w[mb] = rec[mb * 64];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) acc[mb] = mma_h(x, w[mb], acc[mb]);
}

// F16W operands: a stored bf16 value is exactly an fp16 value once it lies
// in the fp16 range (the callers keep it there, scaling a node's aggregate
// row by a power of two where needed); an fp32 accumulator value is rounded
// to bf16 first (the model's activation precision) and then converted.
__device__ __forceinline__ h8 bf_to_h(const bf8 &x) {
  return __builtin_convertvector(__builtin_convertvector(x, f8), h8);
}
__device__ __forceinline__ h8 bf_to_h(const bf8 &x, float sv) {
  return __builtin_convertvector(__builtin_convertvector(x, f8) * sv, h8);
}
__device__ __forceinline__ h8 acc_to_h(const f8 &x) {
  return __builtin_convertvector(__builtin_convertvector(__builtin_convertvector(x, bf8), f8), h8);
}

template <int MB>
__device__ __forceinline__ void zero(f16v (&a)[MB]) {
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int v = 0; v < 16; ++v) a[mb][v] = 0.f;
}

// Stores the wave's 32 rows x 32 MB floats (row r at out + r * stride,
// rows >= nvalid skipped) through a 32 x 32-float LDS staging tile, one
// 128-byte column block at a time: every store instruction then writes 8
// full 128-byte lines instead of 32-byte pieces of 32 rows.
//
// Rows that a later kernel reads (h, P, e) are stored with the nontemporal
// hint.  Measured on the full fp32 event: 6.48 -> 6.28 ms with h, P and the
// updated e stored this way, the time saved showing up mostly in the
// kernels that read those rows next.
//
// The tile has 32 rows of 128 bytes (eight 16-byte chunks); chunk c of row r
// sits at chunk c ^ swz(r), swz(r) = r & 7.  Measured with the 16-byte
// accesses (row writes, one chunk per lane; column-block reads, eight lanes
// per row): no LDS bank conflicts, against 1.0M per 64k writes and reads
// for rows padded to 36 floats, 14.7M for unpadded rows and 2.1M for the
// swizzle (r >> 1) & 7.  The 8-byte writes of 16-bit h rows (store_block16)
// leave about 56 conflict cycles per 32-row unit (about 1 us of a 140 us
// node update): each half-wave writes one half of every chunk it touches,
// and the swizzle (r ^ (r >> 3)) & 7 gave the same count.
constexpr int SST = 32;  // staging row stride in floats
__device__ __forceinline__ int swz(int r) { return r & 7; }
template <int MB>
__device__ __forceinline__ void store_block(float *__restrict__ out, int64_t stride, int nvalid,
                                            const f16v (&acc)[MB], float *stg, int lane) {
  const int n = lane & 31, hh = lane >> 5;
  const int rr = lane >> 3, cc = lane & 7;
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) {
#pragma unroll
    for (int q = 0; q < 4; ++q)
      *(f4 *)(stg + n * SST + 4 * ((2 * q + hh) ^ swz(n))) =
          f4{acc[mb][4 * q], acc[mb][4 * q + 1], acc[mb][4 * q + 2], acc[mb][4 * q + 3]};
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int row = 8 * k + rr;
      const f4 v = *(const f4 *)(stg + row * SST + 4 * (cc ^ swz(row)));
      if (row < nvalid)
        __builtin_nontemporal_store(v, (f4 *)(out + row * stride + mb * 32 + 4 * cc));
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  }
}

// 16-bit rows (bf16 model: h in bf16, the projections in fp16) from
// accumulator blocks, through the same staging tile, two 32-feature blocks
// (128 bytes of a row) at a time, so that every store instruction writes 8
// full 128-byte lines.  PERM keeps feature 8 q + 4 hh + t of each block
// (q, t = 0..3) at position 16 hh + 4 q + t: the projections' order, in
// which a lane's 16 accumulator values of a block are contiguous (the edge
// kernel reads them back with two 16-byte loads per block).
template <int MB, bool PERM, typename T>
__device__ __forceinline__ void store_block16(T *__restrict__ out, int64_t stride, int nvalid,
                                              const f16v (&acc)[MB], float *stg, int lane) {
  typedef T t4 __attribute__((ext_vector_type(4)));
  typedef T t8 __attribute__((ext_vector_type(8)));
  static_assert(MB % 2 == 0, "two blocks per staging round");
  char *sb = (char *)stg;
  const int n = lane & 31, hh = lane >> 5;
  const int rr = lane >> 3, cc = lane & 7;
#pragma unroll
  for (int mp = 0; mp < MB / 2; ++mp) {
#pragma unroll
    for (int b = 0; b < 2; ++b) {
      const f16v &a = acc[2 * mp + b];
      // (chunk = 8 values; chunk c of row n at c ^ swz(n), as in store_block)
      if constexpr (PERM) {
        t8 lo, hi;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          lo[j] = (T)a[j];
          hi[j] = (T)a[8 + j];
        }
        *(t8 *)(sb + n * SST * 4 + 16 * ((4 * b + 2 * hh) ^ swz(n))) = lo;
        *(t8 *)(sb + n * SST * 4 + 16 * ((4 * b + 2 * hh + 1) ^ swz(n))) = hi;
      } else {
#pragma unroll
        for (int q = 0; q < 4; ++q)
          *(t4 *)(sb + n * SST * 4 + 16 * ((4 * b + q) ^ swz(n)) + 8 * hh) =
              t4{(T)a[4 * q], (T)a[4 * q + 1], (T)a[4 * q + 2], (T)a[4 * q + 3]};
      }
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int row = 8 * k + rr;
      const t8 v = *(const t8 *)(sb + row * SST * 4 + 16 * (cc ^ swz(row)));
      if (row < nvalid) __builtin_nontemporal_store(v, (t8 *)(out + row * stride + mp * 64 + cc * 8));
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  }
}

// Weight stream of the node kernel: all records of one tile, cut into chunks
// of NF4 float4 per thread (NF4 * 8 KB), double-buffered through LDS.  While
// the waves multiply out of one buffer, the next chunk is fetched from L2
// into registers and written into the other buffer; one barrier per chunk.
template <int NF4>
struct Stream {
  const f4 *base;
  int nchunks;
  f4 *buf;    // 2 x NF4 * 512 float4
  int c = 0;  // chunk index within the tile's stream
  int k = 0;  // chunks consumed so far (selects the buffer)
  f4 st[NF4];
  __device__ void fetch(int cc, int tid) {
    // a 32-bit byte offset from the uniform base (one register per address)
    const char *b = (const char *)base + (uint32_t)(cc * NF4 * 512 + tid) * 16u;
#pragma unroll
    for (int i = 0; i < NF4; ++i) st[i] = *(const f4 *)(b + i * 512 * 16);
  }
  __device__ void commit(int b, int tid) {
#pragma unroll
    for (int i = 0; i < NF4; ++i) buf[b * NF4 * 512 + i * 512 + tid] = st[i];
  }
  __device__ const f4 *begin(int tid) {
    __syncthreads();
    fetch((c + 1) % nchunks, tid);
    return buf + (k & 1) * NF4 * 512;
  }
  __device__ void end(int tid) {
    commit((k + 1) & 1, tid);
    ++k;
    c = (c + 1) % nchunks;
  }
};

// Chunks of the node kernels' weight stream.  Two-part records (f16x2, bf16
// hi/lo): 6 records, 48 KB (MB = 4), per update chunk and 4, 32 KB, per
// encoder chunk.  One-part records (fp16 weights): the same chunk bytes hold
// twice the records, except in the H = 64 encoder, whose 20 records take 4
// per chunk (16 KB-per-thread-slot chunks) so that the count divides.
template <int MB, bool ENC, int PREC>
constexpr int node_nf4() {
  return PREC == F16W && ENC && MB == 2 ? 1 : (ENC ? 4 * 2 : 4 * 3) * MB * 64 / 512;
}
template <int MB, bool ENC, int PREC>
constexpr int rpc_h() { return node_nf4<MB, ENC, PREC>() * 512 / (rec_parts<PREC>() * MB * 64); }
template <int MB, int PREC>
constexpr int rpc_l1() { return rpc_h<MB, false, PREC>(); }

// Records per 128-byte line pair of the node update's layer-1 inputs (two
// lanes read one line of a row): 2 for fp32 rows, 4 for bf16 rows.  The
// host packs those records in the same order (node_line_k in gnn_api.hip).
template <int PREC>
constexpr int line_group() { return PREC == SPLIT ? 2 : 4; }

template <int MB, bool ENC, int NPROJ, int PREC>
__global__ __launch_bounds__(64 * SW) void node_split(NodeArgs a) {
  constexpr int H = 32 * MB;
  constexpr int G = H / 16;  // k-steps per H-wide operand
  constexpr int NF4 = node_nf4<MB, ENC, PREC>();
  constexpr int RPC_H = rpc_h<MB, ENC, PREC>();
  constexpr int RPC_1 = rpc_l1<MB, PREC>();
  constexpr int REC_H = rec_parts<PREC>() * MB * 64;  // 16-byte slots per record
  constexpr int REC_1 = REC_H;
  static_assert(RPC_H * REC_H == NF4 * 512, "chunk size");
  static_assert(ENC || (3 * G) % RPC_1 == 0, "layer-1 records fill whole chunks");
  using act_t = typename std::conditional<PREC == SPLIT, float, __bf16>::type;
  __shared__ f4 wbuf[2 * NF4 * 512];
  __shared__ float stage[SW][32 * SST];
  // LayerNorm parameters of both layers, [b1 g1 beta1 b2 g2 beta2] with
  // each bias multiplied by its accumulator scale; the encoder adds its
  // first-layer bias and W^T ([F][H]).  Read from LDS, they stay off the
  // vector-memory counter that the row loads and stores wait on.
  constexpr int NPRM = 6 * H + NPROJ * H + (ENC ? H + MAX_F * H : 0);
  __shared__ float prm[NPRM];
  // (the projections' consumer biases, scaled, at prm + PB)
  constexpr int PB = 6 * H + (ENC ? H + MAX_F * H : 0);
  const int tid = threadIdx.x, lane = tid & 63, hh = lane >> 5, n = lane & 31;
  const int wave = tid >> 6;
  float *stg = stage[wave];
  for (int i = tid; i < H; i += 64 * SW) {
    prm[i] = ENC ? 0.f : a.mlp.l0.b[i] * a.s1;
    prm[H + i] = a.mlp.l0.g[i];
    prm[2 * H + i] = a.mlp.l0.beta[i];
    prm[3 * H + i] = a.mlp.l1.b[i] * a.s2;
    prm[4 * H + i] = a.mlp.l1.g[i];
    prm[5 * H + i] = a.mlp.l1.beta[i];
    if constexpr (ENC) prm[6 * H + i] = a.mlp.l0.b[i];
#pragma unroll
    for (int p = 0; p < NPROJ; ++p) prm[PB + p * H + i] = a.pbias[p][i] * a.ps1[p];
  }
  if constexpr (ENC)
    for (int i = tid; i < a.F * H; i += 64 * SW) prm[7 * H + i] = ((const float *)a.mlp.l0.w)[i];
  Stream<NF4> ws{(const f4 *)a.wstream, a.nchunks, wbuf};
  ws.fetch(0, tid);
  ws.commit(0, tid);
  __syncthreads();

  const float eps2 = a.eps * a.s2 * a.s2;
  const int blk = xcd_remap(blockIdx.x, gridDim.x);
  // Rounds of one 32-row unit per wave: K full rounds of SW units per
  // workgroup, then the remaining units spread over all workgroups (unit j
  // to workgroup j % grid, wave j / grid), so that the last round is not
  // carried by a few workgroups only.  A wave without a unit in the last
  // round keeps streaming the weights (barriers) and does nothing else.
  const int64_t G_ = gridDim.x;
  const int64_t full = 32 * SW * G_;
  const int64_t K = a.n_rows / full;
  const int64_t rem_units = (a.n_rows - K * full + 31) / 32;
  const int64_t rounds = K + (blk < rem_units ? 1 : 0);
  const int wv = __builtin_amdgcn_readfirstlane(wave);
  for (int64_t rd = 0; rd < rounds; ++rd) {
    // Keeps loop-invariant loads inside the loop (hoisted, they would stay
    // in registers for the whole kernel).
    asm volatile("" ::: "memory");
    const int64_t unit = rd < K ? (rd * G_ + blk) * SW + wv : K * full / 32 + wv * G_ + blk;
    const bool active = rd < K || wv * G_ + blk < rem_units;
    const int64_t wrow0 = unit * 32;  // the wave's first row (wave-uniform)
    const int nvalid = !active ? 0 : (int)(a.n_rows - wrow0 < 32 ? a.n_rows - wrow0 : 32);
    const int64_t row = wrow0 + n;
    const bool valid = n < nvalid;
    const int64_t r = valid ? row : (nvalid > 0 ? wrow0 + nvalid - 1 : 0);
    if (!active) {
      // one tile's worth of the weight stream: same barriers, same share
      // of every chunk fetch
      for (int c = 0; c < a.nchunks; ++c) {
        (void)ws.begin(tid);
        ws.end(tid);
      }
      continue;
    }

    f16v acc[MB];
    if constexpr (ENC) {
      // the bias is in the accumulators already (the LayerNorm adds zeros)
      small_k_layer<MB>(acc, a.x, a.F, (int)r, prm + 7 * H, prm + 6 * H, hh);
      ln_relu_lds<MB>(acc, prm, a.eps, hh);
    } else {
      // Layer 1 over [h; agg_in; agg_out]: 3G records.  The k-steps of each
      // source are taken in line order (node_line_k): the GRP records of a
      // group cover 16 GRP consecutive features, lanes n and n + 32 reading
      // the two 64-byte halves of one 128-byte line of row n, and a group's
      // records are requested together, one group ahead, into a ring of
      // two groups.
      zero<MB>(acc);
      constexpr int NREC = 3 * G, GRP = line_group<PREC>(), RING = 2 * GRP;
      static_assert(G % GRP == 0, "groups inside one source");
      // Addresses are a per-tile scalar base plus one 32-bit lane offset
      // shared by the three sources: 64-bit per-lane pointers cost the
      // registers that the look-ahead needs (a spill reload would wait for
      // every load in flight).
      const int64_t t0 = wrow0;
      const uint32_t roff =
          (uint32_t)((r - t0) * H + 8 * GRP * hh) * (uint32_t)sizeof(act_t);
      const act_t *const *srcs = (const act_t *const *)a.src;
      using xrec_t = typename std::conditional<PREC == SPLIT, f8, bf8>::type;
      auto load_rec = [&](int rec) {
        const int g = rec % G;
        const char *p = (const char *)(srcs[rec / G] + t0 * H) + roff +
                        (int)sizeof(act_t) * (16 * GRP * (g / GRP) + 8 * (g % GRP));
        if constexpr (PREC == SPLIT)
          return cat8(*(const f4 *)p, *(const f4 *)(p + 16));
        else
          return *(const bf8 *)p;
      };
      xrec_t xr[RING];
#pragma unroll
      for (int i = 0; i < GRP; ++i) xr[i] = load_rec(i);
      // Split and fp16 weights: the node's whole input row is multiplied by
      // a power of two sv <= 1 that keeps it inside the fp16 range of the
      // operands: the aggregates are bounded by max(deg_in, deg_out) times
      // the bound of a message row.  Column n of the product is then sv
      // times the node's, and is divided by sv again after the last record
      // (exact).
      float sv = 1.f, inv_sv = 1.f;
      if constexpr (PREC != BF16) {
        const int32_t din = a.rp_in[r + 1] - a.rp_in[r];
        const int32_t dout = a.rp_out[r + 1] - a.rp_out[r];
        const float m = (float)(din > dout ? (din > 1 ? din : 1) : (dout > 1 ? dout : 1)) *
                        a.row_bound;
        if (m > 32768.f) {
          int e = 0;
          (void)frexpf(m * (1.f / 32768.f), &e);  // m / 2^15 <= 2^e
          sv = ldexpf(1.f, -e);
          inv_sv = ldexpf(1.f, e);
        }
      }
      const f4 *w = nullptr;
#pragma unroll
      for (int i = 0; i < NREC; ++i) {
        if (i % GRP == 0 && i + GRP < NREC)
#pragma unroll
          for (int j = 0; j < GRP; ++j) xr[(i + GRP + j) % RING] = load_rec(i + GRP + j);
        // keeps the loads here: under register pressure the scheduler would
        // sink them next to their use and the look-ahead would be lost
        __builtin_amdgcn_sched_barrier(0);
        if (i % RPC_1 == 0) w = ws.begin(tid) + lane;
        if constexpr (PREC == SPLIT)
          step_h<MB>(acc, (const h8 *)(w + (i % RPC_1) * REC_1), xr[i % RING] * sv);
        else if constexpr (PREC == BF16)
          step_hl<MB>(acc, (const bf8 *)(w + (i % RPC_1) * REC_1), xr[i % RING]);
        else
          step_f<MB>(acc, (const h8 *)(w + (i % RPC_1) * REC_1), bf_to_h(xr[i % RING], sv));
        if (i % RPC_1 == RPC_1 - 1) ws.end(tid);
      }
      if constexpr (PREC != BF16) {
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) acc[mb] *= inv_sv;
      }
      ln_relu_lds<MB>(acc, prm, a.eps * a.s1 * a.s1, hh);
    }

    // Layer 2, then the projection halves.  Record i of this part sits in
    // chunk i / RPC_H at slot i % RPC_H.
    const f4 *wcur = nullptr;
    auto rec_h = [&](int i) {
      if (i % RPC_H == 0) wcur = ws.begin(tid) + lane;
      return wcur + (i % RPC_H) * REC_H;
    };
    auto rec_done = [&](int i) {
      if (i % RPC_H == RPC_H - 1) ws.end(tid);
    };
    f16v hv[MB];
    zero<MB>(hv);
#pragma unroll
    for (int g = 0; g < G; ++g) {
      if constexpr (PREC == SPLIT)
        step_h<MB>(hv, (const h8 *)rec_h(g), acc_x<MB>(acc, g));
      else if constexpr (PREC == BF16)
        step_hl<MB>(hv, (const bf8 *)rec_h(g), to_bf16(acc_x<MB>(acc, g)));
      else
        step_f<MB>(hv, (const h8 *)rec_h(g), acc_to_h(acc_x<MB>(acc, g)));
      rec_done(g);
    }
    ln_relu_lds<MB>(hv, prm + 3 * H, eps2, hh);
    if (a.h_out) {
      if constexpr (PREC == SPLIT)
        store_block<MB>(a.h_out + wrow0 * H, H, nvalid, hv, stg, lane);
      else
        store_block16<MB, false, __bf16>((__bf16 *)a.h_out + wrow0 * H, H, nvalid, hv, stg, lane);
    }
    // the projections read h as it is stored
    using xp_t = typename std::conditional<PREC == BF16, bf8, h8>::type;
    xp_t x1[G], x2[PREC == SPLIT ? G : 1];
#pragma unroll
    for (int g = 0; g < G; ++g) {
      if constexpr (PREC == SPLIT)
        split2(acc_x<MB>(hv, g), x1[g], x2[g]);
      else if constexpr (PREC == BF16)
        x1[g] = to_bf16(acc_x<MB>(hv, g));
      else
        x1[g] = acc_to_h(acc_x<MB>(hv, g));
    }
#pragma unroll
    for (int p = 0; p < NPROJ; ++p)
#pragma unroll
      for (int half = 0; half < 2; ++half) {
        f16v pv[MB];
        zero<MB>(pv);
#pragma unroll
        for (int g = 0; g < G; ++g) {
          const int i = G * (1 + 2 * p + half) + g;
          if constexpr (PREC == SPLIT)
            step_h<MB>(pv, (const h8 *)rec_h(i), x1[g], x2[g]);
          else if constexpr (PREC == BF16)
            step_hl<MB>(pv, (const bf8 *)rec_h(i), x1[g]);
          else
            step_f<MB>(pv, (const h8 *)rec_h(i), x1[g]);
          rec_done(i);
        }
        if (half == 0) {
          // the consumer's layer-1 bias, added once per node here rather
          // than once per edge in the edge kernel
#pragma unroll
          for (int mb = 0; mb < MB; ++mb)
#pragma unroll
            for (int q = 0; q < 4; ++q) {
              const f4 bb = *(const f4 *)(prm + PB + p * H + mb * 32 + 8 * q + 4 * hh);
#pragma unroll
              for (int t = 0; t < 4; ++t) pv[mb][4 * q + t] += bb[t];
            }
        }
        if constexpr (PREC == SPLIT)
          store_block<MB>(a.p_out[p] + wrow0 * 2 * H + half * H, 2 * H, nvalid, pv, stg, lane);
        else
          store_block16<MB, true, _Float16>((_Float16 *)a.p_out[p] + wrow0 * 2 * H + half * H,
                                            2 * H, nvalid, pv, stg, lane);
      }
  }
}

template <int MB, int MODE, int PREC>
__global__ __launch_bounds__((64 * edge_waves<PREC, MODE>())) void edge_split(EdgeArgs a) {
  constexpr int EW = edge_waves<PREC, MODE>();
  constexpr int H = 32 * MB;
  constexpr int G = H / 16;
  constexpr int RP = rec_parts<PREC>();
  constexpr int NR = G * MB * RP * 64;  // 16-byte slots of one H x H matrix
  using act_t = typename std::conditional<PREC == SPLIT, float, __bf16>::type;  // aggregates
  // edge rows: fp32, bf16, or bf16 values in fp16 encoding (F16W)
  using et_t = typename std::conditional<PREC == F16W, _Float16, act_t>::type;
  // ENC_UPD: the edge encoder, then the first update of the edges it
  // encoded, each unit's e0 kept in registers between the two (fp16
  // weights: their three H x H matrices fit in LDS together).
  constexpr bool ENC_UPD = MODE == (int)EdgeMode::EncUpdAgg;
  constexpr bool HAS_E = MODE != (int)EdgeMode::Enc && !ENC_UPD;  // e rows read from HBM
  constexpr bool HAS_WE = MODE != (int)EdgeMode::Enc;             // a W_e product
  constexpr bool HAS_L2 = MODE != (int)EdgeMode::Cls;
  constexpr bool FUSE = MODE == (int)EdgeMode::UpdAgg || ENC_UPD;
  // The update always sums its rows per source here (UpdAgg); the plain
  // update is the fp32-matrix-core kernel's (factored.hip).
  static_assert(MODE != (int)EdgeMode::Upd, "split kernels have no plain update");
  static_assert(!ENC_UPD || PREC == F16W, "the encoder runs inside the update with fp16 weights only");
  __shared__ h8 lds[(HAS_WE ? NR : 0) + (HAS_L2 ? NR : 0) + (ENC_UPD ? NR : 0)];
  __shared__ float prm[6 * H];  // s1 b1, gamma1, beta1, s2 b2, gamma2, beta2
  __shared__ float prm_enc[ENC_UPD ? 6 * H : 1];  // the same for the encoder
  const int lane = threadIdx.x & 63, hh = lane >> 5, n = lane & 31;
  const int blk = xcd_remap(blockIdx.x, gridDim.x);
  const int wv = threadIdx.x >> 6;
  const int64_t gw = (int64_t)blk * EW + wv;
  const int64_t nw = (int64_t)gridDim.x * EW;
  const int64_t units = (a.n_rows + 31) / 32;
  auto row_of = [&](int64_t u) {
    const int64_t row = u * 32 + n;
    return row < a.n_rows ? row : a.n_rows - 1;  // tail lanes recompute the last row
  };
  // The unit of round rd for this wave (-1: none).  Full rounds go
  // workgroup by workgroup (a workgroup's waves take consecutive units); the
  // last, partial round is spread over all workgroups, one wave of each
  // before any takes a second, so that it does not fall on a few CUs only.
  const int64_t full_rounds = units / nw;
  auto unit_at = [&](int64_t rd) -> int64_t {
    if (rd < full_rounds) return rd * nw + gw;
    const int64_t u = full_rounds * nw + (int64_t)wv * gridDim.x + blk;
    return rd == full_rounds && u < units ? u : -1;
  };

  // The next unit's edge indices and e row are requested before the
  // current unit's stores (vector-memory completions are counted in issue
  // order, so a load issued after a store is waited for with that store).
  using xrec_t = typename std::conditional<PREC == SPLIT, f8,
                                           typename std::conditional<PREC == F16W, h8, bf8>::type>::type;
  xrec_t ev[HAS_E ? G : 1];
  auto load_e = [&](int64_t rr) {
    const et_t *ep = (const et_t *)a.e_in + rr * H + 8 * hh;
#pragma unroll
    for (int g = 0; g < G; ++g) {
      if constexpr (PREC == SPLIT)
        ev[g] = cat8(*(const f4 *)(ep + 16 * g), *(const f4 *)(ep + 16 * g + 4));
      else
        ev[g] = *(const xrec_t *)(ep + 16 * g);
    }
  };
  // FUSE: the source of the rows just before and after this lane's row
  // (-1 / -2 outside the edge list) find the runs of equal sources.
  int32_t nsrc = 0, ndst = 0, nprev = -1, nnext = -2;
  auto load_idx = [&](int64_t uu) {
    const int64_t r0 = row_of(uu);
    nsrc = a.src_idx[r0];
    ndst = a.dst_idx[r0];
    if constexpr (FUSE) {
      const int64_t rr = uu * 32 + n;
      nprev = rr >= 1 && rr - 1 < a.n_rows ? a.src_idx[rr - 1] : -1;
      nnext = rr + 1 < a.n_rows ? a.src_idx[rr + 1] : -2;
    }
    // FUSE requests the e row at the end of the unit instead: the next
    // unit's first products wait for its P gathers, issued after this
    // unit's stores anyway, and the registers are needed until then.
    if constexpr (HAS_E && !FUSE) load_e(r0);
  };
  // The first unit's loads go out before the weights are copied into LDS.
  int64_t u = unit_at(0);
  if (u >= 0) {
    load_idx(u);
    if constexpr (FUSE && HAS_E) load_e(row_of(u));
  }
  h8 *lw_e = lds;
  h8 *lw_2 = lds + (HAS_WE ? NR : 0);
  h8 *lw_2enc = lw_2 + NR;  // ENC_UPD: the encoder's W2
  for (int i = threadIdx.x; i < NR; i += 64 * EW) {
    if constexpr (HAS_WE) lw_e[i] = ((const h8 *)a.we)[i];
    if constexpr (HAS_L2) lw_2[i] = ((const h8 *)a.w2)[i];
    if constexpr (ENC_UPD) lw_2enc[i] = ((const h8 *)a.enc.w2)[i];
  }
  for (int i = threadIdx.x; i < H; i += 64 * EW) {
    prm[i] = 0.f;  // (layer-1 bias: inside the gathered P[src] rows)
    prm[H + i] = a.g1[i];
    prm[2 * H + i] = a.beta1[i];
    if constexpr (HAS_L2) {
      prm[3 * H + i] = a.b2[i] * a.s2;
      prm[4 * H + i] = a.g2[i];
      prm[5 * H + i] = a.beta2[i];
    } else {
      prm[3 * H + i] = ((const float *)a.w2)[i];  // classifier head row
    }
    if constexpr (ENC_UPD) {
      prm_enc[i] = 0.f;
      prm_enc[H + i] = a.enc.g1[i];
      prm_enc[2 * H + i] = a.enc.beta1[i];
      prm_enc[3 * H + i] = a.enc.b2[i] * a.enc.s2;
      prm_enc[4 * H + i] = a.enc.g2[i];
      prm_enc[5 * H + i] = a.enc.beta2[i];
    }
  }
  __syncthreads();
  const float eps1 = a.eps * a.s1 * a.s1, eps2 = a.eps * a.s2 * a.s2;

  for (int64_t rd = 0; u >= 0; ++rd) {
    const int64_t un = unit_at(rd + 1);  // the next unit (-1: none)
    // Keeps the LDS record reads inside the loop (they are loop-invariant;
    // hoisted, they would pin every weight in registers).
    asm volatile("" ::: "memory");
    const int64_t row = u * 32 + n;
    const bool valid = row < a.n_rows;
    const int64_t s = clamp_idx(nsrc, a.n_nodes);
    const int64_t d = clamp_idx(ndst, a.n_nodes);

    // Layer 1 = s1 (P[src][0:H] + P[dst][H:2H] + W_e e) (+ s1 b1 in the LayerNorm).
    // The fp32 update and classifier raise the wave's priority while their
    // gathers are issued and summed, so that they go out ahead of the other
    // wave's products (full event: update 0.312 -> 0.308 ms, classifier
    // 0.189 -> 0.187 ms; the encoder and the 16-bit kernels lose by it).
    constexpr bool PRIO = PREC == SPLIT && MODE != (int)EdgeMode::Enc;
    if constexpr (PRIO) __builtin_amdgcn_s_setprio(3);
    f16v acc[MB];
    h8 xe[ENC_UPD ? G : 1];  // ENC_UPD: the unit's e0 as fp16 operands
    if constexpr (PREC == SPLIT) {
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
    } else {
      // fp16 rows in the order of store_block16: this lane's 16 values of
      // block mb are contiguous.  load16 fetches them from P[src][0:H] and
      // P[dst][H:2H] into raw[mb]; sum16 adds the two into acc[mb] in fp32.
      auto load16 = [&](const float *Pv, u4 (&raw)[MB][4]) {
        const _Float16 *ps = (const _Float16 *)Pv + s * 2 * H + 16 * hh;
        const _Float16 *pd = (const _Float16 *)Pv + d * 2 * H + H + 16 * hh;
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) {
          raw[mb][0] = *(const u4 *)(ps + 32 * mb);
          raw[mb][1] = *(const u4 *)(ps + 32 * mb + 8);
          raw[mb][2] = *(const u4 *)(pd + 32 * mb);
          raw[mb][3] = *(const u4 *)(pd + 32 * mb + 8);
        }
      };
      auto sum16 = [&](const u4 (&raw)[MB][4], int mb) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const unsigned a0 = raw[mb][0][j], b0 = raw[mb][2][j];
          const unsigned a1 = raw[mb][1][j], b1 = raw[mb][3][j];
          acc[mb][2 * j] = add_f16<false>(a0, b0);
          acc[mb][2 * j + 1] = add_f16<true>(a0, b0);
          acc[mb][8 + 2 * j] = add_f16<false>(a1, b1);
          acc[mb][8 + 2 * j + 1] = add_f16<true>(a1, b1);
        }
      };
      u4 raw[MB][4];
      if constexpr (ENC_UPD) {
        // The encoder, e0 = LN/ReLU(W2 LN/ReLU(P_enc[src][0:H] +
        // P_enc[dst][H:2H])), layer 2 untransposed: e0 ends in the layout
        // of the next product's operand.
        load16(a.enc.P, raw);
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) sum16(raw, mb);
        ln_relu_lds<MB, false>(acc, prm_enc, a.eps * a.enc.s1 * a.enc.s1, hh);
        h8 xa[G];
#pragma unroll
        for (int g = 0; g < G; ++g) xa[g] = acc_to_h(acc_x<MB>(acc, g));
        zero<MB>(acc);
#pragma unroll
        for (int g = 0; g < G; ++g) step_f<MB>(acc, lw_2enc + g * RP * MB * 64 + lane, xa[g]);
        ln_relu_lds<MB>(acc, prm_enc + 3 * H, a.eps * a.enc.s2 * a.enc.s2, hh);
        // The update's gathers.  Issued before that LayerNorm, to wait
        // under it, they spill registers and cost more than they hide (full
        // event 3.378 ms with the P[src] half there, 3.408 with both,
        // against 3.363).
        load16(a.P, raw);
        // e0 rounded as the encoder stores it (bf16 values); block mb of
        // the accumulators then takes the update's projections
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) {
          xe[2 * mb] = acc_to_h(acc_x<MB>(acc, 2 * mb));
          xe[2 * mb + 1] = acc_to_h(acc_x<MB>(acc, 2 * mb + 1));
          sum16(raw, mb);
        }
      } else {
        load16(a.P, raw);
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) sum16(raw, mb);
      }
    }
    if constexpr (PRIO) __builtin_amdgcn_s_setprio(0);
    if constexpr (ENC_UPD) {
#pragma unroll
      for (int g = 0; g < G; ++g) step_f<MB>(acc, lw_e + g * RP * MB * 64 + lane, xe[g]);
    }
    if constexpr (HAS_E) {
#pragma unroll
      for (int g = 0; g < G; ++g) {
        if constexpr (PREC == SPLIT)
          step_h<MB>(acc, lw_e + g * RP * MB * 64 + lane, ev[g]);
        else if constexpr (PREC == BF16)
          step_hl<MB>(acc, (const bf8 *)(lw_e + g * RP * MB * 64 + lane), ev[g]);
        else
          step_f<MB>(acc, lw_e + g * RP * MB * 64 + lane, ev[g]);
      }
    }
    // (FUSE: after layer 2's LayerNorm, which needs the registers)
    if constexpr (!FUSE)
      if (un >= 0) load_idx(un);
    ln_relu_lds<MB, false>(acc, prm, eps1, hh);  // bias inside P[src]

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
      // (the encoder and the fused update: layer 2 transposed, row-contiguous
      // e stores)
      // Layer 2 transposed: lane l holds feature 32 mb + n of the unit's
      // rows 8 (v / 4) + 4 hh + v % 4.
      f16v t2[MB];
      zero<MB>(t2);
#pragma unroll
      for (int g = 0; g < G; ++g) {
        if constexpr (PREC == SPLIT)
          step_ht<MB>(t2, lw_2 + g * RP * MB * 64 + lane, acc_x<MB>(acc, g));
        else if constexpr (PREC == BF16)
          step_hlt<MB>(t2, (const bf8 *)(lw_2 + g * RP * MB * 64 + lane), to_bf16(acc_x<MB>(acc, g)));
        else
          step_ft<MB>(t2, lw_2 + g * RP * MB * 64 + lane, acc_to_h(acc_x<MB>(acc, g)));
      }
      ln_relu_t<MB>(t2, prm + 3 * H, eps2, n);
      if constexpr (PREC != SPLIT) {
        // the stored rows are the bf16 values; the sums add exactly those
#pragma unroll
        for (int mb = 0; mb < MB; ++mb)
#pragma unroll
          for (int v = 0; v < 16; ++v) t2[mb][v] = (float)(__bf16)t2[mb][v];
      }
      // Bit e of `ends` marks the last row of a run of equal sources
      // (within the unit's valid rows); hc: the unit's first run began in
      // the previous unit; tc: its last run continues in the next one.  All
      // three are wave-uniform; taken before the next unit's indices replace
      // this unit's.
      const int nvalid = (int)(a.n_rows - u * 32 < 32 ? a.n_rows - u * 32 : 32);
      uint32_t ends = 0;
      bool hc = false, tc = false;
      int32_t cur_src = 0;
      if constexpr (FUSE) {
        ends = (uint32_t)__ballot(n < nvalid && (n == nvalid - 1 || nsrc != nnext));
        hc = __ballot(n == 0 && nprev == nsrc) != 0;
        tc = __ballot(n == 31 && nsrc == nnext) != 0;
        cur_src = nsrc;
        if (un >= 0) load_idx(un);
      }
      // e rows: each store writes 32 contiguous elements of a row per
      // half-wave (128 bytes fp32, 64 bytes bf16).  The update's rows go
      // out nontemporal, as the node kernel's (the aggregation that reads
      // them next: 0.136 -> 0.128 ms); the encoder's gain nothing from it.
      et_t *eo = (et_t *)a.e_out + (u * 32 + 4 * hh) * H + n;
      auto st_e = [&](et_t *p, float x) {
        if constexpr (FUSE)
          __builtin_nontemporal_store((et_t)x, p);
        else
          *p = (et_t)x;
      };
      if (nvalid == 32) {
#pragma unroll
        for (int v = 0; v < 16; ++v)
#pragma unroll
          for (int mb = 0; mb < MB; ++mb) st_e(&eo[(8 * (v / 4) + v % 4) * H + 32 * mb], t2[mb][v]);
      } else {
#pragma unroll
        for (int v = 0; v < 16; ++v)
          if (8 * (v / 4) + 4 * hh + v % 4 < nvalid)
#pragma unroll
            for (int mb = 0; mb < MB; ++mb) st_e(&eo[(8 * (v / 4) + v % 4) * H + 32 * mb], t2[mb][v]);
      }
      if constexpr (FUSE) {
      // Exchange halves: afterwards lane l holds block b = p + hh MB/2 of
      // all 32 rows, rows 8 (v / 4) + v % 4 in t2[p][v] and rows
      // 8 (v / 4) + 4 + v % 4 in t2[p + MB/2][v].
      // (Elements are copied to scalars first: this compiler's
      // __builtin_bit_cast of a vector element reads element 0.)
#pragma unroll
      for (int p = 0; p < MB / 2; ++p)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const unsigned lo = __float_as_uint(t2[p][v]);
          const unsigned hi = __float_as_uint(t2[p + MB / 2][v]);
          const auto r = __builtin_amdgcn_permlane32_swap(lo, hi, false, false);
          const unsigned r0 = r[0], r1 = r[1];
          t2[p][v] = __uint_as_float(r0);
          t2[p + MB / 2][v] = __uint_as_float(r1);
        }
      // Run sums in row order, one feature of MB/2 blocks per lane.
      float sum[MB / 2];
#pragma unroll
      for (int p = 0; p < MB / 2; ++p) sum[p] = 0.f;
#pragma unroll
      for (int e = 0; e < 32; ++e) {
        const int v = 4 * (e / 8) + e % 4;
#pragma unroll
        for (int p = 0; p < MB / 2; ++p) sum[p] += (e / 4) % 2 ? t2[p + MB / 2][v] : t2[p][v];
        if (ends & (1u << e)) {
          const bool first = (ends & ((1u << e) - 1u)) == 0u;
          const bool last = (ends >> e) == 1u;
          // pieces stay fp32; a complete run is stored in the row type
          if ((first && hc) || (last && tc)) {
            float *dst = a.agg_part + (u * 2 + (first && hc ? 0 : 1)) * H;
#pragma unroll
            for (int p = 0; p < MB / 2; ++p) dst[32 * (p + hh * (MB / 2)) + n] = sum[p];
          } else {  // (read by the node update: nontemporal, as e)
            act_t *dst = (act_t *)a.agg_out + (int64_t)__builtin_amdgcn_readlane(cur_src, e) * H;
#pragma unroll
            for (int p = 0; p < MB / 2; ++p)
              __builtin_nontemporal_store((act_t)sum[p], &dst[32 * (p + hh * (MB / 2)) + n]);
          }
#pragma unroll
          for (int p = 0; p < MB / 2; ++p) sum[p] = 0.f;
        }
      }
      if constexpr (HAS_E)
        if (un >= 0) load_e(row_of(un));
      }
    }
    u = un;
  }
}

template <int MB, int PREC>
hipError_t node_h(bool enc, const NodeArgs &a, int grid, hipStream_t stream) {
  const int64_t tiles = (a.n_rows + 32 * SW - 1) / (32 * SW);
  if (tiles <= 0) return hipSuccess;
  const unsigned nb = (unsigned)(tiles < grid ? tiles : grid);
  if (!enc) return launch(node_split<MB, false, 1, PREC>, nb, 64 * SW, 0, stream, a);
  if (a.nproj == 2) return launch(node_split<MB, true, 2, PREC>, nb, 64 * SW, 0, stream, a);
  return launch(node_split<MB, true, 1, PREC>, nb, 64 * SW, 0, stream, a);
}

template <int MB, int PREC, int MODE>
hipError_t edge_go(const EdgeArgs &a, int grid, hipStream_t stream) {
  constexpr int EW = edge_waves<PREC, MODE>();
  const int64_t units = (a.n_rows + 31) / 32;
  const int64_t need = (units + EW - 1) / EW;
  if (need <= 0) return hipSuccess;
  const unsigned nb = (unsigned)(need < grid ? need : grid);
  return launch(edge_split<MB, MODE, PREC>, nb, 64 * EW, 0, stream, a);
}

template <int MB, int PREC>
hipError_t edge_h(EdgeMode mode, const EdgeArgs &a, int grid, hipStream_t stream) {
  switch (mode) {
    case EdgeMode::Enc: return edge_go<MB, PREC, 0>(a, grid, stream);
    case EdgeMode::Upd: return hipErrorInvalidValue;  // always UpdAgg here
    case EdgeMode::Cls: return edge_go<MB, PREC, 2>(a, grid, stream);
    case EdgeMode::UpdAgg:
      if (!a.agg_out || !a.agg_part) return hipErrorInvalidValue;
      return edge_go<MB, PREC, 3>(a, grid, stream);
    case EdgeMode::EncUpdAgg:
      if constexpr (PREC == F16W) {
        if (!a.agg_out || !a.agg_part || !a.enc.P || !a.enc.w2) return hipErrorInvalidValue;
        return edge_go<MB, PREC, 4>(a, grid, stream);
      }
      return hipErrorInvalidValue;
  }
  return hipErrorInvalidValue;
}

template <int MB, int PREC>
const void *edge_fn_mb(EdgeMode mode) {
  switch (mode) {
    case EdgeMode::Enc: return (const void *)edge_split<MB, 0, PREC>;
    case EdgeMode::Cls: return (const void *)edge_split<MB, 2, PREC>;
    case EdgeMode::Upd:  // not launched here (UpdAgg is)
    case EdgeMode::UpdAgg: return (const void *)edge_split<MB, 3, PREC>;
    case EdgeMode::EncUpdAgg:
      if constexpr (PREC == F16W) return (const void *)edge_split<MB, 4, PREC>;
      return nullptr;
  }
  return (const void *)edge_split<MB, 3, PREC>;
}

template <int PREC>
const void *edge_fn(EdgeMode mode, int hidden) {
  return hidden == 64 ? edge_fn_mb<2, PREC>(mode) : edge_fn_mb<4, PREC>(mode);
}

}  // namespace

// Chunks of a node stream: the encoder holds (1 + 2 nproj) H x H matrices
// of 2-part records; the update 3H/16 layer-1 records (3 parts when split, 2
// in bf16) and three H x H matrices.
int node_split_chunks(bool enc, int hidden, int nproj, int prec) {
  const int G = hidden / 16;
  auto chunks = [&](auto mbc, auto pc) {
    constexpr int MB = decltype(mbc)::value, PREC = decltype(pc)::value;
    return enc ? (G * (1 + 2 * nproj)) / rpc_h<MB, true, PREC>()
               : (3 * G) / rpc_l1<MB, PREC>() + (3 * G) / rpc_h<MB, false, PREC>();
  };
  using I2 = std::integral_constant<int, 2>;
  using I4 = std::integral_constant<int, 4>;
  using PS = std::integral_constant<int, SPLIT>;
  using PB = std::integral_constant<int, BF16>;
  using PF = std::integral_constant<int, F16W>;
  if (hidden == 64) return prec == 2 ? chunks(I2{}, PF{}) : prec == 1 ? chunks(I2{}, PB{}) : chunks(I2{}, PS{});
  return prec == 2 ? chunks(I4{}, PF{}) : prec == 1 ? chunks(I4{}, PB{}) : chunks(I4{}, PS{});
}

template <int MB>
hipError_t node_p(int prec, bool enc, const NodeArgs &a, int grid, hipStream_t stream) {
  switch (prec) {
    case 0: return node_h<MB, SPLIT>(enc, a, grid, stream);
    case 1: return node_h<MB, BF16>(enc, a, grid, stream);
    case 2: return node_h<MB, F16W>(enc, a, grid, stream);
  }
  return hipErrorInvalidValue;
}

hipError_t launch_node_split(bool enc, int hidden, const NodeArgs &a, int grid, int prec,
                             hipStream_t stream) {
  if (a.F > MAX_F || a.nproj < 1 || a.nproj > 2 || (!enc && a.nproj != 1) || grid <= 0)
    return hipErrorInvalidValue;
  if (a.nchunks != node_split_chunks(enc, hidden, a.nproj, prec)) return hipErrorInvalidValue;
  switch (hidden) {
    case 64: return node_p<2>(prec, enc, a, grid, stream);
    case 128: return node_p<4>(prec, enc, a, grid, stream);
  }
  return hipErrorInvalidValue;
}

int edge_split_grid(EdgeMode mode, int hidden, int prec, int n_cu) {
  const void *fn = prec == 2 ? edge_fn<F16W>(mode, hidden)
                             : prec == 1 ? edge_fn<BF16>(mode, hidden) : edge_fn<SPLIT>(mode, hidden);
  if (!fn) return 0;  // (the fused encoder + update exists with fp16 weights only)
  const int m = mode == EdgeMode::Enc ? 0 : mode == EdgeMode::Cls ? 2 : mode == EdgeMode::EncUpdAgg ? 4 : 3;
  auto waves = [&](auto pc) {
    constexpr int P = decltype(pc)::value;
    return m == 0 ? edge_waves<P, 0>() : m == 2 ? edge_waves<P, 2>() : m == 4 ? edge_waves<P, 4>() : edge_waves<P, 3>();
  };
  const int threads = 64 * (prec == 2 ? waves(std::integral_constant<int, F16W>{})
                            : prec == 1 ? waves(std::integral_constant<int, BF16>{})
                                        : waves(std::integral_constant<int, SPLIT>{}));
  int per_cu = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, fn, threads, 0) != hipSuccess ||
      per_cu < 1)
    per_cu = 1;
  return per_cu * (n_cu > 0 ? n_cu : 1);
}

template <int MB>
hipError_t edge_p(int prec, EdgeMode mode, const EdgeArgs &a, int grid, hipStream_t stream) {
  switch (prec) {
    case 0: return edge_h<MB, SPLIT>(mode, a, grid, stream);
    case 1: return edge_h<MB, BF16>(mode, a, grid, stream);
    case 2: return edge_h<MB, F16W>(mode, a, grid, stream);
  }
  return hipErrorInvalidValue;
}

hipError_t launch_edge_split(EdgeMode mode, int hidden, const EdgeArgs &a, int grid, int prec,
                             hipStream_t stream) {
  if (grid <= 0) return hipErrorInvalidValue;
  switch (hidden) {
    case 64: return edge_p<2>(prec, mode, a, grid, stream);
    case 128: return edge_p<4>(prec, mode, a, grid, stream);
  }
  return hipErrorInvalidValue;
}

}  // namespace gnn
