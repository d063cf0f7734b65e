// Internal declarations shared by the host runtime and the kernel files of
// libgnn.so.  Nothing here is part of the public ABI (include/gnn.h).
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>

namespace gnn {

// Activation storage type of a handle.
enum class Act : int { F32 = 0, BF16 = 1 };

// One Linear layer on the device.  `w` is laid out for the kernel that reads
// it: MFMA operand fragments for the dense layers, plain [out][in] rows for
// the small-K node-encoder layer and the classifier's H->1 head.
struct LayerDev {
  const void *w = nullptr;
  const void *w_lo = nullptr;   // bf16 mode: W - bf16(W), same fragment order

  const float *b = nullptr;
  const float *g = nullptr;     // LayerNorm gamma (nullptr for the head)
  const float *beta = nullptr;  // LayerNorm beta
};

struct MlpDev {
  LayerDev l0, l1;
};

// Arguments of the fused gather-MLP kernel family.  Rows are edges (edge
// encoder, edge update, classifier) or nodes (node encoder, node update).
// Row r of the layer-1 input is the concatenation over s < nsrc of
// src[s][idx[s] ? idx[s][r] : r][0 .. H-1]; gathered indices are clamped to
// [0, n_nodes) so that an invalid index can never fault.
struct GmlpArgs {
  int64_t n_rows = 0;
  int32_t n_nodes = 0;
  const void *src[3] = {nullptr, nullptr, nullptr};
  const int32_t *idx[3] = {nullptr, nullptr, nullptr};
  const float *x = nullptr;  // node encoder: raw features [n_rows][F]
  int32_t F = 0;
  MlpDev mlp;
  void *out = nullptr;          // [n_rows][H] activations (hidden MLPs)
  float *out_logit = nullptr;   // classifier outputs, [n_rows]
  float *out_score = nullptr;
  float eps = 1e-5f;
};

enum class GmlpKind : int { NodeEnc = 0, EdgeEnc = 1, EdgeUpd = 2, NodeUpd = 3, Classifier = 4 };

// Every launcher enqueues on `stream` and returns the launch status.
hipError_t launch_gmlp(GmlpKind kind, Act act, int hidden, const GmlpArgs &a, hipStream_t stream);

// Deterministic CSR segmented sums of the edge rows `e` ([n_edges][H]):
// agg_in[v] = sum over p in [rp_in[v], rp_in[v+1]) of e[perm_in[p]], in
// ascending p, and the same for agg_out.  fp32 accumulation in both modes.
hipError_t launch_segsum(Act act, int hidden, const void *e, const int32_t *rp_in,
                         const int32_t *perm_in, const int32_t *rp_out, const int32_t *perm_out,
                         void *agg_in, void *agg_out, int32_t n_nodes, hipStream_t stream);

// Stable CSR of `keys` (n_edges int32 in [0, n_nodes), clamped if not):
// row_ptr[n_nodes+1] and perm[n_edges] (edge ids, ascending within a row).
struct CsrScratch {
  uint32_t *keys_a, *keys_b, *vals_a, *vals_b;  // n_edges each
  uint32_t *hist;                               // csr_hist_len(n_edges)
};
size_t csr_hist_len(int64_t n_edges);
hipError_t build_csr(const int32_t *keys, int32_t n_edges, int32_t n_nodes, int32_t *row_ptr,
                     int32_t *perm, const CsrScratch &s, hipStream_t stream);

// flag <- 1 if any of the 2*n_edges indices lies outside [0, n_nodes).
hipError_t launch_validate(const int32_t *edge_index, int64_t n_edges, int32_t n_nodes,
                           int32_t *flag, hipStream_t stream);
hipError_t launch_fill_i32(int32_t *p, int64_t n, int32_t v, hipStream_t stream);
// bf16 rows -> fp32 rows (debug export).
hipError_t launch_bf16_to_f32(const void *in, float *out, int64_t n, hipStream_t stream);

}  // namespace gnn
