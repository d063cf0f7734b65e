// Internal declarations shared by the host runtime and the kernel files of
// libgnn.so.  Nothing here is part of the public ABI (include/gnn.h).
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>
#include <tuple>
#include <utility>

struct gnn_handle;

namespace gnn {

// Events of the stage being timed on this thread (profiling on), bound to the
// dispatches of the stage's kernels rather than recorded between them: the
// first kernel launched in the stage marks `start` when it begins, and every
// kernel marks `stop` when it ends (the last one's stands).  Both are null
// when no stage is being timed.
struct StageEvents {
  hipEvent_t start = nullptr, stop = nullptr;
  bool launched = false;
};
StageEvents &stage_events();  // this thread's

template <typename K, typename T, size_t... I>
hipError_t launch_args(K k, dim3 grid, dim3 block, size_t shmem, hipStream_t stream, T &t,
                       std::index_sequence<I...>) {
  void *argv[] = {(void *)&std::get<I>(t)...};
  StageEvents &ev = stage_events();
  if (!ev.stop) return hipLaunchKernel((const void *)k, grid, block, argv, shmem, stream);
  const hipError_t e =
      hipExtLaunchKernel((const void *)k, grid, block, argv, shmem, stream, ev.start, ev.stop, 0);
  if (e == hipSuccess) {
    ev.start = nullptr;
    ev.launched = true;
  }
  return e;
}

// Launches kernel k(args...) on `stream` with the timed stage's events, if
// any (StageEvents).  Returns the launch status, which the runtime also
// leaves for hipGetLastError().
template <typename... P, typename... A>
hipError_t launch(void (*k)(P...), dim3 grid, dim3 block, size_t shmem, hipStream_t stream,
                  A &&...args) {
  static_assert(sizeof...(P) == sizeof...(A), "kernel argument count");
  std::tuple<P...> t(std::forward<A>(args)...);
  return launch_args(k, grid, block, shmem, stream, t, std::index_sequence_for<P...>{});
}

// Activation storage type of a handle.
// Row element types.  F16 is used only for the edge rows of the bf16 model
// with fp16 weights: their values are bf16 numbers, held in fp16 encoding so
// that the fp16 products read them as they are.
enum class Act : int { F32 = 0, BF16 = 1, F16 = 2 };

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

// ---- fp32 kernels with the edge MLPs' first layer regrouped per node ----
// (factored.hip).  P rows are [W_s h_v ; W_d h_v], 2H floats per node.
struct NodeArgs {
  int64_t n_rows = 0;
  const float *x = nullptr;  // encoder: raw features [n_rows][F]
  int32_t F = 0;
  const float *src[3] = {nullptr, nullptr, nullptr};  // update: h, agg_in, agg_out
  MlpDev mlp;                 // biases and LayerNorm parameters; encoder W1 rows
  const float *wstream = nullptr;  // fragment stream: [W1 (update only)] W2 proj...
  int32_t nchunks = 0;             // chunks of the stream (8 k-groups each)
  int32_t nproj = 1;
  float *h_out = nullptr;                     // [n_rows][H] or nullptr
  float *p_out[2] = {nullptr, nullptr};       // [n_rows][2H]
  float eps = 1e-5f;
  // split kernels: power-of-two scales of the layer-1 (update) and layer-2
  // weights; the CSR row pointers and the bound of an h or message row
  // entry, which give each node's aggregate bound (update only)
  float s1 = 1.f, s2 = 1.f;
  const int32_t *rp_in = nullptr, *rp_out = nullptr;
  float row_bound = 0.f;
  // split kernels: the layer-1 bias of the edge MLP that reads projection
  // p, and that MLP's layer-1 scale; the bias goes into the source half
  // P[v][0:H] as the rows are stored, so the edge kernels add none
  const float *pbias[2] = {nullptr, nullptr};
  float ps1[2] = {1.f, 1.f};
};

// UpdAgg: the edge update that also sums its output rows per source node
// (split kernels, fp32 or bf16 rows).  It needs the rows in source order:
// every run of equal src_idx is one node's complete out-edge list.
// EncUpdAgg (fp16 weights only): the edge encoder and the first UpdAgg in
// one pass, e0 handed from one to the other in registers.
enum class EdgeMode : int { Enc = 0, Upd = 1, Cls = 2, UpdAgg = 3, EncUpdAgg = 4 };

struct EdgeArgs {
  int64_t n_rows = 0;
  int32_t n_nodes = 0;
  const int32_t *src_idx = nullptr, *dst_idx = nullptr;
  const float *P = nullptr;      // [n_nodes][2H]
  const float *e_in = nullptr;   // [n_rows][H] (update, classifier)
  const float *we = nullptr;     // fragments of W_e (H x H)
  const float *b1 = nullptr, *g1 = nullptr, *beta1 = nullptr;
  const float *w2 = nullptr;     // fragments of W2 (H x H), or the classifier head [H]
  const float *b2 = nullptr, *g2 = nullptr, *beta2 = nullptr;
  float *e_out = nullptr, *out_logit = nullptr, *out_score = nullptr;
  // classifier: row r's outputs go to position out_idx[r] (nullptr: r)
  const int32_t *out_idx = nullptr;
  float eps = 1e-5f;
  // split kernels: power-of-two scales of the first layer (W_e and the
  // stored P rows) and of W2
  float s1 = 1.f, s2 = 1.f;
  // UpdAgg: the sum of every run of rows with one source node that lies
  // inside one 32-row unit goes to agg_out[src] (row type); a run cut by a
  // unit boundary leaves its piece in agg_part[unit][0] (the unit's first
  // run, continued from the previous unit) or agg_part[unit][1] (its last
  // run, continued in the next), H fp32 each, for launch_segsum_fused.
  void *agg_out = nullptr;
  float *agg_part = nullptr;
  // EncUpdAgg: the edge encoder's projections, W2 records (B operand from
  // the accumulators), LayerNorm parameters and first-layer / W2 scales.
  // The update's W_e records (`we`) then read e0 from the accumulators too.
  struct {
    const float *P = nullptr, *w2 = nullptr;
    const float *g1 = nullptr, *beta1 = nullptr, *b2 = nullptr, *g2 = nullptr, *beta2 = nullptr;
    float s1 = 1.f, s2 = 1.f;
  } enc;
};

hipError_t launch_node_f32(bool enc, int hidden, const NodeArgs &a, int grid,
                           hipStream_t stream);
int node_f32_grid(int n_cu);
int node_stream_chunk_f4(int hidden);
// `grid` = number of persistent workgroups (edge_f32_grid).
hipError_t launch_edge_f32(EdgeMode mode, int hidden, const EdgeArgs &a, int grid,
                           hipStream_t stream);
int edge_f32_grid(EdgeMode mode, int hidden, int n_cu);

// The same kernels on the fp16/bf16 matrix cores (split.hip), by `prec`:
// 0 = fp32 model, split-precision products (fp32 P rows); 1 = bf16 model
// (h, e and the aggregates in bf16, hi/lo bf16 weights, fp16 P rows);
// 2 = the bf16 model with fp16 weights (one product per weight).  Weights
// come as 16-bit records; P rows are stored multiplied by the consumer's s1.
hipError_t launch_node_split(bool enc, int hidden, const NodeArgs &a, int grid, int prec,
                             hipStream_t stream);
int node_split_chunks(bool enc, int hidden, int nproj, int prec);
hipError_t launch_edge_split(EdgeMode mode, int hidden, const EdgeArgs &a, int grid, int prec,
                             hipStream_t stream);
int edge_split_grid(EdgeMode mode, int hidden, int prec, int n_cu);  // 0: no such kernel

// Deterministic CSR segmented sums of the edge rows `e` ([n_edges][H]):
// agg_in[v] = sum over p in [rp_in[v], rp_in[v+1]) of e[perm_in[p]], in
// ascending p, and the same for agg_out; a null perm is the identity.  fp32
// accumulation in both modes.
hipError_t launch_segsum(Act act, int hidden, const void *e, const int32_t *rp_in,
                         const int32_t *perm_in, const int32_t *rp_out, const int32_t *perm_out,
                         void *agg_in, void *agg_out, int32_t n_nodes, hipStream_t stream);
// Rows in source order after an UpdAgg edge update: agg_in as above;
// agg_out[v] is completed for the nodes whose out-edge positions
// [rp_out[v], rp_out[v+1]) span several 32-row units (sum of the fp32 unit
// pieces in agg_part, in unit order) and zeroed for nodes without out-edges;
// the edge update wrote every other row.  act = Act::F16: fp16 edge rows,
// bf16 aggregates.
hipError_t launch_segsum_fused(Act act, int hidden, const void *e, const int32_t *rp_in,
                               const int32_t *perm_in, const int32_t *rp_out,
                               const float *agg_part, void *agg_in, void *agg_out,
                               int32_t n_nodes, int64_t n_edges, hipStream_t stream);

// Stable CSRs of edge_index ([2][n_edges] int32, indices clamped into
// [0, n_nodes)): by destination (row_ptr_in, perm_in) and by source
// (row_ptr_out, perm_out); row_ptr has n_nodes+1 entries, perm lists edge
// ids ascending within each row.  Both sorts run in the same launches.
struct CsrScratch {
  uint2 *pairs_a, *pairs_b;  // 2*n_edges (key, edge id) pairs each
  // look-back words of the sort passes, digit totals, tile counters and an
  // error word: csr_scratch_bytes(n_edges, n_nodes) bytes, 4-byte aligned
  uint32_t *status;
};
// The sort's look-back words hold counts below 2^30: builds of at most
// CSR_MAX_ITEMS - 1 edges (larger ones return hipErrorInvalidValue).
constexpr int32_t CSR_MAX_ITEMS = 1 << 30;
size_t csr_scratch_bytes(int64_t n_edges, int64_t n_nodes);
// Nonzero after a build in which a sort pass gave up waiting for an earlier
// tile (a bounded wait that forward progress of running workgroups ends).
uint32_t *csr_err_word(const CsrScratch &s, int64_t n_edges, int64_t n_nodes);
// Destination- and source-sorted CSR of edge_index (stable: ascending edge id
// within a row).  With eis set (regrouped kernels) it also writes the edges
// in source order, eis[0][p] = src[perm_out[p]], eis[1][p] = dst[perm_out[p]]
// (clamped into [0, n_nodes)), inv[j] = source-order position of edge j, and
// q_in[k] = inv[perm_in[k]].
hipError_t build_csr(const int32_t *edge_index, int32_t n_edges, int32_t n_nodes,
                     int32_t *row_ptr_in, int32_t *perm_in, int32_t *row_ptr_out,
                     int32_t *perm_out, const CsrScratch &s, int32_t *eis, int32_t *inv,
                     int32_t *q_in, hipStream_t stream);
// dst[idx[r]][:] = src[r][:] (fp32, bf16 or fp16 rows of width H, written as fp32).
hipError_t launch_scatter_rows(Act act, const void *src, const int32_t *idx, float *dst,
                               int64_t rows, int H, hipStream_t stream);

// Edge filter (filter.hip): scores[j] = sigmoid(MLP([x_src; x_dst])).
struct FilterArgs {
  int64_t n_edges = 0;
  int32_t n_nodes = 0;
  const float *x = nullptr;  // [n_nodes][F]
  int32_t F = 0;
  const int32_t *edge_index = nullptr;
  const float *w0t = nullptr, *b0 = nullptr, *g0 = nullptr, *beta0 = nullptr;  // W0 as [2F][H]
  const float *w1 = nullptr, *b1 = nullptr, *g1 = nullptr, *beta1 = nullptr;   // fragments
  // f16x2 records of s1 W1 (layer 2 on the fp16 matrix cores); nullptr: the
  // fp32 fragments w1 are used
  const void *w1r = nullptr;
  float s1 = 1.f;
  const float *w2 = nullptr, *b2 = nullptr;                                   // head [H], [1]
  float *scores = nullptr;
  float eps = 1e-5f;
};
hipError_t launch_filter_scores(int hidden, const FilterArgs &a, hipStream_t stream);
// Stable compaction of the edges with score > threshold into out
// ([2][total] contiguous); counts has compact_tiles(n) entries.
size_t compact_tiles(int64_t n);
hipError_t launch_compact(const float *scores, const int32_t *edge_index, int64_t n,
                          float threshold, int32_t *counts, int32_t *total, int32_t *out,
                          hipStream_t stream);

// Graph construction (graph.hip).  Embedding MLP F -> H -> H -> D.
struct EmbedArgs {
  int64_t n = 0;
  const float *x = nullptr;  // [n][F]
  int32_t F = 0, D = 0;
  const float *w0t = nullptr, *b0 = nullptr, *g0 = nullptr, *beta0 = nullptr;  // W0 as [F][H]
  const float *w1 = nullptr, *b1 = nullptr, *g1 = nullptr, *beta1 = nullptr;   // fragments
  // f16x2 records of s1 W1 (layer 2 on the fp16 matrix cores); nullptr: the
  // fp32 fragments w1 are used
  const void *w1r = nullptr;
  float s1 = 1.f;
  const float *w2 = nullptr, *b2 = nullptr;                                   // [D][H], [D]
  float *z = nullptr;                                                         // [n][D]
  float eps = 1e-5f;
};
hipError_t launch_embed(int hidden, const EmbedArgs &a, hipStream_t stream);

// Fixed-radius pairs over the rows of z [n][D].
struct FrnnArgs {
  const float *z = nullptr;
  int64_t n = 0;
  int32_t D = 0, g = 0;       // dimensions, grid dimensions (min(3, D))
  float r2 = 0.f, inv_cell = 0.f;
  uint32_t mask = 0;          // bucket table size - 1 (power of two)
  const int32_t *rp = nullptr, *perm = nullptr;  // buckets: CSR of the points by key
  int32_t *count = nullptr;   // [n] pairs per point
  int64_t *offs = nullptr;    // [n] exclusive offsets
  int64_t *bsum = nullptr;    // [frnn_scan_blocks(n)] scan scratch
  int64_t *total_dev = nullptr;
  int64_t total = 0;          // fill pass: number of pairs (row stride of out)
  int32_t *out = nullptr;     // [2][total]
};
size_t frnn_scan_blocks(int64_t n);
hipError_t launch_frnn_keys(const FrnnArgs &a, int32_t *keys, hipStream_t stream);
// zs: [n][D] scratch for the coordinates in bucket order
hipError_t launch_frnn_count(const FrnnArgs &a, float *zs, hipStream_t stream);
hipError_t launch_frnn_fill(const FrnnArgs &a, const float *zs, hipStream_t stream);

// Weakly-connected components (wcc.hip): labels <- identity, then rounds of
// hooking over the kept edges and pointer jumping; `changed` (zero on entry)
// is set to 1 by a round that joined two trees.  A round whose `prev` (the
// previous round's flag; nullptr in the first round) is 0 does nothing.
hipError_t wcc_launch_init(int32_t *labels, int32_t n, hipStream_t stream);
hipError_t wcc_launch_round(const int32_t *edge_index, const float *scores, float threshold,
                            int64_t n_edges, int32_t n_nodes, int32_t *labels,
                            const int32_t *prev, int32_t *changed, hipStream_t stream);

// flag <- 1 if any of the 2*n_edges indices lies outside [0, n_nodes).
hipError_t launch_validate(const int32_t *edge_index, int64_t n_edges, int32_t n_nodes,
                           int32_t *flag, hipStream_t stream);
hipError_t launch_fill_i32(int32_t *p, int64_t n, int32_t v, hipStream_t stream);
// bf16 rows -> fp32 rows (debug export).
hipError_t launch_bf16_to_f32(const void *in, float *out, int64_t n, hipStream_t stream);

// Detaches a handle's cached workspaces from a stream about to be destroyed
// (host; the stream's work must have finished).
void ws_forget_stream(gnn_handle *h, hipStream_t stream);

// Sets the calling thread's gnn_last_error() text; returns code (host).
int set_error(int code, const char *msg);

// Device address and size of the no-allocation entry point's scratch array
// on `device` (the current device), looked up once per device (noalloc.hip).
int noalloc_scratch(int device, void **ptr, size_t *bytes);

}  // namespace gnn
