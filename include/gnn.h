/*
 * gnn.h -- C ABI of libgnn.so, an MI355X (gfx950) implementation of the
 * interaction-network edge classifier used by GNN-based track finding.
 *
 * Paper section 2.1 ("ExaTrkX") places this step in the pipeline: an
 * interaction network classifies the edges of the hit graph and its per-edge
 * scores go on to the connected-components step.  Section 2.3 describes the
 * custom service backend's contract (hits x raw features in); section 1
 * gives the event scale (about 300k nodes and 1M edges).  This library takes
 * one hit graph in and returns one score per edge.
 *
 * Model (the paper prints no architecture; this is the workload's definition):
 *   every MLP is two Linear layers, each followed by LayerNorm and ReLU;
 *   h0 = MLP_node_enc(x);  e0 = MLP_edge_enc([h_src; h_dst]);
 *   T times: e = MLP_edge([h_src; h_dst; e]);  agg_in(v) = sum of e over
 *            edges into v; agg_out(v) = sum over edges out of v;
 *            h = MLP_node([h; agg_in; agg_out]);
 *   z = w . LNReLU(W [h_src; h_dst; e] + b) + c;  score = sigmoid(z).
 *
 * Every pointer argument of gnn_infer* / gnn_debug_* is a DEVICE pointer on
 * the handle's device, except where noted.  All calls are thread-safe; one
 * handle may run concurrently on several streams (its weights are read-only).
 *
 * Workspace: gnn_infer* and gnn_debug_* need device scratch of at most
 * (E + 3N)*H*act_bytes + 16*N*H + (60 + H/4)*E + 64 KiB bytes (act_bytes 4
 * for fp32, 2 for bf16; about 1.7 GB for N = 300k, E = 1M, H = 128, fp32).  The handle keeps these buffers between calls (at most 16, one
 * per call in flight, each rounded up by 1/8 for growth) and frees them in
 * gnn_destroy; a call that finds an idle buffer large enough orders itself
 * after that buffer's previous call with an event and allocates nothing.
 */
#ifndef GNN_H
#define GNN_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---- status codes ------------------------------------------------------ */
#define GNN_OK 0
#define GNN_E_INVALID_ARG (-1) /* null pointer, bad count, bad dims           */
#define GNN_E_NO_DEVICE (-2)   /* no HIP device visible                        */
#define GNN_E_OOM (-3)         /* device or host allocation failed             */
#define GNN_E_INDEX (-4)       /* edge index out of range (validation on)      */
#define GNN_E_HIP (-5)         /* a HIP runtime call or kernel launch failed   */
#define GNN_E_UNSUPPORTED (-6) /* dims or device the library does not support */

/* ---- model description ------------------------------------------------- */
#define GNN_FP32 0 /* weights and activations fp32                           */
#define GNN_BF16 1 /* activations stored in bf16 and fed to bf16 MFMAs; each
                      weight carried as two bf16 terms (hi = bf16(W),
                      lo = bf16(W - hi)); fp32 accumulation, fp32 LayerNorm
                      statistics, fp32 segment sums                       */

#define GNN_VALIDATE_INDICES 1u /* check every index is in [0, n_nodes) before
                                   computing; costs one host synchronisation */
#define GNN_LITERAL_GATHER 2u   /* evaluate the first layer of every edge MLP per
                                   edge on the gathered [h_src; h_dst; e] rows
                                   instead of the default regrouping
                                   (W_s h)[src] + (W_d h)[dst] + W_e e with the
                                   node projections computed once per node; the
                                   two agree up to fp32 rounding (both dtypes) */
#define GNN_FP32_MFMA 4u        /* fp32, regrouped form: multiply on the fp32
                                   matrix cores (v_mfma_f32_32x32x2_f32).  The
                                   default multiplies fp32 operands split into
                                   fp16 pairs (x = x1 + x2, per-operand error
                                   <= 2^-22 |x|; weights pre-scaled by a power
                                   of two; each node's aggregate row scaled by
                                   a power of two when its degree would leave
                                   the fp16 range) on the fp16 matrix cores,
                                   with fp32 accumulation throughout.  The
                                   default needs every LayerNorm output bound
                                   max|gamma| sqrt(H-1) + max|beta| <= 2^15;
                                   weights that break it select this path by
                                   themselves. */
#define GNN_F16_WEIGHTS 8u      /* GNN_BF16 only (not with GNN_LITERAL_GATHER or
                                   GNN_FP32_MFMA): each weight carried as one
                                   fp16 number (times a power of two) instead
                                   of the bf16 pair hi/lo, so every product is
                                   one fp16 matrix-core operation instead of
                                   two bf16 ones.  Activations stay bf16 in
                                   memory and are rounded to bf16 where they
                                   feed a product, then converted exactly to
                                   fp16 (a node's aggregate row scaled by a
                                   power of two when its degree would leave the
                                   fp16 range).  Needs every LayerNorm output
                                   bound (as above) <= 2^15 and every scaled
                                   weight inside the fp16 range; otherwise
                                   gnn_create fails with GNN_E_UNSUPPORTED.
                                   With T >= 1 the edge encoder then runs in
                                   the first edge update's kernel (its output
                                   stays on chip; the profiler counts it in
                                   GNN_STAGE_EDGE_UPDATE), except in
                                   gnn_debug_stages. */

typedef struct gnn_dims {
  uint32_t struct_size;     /* = sizeof(gnn_dims) (ABI versioning)              */
  int32_t in_features;      /* F: raw features per node, 1..16 (3 for hits)     */
  int32_t hidden;           /* H: 64 or 128                                     */
  int32_t n_iters;          /* T: message-passing iterations, 0..64             */
  int32_t n_mp_weight_sets; /* 1 = one edge MLP and one node MLP shared by all
                               iterations; T = one pair per iteration          */
  int32_t dtype;            /* GNN_FP32 or GNN_BF16                             */
  float ln_eps;             /* LayerNorm epsilon (1e-5)                         */
  uint32_t flags;           /* OR of GNN_VALIDATE_INDICES, GNN_LITERAL_GATHER,
                               GNN_FP32_MFMA, GNN_F16_WEIGHTS, or 0             */
} gnn_dims;

typedef struct gnn_handle gnn_handle;

/* Number of floats in the packed weight blob for `dims`, 0 if dims invalid.
 * Paper section 2.1: the edge-classification step is an interaction network
 * whose trained weights the pipeline loads (section 2.1: trained PyTorch
 * models run through libTorch); this blob is that model's parameter set.
 * Blob order (fp32; W is [out][in] row-major, PyTorch Linear convention):
 *   node_enc (F->H->H), edge_enc (2H->H->H),
 *   n_mp_weight_sets x [edge_mlp (3H->H->H), node_mlp (3H->H->H)],
 *   edge_cls (3H->H->1).
 * A hidden layer stores W, b, gamma, beta; the classifier's last layer
 * stores W[1][H] and b[1]. */
size_t gnn_weight_count(const gnn_dims *dims);

/* Loads one model instance (paper section 2.1: the pipeline loads the trained
 * interaction network once and runs it for every event; section 3.2: one GPU
 * may hold several instances, which here share one handle).
 * Validate dims, convert and upload the HOST fp32 blob `weights` (copied;
 * the caller may free it on return) to the current HIP device.  Returns NULL
 * on error (see gnn_last_error): GNN_E_INVALID_ARG for bad dims or NULL
 * pointers, GNN_E_NO_DEVICE, GNN_E_UNSUPPORTED for a device that is not
 * gfx950 or dims outside the supported set, GNN_E_OOM. */
gnn_handle *gnn_create(const float *weights, const gnn_dims *dims);

/* Score every edge of one hit graph (paper section 2.1: one score per edge).
 *   node_feat   [n_nodes][F] fp32, row-major
 *   edge_index  [2][n_edges] int32: row 0 = source, row 1 = destination;
 *               never modified; self-loops and duplicate edges are allowed
 *   edge_scores [n_edges] fp32 output, sigmoid scores in input edge order
 * Asynchronous on `stream` (0 = the null stream): inputs must stay valid
 * and outputs untouched until the stream passes this work.  Results are
 * bitwise deterministic for a given input.  Returns GNN_OK with no writes
 * when n_edges == 0; GNN_E_INVALID_ARG for n_nodes == 0 < n_edges, negative
 * counts, counts above INT32_MAX or NULL pointers; GNN_E_UNSUPPORTED for
 * n_edges >= 2^30 (the CSR sort's counters are 30 bits wide).  An index
 * outside [0, n_nodes) is reported as GNN_E_INDEX when GNN_VALIDATE_INDICES
 * is set; otherwise it is clamped into range (no fault, meaningless scores). */
int gnn_infer(gnn_handle *h, const float *node_feat, const int32_t *edge_index,
              int64_t n_nodes, int64_t n_edges, float *edge_scores, hipStream_t stream);

/* As gnn_infer, writing the pre-sigmoid logits z instead of the scores
 * (paper section 2.1: the classifier's raw output before the sigmoid that
 * turns it into an edge score; exposed for parity checks, where a logit
 * keeps precision that a saturated score loses).  Same arguments, layouts,
 * ownership and errors as gnn_infer. */
int gnn_infer_logits(gnn_handle *h, const float *node_feat, const int32_t *edge_index,
                     int64_t n_nodes, int64_t n_edges, float *edge_logits,
                     hipStream_t stream);

/* ---- no-allocation inference ----------------------------------------------
 * For callers that cannot allocate device memory: code under HIP stream
 * capture, tight serving loops, harnesses that forbid hipMalloc.
 * gnn_infer_noalloc is gnn_infer (same arguments, layouts, ownership,
 * results bit for bit, errors) except for its workspace: instead of the
 * handle's cached buffers it uses one fixed device array of
 * GNN_NOALLOC_SCRATCH_BYTES bytes inside the library, so it calls no
 * hipMalloc, hipFree or other allocating routine and records no profiling
 * events.  Each GPU the call runs on holds its own copy of that array from
 * the first call on it until the process ends.  An event whose workspace
 * (the bound at the top of this file) exceeds the array is rejected with
 * GNN_E_INVALID_ARG before any work is enqueued: the array holds events up
 * to about 50k hits and 330k edges at H = 128 in fp32 (378 MB of workspace;
 * 255 MB in bf16).  Larger events, such as the paper-scale 300k-hit event
 * (1.7 GB), go through gnn_infer, whose cached workspace allocates only on
 * a handle's first call of a given size.  All calls on one
 * GPU share the array: calls whose work overlaps on that GPU (several
 * streams, several threads, several handles) race and give undefined
 * results, so order them (one stream, or events between streams).  Each call
 * overwrites what the previous one left; nothing needs clearing between
 * calls.  With GNN_VALIDATE_INDICES the call synchronises `stream`, as
 * gnn_infer does. */
#define GNN_NOALLOC_SCRATCH_BYTES ((size_t)512 << 20)
int gnn_infer_noalloc(gnn_handle *h, const float *node_feat, const int32_t *edge_index,
                      int64_t n_nodes, int64_t n_edges, float *edge_scores, hipStream_t stream);

/* ---- edge filter (the step before the GNN) --------------------------------
 * Paper section 2.1: after the embedding step a Filtering MLP scores every
 * candidate edge and applyFiltering keeps the edges above a fixed threshold.
 * Model: s_j = sigmoid(w . phi(W1 phi(W0 [x_src; x_dst] + b0) + b1) + c),
 * phi = LayerNorm then ReLU.  Blob (fp32, W [out][in]): layer 0 (2F -> H:
 * W, b, gamma, beta), layer 1 (H -> H: W, b, gamma, beta), head (H -> 1: W,
 * b). */
typedef struct gnn_filter_dims {
  uint32_t struct_size; /* = sizeof(gnn_filter_dims)          */
  int32_t in_features;  /* F, 1..16                           */
  int32_t hidden;       /* H, 64 or 128                        */
  float ln_eps;         /* LayerNorm epsilon                   */
} gnn_filter_dims;

typedef struct gnn_filter gnn_filter;

size_t gnn_filter_weight_count(const gnn_filter_dims *dims);
gnn_filter *gnn_filter_create(const float *weights, const gnn_filter_dims *dims);
void gnn_filter_destroy(gnn_filter *f);

/* Scores the n_edges candidate edges (edge_scores, [n_edges] fp32 device,
 * may be NULL) and writes the edges with score > threshold, in input order,
 * as a contiguous [2][n_kept] int32 edge_index to edge_index_out (device,
 * room for 2 * n_edges).  *n_kept (host) receives the count, so the call
 * returns after `stream` has drained. */
int gnn_filter_apply(gnn_filter *f, const float *node_feat, const int32_t *edge_index,
                     int64_t n_nodes, int64_t n_edges, float threshold, float *edge_scores,
                     int32_t *edge_index_out, int64_t *n_kept, hipStream_t stream);

/* Track candidates from edge scores (paper section 2.1: weakly-connected
 * components of the scored graph form the track candidates; section 2.3:
 * the service returns one integer label per space point).  Keeps the edges with
 * edge_scores[j] > threshold (every edge when edge_scores is NULL), treats
 * them as undirected and writes labels[v] = the smallest node id of v's
 * connected component -- unique, so results are bitwise reproducible.
 *   edge_index [2][n_edges] int32 (device), edge_scores [n_edges] fp32
 *   (device) or NULL, labels [n_nodes] int32 (device, output).
 * Runs on the current device; the host checks convergence between rounds,
 * so the call returns after `stream` has drained.  GNN_E_INVALID_ARG for
 * bad counts or NULL pointers; out-of-range indices are clamped. */
int gnn_wcc(const int32_t *edge_index, const float *edge_scores, float threshold,
            int64_t n_nodes, int64_t n_edges, int32_t *labels, hipStream_t stream);

/* Hits in, labels out: gnn_infer, then gnn_wcc on its scores.  edge_scores
 * may be NULL (scores then live in a temporary buffer). */
int gnn_infer_labels(gnn_handle *h, const float *node_feat, const int32_t *edge_index,
                     int64_t n_nodes, int64_t n_edges, float threshold, float *edge_scores,
                     int32_t *labels, hipStream_t stream);

/* Unloads the model instance loaded by gnn_create (paper section 2.1).
 * Waits for the device, then frees everything the handle owns: its weights
 * and its cached workspaces.  Calls in progress on other threads must have
 * returned.  NULL-safe. */
void gnn_destroy(gnn_handle *h);

/* Memory management, not a step of the method: frees the inference
 * workspaces the handle keeps between calls (see the note at the top of
 * this file) that no call is using, each after the work of its last call
 * has finished (the function waits for that work).  Buffers held by calls
 * in progress on other threads stay.  Later calls allocate again as needed.
 * Returns the number of bytes freed (0 if none), or GNN_E_INVALID_ARG for a
 * NULL handle, GNN_E_HIP if waiting or freeing fails. */
int64_t gnn_release_workspaces(gnn_handle *h);

/* Memory management, not a step of the method: caps the bytes of inference
 * workspace the handle may hold at once (its cached buffers plus buffers of
 * calls in progress); 0 removes the cap.  A call whose workspace would take
 * the handle past the cap allocates nothing and returns GNN_E_OOM before
 * enqueuing any work (outputs untouched); the handle stays usable.  The
 * initial cap comes from the environment variable GNN_WORKSPACE_LIMIT at
 * gnn_create (digits with an optional k, m or g suffix, binary units; a
 * malformed value makes gnn_create fail with GNN_E_INVALID_ARG), else none.
 * Lowering the cap frees nothing already held (see
 * gnn_release_workspaces).  Returns GNN_OK, or GNN_E_INVALID_ARG for a NULL
 * handle or a negative count. */
int gnn_set_workspace_limit(gnn_handle *h, int64_t bytes);

/* Error reporting, not a step of the method (the paper describes none):
 * the message of the last failed call on this thread ("" if none).  The
 * pointer stays valid until the next failing call on the same thread. */
const char *gnn_last_error(void);

/* ---- graph construction ---------------------------------------------------
 * Paper section 2.1: an embedding network maps every space point into a
 * latent space, and a fixed-radius nearest-neighbour search there proposes
 * the candidate edges.  The paper gives no architecture; the embedding here
 * is z = W3 phi(W2 phi(W1 x + b1) + b2) + b3 (F -> H -> H -> D, phi =
 * LayerNorm then ReLU as in the GNN's MLPs, no activation on the output). */
typedef struct gnn_embed_dims {
  uint32_t struct_size; /* = sizeof(gnn_embed_dims)                        */
  int32_t in_features;  /* F, 1..16                                         */
  int32_t hidden;       /* H, 64 or 128                                     */
  int32_t out_dim;      /* D, 1..16                                         */
  float ln_eps;         /* LayerNorm epsilon                                */
} gnn_embed_dims;
typedef struct gnn_embedder gnn_embedder;

/* Floats in the embedding blob: W1 [H][F], b1, gamma1, beta1, W2 [H][H], b2,
 * gamma2, beta2, W3 [D][H], b3 (host fp32, [out][in] row-major); 0 if dims
 * are invalid. */
size_t gnn_embed_weight_count(const gnn_embed_dims *dims);
/* Copies and uploads the HOST blob; NULL on error (gnn_last_error). */
gnn_embedder *gnn_embed_create(const float *weights, const gnn_embed_dims *dims);
/* z [n_nodes][D] fp32 (device) from node_feat [n_nodes][F] (device),
 * asynchronous on `stream`; fp32 throughout (fp32 matrix cores). */
int gnn_embed_apply(gnn_embedder *m, const float *node_feat, int64_t n_nodes, float *z,
                    hipStream_t stream);
void gnn_embed_destroy(gnn_embedder *m);

/* Every pair i < j of rows of z [n_nodes][dim] (device fp32, dim 1..16)
 * whose squared distance, evaluated in fp32 as d = 0, d = fmaf(t, t, d) with
 * t = z[i][k] - z[j][k] for k = 0 .. dim-1, is below r2.  The count goes to
 * *n_pairs (host).  With edge_index non-NULL and room for max_pairs pairs,
 * the pairs are written as a contiguous [2][n_pairs] int32 edge list (row 0
 * = i, row 1 = j), grouped by ascending i, deterministic order within one i;
 * that write is asynchronous on `stream`, the count is not (the call waits
 * for it).  Returns GNN_OK; GNN_E_INVALID_ARG for bad arguments or when
 * more than max_pairs pairs exist (nothing written, *n_pairs holds the
 * count); GNN_E_UNSUPPORTED above INT32_MAX pairs.  r2 <= 0 or fewer than
 * two rows give no pairs.  The search bins the rows on a grid over their
 * first min(3, dim) coordinates with cells as wide as the radius: its cost
 * grows with the number of rows per cell. */
int gnn_frnn(const float *z, int64_t n_nodes, int32_t dim, float r2, int32_t *edge_index,
             int64_t max_pairs, int64_t *n_pairs, hipStream_t stream);

/* ---- serving: a request queue in front of several model instances --------
 * Paper sections 2.3 and 3.2: the GNN runs as a service, one GPU holding
 * several instances of the model (Fig. 4b) behind a queue of requests from
 * many clients.  A gnn_server runs n_instances worker threads, each with its
 * own HIP stream (default priority), that take requests from one FIFO queue
 * and run each as gnn_infer on the shared handle, then synchronise their
 * stream.  The handle must outlive the server and may not be destroyed while
 * requests are pending. */
typedef struct gnn_server gnn_server;

/* n_instances in 1..64; binds to the current HIP device.  NULL on error
 * (gnn_last_error): GNN_E_INVALID_ARG, GNN_E_NO_DEVICE. */
gnn_server *gnn_server_create(gnn_handle *h, int n_instances);

/* Queue one event, with the arguments and device-pointer layouts of
 * gnn_infer.  The workers' streams are not ordered after any stream of the
 * caller: the inputs must already hold their values on the device when
 * submit is called (for example, synchronise the stream that produced them
 * first), and the buffers must stay valid and the outputs untouched until
 * the request is waited for.  Returns the request id (>= 0), or a negative
 * status: GNN_E_INVALID_ARG for NULL pointers, counts outside 0..INT32_MAX
 * or a server that is shutting down. */
int64_t gnn_server_submit(gnn_server *s, const float *node_feat, const int32_t *edge_index,
                          int64_t n_nodes, int64_t n_edges, float *edge_scores);

/* Block until request `id` has completed and release it; returns the status
 * of its gnn_infer (its message becomes this thread's gnn_last_error).  With
 * latency_ms non-NULL, stores the time from submission to completion
 * (queueing included) in milliseconds.  Only one thread may wait for a
 * request: an id that is unknown, already released, or being waited for by
 * another thread gives GNN_E_INVALID_ARG (that other wait is unaffected). */
int gnn_server_wait(gnn_server *s, int64_t id, double *latency_ms);

/* What gnn_server_wait_info reports about one request.  The device interval
 * comes from two events the worker records on its stream just before and
 * just after the request's gnn_infer, in milliseconds since an event
 * recorded when the server was created; the union of these intervals over
 * a run, divided by its wall time, is the fraction of that time the GPU
 * spent on requests (paper section 3.2, Fig. 4b: GPU utilisation against
 * the number of model instances).  Both are -1 if the request failed. */
typedef struct gnn_request_info {
  uint32_t struct_size;   /* = sizeof(gnn_request_info)                        */
  int32_t status;         /* status of the request's gnn_infer                 */
  double latency_ms;      /* submission to completion, host clock              */
  double device_start_ms; /* device interval of the request's work, relative   */
  double device_end_ms;   /* to the server's creation                          */
} gnn_request_info;

/* gnn_server_wait, filling *info (struct_size set by the caller).  Returns
 * the request's status as gnn_server_wait does; GNN_E_INVALID_ARG also for
 * a NULL info or a wrong struct_size. */
int gnn_server_wait_info(gnn_server *s, int64_t id, gnn_request_info *info);

/* Finish every queued request, stop the workers, free the server.  Results
 * of requests not waited for are discarded.  NULL-safe. */
void gnn_server_destroy(gnn_server *s);

/* ---- profiling -----------------------------------------------------------
 * While profiling is enabled on a handle, every call times each stage with
 * two HIP events bound to the dispatches of the stage's kernels
 * (hipExtLaunchKernel): the first kernel's start and the last one's end, so
 * a stage's time is the time its kernels ran.  Timed dispatches cost the
 * stream a few microseconds each.  A call's total runs from its first
 * stage's start to its last stage's end.  gnn_profile_read waits for those
 * events and returns the accumulated device time per stage since the last
 * enable. */
#define GNN_STAGE_CSR 0         /* destination- and source-sorted CSR build  */
#define GNN_STAGE_NODE_ENC 1    /* node encoder MLP                           */
#define GNN_STAGE_EDGE_ENC 2    /* edge encoder MLP (gathers h_src, h_dst)    */
#define GNN_STAGE_EDGE_UPDATE 3 /* fused gather + edge MLP, once per iteration */
#define GNN_STAGE_AGGREGATE 4   /* CSR segmented sums, once per iteration      */
#define GNN_STAGE_NODE_UPDATE 5 /* node MLP, once per iteration                */
#define GNN_STAGE_CLASSIFIER 6  /* edge classifier + sigmoid                   */
#define GNN_STAGE_TOTAL 7       /* the whole call                              */
#define GNN_N_STAGES 8

typedef struct gnn_profile_stats {
  uint32_t struct_size;            /* = sizeof(gnn_profile_stats)          */
  int32_t n_calls;                 /* profiled calls accumulated           */
  int64_t launches[GNN_N_STAGES];  /* timed stages (one per stage run)     */
  double ms[GNN_N_STAGES];         /* accumulated device milliseconds      */
} gnn_profile_stats;

/* Sampled profiling: each call times only the three per-iteration stages
 * (edge update, aggregation, node update) of its iteration T / 2, and no
 * total.  A timed dispatch costs the stream a few microseconds (about 0.12
 * ms per full-size event when every stage is timed); sampling keeps per-kernel
 * times of every call at a tenth of that. */
#define GNN_PROFILE_SAMPLE 2

/* Profiling mode: 0 off, 1 every stage of every call, GNN_PROFILE_SAMPLE;
 * any other value gives GNN_E_INVALID_ARG.  Resets the counters. */
int gnn_profile_enable(gnn_handle *h, int enable);
/* Synchronise the recorded events and fill *out (struct_size must be set). */
int gnn_profile_read(gnn_handle *h, gnn_profile_stats *out);

/* ---- measurement aid: achievable HBM streaming rates --------------------
 * Not an operation of the method: it gives the roofline figures a measured
 * ceiling beside the 8 TB/s peak.  One launch of a plain grid-stride kernel
 * of 256-thread workgroups streams `bytes` (a positive multiple of 16)
 * through device memory in 16-byte nontemporal accesses:
 *   GNN_PROBE_READ   reads buf; buf2 (>= 4 bytes) is a sink written only
 *                    when the sum equals -1.5e38 (never, for finite data);
 *   GNN_PROBE_WRITE  fills buf (buf2 unused but must be non-NULL);
 *   GNN_PROBE_COPY   copies buf to buf2 (both `bytes` long, disjoint).
 * grid = workgroups (0: 4 per compute unit).  After one untimed launch,
 * `reps` launches (1..1000) are timed with HIP events on `stream`; *ms gets
 * the fastest.  Waits for the stream.  buf and buf2 are device pointers
 * owned by the caller; their contents afterwards are unspecified.  Returns
 * GNN_E_INVALID_ARG for a bad kind, size, grid, reps or NULL pointer,
 * GNN_E_HIP if a launch or event call fails. */
#define GNN_PROBE_READ 0
#define GNN_PROBE_WRITE 1
#define GNN_PROBE_COPY 2
int gnn_hbm_probe(int kind, void *buf, void *buf2, int64_t bytes, int32_t grid, int32_t reps,
                  float *ms, hipStream_t stream);

/* ---- test hooks ---------------------------------------------------------
 * Destination- and source-sorted CSR of edge_index, as the inference path
 * builds it: row_ptr_in [n_nodes+1], perm_in [n_edges] (edge ids with
 * dst == v in ascending id order at row_ptr_in[v] .. row_ptr_in[v+1]-1),
 * and the same by source.  Any output pointer may be NULL.  Waits for the
 * build; GNN_E_HIP if a sort pass gave up waiting on an earlier tile (its
 * wait is bounded; running workgroups always end it in practice). */
int gnn_debug_csr(gnn_handle *h, const int32_t *edge_index, int64_t n_nodes, int64_t n_edges,
                  int32_t *row_ptr_in, int32_t *perm_in, int32_t *row_ptr_out,
                  int32_t *perm_out, hipStream_t stream);

/* Run the encoders and the first `stop_iter` message-passing iterations and
 * copy out, as fp32 in input order, h [n_nodes][H] and e [n_edges][H] and,
 * for stop_iter >= 1, the aggregates of the last iteration run
 * [n_nodes][H] each.  Any output pointer may be NULL. */
int gnn_debug_stages(gnn_handle *h, const float *node_feat, const int32_t *edge_index,
                     int64_t n_nodes, int64_t n_edges, int32_t stop_iter, float *h_out,
                     float *e_out, float *agg_in_out, float *agg_out_out, hipStream_t stream);

#ifdef __cplusplus
}
#endif
#endif /* GNN_H */
