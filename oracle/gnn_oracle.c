/*
 * gnn_oracle.c -- CPU oracle for the interaction-network edge classifier.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path links, loads or
 * calls this file; only the tests, the smoke check and the benchmark's CPU
 * baseline do.  It shares no code, header or table with the HIP library: it
 * parses the weight blob with its own code and evaluates the plain
 * definition of the model in double precision, one row at a time, with no
 * blocking, fusion or reordering beyond what the definition states.
 *
 * What is computed (paper section 2.1, "ExaTrkX": the edge-classification
 * step is an interaction network whose per-edge scores feed the weakly
 * connected components step; section 1 gives the event scale of roughly
 * 300k nodes and 1M edges).  The paper prints no architecture, so the model
 * follows the workload specification used throughout this repository:
 *
 *   MLP(a)  = phi2(W2 phi1(W1 a + b1) + b2),
 *   phi(y)  = ReLU(gamma * (y - mean(y)) / sqrt(var(y) + eps) + beta),
 *             mean and biased variance over the features of one row;
 *   h0_v    = MLP_node_enc(x_v)                                   (F -> H -> H)
 *   e0_j    = MLP_edge_enc([h_src(j); h_dst(j)])                  (2H -> H -> H)
 *   for t = 0 .. T-1 (weight set k = 0 if shared, else t):
 *     e'_j     = MLP_edge^k([h_src(j); h_dst(j); e_j])            (3H -> H -> H)
 *     ain_v    = sum over j with dst(j) = v of e'_j   (ascending j; empty = 0)
 *     aout_v   = sum over j with src(j) = v of e'_j
 *     h'_v     = MLP_node^k([h_v; ain_v; aout_v])                 (3H -> H -> H)
 *   z_j     = w2 . phi1(W1 [h_src(j); h_dst(j); e_j] + b1) + b2   (3H -> H -> 1)
 *   s_j     = 1 / (1 + exp(-z_j))
 *
 * Readings where the specification is silent (each is listed in the design
 * notes): LayerNorm then ReLU after both Linear layers of every hidden MLP;
 * the classifier's last Linear has no LayerNorm (a width-1 LayerNorm is a
 * constant); the classifier and the edge MLP read the same concatenation;
 * the edge encoder reads the encoded h0; no residual connections; within an
 * iteration the edge update uses the old h and e, aggregation sums the new
 * e, and the node update uses the old h.
 *
 * Track candidates (paper section 2.1: the edge scores are passed to the
 * weakly-connected-components step; section 2.3: the custom backend returns
 * one integer label per space point): oracle_wcc keeps the edges whose score
 * exceeds a threshold, treats them as undirected, and labels every node with
 * the smallest node id of its connected component, found by breadth-first
 * search.
 *
 * Edge filtering (paper section 2.1: an MLP scores the candidate edges and a
 * fixed threshold on those scores removes clearly fake ones before the GNN):
 * oracle_filter evaluates s_j = sigmoid(w . phi(W2 phi(W1 [x_src; x_dst] + b1)
 * + b2) + c) per candidate edge and keeps, in input order, the edges with
 * s_j > threshold.
 *
 * Graph construction (paper section 2.1: an embedding network maps every
 * space point into a latent space and a fixed-radius nearest-neighbour
 * search there builds the candidate edges): oracle_embed evaluates
 * z_v = W3 phi(W2 phi(W1 x_v + b1) + b2) + b3 (F -> H -> H -> D; the output
 * layer has no LayerNorm or activation), and oracle_frnn lists every pair
 * i < j of rows of a given fp32 matrix z with d2(i, j) < r2, where d2 is the
 * squared Euclidean distance evaluated in fp32 as d = 0; d = fmaf(t, t, d)
 * with t = z_i[k] - z_j[k] for k = 0 .. D-1 (one rounding per step, the
 * same decision a GPU makes with the same operations), by brute force over
 * all pairs, in ascending (i, j) order.
 *
 * Every function here is pinned by the CPU tests against something other
 * than itself: a torch-CPU library evaluation of one hidden layer, an
 * incidence-matrix brute force on tiny graphs, closed forms (all-zero
 * weights, constant messages), invariances (edge order, node labels), and
 * scipy's connected_components for the labels.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* One Linear layer as stored in the blob. gamma/beta are NULL for the
 * classifier's last layer, which has no LayerNorm. */
typedef struct {
  int fin, fout;
  double *W;     /* [fout][fin] */
  double *b;     /* [fout] */
  double *gamma; /* [fout] or NULL */
  double *beta;  /* [fout] or NULL */
} olayer;

typedef struct { olayer l0, l1; } omlp;

typedef struct {
  int F, H, T, S;
  double eps;
  omlp node_enc, edge_enc, cls;
  omlp *edge_mlp, *node_mlp; /* S each */
  double *store;             /* one allocation behind every array above */
} omodel;

static long layer_floats(int fin, int fout, int hidden) {
  return (long)fin * fout + fout + (hidden ? 2L * fout : 0L);
}

long oracle_weight_count(int F, int H, int S) {
  long n = 0;
  n += layer_floats(F, H, 1) + layer_floats(H, H, 1);          /* node_enc */
  n += layer_floats(2 * H, H, 1) + layer_floats(H, H, 1);      /* edge_enc */
  n += (long)S * 2 * (layer_floats(3 * H, H, 1) + layer_floats(H, H, 1));
  n += layer_floats(3 * H, H, 1) + layer_floats(H, 1, 0);      /* edge_cls */
  return n;
}

static const float *take_layer(olayer *L, const float *p, int fin, int fout,
                               int hidden, double **dst) {
  L->fin = fin;
  L->fout = fout;
  L->W = *dst;
  for (long i = 0; i < (long)fin * fout; ++i) (*dst)[i] = p[i];
  *dst += (long)fin * fout;
  p += (long)fin * fout;
  L->b = *dst;
  for (int i = 0; i < fout; ++i) (*dst)[i] = p[i];
  *dst += fout;
  p += fout;
  if (hidden) {
    L->gamma = *dst;
    for (int i = 0; i < fout; ++i) (*dst)[i] = p[i];
    *dst += fout;
    p += fout;
    L->beta = *dst;
    for (int i = 0; i < fout; ++i) (*dst)[i] = p[i];
    *dst += fout;
    p += fout;
  } else {
    L->gamma = L->beta = NULL;
  }
  return p;
}

static int model_init(omodel *m, const float *w, int F, int H, int T, int S, double eps) {
  if (F <= 0 || H <= 0 || T < 0 || S <= 0) return -1;
  m->F = F; m->H = H; m->T = T; m->S = S; m->eps = eps;
  m->store = (double *)malloc(sizeof(double) * (size_t)oracle_weight_count(F, H, S));
  m->edge_mlp = (omlp *)malloc(sizeof(omlp) * (size_t)S);
  m->node_mlp = (omlp *)malloc(sizeof(omlp) * (size_t)S);
  if (!m->store || !m->edge_mlp || !m->node_mlp) return -3;
  double *d = m->store;
  const float *p = w;
  p = take_layer(&m->node_enc.l0, p, F, H, 1, &d);
  p = take_layer(&m->node_enc.l1, p, H, H, 1, &d);
  p = take_layer(&m->edge_enc.l0, p, 2 * H, H, 1, &d);
  p = take_layer(&m->edge_enc.l1, p, H, H, 1, &d);
  for (int s = 0; s < S; ++s) {
    p = take_layer(&m->edge_mlp[s].l0, p, 3 * H, H, 1, &d);
    p = take_layer(&m->edge_mlp[s].l1, p, H, H, 1, &d);
    p = take_layer(&m->node_mlp[s].l0, p, 3 * H, H, 1, &d);
    p = take_layer(&m->node_mlp[s].l1, p, H, H, 1, &d);
  }
  p = take_layer(&m->cls.l0, p, 3 * H, H, 1, &d);
  p = take_layer(&m->cls.l1, p, H, 1, 0, &d);
  return 0;
}

static void model_free(omodel *m) {
  free(m->store);
  free(m->edge_mlp);
  free(m->node_mlp);
}

/* y = W a + b (one output row at a time, plain dot products). */
static void linear(const olayer *L, const double *a, double *y) {
  for (int o = 0; o < L->fout; ++o) {
    const double *w = L->W + (long)o * L->fin;
    double acc = 0.0;
    /* the simd pragma only lets the compiler split this sum into a few
     * interleaved partial sums (fp64, well below the tolerances used) */
#pragma omp simd reduction(+ : acc)
    for (int k = 0; k < L->fin; ++k) acc += w[k] * a[k];
    y[o] = acc + L->b[o];
  }
}

/* In place: y <- ReLU(gamma * (y - mean) / sqrt(var + eps) + beta). */
static void layernorm_relu(const olayer *L, double eps, double *y) {
  const int n = L->fout;
  double mean = 0.0, var = 0.0;
  for (int i = 0; i < n; ++i) mean += y[i];
  mean /= n;
  for (int i = 0; i < n; ++i) var += (y[i] - mean) * (y[i] - mean);
  var /= n;
  const double inv = 1.0 / sqrt(var + eps);
  for (int i = 0; i < n; ++i) {
    const double v = L->gamma[i] * (y[i] - mean) * inv + L->beta[i];
    y[i] = v > 0.0 ? v : 0.0;
  }
}

/* Hidden MLP: two Linear layers, each followed by LayerNorm and ReLU.
 * tmp has room for H doubles. */
static void mlp_hidden(const omlp *m, double eps, const double *a, double *tmp, double *out) {
  linear(&m->l0, a, tmp);
  layernorm_relu(&m->l0, eps, tmp);
  linear(&m->l1, tmp, out);
  layernorm_relu(&m->l1, eps, out);
}

static double sigmoid(double z) {
  if (z >= 0.0) return 1.0 / (1.0 + exp(-z));
  const double ez = exp(z);
  return ez / (1.0 + ez);
}

int oracle_max_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}

void oracle_set_threads(int n) {
#ifdef _OPENMP
  if (n > 0) omp_set_num_threads(n);
#else
  (void)n;
#endif
}

/* One hidden layer (Linear + LayerNorm + ReLU) applied to `rows` input rows;
 * exported so that a test can pin it against a library evaluation. */
int oracle_hidden_layer(const float *W, const float *b, const float *gamma, const float *beta,
                        int fin, int fout, double eps, const double *in, long rows, double *out) {
  if (fin <= 0 || fout <= 0 || rows < 0) return -1;
  olayer L;
  L.fin = fin;
  L.fout = fout;
  L.W = (double *)malloc(sizeof(double) * (size_t)fin * fout);
  L.b = (double *)malloc(sizeof(double) * (size_t)fout);
  L.gamma = (double *)malloc(sizeof(double) * (size_t)fout);
  L.beta = (double *)malloc(sizeof(double) * (size_t)fout);
  for (long i = 0; i < (long)fin * fout; ++i) L.W[i] = W[i];
  for (int i = 0; i < fout; ++i) {
    L.b[i] = b[i];
    L.gamma[i] = gamma[i];
    L.beta[i] = beta[i];
  }
  for (long r = 0; r < rows; ++r) {
    linear(&L, in + r * fin, out + r * fout);
    layernorm_relu(&L, eps, out + r * fout);
  }
  free(L.W); free(L.b); free(L.gamma); free(L.beta);
  return 0;
}

/* Stable counting sort of edge ids by key: row_ptr[v+1] = #{j : key_j <= v}
 * and perm lists, for each v, the ids j with key_j = v in ascending order.
 * Returns -4 if a key lies outside [0, n_nodes). */
int oracle_csr(long n_nodes, long n_edges, const int32_t *keys, int32_t *row_ptr, int32_t *perm) {
  if (n_nodes < 0 || n_edges < 0) return -1;
  for (long j = 0; j < n_edges; ++j)
    if (keys[j] < 0 || keys[j] >= n_nodes) return -4;
  for (long v = 0; v <= n_nodes; ++v) row_ptr[v] = 0;
  for (long j = 0; j < n_edges; ++j) row_ptr[keys[j] + 1] += 1;
  for (long v = 0; v < n_nodes; ++v) row_ptr[v + 1] += row_ptr[v];
  long *cursor = (long *)malloc(sizeof(long) * (size_t)(n_nodes > 0 ? n_nodes : 1));
  for (long v = 0; v < n_nodes; ++v) cursor[v] = row_ptr[v];
  for (long j = 0; j < n_edges; ++j) perm[cursor[keys[j]]++] = (int32_t)j;
  free(cursor);
  return 0;
}

/*
 * Full forward pass.  Inputs: the fp32 weight blob, x [n_nodes][F] fp32,
 * edge_index [2][n_edges] int32 (row 0 src, row 1 dst).  Outputs (either may
 * be NULL): logits z and scores s, [n_edges] in input edge order.
 *
 * Intermediate dumps (all NULL-able) taken after step `dump_iter`:
 *   0   -> h0 and e0 (the encoders' outputs);
 *   t>0 -> h^t, e^t and the aggregates of iteration t.
 * Returns 0, -1 for bad arguments, -3 on allocation failure, -4 for an
 * out-of-range index.
 */
int oracle_forward(const float *weights, int F, int H, int T, int S, double eps,
                   const float *x, const int32_t *edge_index, long n_nodes, long n_edges,
                   double *logits, double *scores, int dump_iter, double *h_dump,
                   double *e_dump, double *ain_dump, double *aout_dump) {
  if (n_nodes < 0 || n_edges < 0 || (n_edges > 0 && n_nodes == 0)) return -1;
  if (S != 1 && S != T) return -1;
  const int32_t *src = edge_index;
  const int32_t *dst = edge_index + n_edges;
  for (long j = 0; j < n_edges; ++j)
    if (src[j] < 0 || src[j] >= n_nodes || dst[j] < 0 || dst[j] >= n_nodes) return -4;

  omodel m;
  int rc = model_init(&m, weights, F, H, T, S, eps);
  if (rc) return rc;

  const size_t nh = (size_t)n_nodes * H, eh = (size_t)n_edges * H;
  double *h = (double *)malloc(sizeof(double) * (nh ? nh : 1));
  double *h2 = (double *)malloc(sizeof(double) * (nh ? nh : 1));
  double *e = (double *)malloc(sizeof(double) * (eh ? eh : 1));
  double *e2 = (double *)malloc(sizeof(double) * (eh ? eh : 1));
  double *ain = (double *)malloc(sizeof(double) * (nh ? nh : 1));
  double *aout = (double *)malloc(sizeof(double) * (nh ? nh : 1));
  if (!h || !h2 || !e || !e2 || !ain || !aout) {
    rc = -3;
    goto done;
  }

  /* node encoder */
#pragma omp parallel
  {
    double *a = (double *)malloc(sizeof(double) * (size_t)(F > 3 * H ? F : 3 * H));
    double *tmp = (double *)malloc(sizeof(double) * (size_t)H);
#pragma omp for schedule(static)
    for (long v = 0; v < n_nodes; ++v) {
      for (int k = 0; k < F; ++k) a[k] = x[v * F + k];
      mlp_hidden(&m.node_enc, eps, a, tmp, h + v * H);
    }
    /* edge encoder on [h_src; h_dst] */
#pragma omp for schedule(static)
    for (long j = 0; j < n_edges; ++j) {
      memcpy(a, h + (long)src[j] * H, sizeof(double) * H);
      memcpy(a + H, h + (long)dst[j] * H, sizeof(double) * H);
      mlp_hidden(&m.edge_enc, eps, a, tmp, e + j * H);
    }
    free(a);
    free(tmp);
  }
  if (dump_iter == 0) {
    if (h_dump) memcpy(h_dump, h, sizeof(double) * nh);
    if (e_dump) memcpy(e_dump, e, sizeof(double) * eh);
  }

  for (int t = 0; t < T; ++t) {
    const omlp *em = &m.edge_mlp[S == 1 ? 0 : t];
    const omlp *nm = &m.node_mlp[S == 1 ? 0 : t];
#pragma omp parallel
    {
      double *a = (double *)malloc(sizeof(double) * (size_t)3 * H);
      double *tmp = (double *)malloc(sizeof(double) * (size_t)H);
      /* edge update on [h_src; h_dst; e] with the old h and e */
#pragma omp for schedule(static)
      for (long j = 0; j < n_edges; ++j) {
        memcpy(a, h + (long)src[j] * H, sizeof(double) * H);
        memcpy(a + H, h + (long)dst[j] * H, sizeof(double) * H);
        memcpy(a + 2 * H, e + j * H, sizeof(double) * H);
        mlp_hidden(em, eps, a, tmp, e2 + j * H);
      }
      free(a);
      free(tmp);
    }
    /* sum aggregation of the new messages, in ascending edge id */
    memset(ain, 0, sizeof(double) * nh);
    memset(aout, 0, sizeof(double) * nh);
    for (long j = 0; j < n_edges; ++j) {
      double *pi = ain + (long)dst[j] * H, *po = aout + (long)src[j] * H;
      const double *m2 = e2 + j * H;
      for (int f = 0; f < H; ++f) {
        pi[f] += m2[f];
        po[f] += m2[f];
      }
    }
#pragma omp parallel
    {
      double *a = (double *)malloc(sizeof(double) * (size_t)3 * H);
      double *tmp = (double *)malloc(sizeof(double) * (size_t)H);
      /* node update on [h; agg_in; agg_out] with the old h */
#pragma omp for schedule(static)
      for (long v = 0; v < n_nodes; ++v) {
        memcpy(a, h + v * H, sizeof(double) * H);
        memcpy(a + H, ain + v * H, sizeof(double) * H);
        memcpy(a + 2 * H, aout + v * H, sizeof(double) * H);
        mlp_hidden(nm, eps, a, tmp, h2 + v * H);
      }
      free(a);
      free(tmp);
    }
    double *sw = h; h = h2; h2 = sw;
    sw = e; e = e2; e2 = sw;
    if (dump_iter == t + 1) {
      if (h_dump) memcpy(h_dump, h, sizeof(double) * nh);
      if (e_dump) memcpy(e_dump, e, sizeof(double) * eh);
      if (ain_dump) memcpy(ain_dump, ain, sizeof(double) * nh);
      if (aout_dump) memcpy(aout_dump, aout, sizeof(double) * nh);
    }
  }

  /* classifier: one hidden layer on [h_src; h_dst; e], then a plain dot */
#pragma omp parallel
  {
    double *a = (double *)malloc(sizeof(double) * (size_t)3 * H);
    double *tmp = (double *)malloc(sizeof(double) * (size_t)H);
#pragma omp for schedule(static)
    for (long j = 0; j < n_edges; ++j) {
      memcpy(a, h + (long)src[j] * H, sizeof(double) * H);
      memcpy(a + H, h + (long)dst[j] * H, sizeof(double) * H);
      memcpy(a + 2 * H, e + j * H, sizeof(double) * H);
      linear(&m.cls.l0, a, tmp);
      layernorm_relu(&m.cls.l0, eps, tmp);
      double z;
      linear(&m.cls.l1, tmp, &z);
      if (logits) logits[j] = z;
      if (scores) scores[j] = sigmoid(z);
    }
    free(a);
    free(tmp);
  }

done:
  free(h); free(h2); free(e); free(e2); free(ain); free(aout);
  model_free(&m);
  return rc;
}

/* Connected components of the undirected graph of kept edges
 * (score > threshold; all edges when scores is NULL).  labels[v] = smallest
 * node id in v's component.  Returns -4 for an out-of-range index. */
int oracle_wcc(long n_nodes, long n_edges, const int32_t *edge_index, const float *scores,
               float threshold, int32_t *labels) {
  if (n_nodes < 0 || n_edges < 0) return -1;
  const int32_t *src = edge_index, *dst = edge_index + n_edges;
  for (long j = 0; j < n_edges; ++j)
    if (src[j] < 0 || src[j] >= n_nodes || dst[j] < 0 || dst[j] >= n_nodes) return -4;
  /* adjacency lists of the kept edges, both directions */
  long *deg = (long *)calloc((size_t)n_nodes + 1, sizeof(long));
  for (long j = 0; j < n_edges; ++j)
    if (!scores || scores[j] > threshold) {
      deg[src[j] + 1] += 1;
      deg[dst[j] + 1] += 1;
    }
  for (long v = 0; v < n_nodes; ++v) deg[v + 1] += deg[v];
  int32_t *adj = (int32_t *)malloc(sizeof(int32_t) * (size_t)(deg[n_nodes] > 0 ? deg[n_nodes] : 1));
  long *fill = (long *)malloc(sizeof(long) * (size_t)(n_nodes > 0 ? n_nodes : 1));
  for (long v = 0; v < n_nodes; ++v) fill[v] = deg[v];
  for (long j = 0; j < n_edges; ++j)
    if (!scores || scores[j] > threshold) {
      adj[fill[src[j]]++] = dst[j];
      adj[fill[dst[j]]++] = src[j];
    }
  /* BFS from every unlabelled node in increasing id order: the start node
   * is then the smallest id of its component */
  int32_t *queue = (int32_t *)malloc(sizeof(int32_t) * (size_t)(n_nodes > 0 ? n_nodes : 1));
  for (long v = 0; v < n_nodes; ++v) labels[v] = -1;
  for (long v = 0; v < n_nodes; ++v) {
    if (labels[v] >= 0) continue;
    long head = 0, tail = 0;
    labels[v] = (int32_t)v;
    queue[tail++] = (int32_t)v;
    while (head < tail) {
      const int32_t u = queue[head++];
      for (long k = deg[u]; k < deg[u + 1]; ++k) {
        const int32_t w = adj[k];
        if (labels[w] < 0) {
          labels[w] = (int32_t)v;
          queue[tail++] = w;
        }
      }
    }
  }
  free(deg);
  free(adj);
  free(fill);
  free(queue);
  return 0;
}

long oracle_filter_weight_count(int F, int H) {
  return layer_floats(2 * F, H, 1) + layer_floats(H, H, 1) + layer_floats(H, 1, 0);
}

/* Filter scores of every candidate edge (scores, may be NULL) and the ids of
 * the kept edges in input order (kept, may be NULL; its count is returned
 * through *n_kept).  Returns 0, -1 for bad arguments, -4 for a bad index. */
int oracle_filter(const float *weights, int F, int H, double eps, const float *x,
                  const int32_t *edge_index, long n_nodes, long n_edges, double threshold,
                  double *scores, int64_t *kept, int64_t *n_kept) {
  if (F <= 0 || H <= 0 || n_nodes < 0 || n_edges < 0 || (n_edges > 0 && n_nodes == 0)) return -1;
  const int32_t *src = edge_index, *dst = edge_index + n_edges;
  for (long j = 0; j < n_edges; ++j)
    if (src[j] < 0 || src[j] >= n_nodes || dst[j] < 0 || dst[j] >= n_nodes) return -4;
  double *store = (double *)malloc(sizeof(double) * (size_t)oracle_filter_weight_count(F, H));
  double *d = store;
  const float *p = weights;
  omlp m;
  olayer head;
  p = take_layer(&m.l0, p, 2 * F, H, 1, &d);
  p = take_layer(&m.l1, p, H, H, 1, &d);
  p = take_layer(&head, p, H, 1, 0, &d);
  double *sc = (double *)malloc(sizeof(double) * (size_t)(n_edges > 0 ? n_edges : 1));
#pragma omp parallel
  {
    double *a = (double *)malloc(sizeof(double) * (size_t)2 * F);
    double *tmp = (double *)malloc(sizeof(double) * (size_t)H);
    double *hid = (double *)malloc(sizeof(double) * (size_t)H);
#pragma omp for schedule(static)
    for (long j = 0; j < n_edges; ++j) {
      for (int k = 0; k < F; ++k) {
        a[k] = x[(long)src[j] * F + k];
        a[F + k] = x[(long)dst[j] * F + k];
      }
      mlp_hidden(&m, eps, a, tmp, hid);
      double z;
      linear(&head, hid, &z);
      sc[j] = sigmoid(z);
    }
    free(a);
    free(tmp);
    free(hid);
  }
  long cnt = 0;
  for (long j = 0; j < n_edges; ++j) {
    if (scores) scores[j] = sc[j];
    if (sc[j] > threshold) {
      if (kept) kept[cnt] = j;
      ++cnt;
    }
  }
  if (n_kept) *n_kept = cnt;
  free(sc);
  free(store);
  return 0;
}

/* ---- graph construction ---------------------------------------------- */

long oracle_embed_weight_count(int F, int H, int D) {
  return layer_floats(F, H, 1) + layer_floats(H, H, 1) + layer_floats(H, D, 0);
}

/* z[n_nodes][D] = embedding of every row of x[n_nodes][F].  Returns 0, or -1
 * for bad arguments. */
int oracle_embed(const float *weights, int F, int H, int D, double eps, const float *x,
                 long n_nodes, double *z) {
  if (F <= 0 || H <= 0 || D <= 0 || n_nodes < 0) return -1;
  double *store = (double *)malloc(sizeof(double) * (size_t)oracle_embed_weight_count(F, H, D));
  double *d = store;
  const float *p = weights;
  omlp m;
  olayer out;
  p = take_layer(&m.l0, p, F, H, 1, &d);
  p = take_layer(&m.l1, p, H, H, 1, &d);
  p = take_layer(&out, p, H, D, 0, &d);
#pragma omp parallel
  {
    double *a = (double *)malloc(sizeof(double) * (size_t)F);
    double *tmp = (double *)malloc(sizeof(double) * (size_t)H);
    double *hid = (double *)malloc(sizeof(double) * (size_t)H);
#pragma omp for schedule(static)
    for (long v = 0; v < n_nodes; ++v) {
      for (int k = 0; k < F; ++k) a[k] = x[v * F + k];
      mlp_hidden(&m, eps, a, tmp, hid);
      linear(&out, hid, z + v * D);
    }
    free(a);
    free(tmp);
    free(hid);
  }
  free(store);
  return 0;
}

/* fp32 squared distance of rows i and j of z[.][D], one fused multiply-add
 * per coordinate in ascending order. */
static float frnn_d2(const float *zi, const float *zj, int D) {
  float acc = 0.0f;
  for (int k = 0; k < D; ++k) {
    const float t = zi[k] - zj[k];
    acc = fmaf(t, t, acc);
  }
  return acc;
}

/* Every pair i < j with d2 < r2, in ascending (i, j) order.  With pairs
 * non-NULL, writes up to max_pairs of them as (i, j) at pairs[2k],
 * pairs[2k+1]; the total count is returned through *n_pairs either way.
 * Returns 0, or -1 for bad arguments. */
int oracle_frnn(const float *z, long n_nodes, int D, float r2, int64_t *pairs, long max_pairs,
                int64_t *n_pairs) {
  if (n_nodes < 0 || D <= 0) return -1;
  long *cnt = (long *)calloc((size_t)(n_nodes > 0 ? n_nodes : 1), sizeof(long));
#pragma omp parallel for schedule(dynamic, 64)
  for (long i = 0; i < n_nodes; ++i) {
    long c = 0;
    for (long j = i + 1; j < n_nodes; ++j)
      if (frnn_d2(z + i * D, z + j * D, D) < r2) ++c;
    cnt[i] = c;
  }
  long total = 0;
  for (long i = 0; i < n_nodes; ++i) {
    const long c = cnt[i];
    cnt[i] = total;
    total += c;
  }
  if (pairs) {
#pragma omp parallel for schedule(dynamic, 64)
    for (long i = 0; i < n_nodes; ++i) {
      long o = cnt[i];
      for (long j = i + 1; j < n_nodes; ++j)
        if (frnn_d2(z + i * D, z + j * D, D) < r2) {
          if (o < max_pairs) {
            pairs[2 * o] = i;
            pairs[2 * o + 1] = j;
          }
          ++o;
        }
    }
  }
  if (n_pairs) *n_pairs = total;
  free(cnt);
  return 0;
}

/* The partners j > i of one row i, ascending (the pairs of oracle_frnn
 * whose first element is i); returns their count, writing at most max_out
 * of them to out. */
long oracle_frnn_row(const float *z, long n_nodes, int D, float r2, long i, int64_t *out,
                     long max_out) {
  long c = 0;
  for (long j = i + 1; j < n_nodes; ++j)
    if (frnn_d2(z + i * D, z + j * D, D) < r2) {
      if (out && c < max_out) out[c] = j;
      ++c;
    }
  return c;
}
