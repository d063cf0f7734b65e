// Host runtime of libgnn.so: the C ABI declared in include/gnn.h.
//
// gnn_create parses the fp32 weight blob (its own parser), converts every
// dense layer into the MFMA fragment order the kernels read (mlp.hip) and
// uploads it once.  gnn_infer enqueues the whole inference on the caller's
// stream: CSR build (csr.hip), node and edge encoders, T iterations of edge
// update -> segmented sums (agg.hip) -> node update, then the classifier.
// The inference workspace comes from a small cache owned by the handle: an
// idle entry is reused once the stream has been made to wait for the event
// that closed its previous call, so steady-state calls allocate nothing and
// one handle can serve several streams at once.  The other entry points
// allocate stream-ordered (hipMallocAsync/hipFreeAsync) from the device's
// default pool, whose release threshold is raised.
#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/gnn.h"
#include "gnn_internal.h"

using namespace gnn;

namespace {

thread_local std::string g_last_error;

int fail(int code, const char *fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return code;
}

}  // namespace

int gnn::set_error(int code, const char *msg) { return fail(code, "%s", msg ? msg : ""); }

namespace {

// ---------------------------------------------------------------- dims ---

int check_dims(const gnn_dims *d) {
  if (!d) return fail(GNN_E_INVALID_ARG, "dims is NULL");
  if (d->struct_size != sizeof(gnn_dims))
    return fail(GNN_E_INVALID_ARG, "dims.struct_size %u != %zu", d->struct_size,
                sizeof(gnn_dims));
  if (d->in_features < 1 || d->in_features > 16)
    return fail(d->in_features < 1 ? GNN_E_INVALID_ARG : GNN_E_UNSUPPORTED,
                "in_features %d outside 1..16", d->in_features);
  if (d->hidden <= 0 || d->hidden % 32)
    return fail(GNN_E_INVALID_ARG, "hidden %d is not a positive multiple of 32", d->hidden);
  if (d->hidden != 64 && d->hidden != 128)
    return fail(GNN_E_UNSUPPORTED, "hidden %d not supported (64 or 128)", d->hidden);
  if (d->n_iters < 0 || d->n_iters > 64)
    return fail(GNN_E_INVALID_ARG, "n_iters %d outside 0..64", d->n_iters);
  if (!(d->n_mp_weight_sets == 1 || (d->n_mp_weight_sets == d->n_iters && d->n_iters > 0)))
    return fail(GNN_E_INVALID_ARG, "n_mp_weight_sets %d must be 1 or n_iters",
                d->n_mp_weight_sets);
  if (d->dtype != GNN_FP32 && d->dtype != GNN_BF16)
    return fail(GNN_E_INVALID_ARG, "dtype %d unknown", d->dtype);
  if (!(d->ln_eps > 0.f) || !(d->ln_eps < 1.f))
    return fail(GNN_E_INVALID_ARG, "ln_eps %g outside (0, 1)", (double)d->ln_eps);
  if (d->flags & ~(GNN_VALIDATE_INDICES | GNN_LITERAL_GATHER | GNN_FP32_MFMA | GNN_F16_WEIGHTS))
    return fail(GNN_E_INVALID_ARG, "unknown flags");
  if ((d->flags & GNN_F16_WEIGHTS) &&
      (d->dtype != GNN_BF16 || (d->flags & (GNN_LITERAL_GATHER | GNN_FP32_MFMA))))
    return fail(GNN_E_INVALID_ARG,
                "GNN_F16_WEIGHTS needs dtype GNN_BF16 and neither GNN_LITERAL_GATHER nor "
                "GNN_FP32_MFMA");
  return GNN_OK;
}

size_t layer_floats(size_t fin, size_t fout, bool hidden) {
  return fin * fout + fout + (hidden ? 2 * fout : 0);
}

size_t weight_count(const gnn_dims *d) {
  const size_t F = d->in_features, H = d->hidden, S = d->n_mp_weight_sets;
  return layer_floats(F, H, true) + layer_floats(H, H, true) +          // node_enc
         layer_floats(2 * H, H, true) + layer_floats(H, H, true) +      // edge_enc
         S * 2 * (layer_floats(3 * H, H, true) + layer_floats(H, H, true)) +
         layer_floats(3 * H, H, true) + layer_floats(H, 1, false);       // edge_cls
}

// ------------------------------------------------------ weight layout ---

uint16_t f32_to_bf16(float f) {
  uint32_t u;
  memcpy(&u, &f, 4);
  if ((u & 0x7f800000u) == 0x7f800000u && (u & 0x007fffffu)) return 0x7fc0;  // NaN
  u += 0x7fffu + ((u >> 16) & 1u);  // round to nearest even
  return (uint16_t)(u >> 16);
}

// A blob layer: W [fout][fin] then b, gamma, beta.
struct BlobLayer {
  const float *W, *b, *g, *beta;
  int fin, fout;
};

// MFMA fragment orders (see mlp.hip).  With MB = H/32, lane = 0..63,
// i = lane % 32 and hh = lane / 32:
//  fp32, any K:        frag[g][mb][lane][t] = W[32mb+i][8g + 4hh + t]
//  bf16, B from HBM:   frag[g][mb][lane][s] = W[32mb+i][16g + 8hh + s]
//  bf16, B from accs:  frag[g][mb][lane][s] = W[32mb+i][16g + 8(s/4) + 4hh + s%4]
void frag_f32(const BlobLayer &L, float *dst) {
  const int MB = L.fout / 32, G = L.fin / 8;
  for (int g = 0; g < G; ++g)
    for (int mb = 0; mb < MB; ++mb)
      for (int lane = 0; lane < 64; ++lane)
        for (int t = 0; t < 4; ++t)
          dst[(((size_t)g * MB + mb) * 64 + lane) * 4 + t] =
              L.W[(size_t)(mb * 32 + lane % 32) * L.fin + 8 * g + 4 * (lane / 32) + t];
}

float bf16_to_f32(uint16_t b) {
  const uint32_t u = (uint32_t)b << 16;
  float f;
  memcpy(&f, &u, 4);
  return f;
}

// bf16 mode carries every weight as hi = bf16(W) and lo = bf16(W - hi).
void frag_bf16(const BlobLayer &L, bool from_acc, uint16_t *hi, uint16_t *lo) {
  const int MB = L.fout / 32, G = L.fin / 16;
  for (int g = 0; g < G; ++g)
    for (int mb = 0; mb < MB; ++mb)
      for (int lane = 0; lane < 64; ++lane)
        for (int s = 0; s < 8; ++s) {
          const int hh = lane / 32;
          const int k = from_acc ? 16 * g + 8 * (s / 4) + 4 * hh + s % 4 : 16 * g + 8 * hh + s;
          const float wv = L.W[(size_t)(mb * 32 + lane % 32) * L.fin + k];
          const size_t o = (((size_t)g * MB + mb) * 64 + lane) * 8 + s;
          hi[o] = f32_to_bf16(wv);
          lo[o] = f32_to_bf16(wv - bf16_to_f32(hi[o]));
        }
}

// ---- split-precision records (split.hip) ----
// A record holds the A operands of one 16-wide k-step for all MB = fout/32
// output blocks, [mb][part][lane][8] 16-bit values; slot j of lane l
// (hh = l / 32) multiplies input column k(g, hh, j) of row 32 mb + l % 32:
//   B from HBM:   k = 16 g + 8 hh + j
//   B from accs:  k = 16 g + 8 (j / 4) + 4 hh + j % 4

uint16_t f16_bits(_Float16 v) {
  uint16_t b;
  memcpy(&b, &v, 2);
  return b;
}

// Power of two s with max |s W| in [2^13, 2^14) (1 for an all-zero or
// non-finite W), over the whole (fout x fin) layer.
float pow2_scale(const BlobLayer &L) {
  float mx = 0.f;
  const size_t n = (size_t)L.fout * L.fin;
  for (size_t i = 0; i < n; ++i) mx = fmaxf(mx, fabsf(L.W[i]));
  if (!(mx > 0.f) || !std::isfinite(mx)) return 1.f;
  int e = 0;
  (void)frexpf(mx, &e);  // mx = m 2^e, m in [0.5, 1)
  int k = 14 - e;
  k = k < -40 ? -40 : (k > 40 ? 40 : k);
  return ldexpf(1.f, k);
}

// Largest value a LayerNorm/ReLU output of layer L can take:
// |(y - mean) / sqrt(var + eps)| <= sqrt(H - 1) for every feature.
double ln_out_bound(const BlobLayer &L) {
  double b = 0.0;
  const double r = sqrt((double)L.fout - 1.0);
  for (int f = 0; f < L.fout; ++f) {
    const double v = fabs((double)L.g[f]) * r + fabs((double)L.beta[f]);
    if (!(v <= 1e30)) return INFINITY;
    b = v > b ? v : b;
  }
  return b;
}

// f16x2 records of s * W[:, c0 : c0 + K]: parts w1 = fp16(sW), w2 = fp16(sW - w1).
// Input feature of slot j (0..7) of lane half hh in k-step g of a record
// stream (rec_f16x2, rec_bf16x2), by how the kernel supplies the operand:
//   grp = 0: row slices from memory, k = 16 g + 8 hh + j;
//   grp < 0: the previous layer's accumulators, k = 16 g + 8 (j / 4) + 4 hh + j % 4;
//   grp > 0: line order (the node update's layer-1 rows): groups of grp
//            k-steps cover 16 grp consecutive features, lane half hh the
//            8 grp features from 8 grp hh on, k-step g % grp of the group its
//            8 features from 8 (g % grp) on.
inline int node_line_k(int g, int hh, int j, int grp) {
  if (grp < 0) return 16 * g + 8 * (j / 4) + 4 * hh + j % 4;
  if (grp == 0) return 16 * g + 8 * hh + j;
  return 16 * grp * (g / grp) + 8 * grp * hh + 8 * (g % grp) + j;
}

std::vector<uint16_t> rec_f16x2(const BlobLayer &L, int c0, int K, float s, int grp) {
  const int MB = L.fout / 32, G = K / 16;
  std::vector<uint16_t> out((size_t)G * MB * 2 * 64 * 8);
  for (int g = 0; g < G; ++g)
    for (int mb = 0; mb < MB; ++mb)
      for (int lane = 0; lane < 64; ++lane)
        for (int j = 0; j < 8; ++j) {
          const int hh = lane / 32;
          const int k = node_line_k(g, hh, j, grp);
          const float wv = s * L.W[(size_t)(mb * 32 + lane % 32) * L.fin + c0 + k];
          const _Float16 p1 = (_Float16)wv;
          const _Float16 p2 = (_Float16)(wv - (float)p1);
          const size_t o = ((((size_t)g * MB + mb) * 2) * 64 + lane) * 8 + j;
          out[o] = f16_bits(p1);
          out[o + 64 * 8] = f16_bits(p2);
        }
  return out;
}

// bf16 hi/lo records of sc * W[:, c0 : c0 + K]: hi = bf16(sc W), lo =
// bf16(sc W - hi) (the bf16 model's weights; sc a power of two, so the pair
// is sc times the pair of W).
// One-part fp16 records of s * W[:, c0 : c0 + K] (the bf16 model with fp16
// weights), laid out as rec_f16x2's first part: [g][mb][lane] x 8 values.
std::vector<uint16_t> rec_f16x1(const BlobLayer &L, int c0, int K, float s, int grp) {
  const int MB = L.fout / 32, G = K / 16;
  std::vector<uint16_t> out((size_t)G * MB * 64 * 8);
  for (int g = 0; g < G; ++g)
    for (int mb = 0; mb < MB; ++mb)
      for (int lane = 0; lane < 64; ++lane)
        for (int j = 0; j < 8; ++j) {
          const int k = node_line_k(g, lane / 32, j, grp);
          const float wv = s * L.W[(size_t)(mb * 32 + lane % 32) * L.fin + c0 + k];
          out[(((size_t)g * MB + mb) * 64 + lane) * 8 + j] = f16_bits((_Float16)wv);
        }
  return out;
}

std::vector<uint16_t> rec_bf16x2(const BlobLayer &L, int c0, int K, int grp, float sc = 1.f) {
  const int MB = L.fout / 32, G = K / 16;
  std::vector<uint16_t> out((size_t)G * MB * 2 * 64 * 8);
  for (int g = 0; g < G; ++g)
    for (int mb = 0; mb < MB; ++mb)
      for (int lane = 0; lane < 64; ++lane)
        for (int j = 0; j < 8; ++j) {
          const int hh = lane / 32;
          const int k = node_line_k(g, hh, j, grp);
          const float wv = sc * L.W[(size_t)(mb * 32 + lane % 32) * L.fin + c0 + k];
          const uint16_t hi = f32_to_bf16(wv);
          const size_t o = ((((size_t)g * MB + mb) * 2) * 64 + lane) * 8 + j;
          out[o] = hi;
          out[o + 64 * 8] = f32_to_bf16(wv - bf16_to_f32(hi));
        }
  return out;
}

// bf16 model: power of two s for the fp16 projections s P = s [W_s h; W_d h]
// that edge-side layer L reads (columns [0, H) and [H, 2H) of its W), with
// s max_f sum_k |W[f][k]| hb <= 2^15 for an h bound hb, as large as that
// allows within [2^-40, 2^40]; 0 if none fits.
float proj_f16_scale(const BlobLayer &L, int H, double hb) {
  double m = 0.0;
  for (int f = 0; f < L.fout; ++f)
    for (int half = 0; half < 2; ++half) {
      double r = 0.0;
      for (int k = half * H; k < half * H + H; ++k) r += fabs((double)L.W[(size_t)f * L.fin + k]);
      m = r > m ? r : m;
    }
  const double bound = m * hb;
  if (!(bound <= 1e300)) return 0.f;
  if (!(bound > 0.0)) return 1.f;
  int e = 0;
  (void)frexp(32768.0 / bound, &e);  // 2^(e-1) <= 2^15 / bound < 2^e
  int k = e - 1;
  k = k < -40 ? -40 : (k > 40 ? 40 : k);
  const double sc = ldexp(1.0, k);
  return sc * bound <= 32768.0 ? (float)sc : 0.f;
}

// Builds one host staging image of all device weights, section by section,
// each 256-byte aligned; device pointers are fixed up after the upload.
struct Staging {
  std::vector<unsigned char> bytes;
  size_t add(const void *src, size_t n) {
    const size_t off = (bytes.size() + 255) & ~(size_t)255;
    bytes.resize(off + n);
    if (src) memcpy(bytes.data() + off, src, n);
    return off;
  }
};

struct LayerOff {
  size_t w = 0, w_lo = 0, b = 0, g = 0, beta = 0;
  bool has_ln = false, has_lo = false;
};
struct MlpOff {
  LayerOff l0, l1;
};

}  // namespace

// Extra weights of the regrouped first layers: W_e column blocks (H x H) and
// the node-kernel streams with the stacked projections [W_s; W_d].  In the
// split path every matrix is in 16-bit records and the edge kernels
// read W2 from records too; in the fp32 path they are fp32 MFMA fragments.
struct FactDev {
  bool split = false;  // split.hip kernels (fp32 split products, or the bf16 model)
  bool bf16 = false;   // with split: the bf16 model
  int prec = 0;        // split.hip precision: 0 fp32, 1 bf16 hi/lo, 2 bf16 with fp16 weights
  const void *we_cls = nullptr;
  std::vector<const void *> we_em;
  // node-kernel streams: encoder (W2 | two projections) and, per
  // iteration, update (W1 | W2 | projection for the next edge consumer)
  const void *enc_stream = nullptr;
  std::vector<const void *> upd_stream;
  int enc_chunks = 0, upd_chunks = 0;
  // split path: W2 records of the edge-side MLPs and the power-of-two scales
  // (s1: first layer incl. the stored projections; s2: W2)
  const void *w2_ee = nullptr;
  std::vector<const void *> w2_em;
  float s1_ee = 1.f, s2_ee = 1.f, s1_cls = 1.f, s2_ne = 1.f;
  std::vector<float> s1_em, s2_em, s1_nm, s2_nm;
  float row_bound = 0.f;  // bound of any h or e entry (LayerNorm/ReLU outputs)
  int grid_enc = 0, grid_upd = 0, grid_cls = 0, grid_node = 0;  // persistent grids
  // fp16 weights: the first update's W_e records with e0 taken from the
  // accumulators (the edge encoder then runs inside that update)
  const void *we_em0_acc = nullptr;
  int grid_encupd = 0;
};

struct gnn_handle {
  gnn_dims dims;
  int device = 0;
  bool factored = false;
  void *dev_weights = nullptr;
  MlpDev node_enc, edge_enc, cls;
  std::vector<MlpDev> edge_mlp, node_mlp;
  FactDev fd;
  // profiling: recorded (stage, start, end) event pairs not yet read, the
  // running totals and a pool of reusable events.  A call's total shares the
  // events of its first and last stages (its mark owns neither).
  struct Mark {
    int stage;
    hipEvent_t a, b;
    bool own_a, own_b;
  };
  std::mutex prof_mu;
  bool prof_on = false;
  bool prof_sample = false;  // GNN_PROFILE_SAMPLE: one iteration's stages per call
  std::vector<Mark> prof_pending;
  std::vector<hipEvent_t> prof_free;
  int32_t prof_calls = 0;
  int64_t prof_launches[GNN_N_STAGES] = {};
  double prof_ms[GNN_N_STAGES] = {};
  // Inference workspaces kept across calls.  `done` is recorded on `last`
  // after each call that used the entry; a later call (on any stream) waits
  // for it before touching the memory.  `busy` covers the host side of a call.
  struct WsEntry {
    void *base;
    size_t bytes;
    hipEvent_t done;
    hipStream_t last;
    bool busy, recorded;
  };
  std::mutex ws_mu;
  std::vector<WsEntry> ws;
  // Most bytes of workspace the handle may hold at once (cached entries plus
  // call-owned allocations in flight); 0 = no limit.
  size_t ws_limit = 0;
  size_t ws_held = 0;
};

namespace {

// Layer kinds for the converter.
enum class WKind { Plain, PlainT, FragMem, FragAcc };

LayerOff stage_layer(Staging &st, const BlobLayer &L, WKind kind, bool bf16, bool has_ln) {
  LayerOff o;
  o.has_ln = has_ln;
  const size_t nW = (size_t)L.fin * L.fout;
  if (kind == WKind::Plain) {
    o.w = st.add(L.W, nW * sizeof(float));
  } else if (kind == WKind::PlainT) {
    std::vector<float> t(nW);  // [in][out]
    for (int o2 = 0; o2 < L.fout; ++o2)
      for (int k = 0; k < L.fin; ++k) t[(size_t)k * L.fout + o2] = L.W[(size_t)o2 * L.fin + k];
    o.w = st.add(t.data(), nW * sizeof(float));
  } else if (!bf16) {
    std::vector<float> f(nW);
    frag_f32(L, f.data());
    o.w = st.add(f.data(), nW * sizeof(float));
  } else {
    std::vector<uint16_t> hi(nW), lo(nW);
    frag_bf16(L, kind == WKind::FragAcc, hi.data(), lo.data());
    o.w = st.add(hi.data(), nW * sizeof(uint16_t));
    o.w_lo = st.add(lo.data(), nW * sizeof(uint16_t));
    o.has_lo = true;
  }
  o.b = st.add(L.b, L.fout * sizeof(float));
  if (has_ln) {
    o.g = st.add(L.g, L.fout * sizeof(float));
    o.beta = st.add(L.beta, L.fout * sizeof(float));
  }
  return o;
}

// fp32 fragments of an arbitrary (fout x fin) row-major matrix.
size_t stage_frag_f32(Staging &st, const std::vector<float> &W, int fout, int fin) {
  BlobLayer L{W.data(), nullptr, nullptr, nullptr, fin, fout};
  std::vector<float> f(W.size());
  frag_f32(L, f.data());
  return st.add(f.data(), f.size() * sizeof(float));
}

// Column block W[:, c0:c0+H] of an (H x fin) layer, as an (H x H) matrix.
std::vector<float> col_block(const BlobLayer &L, int H, int c0) {
  std::vector<float> P((size_t)H * H);
  for (int o = 0; o < H; ++o)
    for (int k = 0; k < H; ++k) P[(size_t)o * H + k] = L.W[(size_t)o * L.fin + c0 + k];
  return P;
}

std::vector<float> frag_of(const float *W, int fout, int fin) {
  BlobLayer L{W, nullptr, nullptr, nullptr, fin, fout};
  std::vector<float> f((size_t)fout * fin);
  frag_f32(L, f.data());
  return f;
}

void append(std::vector<float> &dst, const std::vector<float> &src) {
  dst.insert(dst.end(), src.begin(), src.end());
}

// Fragments of the two projection halves W[:, 0:H] and W[:, H:2H].
void append_projection(std::vector<float> &dst, const BlobLayer &L, int H) {
  append(dst, frag_of(col_block(L, H, 0).data(), H, H));
  append(dst, frag_of(col_block(L, H, H).data(), H, H));
}

LayerDev fix_layer(const LayerOff &o, const unsigned char *base) {
  LayerDev d;
  d.w = base + o.w;
  if (o.has_lo) d.w_lo = base + o.w_lo;
  d.b = (const float *)(base + o.b);
  if (o.has_ln) {
    d.g = (const float *)(base + o.g);
    d.beta = (const float *)(base + o.beta);
  }
  return d;
}

MlpDev fix_mlp(const MlpOff &o, const unsigned char *base) {
  return MlpDev{fix_layer(o.l0, base), fix_layer(o.l1, base)};
}

struct DeviceGuard {
  int prev = -1;
  explicit DeviceGuard(int dev) {
    if (hipGetDevice(&prev) != hipSuccess) prev = -1;
    if (prev != dev) (void)hipSetDevice(dev);
  }
  ~DeviceGuard() {
    int cur = -1;
    if (prev >= 0 && hipGetDevice(&cur) == hipSuccess && cur != prev) (void)hipSetDevice(prev);
  }
};

size_t align256(size_t n) { return (n + 255) & ~(size_t)255; }

// Workspace carve-up for one call.
struct Workspace {
  void *base = nullptr;
  size_t bytes = 0;
  void *h = nullptr, *e = nullptr, *ain = nullptr, *aout = nullptr;
  float *pa = nullptr, *pb = nullptr;  // node projections (regrouped fp32 path)
  int32_t *rp_in = nullptr, *rp_out = nullptr, *perm_in = nullptr, *perm_out = nullptr;
  CsrScratch csr{};
  int32_t *flag = nullptr;
  // regrouped path: edges in source order ([2][E], written by the CSR
  // build), the in-CSR over that order, and the unit pieces of the fused
  // out-sums ([units][2][H] fp32)
  int32_t *eis = nullptr, *inv = nullptr, *q_in = nullptr;
  float *part = nullptr;
};

size_t plan_workspace(Workspace &w, int64_t N, int64_t E, int H, size_t act_bytes,
                      bool factored, bool fused) {
  size_t off = 0;
  auto take = [&](size_t n) {
    const size_t o = off;
    off += align256(n > 0 ? n : 1);
    return o;
  };
  const size_t o_h = take((size_t)N * H * act_bytes);
  const size_t o_e = take((size_t)E * H * act_bytes);
  const size_t o_ai = take((size_t)N * H * act_bytes);
  const size_t o_ao = take((size_t)N * H * act_bytes);
  const size_t o_rpi = take((size_t)(N + 1) * 4), o_rpo = take((size_t)(N + 1) * 4);
  const size_t o_pi = take((size_t)E * 4), o_po = take((size_t)E * 4);
  const size_t o_sa = take((size_t)E * 16), o_sb = take((size_t)E * 16);
  const size_t o_st = take(csr_scratch_bytes(E, N));
  const size_t o_eis = factored ? take((size_t)E * 8) : 0;
  const size_t o_inv = factored ? take((size_t)E * 4) : 0;
  const size_t o_qin = factored ? take((size_t)E * 4) : 0;
  const size_t o_flag = take(4);
  const size_t o_pa = factored ? take((size_t)N * 2 * H * 4) : 0;
  const size_t o_pb = factored ? take((size_t)N * 2 * H * 4) : 0;
  const size_t o_part = fused ? take((size_t)((E + 31) / 32) * 2 * H * 4) : 0;
  if (w.base) {
    if (factored) {
      w.pa = (float *)((unsigned char *)w.base + o_pa);
      w.pb = (float *)((unsigned char *)w.base + o_pb);
    }
    if (fused) w.part = (float *)((unsigned char *)w.base + o_part);
    unsigned char *b = (unsigned char *)w.base;
    w.h = b + o_h;
    w.e = b + o_e;
    w.ain = b + o_ai;
    w.aout = b + o_ao;
    w.rp_in = (int32_t *)(b + o_rpi);
    w.rp_out = (int32_t *)(b + o_rpo);
    w.perm_in = (int32_t *)(b + o_pi);
    w.perm_out = (int32_t *)(b + o_po);
    w.csr.pairs_a = (uint2 *)(b + o_sa);
    w.csr.pairs_b = (uint2 *)(b + o_sb);
    w.csr.status = (uint32_t *)(b + o_st);
    w.flag = (int32_t *)(b + o_flag);
    if (factored) {
      w.eis = (int32_t *)(b + o_eis);
      w.inv = (int32_t *)(b + o_inv);
      w.q_in = (int32_t *)(b + o_qin);
    }
  }
  return off;
}

int check_counts(gnn_handle *h, int64_t N, int64_t E) {
  if (!h) return fail(GNN_E_INVALID_ARG, "handle is NULL");
  if (N < 0 || E < 0) return fail(GNN_E_INVALID_ARG, "negative count (n_nodes %lld, n_edges %lld)",
                                  (long long)N, (long long)E);
  if (N > INT32_MAX || E > INT32_MAX)
    return fail(GNN_E_INVALID_ARG, "count above INT32_MAX");
  if (E > 0 && N == 0) return fail(GNN_E_INVALID_ARG, "n_edges > 0 with n_nodes == 0");
  if (E >= CSR_MAX_ITEMS)
    return fail(GNN_E_UNSUPPORTED, "n_edges %lld: the CSR build takes at most 2^30 - 1 edges",
                (long long)E);
  return GNN_OK;
}

#define HIP_TRY(expr)                                                                \
  do {                                                                               \
    hipError_t e_ = (expr);                                                          \
    if (e_ != hipSuccess) {                                                          \
      rc = fail(GNN_E_HIP, "%s failed: %s", #expr, hipGetErrorString(e_));           \
      goto out;                                                                      \
    }                                                                                \
  } while (0)

// Times the stages of a call when profiling is on.  Each stage gets two
// events that its kernels' dispatches mark themselves (StageEvents): the
// first kernel's start and the last one's end, so a stage's time is the time
// its kernels ran, with no marker work added to the stream.  The call's total
// runs from its first stage's start to its last stage's end.
struct StageTimer {
  gnn_handle *h;
  bool on, sample;
  hipEvent_t a = nullptr, b = nullptr;          // the open stage's events
  hipEvent_t first = nullptr, last_b = nullptr;  // the call's first start, last end
  StageTimer(gnn_handle *h_, bool count_call) : h(h_) {
    std::lock_guard<std::mutex> lk(h->prof_mu);
    on = h->prof_on;
    sample = h->prof_sample;
    if (on && count_call) ++h->prof_calls;
  }
  ~StageTimer() {  // a stage left open by an error
    gnn::stage_events() = gnn::StageEvents{};
    if (a) put(a);
    if (b) put(b);
  }
  hipEvent_t get() {
    std::lock_guard<std::mutex> lk(h->prof_mu);
    hipEvent_t e = nullptr;
    if (!h->prof_free.empty()) {
      e = h->prof_free.back();
      h->prof_free.pop_back();
    } else if (hipEventCreate(&e) != hipSuccess) {
      (void)hipGetLastError();
      e = nullptr;
    }
    return e;
  }
  void put(hipEvent_t e) {
    std::lock_guard<std::mutex> lk(h->prof_mu);
    h->prof_free.push_back(e);
  }
  // in_sample: the stage belongs to the iteration that GNN_PROFILE_SAMPLE
  // times (every stage is timed in the full mode)
  void begin(bool in_sample = false) {
    if (!on || (sample && !in_sample)) return;
    a = get();
    b = get();
    if (!a || !b) {
      if (a) put(a);
      if (b) put(b);
      a = b = nullptr;
      return;
    }
    gnn::stage_events() = gnn::StageEvents{a, b, false};
  }
  void end(int stage) {
    if (!a) return;
    gnn::StageEvents &ev = gnn::stage_events();
    const bool launched = ev.launched;
    ev = gnn::StageEvents{};
    if (!launched) {  // nothing ran in this stage
      put(a);
      put(b);
    } else {
      std::lock_guard<std::mutex> lk(h->prof_mu);
      h->prof_pending.push_back({stage, a, b, true, true});
      if (!first) first = a;
      last_b = b;
    }
    a = b = nullptr;
  }
  // Records the call's total (events owned by the first and last stages).
  void finish(int stage) {
    if (!first || sample) return;
    std::lock_guard<std::mutex> lk(h->prof_mu);
    h->prof_pending.push_back({stage, first, last_b, false, false});
  }
};

// Parses a byte count: decimal digits with an optional binary suffix k, m or
// g (either case).  Returns false for anything else or on overflow.
bool parse_bytes(const char *txt, size_t *out) {
  if (!txt || !*txt) return false;
  size_t v = 0;
  const char *p = txt;
  for (; *p >= '0' && *p <= '9'; ++p) {
    const size_t d = (size_t)(*p - '0');
    if (v > (SIZE_MAX - d) / 10) return false;
    v = v * 10 + d;
  }
  if (p == txt) return false;
  int shift = 0;
  if (*p) {
    switch (*p) {
      case 'k': case 'K': shift = 10; break;
      case 'm': case 'M': shift = 20; break;
      case 'g': case 'G': shift = 30; break;
      default: return false;
    }
    if (p[1]) return false;
  }
  if (shift && v > (SIZE_MAX >> shift)) return false;
  *out = v << shift;
  return true;
}

// Fails with GNN_E_OOM if taking `more` bytes would exceed the handle's
// workspace limit (caller holds ws_mu).
int ws_check_limit(gnn_handle *h, size_t more) {
  if (h->ws_limit && h->ws_held + more > h->ws_limit)
    return fail(GNN_E_OOM,
                "workspace limit of %zu bytes reached: the handle holds %zu bytes and this call "
                "needs %zu more (see gnn_set_workspace_limit)",
                h->ws_limit, h->ws_held, more);
  return GNN_OK;
}

// Most cached workspaces per handle; beyond this, calls share entries
// (ordered by events) rather than allocate more.
constexpr size_t kMaxCachedWorkspaces = 16;

size_t ws_round(size_t bytes) {
  const size_t mib = size_t(1) << 20, b = bytes + bytes / 8;  // slack for growing events
  return (b + mib - 1) / mib * mib;
}

// Gives a call on `stream` a workspace of at least `bytes`.  Preference: an
// idle cached entry last used on this stream, then one whose last call has
// finished, then a new cached entry, then (cache full) an idle entry still in
// use on another stream, then replacing an idle entry that is too small.
// With every entry busy on the host, the call gets a stream-ordered
// allocation of its own (*slot = -1), freed at its end.
int ws_acquire(gnn_handle *h, size_t bytes, hipStream_t stream, void **base, int *slot) {
  std::lock_guard<std::mutex> lk(h->ws_mu);
  auto &ws = h->ws;
  int pick = -1, rank = 3;
  for (int i = 0; i < (int)ws.size(); ++i) {
    const auto &e = ws[i];
    if (e.busy || e.bytes < bytes) continue;
    // (a query that does not return hipSuccess, "not ready" included, is
    // cleared from the thread's last-error state, which the launch wrappers
    // of this call report)
    int r = 1;
    if (e.last == stream) {
      r = 0;
    } else if (e.recorded && hipEventQuery(e.done) != hipSuccess) {
      (void)hipGetLastError();
      r = 2;
    }
    if (r < rank || (r == rank && e.bytes < ws[pick].bytes)) {
      pick = i;
      rank = r;
    }
  }
  // A buffer still in use on another stream is taken (after its work) only
  // when the cache has no room for a new one, or the workspace limit none.
  if (pick >= 0 && rank == 2 && ws.size() < kMaxCachedWorkspaces &&
      !(h->ws_limit && h->ws_held + ws_round(bytes) > h->ws_limit))
    pick = -1;
  if (pick < 0) {
    int victim = -1;
    for (int i = 0; i < (int)ws.size() && victim < 0; ++i)  // emptied by a release
      if (!ws[i].busy && !ws[i].base) victim = i;
    if (victim < 0 && ws.size() >= kMaxCachedWorkspaces)
      for (int i = 0; i < (int)ws.size() && victim < 0; ++i)
        if (!ws[i].busy) victim = i;
    if (ws.size() >= kMaxCachedWorkspaces && victim < 0) {
      *slot = -1;
      if (const int lr = ws_check_limit(h, bytes)) return lr;
      const hipError_t ae = hipMallocAsync(base, bytes, stream);
      if (ae == hipSuccess) {
        h->ws_held += bytes;
        return GNN_OK;
      }
      (void)hipGetLastError();
      return fail(ae == hipErrorOutOfMemory ? GNN_E_OOM : GNN_E_HIP,
                  "hipMallocAsync(%zu bytes) failed: %s", bytes, hipGetErrorString(ae));
    }
    if (victim >= 0) {
      // Replaced in place: busy entries keep their indices.  Its last call
      // must end before the memory goes back.
      auto &v = ws[victim];
      if (v.base && ws_check_limit(h, ws_round(bytes) - std::min(v.bytes, ws_round(bytes))))
        return GNN_E_OOM;
      if (v.base && ((v.recorded && hipEventSynchronize(v.done) != hipSuccess) ||
                     hipFree(v.base) != hipSuccess)) {
        (void)hipGetLastError();
        return fail(GNN_E_HIP, "releasing a cached workspace failed");
      }
      h->ws_held -= v.bytes;
      v.base = nullptr;
      v.bytes = 0;
      v.recorded = false;
      pick = victim;
    } else {
      if (const int lr = ws_check_limit(h, ws_round(bytes))) return lr;
      gnn_handle::WsEntry e{nullptr, 0, nullptr, stream, false, false};
      if (hipEventCreateWithFlags(&e.done, hipEventDisableTiming) != hipSuccess) {
        (void)hipGetLastError();
        return fail(GNN_E_HIP, "hipEventCreate for a workspace failed");
      }
      ws.push_back(e);
      pick = (int)ws.size() - 1;
    }
    auto &e = ws[pick];
    const size_t want = ws_round(bytes);
    if (const int lr = ws_check_limit(h, want)) return lr;
    const hipError_t ae = hipMalloc(&e.base, want);
    if (ae != hipSuccess) {  // the entry stays, empty, for a later call
      (void)hipGetLastError();
      e.base = nullptr;
      return fail(ae == hipErrorOutOfMemory ? GNN_E_OOM : GNN_E_HIP,
                  "hipMalloc(%zu bytes) of a workspace failed: %s", want, hipGetErrorString(ae));
    }
    e.bytes = want;
    h->ws_held += want;
  }
  auto &e = ws[pick];
  if (e.recorded && hipStreamWaitEvent(stream, e.done, 0) != hipSuccess)
    return fail(GNN_E_HIP, "hipStreamWaitEvent on a cached workspace failed");
  e.busy = true;
  e.last = stream;
  *base = e.base;
  *slot = pick;
  return GNN_OK;
}

// Ends the host side of a call: marks the end of its work on `stream` so the
// next user of the entry can wait for it.
int ws_release(gnn_handle *h, int slot, void *base, size_t bytes, hipStream_t stream) {
  if (slot < 0) {
    {
      std::lock_guard<std::mutex> lk(h->ws_mu);
      h->ws_held -= bytes;
    }
    const hipError_t fe = hipFreeAsync(base, stream);
    return fe == hipSuccess ? GNN_OK
                            : fail(GNN_E_HIP, "hipFreeAsync failed: %s", hipGetErrorString(fe));
  }
  std::lock_guard<std::mutex> lk(h->ws_mu);
  auto &e = h->ws[slot];
  int rc = GNN_OK;
  if (hipEventRecord(e.done, stream) == hipSuccess) {
    e.recorded = true;
  } else {  // no event to wait for: finish the call's work here instead
    (void)hipGetLastError();
    e.recorded = false;
    if (hipStreamSynchronize(stream) != hipSuccess)
      rc = fail(GNN_E_HIP, "closing a call on its workspace failed");
  }
  e.busy = false;
  return rc;
}

// What a call should produce.
struct RunOut {
  float *scores = nullptr, *logits = nullptr;  // classifier outputs
  int stop_iter = -1;                          // >= 0: stop after that many iterations
  float *h = nullptr, *e = nullptr, *ain = nullptr, *aout = nullptr;  // debug exports
  bool csr_only = false;
  int32_t *rp_in = nullptr, *perm_in = nullptr, *rp_out = nullptr, *perm_out = nullptr;
  // A caller-provided workspace of ext_bytes bytes instead of the handle's
  // cache (no allocation, no profiling events): the no-allocation entry point.
  void *ext_base = nullptr;
  size_t ext_bytes = 0;
};

int run(gnn_handle *hd, const float *x, const int32_t *ei, int64_t N, int64_t E,
        hipStream_t stream, const RunOut &ro) {
  const gnn_dims &d = hd->dims;
  const int H = d.hidden;
  const Act act = d.dtype == GNN_BF16 ? Act::BF16 : Act::F32;
  // the edge rows of the bf16 model with fp16 weights are held in fp16
  const Act eact = hd->factored && hd->fd.split && hd->fd.prec == 2 ? Act::F16 : act;
  const size_t ab = act == Act::F32 ? 4 : 2;
  const int32_t n = (int32_t)N, m = (int32_t)E;
  int rc = GNN_OK;
  Workspace w;
  DeviceGuard guard(hd->device);
  // The launch wrappers report hipGetLastError(): drop whatever an earlier
  // runtime call of this thread left there, so that only this call's own
  // launches are reported.
  (void)hipGetLastError();
  StageTimer st(hd, ro.ext_base == nullptr);
  if (ro.ext_base) st.on = false;  // creating events may allocate

  const bool fac = hd->factored;
  // the edge update sums its rows per source itself (split kernels)
  const bool fused = fac && hd->fd.split;
  w.bytes = plan_workspace(w, N, E, H, ab, fac, fused);
  int slot = -1;
  if (ro.ext_base) {
    if (w.bytes > ro.ext_bytes)
      return fail(GNN_E_INVALID_ARG,
                  "this event needs %zu bytes of scratch (n_nodes %lld, n_edges %lld); the "
                  "no-allocation entry point has %zu",
                  w.bytes, (long long)N, (long long)E, ro.ext_bytes);
    w.base = ro.ext_base;
  } else {
    rc = ws_acquire(hd, w.bytes, stream, &w.base, &slot);
    if (rc != GNN_OK) return rc;
  }
  plan_workspace(w, N, E, H, ab, fac, fused);

  if (d.flags & GNN_VALIDATE_INDICES) {
    int32_t bad = 0;
    HIP_TRY(launch_fill_i32(w.flag, 1, 0, stream));
    HIP_TRY(launch_validate(ei, E, n, w.flag, stream));
    HIP_TRY(hipMemcpyAsync(&bad, w.flag, 4, hipMemcpyDeviceToHost, stream));
    HIP_TRY(hipStreamSynchronize(stream));
    if (bad) {
      rc = fail(GNN_E_INDEX, "edge_index holds an index outside [0, %d)", n);
      goto out;
    }
  }

  {
    int32_t *rpi = ro.rp_in ? ro.rp_in : w.rp_in, *pi = ro.perm_in ? ro.perm_in : w.perm_in;
    int32_t *rpo = ro.rp_out ? ro.rp_out : w.rp_out, *po = ro.perm_out ? ro.perm_out : w.perm_out;
    st.begin();
    // The regrouped kernels keep the edge rows in source order (a node's
    // out-edges are consecutive); outputs go back to input order.  The CSR
    // build writes that order as well.
    HIP_TRY(build_csr(ei, m, n, rpi, pi, rpo, po, w.csr, w.eis, w.inv, w.q_in, stream));
    st.end(GNN_STAGE_CSR);
    if (ro.csr_only) {
      // the sort's look-back wait is bounded; report a pass that gave up
      uint32_t err = 0;
      HIP_TRY(hipMemcpyAsync(&err, csr_err_word(w.csr, m, n), 4, hipMemcpyDeviceToHost, stream));
      HIP_TRY(hipStreamSynchronize(stream));
      if (err) rc = fail(GNN_E_HIP, "CSR sort: a tile's look-back wait ran out");
      goto out;
    }
    w.rp_in = rpi;
    w.perm_in = pi;
    w.rp_out = rpo;
    w.perm_out = po;
  }

  if (fac) {
    const FactDev &fd = hd->fd;
    const int T = ro.stop_iter >= 0 ? (ro.stop_iter < d.n_iters ? ro.stop_iter : d.n_iters)
                                    : d.n_iters;
    auto set_of = [&](int t) { return d.n_mp_weight_sets == 1 ? 0 : t; };
    // node encoder -> h0, projections for the edge encoder (pa) and for the
    // first edge update, or the classifier when there is no iteration (pb)
    NodeArgs na;
    na.n_rows = N;
    na.x = x;
    na.F = d.in_features;
    na.mlp = hd->node_enc;
    na.wstream = (const float *)fd.enc_stream;
    na.nchunks = fd.enc_chunks;
    na.s2 = fd.s2_ne;
    na.nproj = 2;
    // with no iteration h0 feeds the classifier only through pb
    na.h_out = T == 0 && ro.stop_iter < 0 ? nullptr : (float *)w.h;
    na.p_out[0] = w.pa;
    na.p_out[1] = w.pb;
    // the edge MLP that reads the projections stored after node update t
    // (t = -1: the node encoder's second projection)
    auto consumer = [&](int t, const MlpDev **m, float *s1) {
      if (t + 1 < T) {
        *m = &hd->edge_mlp[set_of(t + 1)];
        *s1 = fd.split ? fd.s1_em[set_of(t + 1)] : 1.f;
      } else {
        *m = &hd->cls;
        *s1 = fd.split ? fd.s1_cls : 1.f;
      }
    };
    {
      na.pbias[0] = hd->edge_enc.l0.b;
      na.ps1[0] = fd.split ? fd.s1_ee : 1.f;
      const MlpDev *m2 = nullptr;
      consumer(-1, &m2, &na.ps1[1]);
      na.pbias[1] = m2->l0.b;
    }
    na.eps = d.ln_eps;
    st.begin();
    HIP_TRY(fd.split ? launch_node_split(true, H, na, fd.grid_node, fd.prec, stream)
                     : launch_node_f32(true, H, na, fd.grid_node, stream));
    st.end(GNN_STAGE_NODE_ENC);

    auto edge_args = [&](const float *P, const MlpDev &m) {
      EdgeArgs ea;
      ea.n_rows = E;
      ea.n_nodes = n;
      ea.src_idx = w.eis;
      ea.dst_idx = w.eis + E;
      ea.P = P;
      ea.b1 = m.l0.b;
      ea.g1 = m.l0.g;
      ea.beta1 = m.l0.beta;
      ea.w2 = (const float *)m.l1.w;
      ea.b2 = m.l1.b;
      ea.g2 = m.l1.g;
      ea.beta2 = m.l1.beta;
      ea.eps = d.ln_eps;
      return ea;
    };
    auto launch_edge = [&](EdgeMode mode, const EdgeArgs &ea, int grid) {
      return fd.split ? launch_edge_split(mode, H, ea, grid, fd.prec, stream)
                      : launch_edge_f32(mode, H, ea, grid, stream);
    };
    // With fp16 weights the edge encoder runs inside the first update, so
    // that e0 never goes to HBM and back (not for gnn_debug_stages, which
    // copies e0 out when stop_iter is 0 and runs the two kernels apart).
    const bool enc_in_upd = fd.prec == 2 && fused && T >= 1 && ro.stop_iter < 0;
    EdgeArgs enc_a = edge_args(w.pa, hd->edge_enc);
    enc_a.e_out = (float *)w.e;
    if (fd.split) {
      enc_a.w2 = (const float *)fd.w2_ee;
      enc_a.s1 = fd.s1_ee;
      enc_a.s2 = fd.s2_ee;
    }
    if (!enc_in_upd) {
      st.begin();
      HIP_TRY(launch_edge(EdgeMode::Enc, enc_a, fd.grid_enc));
      st.end(GNN_STAGE_EDGE_ENC);
    }
    for (int t = 0; t < T; ++t) {
      const int k = set_of(t);
      EdgeArgs ea = edge_args(w.pb, hd->edge_mlp[k]);
      ea.e_in = (const float *)w.e;
      ea.we = (const float *)fd.we_em[k];
      ea.e_out = (float *)w.e;  // in place: a wave reads its rows before writing them
      if (fd.split) {
        ea.w2 = (const float *)fd.w2_em[k];
        ea.s1 = fd.s1_em[k];
        ea.s2 = fd.s2_em[k];
      }
      if (fused) {
        ea.agg_out = w.aout;
        ea.agg_part = w.part;
      }
      EdgeMode mode = fused ? EdgeMode::UpdAgg : EdgeMode::Upd;
      int grid = fd.grid_upd;
      if (t == 0 && enc_in_upd) {
        ea.enc.P = enc_a.P;
        ea.enc.w2 = enc_a.w2;
        ea.enc.g1 = enc_a.g1;
        ea.enc.beta1 = enc_a.beta1;
        ea.enc.b2 = enc_a.b2;
        ea.enc.g2 = enc_a.g2;
        ea.enc.beta2 = enc_a.beta2;
        ea.enc.s1 = enc_a.s1;
        ea.enc.s2 = enc_a.s2;
        ea.we = (const float *)fd.we_em0_acc;  // e0 from the accumulators
        mode = EdgeMode::EncUpdAgg;
        grid = fd.grid_encupd;
      }
      st.begin(t == T / 2);
      HIP_TRY(launch_edge(mode, ea, grid));
      st.end(GNN_STAGE_EDGE_UPDATE);
      st.begin(t == T / 2);
      if (fused)
        HIP_TRY(launch_segsum_fused(eact, H, w.e, w.rp_in, w.q_in, w.rp_out, w.part, w.ain,
                                    w.aout, n, E, stream));
      else  // source-order rows: the out-CSR is the identity
        HIP_TRY(launch_segsum(act, H, w.e, w.rp_in, w.q_in, w.rp_out, nullptr, w.ain, w.aout,
                              n, stream));
      st.end(GNN_STAGE_AGGREGATE);
      NodeArgs nu;
      nu.n_rows = N;
      nu.src[0] = (const float *)w.h;
      nu.src[1] = (const float *)w.ain;
      nu.src[2] = (const float *)w.aout;
      nu.mlp = hd->node_mlp[k];
      nu.wstream = (const float *)fd.upd_stream[t];
      nu.nchunks = fd.upd_chunks;
      if (fd.split) {
        nu.s1 = fd.s1_nm[k];
        nu.s2 = fd.s2_nm[k];
        nu.rp_in = w.rp_in;
        nu.rp_out = w.rp_out;
        nu.row_bound = fd.row_bound;
      }
      nu.nproj = 1;
      // In place: a wave reads its rows before writing them.  The last
      // update's h reaches the classifier only through its projections, so
      // it is not stored unless the stages are being exported.
      nu.h_out = t == T - 1 && ro.stop_iter < 0 ? nullptr : (float *)w.h;
      nu.p_out[0] = w.pb;
      {
        const MlpDev *mc = nullptr;
        consumer(t, &mc, &nu.ps1[0]);
        nu.pbias[0] = mc->l0.b;
      }
      nu.eps = d.ln_eps;
      st.begin(t == T / 2);
      HIP_TRY(fd.split ? launch_node_split(false, H, nu, fd.grid_node, fd.prec, stream)
                       : launch_node_f32(false, H, nu, fd.grid_node, stream));
      st.end(GNN_STAGE_NODE_UPDATE);
    }
    if (ro.stop_iter >= 0) {
      const int64_t nh = N * H, eh = E * H;
      struct { float *dst; void *src; int64_t n; bool agg; } ex[4] = {
          {ro.h, w.h, nh, false}, {ro.e, w.e, eh, false},
          {ro.ain, w.ain, nh, true}, {ro.aout, w.aout, nh, true}};
      for (auto &x2 : ex) {
        if (!x2.dst || x2.n == 0 || (x2.agg && T == 0)) continue;
        if (x2.src == w.e)  // back to input order
          HIP_TRY(launch_scatter_rows(eact, w.e, w.perm_out, x2.dst, E, H, stream));
        else if (act == Act::F32)
          HIP_TRY(hipMemcpyAsync(x2.dst, x2.src, x2.n * 4, hipMemcpyDeviceToDevice, stream));
        else
          HIP_TRY(launch_bf16_to_f32(x2.src, x2.dst, x2.n, stream));
      }
      goto out;
    }
    {
      EdgeArgs ea = edge_args(w.pb, hd->cls);
      ea.out_idx = w.perm_out;
      ea.e_in = (const float *)w.e;
      ea.we = (const float *)fd.we_cls;
      ea.g2 = ea.beta2 = nullptr;
      ea.s1 = fd.s1_cls;
      ea.out_score = ro.scores;
      ea.out_logit = ro.logits;
      st.begin();
      HIP_TRY(launch_edge(EdgeMode::Cls, ea, fd.grid_cls));
      st.end(GNN_STAGE_CLASSIFIER);
    }
    goto out;
  }

  {
    GmlpArgs a;
    a.n_nodes = n;
    a.eps = d.ln_eps;
    // node encoder
    a.n_rows = N;
    a.x = x;
    a.F = d.in_features;
    a.mlp = hd->node_enc;
    a.out = w.h;
    st.begin();
    HIP_TRY(launch_gmlp(GmlpKind::NodeEnc, act, H, a, stream));
    st.end(GNN_STAGE_NODE_ENC);
    // edge encoder on [h_src; h_dst]
    a = GmlpArgs();
    a.n_nodes = n;
    a.eps = d.ln_eps;
    a.n_rows = E;
    a.src[0] = w.h; a.idx[0] = ei;
    a.src[1] = w.h; a.idx[1] = ei + E;
    a.mlp = hd->edge_enc;
    a.out = w.e;
    st.begin();
    HIP_TRY(launch_gmlp(GmlpKind::EdgeEnc, act, H, a, stream));
    st.end(GNN_STAGE_EDGE_ENC);

    const int T = ro.stop_iter >= 0 ? (ro.stop_iter < d.n_iters ? ro.stop_iter : d.n_iters)
                                    : d.n_iters;
    for (int t = 0; t < T; ++t) {
      const int k = d.n_mp_weight_sets == 1 ? 0 : t;
      // edge update on [h_src; h_dst; e], in place (a wave reads its own e
      // rows completely before it writes them)
      a = GmlpArgs();
      a.n_nodes = n;
      a.eps = d.ln_eps;
      a.n_rows = E;
      a.src[0] = w.h; a.idx[0] = ei;
      a.src[1] = w.h; a.idx[1] = ei + E;
      a.src[2] = w.e;
      a.mlp = hd->edge_mlp[k];
      a.out = w.e;
      st.begin(t == T / 2);
      HIP_TRY(launch_gmlp(GmlpKind::EdgeUpd, act, H, a, stream));
      st.end(GNN_STAGE_EDGE_UPDATE);
      st.begin(t == T / 2);
      HIP_TRY(launch_segsum(act, H, w.e, w.rp_in, w.perm_in, w.rp_out, w.perm_out, w.ain,
                            w.aout, n, stream));
      st.end(GNN_STAGE_AGGREGATE);
      // node update on [h; agg_in; agg_out], in place
      a = GmlpArgs();
      a.n_nodes = n;
      a.eps = d.ln_eps;
      a.n_rows = N;
      a.src[0] = w.h;
      a.src[1] = w.ain;
      a.src[2] = w.aout;
      a.mlp = hd->node_mlp[k];
      a.out = w.h;
      st.begin(t == T / 2);
      HIP_TRY(launch_gmlp(GmlpKind::NodeUpd, act, H, a, stream));
      st.end(GNN_STAGE_NODE_UPDATE);
    }

    if (ro.stop_iter >= 0) {
      const int64_t nh = N * H, eh = E * H;
      struct { float *dst; void *src; int64_t n; bool agg; } ex[4] = {
          {ro.h, w.h, nh, false}, {ro.e, w.e, eh, false},
          {ro.ain, w.ain, nh, true}, {ro.aout, w.aout, nh, true}};
      for (auto &x2 : ex) {
        if (!x2.dst || x2.n == 0 || (x2.agg && T == 0)) continue;
        if (act == Act::F32)
          HIP_TRY(hipMemcpyAsync(x2.dst, x2.src, x2.n * 4, hipMemcpyDeviceToDevice, stream));
        else
          HIP_TRY(launch_bf16_to_f32(x2.src, x2.dst, x2.n, stream));
      }
      goto out;
    }

    // classifier on [h_src; h_dst; e]
    a = GmlpArgs();
    a.n_nodes = n;
    a.eps = d.ln_eps;
    a.n_rows = E;
    a.src[0] = w.h; a.idx[0] = ei;
    a.src[1] = w.h; a.idx[1] = ei + E;
    a.src[2] = w.e;
    a.mlp = hd->cls;
    a.out_score = ro.scores;
    a.out_logit = ro.logits;
    st.begin();
    HIP_TRY(launch_gmlp(GmlpKind::Classifier, act, H, a, stream));
    st.end(GNN_STAGE_CLASSIFIER);
  }

out:
  st.finish(GNN_STAGE_TOTAL);
  if (!ro.ext_base) {
    const int rr = ws_release(hd, slot, w.base, w.bytes, stream);
    if (rc == GNN_OK) rc = rr;
  }
  return rc;
}

int common_checks(gnn_handle *h, const float *x, const int32_t *ei, int64_t N, int64_t E,
                  const void *out) {
  int rc = check_counts(h, N, E);
  if (rc) return rc;
  if (E == 0) return GNN_OK;
  if (!x || !ei || !out) return fail(GNN_E_INVALID_ARG, "NULL input or output pointer");
  return GNN_OK;
}

}  // namespace

namespace gnn {

StageEvents &stage_events() {
  static thread_local StageEvents ev;
  return ev;
}

// Detaches the handle's cached workspaces from `stream` before the caller
// destroys it: entries whose last call ran there wait for that call (already
// finished when the stream has been synchronised) and then hold no event
// recorded on it, so no later call queries or waits on an event of a
// destroyed stream.
void ws_forget_stream(gnn_handle *h, hipStream_t stream) {
  if (!h) return;
  DeviceGuard guard(h->device);
  std::lock_guard<std::mutex> lk(h->ws_mu);
  for (auto &e : h->ws) {
    if (e.busy || e.last != stream) continue;
    if (e.recorded && hipEventSynchronize(e.done) != hipSuccess) (void)hipGetLastError();
    e.recorded = false;
    e.last = nullptr;
  }
}

}  // namespace gnn

extern "C" {

size_t gnn_weight_count(const gnn_dims *dims) {
  if (check_dims(dims) != GNN_OK) return 0;
  return weight_count(dims);
}

const char *gnn_last_error(void) { return g_last_error.c_str(); }

gnn_handle *gnn_create(const float *weights, const gnn_dims *dims) {
  if (check_dims(dims) != GNN_OK) return nullptr;
  if (!weights) {
    fail(GNN_E_INVALID_ARG, "weights is NULL");
    return nullptr;
  }
  size_t ws_limit = 0;
  if (const char *lim = getenv("GNN_WORKSPACE_LIMIT")) {
    if (!parse_bytes(lim, &ws_limit)) {
      fail(GNN_E_INVALID_ARG,
           "GNN_WORKSPACE_LIMIT='%s' is not a byte count (digits, optional k/m/g suffix)", lim);
      return nullptr;
    }
  }
  int ndev = 0;
  if (hipGetDeviceCount(&ndev) != hipSuccess || ndev <= 0) {
    (void)hipGetLastError();
    fail(GNN_E_NO_DEVICE, "no HIP device visible");
    return nullptr;
  }
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) {
    fail(GNN_E_NO_DEVICE, "hipGetDevice failed");
    return nullptr;
  }
  hipDeviceProp_t prop;
  if (hipGetDeviceProperties(&prop, dev) != hipSuccess) {
    fail(GNN_E_HIP, "hipGetDeviceProperties failed");
    return nullptr;
  }
  if (strncmp(prop.gcnArchName, "gfx950", 6) != 0) {
    fail(GNN_E_UNSUPPORTED, "device %d is %s; this library is built for gfx950 only", dev,
         prop.gcnArchName);
    return nullptr;
  }
  // Keep freed stream-ordered memory in the pool instead of returning it to
  // the driver after every call.
  hipMemPool_t pool;
  if (hipDeviceGetDefaultMemPool(&pool, dev) == hipSuccess) {
    uint64_t thr = UINT64_MAX;
    (void)hipMemPoolSetAttribute(pool, hipMemPoolAttrReleaseThreshold, &thr);
  }

  const gnn_dims &d = *dims;
  const int F = d.in_features, H = d.hidden, S = d.n_mp_weight_sets;
  const bool bf16 = d.dtype == GNN_BF16;
  const bool f16w = bf16 && (d.flags & GNN_F16_WEIGHTS);
  const float *p = weights;
  auto next = [&](int fin, int fout, bool ln) {
    BlobLayer L{p, nullptr, nullptr, nullptr, fin, fout};
    p += (size_t)fin * fout;
    L.b = p;
    p += fout;
    if (ln) {
      L.g = p;
      p += fout;
      L.beta = p;
      p += fout;
    }
    return L;
  };
  Staging st;
  MlpOff o_ne, o_ee, o_cls;
  std::vector<MlpOff> o_em(S), o_nm(S);
  const bool factored = !(d.flags & GNN_LITERAL_GATHER);
  const int T = d.n_iters;
  size_t o_we_cls = 0, o_enc_stream = 0, o_w2_ee = 0, o_we_em0_acc = 0;
  std::vector<size_t> o_we_em(S), o_upd_stream(T), o_w2_em(S);
  bool split = false;
  FactDev fdh;  // scales of the split path (pointers are fixed up below)
  {
    BlobLayer a0 = next(F, H, true), a1 = next(H, H, true);
    o_ne = {stage_layer(st, a0, WKind::PlainT, bf16, true),
            stage_layer(st, a1, WKind::FragAcc, bf16, true)};
    BlobLayer b0 = next(2 * H, H, true), b1 = next(H, H, true);
    o_ee = {stage_layer(st, b0, WKind::FragMem, bf16, true),
            stage_layer(st, b1, WKind::FragAcc, bf16, true)};
    std::vector<BlobLayer> e0s, e1s, n0s, n1s;
    for (int s = 0; s < S; ++s) {
      BlobLayer e0 = next(3 * H, H, true), e1 = next(H, H, true);
      o_em[s] = {stage_layer(st, e0, WKind::FragMem, bf16, true),
                 stage_layer(st, e1, WKind::FragAcc, bf16, true)};
      BlobLayer n0 = next(3 * H, H, true), n1 = next(H, H, true);
      o_nm[s] = {stage_layer(st, n0, WKind::FragMem, bf16, true),
                 stage_layer(st, n1, WKind::FragAcc, bf16, true)};
      e0s.push_back(e0);
      e1s.push_back(e1);
      n0s.push_back(n0);
      n1s.push_back(n1);
    }
    BlobLayer c0 = next(3 * H, H, true), c1 = next(H, 1, false);
    o_cls = {stage_layer(st, c0, WKind::FragMem, bf16, true),
             stage_layer(st, c1, WKind::Plain, bf16, false)};
    // The edge consumer of the projections computed after node update t
    // (t = -1: the node encoder's second projection).
    auto next_edge_l1 = [&](int t) -> const BlobLayer & {
      return t + 1 < T ? e0s[S == 1 ? 0 : t + 1] : c0;
    };
    if (factored && !bf16) {
      // Split products need every LayerNorm output that feeds an f16x2
      // product inside the fp16 range (with a factor 2 to spare).
      double bound = 0.0;
      for (const BlobLayer *L : {&a0, &a1, &b0, &b1}) bound = fmax(bound, ln_out_bound(*L));
      for (int s = 0; s < S; ++s)
        for (const BlobLayer *L : {&e0s[s], &e1s[s], &n0s[s], &n1s[s]})
          bound = fmax(bound, ln_out_bound(*L));
      split = !(d.flags & GNN_FP32_MFMA) && bound <= 32768.0;
      fdh.row_bound = (float)bound;
    }
    if (factored && bf16) {
      // The bf16 model on the same kernels: hi/lo bf16 records (or, with
      // GNN_F16_WEIGHTS, one fp16 record part); the fp16 projections and the
      // W_e records of their consumer carry that consumer's scale (bias and
      // eps follow in the kernel).
      split = true;
      if (f16w) {
        // fp16 operands: every LayerNorm output that feeds a product must
        // lie inside the fp16 range (as for the split products), and the
        // node update scales aggregate rows by the message-row bound
        double bound = 0.0;
        for (const BlobLayer *L : {&a0, &a1, &b0, &b1}) bound = fmax(bound, ln_out_bound(*L));
        for (int s = 0; s < S; ++s)
          for (const BlobLayer *L : {&e0s[s], &e1s[s], &n0s[s], &n1s[s]})
            bound = fmax(bound, ln_out_bound(*L));
        if (!(bound <= 32768.0)) {
          fail(GNN_E_UNSUPPORTED,
               "GNN_F16_WEIGHTS: a LayerNorm output bound %g exceeds the fp16 range", bound);
          return nullptr;
        }
        fdh.row_bound = (float)bound;
      }
      double hb = ln_out_bound(a1);
      for (int s = 0; s < S; ++s) hb = fmax(hb, ln_out_bound(n1s[s]));
      fdh.s1_ee = proj_f16_scale(b0, H, hb);
      fdh.s1_cls = proj_f16_scale(c0, H, hb);
      bool fits = fdh.s1_ee > 0.f && fdh.s1_cls > 0.f;
      for (int s = 0; s < S; ++s) {
        fdh.s1_em.push_back(proj_f16_scale(e0s[s], H, hb));
        fits = fits && fdh.s1_em[s] > 0.f;
      }
      if (!fits) {
        fail(GNN_E_UNSUPPORTED,
             "bf16 model: no power-of-two scale keeps these weights' node projections inside "
             "the fp16 range");
        return nullptr;
      }
      auto add16 = [&](const std::vector<uint16_t> &v) {
        return st.add(v.data(), v.size() * sizeof(uint16_t));
      };
      auto cat = [](std::vector<uint16_t> &dst, const std::vector<uint16_t> &src) {
        dst.insert(dst.end(), src.begin(), src.end());
      };
      // Records: hi/lo bf16 pairs, or with GNN_F16_WEIGHTS one fp16 part of
      // the weights times a power of two (W2, the node MLPs and the node
      // encoder's W2 then carry pow2_scale; the projections and W_e carry
      // the fp16 projections' consumer scale either way).
      bool f16_fits = true;
      auto rec = [&](const BlobLayer &L, int c0, int K, int grp, float sc) {
        if (!f16w) return rec_bf16x2(L, c0, K, grp, sc);
        for (int f = 0; f < L.fout; ++f)
          for (int k = c0; k < c0 + K; ++k)
            if (!(fabsf(sc * L.W[(size_t)f * L.fin + k]) <= 65504.f)) f16_fits = false;
        return rec_f16x1(L, c0, K, sc, grp);
      };
      auto s2_of = [&](const BlobLayer &L) { return f16w ? pow2_scale(L) : 1.f; };
      fdh.s2_ee = s2_of(b1);
      fdh.s2_ne = s2_of(a1);
      for (int s = 0; s < S; ++s) {
        fdh.s2_em.push_back(s2_of(e1s[s]));
        fdh.s1_nm.push_back(s2_of(n0s[s]));
        fdh.s2_nm.push_back(s2_of(n1s[s]));
        o_we_em[s] = add16(rec(e0s[s], 2 * H, H, 0, fdh.s1_em[s]));
        o_w2_em[s] = add16(rec(e1s[s], 0, H, -1, fdh.s2_em[s]));
      }
      o_we_cls = add16(rec(c0, 2 * H, H, 0, fdh.s1_cls));
      o_w2_ee = add16(rec(b1, 0, H, -1, fdh.s2_ee));
      if (f16w) o_we_em0_acc = add16(rec(e0s[0], 2 * H, H, -1, fdh.s1_em[0]));
      auto scale_of = [&](const BlobLayer &L) {
        if (&L == &c0) return fdh.s1_cls;
        for (int s = 0; s < S; ++s)
          if (&L == &e0s[s]) return fdh.s1_em[s];
        return fdh.s1_ee;
      };
      auto proj = [&](std::vector<uint16_t> &dst, const BlobLayer &L) {
        const float sc = scale_of(L);
        cat(dst, rec(L, 0, H, -1, sc));
        cat(dst, rec(L, H, H, -1, sc));
      };
      std::vector<uint16_t> es = rec(a1, 0, H, -1, fdh.s2_ne);
      proj(es, b0);
      proj(es, next_edge_l1(-1));
      o_enc_stream = add16(es);
      for (int t = 0; t < T; ++t) {
        const int k = S == 1 ? 0 : t;
        std::vector<uint16_t> us = rec(n0s[k], 0, 3 * H, 4, fdh.s1_nm[k]);
        cat(us, rec(n1s[k], 0, H, -1, fdh.s2_nm[k]));
        proj(us, next_edge_l1(t));
        o_upd_stream[t] = add16(us);
      }
      if (!f16_fits) {
        fail(GNN_E_UNSUPPORTED, "GNN_F16_WEIGHTS: a scaled weight exceeds the fp16 range");
        return nullptr;
      }
    } else if (factored && split) {
      auto add16 = [&](const std::vector<uint16_t> &v) {
        return st.add(v.data(), v.size() * sizeof(uint16_t));
      };
      auto cat = [](std::vector<uint16_t> &dst, const std::vector<uint16_t> &src) {
        dst.insert(dst.end(), src.begin(), src.end());
      };
      fdh.s1_ee = pow2_scale(b0);
      fdh.s2_ee = pow2_scale(b1);
      fdh.s1_cls = pow2_scale(c0);
      fdh.s2_ne = pow2_scale(a1);
      for (int s = 0; s < S; ++s) {
        fdh.s1_em.push_back(pow2_scale(e0s[s]));
        fdh.s2_em.push_back(pow2_scale(e1s[s]));
        fdh.s1_nm.push_back(pow2_scale(n0s[s]));
        fdh.s2_nm.push_back(pow2_scale(n1s[s]));
        o_we_em[s] = add16(rec_f16x2(e0s[s], 2 * H, H, fdh.s1_em[s], 0));
        o_w2_em[s] = add16(rec_f16x2(e1s[s], 0, H, fdh.s2_em[s], -1));
      }
      o_we_cls = add16(rec_f16x2(c0, 2 * H, H, fdh.s1_cls, 0));
      o_w2_ee = add16(rec_f16x2(b1, 0, H, fdh.s2_ee, -1));
      // Projections of h (B operand from the accumulators), scaled by the
      // consumer's first-layer scale.
      auto scale_of = [&](const BlobLayer &L) {
        if (&L == &c0) return fdh.s1_cls;
        for (int s = 0; s < S; ++s)
          if (&L == &e0s[s]) return fdh.s1_em[s];
        return fdh.s1_ee;
      };
      auto proj = [&](std::vector<uint16_t> &dst, const BlobLayer &L) {
        const float sc = scale_of(L);
        cat(dst, rec_f16x2(L, 0, H, sc, -1));
        cat(dst, rec_f16x2(L, H, H, sc, -1));
      };
      std::vector<uint16_t> es = rec_f16x2(a1, 0, H, fdh.s2_ne, -1);
      proj(es, b0);
      proj(es, next_edge_l1(-1));
      o_enc_stream = add16(es);
      for (int t = 0; t < T; ++t) {
        const int k = S == 1 ? 0 : t;
        std::vector<uint16_t> us = rec_f16x2(n0s[k], 0, 3 * H, fdh.s1_nm[k], 2);
        cat(us, rec_f16x2(n1s[k], 0, H, fdh.s2_nm[k], -1));
        proj(us, next_edge_l1(t));
        o_upd_stream[t] = add16(us);
      }
    } else if (factored) {
      for (int s = 0; s < S; ++s)
        o_we_em[s] = stage_frag_f32(st, col_block(e0s[s], H, 2 * H), H, H);
      o_we_cls = stage_frag_f32(st, col_block(c0, H, 2 * H), H, H);
      // Node encoder stream: W2 | projection for the edge encoder |
      // projection for the first edge update (the classifier if T == 0).
      std::vector<float> es = frag_of(a1.W, H, H);
      append_projection(es, b0, H);
      append_projection(es, next_edge_l1(-1), H);
      o_enc_stream = st.add(es.data(), es.size() * sizeof(float));
      // Node update t: W1 | W2 | projection for edge update t+1 (or the
      // classifier after the last iteration).
      for (int t = 0; t < T; ++t) {
        const int k = S == 1 ? 0 : t;
        std::vector<float> us = frag_of(n0s[k].W, H, 3 * H);
        append(us, frag_of(n1s[k].W, H, H));
        append_projection(us, next_edge_l1(t), H);
        o_upd_stream[t] = st.add(us.data(), us.size() * sizeof(float));
      }
    }
  }

  gnn_handle *h = new gnn_handle();
  h->dims = d;
  h->ws_limit = ws_limit;
  h->device = dev;
  if (hipMalloc(&h->dev_weights, st.bytes.size()) != hipSuccess) {
    (void)hipGetLastError();
    delete h;
    fail(GNN_E_OOM, "hipMalloc of %zu weight bytes failed", st.bytes.size());
    return nullptr;
  }
  if (hipMemcpy(h->dev_weights, st.bytes.data(), st.bytes.size(), hipMemcpyHostToDevice) !=
      hipSuccess) {
    (void)hipFree(h->dev_weights);
    delete h;
    fail(GNN_E_HIP, "weight upload failed");
    return nullptr;
  }
  const unsigned char *base = (const unsigned char *)h->dev_weights;
  h->node_enc = fix_mlp(o_ne, base);
  h->edge_enc = fix_mlp(o_ee, base);
  h->cls = fix_mlp(o_cls, base);
  for (int s = 0; s < S; ++s) {
    h->edge_mlp.push_back(fix_mlp(o_em[s], base));
    h->node_mlp.push_back(fix_mlp(o_nm[s], base));
  }
  h->factored = factored;
  if (factored) {
    FactDev &fd = h->fd;
    fd = fdh;
    fd.split = split;
    fd.bf16 = bf16;
    fd.we_cls = base + o_we_cls;
    for (int s = 0; s < S; ++s) fd.we_em.push_back(base + o_we_em[s]);
    fd.enc_stream = base + o_enc_stream;
    for (int t = 0; t < T; ++t) fd.upd_stream.push_back(base + o_upd_stream[t]);
    int n_cu = 0;
    if (hipDeviceGetAttribute(&n_cu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
      n_cu = 256;
    if (split) {
      fd.w2_ee = base + o_w2_ee;
      for (int s = 0; s < S; ++s) fd.w2_em.push_back(base + o_w2_em[s]);
      fd.prec = !bf16 ? 0 : (f16w ? 2 : 1);
      fd.enc_chunks = node_split_chunks(true, H, 2, fd.prec);
      fd.upd_chunks = node_split_chunks(false, H, 1, fd.prec);
      fd.grid_enc = edge_split_grid(EdgeMode::Enc, H, fd.prec, n_cu);
      fd.grid_upd = edge_split_grid(EdgeMode::UpdAgg, H, fd.prec, n_cu);
      fd.grid_cls = edge_split_grid(EdgeMode::Cls, H, fd.prec, n_cu);
      if (f16w) {
        fd.we_em0_acc = base + o_we_em0_acc;
        fd.grid_encupd = edge_split_grid(EdgeMode::EncUpdAgg, H, fd.prec, n_cu);
      }
    } else {
      const int kg = H / 8;  // k-groups of one H-wide operand; 8 per chunk
      fd.enc_chunks = (kg + 4 * kg) / 8;
      fd.upd_chunks = (3 * kg + kg + 2 * kg) / 8;
      fd.grid_enc = edge_f32_grid(EdgeMode::Enc, H, n_cu);
      fd.grid_upd = edge_f32_grid(EdgeMode::Upd, H, n_cu);
      fd.grid_cls = edge_f32_grid(EdgeMode::Cls, H, n_cu);
    }
    fd.grid_node = node_f32_grid(n_cu);
  }
  return h;
}

int64_t gnn_release_workspaces(gnn_handle *h) {
  if (!h) return fail(GNN_E_INVALID_ARG, "handle is NULL");
  DeviceGuard guard(h->device);
  std::lock_guard<std::mutex> lk(h->ws_mu);
  int64_t freed = 0;
  for (auto &e : h->ws) {
    if (e.busy || !e.base) continue;
    if ((e.recorded && hipEventSynchronize(e.done) != hipSuccess) ||
        hipFree(e.base) != hipSuccess) {
      (void)hipGetLastError();
      return fail(GNN_E_HIP, "releasing a cached workspace failed");
    }
    freed += (int64_t)e.bytes;
    h->ws_held -= e.bytes;
    e.base = nullptr;
    e.bytes = 0;
    e.recorded = false;
  }
  return freed;
}

int gnn_set_workspace_limit(gnn_handle *h, int64_t bytes) {
  if (!h) return fail(GNN_E_INVALID_ARG, "handle is NULL");
  if (bytes < 0) return fail(GNN_E_INVALID_ARG, "negative workspace limit %lld", (long long)bytes);
  std::lock_guard<std::mutex> lk(h->ws_mu);
  h->ws_limit = (size_t)bytes;
  return GNN_OK;
}

void gnn_destroy(gnn_handle *h) {
  if (!h) return;
  {
    DeviceGuard guard(h->device);
    (void)hipDeviceSynchronize();
    (void)hipFree(h->dev_weights);
    for (auto &mk : h->prof_pending) {
      if (mk.own_a) (void)hipEventDestroy(mk.a);
      if (mk.own_b) (void)hipEventDestroy(mk.b);
    }
    for (auto e : h->prof_free) (void)hipEventDestroy(e);
    for (auto &e : h->ws) {
      if (e.base) (void)hipFree(e.base);
      (void)hipEventDestroy(e.done);
    }
  }
  delete h;
}

int gnn_profile_enable(gnn_handle *h, int enable) {
  if (!h) return fail(GNN_E_INVALID_ARG, "handle is NULL");
  gnn_profile_stats scratch;
  scratch.struct_size = sizeof scratch;
  int rc = gnn_profile_read(h, &scratch);  // drains pending events
  if (rc) return rc;
  if (enable < 0 || enable > GNN_PROFILE_SAMPLE)
    return fail(GNN_E_INVALID_ARG, "profiling mode %d is not 0, 1 or GNN_PROFILE_SAMPLE", enable);
  std::lock_guard<std::mutex> lk(h->prof_mu);
  h->prof_on = enable != 0;
  h->prof_sample = enable == GNN_PROFILE_SAMPLE;
  h->prof_calls = 0;
  // events for about 64 calls (two per timed stage), so that none is
  // created while timing
  if (h->prof_on) {
    DeviceGuard guard(h->device);
    while (h->prof_free.size() < 4096) {
      hipEvent_t e = nullptr;
      if (hipEventCreate(&e) != hipSuccess) break;
      h->prof_free.push_back(e);
    }
  }
  for (int i = 0; i < GNN_N_STAGES; ++i) {
    h->prof_launches[i] = 0;
    h->prof_ms[i] = 0.0;
  }
  return GNN_OK;
}

int gnn_profile_read(gnn_handle *h, gnn_profile_stats *out) {
  if (!h || !out) return fail(GNN_E_INVALID_ARG, "NULL argument");
  if (out->struct_size != sizeof(gnn_profile_stats))
    return fail(GNN_E_INVALID_ARG, "gnn_profile_stats.struct_size mismatch");
  DeviceGuard guard(h->device);
  std::vector<gnn_handle::Mark> marks;
  {
    std::lock_guard<std::mutex> lk(h->prof_mu);
    marks.swap(h->prof_pending);
  }
  int rc = GNN_OK;
  std::vector<double> add(GNN_N_STAGES, 0.0);
  std::vector<int64_t> cnt(GNN_N_STAGES, 0);
  for (auto &mk : marks) {
    float ms = 0.f;
    if (hipEventSynchronize(mk.b) != hipSuccess ||
        hipEventElapsedTime(&ms, mk.a, mk.b) != hipSuccess) {
      rc = fail(GNN_E_HIP, "profiling event query failed");
      continue;
    }
    add[mk.stage] += ms;
    cnt[mk.stage] += 1;
  }
  std::lock_guard<std::mutex> lk(h->prof_mu);
  for (auto &mk : marks) {
    if (mk.own_a) h->prof_free.push_back(mk.a);
    if (mk.own_b) h->prof_free.push_back(mk.b);
  }
  for (int i = 0; i < GNN_N_STAGES; ++i) {
    h->prof_ms[i] += add[i];
    h->prof_launches[i] += cnt[i];
    out->ms[i] = h->prof_ms[i];
    out->launches[i] = h->prof_launches[i];
  }
  out->n_calls = h->prof_calls;
  return rc;
}

int gnn_infer(gnn_handle *h, const float *node_feat, const int32_t *edge_index, int64_t n_nodes,
              int64_t n_edges, float *edge_scores, hipStream_t stream) {
  int rc = common_checks(h, node_feat, edge_index, n_nodes, n_edges, edge_scores);
  if (rc || n_edges == 0) return rc;
  RunOut ro;
  ro.scores = edge_scores;
  return run(h, node_feat, edge_index, n_nodes, n_edges, stream, ro);
}

int gnn_infer_noalloc(gnn_handle *h, const float *node_feat, const int32_t *edge_index,
                      int64_t n_nodes, int64_t n_edges, float *edge_scores, hipStream_t stream) {
  int rc = common_checks(h, node_feat, edge_index, n_nodes, n_edges, edge_scores);
  if (rc || n_edges == 0) return rc;
  RunOut ro;
  ro.scores = edge_scores;
  {
    DeviceGuard guard(h->device);
    rc = noalloc_scratch(h->device, &ro.ext_base, &ro.ext_bytes);
  }
  if (rc) return rc;
  return run(h, node_feat, edge_index, n_nodes, n_edges, stream, ro);
}

int gnn_infer_logits(gnn_handle *h, const float *node_feat, const int32_t *edge_index,
                     int64_t n_nodes, int64_t n_edges, float *edge_logits, hipStream_t stream) {
  int rc = common_checks(h, node_feat, edge_index, n_nodes, n_edges, edge_logits);
  if (rc || n_edges == 0) return rc;
  RunOut ro;
  ro.logits = edge_logits;
  return run(h, node_feat, edge_index, n_nodes, n_edges, stream, ro);
}

struct gnn_filter {
  gnn_filter_dims dims;
  int device = 0;
  void *dev = nullptr;
  FilterArgs tmpl;  // weight pointers
};

namespace {
int check_filter_dims(const gnn_filter_dims *d) {
  if (!d) return fail(GNN_E_INVALID_ARG, "dims is NULL");
  if (d->struct_size != sizeof(gnn_filter_dims))
    return fail(GNN_E_INVALID_ARG, "gnn_filter_dims.struct_size mismatch");
  if (d->in_features < 1 || d->in_features > 16)
    return fail(GNN_E_INVALID_ARG, "in_features %d outside 1..16", d->in_features);
  if (d->hidden != 64 && d->hidden != 128)
    return fail(d->hidden > 0 && d->hidden % 32 == 0 ? GNN_E_UNSUPPORTED : GNN_E_INVALID_ARG,
                "hidden %d not supported (64 or 128)", d->hidden);
  if (!(d->ln_eps > 0.f) || !(d->ln_eps < 1.f))
    return fail(GNN_E_INVALID_ARG, "ln_eps outside (0, 1)");
  return GNN_OK;
}
}  // namespace

size_t gnn_filter_weight_count(const gnn_filter_dims *d) {
  if (check_filter_dims(d)) return 0;
  const size_t F = d->in_features, H = d->hidden;
  return layer_floats(2 * F, H, true) + layer_floats(H, H, true) + layer_floats(H, 1, false);
}

gnn_filter *gnn_filter_create(const float *weights, const gnn_filter_dims *dims) {
  if (check_filter_dims(dims)) return nullptr;
  if (!weights) {
    fail(GNN_E_INVALID_ARG, "weights is NULL");
    return nullptr;
  }
  int ndev = 0, dev = 0;
  if (hipGetDeviceCount(&ndev) != hipSuccess || ndev <= 0 || hipGetDevice(&dev) != hipSuccess) {
    (void)hipGetLastError();
    fail(GNN_E_NO_DEVICE, "no HIP device visible");
    return nullptr;
  }
  const int F = dims->in_features, H = dims->hidden;
  const float *p = weights;
  auto next = [&](int fin, int fout, bool ln) {
    BlobLayer L{p, nullptr, nullptr, nullptr, fin, fout};
    p += (size_t)fin * fout;
    L.b = p;
    p += fout;
    if (ln) {
      L.g = p;
      p += fout;
      L.beta = p;
      p += fout;
    }
    return L;
  };
  BlobLayer l0 = next(2 * F, H, true), l1 = next(H, H, true), l2 = next(H, 1, false);
  Staging st;
  LayerOff o0 = stage_layer(st, l0, WKind::PlainT, false, true);
  LayerOff o1 = stage_layer(st, l1, WKind::FragAcc, false, true);
  LayerOff o2 = stage_layer(st, l2, WKind::Plain, false, false);
  // Layer 2 on the fp16 matrix cores from split operands when its input, a
  // LayerNorm/ReLU output, stays inside half the fp16 range (else fp32).
  const bool split = ln_out_bound(l0) <= 32768.0;
  const float s1 = split ? pow2_scale(l1) : 1.f;
  size_t o_w1r = 0;
  if (split) {
    const std::vector<uint16_t> r = rec_f16x2(l1, 0, H, s1, -1);
    o_w1r = st.add(r.data(), r.size() * sizeof(uint16_t));
  }
  gnn_filter *f = new gnn_filter();
  f->dims = *dims;
  f->device = dev;
  if (hipMalloc(&f->dev, st.bytes.size()) != hipSuccess ||
      hipMemcpy(f->dev, st.bytes.data(), st.bytes.size(), hipMemcpyHostToDevice) != hipSuccess) {
    (void)hipGetLastError();
    if (f->dev) (void)hipFree(f->dev);
    delete f;
    fail(GNN_E_OOM, "filter weight upload failed");
    return nullptr;
  }
  const unsigned char *base = (const unsigned char *)f->dev;
  LayerDev d0 = fix_layer(o0, base), d1 = fix_layer(o1, base), d2 = fix_layer(o2, base);
  f->tmpl.F = F;
  f->tmpl.eps = dims->ln_eps;
  f->tmpl.w0t = (const float *)d0.w;
  f->tmpl.b0 = d0.b;
  f->tmpl.g0 = d0.g;
  f->tmpl.beta0 = d0.beta;
  f->tmpl.w1 = (const float *)d1.w;
  f->tmpl.b1 = d1.b;
  f->tmpl.g1 = d1.g;
  f->tmpl.beta1 = d1.beta;
  f->tmpl.w2 = (const float *)d2.w;
  f->tmpl.b2 = d2.b;
  if (split) {
    f->tmpl.w1r = base + o_w1r;
    f->tmpl.s1 = s1;
  }
  return f;
}

void gnn_filter_destroy(gnn_filter *f) {
  if (!f) return;
  {
    DeviceGuard guard(f->device);
    (void)hipDeviceSynchronize();
    (void)hipFree(f->dev);
  }
  delete f;
}

// ------------------------------------------------------ embedding MLP ---

struct gnn_embedder {
  gnn_embed_dims dims;
  int device = 0;
  void *dev = nullptr;
  EmbedArgs tmpl;  // weight pointers
};

namespace {
int check_embed_dims(const gnn_embed_dims *d) {
  if (!d) return fail(GNN_E_INVALID_ARG, "dims is NULL");
  if (d->struct_size != sizeof(gnn_embed_dims))
    return fail(GNN_E_INVALID_ARG, "gnn_embed_dims.struct_size mismatch");
  if (d->in_features < 1 || d->in_features > 16)
    return fail(GNN_E_INVALID_ARG, "in_features %d outside 1..16", d->in_features);
  if (d->hidden != 64 && d->hidden != 128)
    return fail(d->hidden > 0 && d->hidden % 32 == 0 ? GNN_E_UNSUPPORTED : GNN_E_INVALID_ARG,
                "hidden %d not supported (64 or 128)", d->hidden);
  if (d->out_dim < 1 || d->out_dim > 16)
    return fail(GNN_E_INVALID_ARG, "out_dim %d outside 1..16", d->out_dim);
  if (!(d->ln_eps > 0.f) || !(d->ln_eps < 1.f))
    return fail(GNN_E_INVALID_ARG, "ln_eps outside (0, 1)");
  return GNN_OK;
}
}  // namespace

size_t gnn_embed_weight_count(const gnn_embed_dims *d) {
  if (check_embed_dims(d)) return 0;
  const size_t F = d->in_features, H = d->hidden, D = d->out_dim;
  return layer_floats(F, H, true) + layer_floats(H, H, true) + layer_floats(H, D, false);
}

gnn_embedder *gnn_embed_create(const float *weights, const gnn_embed_dims *dims) {
  if (check_embed_dims(dims)) return nullptr;
  if (!weights) {
    fail(GNN_E_INVALID_ARG, "weights is NULL");
    return nullptr;
  }
  int ndev = 0, dev = 0;
  if (hipGetDeviceCount(&ndev) != hipSuccess || ndev <= 0 || hipGetDevice(&dev) != hipSuccess) {
    (void)hipGetLastError();
    fail(GNN_E_NO_DEVICE, "no HIP device visible");
    return nullptr;
  }
  const int F = dims->in_features, H = dims->hidden, D = dims->out_dim;
  const float *p = weights;
  auto next = [&](int fin, int fout, bool ln) {
    BlobLayer L{p, nullptr, nullptr, nullptr, fin, fout};
    p += (size_t)fin * fout;
    L.b = p;
    p += fout;
    if (ln) {
      L.g = p;
      p += fout;
      L.beta = p;
      p += fout;
    }
    return L;
  };
  BlobLayer l0 = next(F, H, true), l1 = next(H, H, true), l2 = next(H, D, false);
  Staging st;
  LayerOff o0 = stage_layer(st, l0, WKind::PlainT, false, true);
  LayerOff o1 = stage_layer(st, l1, WKind::FragAcc, false, true);
  LayerOff o2 = stage_layer(st, l2, WKind::Plain, false, false);
  // layer 2 on split fp16 products unless its input leaves the fp16 range
  const bool split = ln_out_bound(l0) <= 32768.0;
  const float s1 = split ? pow2_scale(l1) : 1.f;
  size_t o_w1r = 0;
  if (split) {
    const std::vector<uint16_t> r = rec_f16x2(l1, 0, H, s1, -1);
    o_w1r = st.add(r.data(), r.size() * sizeof(uint16_t));
  }
  gnn_embedder *m = new gnn_embedder();
  m->dims = *dims;
  m->device = dev;
  if (hipMalloc(&m->dev, st.bytes.size()) != hipSuccess ||
      hipMemcpy(m->dev, st.bytes.data(), st.bytes.size(), hipMemcpyHostToDevice) != hipSuccess) {
    (void)hipGetLastError();
    if (m->dev) (void)hipFree(m->dev);
    delete m;
    fail(GNN_E_OOM, "embedding weight upload failed");
    return nullptr;
  }
  const unsigned char *base = (const unsigned char *)m->dev;
  LayerDev d0 = fix_layer(o0, base), d1 = fix_layer(o1, base), d2 = fix_layer(o2, base);
  m->tmpl.F = F;
  m->tmpl.D = D;
  m->tmpl.eps = dims->ln_eps;
  m->tmpl.w0t = (const float *)d0.w;
  m->tmpl.b0 = d0.b;
  m->tmpl.g0 = d0.g;
  m->tmpl.beta0 = d0.beta;
  m->tmpl.w1 = (const float *)d1.w;
  m->tmpl.b1 = d1.b;
  m->tmpl.g1 = d1.g;
  m->tmpl.beta1 = d1.beta;
  if (split) {
    m->tmpl.w1r = base + o_w1r;
    m->tmpl.s1 = s1;
  }
  m->tmpl.w2 = (const float *)d2.w;
  m->tmpl.b2 = d2.b;
  return m;
}

int gnn_embed_apply(gnn_embedder *m, const float *node_feat, int64_t n_nodes, float *z,
                    hipStream_t stream) {
  if (!m) return fail(GNN_E_INVALID_ARG, "embedder is NULL");
  if (n_nodes < 0 || n_nodes > INT32_MAX)
    return fail(GNN_E_INVALID_ARG, "n_nodes outside 0..INT32_MAX");
  if (n_nodes == 0) return GNN_OK;
  if (!node_feat || !z) return fail(GNN_E_INVALID_ARG, "NULL input or output pointer");
  DeviceGuard guard(m->device);
  EmbedArgs a = m->tmpl;
  a.n = n_nodes;
  a.x = node_feat;
  a.z = z;
  const hipError_t e = launch_embed(m->dims.hidden, a, stream);
  if (e != hipSuccess) return fail(GNN_E_HIP, "embedding launch failed: %s", hipGetErrorString(e));
  return GNN_OK;
}

void gnn_embed_destroy(gnn_embedder *m) {
  if (!m) return;
  {
    DeviceGuard guard(m->device);
    (void)hipDeviceSynchronize();
    (void)hipFree(m->dev);
  }
  delete m;
}

int gnn_filter_apply(gnn_filter *f, const float *node_feat, const int32_t *edge_index,
                     int64_t n_nodes, int64_t n_edges, float threshold, float *edge_scores,
                     int32_t *edge_index_out, int64_t *n_kept, hipStream_t stream) {
  if (!f) return fail(GNN_E_INVALID_ARG, "filter is NULL");
  if (n_nodes < 0 || n_edges < 0 || n_nodes > INT32_MAX || n_edges > INT32_MAX)
    return fail(GNN_E_INVALID_ARG, "bad count");
  if (n_edges > 0 && n_nodes == 0) return fail(GNN_E_INVALID_ARG, "n_edges > 0 with n_nodes == 0");
  if (!n_kept) return fail(GNN_E_INVALID_ARG, "n_kept is NULL");
  *n_kept = 0;
  if (n_edges == 0) return GNN_OK;
  if (!node_feat || !edge_index || !edge_index_out)
    return fail(GNN_E_INVALID_ARG, "NULL input or output pointer");
  DeviceGuard guard(f->device);
  const size_t nt = compact_tiles(n_edges);
  const size_t sc_bytes = edge_scores ? 0 : align256((size_t)n_edges * 4);
  const size_t bytes = sc_bytes + align256((nt + 1) * 4) + 256;
  int rc = GNN_OK;
  unsigned char *ws = nullptr;
  {
    hipError_t ae = hipMallocAsync((void **)&ws, bytes, stream);
    if (ae != hipSuccess) {
      (void)hipGetLastError();
      return fail(GNN_E_OOM, "hipMallocAsync failed: %s", hipGetErrorString(ae));
    }
  }
  float *scores = edge_scores ? edge_scores : (float *)ws;
  int32_t *counts = (int32_t *)(ws + sc_bytes);
  int32_t *total = counts + nt;
  int32_t host_total = 0;
  FilterArgs a = f->tmpl;
  a.n_edges = n_edges;
  a.n_nodes = (int32_t)n_nodes;
  a.x = node_feat;
  a.edge_index = edge_index;
  a.scores = scores;
  HIP_TRY(launch_filter_scores(f->dims.hidden, a, stream));
  HIP_TRY(launch_compact(scores, edge_index, n_edges, threshold, counts, total, edge_index_out,
                         stream));
  HIP_TRY(hipMemcpyAsync(&host_total, total, 4, hipMemcpyDeviceToHost, stream));
  HIP_TRY(hipStreamSynchronize(stream));
  *n_kept = host_total;
out:
  {
    hipError_t fe = hipFreeAsync(ws, stream);
    if (fe != hipSuccess && rc == GNN_OK)
      rc = fail(GNN_E_HIP, "hipFreeAsync failed: %s", hipGetErrorString(fe));
  }
  return rc;
}

int gnn_wcc(const int32_t *edge_index, const float *edge_scores, float threshold,
            int64_t n_nodes, int64_t n_edges, int32_t *labels, hipStream_t stream) {
  if (n_nodes < 0 || n_edges < 0) return fail(GNN_E_INVALID_ARG, "negative count");
  if (n_nodes > INT32_MAX || n_edges > INT32_MAX)
    return fail(GNN_E_INVALID_ARG, "count above INT32_MAX");
  if (n_edges > 0 && n_nodes == 0) return fail(GNN_E_INVALID_ARG, "n_edges > 0 with n_nodes == 0");
  if (n_nodes == 0) return GNN_OK;
  if (!labels || (n_edges > 0 && !edge_index))
    return fail(GNN_E_INVALID_ARG, "NULL labels or edge_index");
  const int32_t n = (int32_t)n_nodes;
  // Hooking onto the smaller root plus full compression converges in a few
  // rounds on graphs of tracks (and in O(log n) on typical graphs); a call
  // that has not converged after max_rounds fails instead of returning
  // partial labels.  Rounds are queued GROUP at a time, each with its own
  // flag (zeroed up front); a round after one that joined nothing returns at
  // once, so the host reads one flag per group instead of one per round.
  const int max_rounds = 256, GROUP = 4;
  int rc = GNN_OK;
  bool converged = n_edges == 0;
  int32_t *changed = nullptr;
  {
    hipError_t ae = hipMallocAsync((void **)&changed, max_rounds * sizeof(int32_t), stream);
    if (ae != hipSuccess) {
      (void)hipGetLastError();
      return fail(GNN_E_OOM, "hipMallocAsync failed: %s", hipGetErrorString(ae));
    }
  }
  HIP_TRY(wcc_launch_init(labels, n, stream));
  HIP_TRY(launch_fill_i32(changed, max_rounds, 0, stream));
  for (int r0 = 0; r0 < max_rounds && n_edges > 0; r0 += GROUP) {
    const int r1 = r0 + GROUP < max_rounds ? r0 + GROUP : max_rounds;
    for (int r = r0; r < r1; ++r)
      HIP_TRY(wcc_launch_round(edge_index, edge_scores, threshold, n_edges, n, labels,
                               r > 0 ? changed + r - 1 : nullptr, changed + r, stream));
    int32_t host_changed = 0;
    HIP_TRY(hipMemcpyAsync(&host_changed, changed + r1 - 1, sizeof(int32_t),
                           hipMemcpyDeviceToHost, stream));
    HIP_TRY(hipStreamSynchronize(stream));
    if (!host_changed) {
      converged = true;
      break;
    }
  }
  if (!converged) rc = fail(GNN_E_UNSUPPORTED, "components did not converge in %d rounds",
                            max_rounds);
out:
  {
    hipError_t fe = hipFreeAsync(changed, stream);
    if (fe != hipSuccess && rc == GNN_OK)
      rc = fail(GNN_E_HIP, "hipFreeAsync failed: %s", hipGetErrorString(fe));
  }
  return rc;
}

int gnn_infer_labels(gnn_handle *h, const float *node_feat, const int32_t *edge_index,
                     int64_t n_nodes, int64_t n_edges, float threshold, float *edge_scores,
                     int32_t *labels, hipStream_t stream) {
  int rc = check_counts(h, n_nodes, n_edges);
  if (rc) return rc;
  if (n_nodes > 0 && !labels) return fail(GNN_E_INVALID_ARG, "labels is NULL");
  float *scores = edge_scores;
  if (n_edges > 0 && !scores) {
    hipError_t ae = hipMallocAsync((void **)&scores, (size_t)n_edges * sizeof(float), stream);
    if (ae != hipSuccess) {
      (void)hipGetLastError();
      return fail(GNN_E_OOM, "hipMallocAsync failed: %s", hipGetErrorString(ae));
    }
  }
  rc = gnn_infer(h, node_feat, edge_index, n_nodes, n_edges, scores, stream);
  if (rc == GNN_OK) rc = gnn_wcc(edge_index, scores, threshold, n_nodes, n_edges, labels, stream);
  if (scores != edge_scores) (void)hipFreeAsync(scores, stream);
  return rc;
}

int gnn_debug_csr(gnn_handle *h, const int32_t *edge_index, int64_t n_nodes, int64_t n_edges,
                  int32_t *row_ptr_in, int32_t *perm_in, int32_t *row_ptr_out, int32_t *perm_out,
                  hipStream_t stream) {
  int rc = check_counts(h, n_nodes, n_edges);
  if (rc) return rc;
  if (n_edges == 0) return GNN_OK;
  if (!edge_index) return fail(GNN_E_INVALID_ARG, "edge_index is NULL");
  RunOut ro;
  ro.csr_only = true;
  ro.rp_in = row_ptr_in;
  ro.perm_in = perm_in;
  ro.rp_out = row_ptr_out;
  ro.perm_out = perm_out;
  return run(h, nullptr, edge_index, n_nodes, n_edges, stream, ro);
}

int gnn_debug_stages(gnn_handle *h, const float *node_feat, const int32_t *edge_index,
                     int64_t n_nodes, int64_t n_edges, int32_t stop_iter, float *h_out,
                     float *e_out, float *agg_in_out, float *agg_out_out, hipStream_t stream) {
  int rc = check_counts(h, n_nodes, n_edges);
  if (rc) return rc;
  if (n_edges == 0) return GNN_OK;
  if (!node_feat || !edge_index) return fail(GNN_E_INVALID_ARG, "NULL input pointer");
  if (stop_iter < 0) return fail(GNN_E_INVALID_ARG, "stop_iter < 0");
  RunOut ro;
  ro.stop_iter = stop_iter;
  ro.h = h_out;
  ro.e = e_out;
  ro.ain = agg_in_out;
  ro.aout = agg_out_out;
  return run(h, node_feat, edge_index, n_nodes, n_edges, stream, ro);
}

}  // extern "C"
