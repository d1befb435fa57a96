// One training step of the 3-layer GraphSAGE model the paper evaluates
// (Section 8.1, Table 2: LayerNorm before each layer, mean aggregation), with
// optional masked label propagation (Section 6.1 step 1, Lemma 2), built from
// the library's kernels, ordered on the caller's stream without host
// synchronization (the weight gradients run on the side stream, forked from
// and joined back to it).
//
// Layer l reads H (n x f), and writes the row-major concatenation
//   C = [ LayerNorm(H) | D^-1 A LayerNorm(H) | 1 | 0 0 0 ]
// so that the layer's UPDATE
//   O = Y W_self + Z W_neigh + b
// is one MFMA product C Wp with the packed weights Wp = [W_self; W_neigh; b; 0].
// The aggregation writes straight into the middle block through its row
// stride; the ones column carries the bias, and the weight gradient of the
// same product yields dW_self, dW_neigh and db together. Column layout of a
// row: Y in [0, f), Z in [zo, zo + f), the ones column at oc, zero padding up
// to K (the GEMMs' inner size); rows are ldc >= K floats apart. Wide layers
// (f >= 128) start Z on a 128-byte boundary and every row is a multiple of
// 128 bytes, so the gathered rows of the aggregations touch no extra cache
// line (a 516-float stride costs 28% at f = 256).
//
// A layer whose output is narrower than its input (the class layer, fo < f)
// aggregates the narrower operand instead: since D^-1 A Y W_neigh =
// D^-1 A (Y W_neigh), it computes T = Y W_neigh, writes M = D^-1 A T into the
// middle block (fo wide) and packs [W_self; I; b; 0], so the same product
// adds M. Its backward aggregates the fo-wide gradient: G = (D^-1 A)^T dO,
// dY = [dO | G] [W_self | W_neigh]^T in one product, and the weight gradients
// come from Y^T [dO | G].

#include "common.h"

namespace gcn {
namespace {

constexpr int kThreadsS = 256;

inline int64_t round4(int64_t v) { return (v + 3) & ~int64_t(3); }

// Columns of C below K that no kernel of the layer writes: [f, zo),
// [zo + zw, oc) (zw: the width of the middle block's data), the ones column
// oc and (oc, K).
__global__ __launch_bounds__(kThreadsS) void k_concat_tail(int64_t n, int64_t f, int64_t zo,
                                                           int64_t zw, int64_t oc, int64_t K,
                                                           float* __restrict__ c, int64_t ldc) {
  const int64_t a = zo - f, b = oc - zo - zw;  // the two padding runs
  const int64_t per_row = K - f - zw;
  const int64_t t = (int64_t)blockIdx.x * kThreadsS + threadIdx.x;
  if (t >= n * per_row) return;
  const int64_t i = t / per_row, k = t % per_row;
  int64_t col;
  if (k < a)
    col = f + k;
  else if (k < a + b)
    col = zo + zw + (k - a);
  else
    col = oc + (k - a - b);
  c[i * ldc + col] = (col == oc) ? 1.f : 0.f;
}

// Wp [K x fop]: rows [0, f) = W_self, [zo, zo + f) = W_neigh (or, when the
// layer aggregates Y W_neigh, [zo, zo + fo) = the identity), row oc = b,
// every other entry 0 (fo columns used of fop).
__global__ __launch_bounds__(kThreadsS) void k_pack_weights(int64_t f, int64_t zo, int64_t oc,
                                                            int64_t K, int64_t fo, int64_t fop,
                                                            bool ident,
                                                            const float* __restrict__ ws,
                                                            const float* __restrict__ wn,
                                                            const float* __restrict__ b,
                                                            float* __restrict__ wp) {
  const int64_t t = (int64_t)blockIdx.x * kThreadsS + threadIdx.x;
  if (t >= K * fop) return;
  const int64_t r = t / fop, c = t % fop;
  float v = 0.f;
  if (c < fo) {
    if (r < f)
      v = ws[r * fo + c];
    else if (ident && r >= zo && r < zo + fo)
      v = r - zo == c ? 1.f : 0.f;
    else if (!ident && r >= zo && r < zo + f)
      v = wn[(r - zo) * fo + c];
    else if (r == oc)
      v = b[c];
  }
  wp[t] = v;
}

// dst [rows x ldd] = src [rows x cols] (ld lds) in the first cols columns,
// 0 in the columns [cols, ldd).
__global__ __launch_bounds__(kThreadsS) void k_pad_cols(int64_t rows, int64_t cols,
                                                        const float* __restrict__ src, int64_t lds,
                                                        float* __restrict__ dst, int64_t ldd) {
  const int64_t t = (int64_t)blockIdx.x * kThreadsS + threadIdx.x;
  if (t >= rows * ldd) return;
  const int64_t r = t / ldd, c = t % ldd;
  dst[t] = c < cols ? src[r * lds + c] : 0.f;
}

// B [f x 2 fop] = [W_self | 0 | W_neigh | 0] (the weights of the input
// gradient of a layer that aggregates Y W_neigh: dY = [dO | G] B^T).
__global__ __launch_bounds__(kThreadsS) void k_pack_bcat(int64_t f, int64_t fo, int64_t fop,
                                                         const float* __restrict__ ws,
                                                         const float* __restrict__ wn,
                                                         float* __restrict__ bc) {
  const int64_t t = (int64_t)blockIdx.x * kThreadsS + threadIdx.x;
  if (t >= f * 2 * fop) return;
  const int64_t r = t / (2 * fop), c = t % (2 * fop);
  float v = 0.f;
  if (c < fo)
    v = ws[r * fo + c];
  else if (c >= fop && c < fop + fo)
    v = wn[r * fo + c - fop];
  bc[t] = v;
}

// Zero the padding columns [fo, fop) and [fop + fo, 2 fop) of DG [n x 2 fop]
// (the blocks dO and G of the input-gradient product's left operand).
__global__ __launch_bounds__(kThreadsS) void k_zero_dg_pad(int64_t n, int64_t fo, int64_t fop,
                                                           float* __restrict__ dg) {
  const int64_t pad = fop - fo;
  const int64_t t = (int64_t)blockIdx.x * kThreadsS + threadIdx.x;
  if (t >= n * 2 * pad) return;
  const int64_t i = t / (2 * pad), k = t % (2 * pad);
  const int64_t col = k < pad ? fo + k : fop + fo + (k - pad);
  dg[i * 2 * fop + col] = 0.f;
}

// [dO | G] before the transposed aggregation writes G: row i of dg (2 fop
// wide) gets dO's fo columns and zeros up to fop, and the piece of the G half
// that holds its last columns and padding is zeroed (the aggregation then
// writes the fo columns of G). Thread t takes 16-byte piece t % q of row
// t / q, q = fop / 4 + (fo % 4 != 0); dO rows 16-byte aligned, ldo >= fop.
__global__ __launch_bounds__(kThreadsS) void k_fill_dg(int64_t n, int64_t fo, int64_t fop,
                                                       const float* __restrict__ d_o,
                                                       int64_t ldo, float* __restrict__ dg) {
  const int64_t q = fop / 4 + (fo % 4 != 0 ? 1 : 0);
  const int64_t t = (int64_t)blockIdx.x * kThreadsS + threadIdx.x;
  if (t >= n * q) return;
  const int64_t i = t / q, p = t % q;
  float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
  int64_t col = fop + 4 * (fo / 4);  // the extra piece: the G half's last one
  if (p < fop / 4) {
    col = 4 * p;
    v = *reinterpret_cast<const float4*>(d_o + i * ldo + col);
    if (col + 0 >= fo) v.x = 0.f;
    if (col + 1 >= fo) v.y = 0.f;
    if (col + 2 >= fo) v.z = 0.f;
    if (col + 3 >= fo) v.w = 0.f;
  }
  *reinterpret_cast<float4*>(dg + i * 2 * fop + col) = v;
}

// dwp [f x 2 fop] = Y^T [dO | G] -> dW_self, dW_neigh (the bias comes from
// the column sum of dO).
__global__ __launch_bounds__(kThreadsS) void k_unpack_grads_tf(int64_t f, int64_t fo,
                                                               int64_t fop,
                                                               const float* __restrict__ dwp,
                                                               float* __restrict__ dws,
                                                               float* __restrict__ dwn) {
  const int64_t t = (int64_t)blockIdx.x * kThreadsS + threadIdx.x;
  if (t >= 2 * f * fo) return;
  const int64_t r = t / fo, c = t % fo;
  if (r < f)
    dws[r * fo + c] = dwp[r * 2 * fop + c];
  else
    dwn[(r - f) * fo + c] = dwp[(r - f) * 2 * fop + fop + c];
}

// The inverse of k_pack_weights for the gradient.
__global__ __launch_bounds__(kThreadsS) void k_unpack_grads(int64_t f, int64_t zo, int64_t oc,
                                                            int64_t fo, int64_t fop,
                                                            const float* __restrict__ dwp,
                                                            float* __restrict__ dws,
                                                            float* __restrict__ dwn,
                                                            float* __restrict__ db) {
  const int64_t t = (int64_t)blockIdx.x * kThreadsS + threadIdx.x;
  if (t >= (2 * f + 1) * fo) return;
  const int64_t r = t / fo, c = t % fo;
  if (r < f)
    dws[r * fo + c] = dwp[r * fop + c];
  else if (r < 2 * f)
    dwn[(r - f) * fo + c] = dwp[(zo + r - f) * fop + c];
  else
    db[c] = dwp[oc * fop + c];
}

// Masked label propagation, forward: Xp = X + E[y] on rows with mask = 1.
// One row per wavefront, the lanes striding over its features.
__global__ __launch_bounds__(kThreadsS) void k_embed_labels(int64_t n, int64_t f, int C,
                                                            const float* __restrict__ x,
                                                            int64_t ldx,
                                                            const uint8_t* __restrict__ mask,
                                                            const int32_t* __restrict__ y,
                                                            const float* __restrict__ e,
                                                            float* __restrict__ xp, int64_t ldp) {
  const int64_t i = (int64_t)blockIdx.x * (kThreadsS / 64) + (threadIdx.x >> 6);
  if (i >= n) return;
  const int lane = threadIdx.x & 63;
  const int32_t k = y[i];
  const bool on = mask[i] && k >= 0 && k < C;
  for (int64_t c = lane; c < f; c += 64) {
    float v = x[i * ldx + c];
    if (on) v += e[(int64_t)k * f + c];
    xp[i * ldp + c] = v;
  }
}

// The same with 16-byte pieces (f, ldx, ldp multiples of 4, aligned rows):
// thread t takes piece t % q of row t / q (q = f / 4).
__global__ __launch_bounds__(kThreadsS) void k_embed_labels_v(int64_t n, int64_t f, int C,
                                                              const float* __restrict__ x,
                                                              int64_t ldx,
                                                              const uint8_t* __restrict__ mask,
                                                              const int32_t* __restrict__ y,
                                                              const float* __restrict__ e,
                                                              float* __restrict__ xp, int64_t ldp) {
  const int64_t q = f / 4;
  const int64_t t = (int64_t)blockIdx.x * kThreadsS + threadIdx.x;
  if (t >= n * q) return;
  const int64_t i = t / q, c = 4 * (t % q);
  const int32_t k = y[i];
  const bool on = mask[i] && k >= 0 && k < C;
  float4 v = *reinterpret_cast<const float4*>(x + i * ldx + c);
  if (on) {
    const float4 w = *reinterpret_cast<const float4*>(e + (int64_t)k * f + c);
    v.x += w.x;
    v.y += w.y;
    v.z += w.z;
    v.w += w.w;
  }
  *reinterpret_cast<float4*>(xp + i * ldp + c) = v;
}

// Masked label propagation, backward: Xp = X + M E with M the one-hot matrix
// of the embedded rows' labels (row i: 1 at column y[i] if mask[i]), so
// dE = M^T dXp, a weight-gradient product. Thread t writes the 4 entries
// [4 (t % q), 4 (t % q) + 4) of row t / q of M (q = ldo / 4).
__global__ __launch_bounds__(kThreadsS) void k_onehot(int64_t n, int C, int64_t ldo,
                                                      const uint8_t* __restrict__ mask,
                                                      const int32_t* __restrict__ y,
                                                      float* __restrict__ m) {
  const int64_t t = (int64_t)blockIdx.x * kThreadsS + threadIdx.x;
  const int64_t q = ldo / 4;
  if (t >= n * q) return;
  const int64_t i = t / q;
  const int c0 = (int)(t - i * q) * 4;
  const int32_t k = y[i];
  const int hot = mask[i] && k >= 0 && k < C ? k : -1;
  float4 v;
  v.x = hot == c0 ? 1.f : 0.f;
  v.y = hot == c0 + 1 ? 1.f : 0.f;
  v.z = hot == c0 + 2 ? 1.f : 0.f;
  v.w = hot == c0 + 3 ? 1.f : 0.f;
  *reinterpret_cast<float4*>(m + i * ldo + c0) = v;
}

// Column sums of dO (the bias gradient) in a fixed order: workgroup b adds
// rows [b R, (b + 1) R) in row order (thread = column, eight rows loaded
// ahead of the additions), then k_colsum_reduce runs one workgroup per
// column: thread t adds the partials t, t + 256, ... in turn, and a fixed
// tree combines the 256 sums.
constexpr int kColsumRows = 1024;
constexpr int kColsumAhead = 8;

__global__ __launch_bounds__(kThreadsS) void k_colsum_partial(int64_t n, int64_t N,
                                                              const float* __restrict__ d,
                                                              int64_t ld,
                                                              float* __restrict__ part) {
  const int64_t c = (int64_t)blockIdx.y * kThreadsS + threadIdx.x;
  if (c >= N) return;
  const int64_t i0 = (int64_t)blockIdx.x * kColsumRows;
  const int64_t i1 = std::min(n, i0 + kColsumRows);
  float s = 0.f;
  int64_t i = i0;
  for (; i + kColsumAhead <= i1; i += kColsumAhead) {
    float v[kColsumAhead];
#pragma unroll
    for (int k = 0; k < kColsumAhead; ++k) v[k] = d[(i + k) * ld + c];
#pragma unroll
    for (int k = 0; k < kColsumAhead; ++k) s += v[k];
  }
  for (; i < i1; ++i) s += d[i * ld + c];
  part[(int64_t)blockIdx.x * N + c] = s;
}

__global__ __launch_bounds__(kThreadsS) void k_colsum_reduce(int64_t nb, int64_t N,
                                                             const float* __restrict__ part,
                                                             float* __restrict__ out) {
  __shared__ float red[kThreadsS];
  const int64_t c = blockIdx.x;
  float s = 0.f;
  for (int64_t b = threadIdx.x; b < nb; b += kThreadsS) s += part[b * N + c];
  red[threadIdx.x] = s;
  __syncthreads();
  for (int off = kThreadsS / 2; off > 0; off >>= 1) {
    if ((int)threadIdx.x < off) red[threadIdx.x] += red[threadIdx.x + off];
    __syncthreads();
  }
  if (threadIdx.x == 0) out[c] = red[0];
}

inline unsigned blocks(int64_t work) {
  return (unsigned)std::max<int64_t>(1, ceil_div(work, kThreadsS));
}

// Buffers of one layer.
struct Layer {
  int64_t f = 0, fp = 0, zo = 0, oc = 0, K = 0, ldc = 0, fo = 0, fop = 0;
  bool tf = false;        // fo < f: the layer aggregates Y W_neigh (M) instead of Y (Z)
  float* c = nullptr;     // [n x ldc] = [Y | Z | 1 000] or [Y | M | 1 000]
  float* rstd = nullptr;  // [n]
  float* wp = nullptr;    // [K x fop]
  float* wn = nullptr;    // tf: W_neigh padded to [f x fop]
  float* bc = nullptr;    // tf: [W_self | 0 | W_neigh | 0], [f x 2 fop]
  float* o = nullptr;     // [n x fop] pre-activation; after ReLU the layer output
};

inline int64_t round32(int64_t v) { return (v + 31) & ~int64_t(31); }

void set_layout(Layer& y, int64_t f, int64_t fo) {
  y.f = f;
  y.fp = round4(f);
  y.tf = fo < f;
  y.zo = f >= 128 ? round32(f) : y.fp;
  y.oc = y.zo + (y.tf ? round4(fo) : y.fp);
  y.K = y.oc + 4;
  y.ldc = round32(y.K);
  y.fo = fo;
  y.fop = round4(fo);
}

struct Sage {
  int64_t n = 0;
  Layer L[3];
  float* xp = nullptr;    // input with label embeddings ([n x fp of layer 1])
  float* tmid = nullptr;  // Y W_neigh of the layers that aggregate it
};

gcn_status check_args(const gcn_graph* g, const float* X, int64_t ldx, int64_t f_in,
                      int64_t hidden, int64_t n_classes, const float* const* params,
                      const int32_t* labels, const uint8_t* lp_mask, const float* E, double eps) {
  GCN_CHECK(check_graph(g));
  if (g->n_rows != g->n_cols) {
    set_error("the GraphSAGE model needs a square graph");
    return GCN_EINVAL;
  }
  if (!X || !params || f_in <= 0 || hidden <= 0 || n_classes <= 0 || n_classes > 64 ||
      ldx < f_in || !(eps >= 0.0)) {
    set_error("invalid GraphSAGE arguments (1 <= n_classes <= 64, ldx >= f_in, eps >= 0)");
    return GCN_EINVAL;
  }
  for (int k = 0; k < 9; ++k)
    if (!params[k]) {
      set_error("params[%d] must be non-NULL", k);
      return GCN_EINVAL;
    }
  if (lp_mask && (!E || !labels)) {
    set_error("label propagation needs the labels and the embedding E");
    return GCN_EINVAL;
  }
  return GCN_OK;
}

void sage_free(Sage& m, hipStream_t s) {
  tfree(m.tmid, s);
  m.tmid = nullptr;
  tfree(m.xp, s);
  for (int l = 2; l >= 0; --l) {
    tfree(m.L[l].o, s);
    tfree(m.L[l].bc, s);
    tfree(m.L[l].wn, s);
    tfree(m.L[l].wp, s);
    tfree(m.L[l].rstd, s);
    tfree(m.L[l].c, s);
    m.L[l] = Layer();
  }
  m.xp = nullptr;
}

// Shapes, buffers, packed weights and the forward pass; on return L[2].o
// holds the logits and L[0..1].o the ReLU outputs of layers 1 and 2.
gcn_status sage_forward(const gcn_graph* g, const float* X, int64_t ldx, int64_t f_in,
                        int64_t hidden, int64_t n_classes, const float* const* params,
                        const int32_t* labels, const uint8_t* lp_mask, const float* E, double eps,
                        Sage& m, hipStream_t s) {
  const int64_t n = g->n_rows;
  m.n = n;
  Layer* L = m.L;
  const int64_t dims[4] = {f_in, hidden, hidden, n_classes};
  for (int l = 0; l < 3; ++l) set_layout(L[l], dims[l], dims[l + 1]);
  gcn_status st = GCN_OK;
  for (int l = 0; l < 3 && st == GCN_OK; ++l) {
    st = talloc(&L[l].c, n * L[l].ldc, s, "concatenated layer input");
    if (st == GCN_OK) st = talloc(&L[l].rstd, n, s, "LayerNorm 1/std");
    if (st == GCN_OK) st = talloc(&L[l].wp, L[l].K * L[l].fop, s, "packed weights");
    if (st == GCN_OK) st = talloc(&L[l].o, n * L[l].fop, s, "layer output");
    if (st == GCN_OK && L[l].tf) st = talloc(&L[l].wn, L[l].f * L[l].fop, s, "padded W_neigh");
    if (st == GCN_OK && L[l].tf) st = talloc(&L[l].bc, L[l].f * 2 * L[l].fop, s, "[W_self | W_neigh]");
  }
  int64_t t_max = 0;
  for (int l = 0; l < 3; ++l)
    if (L[l].tf) t_max = std::max(t_max, n * L[l].fop);
  if (st == GCN_OK && t_max > 0) st = talloc(&m.tmid, t_max, s, "Y W_neigh");
  if (st == GCN_OK && lp_mask) st = talloc(&m.xp, n * L[0].fp, s, "input with label embeddings");
  GCN_CHECK(st);
  // packed weights and the constant columns of each C
  for (int l = 0; l < 3; ++l) {
    Layer& y = L[l];
    hipLaunchKernelGGL(k_pack_weights, dim3(blocks(y.K * y.fop)), dim3(kThreadsS), 0, s, y.f,
                       y.zo, y.oc, y.K, y.fo, y.fop, y.tf, params[3 * l], params[3 * l + 1],
                       params[3 * l + 2], y.wp);
    GCN_HIP(hipGetLastError());
    const int64_t zw = y.tf ? y.fo : y.f;  // columns of the middle block the layer writes
    hipLaunchKernelGGL(k_concat_tail, dim3(blocks(n * (y.K - y.f - zw))), dim3(kThreadsS), 0, s, n,
                       y.f, y.zo, zw, y.oc, y.K, y.c, y.ldc);
    GCN_HIP(hipGetLastError());
    if (y.tf) {
      hipLaunchKernelGGL(k_pad_cols, dim3(blocks(y.f * y.fop)), dim3(kThreadsS), 0, s, y.f, y.fo,
                         params[3 * l + 1], y.fo, y.wn, y.fop);
      GCN_HIP(hipGetLastError());
      hipLaunchKernelGGL(k_pack_bcat, dim3(blocks(y.f * 2 * y.fop)), dim3(kThreadsS), 0, s, y.f,
                         y.fo, y.fop, params[3 * l], params[3 * l + 1], y.bc);
      GCN_HIP(hipGetLastError());
    }
  }
  const float* h = X;
  int64_t ldh = ldx;
  if (lp_mask) {
    const bool vec = f_in % 4 == 0 && ldx % 4 == 0 && L[0].fp % 4 == 0 &&
                     reinterpret_cast<uintptr_t>(X) % 16 == 0 &&
                     reinterpret_cast<uintptr_t>(E) % 16 == 0 &&
                     reinterpret_cast<uintptr_t>(m.xp) % 16 == 0;
    if (vec)
      hipLaunchKernelGGL(k_embed_labels_v, dim3(blocks(n * (f_in / 4))), dim3(kThreadsS), 0, s, n,
                         f_in, (int)n_classes, X, ldx, lp_mask, labels, E, m.xp, L[0].fp);
    else
      hipLaunchKernelGGL(k_embed_labels, dim3(blocks(n * 64)), dim3(kThreadsS), 0, s, n, f_in,
                         (int)n_classes, X, ldx, lp_mask, labels, E, m.xp, L[0].fp);
    GCN_HIP(hipGetLastError());
    h = m.xp;
    ldh = L[0].fp;
  }
  for (int l = 0; l < 3 && st == GCN_OK; ++l) {
    Layer& y = L[l];
    st = layernorm_fwd(n, y.f, h, ldh, eps, y.c, y.ldc, y.rstd, s);
    if (st == GCN_OK && !y.tf) {
      st = aggregate_f32(g->csr, y.c, y.ldc, y.c + y.zo, y.ldc, y.f, false, s);
    } else if (st == GCN_OK) {
      // M = D^-1 A (Y W_neigh): the aggregation gathers fo-wide rows
      st = gemm_f32(GCN_GEMM_NN, n, y.fo, y.f, y.c, y.ldc, y.wn, y.fop, m.tmid, y.fop, s);
      if (st == GCN_OK)
        st = aggregate_f32(g->csr, m.tmid, y.fop, y.c + y.zo, y.ldc, y.fo, false, s);
    }
    // the ReLU of layers 1 and 2 is applied as the product is stored
    if (st == GCN_OK)
      st = gemm_f32(GCN_GEMM_NN, n, y.fop, y.K, y.c, y.ldc, y.wp, y.fop, y.o, y.fop, s, nullptr, 0,
                    l < 2);
    h = y.o;
    ldh = y.fop;
  }
  return st;
}

gcn_status copy_rows(float* dst, int64_t ldd, const float* src, int64_t lds, int64_t n,
                     int64_t cols, hipStream_t s) {
  if (!dst || n == 0) return GCN_OK;
  GCN_HIP(hipMemcpy2DAsync(dst, ldd * sizeof(float), src, lds * sizeof(float),
                           cols * sizeof(float), n, hipMemcpyDeviceToDevice, s));
  return GCN_OK;
}

// dE = M^T dXp with M the one-hot rows of the embedded rows' labels (*part
// receives M, released by the caller).
gcn_status embed_grad(int64_t n, int C, int64_t f_in, const uint8_t* lp_mask,
                      const int32_t* labels, const float* dxp, int64_t ldp, float* dE,
                      float** part, hipStream_t s) {
  const int64_t ldo = (C + 3) & ~int64_t(3);
  GCN_CHECK(talloc(part, n * ldo, s, "label one-hot rows"));
  hipLaunchKernelGGL(k_onehot, dim3(blocks(n * (ldo / 4))), dim3(kThreadsS), 0, s, n, C, ldo,
                     lp_mask, labels, *part);
  GCN_HIP(hipGetLastError());
  return gemm_f32(GCN_GEMM_TN, C, f_in, n, *part, ldo, dxp, ldp, dE, f_in, s);
}

// Backward pass and loss after sage_forward.
gcn_status sage_backward(const gcn_graph* g, int64_t f_in, int64_t n_classes,
                         const int32_t* labels, const uint8_t* lp_mask, float* const* grads,
                         float* dE, double* loss, Sage& m, hipStream_t s) {
  const int64_t n = m.n;
  const int C = (int)n_classes;
  Layer* L = m.L;
  float *dlogits = nullptr, *dc = nullptr, *t = nullptr, *dwp = nullptr, *part = nullptr;
  float* colpart = nullptr;
  const int64_t n_colsum = std::max<int64_t>(1, ceil_div(n, kColsumRows));
  const int64_t ld_dc = std::max(std::max(L[0].ldc, L[1].ldc), L[2].ldc);
  const int64_t ld_t = std::max(L[0].fp, L[1].fp);
  int64_t w_max = 0;
  for (int l = 0; l < 3; ++l) {
    w_max = std::max(w_max, L[l].K * L[l].fop);
    if (L[l].tf) w_max = std::max(w_max, L[l].f * 2 * L[l].fop);
  }
  // [dO | G] of each layer that aggregates Y W_neigh: read on both streams,
  // so one buffer per layer
  float* dgl[3] = {nullptr, nullptr, nullptr};
  gcn_status st = talloc(&dlogits, n * L[2].fop, s, "dlogits");
  if (st == GCN_OK) st = talloc(&dc, n * ld_dc, s, "dC");
  if (st == GCN_OK) st = talloc(&t, n * ld_t, s, "transposed aggregation");
  if (st == GCN_OK) st = talloc(&dwp, w_max, s, "packed weight gradient");
  if (st == GCN_OK)
    st = talloc(&colpart, n_colsum * std::max(L[1].fop, L[2].fop), s, "bias gradient partials");
  for (int l = 0; l < 3 && st == GCN_OK; ++l)
    if (L[l].tf) st = talloc(&dgl[l], n * 2 * L[l].fop, s, "[dO | G]");
  if (st == GCN_OK)
    st = softmax_xent(n, C, L[2].o, L[2].fop, labels, dlogits, L[2].fop, loss, s, lp_mask);
  // The weight gradients of a layer (product, bias sums, unpacking) read only
  // that layer's C and dO, so they run on the side stream. They are forked
  // after the input-gradient product (also matrix-core bound), so that they
  // overlap the memory-bound transposed aggregation and LayerNorm backward
  // on s. dwp and colpart are used on the side stream only.
  SideWork side;
  if (st == GCN_OK) st = side.init(s);
  const hipStream_t s2 = side.side;
  float* dO = dlogits;
  int64_t ld_do = L[2].fop;
  for (int l = 2; l >= 0 && st == GCN_OK; --l) {
    Layer& y = L[l];
    const bool input_grad = l > 0 || lp_mask;
    if (y.tf) {
      // DG = [dO | G] with G = (D^-1 A)^T dO, fo wide; padding columns zero
      const int64_t ldg = 2 * y.fop;
      float* dg = dgl[l];
      hipError_t e = hipSuccess;
      if (ld_do >= y.fop && ld_do % 4 == 0 && reinterpret_cast<uintptr_t>(dO) % 16 == 0) {
        const int64_t q = y.fop / 4 + (y.fo % 4 != 0 ? 1 : 0);
        hipLaunchKernelGGL(k_fill_dg, dim3(blocks(n * q)), dim3(kThreadsS), 0, s, n, y.fo, y.fop,
                           (const float*)dO, ld_do, dg);
        e = hipGetLastError();
      } else {
        hipLaunchKernelGGL(k_zero_dg_pad, dim3(blocks(n * 2 * (y.fop - y.fo))), dim3(kThreadsS),
                           0, s, n, y.fo, y.fop, dg);
        e = hipGetLastError();
        if (e == hipSuccess) st = copy_rows(dg, ldg, dO, ld_do, n, y.fo, s);
      }
      if (e != hipSuccess) {
        st = hip_fail(e, "[dO | G] fill", __FILE__, __LINE__);
        break;
      }
      if (st == GCN_OK) st = aggregate_f32(g->csc, dO, ld_do, dg + y.fop, ldg, y.fo, false, s);
      if (st == GCN_OK) st = side.fork();  // DG is complete on s
      if (st != GCN_OK) break;
      // weight gradients on the side stream: [dW_self | dW_neigh] = Y^T DG, db = colsum dO
      st = gemm_f32(GCN_GEMM_TN, y.f, ldg, n, y.c, y.ldc, dg, ldg, dwp, ldg, s2);
      if (st != GCN_OK) break;
      {
        ProfScope ps("bias_grad", s2);
        hipLaunchKernelGGL(k_colsum_partial,
                           dim3((unsigned)n_colsum, (unsigned)ceil_div(y.fo, kThreadsS)),
                           dim3(kThreadsS), 0, s2, n, y.fo, (const float*)dO, ld_do, colpart);
        hipLaunchKernelGGL(k_colsum_reduce, dim3((unsigned)y.fo), dim3(kThreadsS), 0, s2,
                           n_colsum, y.fo, (const float*)colpart, grads[3 * l + 2]);
      }
      hipLaunchKernelGGL(k_unpack_grads_tf, dim3(blocks(2 * y.f * y.fo)), dim3(kThreadsS), 0, s2,
                         y.f, y.fo, y.fop, (const float*)dwp, grads[3 * l], grads[3 * l + 1]);
      e = hipGetLastError();
      if (e != hipSuccess) {
        st = hip_fail(e, "tf layer gradients", __FILE__, __LINE__);
        break;
      }
      if (!input_grad) break;
      if (l > 0 && sage_tf_bwd_fusable(y.f, ldg, dg, ldg)) {
        // dY in registers, straight into the LayerNorm backward and the
        // ReLU mask of the layer below (whose output it overwrites)
        Layer& below = L[l - 1];
        st = sage_tf_bwd_fused(n, y.f, ldg, dg, ldg, y.bc, ldg, y.c, y.ldc, y.rstd, below.o,
                               below.fop, s);
        dO = below.o;
        ld_do = below.fop;
        continue;
      }
      // dY = dO W_self^T + G W_neigh^T = DG [W_self | W_neigh]^T, then the LayerNorm backward
      st = gemm_f32(GCN_GEMM_NT, n, y.f, ldg, dg, ldg, y.bc, ldg, dc, y.ldc, s);
      if (st != GCN_OK) break;
      if (l > 0) {
        Layer& below = L[l - 1];
        st = layernorm_bwd(n, y.f, y.c, y.ldc, y.rstd, dc, y.ldc, nullptr, 0, below.o, below.fop,
                           below.o, below.fop, s);
        dO = below.o;
        ld_do = below.fop;
        continue;
      }
      st = layernorm_bwd(n, y.f, y.c, y.ldc, y.rstd, dc, y.ldc, nullptr, 0, nullptr, 0, m.xp, y.fp,
                         s);
      if (st == GCN_OK) st = embed_grad(n, C, f_in, lp_mask, labels, m.xp, y.fp, dE, &part, s);
      break;
    }
    // dC = dO Wp^T; the input gradient of the layer is
    // dY = dC[:, Y block] + A^T dC[:, Z block], then the LayerNorm backward
    // dC over the Y and Z blocks only (the ones and padding columns are not read)
    if (input_grad) st = gemm_f32(GCN_GEMM_NT, n, y.zo + y.f, y.fo, dO, ld_do, y.wp, y.fop, dc,
                                  y.ldc, s);
    if (st == GCN_OK) st = side.fork();  // dO of this layer and dC are complete on s
    if (st != GCN_OK) break;
    // only the fo real columns of dO enter the products: the padding columns of
    // the logits gradient are never written. The product covers rows [0, oc)
    // of the packed gradient (the W blocks); the bias row oc is the column sum
    // of dO, computed on its own so that a 2f + 4 row count does not cost a
    // whole extra tile of the product.
    st = gemm_f32(GCN_GEMM_TN, y.oc, y.fo, n, y.c, y.ldc, dO, ld_do, dwp, y.fop, s2);
    if (st != GCN_OK) break;
    {
      ProfScope ps("bias_grad", s2);
      hipLaunchKernelGGL(k_colsum_partial,
                         dim3((unsigned)n_colsum, (unsigned)ceil_div(y.fo, kThreadsS)),
                         dim3(kThreadsS), 0, s2, n, y.fo, (const float*)dO, ld_do, colpart);
      hipLaunchKernelGGL(k_colsum_reduce, dim3((unsigned)y.fo), dim3(kThreadsS), 0, s2,
                         n_colsum, y.fo, (const float*)colpart, dwp + y.oc * y.fop);
    }
    if (hipGetLastError() != hipSuccess) {
      st = hip_fail(hipErrorLaunchFailure, "bias gradient", __FILE__, __LINE__);
      break;
    }
    hipLaunchKernelGGL(k_unpack_grads, dim3(blocks((2 * y.f + 1) * y.fo)), dim3(kThreadsS), 0, s2,
                       y.f, y.zo, y.oc, y.fo, y.fop, (const float*)dwp, grads[3 * l],
                       grads[3 * l + 1], grads[3 * l + 2]);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) {
      st = hip_fail(e, "k_unpack_grads", __FILE__, __LINE__);
      break;
    }
    if (!input_grad) break;
    st = aggregate_f32(g->csc, dc + y.zo, y.ldc, t, y.fp, y.f, false, s);
    if (st != GCN_OK) break;
    if (l > 0) {
      // the gradient of the layer below, masked by its ReLU, overwrites its output
      Layer& below = L[l - 1];
      st = layernorm_bwd(n, y.f, y.c, y.ldc, y.rstd, dc, y.ldc, t, y.fp, below.o, below.fop,
                         below.o, below.fop, s);
      dO = below.o;
      ld_do = below.fop;
    } else {
      // label propagation: dXp, then the embedding gradient
      st = layernorm_bwd(n, y.f, y.c, y.ldc, y.rstd, dc, y.ldc, t, y.fp, nullptr, 0, m.xp, y.fp,
                         s);
      if (st == GCN_OK) st = embed_grad(n, C, f_in, lp_mask, labels, m.xp, y.fp, dE, &part, s);
    }
  }
  // the side work ends before its buffers are released on s
  const gcn_status sj = side.join();
  if (st == GCN_OK) st = sj;
  tfree(part, s);
  for (int l = 2; l >= 0; --l) tfree(dgl[l], s);
  tfree(colpart, s);
  tfree(dwp, s);
  tfree(t, s);
  tfree(dc, s);
  tfree(dlogits, s);
  return st;
}


}  // namespace
}  // namespace gcn

using namespace gcn;

extern "C" gcn_status gcn_sage3_forward(const gcn_graph* g, const float* X, int64_t ldx,
                                        int64_t f_in, int64_t hidden, int64_t n_classes,
                                        const float* const* params, const int32_t* labels,
                                        const uint8_t* lp_mask, const float* E, double eps,
                                        float* H1, int64_t ldh1, float* H2, int64_t ldh2,
                                        float* logits, int64_t ldl, void* stream_) {
  clear_error();
  GCN_CHECK(check_args(g, X, ldx, f_in, hidden, n_classes, params, labels, lp_mask, E, eps));
  if ((H1 && ldh1 < hidden) || (H2 && ldh2 < hidden) || (logits && ldl < n_classes)) {
    set_error("output leading dimensions must cover the output widths");
    return GCN_EINVAL;
  }
  hipStream_t s = (hipStream_t)stream_;
  Sage m;
  gcn_status st = sage_forward(g, X, ldx, f_in, hidden, n_classes, params, labels, lp_mask, E,
                               eps, m, s);
  if (st == GCN_OK) st = copy_rows(H1, ldh1, m.L[0].o, m.L[0].fop, m.n, hidden, s);
  if (st == GCN_OK) st = copy_rows(H2, ldh2, m.L[1].o, m.L[1].fop, m.n, hidden, s);
  if (st == GCN_OK) st = copy_rows(logits, ldl, m.L[2].o, m.L[2].fop, m.n, n_classes, s);
  sage_free(m, s);
  return st;
}

extern "C" gcn_status gcn_sage3_step(const gcn_graph* g, const float* X, int64_t ldx, int64_t f_in,
                                     int64_t hidden, int64_t n_classes,
                                     const float* const* params, const int32_t* labels,
                                     const uint8_t* lp_mask, const float* E, double eps,
                                     float* const* grads, float* dE, double* loss,
                                     void* stream_) {
  clear_error();
  GCN_CHECK(check_args(g, X, ldx, f_in, hidden, n_classes, params, labels, lp_mask, E, eps));
  if (!grads || !labels || !loss || (lp_mask && !dE)) {
    set_error("the step needs labels, grads, loss (and dE with label propagation)");
    return GCN_EINVAL;
  }
  for (int k = 0; k < 9; ++k)
    if (!grads[k]) {
      set_error("grads[%d] must be non-NULL", k);
      return GCN_EINVAL;
    }
  hipStream_t s = (hipStream_t)stream_;
  Sage m;
  gcn_status st = sage_forward(g, X, ldx, f_in, hidden, n_classes, params, labels, lp_mask, E,
                               eps, m, s);
  if (st == GCN_OK)
    st = sage_backward(g, f_in, n_classes, labels, lp_mask, grads, dE, loss, m, s);
  sage_free(m, s);
  return st;
}
