// One training step of a 2-layer GCN built from the library's kernels:
// aggregation (Section 4 of SuperGCN, arXiv 2411.16025) interleaved with the
// dense UPDATE of each layer (Section 2.1). Everything is ordered on the
// caller's stream without host synchronization (without the fused backward,
// one product runs on the side stream, forked from and joined back to it).
//
// Each layer multiplies A_hat, its input and its weights; the association is
// chosen so that the aggregation gathers the narrower operand. Layer 1
// aggregates first when f_in <= hidden, as the paper's AGGREGATE-then-UPDATE:
// P = A_hat X, H1 = relu(P W1). Its weight gradient is then dW1 = P^T dZ1
// with dZ1 the gradient at P W1 (dH1 masked by H1 > 0), and no aggregation
// runs in its backward (the input gradient is not needed); for f_in <= 112
// and at most 48 classes, dZ1, dW1 and dW2 then come from one fused pass over
// the rows that keeps dZ1 in registers, and (hidden <= 256) H1 and Z2 = H1 W2
// from one forward pass that keeps H1 in registers for Z2. Otherwise it
// transforms first:
// H1 = relu(A_hat (X W1)), dW1 = X^T (A_hat^T dZ1). Layer 2 transforms first
// (its output, the classes, is the narrower side): logits = A_hat (H1 W2).

#include "common.h"

using namespace gcn;

extern "C" gcn_status gcn_gcn2_step(const gcn_graph* g, const float* X, int64_t ldx, int64_t f_in,
                                    const float* W1, int64_t hidden, const float* W2,
                                    int64_t n_classes, const int32_t* labels, float* dW1,
                                    float* dW2, double* loss, void* stream_) {
  clear_error();
  GCN_CHECK(check_graph(g));
  if (g->n_rows != g->n_cols) {
    set_error("the GCN step needs a square graph");
    return GCN_EINVAL;
  }
  if (!X || !W1 || !W2 || !labels || !dW1 || !dW2 || !loss || f_in <= 0 || hidden <= 0 ||
      n_classes <= 0 || n_classes > 64 || ldx < f_in) {
    set_error("invalid GCN step arguments (1 <= n_classes <= 64)");
    return GCN_EINVAL;
  }
  hipStream_t s = (hipStream_t)stream_;
  const int64_t n = g->n_rows;
  const int64_t ldh = (hidden + 3) & ~int64_t(3);
  const int64_t ldc = (n_classes + 3) & ~int64_t(3);
  // layer 1 aggregates first when its input is no wider than its output
  const bool agg_first = f_in <= hidden;
  const int64_t ldp = agg_first ? (f_in + 3) & ~int64_t(3) : ldh;
  // P: A_hat X (aggregation first) or X W1 (transform first)
  float *p = nullptr, *h1 = nullptr, *z2 = nullptr, *lg = nullptr, *dl = nullptr, *dz2 = nullptr;
  float *dz1 = nullptr, *dh1 = nullptr;
  float* w2p = nullptr;  // W2 with rows padded to a multiple of 4 floats (16-byte aligned rows)
  gcn_status st = talloc(&p, n * ldp, s, "P");
  if (st == GCN_OK) st = talloc(&w2p, hidden * ldc, s, "W2 copy");
  if (st == GCN_OK) {
    hipError_t e = hipMemcpy2DAsync(w2p, ldc * sizeof(float), W2, n_classes * sizeof(float),
                                    n_classes * sizeof(float), hidden, hipMemcpyDeviceToDevice, s);
    if (e != hipSuccess) st = hip_fail(e, "hipMemcpy2DAsync", __FILE__, __LINE__);
  }
  if (st == GCN_OK) st = talloc(&h1, n * ldh, s, "H1");
  if (st == GCN_OK) st = talloc(&z2, n * ldc, s, "Z2");
  if (st == GCN_OK) st = talloc(&lg, n * ldc, s, "logits");
  if (st == GCN_OK) st = talloc(&dl, n * ldc, s, "dlogits");
  if (st == GCN_OK) st = talloc(&dz2, n * ldc, s, "dZ2");
  // forward
  const bool fwd_fused = agg_first && layer1_fwd_fusable(f_in, hidden, n_classes, p, ldp, h1, ldh);
  if (agg_first) {
    if (st == GCN_OK) st = aggregate_f32(g->csr, X, ldx, p, ldp, f_in, false, s);
    if (fwd_fused) {
      // H1 = relu(P W1) and Z2 = H1 W2 in one pass (Z2 from H1 in registers)
      if (st == GCN_OK)
        st = layer1_fwd_fused(n, f_in, hidden, n_classes, p, ldp, W1, hidden, w2p, ldc, h1, ldh,
                              z2, ldc, s);
    } else if (st == GCN_OK) {
      // H1 = relu(P W1), the ReLU applied as the product stores its tile
      st = gemm_f32(GCN_GEMM_NN, n, hidden, f_in, p, ldp, W1, hidden, h1, ldh, s, nullptr, 0, true);
    }
  } else {
    if (st == GCN_OK) st = gemm_f32(GCN_GEMM_NN, n, hidden, f_in, X, ldx, W1, hidden, p, ldh, s);
    if (st == GCN_OK) st = aggregate_f32(g->csr, p, ldh, h1, ldh, hidden, true, s);  // + ReLU
  }
  if (st == GCN_OK && !fwd_fused)
    st = gemm_f32(GCN_GEMM_NN, n, n_classes, hidden, h1, ldh, w2p, ldc, z2, ldc, s);
  if (st == GCN_OK) st = aggregate_f32(g->csr, z2, ldc, lg, ldc, n_classes, false, s);
  if (st == GCN_OK) st = softmax_xent(n, (int)n_classes, lg, ldc, labels, dl, ldc, loss, s);
  // backward
  if (st == GCN_OK) st = aggregate_f32(g->csc, dl, ldc, dz2, ldc, n_classes, false, s);
  if (agg_first && layer1_bwd_fusable(f_in, hidden, n_classes, dz2, ldc, w2p, ldc)) {
    // dZ1 = (dZ2 W2^T) masked by H1 > 0, dW1 = P^T dZ1 and dW2 = H1^T dZ2 in
    // one pass over the rows, dZ1 kept in registers
    if (st == GCN_OK)
      st = layer1_bwd_fused(n, f_in, hidden, n_classes, p, ldp, h1, ldh, dz2, ldc, w2p, ldc, dW1,
                            dW2, s);
  } else {
    if (st == GCN_OK) st = talloc(&dz1, n * ldh, s, "dZ1");
    // dW2 = H1^T dZ2 reads only H1 and dZ2: on the side stream it overlaps
    // the rest of the backward
    SideWork side;
    if (st == GCN_OK) st = side.init(s);
    if (st == GCN_OK) st = side.fork();
    if (st == GCN_OK) st = gemm_f32(GCN_GEMM_TN, hidden, n_classes, n, h1, ldh, dz2, ldc, dW2,
                                    n_classes, side.side);
    // dH1 = dZ2 W2^T with the ReLU mask (H1 > 0) applied as it is stored:
    // with the aggregation first this is already dZ1 (the gradient at P W1)
    dh1 = agg_first ? dz1 : p;  // (X W1 is dead after the first aggregation)
    if (st == GCN_OK) st = gemm_f32(GCN_GEMM_NT, n, hidden, n_classes, dz2, ldc, w2p, ldc, dh1,
                                    ldh, s, h1, ldh);
    if (agg_first) {
      // dW1 = P^T dZ1
      if (st == GCN_OK)
        st = gemm_f32(GCN_GEMM_TN, f_in, hidden, n, p, ldp, dz1, ldh, dW1, hidden, s);
    } else {
      // dZ1 = A_hat^T dH1, dW1 = X^T dZ1
      if (st == GCN_OK) st = aggregate_f32(g->csc, dh1, ldh, dz1, ldh, hidden, false, s);
      if (st == GCN_OK)
        st = gemm_f32(GCN_GEMM_TN, f_in, hidden, n, X, ldx, dz1, ldh, dW1, hidden, s);
    }
    // the side work ends before the buffers it reads are released on s
    const gcn_status sj = side.join();
    if (st == GCN_OK) st = sj;
  }
  tfree(dz1, s);
  tfree(dz2, s);
  tfree(dl, s);
  tfree(lg, s);
  tfree(z2, s);
  tfree(h1, s);
  tfree(p, s);
  tfree(w2p, s);
  return st;
}
