/* gcnagg.h -- C ABI of the GCN aggregation library for AMD Instinct MI355X
 * (gfx950).
 *
 * The library computes the graph aggregation step of full-batch GCN training
 * as described in SuperGCN (Chen et al., "Scaling Large-scale GNN Training
 * to Thousands of Processors on CPU-based Supercomputers", arXiv 2411.16025):
 *
 *   forward   Y  = A_hat X            (Section 4: Index_add / SpMM)
 *   backward  dX = A_hat^T G
 *   with A_hat = D~^-1/2 (A + I) D~^-1/2, the GCN propagation matrix
 *   (Section 2.1 cites GCN; Lemma 2 in Section 6.3 writes a layer as A H W),
 *
 * plus the consumer side of the paper's quantized boundary exchange
 * (Section 6.1, step 3): halo feature rows arrive as 8-bit codes with a
 * per-row zero point and scale (Section 2.4) and are dequantized inside the
 * aggregation.
 *
 * Conventions shared by every call:
 *  - Pointers are DEVICE pointers unless a parameter says "host".
 *  - `stream` is a hipStream_t passed as void* (NULL = the default stream).
 *    Work is enqueued on it; a call returns before the work completes unless
 *    stated otherwise. Inputs must stay valid until the stream reaches it.
 *  - Matrices are row-major with an explicit leading dimension (elements
 *    between consecutive rows), ld >= F.
 *  - Edge (s -> d) means "row s of the input is added into row d of the
 *    output": the stored entry has row d and column s (Section 4: rows of
 *    src are added to dst at the positions idx names).
 *  - Every call returns a gcn_status and never throws. On failure,
 *    gcn_last_error() returns a message for the calling thread. Argument
 *    errors are detected before any work is enqueued, so outputs are left
 *    untouched.
 *  - Calls that share a gcn_graph may run concurrently only if none of them
 *    is gcn_normalize or gcn_graph_free.
 *  - Temporaries are allocated stream-ordered from the device's default
 *    memory pool; on first use the library sets that pool's release
 *    threshold to keep freed blocks for reuse (they stay reserved for the
 *    process).
 */
#ifndef GCNAGG_H
#define GCNAGG_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct gcn_graph gcn_graph; /* opaque; owns its device arrays */

typedef enum {
  GCN_OK = 0,
  GCN_EINVAL = 1, /* null pointer, non-positive size, ld < F, unknown dtype/flag, bad shape */
  GCN_ERANGE = 2, /* vertex id out of range, n_local_cols > n_cols, sizes beyond int32 ids */
  GCN_ENOMEM = 3, /* device allocation failed */
  GCN_EHIP = 4,   /* a HIP runtime call failed */
  GCN_ESTATE = 5  /* freed / corrupted handle, a handle used while another device is
                     current, or a call out of order */
} gcn_status;

/* gcn_build_csr flags */
enum {
  GCN_SYMMETRIZE = 1u,    /* also store the reverse of every edge (square graphs only) */
  GCN_ADD_SELF_LOOPS = 2u /* drop drawn self pairs, then store one (i, i) per
                             i < min(n_rows, n_cols) */
};

/* input element types of the aggregation calls; accumulation and output are fp32 */
enum { GCN_DT_F32 = 0, GCN_DT_BF16 = 1 };

/* gcn_aggregate_fwd_q8halo flags */
enum {
  GCN_Q8_USE_CSC = 1u, /* aggregate with A_hat^T instead of A_hat */
  GCN_Q_CODES_2BIT = 2u /* halo codes are 2-bit, packed four per byte (see
                           gcn_layernorm_quantize); ldq >= (F + 3) / 4 */
};

/* Build the sparse structure of A (or A + I) from an edge list: the
 * "clustering and sorting" step of Section 4 done on the device. Entries are
 * sorted by (row, column) and deduplicated, so A is binary. The transpose is
 * built as well (for symmetric graphs it is the same matrix and shares the
 * arrays), so the backward pass reads A^T row by row without atomics. Rows
 * are then binned by length for the aggregation kernels. Every stored value
 * is 1.0 until gcn_normalize runs (an unnormalized graph aggregates like
 * Index_add).
 *
 *  n_rows, n_cols  output rows / input rows of the operator, 1 .. 2^31-1.
 *                  Columns >= n_rows of a rectangular graph are halo nodes.
 *  n_edges         number of (src, dst) pairs, >= 0.
 *  src, dst        int32 device arrays [n_edges]; src in [0, n_cols),
 *                  dst in [0, n_rows) (checked on the device -> GCN_ERANGE).
 *  flags           GCN_SYMMETRIZE (requires n_rows == n_cols) | GCN_ADD_SELF_LOOPS.
 *  out             host pointer that receives the new handle.
 * Synchronizes `stream` (the entry count and bin sizes are read back).
 * Device memory: about 24 bytes per stored entry while building, 8 per
 * entry afterwards (twice that for a non-symmetric graph). */
gcn_status gcn_build_csr(int64_t n_rows, int64_t n_cols, int64_t n_edges, const int32_t* src,
                         const int32_t* dst, uint32_t flags, void* stream, gcn_graph** out);

/* Overwrite the stored values of A and A^T with the entries of
 * A_hat = D~^-1/2 (A + I) D~^-1/2: entry (r, c) becomes
 * (float)(1 / sqrt((double)(deg[r] + 1) * (double)(deg[c] + 1))), computed
 * with IEEE double division and square root.
 *  deg  NULL: deg[v] = number of stored entries of row v other than (v, v)
 *       (square graphs only); otherwise an int32 device array indexed by
 *       node id, [max(n_rows, n_cols)] entries, of caller-supplied degrees
 *       without the self-loop (e.g. global degrees of a partition whose cut
 *       edges live on other workers), each >= 0 (else GCN_EINVAL).
 *  Synchronizes `stream` when deg is supplied (the degrees are checked). */
gcn_status gcn_normalize(gcn_graph* g, const int32_t* deg, void* stream);

/* As gcn_normalize, with separate degree arrays for the rows and for the
 * columns: entry (r, c) becomes
 * (float)(1 / sqrt((double)(deg_rows[r] + 1) * (double)(deg_cols[c] + 1))).
 * This normalizes an operator whose row and column ids are different node
 * sets, such as the pre-aggregation matrix of Section 5.2 (rows: the
 * receiver's nodes in the vertex cover; columns: the sender's nodes) or a
 * receiver whose columns are its own nodes followed by received rows.
 *  deg_rows  int32 device array [n_rows], degrees without the self-loop, >= 0.
 *  deg_cols  int32 device array [n_cols], likewise.
 * A^T receives the transposed values. A symmetric graph (GCN_SYMMETRIZE)
 * stores one structure for both directions; when deg_rows and deg_cols are
 * different arrays its A^T first gets entries of its own (8 bytes per entry),
 * since its values are then not those of A.
 *  Negative degrees or NULL arrays -> GCN_EINVAL. Synchronizes `stream`. */
gcn_status gcn_normalize_rc(gcn_graph* g, const int32_t* deg_rows, const int32_t* deg_cols,
                            void* stream);

/* Overwrite the stored values with those of the mean operator D^-1 A
 * (GraphSAGE's mean AGGREGATE, Section 2.1, the model of the evaluation):
 * entry (r, c) becomes (float)(1 / (double)len(r)), len(r) = stored entries of
 * row r of A (self-loops and drawn self pairs count when stored; a graph
 * built without GCN_ADD_SELF_LOOPS gives the mean over neighbours). A^T
 * receives the transposed values; for a symmetric graph it then keeps the
 * shared structure but gets entries of its own (8 bytes per entry more).
 * Asynchronous on `stream`. */
gcn_status gcn_normalize_mean(gcn_graph* g, void* stream);

/* Y[n_rows x F] = A_hat X. X is [n_cols x F] (ldx), fp32 or bf16 (dtype);
 * Y is fp32 (ldy). Accumulation is fp32; each output element is summed in
 * an order fixed by the graph alone, so repeated calls give identical bits. */
gcn_status gcn_aggregate_fwd(const gcn_graph* g, const void* X, int64_t ldx, int dtype, float* Y,
                             int64_t ldy, int64_t F, void* stream);

/* dX[n_cols x F] = A_hat^T G, G is [n_rows x F]. Same rules as the forward. */
gcn_status gcn_aggregate_bwd(const gcn_graph* g, const void* G, int64_t ldg, int dtype, float* dX,
                             int64_t lddx, int64_t F, void* stream);

/* gcn_aggregate_fwd for callers that cannot allocate device memory (code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): same arguments, same kernels and identical results, but the
 * partial rows of long rows live in a fixed array of the library, 2^24 floats
 * (64 MiB) per device, held by every device the library runs on until the
 * process ends. The call allocates nothing and frees nothing.
 *  Returns GCN_ERANGE, before any work is enqueued, when the graph's plan
 *  needs more: (rows cut into chunks or column-blocked pieces, counted as
 *  partial rows) * round_up(F, 4) floats > 2^24.
 * Every call on one device shares that array and leaves its contents behind
 * (each call writes every partial row it reads, so nothing needs clearing):
 * calls that may overlap on one device -- on different streams, or from
 * different threads -- race and must be serialized by the caller. */
gcn_status gcn_aggregate_fwd_noalloc(const gcn_graph* g, const void* X, int64_t ldx, int dtype,
                                     float* Y, int64_t ldy, int64_t F, void* stream);

/* Forward aggregation whose input rows >= n_local_cols are halo rows held as
 * uint8 codes (Section 6.1 step 3; quantization of Section 2.4 with b = 8):
 *   x[j, f] = X_local[j, f]                                   j <  n_local_cols
 *   x[j, f] = fmaf((float)Q_halo[h, f], halo_scale[h * ldp], halo_min[h * ldp]),
 *             h = j - n_local_cols                             j >= n_local_cols
 *   Y = A_hat x   (or A_hat^T x with GCN_Q8_USE_CSC; then x has n_rows rows
 *                  and Y has n_cols rows).
 *  X_local     fp32 [n_local_cols x F] (ldx); may be NULL if n_local_cols == 0.
 *  Q_halo      uint8 [n_in - n_local_cols x F] (ldq), n_in = rows of x; with
 *              GCN_Q_CODES_2BIT the codes are 2-bit (Section 7.3's Int2),
 *              packed four per byte, and the code is taken from byte f / 4.
 *  halo_min, halo_scale   fp32 zero point Z and scale S of halo row h at
 *              element h * ldp (ldp >= 1). ldp = 1: two plain arrays;
 *              ldp = 2 with halo_scale == halo_min + 1: (Z, S) pairs side by
 *              side, so a gather's two 4-byte parameter loads touch one cache
 *              line.
 *  Y           fp32 output (ldy). */
gcn_status gcn_aggregate_fwd_q8halo(const gcn_graph* g, int64_t n_local_cols, const float* X_local,
                                    int64_t ldx, const uint8_t* Q_halo, int64_t ldq,
                                    const float* halo_min, const float* halo_scale, int64_t ldp,
                                    float* Y, int64_t ldy, int64_t F, uint32_t flags,
                                    void* stream);

/* Per-row uint8 quantization (Section 2.4 with b = 8, the producer side of
 * the quantized exchange): Z = min_f X[i, f], S = (max - min) / 255 in fp32,
 * Q[i, f] = clamp(rint((X[i, f] - Z) / S), 0, 255) with IEEE fp32 division
 * and round-half-even (the paper's implementation drops the stochastic
 * rounding, Section 7.3); every code is 0 when S == 0.
 *  X [n x F] fp32 (ldx) -> Q [n x F] uint8 (ldq); zmin[i * ldp] and
 *  scale[i * ldp] fp32 (ldp >= 1; ldp = 2 with scale = zmin + 1 writes the
 *  (Z, S) pairs that gcn_aggregate_fwd_q8halo reads with one load). */
gcn_status gcn_quantize_rows_u8(int64_t n, int64_t F, const float* X, int64_t ldx, uint8_t* Q,
                                int64_t ldq, float* zmin, float* scale, int64_t ldp,
                                void* stream);

/* ---- the dense side of a layer: UPDATE of Section 2.1 ------------------ */

/* GEMM operations */
enum { GCN_GEMM_NN = 0, GCN_GEMM_NT = 1, GCN_GEMM_TN = 2 };

/* fp32 GEMM on the matrix cores, row-major operands:
 *   GCN_GEMM_NN  C[M x N] = A[M x K] B[K x N]
 *   GCN_GEMM_NT  C[M x N] = A[M x K] B[N x K]^T
 *   GCN_GEMM_TN  C[M x N] = A[K x M]^T B[K x N]   (K may be millions: split
 *                into fixed chunks whose partial products are added in chunk
 *                order, so results repeat bit for bit; needs M * N < 2^31)
 * lda, ldb, ldc are the row strides of the stored matrices. fp32 inputs and
 * fp32 accumulation. */
gcn_status gcn_gemm_f32(int op, int64_t M, int64_t N, int64_t K, const float* A, int64_t lda,
                        const float* B, int64_t ldb, float* C, int64_t ldc, void* stream);

/* H[i, f] = max(H[i, f], 0) in place, H [n x F] (ld). */
gcn_status gcn_relu(int64_t n, int64_t F, float* H, int64_t ld, void* stream);

/* dH[i, f] = 0 where H[i, f] <= 0 (H is the ReLU output), in place. */
gcn_status gcn_relu_bwd(int64_t n, int64_t F, const float* H, int64_t ldh, float* dH, int64_t ld,
                        void* stream);

/* Softmax cross-entropy over n rows of C <= 64 logits: *loss (device double)
 * = mean_i (logsumexp(z_i) - z_i[y_i]), dlogits = (softmax(z) - onehot(y)) / n.
 * labels (int32 [n]) must lie in [0, C). Row losses are added in a fixed order
 * in double. */
gcn_status gcn_softmax_xent(int64_t n, int64_t C, const float* logits, int64_t ld,
                            const int32_t* labels, float* dlogits, int64_t ldd, double* loss,
                            void* stream);

/* One training step of a 2-layer GCN on a square graph (Section 2.1: each
 * layer aggregates, then applies a linear transform):
 *   H1 = relu(A_hat X W1), logits = A_hat (H1 W2),
 *   loss = mean softmax cross-entropy, then the exact backward:
 *   dZ2 = A_hat^T dlogits, dW2 = H1^T dZ2, dZ1 = dZ2 W2^T masked by H1 > 0,
 *   dW1 = (A_hat X)^T dZ1.
 *  Layer 1 is evaluated as relu((A_hat X) W1) with dW1 = (A_hat X)^T dZ1 when
 *  f_in <= hidden (the aggregation gathers the narrower rows and the backward
 *  needs none), else as relu(A_hat (X W1)) with dW1 = X^T (A_hat^T dZ1). The
 *  two agree up to fp32 rounding. In the first order, with f_in <= 112 and
 *  n_classes <= 48, dZ1, dW1 and dW2 come from one fused pass over the rows
 *  (dZ1 is never stored), and for hidden <= 256 so do H1 and H1 W2; the sums
 *  are the same up to their order.
 *  X [n x f_in] (ldx), W1 [f_in x hidden], W2 [hidden x n_classes] (dense,
 *  row-major), labels int32 [n] in [0, n_classes), n_classes <= 64.
 *  Outputs: dW1, dW2 (same shapes as W1, W2), *loss (device double).
 * No bias, dropout or normalization layer. Intermediates are allocated
 * stream-ordered for the duration of the call. Without the fused pass, dW2
 * is computed on a second, library-owned stream of the current device
 * (non-blocking, default priority), forked from `stream` by an event and
 * joined back to it before the call returns, so all outputs are ordered on
 * `stream`. */
gcn_status gcn_gcn2_step(const gcn_graph* g, const float* X, int64_t ldx, int64_t f_in,
                         const float* W1, int64_t hidden, const float* W2, int64_t n_classes,
                         const int32_t* labels, float* dW1, float* dW2, double* loss,
                         void* stream);

/* LayerNorm-then-quantize producer for boundary rows (Section 6.1 steps 2
 * and 3; Section 7.3 computes the parameters and the codes in one fused pass
 * and fixes the bit width at 2).
 *  flags   GCN_LAYERNORM: first y = (x - mean) / sqrt(var + eps) * gamma + beta
 *          per row over the F features (biased variance, computed in double,
 *          rounded once to fp32; gamma/beta fp32 [F] or NULL for 1 and 0);
 *          without it y = x.
 *  bits    8: one code byte per feature (as gcn_quantize_rows_u8);
 *          2: codes 0..3 packed four per byte, feature f in bits
 *             [2 (f % 4), 2 (f % 4) + 2) of byte f / 4 (padding codes 0).
 *  Codes: Z = min y, S = (max y - min y) / (2^bits - 1), q = clamp(rint((y - Z)
 *  / S), 0, 2^bits - 1) in fp32, all 0 when S == 0; Z and S at zmin[i * ldp],
 *  scale[i * ldp]. Q [n x ldq] needs ldq >= F (8-bit) or (F + 3) / 4 (2-bit).
 *  Y (optional, [n x F], ldy) receives the normalized rows. */
enum { GCN_LAYERNORM = 1u };
gcn_status gcn_layernorm_quantize(int64_t n, int64_t F, const float* X, int64_t ldx,
                                  const float* gamma, const float* beta, double eps,
                                  uint32_t flags, int bits, float* Y, int64_t ldy, uint8_t* Q,
                                  int64_t ldq, float* zmin, float* scale, int64_t ldp,
                                  void* stream);

/* Row LayerNorm without affine parameters (applied before every layer,
 * Section 6.1 step 2 and Table 2): Y = (X - mean) / sqrt(var + eps) per row
 * over the F features, biased variance, statistics in double, each value
 * rounded once to fp32. rstd (optional, fp32 [n]) receives 1 / sqrt(var + eps).
 * Asynchronous. */
gcn_status gcn_layernorm_fwd(int64_t n, int64_t F, const float* X, int64_t ldx, double eps,
                             float* Y, int64_t ldy, float* rstd, void* stream);

/* Gradient of gcn_layernorm_fwd: dX = rstd * (g - mean(g) - Y * mean(g * Y))
 * per row, with g = dY + dY2 (dY2 optional, NULL for none) and Y, rstd from
 * the forward pass; with mask (optional) dX is zeroed where mask <= 0 (the
 * ReLU of the layer below: pass its output). mask may be dX itself (same ld).
 * Row means in double. Asynchronous. */
gcn_status gcn_layernorm_bwd(int64_t n, int64_t F, const float* Y, int64_t ldy, const float* rstd,
                             const float* dY, int64_t lddy, const float* dY2, int64_t lddy2,
                             const float* mask, int64_t ldm, float* dX, int64_t lddx,
                             void* stream);

/* Forward pass (inference) of the 3-layer GraphSAGE model of gcn_sage3_step,
 * the same kernels in the same order, so its outputs are bit-identical to the
 * step's activations. Arguments as for gcn_sage3_step (labels may be NULL
 * without lp_mask); outputs, each optional (NULL) and fp32 device row-major:
 * H1, H2 [n x hidden] the ReLU outputs of layers 1 and 2, logits
 * [n x n_classes]. Asynchronous. */
gcn_status gcn_sage3_forward(const gcn_graph* g, const float* X, int64_t ldx, int64_t f_in,
                             int64_t hidden, int64_t n_classes, const float* const* params,
                             const int32_t* labels, const uint8_t* lp_mask, const float* E,
                             double eps, float* H1, int64_t ldh1, float* H2, int64_t ldh2,
                             float* logits, int64_t ldl, void* stream);

/* One training step (forward, loss, backward) of the 3-layer GraphSAGE model
 * of the evaluation (Section 8.1, Table 2), with optional masked label
 * propagation (Section 6.1 step 1, Lemma 2). Layer l (l = 1, 2, 3):
 *   Y = LayerNorm(H) (as gcn_layernorm_fwd), Z = A Y with the graph's values
 *   (after gcn_normalize_mean: the neighbour mean), O = Y W_self + Z W_neigh + b,
 *   H = relu(O) for l = 1, 2; the logits are O of layer 3. A layer whose output
 *   is narrower than its input evaluates Z W_neigh as A (Y W_neigh), so that
 *   its aggregations (forward and backward) gather the narrower rows; the two
 *   agree up to fp32 rounding. With hidden a multiple of 16 up to 256, the
 *   input gradient of such a layer and the LayerNorm backward of its input
 *   run as one pass (the same sums, in another order).
 * Loss: mean softmax cross-entropy over the rows that count (all rows, or
 * those with lp_mask = 0). Label propagation: rows with lp_mask = 1 get E[label]
 * added to their input features and are left out of the loss. Dropout is not
 * applied.
 *  g        square graph, aggregated as stored (A for the forward, A^T for the
 *           backward).
 *  X        fp32 device [n x f_in] (ldx); labels int32 [n] in [0, n_classes).
 *  params   host array of 9 device pointers, fp32 row-major:
 *           W_self1, W_neigh1 [f_in x hidden], b1 [hidden],
 *           W_self2, W_neigh2 [hidden x hidden], b2 [hidden],
 *           W_self3, W_neigh3 [hidden x n_classes], b3 [n_classes].
 *  grads    host array of 9 device pointers of the same shapes (outputs).
 *  lp_mask  uint8 device [n] or NULL; E fp32 [n_classes x f_in] and dE (output,
 *           same shape) are required with it.
 *  eps      LayerNorm epsilon; loss: device double, the mean loss.
 *  1 <= n_classes <= 64. Asynchronous; temporaries are stream-ordered
 *  (about 4 n (2 f_in + 3 (2 hidden + 4) + 4 hidden) bytes). The weight
 *  gradients of each layer run on a second, library-owned stream of the
 *  current device, forked from `stream` by an event and joined back to it
 *  before the call returns: all outputs are ordered on `stream`. */
gcn_status gcn_sage3_step(const gcn_graph* g, const float* X, int64_t ldx, int64_t f_in,
                          int64_t hidden, int64_t n_classes, const float* const* params,
                          const int32_t* labels, const uint8_t* lp_mask, const float* E,
                          double eps, float* const* grads, float* dE, double* loss,
                          void* stream);

/* ---- hybrid pre/post-aggregation (Algorithm 1, Sections 5.2 and 5.3) ---- */

/* Split the cut edges that a sending worker has into a receiving worker.
 * Sending a source node's row serves all of its cut edges (post-aggregation
 * on the receiver); sending the sender's partial sum for a destination node
 * serves all of that node's cut edges (pre-aggregation on the sender). The
 * split takes a minimum vertex cover of the bipartite remote graph (Eq. 1;
 * each connected component is solved separately by Hopcroft-Karp maximum
 * matching and Koenig's construction, in parallel host threads): an edge whose
 * source is in the cover is a post-aggregation edge, every other edge is a
 * pre-aggregation edge (its destination is then in the cover). The rows to
 * send are the cover's nodes, as many as a maximum matching has edges.
 * Host-side; every array is a host array.
 *  n_src, n_dst  sender-local source ids [0, n_src), receiver-local
 *                destination ids [0, n_dst); n_src + n_dst < 2^31.
 *  src, dst      int32 [n_edges]; repeated pairs are allowed (out of range
 *                -> GCN_ERANGE, nothing written).
 *  is_post       uint8 [n_edges] or NULL: 1 for post-, 0 for pre-aggregation.
 *  src_slot      int32 [n_src] or NULL: position of the source among the
 *                covered sources (their send-buffer row, in increasing id
 *                order), -1 if not covered.
 *  dst_slot      int32 [n_dst] or NULL: likewise for covered destinations
 *                (the row of the sender's partial-sum buffer).
 *  volume        int64 or NULL: rows to send = size of the cover.
 * Which minimum cover is returned when several exist is unspecified; its
 * size is not. Host memory: about 40 bytes per edge and node. */
gcn_status gcn_prepost_split(int64_t n_src, int64_t n_dst, int64_t n_edges, const int32_t* src,
                             const int32_t* dst, uint8_t* is_post, int32_t* src_slot,
                             int32_t* dst_slot, int64_t* volume);

/* Post-aggregation combine on the receiver (Section 5.2): add the received
 * partial sums to the rows they belong to, Y[idx[j], :] += P[j, :] for
 * j < n, in fp32. P [n x F] (ldp) and Y [n_y x F] (ldy) are fp32 device
 * arrays; idx is an int32 device array [n] of distinct row ids (the covered
 * destinations, e.g. those with dst_slot >= 0 in slot order). Rows whose idx
 * lies outside [0, n_y) are skipped, no error is reported for them; repeated
 * ids race. Asynchronous on `stream`. */
gcn_status gcn_add_rows(int64_t n, int64_t F, const float* P, int64_t ldp, const int32_t* idx,
                        int64_t n_y, float* Y, int64_t ldy, void* stream);

/* gcn_add_rows for partial sums that were quantized by their sender
 * (Section 6.1 steps 2-3 applied to the pre-aggregated rows of Section 5.2:
 * the sender quantizes them like any boundary row, e.g. with
 * gcn_layernorm_quantize without GCN_LAYERNORM):
 *   Y[idx[j], f] += fmaf((float)q[j, f], scale[j * ldp], zmin[j * ldp])
 * in fp32 (the dequantized value rounded once, then the add), j < n.
 *  bits  8: Q [n x ldq] uint8 codes, ldq >= F; 2: codes packed four per byte
 *        along the features (feature f in bits [2 (f % 4), 2 (f % 4) + 2) of
 *        byte f / 4), ldq >= (F + 3) / 4.
 *  zmin, scale  fp32 zero point and scale of row j at element j * ldp
 *        (ldp >= 1; ldp = 2 with scale == zmin + 1 reads the pairs
 *        gcn_layernorm_quantize writes).
 *  idx, n_y, Y, ldy  as for gcn_add_rows (distinct ids; ids outside
 *        [0, n_y) are skipped).
 * Other bit widths -> GCN_EINVAL. Asynchronous on `stream`. */
gcn_status gcn_add_rows_q(int64_t n, int64_t F, int bits, const uint8_t* Q, int64_t ldq,
                          const float* zmin, const float* scale, int64_t ldp, const int32_t* idx,
                          int64_t n_y, float* Y, int64_t ldy, void* stream);

/* ---- support calls ---------------------------------------------------- */

/* Release every device array of the graph (after synchronizing the device
 * work that uses it is the caller's job). NULL is ignored. */
void gcn_graph_free(gcn_graph* g);

/* Host outputs (any may be NULL): shape and stored-entry count. */
gcn_status gcn_graph_info(const gcn_graph* g, int64_t* n_rows, int64_t* n_cols, int64_t* nnz);

/* Copy the canonical arrays of A (which = 0) or A^T (which = 1) to HOST
 * memory: ptr [n_major + 1] (int64), idx [nnz] (int32 columns, increasing
 * within a row), val [nnz] (fp32). Any output may be NULL. Synchronizes. */
gcn_status gcn_graph_export(const gcn_graph* g, int which, int64_t* ptr, int32_t* idx, float* val,
                            void* stream);

/* Row-length classes the aggregation kernels use, for A (which = 0) or A^T
 * (which = 1). Writes up to `cap` records of 5 int64 each to host memory:
 * {first_len, last_len, rows, entries, entries with column >= halo_from},
 * last_len = -1 meaning unbounded (pass halo_from = -1 to skip the last
 * count, which is then 0). Returns the number of classes in *n_classes (10:
 * empty rows, 1, 2, 3-4, 5-8, 9-16, 17-32 entries, medium rows, rows cut into
 * fixed-length chunks, and rows cut at column-block boundaries, the last bin
 * empty when the plan blocks no row). Synchronizes `stream` when
 * halo_from >= 0.
 *
 * The plan's bounds can be set at build time through the environment:
 * GCN_MEDIUM_MAX (longest medium row, default 48 where rows are column-blocked,
 * else 256), GCN_CHUNK_LEN (entries per chunk, 2048), GCN_BLOCKED_MIN
 * (shortest column-blocked row, 49), GCN_COL_BLOCKS (column blocks, 64; 1
 * blocks nothing), GCN_SEGMENT_MIN (entries per segment a blocked row is cut
 * for, 24: about len / 24 segments, a power of two up to GCN_COL_BLOCKS; 0
 * cuts at every block), GCN_PIECE_MAX
 * (entries per blocked piece, 256) and GCN_BLOCK_MIN_COLS (fewest columns
 * for which rows are blocked, 2^20). Out-of-range values are ignored. */
gcn_status gcn_graph_bins(const gcn_graph* g, int which, int64_t halo_from, int64_t* records,
                          int cap, int* n_classes, void* stream);

/* Per-kernel device timing. While enabled, every kernel launch of the
 * library is bracketed by HIP events on its stream; gcn_profile_read
 * synchronizes those events and returns, per kernel name, the number of
 * launches and their summed duration in milliseconds (host arrays of `cap`
 * entries; names are static strings). Disabling clears the records. */
gcn_status gcn_profile_enable(int on);
gcn_status gcn_profile_read(const char** names, int64_t* launches, double* total_ms, int cap,
                            int* n_kernels);

/* Message describing the last failure on the calling thread ("" if none). */
const char* gcn_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* GCNAGG_H */
