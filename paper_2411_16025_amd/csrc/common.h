// Internal declarations shared by the library's translation units.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <cstdio>
#include <string>

#include "../../include/gcnagg.h"

namespace gcn {

constexpr uint64_t kMagic = 0x47434E4147473031ULL;  // "GCNAGG01"
constexpr uint64_t kFreed = 0xDEADDEADDEADDEADULL;

// One stored entry of a sparse matrix: column id and value side by side, so
// the aggregation loads both with one 8-byte access.
struct __align__(8) Ent {
  int32_t col;
  float val;
};

// Row-length classes (the binning that balances work across wavefronts; the
// bounds are in row_class in build.hip): 0 empty; 1 and 2 rows of exactly one
// and two entries; 3..6 rows of 3-4, 5-8, 9-16 and 17-32 entries; kMedium
// rows of 33 .. medium_max entries; kChunked longer rows, run one workgroup
// per chunk of at most chunk_len entries, or, from blocked_min entries on, as
// column-blocked pieces (see Plan). Classes 1 .. kMedium run one row per lane
// group.
constexpr int kNumClasses = 9;
constexpr int kClassEmpty = 0;
constexpr int kFirstShort = 1;
constexpr int kLastShort = 6;
constexpr int kMedium = 7;
constexpr int kChunked = 8;

struct Plan {
  int32_t* rows = nullptr;        // [n_major] row ids grouped by class (order: see build_plan)
  // first entry and length of each row of the classes 1 .. kMedium, in the
  // order of `rows` from class_off[1] (the row kernels read them with the
  // row id instead of the row pointer)
  int64_t* rbeg = nullptr;
  int32_t* rlen = nullptr;
  int64_t class_off[kNumClasses + 1] = {};  // host copy of the class boundaries in `rows`
  int64_t class_nnz[kNumClasses] = {};      // host: stored entries per class
  int64_t medium_max = 48;                  // longest row of the medium class (256 unblocked)
  int64_t chunk_len = 2048;                 // entries per chunk of a chunked row
  // chunk table for rows of the chunked class
  int64_t n_chunks = 0;
  int32_t* chunk_row = nullptr;   // [n_chunks]
  int64_t* chunk_beg = nullptr;   // [n_chunks] first entry
  int64_t* chunk_end = nullptr;   // [n_chunks] one past the last entry
  int32_t* chunk_part = nullptr;  // [n_chunks] partial-row slot, -1 = writes the output row
  // Column-blocked rows: the first n_blocked rows of the chunked class (those
  // of at least blocked_min entries) are cut where the column crosses a
  // multiple of block_width, and each segment into pieces of at most
  // piece_max entries. The pieces run ordered by column block, so the rows
  // the wavefronts in flight gather come from one column range and hub rows
  // are reused in cache; every piece writes a partial row (slots from
  // n_parts - n_pieces on, in entry order within each row).
  int64_t col_blocks = 64;
  int64_t blocked_min = 49;
  int64_t piece_max = 256;
  int64_t seg_min = 24;             // entries per segment aimed at (0: one per block)
  int64_t block_width = 0;
  int64_t n_blocked = 0;
  int64_t blocked_nnz = 0;          // host: stored entries of the blocked rows
  int64_t n_pieces = 0;
  int64_t* piece_beg = nullptr;     // [n_pieces] first entry, in launch order
  int32_t* piece_len = nullptr;     // [n_pieces] entries
  int32_t* piece_part = nullptr;    // [n_pieces] partial-row slot
  // rows summed from partial rows (multi-chunk rows, then the blocked rows)
  int64_t n_giant = 0;
  int64_t n_parts = 0;
  int32_t* giant_row = nullptr;       // [n_giant]
  int32_t* giant_part_off = nullptr;  // [n_giant + 1] first partial slot of each giant row
};

struct Mat {
  int64_t n_major = 0, n_minor = 0, nnz = 0;
  int64_t* ptr = nullptr;  // [n_major + 1]
  Ent* ent = nullptr;      // [nnz]
  Plan plan;
};

}  // namespace gcn

struct gcn_graph {
  uint64_t magic;
  int device;
  int64_t n_rows, n_cols;
  uint32_t flags;
  bool csc_shared;   // symmetric structure: csc aliases csr's ptr and plan
  bool csc_own_ent;  // ... but csc holds its own entries (mean values are not symmetric)
  bool normalized;
  int norm_mode;     // 0 none (values 1), 1 symmetric D^-1/2 (A+I) D^-1/2, 2 mean D^-1 A
  gcn::Mat csr;     // rows = destination nodes
  gcn::Mat csc;     // rows = source nodes (A^T)
};

namespace gcn {

// ---- error reporting -------------------------------------------------------
void set_error(const char* fmt, ...) __attribute__((format(printf, 1, 2)));
void clear_error();
gcn_status hip_fail(hipError_t e, const char* what, const char* file, int line);

#define GCN_HIP(call)                                                       \
  do {                                                                      \
    hipError_t e_ = (call);                                                 \
    if (e_ != hipSuccess) return ::gcn::hip_fail(e_, #call, __FILE__, __LINE__); \
  } while (0)

#define GCN_CHECK(expr)                        \
  do {                                         \
    gcn_status s_ = (expr);                    \
    if (s_ != GCN_OK) return s_;               \
  } while (0)

gcn_status dmalloc(void** p, size_t bytes, const char* what);
template <class T>
gcn_status dalloc(T** p, int64_t count, const char* what) {
  return dmalloc(reinterpret_cast<void**>(p), (size_t)(count > 0 ? count : 1) * sizeof(T), what);
}
void dfree(void* p);
// Stream-ordered temporaries (hipMallocAsync / hipFreeAsync on `stream`).
gcn_status tmalloc(void** p, size_t bytes, hipStream_t stream, const char* what);
template <class T>
gcn_status talloc(T** p, int64_t count, hipStream_t stream, const char* what) {
  return tmalloc(reinterpret_cast<void**>(p), (size_t)(count > 0 ? count : 1) * sizeof(T), stream,
                 what);
}
void tfree(void* p, hipStream_t stream);

// Work that may overlap the caller's stream runs on a second stream of the
// current device (non-blocking, default priority, created on first use and
// kept until the process ends). fork() makes the side stream wait for all
// work enqueued on `main` so far; join() makes `main` wait for all work
// enqueued on the side stream. The destructor joins, so on every return path
// the side work is ordered before whatever the caller enqueues next.
struct SideWork {
  hipStream_t main = nullptr, side = nullptr;
  hipEvent_t ev_fork = nullptr, ev_join = nullptr;
  bool pending = false;  // side work enqueued since the last join
  gcn_status init(hipStream_t m);
  gcn_status fork();
  gcn_status join();
  ~SideWork();
};

// Stream-ordered temporaries released when the scope ends, on every return
// path (error returns included).
struct TempScope {
  hipStream_t stream;
  void* ptrs[32];
  int n = 0;
  explicit TempScope(hipStream_t s) : stream(s) {}
  TempScope(const TempScope&) = delete;
  TempScope& operator=(const TempScope&) = delete;
  ~TempScope() {
    for (int i = n - 1; i >= 0; --i) tfree(ptrs[i], stream);
  }
  template <class T>
  gcn_status alloc(T** p, int64_t count, const char* what) {
    if (n == 32) {
      set_error("too many temporaries for %s", what);
      return GCN_ENOMEM;
    }
    GCN_CHECK(talloc(p, count, stream, what));
    ptrs[n++] = *p;
    return GCN_OK;
  }
};

gcn_status check_graph(const gcn_graph* g);

// ---- per-kernel profiling (see gcn_profile_enable) --------------------------
bool profiling();
struct ProfScope {
  const char* name;
  hipStream_t stream;
  hipEvent_t start = nullptr;
  ProfScope(const char* n, hipStream_t s);
  ~ProfScope();
};

// ---- device primitives (sort.hip) -------------------------------------------
// Stable LSD radix sort of n 64-bit keys on bits [0, bits); keys end up in
// *keys (buffers may be swapped; both must hold n keys).
gcn_status radix_sort_u64(uint64_t** keys, uint64_t** alt, int64_t n, int bits,
                          hipStream_t stream);
// Stable partition pass: sort by bits [lo_bit, lo_bit + 8) only.
gcn_status radix_pass_u64(const uint64_t* in, uint64_t* out, int64_t n, int shift,
                          hipStream_t stream);
// Exclusive scan of int64 values; out[n] receives the total. in == out allowed.
gcn_status scan_i64(const int64_t* in, int64_t* out, int64_t n, hipStream_t stream);

// ---- aggregation and dense operations (aggregate.hip, dense.hip) -------------
// Y = M X for fp32 X (M is a graph's CSR or CSC); relu clamps the result at 0.
gcn_status aggregate_f32(const Mat& m, const float* X, int64_t ldx, float* Y, int64_t ldy,
                         int64_t F, bool relu, hipStream_t stream);
// mask (optional, [M x N], ldm): C[i, j] = 0 where mask[i, j] <= 0 (NN and NT)
// C = A op(B); with mask, C = 0 where mask <= 0; with relu, C = max(C, 0).
gcn_status gemm_f32(int op, int64_t M, int64_t N, int64_t K, const float* A, int64_t lda,
                    const float* B, int64_t ldb, float* C, int64_t ldc, hipStream_t stream,
                    const float* mask = nullptr, int64_t ldm = 0, bool relu = false);
// Input gradient of a GraphSAGE layer whose output is narrower than its
// input, fused with the LayerNorm backward: dY = DG B^T (DG [n x K] with
// 16-byte aligned rows, B [F x K]), then dX = rstd (dY - mean(dY) - Y
// mean(dY Y)) where dx > 0 on entry (the ReLU output below), else 0.
bool sage_tf_bwd_fusable(int64_t F, int64_t K, const float* dg, int64_t ldg);
gcn_status sage_tf_bwd_fused(int64_t n, int64_t F, int64_t K, const float* dg, int64_t ldg,
                             const float* bw, int64_t ldb, const float* y, int64_t ldy,
                             const float* rstd, float* dx, int64_t ldx, hipStream_t stream);
// Forward of a GCN first layer that aggregates first: H1 = relu(P W1) and
// Z2 = H1 W2 in one pass over the rows. P [n x f_in] (ldp), H1 [n x hidden]
// (ldh, 16-byte aligned rows), W1 [f_in x hidden] (ldw1), W2 [hidden x C]
// (ldw2), Z2 [n x C] (ldz).
bool layer1_fwd_fusable(int64_t f_in, int64_t hidden, int64_t C, const float* P, int64_t ldp,
                        const float* H1, int64_t ldh);
gcn_status layer1_fwd_fused(int64_t n, int64_t f_in, int64_t hidden, int64_t C, const float* P,
                            int64_t ldp, const float* W1, int64_t ldw1, const float* W2,
                            int64_t ldw2, float* H1, int64_t ldh, float* Z2, int64_t ldz,
                            hipStream_t stream);
// Backward of a GCN first layer that aggregates first (H1 = relu(P W1),
// Z2 = H1 W2) in one pass over the rows: dW1 = P^T ((dZ2 W2^T) masked by
// H1 > 0) and dW2 = H1^T dZ2, both [rows x cols] with leading dimension cols.
// W2 is [hidden x C] with 16-byte aligned rows (ldw % 4 == 0), dZ2 likewise.
bool layer1_bwd_fusable(int64_t f_in, int64_t hidden, int64_t C, const float* dZ2, int64_t ldc,
                        const float* W2, int64_t ldw);
gcn_status layer1_bwd_fused(int64_t n, int64_t f_in, int64_t hidden, int64_t C, const float* P,
                            int64_t ldp, const float* H1, int64_t ldh, const float* dZ2,
                            int64_t ldc, const float* W2, int64_t ldw, float* dW1, float* dW2,
                            hipStream_t stream);
gcn_status relu_fwd(int64_t n, int64_t F, float* H, int64_t ld, hipStream_t stream);
gcn_status relu_bwd(int64_t n, int64_t F, const float* H, int64_t ldh, float* dH, int64_t ld,
                    hipStream_t stream);
gcn_status softmax_xent(int64_t n, int C, const float* z, int64_t ldz, const int32_t* y,
                        float* dz, int64_t ldd, double* loss, hipStream_t stream,
                        const uint8_t* skip = nullptr);
// Row LayerNorm without affine parameters (statistics in double); rstd
// (optional) receives 1 / sqrt(var + eps) per row.
gcn_status layernorm_fwd(int64_t n, int64_t F, const float* X, int64_t ldx, double eps, float* Y,
                         int64_t ldy, float* rstd, hipStream_t stream);
// dX = rstd * (g - mean(g) - Y * mean(g * Y)), g = G1 (+ G2), times (mask > 0)
// when mask is given (mask may be dX itself).
gcn_status layernorm_bwd(int64_t n, int64_t F, const float* Y, int64_t ldy, const float* rstd,
                         const float* G1, int64_t ld1, const float* G2, int64_t ld2,
                         const float* mask, int64_t ldm, float* dX, int64_t lddx,
                         hipStream_t stream);

// ---- plan building (build.hip) ----------------------------------------------
gcn_status build_plan(Mat& m, hipStream_t stream);
void free_mat(Mat& m, bool arrays);

inline int bits_for(uint64_t max_value) {
  int b = 0;
  while (b < 64 && (max_value >> b) != 0) ++b;
  return b;
}

inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

}  // namespace gcn
