// Device construction of the sparse operator: edge list -> sorted,
// deduplicated CSR of A (or A + I) and of A^T, degree normalization into
// A_hat = D~^-1/2 (A + I) D~^-1/2, and the row-length binning the
// aggregation kernels launch from.
//
// Paper: SuperGCN (arXiv 2411.16025) Section 4 -- "clustering and sorting":
// the index array is sorted so every destination row's source rows are
// contiguous, which lets the aggregation keep the destination row in
// registers. Section 4's 2D parallelism and FLOPS-based load balancing are
// realized by the row-length classes and the chunk table built here.

#include <algorithm>
#include <cmath>
#include <cstdlib>

#include "scan.h"

namespace gcn {

namespace {

constexpr int kThreads = 256;

inline unsigned grid_for(int64_t n, int per_block = kThreads) {
  return (unsigned)std::max<int64_t>(1, ceil_div(n, per_block));
}

// ---- keys ------------------------------------------------------------------

__global__ void k_edge_keys(const int32_t* __restrict__ src, const int32_t* __restrict__ dst,
                            int64_t n_edges, int64_t n_rows, int64_t n_cols, uint32_t flags,
                            int colbits, uint64_t sentinel, uint64_t* __restrict__ keys,
                            int* __restrict__ err) {
  const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= n_edges) return;
  const int64_t s = src[e], d = dst[e];
  uint64_t k0 = sentinel, k1 = sentinel;
  if (s < 0 || s >= n_cols || d < 0 || d >= n_rows) {
    atomicOr(err, 1);
  } else if (!((flags & GCN_ADD_SELF_LOOPS) && s == d)) {
    k0 = ((uint64_t)d << colbits) | (uint64_t)s;
    k1 = ((uint64_t)s << colbits) | (uint64_t)d;
  }
  keys[e] = k0;
  if (flags & GCN_SYMMETRIZE) keys[n_edges + e] = k1;
}

__global__ void k_diag_keys(int64_t n_diag, int colbits, uint64_t* __restrict__ keys) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n_diag) keys[i] = ((uint64_t)i << colbits) | (uint64_t)i;
}

// 1 for the first copy of each distinct valid key in a sorted array.
struct UniqueFlag {
  const uint64_t* keys;
  uint64_t sentinel;
  __device__ int64_t operator()(int64_t i) const {
    const uint64_t k = keys[i];
    return (k < sentinel && (i == 0 || keys[i - 1] != k)) ? 1 : 0;
  }
};

__global__ void k_compact(const uint64_t* __restrict__ keys, const int64_t* __restrict__ pos,
                          int64_t m, uint64_t sentinel, int colbits, Ent* __restrict__ ent,
                          int32_t* __restrict__ major) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= m) return;
  const uint64_t k = keys[i];
  if (k >= sentinel || (i > 0 && keys[i - 1] == k)) return;
  const int64_t p = pos[i];
  ent[p].col = (int32_t)(k & ((1ull << colbits) - 1ull));
  ent[p].val = 1.0f;
  major[p] = (int32_t)(k >> colbits);
}

// ptr[r] = first position p with major[p] >= r (major is sorted).
__global__ void k_row_ptr(const int32_t* __restrict__ major, int64_t nnz, int64_t n_major,
                          int64_t* __restrict__ ptr) {
  const int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (r > n_major) return;
  int64_t lo = 0, hi = nnz;
  while (lo < hi) {
    const int64_t mid = (lo + hi) >> 1;
    if ((int64_t)major[mid] < r)
      lo = mid + 1;
    else
      hi = mid;
  }
  ptr[r] = lo;
}

// keys of the transpose: (col << rowbits) | row for every stored entry
__global__ void k_transpose_keys(const Ent* __restrict__ ent, const int32_t* __restrict__ major,
                                 int64_t nnz, int rowbits, uint64_t* __restrict__ keys) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < nnz) keys[i] = ((uint64_t)(uint32_t)ent[i].col << rowbits) | (uint64_t)(uint32_t)major[i];
}

__global__ void k_unpack_sorted(const uint64_t* __restrict__ keys, int64_t nnz, int minorbits,
                                Ent* __restrict__ ent, int32_t* __restrict__ major) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= nnz) return;
  const uint64_t k = keys[i];
  ent[i].col = (int32_t)(k & ((1ull << minorbits) - 1ull));
  ent[i].val = 1.0f;
  major[i] = (int32_t)(k >> minorbits);
}

// ---- binning -----------------------------------------------------------------

__device__ inline int row_class(int64_t len, int64_t medium_max) {
  if (len == 0) return kClassEmpty;
  if (len == 1) return 1;
  if (len == 2) return 2;
  if (len <= 4) return 3;
  if (len <= 8) return 4;
  if (len <= 16) return 5;
  if (len <= 32) return 6;
  if (len <= medium_max) return kMedium;
  return kChunked;
}

// Sort key of a row: class in bits [60, 64), then, for the classes of 3 or
// more entries, decreasing length (kLenMask - min(len, kLenMask)) in bits
// [32, 60), then the row id. Rows a wavefront takes together then have about
// the same length, and long rows and full chunks start first.
constexpr uint64_t kLenMask = (1ull << 28) - 1;

__global__ void k_class_keys(const int64_t* __restrict__ ptr, int64_t n_major, int64_t medium_max,
                             uint64_t* __restrict__ keys) {
  const int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (r >= n_major) return;
  const int64_t len = ptr[r + 1] - ptr[r];
  const int c = row_class(len, medium_max);
  const uint64_t l = (uint64_t)len < kLenMask ? (uint64_t)len : kLenMask;
  const uint64_t lcode = c >= kFirstShort + 2 ? kLenMask - l : 0;
  keys[r] = ((uint64_t)c << 60) | (lcode << 32) | (uint64_t)r;
}

// per-class row and entry counts (integer sums, so the atomics are exact)
__global__ void k_class_count(const int64_t* __restrict__ ptr, int64_t n_major, int64_t medium_max,
                              unsigned long long* __restrict__ counts) {
  __shared__ unsigned long long rows[kNumClasses], ents[kNumClasses];
  if (threadIdx.x < kNumClasses) {
    rows[threadIdx.x] = 0;
    ents[threadIdx.x] = 0;
  }
  __syncthreads();
  const int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (r < n_major) {
    const int64_t len = ptr[r + 1] - ptr[r];
    const int c = row_class(len, medium_max);
    atomicAdd(&rows[c], 1ull);
    atomicAdd(&ents[c], (unsigned long long)len);
  }
  __syncthreads();
  if (threadIdx.x < kNumClasses) {
    atomicAdd(&counts[threadIdx.x], rows[threadIdx.x]);
    atomicAdd(&counts[kNumClasses + threadIdx.x], ents[threadIdx.x]);
  }
}

// first entry and length of each row of a run of `rows`
__global__ void k_row_begins(const int32_t* __restrict__ rows, int64_t n,
                             const int64_t* __restrict__ ptr, int64_t* __restrict__ beg,
                             int32_t* __restrict__ len) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const int64_t b = ptr[rows[i]];
  beg[i] = b;
  len[i] = (int32_t)(ptr[rows[i] + 1] - b);
}

__global__ void k_low32(const uint64_t* __restrict__ keys, int64_t n, int32_t* __restrict__ out) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) out[i] = (int32_t)(keys[i] & 0xFFFFFFFFull);
}

struct ChunkCount {
  const int32_t* rows;
  const int64_t* ptr;
  int64_t chunk_len;
  int giant_only;  // 0: chunks of every row; 1: chunks of rows with > 1 chunk; 2: 1 per giant row
  __device__ int64_t operator()(int64_t i) const {
    const int32_t r = rows[i];
    const int64_t c = (ptr[r + 1] - ptr[r] + chunk_len - 1) / chunk_len;
    if (giant_only == 0) return c;
    if (giant_only == 1) return c > 1 ? c : 0;
    return c > 1 ? 1 : 0;
  }
};

__global__ void k_chunks(const int32_t* __restrict__ rows, int64_t n, const int64_t* __restrict__ ptr,
                         int64_t chunk_len, const int64_t* __restrict__ chunk_off,
                         const int64_t* __restrict__ part_off, const int64_t* __restrict__ giant_idx,
                         int32_t* __restrict__ chunk_row, int64_t* __restrict__ chunk_beg,
                         int64_t* __restrict__ chunk_end, int32_t* __restrict__ chunk_part,
                         int32_t* __restrict__ giant_row,
                         int32_t* __restrict__ giant_part_off, int64_t n_giant) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const int32_t r = rows[i];
  const int64_t b = ptr[r], len = ptr[r + 1] - b;
  const int64_t nc = (len + chunk_len - 1) / chunk_len;
  const int64_t c0 = chunk_off[i];
  for (int64_t k = 0; k < nc; ++k) {
    chunk_row[c0 + k] = r;
    chunk_beg[c0 + k] = b + k * chunk_len;
    chunk_end[c0 + k] = b + ((k + 1) * chunk_len < len ? (k + 1) * chunk_len : len);
    chunk_part[c0 + k] = nc > 1 ? (int32_t)(part_off[i] + k) : -1;
  }
  if (nc > 1) {
    const int64_t gi = giant_idx[i];
    giant_row[gi] = r;
    giant_part_off[gi] = (int32_t)part_off[i];
  }
  if (i == n - 1) giant_part_off[n_giant] = (int32_t)part_off[n];
}

// ---- column-blocked pieces of the longest rows ----------------------------------

struct BlockedCount {  // 1 for a row of at least min_len entries
  const int32_t* rows;
  const int64_t* ptr;
  int64_t min_len;
  __device__ int64_t operator()(int64_t i) const {
    const int32_t r = rows[i];
    return ptr[r + 1] - ptr[r] >= min_len ? 1 : 0;
  }
};

// bnd[i * (B + 1) + k] = first entry of row rows[i] whose column is at least
// k * width (k = 0 .. B; the columns of a row increase).
__global__ void k_block_bounds(const int32_t* __restrict__ rows, int64_t n,
                               const int64_t* __restrict__ ptr, const Ent* __restrict__ ent,
                               int B, int64_t width, int64_t* __restrict__ bnd) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= n * (B + 1)) return;
  const int64_t i = t / (B + 1);
  const int k = (int)(t % (B + 1));
  const int32_t r = rows[i];
  int64_t lo = ptr[r], hi = ptr[r + 1];
  if (k == 0) {
    bnd[t] = lo;
    return;
  }
  if (k == B) {
    bnd[t] = hi;
    return;
  }
  const int64_t c = (int64_t)k * width;
  while (lo < hi) {
    const int64_t mid = lo + ((hi - lo) >> 1);
    if ((int64_t)ent[mid].col < c)
      lo = mid + 1;
    else
      hi = mid;
  }
  bnd[t] = lo;
}

struct RowLength {
  const int32_t* rows;
  const int64_t* ptr;
  __device__ int64_t operator()(int64_t i) const {
    const int32_t r = rows[i];
    return ptr[r + 1] - ptr[r];
  }
};

// Column blocks merged into one segment of a row of len entries: a row is
// cut into about len / seg_min segments (a power of two, at most B), each
// spanning ceil(B / segments) consecutive blocks; seg_min = 0 cuts every row
// at every block boundary.
__device__ inline int seg_span(int64_t len, int B, int64_t seg_min) {
  if (seg_min <= 0) return 1;
  const int64_t want = len / seg_min;
  int segs = 1;
  while (segs * 2 <= B && (int64_t)segs * 2 <= want) segs *= 2;
  return (B + segs - 1) / segs;
}

struct PieceCount {  // pieces of the segment starting at block t % B of row t / B
  const int64_t* bnd;
  int B;
  int64_t piece_max, seg_min;
  __device__ int64_t operator()(int64_t t) const {
    const int64_t* b = bnd + (t / B) * (B + 1);
    const int k = (int)(t % B);
    const int span = seg_span(b[B] - b[0], B, seg_min);
    if (k % span) return 0;
    const int e = k + span < B ? k + span : B;
    return (b[e] - b[k] + piece_max - 1) / piece_max;
  }
};

// Pieces in partial-slot order (row, segment, position): start, length and
// the launch sort key (the segment's middle block, then decreasing length,
// then slot). Block 0 of a row also records the row and its first partial
// slot.
__global__ void k_make_pieces(const int32_t* __restrict__ rows, int64_t n, int B,
                              int64_t piece_max, int64_t seg_min, const int64_t* __restrict__ bnd,
                              const int64_t* __restrict__ piece_off, int64_t part0,
                              int64_t* __restrict__ tbeg, int32_t* __restrict__ tlen,
                              uint64_t* __restrict__ keys, int32_t* __restrict__ giant_row,
                              int32_t* __restrict__ giant_part_off) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= n * B) return;
  const int64_t i = t / B;
  const int k = (int)(t % B);
  const int64_t* rb = bnd + i * (B + 1);
  const int span = seg_span(rb[B] - rb[0], B, seg_min);
  if (k % span == 0) {
    const int e = k + span < B ? k + span : B;
    const uint64_t mid = (uint64_t)(k + (e - k - 1) / 2);
    const int64_t s0 = rb[k], s1 = rb[e];
    int64_t j = piece_off[t];
    for (int64_t pos = s0; pos < s1; pos += piece_max, ++j) {
      const int64_t len = s1 - pos < piece_max ? s1 - pos : piece_max;
      tbeg[j] = pos;
      tlen[j] = (int32_t)len;
      keys[j] = (mid << 41) | ((uint64_t)(piece_max - len) << 32) | (uint64_t)j;
    }
  }
  if (k == 0) {
    giant_row[i] = rows[i];
    giant_part_off[i] = (int32_t)(part0 + piece_off[t]);
  }
  if (t == n * B - 1) giant_part_off[n] = (int32_t)(part0 + piece_off[n * B]);
}

// launch-order piece table from the sorted keys
__global__ void k_order_pieces(const uint64_t* __restrict__ keys, int64_t n,
                               const int64_t* __restrict__ tbeg, const int32_t* __restrict__ tlen,
                               int64_t part0, int64_t* __restrict__ pbeg,
                               int32_t* __restrict__ plen, int32_t* __restrict__ ppart) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= n) return;
  const int64_t j = (int64_t)(keys[t] & 0xFFFFFFFFull);
  pbeg[t] = tbeg[j];
  plen[t] = tlen[j];
  ppart[t] = (int32_t)(part0 + j);
}

// per-class count of entries whose column is >= halo_from
__global__ void k_class_halo(const int64_t* __restrict__ ptr, const Ent* __restrict__ ent,
                             int64_t n_major, int64_t medium_max, int64_t blocked_min,
                             int64_t halo_from, unsigned long long* __restrict__ counts) {
  __shared__ unsigned long long cnt[kNumClasses + 1];
  if (threadIdx.x < kNumClasses + 1) cnt[threadIdx.x] = 0;
  __syncthreads();
  const int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (r < n_major) {
    int64_t lo = ptr[r], hi = ptr[r + 1];
    const int64_t end = hi;
    int c = row_class(hi - lo, medium_max);
    if (c == kChunked && blocked_min > 0 && hi - lo >= blocked_min) c = kNumClasses;
    while (lo < hi) {  // first column >= halo_from
      const int64_t mid = (lo + hi) >> 1;
      if ((int64_t)ent[mid].col < halo_from)
        lo = mid + 1;
      else
        hi = mid;
    }
    if (end > lo) atomicAdd(&cnt[c], (unsigned long long)(end - lo));
  }
  __syncthreads();
  if (threadIdx.x < kNumClasses + 1 && cnt[threadIdx.x])
    atomicAdd(&counts[threadIdx.x], cnt[threadIdx.x]);
}

// ---- normalization -------------------------------------------------------------

// deg[v] = stored entries of row v other than (v, v)
__global__ void k_degrees(const int64_t* __restrict__ ptr, const Ent* __restrict__ ent,
                          int64_t n_major, int32_t* __restrict__ deg) {
  const int64_t v = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (v >= n_major) return;
  int64_t lo = ptr[v], hi = ptr[v + 1];
  const int64_t len = hi - lo;
  while (lo < hi) {  // columns are increasing: binary search for v
    const int64_t mid = (lo + hi) >> 1;
    if ((int64_t)ent[mid].col < v)
      lo = mid + 1;
    else
      hi = mid;
  }
  const bool has_self = lo < ptr[v + 1] && (int64_t)ent[lo].col == v;
  deg[v] = (int32_t)(len - (has_self ? 1 : 0));
}

__global__ void k_check_degrees(const int32_t* __restrict__ deg, int64_t n, int* __restrict__ err) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n && deg[i] < 0) atomicOr(err, 1);
}

constexpr int kNormPerThread = 16;
constexpr int64_t kNormTile = (int64_t)kThreads * kNormPerThread;

// last row r with ptr[r] <= k, searched in [lo, hi]
__device__ inline int64_t row_of(const int64_t* ptr, int64_t lo, int64_t hi, int64_t k) {
  while (lo < hi) {
    const int64_t mid = (lo + hi + 1) >> 1;
    if (ptr[mid] <= k)
      lo = mid;
    else
      hi = mid - 1;
  }
  return lo;
}

// val of entry (r, c) = fp32(1 / sqrt((deg_major[r] + 1) * (deg_minor[c] + 1))) in
// IEEE double
__global__ __launch_bounds__(kThreads) void k_normalize(const int64_t* __restrict__ ptr,
                                                        int64_t n_major, Ent* __restrict__ ent,
                                                        int64_t nnz,
                                                        const int32_t* __restrict__ deg_major,
                                                        const int32_t* __restrict__ deg_minor) {
  __shared__ int64_t r_lo, r_hi;
  const int64_t k0 = (int64_t)blockIdx.x * kNormTile;
  const int64_t k1 = std::min(nnz, k0 + kNormTile) - 1;
  if (threadIdx.x == 0) r_lo = row_of(ptr, 0, n_major - 1, k0);
  if (threadIdx.x == 1) r_hi = row_of(ptr, 0, n_major - 1, k1);
  __syncthreads();
  for (int j = 0; j < kNormPerThread; ++j) {
    const int64_t k = k0 + (int64_t)j * kThreads + threadIdx.x;
    if (k > k1) break;
    const int64_t r = row_of(ptr, r_lo, r_hi, k);
    const double dr = (double)deg_major[r] + 1.0;
    const double dc = (double)deg_minor[ent[k].col] + 1.0;
    ent[k].val = (float)(1.0 / sqrt(dr * dc));
  }
}

// val of entry k = fp32(1 / (stored entries of the row of A it belongs to)) in
// IEEE double: for A's CSR that row is the entry's major row, for the CSC it is
// the entry's minor index. a_ptr is A's row pointer.
__global__ __launch_bounds__(kThreads) void k_normalize_mean(const int64_t* __restrict__ ptr,
                                                             int64_t n_major,
                                                             Ent* __restrict__ ent, int64_t nnz,
                                                             const int64_t* __restrict__ a_ptr,
                                                             bool by_minor) {
  __shared__ int64_t r_lo, r_hi;
  const int64_t k0 = (int64_t)blockIdx.x * kNormTile;
  const int64_t k1 = std::min(nnz, k0 + kNormTile) - 1;
  if (!by_minor) {
    if (threadIdx.x == 0) r_lo = row_of(ptr, 0, n_major - 1, k0);
    if (threadIdx.x == 1) r_hi = row_of(ptr, 0, n_major - 1, k1);
    __syncthreads();
  }
  for (int j = 0; j < kNormPerThread; ++j) {
    const int64_t k = k0 + (int64_t)j * kThreads + threadIdx.x;
    if (k > k1) break;
    const int64_t r = by_minor ? (int64_t)ent[k].col : row_of(ptr, r_lo, r_hi, k);
    ent[k].val = (float)(1.0 / (double)(a_ptr[r + 1] - a_ptr[r]));
  }
}

// ---- export ----------------------------------------------------------------------

__global__ void k_split(const Ent* __restrict__ ent, int64_t nnz, int32_t* __restrict__ idx,
                        float* __restrict__ val) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= nnz) return;
  const Ent e = ent[i];
  if (idx) idx[i] = e.col;
  if (val) val[i] = e.val;
}

int64_t env_int(const char* name, int64_t dflt, int64_t lo, int64_t hi) {
  const char* s = std::getenv(name);
  if (!s || !*s) return dflt;
  const long long v = std::atoll(s);
  return (v < lo || v > hi) ? dflt : (int64_t)v;
}

// Sorted CSR from already-generated keys (sentinel-padded). Takes ownership
// of nothing; `major` receives the row id of every stored entry.
gcn_status keys_to_csr(uint64_t** keys, uint64_t** alt, int64_t m, int keybits, int colbits,
                       uint64_t sentinel, Mat& mat, int32_t** major, int64_t* nnz_host,
                       int* err_dev, int* err_host, hipStream_t stream) {
  GCN_CHECK(radix_sort_u64(keys, alt, m, keybits, stream));
  // positions of the distinct keys, written into the spare key buffer
  int64_t* pos = reinterpret_cast<int64_t*>(*alt);
  int64_t* scratch = nullptr;
  GCN_CHECK(talloc(&scratch, scan_scratch_elems(m), stream, "scan scratch"));
  gcn_status st = scan_functor(UniqueFlag{*keys, sentinel}, m, pos, scratch, stream);
  tfree(scratch, stream);
  GCN_CHECK(st);
  // one host synchronization: entry count and the id-range flag
  int64_t* pinned = nullptr;
  GCN_HIP(hipHostMalloc((void**)&pinned, 2 * sizeof(int64_t), hipHostMallocDefault));
  pinned[0] = pinned[1] = 0;
  hipError_t e1 = hipMemcpyAsync(&pinned[0], pos + m, sizeof(int64_t), hipMemcpyDeviceToHost, stream);
  hipError_t e2 = err_dev ? hipMemcpyAsync(&pinned[1], err_dev, sizeof(int), hipMemcpyDeviceToHost,
                                           stream)
                          : hipSuccess;
  hipError_t e3 = hipStreamSynchronize(stream);
  const int64_t nnz = pinned[0];
  const int errv = (int)pinned[1];
  (void)hipHostFree(pinned);
  if (e1 != hipSuccess) return hip_fail(e1, "hipMemcpyAsync(nnz)", __FILE__, __LINE__);
  if (e2 != hipSuccess) return hip_fail(e2, "hipMemcpyAsync(err)", __FILE__, __LINE__);
  if (e3 != hipSuccess) return hip_fail(e3, "hipStreamSynchronize", __FILE__, __LINE__);
  *err_host = errv;
  *nnz_host = nnz;
  if (errv) return GCN_OK;  // caller reports the range error
  mat.nnz = nnz;
  GCN_CHECK(dalloc(&mat.ent, nnz, "entries"));
  GCN_CHECK(dalloc(&mat.ptr, mat.n_major + 1, "row pointers"));
  GCN_CHECK(talloc(major, nnz, stream, "entry rows"));
  if (m > 0) {
    hipLaunchKernelGGL(k_compact, dim3(grid_for(m)), dim3(kThreads), 0, stream, *keys,
                       (const int64_t*)pos, m, sentinel, colbits, mat.ent, *major);
    GCN_HIP(hipGetLastError());
  }
  hipLaunchKernelGGL(k_row_ptr, dim3(grid_for(mat.n_major + 1)), dim3(kThreads), 0, stream,
                     (const int32_t*)*major, nnz, mat.n_major, mat.ptr);
  GCN_HIP(hipGetLastError());
  return GCN_OK;
}

// CSR of the transpose from the entries of a CSR (no duplicates, no padding).
gcn_status transpose_csr(const Mat& a, const int32_t* a_major, Mat& t, hipStream_t stream) {
  const int64_t nnz = a.nnz;
  t.nnz = nnz;
  const int rowbits = bits_for((uint64_t)(a.n_major > 0 ? a.n_major - 1 : 0));
  const int colbits = bits_for((uint64_t)(a.n_minor > 0 ? a.n_minor - 1 : 0));
  uint64_t *keys = nullptr, *alt = nullptr;
  int32_t* major = nullptr;
  gcn_status st = talloc(&keys, nnz, stream, "transpose keys");
  if (st == GCN_OK) st = talloc(&alt, nnz, stream, "transpose keys");
  if (st == GCN_OK) st = dalloc(&t.ent, nnz, "transpose entries");
  if (st == GCN_OK) st = dalloc(&t.ptr, t.n_major + 1, "transpose row pointers");
  if (st == GCN_OK) st = talloc(&major, nnz, stream, "transpose rows");
  if (st == GCN_OK && nnz > 0) {
    hipLaunchKernelGGL(k_transpose_keys, dim3(grid_for(nnz)), dim3(kThreads), 0, stream, a.ent,
                       a_major, nnz, rowbits, keys);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) st = hip_fail(e, "k_transpose_keys", __FILE__, __LINE__);
    if (st == GCN_OK) st = radix_sort_u64(&keys, &alt, nnz, rowbits + colbits, stream);
    if (st == GCN_OK) {
      hipLaunchKernelGGL(k_unpack_sorted, dim3(grid_for(nnz)), dim3(kThreads), 0, stream,
                         (const uint64_t*)keys, nnz, rowbits, t.ent, major);
      e = hipGetLastError();
      if (e != hipSuccess) st = hip_fail(e, "k_unpack_sorted", __FILE__, __LINE__);
    }
  }
  if (st == GCN_OK) {
    hipLaunchKernelGGL(k_row_ptr, dim3(grid_for(t.n_major + 1)), dim3(kThreads), 0, stream,
                       (const int32_t*)major, nnz, t.n_major, t.ptr);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) st = hip_fail(e, "k_row_ptr", __FILE__, __LINE__);
  }
  tfree(major, stream);
  tfree(alt, stream);
  tfree(keys, stream);
  return st;
}

}  // namespace

// ---- plan --------------------------------------------------------------------------

gcn_status build_plan(Mat& m, hipStream_t stream) {
  Plan& p = m.plan;
  TempScope tmp(stream);
  p.col_blocks = env_int("GCN_COL_BLOCKS", 64, 1, 256);
  const int64_t block_min_cols = env_int("GCN_BLOCK_MIN_COLS", 1 << 20, 0, 1ll << 40);
  const bool blocking = p.col_blocks > 1 && m.n_minor >= block_min_cols;
  // with column blocking, rows past 48 entries gain from it; without, rows up
  // to 256 entries run fastest one per lane group
  p.medium_max = env_int("GCN_MEDIUM_MAX", blocking ? 48 : 256, 32, 1 << 20);
  p.chunk_len = env_int("GCN_CHUNK_LEN", 2048, 64, 1 << 24);
  if (p.chunk_len < p.medium_max) p.chunk_len = p.medium_max;
  p.blocked_min = env_int("GCN_BLOCKED_MIN", 49, 1, (int64_t)kLenMask);
  if (p.blocked_min <= p.medium_max) p.blocked_min = p.medium_max + 1;
  p.piece_max = env_int("GCN_PIECE_MAX", 256, 16, 511);
  p.seg_min = env_int("GCN_SEGMENT_MIN", 24, 0, 1 << 20);
  // a row cut into one segment would only pay for its partial row
  if (p.blocked_min < 2 * p.seg_min) p.blocked_min = 2 * p.seg_min;
  const int64_t n = m.n_major;
  uint64_t *keys = nullptr, *sorted = nullptr;
  unsigned long long* counts = nullptr;
  GCN_CHECK(tmp.alloc(&keys, n, "class keys"));
  GCN_CHECK(tmp.alloc(&sorted, n, "class keys"));
  GCN_CHECK(tmp.alloc(&counts, 2 * kNumClasses, "class counts"));
  GCN_CHECK(dalloc(&p.rows, n, "class rows"));
  GCN_HIP(hipMemsetAsync(counts, 0, 2 * kNumClasses * sizeof(unsigned long long), stream));
  hipLaunchKernelGGL(k_class_keys, dim3(grid_for(n)), dim3(kThreads), 0, stream, m.ptr, n,
                     p.medium_max, keys);
  GCN_HIP(hipGetLastError());
  hipLaunchKernelGGL(k_class_count, dim3(grid_for(n)), dim3(kThreads), 0, stream, m.ptr, n,
                     p.medium_max, counts);
  GCN_HIP(hipGetLastError());
  // four stable 8-bit passes over bits [32, 64): by length code, then by class
  GCN_CHECK(radix_pass_u64(keys, sorted, n, 32, stream));
  GCN_CHECK(radix_pass_u64(sorted, keys, n, 40, stream));
  GCN_CHECK(radix_pass_u64(keys, sorted, n, 48, stream));
  GCN_CHECK(radix_pass_u64(sorted, keys, n, 56, stream));
  hipLaunchKernelGGL(k_low32, dim3(grid_for(n)), dim3(kThreads), 0, stream,
                     (const uint64_t*)keys, n, p.rows);
  GCN_HIP(hipGetLastError());
  unsigned long long host_counts[2 * kNumClasses];
  GCN_HIP(hipMemcpyAsync(host_counts, counts, sizeof(host_counts), hipMemcpyDeviceToHost, stream));
  GCN_HIP(hipStreamSynchronize(stream));
  p.class_off[0] = 0;
  for (int c = 0; c < kNumClasses; ++c) {
    p.class_off[c + 1] = p.class_off[c] + (int64_t)host_counts[c];
    p.class_nnz[c] = (int64_t)host_counts[kNumClasses + c];
  }
  // rows up to the medium class read their start and length from here (one
  // load fewer in their chain of dependent loads)
  const int64_t n_rowk = p.class_off[kMedium + 1] - p.class_off[kFirstShort];
  if (n_rowk > 0) {
    GCN_CHECK(dalloc(&p.rbeg, n_rowk, "row starts"));
    GCN_CHECK(dalloc(&p.rlen, n_rowk, "row lengths"));
    hipLaunchKernelGGL(k_row_begins, dim3(grid_for(n_rowk)), dim3(kThreads), 0, stream,
                       (const int32_t*)(p.rows + p.class_off[kFirstShort]), n_rowk,
                       (const int64_t*)m.ptr, p.rbeg, p.rlen);
    GCN_HIP(hipGetLastError());
  }
  // chunked class: the longest rows (a prefix, the class being ordered by
  // decreasing length) become column-blocked pieces when the matrix has
  // enough columns for the gathered rows to outgrow the caches; the others
  // get the chunk table
  const int64_t nc_rows = p.class_off[kChunked + 1] - p.class_off[kChunked];
  p.n_chunks = p.n_giant = p.n_parts = 0;
  p.n_blocked = p.blocked_nnz = p.n_pieces = 0;
  if (nc_rows == 0) return GCN_OK;
  const int32_t* crow = p.rows + p.class_off[kChunked];
  const int B = (int)p.col_blocks;
  p.block_width = blocking ? ceil_div(m.n_minor, (int64_t)B) : 0;
  int64_t* scratch = nullptr;
  GCN_CHECK(tmp.alloc(&scratch, scan_scratch_elems(nc_rows), "scan scratch"));
  if (blocking) {
    int64_t* flag_off = nullptr;
    GCN_CHECK(tmp.alloc(&flag_off, nc_rows + 1, "blocked-row scan"));
    GCN_CHECK(scan_functor(BlockedCount{crow, m.ptr, p.blocked_min}, nc_rows, flag_off, scratch,
                           stream));
    GCN_HIP(hipMemcpyAsync(&p.n_blocked, flag_off + nc_rows, 8, hipMemcpyDeviceToHost, stream));
    GCN_HIP(hipStreamSynchronize(stream));
  }
  const int64_t nb = p.n_blocked;
  const int32_t* chrow = crow + nb;  // rows of the chunk table
  const int64_t nch = nc_rows - nb;
  int64_t *chunk_off = nullptr, *part_off = nullptr, *giant_idx = nullptr;
  int64_t *bnd = nullptr, *piece_off = nullptr, *pscratch = nullptr, *len_off = nullptr;
  int64_t tot[5] = {0, 0, 0, 0, 0};
  if (nch > 0) {
    GCN_CHECK(tmp.alloc(&chunk_off, nch + 1, "chunk offsets"));
    GCN_CHECK(tmp.alloc(&part_off, nch + 1, "partial offsets"));
    GCN_CHECK(tmp.alloc(&giant_idx, nch + 1, "giant index"));
    GCN_CHECK(scan_functor(ChunkCount{chrow, m.ptr, p.chunk_len, 0}, nch, chunk_off, scratch,
                           stream));
    GCN_CHECK(scan_functor(ChunkCount{chrow, m.ptr, p.chunk_len, 1}, nch, part_off, scratch,
                           stream));
    GCN_CHECK(scan_functor(ChunkCount{chrow, m.ptr, p.chunk_len, 2}, nch, giant_idx, scratch,
                           stream));
    GCN_HIP(hipMemcpyAsync(&tot[0], chunk_off + nch, 8, hipMemcpyDeviceToHost, stream));
    GCN_HIP(hipMemcpyAsync(&tot[1], part_off + nch, 8, hipMemcpyDeviceToHost, stream));
    GCN_HIP(hipMemcpyAsync(&tot[2], giant_idx + nch, 8, hipMemcpyDeviceToHost, stream));
  }
  if (nb > 0) {
    GCN_CHECK(tmp.alloc(&bnd, nb * (B + 1), "block bounds"));
    GCN_CHECK(tmp.alloc(&piece_off, nb * B + 1, "piece offsets"));
    GCN_CHECK(tmp.alloc(&pscratch, scan_scratch_elems(nb * B), "scan scratch"));
    hipLaunchKernelGGL(k_block_bounds, dim3(grid_for(nb * (B + 1))), dim3(kThreads), 0, stream,
                       crow, nb, (const int64_t*)m.ptr, (const Ent*)m.ent, B, p.block_width, bnd);
    GCN_HIP(hipGetLastError());
    GCN_CHECK(scan_functor(PieceCount{bnd, B, p.piece_max, p.seg_min}, nb * B, piece_off, pscratch,
                           stream));
    GCN_HIP(hipMemcpyAsync(&tot[3], piece_off + nb * B, 8, hipMemcpyDeviceToHost, stream));
    // entries of the blocked rows
    GCN_CHECK(tmp.alloc(&len_off, nb + 1, "blocked entry scan"));
    GCN_CHECK(scan_functor(RowLength{crow, m.ptr}, nb, len_off, pscratch, stream));
    GCN_HIP(hipMemcpyAsync(&tot[4], len_off + nb, 8, hipMemcpyDeviceToHost, stream));
  }
  GCN_HIP(hipStreamSynchronize(stream));
  p.n_chunks = tot[0];
  const int64_t n_cparts = tot[1], n_cgiant = tot[2];
  p.n_pieces = tot[3];
  p.blocked_nnz = tot[4];
  p.n_parts = n_cparts + p.n_pieces;
  p.n_giant = n_cgiant + nb;
  if (p.n_parts >= (1ll << 31)) {
    set_error("too many partial rows (%lld)", (long long)p.n_parts);
    return GCN_ERANGE;
  }
  GCN_CHECK(dalloc(&p.giant_row, p.n_giant, "giant rows"));
  GCN_CHECK(dalloc(&p.giant_part_off, p.n_giant + 1, "giant partial offsets"));
  if (nch > 0) {
    GCN_CHECK(dalloc(&p.chunk_row, p.n_chunks, "chunk rows"));
    GCN_CHECK(dalloc(&p.chunk_beg, p.n_chunks, "chunk starts"));
    GCN_CHECK(dalloc(&p.chunk_end, p.n_chunks, "chunk ends"));
    GCN_CHECK(dalloc(&p.chunk_part, p.n_chunks, "chunk partial slots"));
    hipLaunchKernelGGL(k_chunks, dim3(grid_for(nch)), dim3(kThreads), 0, stream, chrow, nch,
                       m.ptr, p.chunk_len, (const int64_t*)chunk_off, (const int64_t*)part_off,
                       (const int64_t*)giant_idx, p.chunk_row, p.chunk_beg, p.chunk_end,
                       p.chunk_part, p.giant_row, p.giant_part_off, n_cgiant);
    GCN_HIP(hipGetLastError());
  }
  if (nb > 0) {
    int64_t* tbeg = nullptr;
    int32_t* tlen = nullptr;
    uint64_t *keys = nullptr, *alt = nullptr;
    GCN_CHECK(tmp.alloc(&tbeg, p.n_pieces, "piece starts"));
    GCN_CHECK(tmp.alloc(&tlen, p.n_pieces, "piece lengths"));
    GCN_CHECK(tmp.alloc(&keys, p.n_pieces, "piece keys"));
    GCN_CHECK(tmp.alloc(&alt, p.n_pieces, "piece keys"));
    hipLaunchKernelGGL(k_make_pieces, dim3(grid_for(nb * B)), dim3(kThreads), 0, stream, crow,
                       nb, B, p.piece_max, p.seg_min, (const int64_t*)bnd,
                       (const int64_t*)piece_off,
                       n_cparts, tbeg, tlen, keys, p.giant_row + n_cgiant,
                       p.giant_part_off + n_cgiant);
    GCN_HIP(hipGetLastError());
    // stable passes over bits [32, 56): decreasing length, then block
    GCN_CHECK(radix_pass_u64(keys, alt, p.n_pieces, 32, stream));
    GCN_CHECK(radix_pass_u64(alt, keys, p.n_pieces, 40, stream));
    GCN_CHECK(radix_pass_u64(keys, alt, p.n_pieces, 48, stream));
    GCN_CHECK(dalloc(&p.piece_beg, p.n_pieces, "piece starts"));
    GCN_CHECK(dalloc(&p.piece_len, p.n_pieces, "piece lengths"));
    GCN_CHECK(dalloc(&p.piece_part, p.n_pieces, "piece partial slots"));
    hipLaunchKernelGGL(k_order_pieces, dim3(grid_for(p.n_pieces)), dim3(kThreads), 0, stream,
                       (const uint64_t*)alt, p.n_pieces, (const int64_t*)tbeg,
                       (const int32_t*)tlen, n_cparts, p.piece_beg, p.piece_len, p.piece_part);
    GCN_HIP(hipGetLastError());
  }
  return GCN_OK;
}

void free_mat(Mat& m, bool arrays) {
  Plan& p = m.plan;
  dfree(p.rows);
  dfree(p.rbeg);
  dfree(p.rlen);
  dfree(p.chunk_row);
  dfree(p.chunk_beg);
  dfree(p.chunk_end);
  dfree(p.chunk_part);
  dfree(p.giant_row);
  dfree(p.giant_part_off);
  dfree(p.piece_beg);
  dfree(p.piece_len);
  dfree(p.piece_part);
  p = Plan();
  if (arrays) {
    dfree(m.ptr);
    dfree(m.ent);
  }
  m.ptr = nullptr;
  m.ent = nullptr;
}

}  // namespace gcn

using namespace gcn;

namespace {

void destroy(gcn_graph* g) {
  if (!g) return;
  if (!g->csc_shared) free_mat(g->csc, true);
  if (g->csc_shared && g->csc_own_ent) dfree(g->csc.ent);
  free_mat(g->csr, true);
  g->magic = kFreed;
  delete g;
}

gcn_status build_impl(int64_t n_rows, int64_t n_cols, int64_t n_edges, const int32_t* src,
                      const int32_t* dst, uint32_t flags, hipStream_t stream, gcn_graph* g) {
  const int64_t n_diag = (flags & GCN_ADD_SELF_LOOPS) ? std::min(n_rows, n_cols) : 0;
  const int64_t m = n_edges * ((flags & GCN_SYMMETRIZE) ? 2 : 1) + n_diag;
  const int colbits = bits_for((uint64_t)(n_cols - 1));
  const int rowbits = bits_for((uint64_t)n_rows);  // room for the sentinel row n_rows
  const uint64_t sentinel = (uint64_t)n_rows << colbits;
  g->csr.n_major = n_rows;
  g->csr.n_minor = n_cols;
  g->csc.n_major = n_cols;
  g->csc.n_minor = n_rows;

  uint64_t *keys = nullptr, *alt = nullptr;
  int* err = nullptr;
  int32_t* major = nullptr;
  gcn_status st = talloc(&keys, m + 1, stream, "edge keys");
  if (st == GCN_OK) st = talloc(&alt, m + 1, stream, "edge keys");
  if (st == GCN_OK) st = talloc(&err, 1, stream, "error flag");
  if (st == GCN_OK) {
    hipError_t e = hipMemsetAsync(err, 0, sizeof(int), stream);
    if (e != hipSuccess) st = hip_fail(e, "hipMemsetAsync", __FILE__, __LINE__);
  }
  if (st == GCN_OK && n_edges > 0) {
    ProfScope ps("edge_keys", stream);
    hipLaunchKernelGGL(k_edge_keys, dim3(grid_for(n_edges)), dim3(kThreads), 0, stream, src, dst,
                       n_edges, n_rows, n_cols, flags, colbits, sentinel, keys, err);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) st = hip_fail(e, "k_edge_keys", __FILE__, __LINE__);
  }
  if (st == GCN_OK && n_diag > 0) {
    hipLaunchKernelGGL(k_diag_keys, dim3(grid_for(n_diag)), dim3(kThreads), 0, stream, n_diag,
                       colbits, keys + (m - n_diag));
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) st = hip_fail(e, "k_diag_keys", __FILE__, __LINE__);
  }
  int64_t nnz = 0;
  int err_host = 0;
  if (st == GCN_OK)
    st = keys_to_csr(&keys, &alt, m, rowbits + colbits, colbits, sentinel, g->csr, &major, &nnz,
                     err, &err_host, stream);
  tfree(alt, stream);
  tfree(keys, stream);
  tfree(err, stream);
  if (st == GCN_OK && err_host) {
    set_error("edge list holds a vertex id outside [0, n_cols) for src or [0, n_rows) for dst");
    st = GCN_ERANGE;
  }
  if (st == GCN_OK) {
    if (flags & GCN_SYMMETRIZE) {
      g->csc_shared = true;
      g->csc = g->csr;  // arrays shared; plan rebuilt below is shared too
    } else {
      g->csc_shared = false;
      st = transpose_csr(g->csr, major, g->csc, stream);
    }
  }
  tfree(major, stream);
  if (st == GCN_OK) st = build_plan(g->csr, stream);
  if (st == GCN_OK) {
    if (g->csc_shared)
      g->csc = g->csr;
    else
      st = build_plan(g->csc, stream);
  }
  if (st == GCN_OK) {
    hipError_t e = hipStreamSynchronize(stream);
    if (e != hipSuccess) st = hip_fail(e, "hipStreamSynchronize", __FILE__, __LINE__);
  }
  return st;
}

}  // namespace

extern "C" gcn_status gcn_build_csr(int64_t n_rows, int64_t n_cols, int64_t n_edges,
                                    const int32_t* src, const int32_t* dst, uint32_t flags,
                                    void* stream, gcn_graph** out) {
  clear_error();
  if (!out) {
    set_error("out is NULL");
    return GCN_EINVAL;
  }
  *out = nullptr;
  if (n_rows <= 0 || n_cols <= 0) {
    set_error("n_rows and n_cols must be positive (got %lld, %lld)", (long long)n_rows,
              (long long)n_cols);
    return GCN_EINVAL;
  }
  if (n_rows >= (1ll << 31) || n_cols >= (1ll << 31)) {
    set_error("n_rows and n_cols must be below 2^31 (ids are int32)");
    return GCN_ERANGE;
  }
  if (n_edges < 0) {
    set_error("n_edges must be >= 0");
    return GCN_EINVAL;
  }
  if (n_edges > 0 && (!src || !dst)) {
    set_error("src and dst must be non-NULL when n_edges > 0");
    return GCN_EINVAL;
  }
  if (flags & ~(uint32_t)(GCN_SYMMETRIZE | GCN_ADD_SELF_LOOPS)) {
    set_error("unknown build flag bits 0x%x", flags);
    return GCN_EINVAL;
  }
  if ((flags & GCN_SYMMETRIZE) && n_rows != n_cols) {
    set_error("GCN_SYMMETRIZE needs a square graph");
    return GCN_EINVAL;
  }
  if (n_edges > (1ll << 40)) {
    set_error("n_edges too large");
    return GCN_ERANGE;
  }
  int dev = 0;
  GCN_HIP(hipGetDevice(&dev));
  gcn_graph* g = new (std::nothrow) gcn_graph();
  if (!g) {
    set_error("host allocation failed");
    return GCN_ENOMEM;
  }
  g->magic = kMagic;
  g->device = dev;
  g->n_rows = n_rows;
  g->n_cols = n_cols;
  g->flags = flags;
  g->normalized = false;
  g->norm_mode = 0;
  g->csc_own_ent = false;
  g->csc_shared = false;
  gcn_status st = build_impl(n_rows, n_cols, n_edges, src, dst, flags, (hipStream_t)stream, g);
  if (st != GCN_OK) {
    (void)hipStreamSynchronize((hipStream_t)stream);
    destroy(g);
    return st;
  }
  *out = g;
  return GCN_OK;
}

extern "C" void gcn_graph_free(gcn_graph* g) {
  if (!g || g->magic != kMagic) return;
  destroy(g);
}

extern "C" gcn_status gcn_graph_info(const gcn_graph* g, int64_t* n_rows, int64_t* n_cols,
                                     int64_t* nnz) {
  clear_error();
  GCN_CHECK(check_graph(g));
  if (n_rows) *n_rows = g->n_rows;
  if (n_cols) *n_cols = g->n_cols;
  if (nnz) *nnz = g->csr.nnz;
  return GCN_OK;
}

namespace {

// 1 if any of deg[0, n) is negative (synchronizes the stream)
gcn_status check_degrees(const int32_t* deg, int64_t n, hipStream_t stream) {
  if (n == 0) return GCN_OK;
  int* err = nullptr;
  GCN_CHECK(talloc(&err, 1, stream, "error flag"));
  int host_err = 0;
  hipError_t e = hipMemsetAsync(err, 0, sizeof(int), stream);
  if (e == hipSuccess) {
    hipLaunchKernelGGL(k_check_degrees, dim3(grid_for(n)), dim3(kThreads), 0, stream, deg, n, err);
    e = hipGetLastError();
  }
  if (e == hipSuccess) e = hipMemcpyAsync(&host_err, err, sizeof(int), hipMemcpyDeviceToHost, stream);
  if (e == hipSuccess) e = hipStreamSynchronize(stream);
  tfree(err, stream);
  if (e != hipSuccess) return hip_fail(e, "degree check", __FILE__, __LINE__);
  if (host_err) {
    set_error("supplied degrees must be >= 0");
    return GCN_EINVAL;
  }
  return GCN_OK;
}

// A symmetric graph's transpose shares the structure and, until now, the
// entries of A; give it entries of its own (8 bytes per entry) for values
// that are not symmetric.
gcn_status own_csc_entries(gcn_graph* g, hipStream_t stream) {
  if (!g->csc_shared || g->csc_own_ent) return GCN_OK;
  const int64_t nnz = g->csr.nnz;
  Ent* e = nullptr;
  GCN_CHECK(dalloc(&e, nnz, "transpose entries"));
  hipError_t err = nnz > 0 ? hipMemcpyAsync(e, g->csr.ent, nnz * sizeof(Ent),
                                            hipMemcpyDeviceToDevice, stream)
                           : hipSuccess;
  if (err != hipSuccess) {
    dfree(e);
    return hip_fail(err, "hipMemcpyAsync(transpose entries)", __FILE__, __LINE__);
  }
  g->csc.ent = e;
  g->csc_own_ent = true;
  return GCN_OK;
}

// values of A from row degrees and column degrees; A^T takes them swapped.
// Entry (r, c) of A gets f(deg_rows[r], deg_cols[c]); entry (c, r) of A^T
// the same value. With shared entries (a symmetric graph) entry (c, r) of
// A^T is entry (c, r) of A, f(deg_rows[c], deg_cols[r]): equal for every
// entry only when the two arrays are the same, so different arrays give the
// transpose entries of its own first.
gcn_status normalize_with(gcn_graph* g, const int32_t* deg_rows, const int32_t* deg_cols,
                          hipStream_t stream) {
  if (deg_rows != deg_cols) GCN_CHECK(own_csc_entries(g, stream));
  for (int which = 0; which < 2; ++which) {
    if (which == 1 && g->csc_shared && !g->csc_own_ent) break;
    Mat& m = which ? g->csc : g->csr;
    if (m.nnz == 0) continue;
    ProfScope ps("normalize", stream);
    hipLaunchKernelGGL(k_normalize, dim3(grid_for(m.nnz, (int)kNormTile)), dim3(kThreads), 0,
                       stream, (const int64_t*)m.ptr, m.n_major, m.ent, m.nnz,
                       which ? deg_cols : deg_rows, which ? deg_rows : deg_cols);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return hip_fail(e, "k_normalize", __FILE__, __LINE__);
  }
  g->normalized = true;
  g->norm_mode = 1;
  return GCN_OK;
}

}  // namespace

extern "C" gcn_status gcn_normalize(gcn_graph* g, const int32_t* deg, void* stream_) {
  clear_error();
  GCN_CHECK(check_graph(g));
  hipStream_t stream = (hipStream_t)stream_;
  if (!deg && g->n_rows != g->n_cols) {
    set_error("a rectangular graph needs a supplied degree array");
    return GCN_EINVAL;
  }
  if (deg) {
    GCN_CHECK(check_degrees(deg, std::max(g->n_rows, g->n_cols), stream));
    return normalize_with(g, deg, deg, stream);
  }
  int32_t* own = nullptr;
  GCN_CHECK(talloc(&own, g->n_rows, stream, "degrees"));
  hipLaunchKernelGGL(k_degrees, dim3(grid_for(g->n_rows)), dim3(kThreads), 0, stream, g->csr.ptr,
                     (const Ent*)g->csr.ent, g->n_rows, own);
  hipError_t e = hipGetLastError();
  gcn_status st = e != hipSuccess ? hip_fail(e, "k_degrees", __FILE__, __LINE__)
                                  : normalize_with(g, own, own, stream);
  tfree(own, stream);
  return st;
}

extern "C" gcn_status gcn_normalize_mean(gcn_graph* g, void* stream_) {
  clear_error();
  GCN_CHECK(check_graph(g));
  hipStream_t stream = (hipStream_t)stream_;
  // the transpose keeps the shared structure but needs values of its own
  GCN_CHECK(own_csc_entries(g, stream));
  for (int which = 0; which < 2; ++which) {
    Mat& m = which ? g->csc : g->csr;
    if (m.nnz == 0) continue;
    ProfScope ps("normalize", stream);
    hipLaunchKernelGGL(k_normalize_mean, dim3(grid_for(m.nnz, (int)kNormTile)), dim3(kThreads), 0,
                       stream, (const int64_t*)m.ptr, m.n_major, m.ent, m.nnz,
                       (const int64_t*)g->csr.ptr, which == 1);
    GCN_HIP(hipGetLastError());
  }
  g->normalized = true;
  g->norm_mode = 2;
  return GCN_OK;
}

extern "C" gcn_status gcn_normalize_rc(gcn_graph* g, const int32_t* deg_rows,
                                       const int32_t* deg_cols, void* stream_) {
  clear_error();
  GCN_CHECK(check_graph(g));
  hipStream_t stream = (hipStream_t)stream_;
  if (!deg_rows || !deg_cols) {
    set_error("deg_rows and deg_cols must not be NULL");
    return GCN_EINVAL;
  }
  GCN_CHECK(check_degrees(deg_rows, g->n_rows, stream));
  GCN_CHECK(check_degrees(deg_cols, g->n_cols, stream));
  return normalize_with(g, deg_rows, deg_cols, stream);
}

extern "C" gcn_status gcn_graph_export(const gcn_graph* g, int which, int64_t* ptr, int32_t* idx,
                                       float* val, void* stream_) {
  clear_error();
  GCN_CHECK(check_graph(g));
  if (which != 0 && which != 1) {
    set_error("which must be 0 (A) or 1 (A^T)");
    return GCN_EINVAL;
  }
  hipStream_t stream = (hipStream_t)stream_;
  const Mat& m = which ? g->csc : g->csr;
  if (ptr)
    GCN_HIP(hipMemcpyAsync(ptr, m.ptr, (m.n_major + 1) * sizeof(int64_t), hipMemcpyDeviceToHost,
                           stream));
  if ((idx || val) && m.nnz > 0) {
    TempScope tmp(stream);
    int32_t* didx = nullptr;
    float* dval = nullptr;
    GCN_CHECK(tmp.alloc(&didx, m.nnz, "export columns"));
    GCN_CHECK(tmp.alloc(&dval, m.nnz, "export values"));
    hipLaunchKernelGGL(k_split, dim3(grid_for(m.nnz)), dim3(kThreads), 0, stream,
                       (const Ent*)m.ent, m.nnz, didx, dval);
    GCN_HIP(hipGetLastError());
    if (idx)
      GCN_HIP(hipMemcpyAsync(idx, didx, m.nnz * sizeof(int32_t), hipMemcpyDeviceToHost, stream));
    if (val)
      GCN_HIP(hipMemcpyAsync(val, dval, m.nnz * sizeof(float), hipMemcpyDeviceToHost, stream));
  }
  GCN_HIP(hipStreamSynchronize(stream));
  return GCN_OK;
}

extern "C" gcn_status gcn_graph_bins(const gcn_graph* g, int which, int64_t halo_from,
                                     int64_t* records, int cap, int* n_classes, void* stream_) {
  clear_error();
  GCN_CHECK(check_graph(g));
  if (which != 0 && which != 1) {
    set_error("which must be 0 (A) or 1 (A^T)");
    return GCN_EINVAL;
  }
  const Mat& m = which ? g->csc : g->csr;
  const Plan& p = m.plan;
  // the chunked class is reported as two bins: chunk-table rows, then the
  // column-blocked rows (none when the plan blocks nothing)
  constexpr int kBins = kNumClasses + 1;
  unsigned long long halo[kBins] = {};
  const int64_t bmin = p.n_blocked > 0 ? p.blocked_min : 0;
  if (halo_from >= 0 && m.n_major > 0) {
    hipStream_t stream = (hipStream_t)stream_;
    TempScope tmp(stream);
    unsigned long long* d = nullptr;
    GCN_CHECK(tmp.alloc(&d, kBins, "halo counts"));
    GCN_HIP(hipMemsetAsync(d, 0, sizeof(halo), stream));
    hipLaunchKernelGGL(k_class_halo, dim3(grid_for(m.n_major)), dim3(kThreads), 0, stream,
                       (const int64_t*)m.ptr, (const Ent*)m.ent, m.n_major, p.medium_max, bmin,
                       halo_from, d);
    GCN_HIP(hipGetLastError());
    GCN_HIP(hipMemcpyAsync(halo, d, sizeof(halo), hipMemcpyDeviceToHost, stream));
    GCN_HIP(hipStreamSynchronize(stream));
  }
  static const int64_t lo[kNumClasses] = {0, 1, 2, 3, 5, 9, 17, 33, -1};
  static const int64_t hi[kNumClasses] = {0, 1, 2, 4, 8, 16, 32, -1, -1};
  for (int c = 0; c < kBins && c < cap && records; ++c) {
    int64_t* rec = records + 5 * c;
    if (c < kChunked) {
      rec[0] = lo[c];
      rec[1] = c == kMedium ? p.medium_max : hi[c];
      rec[2] = p.class_off[c + 1] - p.class_off[c];
      rec[3] = p.class_nnz[c];
    } else if (c == kChunked) {
      rec[0] = p.medium_max + 1;
      rec[1] = p.n_blocked > 0 ? p.blocked_min - 1 : -1;
      rec[2] = p.class_off[c + 1] - p.class_off[c] - p.n_blocked;
      rec[3] = p.class_nnz[c] - p.blocked_nnz;
    } else {
      rec[0] = p.blocked_min;
      rec[1] = -1;
      rec[2] = p.n_blocked;
      rec[3] = p.blocked_nnz;
    }
    rec[4] = (int64_t)halo[c];
  }
  if (n_classes) *n_classes = kBins;
  return GCN_OK;
}
