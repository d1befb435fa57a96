// Stable LSD radix sort of 64-bit keys (8-bit digits) and the generic scan.
//
// Each pass: (1) every 4096-key tile counts its digits into LDS, (2) the
// digit-major table of tile counts is prefix-summed, (3) every tile ranks its
// keys stably (wavefront ballots give the rank among equal digits in a
// wavefront, LDS prefix sums across wavefronts and rounds), stages them in
// LDS in digit order, and writes each digit run to its global position, so
// stores of equal digits are contiguous. No global atomics; the result is
// the unique stable order.

#include "scan.h"

namespace gcn {

namespace {

constexpr int kThreads = 256;
constexpr int kItems = 16;
constexpr int kTile = kThreads * kItems;  // keys per tile
constexpr int kWaves = kThreads / 64;

__global__ __launch_bounds__(kThreads) void k_radix_hist(const uint64_t* __restrict__ keys,
                                                         int64_t n, int shift,
                                                         uint32_t* __restrict__ hist,
                                                         int64_t n_tiles) {
  __shared__ uint32_t cnt[kWaves][256];
  const int t = threadIdx.x, w = t >> 6;
  for (int i = t; i < kWaves * 256; i += kThreads) (&cnt[0][0])[i] = 0;
  __syncthreads();
  const int64_t base = (int64_t)blockIdx.x * kTile;
#pragma unroll 4
  for (int j = 0; j < kItems; ++j) {
    const int64_t i = base + j * kThreads + t;
    if (i < n) atomicAdd(&cnt[w][(keys[i] >> shift) & 255u], 1u);
  }
  __syncthreads();
  uint32_t s = 0;
#pragma unroll
  for (int k = 0; k < kWaves; ++k) s += cnt[k][t];
  hist[(int64_t)t * n_tiles + blockIdx.x] = s;
}

__global__ __launch_bounds__(kThreads) void k_radix_scatter(const uint64_t* __restrict__ in,
                                                            uint64_t* __restrict__ out, int64_t n,
                                                            int shift,
                                                            const uint32_t* __restrict__ hist,
                                                            const int64_t* __restrict__ offs,
                                                            int64_t n_tiles) {
  __shared__ uint64_t stage[kTile];
  __shared__ int64_t lds_scan[kThreads];
  __shared__ uint32_t tile_excl[256];
  __shared__ uint32_t run[256];
  __shared__ uint32_t wcnt[kWaves][256];
  const int t = threadIdx.x, w = t >> 6, lane = t & 63;
  const int64_t tile = blockIdx.x;
  const int64_t base = tile * kTile;
  const int tile_n = (int)((n - base) < kTile ? (n - base) : kTile);

  // exclusive prefix over digits of this tile's counts
  const uint32_t my_cnt = hist[(int64_t)t * n_tiles + tile];
  tile_excl[t] = (uint32_t)block_exclusive_scan(my_cnt, lds_scan, nullptr);
  run[t] = 0;
  const uint64_t lt_mask = (lane == 0) ? 0ull : (~0ull >> (64 - lane));

  for (int j = 0; j < kItems; ++j) {
    for (int i = t; i < kWaves * 256; i += kThreads) (&wcnt[0][0])[i] = 0;
    __syncthreads();
    const int li = j * kThreads + t;
    const bool valid = li < tile_n;
    uint64_t key = 0;
    uint32_t d = 0;
    if (valid) {
      key = in[base + li];
      d = (uint32_t)(key >> shift) & 255u;
    }
    uint64_t peers = __ballot(valid);
#pragma unroll
    for (int bit = 0; bit < 8; ++bit) {
      const bool b = (d >> bit) & 1u;
      const uint64_t m = __ballot(b);
      peers &= b ? m : ~m;
    }
    const uint32_t rank = (uint32_t)__popcll(peers & lt_mask);
    if (valid && rank == 0) wcnt[w][d] = (uint32_t)__popcll(peers);
    __syncthreads();
    {
      // digit t: prefix over wavefronts, continuing the running count
      uint32_t pre = run[t];
#pragma unroll
      for (int k = 0; k < kWaves; ++k) {
        const uint32_t c = wcnt[k][t];
        wcnt[k][t] = pre;
        pre += c;
      }
      run[t] = pre;
    }
    __syncthreads();
    if (valid) stage[tile_excl[d] + wcnt[w][d] + rank] = key;
    __syncthreads();
  }
  for (int j = 0; j < kItems; ++j) {
    const int lp = j * kThreads + t;
    if (lp < tile_n) {
      const uint64_t key = stage[lp];
      const uint32_t d = (uint32_t)(key >> shift) & 255u;
      out[offs[(int64_t)d * n_tiles + tile] + (lp - tile_excl[d])] = key;
    }
  }
}

}  // namespace

namespace {

struct RadixWork {
  int64_t n_tiles = 0, cells = 0;
  uint32_t* hist = nullptr;
  int64_t* offs = nullptr;
  int64_t* scratch = nullptr;
  hipStream_t stream = nullptr;
  gcn_status init(int64_t n, hipStream_t s) {
    stream = s;
    n_tiles = ceil_div(n, kTile);
    cells = 256 * n_tiles;
    GCN_CHECK(talloc(&hist, cells, s, "radix histogram"));
    GCN_CHECK(talloc(&offs, cells + 1, s, "radix offsets"));
    GCN_CHECK(talloc(&scratch, scan_scratch_elems(cells), s, "scan scratch"));
    return GCN_OK;
  }
  ~RadixWork() {
    tfree(scratch, stream);
    tfree(offs, stream);
    tfree(hist, stream);
  }
  gcn_status pass(const uint64_t* in, uint64_t* out, int64_t n, int shift) {
    {
      ProfScope p("radix_hist", stream);
      hipLaunchKernelGGL(k_radix_hist, dim3((unsigned)n_tiles), dim3(kThreads), 0, stream, in, n,
                         shift, hist, n_tiles);
      GCN_HIP(hipGetLastError());
    }
    GCN_CHECK(scan_functor(ArrayInput<uint32_t>{hist}, cells, offs, scratch, stream));
    {
      ProfScope p("radix_scatter", stream);
      hipLaunchKernelGGL(k_radix_scatter, dim3((unsigned)n_tiles), dim3(kThreads), 0, stream, in,
                         out, n, shift, (const uint32_t*)hist, (const int64_t*)offs, n_tiles);
      GCN_HIP(hipGetLastError());
    }
    return GCN_OK;
  }
};

}  // namespace

gcn_status radix_pass_u64(const uint64_t* in, uint64_t* out, int64_t n, int shift,
                          hipStream_t stream) {
  if (n == 0) return GCN_OK;
  RadixWork w;
  GCN_CHECK(w.init(n, stream));
  return w.pass(in, out, n, shift);
}

gcn_status radix_sort_u64(uint64_t** keys, uint64_t** alt, int64_t n, int bits,
                          hipStream_t stream) {
  if (n == 0) return GCN_OK;
  RadixWork w;
  GCN_CHECK(w.init(n, stream));
  for (int shift = 0; shift < bits; shift += 8) {
    GCN_CHECK(w.pass(*keys, *alt, n, shift));
    uint64_t* tmp = *keys;
    *keys = *alt;
    *alt = tmp;
  }
  return GCN_OK;
}

gcn_status scan_i64(const int64_t* in, int64_t* out, int64_t n, hipStream_t stream) {
  int64_t* scratch = nullptr;
  GCN_CHECK(talloc(&scratch, scan_scratch_elems(n), stream, "scan scratch"));
  gcn_status st = scan_functor(ArrayInput<int64_t>{in}, n, out, scratch, stream);
  tfree(scratch, stream);
  return st;
}

}  // namespace gcn
