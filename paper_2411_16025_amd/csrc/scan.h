// Device-wide exclusive prefix sum over a functor-produced int64 sequence.
//
// Three phases (reduce tiles, scan the tile sums, rescan tiles with their
// offsets), so the result does not depend on scheduling. Used for radix-sort
// digit offsets, deduplication positions and chunk tables.
#pragma once

#include "common.h"

namespace gcn {

constexpr int kScanThreads = 256;
constexpr int kScanItems = 8;
constexpr int64_t kScanTile = kScanThreads * kScanItems;

template <class T>
struct ArrayInput {
  const T* p;
  __device__ int64_t operator()(int64_t i) const { return (int64_t)p[i]; }
};

// Exclusive scan of 256 per-thread values held in LDS; returns this thread's
// exclusive prefix and writes the block total to *total.
__device__ inline int64_t block_exclusive_scan(int64_t v, int64_t* lds, int64_t* total) {
  const int t = threadIdx.x;
  lds[t] = v;
  __syncthreads();
  for (int off = 1; off < kScanThreads; off <<= 1) {
    int64_t add = (t >= off) ? lds[t - off] : 0;
    __syncthreads();
    lds[t] += add;
    __syncthreads();
  }
  const int64_t incl = lds[t];
  if (total) *total = lds[kScanThreads - 1];
  __syncthreads();
  return incl - v;
}

template <class In>
__global__ __launch_bounds__(kScanThreads) void k_scan_reduce(In in, int64_t n, int64_t* sums) {
  __shared__ int64_t lds[kScanThreads];
  const int64_t base = (int64_t)blockIdx.x * kScanTile + (int64_t)threadIdx.x * kScanItems;
  int64_t s = 0;
#pragma unroll
  for (int j = 0; j < kScanItems; ++j)
    if (base + j < n) s += in(base + j);
  int64_t total;
  block_exclusive_scan(s, lds, &total);
  if (threadIdx.x == 0) sums[blockIdx.x] = total;
}

template <class In>
__global__ __launch_bounds__(kScanThreads) void k_scan_down(In in, int64_t n, const int64_t* offs,
                                                            int64_t* out) {
  __shared__ int64_t lds[kScanThreads];
  const int64_t base = (int64_t)blockIdx.x * kScanTile + (int64_t)threadIdx.x * kScanItems;
  int64_t v[kScanItems];
  int64_t s = 0;
#pragma unroll
  for (int j = 0; j < kScanItems; ++j) {
    v[j] = (base + j < n) ? in(base + j) : 0;
    s += v[j];
  }
  int64_t total;
  int64_t run = block_exclusive_scan(s, lds, &total) + (offs ? offs[blockIdx.x] : 0);
#pragma unroll
  for (int j = 0; j < kScanItems; ++j) {
    if (base + j < n) out[base + j] = run;
    run += v[j];
  }
  // the block holding the last element also writes the grand total at out[n]
  if (base <= n - 1 && n - 1 < base + kScanItems) out[n] = run;
  if (n == 0 && blockIdx.x == 0 && threadIdx.x == 0) out[0] = 0;
}

// out[0..n] = exclusive scan of in(0..n-1), out[n] = total. `scratch` must
// hold scan_scratch_elems(n) int64 values.
inline int64_t scan_scratch_elems(int64_t n) {
  int64_t total = 0;
  int64_t m = ceil_div(n, kScanTile);
  while (m > 1) {
    total += m + 1;
    m = ceil_div(m, kScanTile);
  }
  return total + 2;
}

template <class In>
gcn_status scan_functor(In in, int64_t n, int64_t* out, int64_t* scratch, hipStream_t stream) {
  const int64_t nb = ceil_div(n, kScanTile);
  if (nb <= 1) {
    hipLaunchKernelGGL(k_scan_down<In>, dim3(1), dim3(kScanThreads), 0, stream, in, n,
                       (const int64_t*)nullptr, out);
    GCN_HIP(hipGetLastError());
    return GCN_OK;
  }
  int64_t* sums = scratch;  // nb + 1 entries
  hipLaunchKernelGGL(k_scan_reduce<In>, dim3((unsigned)nb), dim3(kScanThreads), 0, stream, in, n,
                     sums);
  GCN_HIP(hipGetLastError());
  GCN_CHECK(scan_functor(ArrayInput<int64_t>{sums}, nb, sums, scratch + nb + 1, stream));
  hipLaunchKernelGGL(k_scan_down<In>, dim3((unsigned)nb), dim3(kScanThreads), 0, stream, in, n,
                     (const int64_t*)sums, out);
  GCN_HIP(hipGetLastError());
  return GCN_OK;
}

}  // namespace gcn
