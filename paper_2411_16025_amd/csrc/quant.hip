// Per-row uint8 quantization, the producer side of the quantized boundary
// exchange (SuperGCN, arXiv 2411.16025, Section 2.4 and Section 7.3): the
// zero point and scale of a row are computed and the row is quantized in the
// same pass, with round-half-even in place of stochastic rounding.

#include "common.h"

namespace gcn {
namespace {

constexpr int kBlock = 256;

// One wavefront per row: min/max by a butterfly (exact in any order), then
// q = clamp(rint((x - Z) / S), 0, 255) with IEEE fp32 division.
__global__ __launch_bounds__(kBlock) void k_quantize_rows(int64_t n, int F,
                                                          const float* __restrict__ x, int64_t ldx,
                                                          uint8_t* __restrict__ q, int64_t ldq,
                                                          float* __restrict__ zmin,
                                                          float* __restrict__ scale, int64_t ldp) {
  const int lane = threadIdx.x & 63;
  const int64_t i = (int64_t)blockIdx.x * (kBlock / 64) + (threadIdx.x >> 6);
  if (i >= n) return;
  const float* row = x + i * ldx;
  float mn = row[0], mx = row[0];
  for (int f = lane; f < F; f += 64) {
    mn = fminf(mn, row[f]);
    mx = fmaxf(mx, row[f]);
  }
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    mn = fminf(mn, __shfl_xor(mn, off, 64));
    mx = fmaxf(mx, __shfl_xor(mx, off, 64));
  }
  const float s = (mx - mn) / 255.0f;
  if (lane == 0) {
    zmin[i * ldp] = mn;
    scale[i * ldp] = s;
  }
  uint8_t* qr = q + i * ldq;
  for (int f = lane; f < F; f += 64) {
    float c = 0.0f;
    if (s != 0.0f) c = __builtin_rintf((row[f] - mn) / s);
    c = fminf(255.0f, fmaxf(0.0f, c));
    qr[f] = (uint8_t)c;
  }
}

}  // namespace
}  // namespace gcn

using namespace gcn;

extern "C" gcn_status gcn_quantize_rows_u8(int64_t n, int64_t F, const float* X, int64_t ldx,
                                           uint8_t* Q, int64_t ldq, float* zmin, float* scale,
                                           int64_t ldp, void* stream) {
  clear_error();
  if (n < 0 || F <= 0 || F >= (1ll << 31)) {
    set_error("need n >= 0 and F in [1, 2^31)");
    return GCN_EINVAL;
  }
  if (n == 0) return GCN_OK;
  if (!X || !Q || !zmin || !scale || ldx < F || ldq < F || ldp < 1) {
    set_error("X, Q, zmin, scale must be non-NULL with ldx, ldq >= F and ldp >= 1");
    return GCN_EINVAL;
  }
  hipStream_t s = (hipStream_t)stream;
  ProfScope ps("quantize_rows_u8", s);
  const int64_t blocks = ceil_div(n, kBlock / 64);
  hipLaunchKernelGGL(k_quantize_rows, dim3((unsigned)blocks), dim3(kBlock), 0, s, n, (int)F, X, ldx,
                     Q, ldq, zmin, scale, ldp);
  GCN_HIP(hipGetLastError());
  return GCN_OK;
}
