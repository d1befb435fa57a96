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

// Wavefront sums of a double (butterfly; every lane ends with the total).
__device__ inline double wave_sum(double v) {
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) v += __shfl_xor(v, off, 64);
  return v;
}

struct RowNorm {
  double mean, inv;
  const float* gamma;
  const float* beta;
  bool on;
  __device__ inline float apply(float x, int64_t f) const {
    if (!on) return x;
    const double g = gamma ? (double)gamma[f] : 1.0;
    const double b = beta ? (double)beta[f] : 0.0;
    return (float)(((double)x - mean) * inv * g + b);
  }
};

// One wavefront per row: optional LayerNorm in double (Section 6.1 step 2),
// rounded once to fp32, then the per-row b-bit quantization of those values
// (Section 2.4; Section 7.3 computes the parameters and the codes in one
// pass). 2-bit codes: feature f in bits [2 (f % 4), 2 (f % 4) + 2) of byte
// f / 4, padding codes 0.
__global__ __launch_bounds__(kBlock) void k_ln_quantize(int64_t n, int F, const float* __restrict__ x,
                                                        int64_t ldx, const float* __restrict__ gamma,
                                                        const float* __restrict__ beta, double eps,
                                                        int ln, int bits, float* __restrict__ y,
                                                        int64_t ldy, uint8_t* __restrict__ q,
                                                        int64_t ldq, float* __restrict__ zmin,
                                                        float* __restrict__ scale, int64_t ldp) {
  const int lane = threadIdx.x & 63;
  const int64_t i = (int64_t)blockIdx.x * (kBlock / 64) + (threadIdx.x >> 6);
  if (i >= n) return;
  const float* row = x + i * ldx;
  RowNorm nm{0.0, 1.0, gamma, beta, ln != 0};
  if (ln) {
    double s = 0.0;
    for (int f = lane; f < F; f += 64) s += (double)row[f];
    const double mean = wave_sum(s) / (double)F;
    double v = 0.0;
    for (int f = lane; f < F; f += 64) {
      const double d = (double)row[f] - mean;
      v += d * d;
    }
    nm.mean = mean;
    nm.inv = 1.0 / sqrt(wave_sum(v) / (double)F + eps);
  }
  float mn = nm.apply(row[0], 0), mx = mn;
  for (int f = lane; f < F; f += 64) {
    const float t = nm.apply(row[f], f);
    mn = fminf(mn, t);
    mx = fmaxf(mx, t);
    if (y) y[i * ldy + f] = t;
  }
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    mn = fminf(mn, __shfl_xor(mn, off, 64));
    mx = fmaxf(mx, __shfl_xor(mx, off, 64));
  }
  const float levels = (float)((1 << bits) - 1);
  const float s = (mx - mn) / levels;
  if (lane == 0) {
    zmin[i * ldp] = mn;
    scale[i * ldp] = s;
  }
  uint8_t* qr = q + i * ldq;
  if (bits == 8) {
    for (int f = lane; f < F; f += 64) {
      float c = 0.0f;
      if (s != 0.0f) c = __builtin_rintf((nm.apply(row[f], f) - mn) / s);
      qr[f] = (uint8_t)fminf(levels, fmaxf(0.0f, c));
    }
  } else {
    for (int k = lane; 4 * k < F; k += 64) {
      uint32_t byte = 0;
      for (int e = 0; e < 4 && 4 * k + e < F; ++e) {
        const int f = 4 * k + e;
        float c = 0.0f;
        if (s != 0.0f) c = __builtin_rintf((nm.apply(row[f], f) - mn) / s);
        byte |= (uint32_t)fminf(levels, fmaxf(0.0f, c)) << (2 * e);
      }
      qr[k] = (uint8_t)byte;
    }
  }
}

}  // namespace
}  // namespace gcn

using namespace gcn;

extern "C" gcn_status gcn_layernorm_quantize(int64_t n, int64_t F, const float* X, int64_t ldx,
                                             const float* gamma, const float* beta, double eps,
                                             uint32_t flags, int bits, float* Y, int64_t ldy,
                                             uint8_t* Q, int64_t ldq, float* zmin, float* scale,
                                             int64_t ldp, void* stream) {
  clear_error();
  if (n < 0 || F <= 0 || F >= (1ll << 31) || (bits != 8 && bits != 2) ||
      (flags & ~(uint32_t)GCN_LAYERNORM) || !(eps >= 0.0)) {
    set_error("need n >= 0, F in [1, 2^31), bits 8 or 2, known flags and eps >= 0");
    return GCN_EINVAL;
  }
  if (n == 0) return GCN_OK;
  const int64_t qbytes = bits == 8 ? F : (F + 3) / 4;
  if (!X || !Q || !zmin || !scale || ldx < F || ldq < qbytes || ldp < 1 || (Y && ldy < F)) {
    set_error("X, Q, zmin, scale must be non-NULL with ldx >= F, ldq >= code bytes per row, "
              "ldp >= 1 (and ldy >= F when Y is given)");
    return GCN_EINVAL;
  }
  hipStream_t s = (hipStream_t)stream;
  ProfScope ps("layernorm_quantize", s);
  hipLaunchKernelGGL(k_ln_quantize, dim3((unsigned)ceil_div(n, kBlock / 64)), dim3(kBlock), 0, s, n,
                     (int)F, X, ldx, gamma, beta, eps, (int)(flags & GCN_LAYERNORM), bits, Y, ldy,
                     Q, ldq, zmin, scale, ldp);
  GCN_HIP(hipGetLastError());
  return GCN_OK;
}

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
