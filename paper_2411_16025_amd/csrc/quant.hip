// Row-wise kernels: per-row b-bit quantization (b = 8 or 2), the producer
// side of the quantized boundary exchange (SuperGCN, arXiv 2411.16025,
// Sections 2.4, 6.1 and 7.3: the zero point and scale of a row are computed
// and the row is quantized in the same pass, with round-half-even in place of
// stochastic rounding), optionally after a row LayerNorm (Section 6.1 step 2);
// and the LayerNorm forward and backward of the GraphSAGE model (Table 2).

#include <algorithm>

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
                                                        float* __restrict__ scale, int64_t ldp,
                                                        float* __restrict__ rstd) {
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
    if (rstd && lane == 0) rstd[i] = (float)nm.inv;
  }
  if (bits == 0) {  // LayerNorm only
    for (int f = lane; f < F; f += 64) y[i * ldy + f] = nm.apply(row[f], f);
    return;
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

// Register-resident variant for rows of at most 4 * G * NV features in
// 16-byte aligned storage (ldx % 4 == 0): a slot of G lanes holds a whole row
// (NV float4 per lane), so the row is read from memory once; a wavefront
// holds 64 / G rows per group and R groups are loaded before any arithmetic.
// The values of k_ln_quantize: statistics in double (their summation order
// and the last ulps of double in 1 / sqrt(var + eps) differ), values rounded
// once to fp32, the codes of IEEE fp32 division.
//
// A slot's butterfly pairs lanes within the slot: the partner at distance 1
// and 2 comes from a quad permutation, at 4 and 8 from the mirror of the
// half row and of the row (after the earlier steps every lane of a quad,
// then of a half row, holds the same value, so the mirror partner carries
// the same operand as lane ^ 4 or lane ^ 8), further ones from a wavefront
// shuffle. The DPP moves need no LDS round trip; the sums are those of the
// xor butterfly, bit for bit.
template <int CTRL>
__device__ inline int dpp_mov(int x) {
  return __builtin_amdgcn_mov_dpp(x, CTRL, 0xF, 0xF, false);
}

template <int OFF>
__device__ inline int slot_partner(int x) {
  if constexpr (OFF == 1) return dpp_mov<0xB1>(x);   // quad_perm [1, 0, 3, 2]
  if constexpr (OFF == 2) return dpp_mov<0x4E>(x);   // quad_perm [2, 3, 0, 1]
  if constexpr (OFF == 4) return dpp_mov<0x141>(x);  // row_half_mirror
  if constexpr (OFF == 8) return dpp_mov<0x140>(x);  // row_mirror
  return __shfl_xor(x, OFF, 64);
}

template <int OFF>
__device__ inline float slot_partner(float v) {
  return __int_as_float(slot_partner<OFF>(__float_as_int(v)));
}

template <int OFF>
__device__ inline double slot_partner(double v) {
  const long long b = __double_as_longlong(v);
  const int lo = slot_partner<OFF>((int)b);
  const int hi = slot_partner<OFF>((int)(b >> 32));
  return __longlong_as_double((long long)(((unsigned long long)(unsigned)hi << 32) | (unsigned)lo));
}

template <int G, int OFF = 1>
__device__ inline double slot_sum(double v) {
  if constexpr (OFF < G) {
    v += slot_partner<OFF>(v);
    return slot_sum<G, 2 * OFF>(v);
  } else {
    return v;
  }
}

template <int G, int OFF = 1>
__device__ inline void slot_minmax(float& mn, float& mx) {
  if constexpr (OFF < G) {
    mn = fminf(mn, slot_partner<OFF>(mn));
    mx = fmaxf(mx, slot_partner<OFF>(mx));
    slot_minmax<G, 2 * OFF>(mn, mx);
  }
}

// clamp(rint((t - Z) / S), 0, levels) with IEEE fp32 division
__device__ inline uint32_t code_of(float a, float s, float levels) {
  return (uint32_t)fminf(levels, fmaxf(0.0f, __builtin_rintf(a / s)));
}

// The same code from the row's correctly rounded reciprocal rs = RN(1 / S):
// q = RN(a rs) is within one ulp of a / S, the residual a - q S is exact in
// an fma, and RN(q + (a - q S) rs) is the correctly rounded quotient RN(a / S)
// (Markstein's theorem for round-to-nearest division). Valid while the
// residual cannot underflow where it matters: S in [2^-100, 2^100] (quotients
// below 1/4 round to code 0 either way). Adding 1.5 * 2^23 then rounds the
// quotient to an integer, half to even (the spacing of floats there is 1),
// and leaves it in the low mantissa bits: the returned word is 0x4B400000 +
// code, bits 8 to 21 clear, so a byte of it, or a 2-bit field shifted into a
// byte, is the code. Clamping the sum to [1.5 * 2^23, 1.5 * 2^23 + levels]
// keeps the quotient's range (a in [0, max - min], so RN(a / S) is at most
// levels up to a rounding) and maps NaN to code 0, as the division form
// does. A row with S = 0 passes rs = 0 and gets code 0.
__device__ inline uint32_t code_word_rcp(float a, float s, float rs, float levels) {
  constexpr float kMagic = 0x1.8p23f;
  const float q = a * rs;
  const float e = __builtin_fmaf(-q, s, a);
  const float w = __builtin_fmaf(e, rs, q) + kMagic;
  return __float_as_uint(fminf(kMagic + levels, fmaxf(kMagic, w)));
}

// 1 / sqrt(x) for finite x > 0: the hardware estimate refined by two Newton
// steps on the residual e = 1 - x r^2 (r += r e / 2; each step squares the
// relative error), a few ulps of double from the quotient of the correctly
// rounded square root. The normalized values are rounded to fp32 afterwards,
// so such an ulp decides a value only when its exact product lies within
// about 2^-50 of a rounding boundary of fp32.
__device__ inline double inv_sqrt(double x) {
  double r = __builtin_amdgcn_rsq(x);
#pragma unroll
  for (int k = 0; k < 2; ++k) {
    const double e = __builtin_fma(-x * r, r, 1.0);
    r = __builtin_fma(0.5 * r, e, r);
  }
  return r;
}

__device__ inline bool rcp_ok(float s) { return s >= 0x1p-100f && s <= 0x1p100f; }

struct QuantArgs {
  int64_t n;
  int F;
  const float* x;
  int64_t ldx;
  const float* gamma;
  const float* beta;
  double eps;
  int ln, bits;
  float* y;
  int64_t ldy;
  uint8_t* q;
  int64_t ldq;
  float* zmin;
  float* scale;
  int64_t ldp;
  bool q_dword, y_vec;  // Q rows 4-byte aligned; Y rows 16-byte aligned
  float* rstd;          // optional 1 / sqrt(var + eps) per row (bits == 0 only)
};

// LN: LayerNorm first; BITS: 8 or 2 (codes), 0 (LayerNorm output only);
// FULL: every lane's features lie inside the row (F = 4 G NV) and the stores
// are aligned (Q rows 4-byte aligned for 8-bit codes, Y rows 16-byte), so no
// feature is guarded. Each variant is its own kernel: the run-time choices
// cost more issue slots than the memory traffic leaves room for.
template <int G, int NV, int R, bool AFFINE, bool LN, int BITS, bool FULL>
__global__ __launch_bounds__(kBlock) void k_ln_quantize_v(QuantArgs a) {
  constexpr int E = 64 / G;
  const int lane = threadIdx.x & 63;
  const int sl = lane % G;
  // the wavefront walks its row groups (E * R rows each) with a stride of
  // the grid's wavefronts, loading the next group while it works on this one
  const int64_t n_iter = (a.n + E * R - 1) / (E * R);
  const int64_t stride = (int64_t)gridDim.x * (kBlock / 64);
  int64_t it = (int64_t)blockIdx.x * (kBlock / 64) + (threadIdx.x >> 6);
  const int F = FULL ? 4 * G * NV : a.F;
  auto inside = [&](int f) { return FULL || f < F; };
  auto load = [&](int64_t iter, float (&v)[R][NV][4]) {
#pragma unroll
    for (int r = 0; r < R; ++r) {
      const int64_t i = iter * (E * R) + (int64_t)r * E + lane / G;
#pragma unroll
      for (int j = 0; j < NV; ++j) {
        const int f = 4 * (sl + j * G);
        if (i < a.n && (FULL || f + 4 <= F)) {
          const float4 t = *reinterpret_cast<const float4*>(a.x + i * a.ldx + f);
          v[r][j][0] = t.x;
          v[r][j][1] = t.y;
          v[r][j][2] = t.z;
          v[r][j][3] = t.w;
        } else {
#pragma unroll
          for (int e = 0; e < 4; ++e)
            v[r][j][e] = (i < a.n && f + e < F) ? a.x[i * a.ldx + f + e] : 0.0f;
        }
      }
    }
  };
  if (it >= n_iter) return;  // whole wavefronts leave together
  constexpr float levels = (float)((1 << (BITS > 0 ? BITS : 1)) - 1);
  auto process = [&](int64_t it, float (&v)[R][NV][4]) {
#pragma unroll
    for (int r = 0; r < R; ++r) {
      const int64_t i = it * (E * R) + (int64_t)r * E + lane / G;
      const bool live = i < a.n;
      if constexpr (LN) {
        double s = 0.0;
#pragma unroll
        for (int j = 0; j < NV; ++j)
#pragma unroll
          for (int e = 0; e < 4; ++e) s += (double)v[r][j][e];  // masked entries are 0
        const double mean = slot_sum<G>(s) / (double)F;
        double d[NV][4];
        double var = 0.0;
#pragma unroll
        for (int j = 0; j < NV; ++j)
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            d[j][e] = (double)v[r][j][e] - mean;
            if (inside(4 * (sl + j * G) + e)) var = __builtin_fma(d[j][e], d[j][e], var);
          }
        const double inv = inv_sqrt(slot_sum<G>(var) / (double)F + a.eps);
        if (BITS == 0 && a.rstd && live && sl == 0) a.rstd[i] = (float)inv;
#pragma unroll
        for (int j = 0; j < NV; ++j)
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const int f = 4 * (sl + j * G) + e;
            if (inside(f)) {
              if (AFFINE) {
                const double g = a.gamma ? (double)a.gamma[f] : 1.0;
                const double b = a.beta ? (double)a.beta[f] : 0.0;
                v[r][j][e] = (float)(d[j][e] * inv * g + b);
              } else {
                v[r][j][e] = (float)(d[j][e] * inv + 0.0);  // + 0 turns -0 into +0
              }
            }
          }
      }
      if constexpr (BITS == 0) {  // LayerNorm only
        if (!live) continue;
        float* yr = a.y + i * a.ldy;
#pragma unroll
        for (int j = 0; j < NV; ++j) {
          const int f = 4 * (sl + j * G);
          if (!FULL && f >= F) continue;
          if (FULL || (f + 4 <= F && a.y_vec))
            *reinterpret_cast<float4*>(yr + f) = make_float4(v[r][j][0], v[r][j][1], v[r][j][2], v[r][j][3]);
          else
            for (int e = 0; e < 4 && f + e < F; ++e) yr[f + e] = v[r][j][e];
        }
        continue;
      } else {
        float mn = __builtin_inff(), mx = -__builtin_inff();
#pragma unroll
        for (int j = 0; j < NV; ++j)
#pragma unroll
          for (int e = 0; e < 4; ++e)
            if (inside(4 * (sl + j * G) + e)) {
              mn = fminf(mn, v[r][j][e]);
              mx = fmaxf(mx, v[r][j][e]);
            }
        slot_minmax<G>(mn, mx);
        const float s = (mx - mn) / levels;
        const float rs = s != 0.0f ? 1.0f / s : 0.0f;
        // one path per wavefront: the reciprocal form while every live row's
        // scale allows it (almost always), IEEE division otherwise
        const bool fast = __all(!live || s == 0.0f || rcp_ok(s));
        if (!live) continue;
        if (sl == 0) {
          a.zmin[i * a.ldp] = mn;
          a.scale[i * a.ldp] = s;
        }
        uint8_t* qr = a.q + i * a.ldq;
        // the path is chosen once per row group: a choice per feature costs
        // a branch per feature
        auto write = [&](auto code) {
#pragma unroll
          for (int j = 0; j < NV; ++j) {
            const int f = 4 * (sl + j * G);
            if (!FULL && f >= F) continue;
            // code words: the code in the low bits, bits 8 to 21 clear
            uint32_t c[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              const uint32_t cc = code(v[r][j][e] - mn);
              c[e] = inside(f + e) ? cc : 0u;
            }
            const bool whole = FULL || f + 4 <= F;
            if constexpr (BITS == 2) {
              qr[f / 4] = (uint8_t)(c[0] | (c[1] << 2) | (c[2] << 4) | (c[3] << 6));
            } else {
              if (whole && (FULL || a.q_dword))
                *reinterpret_cast<uint32_t*>(qr + f) = (c[0] & 0xFFu) | ((c[1] & 0xFFu) << 8) |
                                                       ((c[2] & 0xFFu) << 16) | (c[3] << 24);
              else
                for (int e = 0; e < 4 && f + e < F; ++e) qr[f + e] = (uint8_t)c[e];
            }
            if (a.y) {
              float* yr = a.y + i * a.ldy;
              if (whole && (FULL || a.y_vec))
                *reinterpret_cast<float4*>(yr + f) = make_float4(v[r][j][0], v[r][j][1], v[r][j][2], v[r][j][3]);
              else
                for (int e = 0; e < 4 && f + e < F; ++e) yr[f + e] = v[r][j][e];
            }
          }
        };
        if (fast)
          write([&](float t) { return code_word_rcp(t, s, rs, levels); });
        else
          write([&](float t) { return s != 0.0f ? code_of(t, s, levels) : 0u; });
      }
    }
  };
  if constexpr (!LN) {
    // one row group per wavefront (the grid covers the rows)
    float v[R][NV][4];
    load(it, v);
    process(it, v);
  } else {
    // the walk, unrolled by two so that the prefetched group is worked on in
    // the registers it was loaded into
    float va[R][NV][4], vb[R][NV][4];
    load(it, va);
    for (;;) {
      if (it + stride < n_iter) load(it + stride, vb);
      process(it, va);
      it += stride;
      if (it >= n_iter) break;
      if (it + stride < n_iter) load(it + stride, va);
      process(it, vb);
      it += stride;
      if (it >= n_iter) break;
    }
  }
}

template <int G, int NV, int R, bool AFFINE, bool LN, int BITS>
void launch_v_full(const QuantArgs& a, hipStream_t s, dim3 grid) {
  const bool full = a.F == 4 * G * NV && (BITS != 8 || a.q_dword) && (!a.y || a.y_vec);
  if (full)
    hipLaunchKernelGGL((k_ln_quantize_v<G, NV, R, AFFINE, LN, BITS, true>), grid, dim3(kBlock), 0,
                       s, a);
  else
    hipLaunchKernelGGL((k_ln_quantize_v<G, NV, R, AFFINE, LN, BITS, false>), grid, dim3(kBlock), 0,
                       s, a);
}

// With LayerNorm a wavefront works on a row group long enough that the next
// group's loads are best issued meanwhile: the grid is capped at 32
// workgroups per CU and every wavefront walks several groups, prefetching.
// Without it one group per wavefront over a grid that covers the rows is
// fastest (4M x 128 rows, Int2: 0.404 ms with one group of 8 rows per
// wavefront, 0.417 with two, 0.441 with four; 8-bit 0.470 / 0.498 / 0.500):
// the kernels without LayerNorm take exactly one row group per wavefront and
// rely on this grid covering every row.
constexpr int64_t kQuantBlocksLN = 256 * 32;

template <int G, int NV, int R>
gcn_status launch_v(const QuantArgs& a, hipStream_t s) {
  const int64_t rows_per_block = (int64_t)(kBlock / 64) * (64 / G) * R;
  const int64_t need = ceil_div(a.n, rows_per_block);
  const dim3 grid((unsigned)(a.ln ? std::min<int64_t>(need, kQuantBlocksLN) : need));
  const bool affine = a.ln && (a.gamma || a.beta);
  if (a.bits == 0) {  // LayerNorm only
    if (affine)
      launch_v_full<G, NV, R, true, true, 0>(a, s, grid);
    else
      launch_v_full<G, NV, R, false, true, 0>(a, s, grid);
  } else if (a.bits == 8) {
    if (!a.ln)
      launch_v_full<G, NV, R, false, false, 8>(a, s, grid);
    else if (affine)
      launch_v_full<G, NV, R, true, true, 8>(a, s, grid);
    else
      launch_v_full<G, NV, R, false, true, 8>(a, s, grid);
  } else {
    if (!a.ln)
      launch_v_full<G, NV, R, false, false, 2>(a, s, grid);
    else if (affine)
      launch_v_full<G, NV, R, true, true, 2>(a, s, grid);
    else
      launch_v_full<G, NV, R, false, true, 2>(a, s, grid);
  }
  GCN_HIP(hipGetLastError());
  return GCN_OK;
}

// The register-resident kernel when the layout allows it (returns false
// otherwise, and the row-per-wavefront kernel runs). Up to 16 features per
// lane and 8 lanes or more per row.
bool try_vector(const QuantArgs& a, hipStream_t s, gcn_status* st) {
  if (a.ldx % 4 != 0 || reinterpret_cast<uintptr_t>(a.x) % 16 != 0 || a.F > 1024) return false;
  if (a.F <= 32)
    *st = launch_v<8, 1, 2>(a, s);
  else if (a.F <= 64)
    *st = launch_v<8, 2, 2>(a, s);
  else if (a.F <= 128)
    *st = launch_v<8, 4, 1>(a, s);
  else if (a.F <= 256)
    *st = launch_v<16, 4, 1>(a, s);
  else if (a.F <= 512)
    *st = launch_v<32, 4, 1>(a, s);
  else
    *st = launch_v<64, 4, 1>(a, s);
  return true;
}

QuantArgs make_args(int64_t n, int64_t F, const float* X, int64_t ldx, const float* gamma,
                    const float* beta, double eps, int ln, int bits, float* Y, int64_t ldy,
                    uint8_t* Q, int64_t ldq, float* zmin, float* scale, int64_t ldp) {
  QuantArgs a{n, (int)F, X, ldx, gamma, beta, eps, ln, bits, Y, ldy, Q, ldq, zmin, scale, ldp,
              false, false, nullptr};
  a.q_dword = reinterpret_cast<uintptr_t>(Q) % 4 == 0 && ldq % 4 == 0;
  a.y_vec = Y && reinterpret_cast<uintptr_t>(Y) % 16 == 0 && ldy % 4 == 0;
  return a;
}

// ---- LayerNorm backward -----------------------------------------------------------

// dx = rstd * (g - mean(g) - y * mean(g * y)) per row, g = g1 (+ g2), then
// optionally dx *= (mask > 0) (the ReLU of the layer below). y is the
// normalized output of the forward pass. Row means in double.
struct LnBwdArgs {
  int64_t n;
  int F;
  const float* y;
  int64_t ldy;
  const float* rstd;
  const float* g1;
  int64_t ld1;
  const float* g2;
  int64_t ld2;
  const float* mask;  // may alias dx (read before dx is written, by the same lane)
  int64_t ldm;
  float* dx;
  int64_t ldx;
};

// Vector path (F a multiple of 4): G lanes per row, NV 16-byte pieces per
// lane. Every load takes an address inside its row (pieces past F read the
// row's first piece, rows past n the last row) and values outside the row are
// zeroed afterwards, so all loads of a lane are issued before any arithmetic,
// without branches. G2 and MASK say whether the second gradient and the mask
// are given.
template <int G, int NV, bool G2, bool MASK>
__global__ __launch_bounds__(kBlock) void k_ln_bwd_v(LnBwdArgs a) {
  constexpr int E = 64 / G;
  const int lane = threadIdx.x & 63;
  const int sl = lane % G;
  const int64_t i = ((int64_t)blockIdx.x * (kBlock / 64) + (threadIdx.x >> 6)) * E + lane / G;
  const bool live = i < a.n;
  const int64_t ic = live ? i : a.n - 1;
  float4 yv[NV], gv[NV], hv[NV], mv[NV];
#pragma unroll
  for (int j = 0; j < NV; ++j) {
    const int f = 4 * (sl + j * G);
    const int fo = f < a.F ? f : 0;
    yv[j] = *reinterpret_cast<const float4*>(a.y + ic * a.ldy + fo);
    gv[j] = *reinterpret_cast<const float4*>(a.g1 + ic * a.ld1 + fo);
    if constexpr (G2) hv[j] = *reinterpret_cast<const float4*>(a.g2 + ic * a.ld2 + fo);
    if constexpr (MASK) mv[j] = *reinterpret_cast<const float4*>(a.mask + ic * a.ldm + fo);
  }
  float yf[NV][4], gf[NV][4];
  bool keep[NV][4];
#pragma unroll
  for (int j = 0; j < NV; ++j) {
    const int f = 4 * (sl + j * G);
    const float yy[4] = {yv[j].x, yv[j].y, yv[j].z, yv[j].w};
    float gg[4] = {gv[j].x, gv[j].y, gv[j].z, gv[j].w};
    if constexpr (G2) {
      gg[0] += hv[j].x;
      gg[1] += hv[j].y;
      gg[2] += hv[j].z;
      gg[3] += hv[j].w;
    }
    const float mm[4] = {MASK ? mv[j].x : 1.f, MASK ? mv[j].y : 1.f, MASK ? mv[j].z : 1.f,
                         MASK ? mv[j].w : 1.f};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const bool ok = live && f < a.F;
      yf[j][e] = ok ? yy[e] : 0.f;
      gf[j][e] = ok ? gg[e] : 0.f;
      keep[j][e] = mm[e] > 0.f;
    }
  }
  double s1 = 0.0, s2 = 0.0;
#pragma unroll
  for (int j = 0; j < NV; ++j)
#pragma unroll
    for (int e = 0; e < 4; ++e) {  // entries outside the row are 0
      s1 += (double)gf[j][e];
      s2 += (double)gf[j][e] * (double)yf[j][e];
    }
  const double m1 = slot_sum<G>(s1) / (double)a.F;
  const double m2 = slot_sum<G>(s2) / (double)a.F;
  if (!live) return;
  const double r = (double)a.rstd[i];
  float* out = a.dx + i * a.ldx;
#pragma unroll
  for (int j = 0; j < NV; ++j) {
    const int f = 4 * (sl + j * G);
    if (f >= a.F) continue;
    float o[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float d = (float)(r * ((double)gf[j][e] - m1 - (double)yf[j][e] * m2));
      o[e] = keep[j][e] ? d : 0.f;
    }
    *reinterpret_cast<float4*>(out + f) = make_float4(o[0], o[1], o[2], o[3]);
  }
}

// One wavefront per row for wide rows, unaligned storage or F % 4 != 0.
__global__ __launch_bounds__(kBlock) void k_ln_bwd(LnBwdArgs a) {
  const int lane = threadIdx.x & 63;
  const int64_t i = (int64_t)blockIdx.x * (kBlock / 64) + (threadIdx.x >> 6);
  if (i >= a.n) return;
  auto g_at = [&](int f) {
    return a.g1[i * a.ld1 + f] + (a.g2 ? a.g2[i * a.ld2 + f] : 0.f);
  };
  double s1 = 0.0, s2 = 0.0;
  for (int f = lane; f < a.F; f += 64) {
    const double gf = (double)g_at(f);
    s1 += gf;
    s2 += gf * (double)a.y[i * a.ldy + f];
  }
  const double m1 = wave_sum(s1) / (double)a.F;
  const double m2 = wave_sum(s2) / (double)a.F;
  const double r = (double)a.rstd[i];
  for (int f = lane; f < a.F; f += 64) {
    const float d = (float)(r * ((double)g_at(f) - m1 - (double)a.y[i * a.ldy + f] * m2));
    const bool keep = !a.mask || a.mask[i * a.ldm + f] > 0.f;
    a.dx[i * a.ldx + f] = keep ? d : 0.f;
  }
}

template <int G, int NV>
void launch_bwd_v(const LnBwdArgs& a, hipStream_t s) {
  const dim3 grid((unsigned)ceil_div(a.n, (int64_t)(kBlock / 64) * (64 / G)));
  if (a.g2 && a.mask)
    hipLaunchKernelGGL((k_ln_bwd_v<G, NV, true, true>), grid, dim3(kBlock), 0, s, a);
  else if (a.g2)
    hipLaunchKernelGGL((k_ln_bwd_v<G, NV, true, false>), grid, dim3(kBlock), 0, s, a);
  else if (a.mask)
    hipLaunchKernelGGL((k_ln_bwd_v<G, NV, false, true>), grid, dim3(kBlock), 0, s, a);
  else
    hipLaunchKernelGGL((k_ln_bwd_v<G, NV, false, false>), grid, dim3(kBlock), 0, s, a);
}

bool al16(const void* p, int64_t ld) { return reinterpret_cast<uintptr_t>(p) % 16 == 0 && ld % 4 == 0; }

}  // namespace

gcn_status layernorm_fwd(int64_t n, int64_t F, const float* X, int64_t ldx, double eps, float* Y,
                         int64_t ldy, float* rstd, hipStream_t s) {
  if (n == 0) return GCN_OK;
  ProfScope ps("layernorm_fwd", s);
  QuantArgs a = make_args(n, F, X, ldx, nullptr, nullptr, eps, 1, 0, Y, ldy, nullptr, 0, nullptr,
                          nullptr, 1);
  a.rstd = rstd;
  gcn_status st = GCN_OK;
  if (try_vector(a, s, &st)) return st;
  hipLaunchKernelGGL(k_ln_quantize, dim3((unsigned)ceil_div(n, kBlock / 64)), dim3(kBlock), 0, s,
                     n, (int)F, X, ldx, nullptr, nullptr, eps, 1, 0, Y, ldy, nullptr, 0, nullptr,
                     nullptr, 1, rstd);
  GCN_HIP(hipGetLastError());
  return GCN_OK;
}

gcn_status layernorm_bwd(int64_t n, int64_t F, const float* Y, int64_t ldy, const float* rstd,
                         const float* G1, int64_t ld1, const float* G2, int64_t ld2,
                         const float* mask, int64_t ldm, float* dX, int64_t lddx, hipStream_t s) {
  if (n == 0) return GCN_OK;
  ProfScope ps("layernorm_bwd", s);
  const LnBwdArgs a{n, (int)F, Y, ldy, rstd, G1, ld1, G2, ld2, mask, ldm, dX, lddx};
  const bool vec = al16(Y, ldy) && al16(G1, ld1) && (!G2 || al16(G2, ld2)) &&
                   (!mask || al16(mask, ldm)) && al16(dX, lddx) && F <= 1024 && F % 4 == 0;
  if (!vec)
    hipLaunchKernelGGL(k_ln_bwd, dim3((unsigned)ceil_div(n, kBlock / 64)), dim3(kBlock), 0, s, a);
  else if (F <= 32)
    launch_bwd_v<8, 1>(a, s);
  else if (F <= 64)
    launch_bwd_v<8, 2>(a, s);
  else if (F <= 128)
    launch_bwd_v<8, 4>(a, s);
  else if (F <= 256)
    launch_bwd_v<16, 4>(a, s);
  else if (F <= 512)
    launch_bwd_v<32, 4>(a, s);
  else
    launch_bwd_v<64, 4>(a, s);
  GCN_HIP(hipGetLastError());
  return GCN_OK;
}

}  // namespace gcn

using namespace gcn;

extern "C" gcn_status gcn_layernorm_fwd(int64_t n, int64_t F, const float* X, int64_t ldx,
                                        double eps, float* Y, int64_t ldy, float* rstd,
                                        void* stream) {
  clear_error();
  if (n < 0 || F <= 0 || F >= (1ll << 31) || !(eps >= 0.0)) {
    set_error("need n >= 0, F in [1, 2^31) and eps >= 0");
    return GCN_EINVAL;
  }
  if (n > 0 && (!X || !Y || ldx < F || ldy < F)) {
    set_error("X and Y must be non-NULL with ldx, ldy >= F");
    return GCN_EINVAL;
  }
  return layernorm_fwd(n, F, X, ldx, eps, Y, ldy, rstd, (hipStream_t)stream);
}

extern "C" gcn_status gcn_layernorm_bwd(int64_t n, int64_t F, const float* Y, int64_t ldy,
                                        const float* rstd, const float* dY, int64_t lddy,
                                        const float* dY2, int64_t lddy2, const float* mask,
                                        int64_t ldm, float* dX, int64_t lddx, void* stream) {
  clear_error();
  if (n < 0 || F <= 0 || F >= (1ll << 31)) {
    set_error("need n >= 0 and F in [1, 2^31)");
    return GCN_EINVAL;
  }
  if (n > 0 && (!Y || !rstd || !dY || !dX || ldy < F || lddy < F || lddx < F ||
                (dY2 && lddy2 < F) || (mask && ldm < F))) {
    set_error("Y, rstd, dY, dX must be non-NULL with leading dimensions >= F");
    return GCN_EINVAL;
  }
  return layernorm_bwd(n, F, Y, ldy, rstd, dY, lddy, dY2, lddy2, mask, ldm, dX, lddx,
                       (hipStream_t)stream);
}

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
  gcn_status st = GCN_OK;
  if (try_vector(make_args(n, F, X, ldx, gamma, beta, eps, (int)(flags & GCN_LAYERNORM), bits, Y,
                           ldy, Q, ldq, zmin, scale, ldp),
                 s, &st))
    return st;
  hipLaunchKernelGGL(k_ln_quantize, dim3((unsigned)ceil_div(n, kBlock / 64)), dim3(kBlock), 0, s, n,
                     (int)F, X, ldx, gamma, beta, eps, (int)(flags & GCN_LAYERNORM), bits, Y, ldy,
                     Q, ldq, zmin, scale, ldp, nullptr);
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
  gcn_status st = GCN_OK;
  if (try_vector(make_args(n, F, X, ldx, nullptr, nullptr, 0.0, 0, 8, nullptr, 0, Q, ldq, zmin,
                           scale, ldp),
                 s, &st))
    return st;
  const int64_t blocks = ceil_div(n, kBlock / 64);
  hipLaunchKernelGGL(k_quantize_rows, dim3((unsigned)blocks), dim3(kBlock), 0, s, n, (int)F, X, ldx,
                     Q, ldq, zmin, scale, ldp);
  GCN_HIP(hipGetLastError());
  return GCN_OK;
}
