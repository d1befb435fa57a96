// Aggregation kernels: Y = A_hat X, dX = A_hat^T G, and the variant whose
// halo input rows are uint8 codes dequantized on read.
//
// Paper: SuperGCN (arXiv 2411.16025) Section 4 -- the destination row is
// accumulated in registers while its (sorted, clustered) source rows stream
// past ("loop reordering", "vector register-optimized kernel"), the inner
// kernel is specialized to the feature width, and work is balanced by
// entries rather than rows ("2D dynamic parallelism", "FLOPS-based load
// balancing"). Section 6.1 step 3 and Section 2.4 define the dequantization
// h = q * S + Z fused here into the gather.
//
// Mapping to gfx950 (wave64, 16-byte lanes):
//  * A lane owns VEC consecutive features; G lanes ("a slot") cover one
//    feature tile of G*VEC floats of one row; a wavefront holds E = 64/G
//    slots. Feature tiles beyond G*VEC use blockIdx.y.
//  * Rows are binned by length (see build.hip):
//      empty rows           -> zero fill
//      1..32 entries        -> one row per slot, E rows per wavefront
//      33..medium_max       -> one wavefront per row, slots interleave entries
//      longer rows          -> one 256-thread workgroup per chunk of entries,
//                              slots reduced in fixed order through LDS; a row
//                              with several chunks writes partial rows that a
//                              last kernel sums in chunk order.
//  * Every output element is summed in an order fixed by the graph and F:
//    no atomics, identical bits on every run.
//  * Source rows are gathered with 16-byte loads; the (column, value) pair
//    of an entry is one 8-byte load; outputs use nontemporal stores so the
//    L2 and the Infinity Cache keep the gathered rows.

#include <algorithm>

#include "common.h"

namespace gcn {

namespace {

typedef float f4 __attribute__((ext_vector_type(4)));
typedef uint16_t us4 __attribute__((ext_vector_type(4)));

constexpr int kBlock = 256;
constexpr int kWavesPerBlock = kBlock / 64;

// ---- gather policies ----------------------------------------------------------

template <int VEC>
struct SrcF32 {
  const float* __restrict__ x;
  int64_t ld;
  int F;
  // features [f0, f0 + VEC) of input row j (f0 < F)
  __device__ inline void load(int32_t j, int f0, float* out) const {
    const float* p = x + (int64_t)j * ld + f0;
    if constexpr (VEC == 4) {
      if (f0 + 4 <= F) {
        const f4 v = *reinterpret_cast<const f4*>(p);
        out[0] = v.x; out[1] = v.y; out[2] = v.z; out[3] = v.w;
      } else {
#pragma unroll
        for (int v = 0; v < 4; ++v) out[v] = (f0 + v < F) ? p[v] : 0.f;
      }
    } else {
      out[0] = p[0];
    }
  }
};

__device__ inline float bf16_to_f32(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }

template <int VEC>
struct SrcBF16 {
  const uint16_t* __restrict__ x;
  int64_t ld;
  int F;
  __device__ inline void load(int32_t j, int f0, float* out) const {
    const uint16_t* p = x + (int64_t)j * ld + f0;
    if constexpr (VEC == 4) {
      if (f0 + 4 <= F) {
        const us4 v = *reinterpret_cast<const us4*>(p);
        out[0] = bf16_to_f32(v.x); out[1] = bf16_to_f32(v.y);
        out[2] = bf16_to_f32(v.z); out[3] = bf16_to_f32(v.w);
      } else {
#pragma unroll
        for (int v = 0; v < 4; ++v) out[v] = (f0 + v < F) ? bf16_to_f32(p[v]) : 0.f;
      }
    } else {
      out[0] = bf16_to_f32(p[0]);
    }
  }
};

// Input rows j < n_local are fp32; rows j >= n_local are uint8 codes with a
// per-row zero point and scale: x = fmaf(q, S, Z), exactly one rounding.
template <int VEC>
struct SrcQ8 {
  const float* __restrict__ x;
  int64_t ldx;
  int64_t n_local;
  const uint8_t* __restrict__ q;
  int64_t ldq;
  const float* __restrict__ zmin;
  const float* __restrict__ scale;
  int F;
  __device__ inline void load(int32_t j, int f0, float* out) const {
    if ((int64_t)j < n_local) {
      SrcF32<VEC>{x, ldx, F}.load(j, f0, out);
      return;
    }
    const int64_t h = (int64_t)j - n_local;
    const uint8_t* p = q + h * ldq + f0;
    const float z = zmin[h], s = scale[h];
    if constexpr (VEC == 4) {
      if (f0 + 4 <= F) {
        const uint32_t w = *reinterpret_cast<const uint32_t*>(p);
        out[0] = __builtin_fmaf((float)(w & 255u), s, z);
        out[1] = __builtin_fmaf((float)((w >> 8) & 255u), s, z);
        out[2] = __builtin_fmaf((float)((w >> 16) & 255u), s, z);
        out[3] = __builtin_fmaf((float)(w >> 24), s, z);
      } else {
#pragma unroll
        for (int v = 0; v < 4; ++v) out[v] = (f0 + v < F) ? __builtin_fmaf((float)p[v], s, z) : 0.f;
      }
    } else {
      out[0] = __builtin_fmaf((float)p[0], s, z);
    }
  }
};

// ---- helpers -------------------------------------------------------------------

template <int VEC>
__device__ inline void store_row(float* __restrict__ y, int f0, int F, const float* acc) {
  if constexpr (VEC == 4) {
    if (f0 + 4 <= F) {
      f4 v = {acc[0], acc[1], acc[2], acc[3]};
      __builtin_nontemporal_store(v, reinterpret_cast<f4*>(y + f0));
    } else {
#pragma unroll
      for (int v = 0; v < 4; ++v)
        if (f0 + v < F) __builtin_nontemporal_store(acc[v], y + f0 + v);
    }
  } else {
    __builtin_nontemporal_store(acc[0], y + f0);
  }
}

// acc += sum over k = first, first + stride, ... < end of val[k] * x[col[k]],
// in increasing k; U gathers are issued before they are consumed.
template <int VEC, int U, class Src>
__device__ inline void accumulate(const Ent* __restrict__ ent, int64_t first, int64_t end,
                                  int64_t stride, const Src& src, int f0, bool active,
                                  float* acc) {
  for (int64_t k = first; k < end; k += (int64_t)U * stride) {
    float w[U];
    float xv[U][VEC];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int64_t ku = k + (int64_t)u * stride;
      w[u] = 0.f;
#pragma unroll
      for (int v = 0; v < VEC; ++v) xv[u][v] = 0.f;
      if (ku < end) {
        const Ent e = ent[ku];
        w[u] = e.val;
        if (active) src.load(e.col, f0, xv[u]);
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      if (k + (int64_t)u * stride < end) {
#pragma unroll
        for (int v = 0; v < VEC; ++v) acc[v] = __builtin_fmaf(w[u], xv[u][v], acc[v]);
      }
    }
  }
}

// Sum the E slots of a wavefront (butterfly over lane distance G, 2G, ...).
// Every slot ends with the same total, combined in the same fixed order.
template <int VEC, int G>
__device__ inline void reduce_slots(float* acc) {
#pragma unroll
  for (int off = G; off < 64; off <<= 1) {
#pragma unroll
    for (int v = 0; v < VEC; ++v) acc[v] += __shfl_xor(acc[v], off, 64);
  }
}

struct ShortArgs {
  int64_t row_off[kLastShort - kFirstShort + 2];   // rows of short class c start at row_off[c-1]
  int64_t wave_off[kLastShort - kFirstShort + 2];  // first wavefront of each short class
};

// ---- kernels ---------------------------------------------------------------------

// Zero rows that have no entries.
template <int VEC, int G>
__global__ __launch_bounds__(kBlock) void k_zero_rows(const int32_t* __restrict__ rows,
                                                      int64_t n, float* __restrict__ y,
                                                      int64_t ldy, int F) {
  constexpr int E = 64 / G;
  const int lane = threadIdx.x & 63;
  const int64_t i = ((int64_t)blockIdx.x * kWavesPerBlock + (threadIdx.x >> 6)) * E + lane / G;
  const int f0 = (int)blockIdx.y * G * VEC + (lane % G) * VEC;
  if (i >= n || f0 >= F) return;
  float z[VEC];
#pragma unroll
  for (int v = 0; v < VEC; ++v) z[v] = 0.f;
  store_row<VEC>(y + (int64_t)rows[i] * ldy, f0, F, z);
}

// Rows with 1..32 entries: one row per slot, E rows per wavefront, the rows
// of one wavefront from one length class.
template <int VEC, int G, class Src>
__global__ __launch_bounds__(kBlock) void k_short(const int64_t* __restrict__ ptr,
                                                  const Ent* __restrict__ ent,
                                                  const int32_t* __restrict__ rows, ShortArgs sa,
                                                  Src src, float* __restrict__ y, int64_t ldy,
                                                  int F) {
  constexpr int E = 64 / G;
  constexpr int NS = kLastShort - kFirstShort + 1;
  const int lane = threadIdx.x & 63;
  const int64_t wave = (int64_t)blockIdx.x * kWavesPerBlock + (threadIdx.x >> 6);
  int c = 0;
#pragma unroll
  for (int k = 1; k < NS; ++k)
    if (wave >= sa.wave_off[k]) c = k;
  const int64_t i = sa.row_off[c] + (wave - sa.wave_off[c]) * E + lane / G;
  const int f0 = (int)blockIdx.y * G * VEC + (lane % G) * VEC;
  if (wave >= sa.wave_off[NS] || i >= sa.row_off[c + 1] || f0 >= F) return;
  const int32_t r = rows[i];
  const int64_t b = ptr[r], e = ptr[r + 1];
  float acc[VEC];
#pragma unroll
  for (int v = 0; v < VEC; ++v) acc[v] = 0.f;
  accumulate<VEC, 4>(ent, b, e, 1, src, f0, true, acc);
  store_row<VEC>(y + (int64_t)r * ldy, f0, F, acc);
}

// Rows with 33..medium_max entries: one wavefront per row.
template <int VEC, int G, class Src>
__global__ __launch_bounds__(kBlock) void k_medium(const int64_t* __restrict__ ptr,
                                                   const Ent* __restrict__ ent,
                                                   const int32_t* __restrict__ rows, int64_t n,
                                                   Src src, float* __restrict__ y, int64_t ldy,
                                                   int F) {
  constexpr int E = 64 / G;
  const int lane = threadIdx.x & 63;
  const int64_t i = (int64_t)blockIdx.x * kWavesPerBlock + (threadIdx.x >> 6);
  if (i >= n) return;  // whole wavefront leaves together
  const int slot = lane / G;
  const int f0 = (int)blockIdx.y * G * VEC + (lane % G) * VEC;
  const bool active = f0 < F;
  const int32_t r = rows[i];
  const int64_t b = ptr[r], e = ptr[r + 1];
  float acc[VEC];
#pragma unroll
  for (int v = 0; v < VEC; ++v) acc[v] = 0.f;
  accumulate<VEC, 4>(ent, b + slot, e, E, src, f0, active, acc);
  reduce_slots<VEC, G>(acc);
  if (slot == 0 && active) store_row<VEC>(y + (int64_t)r * ldy, f0, F, acc);
}

// One workgroup per chunk of a long row. The 4*E slots of the workgroup
// interleave the chunk's entries; wavefront sums meet in LDS and are added in
// wavefront order. Single-chunk rows write Y, others a partial row.
template <int VEC, int G, class Src>
__global__ __launch_bounds__(kBlock) void k_chunk(const int64_t* __restrict__ ptr,
                                                  const Ent* __restrict__ ent,
                                                  const int32_t* __restrict__ chunk_row,
                                                  const int64_t* __restrict__ chunk_beg,
                                                  const int32_t* __restrict__ chunk_part,
                                                  int64_t chunk_len, Src src,
                                                  float* __restrict__ y, int64_t ldy,
                                                  float* __restrict__ parts, int64_t ldp, int F) {
  constexpr int E = 64 / G;
  __shared__ float red[kWavesPerBlock][G * VEC];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int slot = lane / G, gl = lane % G;
  const int64_t c = blockIdx.x;
  const int32_t r = chunk_row[c];
  const int64_t beg = chunk_beg[c];
  const int64_t end = std::min(beg + chunk_len, ptr[r + 1]);
  const int f0 = (int)blockIdx.y * G * VEC + gl * VEC;
  const bool active = f0 < F;
  float acc[VEC];
#pragma unroll
  for (int v = 0; v < VEC; ++v) acc[v] = 0.f;
  accumulate<VEC, 4>(ent, beg + wave * E + slot, end, (int64_t)kWavesPerBlock * E, src, f0,
                     active, acc);
  reduce_slots<VEC, G>(acc);
  if (slot == 0) {
#pragma unroll
    for (int v = 0; v < VEC; ++v) red[wave][gl * VEC + v] = acc[v];
  }
  __syncthreads();
  if (wave == 0 && slot == 0 && active) {
#pragma unroll
    for (int v = 0; v < VEC; ++v) {
      float s = red[0][gl * VEC + v];
#pragma unroll
      for (int w = 1; w < kWavesPerBlock; ++w) s += red[w][gl * VEC + v];
      acc[v] = s;
    }
    const int32_t part = chunk_part[c];
    if (part < 0)
      store_row<VEC>(y + (int64_t)r * ldy, f0, F, acc);
    else
      store_row<VEC>(parts + (int64_t)part * ldp, f0, F, acc);
  }
}

// Sum the partial rows of each multi-chunk row in chunk order: slot s adds
// partials s, s + E, ...; the slots are then combined by the butterfly.
template <int VEC, int G>
__global__ __launch_bounds__(kBlock) void k_reduce_parts(const int32_t* __restrict__ giant_row,
                                                         const int32_t* __restrict__ part_off,
                                                         int64_t n_giant,
                                                         const float* __restrict__ parts,
                                                         int64_t ldp, float* __restrict__ y,
                                                         int64_t ldy, int F) {
  constexpr int E = 64 / G;
  const int lane = threadIdx.x & 63;
  const int64_t i = (int64_t)blockIdx.x * kWavesPerBlock + (threadIdx.x >> 6);
  if (i >= n_giant) return;
  const int slot = lane / G;
  const int f0 = (int)blockIdx.y * G * VEC + (lane % G) * VEC;
  const bool active = f0 < F;
  float acc[VEC];
#pragma unroll
  for (int v = 0; v < VEC; ++v) acc[v] = 0.f;
  if (active) {
    for (int64_t p = part_off[i] + slot; p < part_off[i + 1]; p += E) {
      const float* src = parts + p * ldp + f0;
      if constexpr (VEC == 4) {
        if (f0 + 4 <= F) {
          const f4 v4 = *reinterpret_cast<const f4*>(src);
          acc[0] += v4.x; acc[1] += v4.y; acc[2] += v4.z; acc[3] += v4.w;
        } else {
#pragma unroll
          for (int v = 0; v < 4; ++v)
            if (f0 + v < F) acc[v] += src[v];
        }
      } else {
        acc[0] += src[0];
      }
    }
  }
  reduce_slots<VEC, G>(acc);
  if (slot == 0 && active) store_row<VEC>(y + (int64_t)giant_row[i] * ldy, f0, F, acc);
}

// ---- launch ------------------------------------------------------------------------

inline unsigned blocks_for_waves(int64_t waves) {
  return (unsigned)std::max<int64_t>(1, ceil_div(waves, kWavesPerBlock));
}

template <int VEC, int G, class Src>
gcn_status launch_all(const Mat& m, const Src& src, float* y, int64_t ldy, int F,
                      hipStream_t stream) {
  constexpr int E = 64 / G;
  const Plan& p = m.plan;
  const unsigned tiles = (unsigned)ceil_div(F, G * VEC);
  // empty rows
  const int64_t n_empty = p.class_off[kClassEmpty + 1] - p.class_off[kClassEmpty];
  if (n_empty > 0) {
    ProfScope ps("agg_zero_rows", stream);
    hipLaunchKernelGGL((k_zero_rows<VEC, G>), dim3(blocks_for_waves(ceil_div(n_empty, E)), tiles),
                       dim3(kBlock), 0, stream, (const int32_t*)(p.rows + p.class_off[kClassEmpty]),
                       n_empty, y, ldy, F);
    GCN_HIP(hipGetLastError());
  }
  // short rows
  ShortArgs sa;
  int64_t waves = 0;
  for (int c = kFirstShort; c <= kLastShort + 1; ++c) {
    sa.row_off[c - kFirstShort] = p.class_off[c];
    sa.wave_off[c - kFirstShort] = waves;
    if (c <= kLastShort) waves += ceil_div(p.class_off[c + 1] - p.class_off[c], E);
  }
  if (waves > 0) {
    ProfScope ps("agg_short", stream);
    hipLaunchKernelGGL((k_short<VEC, G, Src>), dim3(blocks_for_waves(waves), tiles), dim3(kBlock),
                       0, stream, (const int64_t*)m.ptr, (const Ent*)m.ent,
                       (const int32_t*)p.rows, sa, src, y, ldy, F);
    GCN_HIP(hipGetLastError());
  }
  // medium rows
  const int64_t n_med = p.class_off[kMedium + 1] - p.class_off[kMedium];
  if (n_med > 0) {
    ProfScope ps("agg_medium", stream);
    hipLaunchKernelGGL((k_medium<VEC, G, Src>), dim3(blocks_for_waves(n_med), tiles), dim3(kBlock),
                       0, stream, (const int64_t*)m.ptr, (const Ent*)m.ent,
                       (const int32_t*)(p.rows + p.class_off[kMedium]), n_med, src, y, ldy, F);
    GCN_HIP(hipGetLastError());
  }
  // long rows
  if (p.n_chunks > 0) {
    float* parts = nullptr;
    const int64_t ldp = (F + 3) & ~3;
    if (p.n_parts > 0) GCN_CHECK(talloc(&parts, p.n_parts * ldp, stream, "partial rows"));
    {
      ProfScope ps("agg_chunk", stream);
      hipLaunchKernelGGL((k_chunk<VEC, G, Src>), dim3((unsigned)p.n_chunks, tiles), dim3(kBlock), 0,
                         stream, (const int64_t*)m.ptr, (const Ent*)m.ent,
                         (const int32_t*)p.chunk_row, (const int64_t*)p.chunk_beg,
                         (const int32_t*)p.chunk_part, p.chunk_len, src, y, ldy, parts, ldp, F);
      hipError_t e = hipGetLastError();
      if (e != hipSuccess) {
        tfree(parts, stream);
        return hip_fail(e, "k_chunk", __FILE__, __LINE__);
      }
    }
    if (p.n_giant > 0) {
      ProfScope ps("agg_reduce_parts", stream);
      hipLaunchKernelGGL((k_reduce_parts<VEC, G>), dim3(blocks_for_waves(p.n_giant), tiles),
                         dim3(kBlock), 0, stream, (const int32_t*)p.giant_row,
                         (const int32_t*)p.giant_part_off, p.n_giant, (const float*)parts, ldp, y,
                         ldy, F);
      hipError_t e = hipGetLastError();
      if (e != hipSuccess) {
        tfree(parts, stream);
        return hip_fail(e, "k_reduce_parts", __FILE__, __LINE__);
      }
    }
    tfree(parts, stream);
  }
  return GCN_OK;
}

// Lanes per slot: smallest power of two covering min(F, 256) features with
// 4-float lanes (at least 4 lanes); the scalar path always uses 64 lanes.
int lanes_for(int F, bool vec4) {
  if (!vec4) return 64;
  const int need = (std::min(F, 256) + 3) / 4;
  int g = 4;
  while (g < need) g <<= 1;
  return g;
}

template <template <int> class SrcT, class Make>
gcn_status dispatch(const Mat& m, bool vec4, int F, float* y, int64_t ldy, hipStream_t stream,
                    Make make) {
  if (!vec4) return launch_all<1, 64>(m, make(SrcT<1>{}), y, ldy, F, stream);
  switch (lanes_for(F, true)) {
    case 4: return launch_all<4, 4>(m, make(SrcT<4>{}), y, ldy, F, stream);
    case 8: return launch_all<4, 8>(m, make(SrcT<4>{}), y, ldy, F, stream);
    case 16: return launch_all<4, 16>(m, make(SrcT<4>{}), y, ldy, F, stream);
    case 32: return launch_all<4, 32>(m, make(SrcT<4>{}), y, ldy, F, stream);
    default: return launch_all<4, 64>(m, make(SrcT<4>{}), y, ldy, F, stream);
  }
}

bool aligned(const void* p, uintptr_t a) { return ((uintptr_t)p % a) == 0; }

gcn_status check_common(const gcn_graph* g, int64_t F) {
  GCN_CHECK(check_graph(g));
  if (F <= 0 || F >= (1ll << 31)) {
    set_error("F must be in [1, 2^31) (got %lld)", (long long)F);
    return GCN_EINVAL;
  }
  return GCN_OK;
}

gcn_status aggregate(const gcn_graph* g, const Mat& m, const void* X, int64_t ldx, int dtype,
                     float* Y, int64_t ldy, int64_t F, void* stream) {
  if (!X || !Y) {
    set_error("input and output pointers must be non-NULL");
    return GCN_EINVAL;
  }
  if (ldx < F || ldy < F) {
    set_error("leading dimensions must be >= F (ldx=%lld ldy=%lld F=%lld)", (long long)ldx,
              (long long)ldy, (long long)F);
    return GCN_EINVAL;
  }
  if (dtype != GCN_DT_F32 && dtype != GCN_DT_BF16) {
    set_error("unknown dtype %d", dtype);
    return GCN_EINVAL;
  }
  const int Fi = (int)F;
  hipStream_t s = (hipStream_t)stream;
  const bool yvec = aligned(Y, 16) && ldy % 4 == 0;
  if (dtype == GCN_DT_F32) {
    const bool vec4 = yvec && aligned(X, 16) && ldx % 4 == 0;
    return dispatch<SrcF32>(m, vec4, Fi, Y, ldy, s, [&](auto t) {
      t.x = (const float*)X;
      t.ld = ldx;
      t.F = Fi;
      return t;
    });
  }
  const bool vec4 = yvec && aligned(X, 8) && ldx % 4 == 0;
  return dispatch<SrcBF16>(m, vec4, Fi, Y, ldy, s, [&](auto t) {
    t.x = (const uint16_t*)X;
    t.ld = ldx;
    t.F = Fi;
    return t;
  });
}

}  // namespace

}  // namespace gcn

using namespace gcn;

extern "C" gcn_status gcn_aggregate_fwd(const gcn_graph* g, const void* X, int64_t ldx, int dtype,
                                        float* Y, int64_t ldy, int64_t F, void* stream) {
  clear_error();
  GCN_CHECK(check_common(g, F));
  return aggregate(g, g->csr, X, ldx, dtype, Y, ldy, F, stream);
}

extern "C" gcn_status gcn_aggregate_bwd(const gcn_graph* g, const void* G, int64_t ldg, int dtype,
                                        float* dX, int64_t lddx, int64_t F, void* stream) {
  clear_error();
  GCN_CHECK(check_common(g, F));
  return aggregate(g, g->csc, G, ldg, dtype, dX, lddx, F, stream);
}

extern "C" gcn_status gcn_aggregate_fwd_q8halo(const gcn_graph* g, int64_t n_local_cols,
                                               const float* X_local, int64_t ldx,
                                               const uint8_t* Q_halo, int64_t ldq,
                                               const float* halo_min, const float* halo_scale,
                                               float* Y, int64_t ldy, int64_t F, uint32_t flags,
                                               void* stream) {
  clear_error();
  GCN_CHECK(check_common(g, F));
  if (flags & ~(uint32_t)GCN_Q8_USE_CSC) {
    set_error("unknown q8halo flag bits 0x%x", flags);
    return GCN_EINVAL;
  }
  const Mat& m = (flags & GCN_Q8_USE_CSC) ? g->csc : g->csr;
  const int64_t n_in = m.n_minor;
  if (n_local_cols < 0 || n_local_cols > n_in) {
    set_error("n_local_cols=%lld outside [0, %lld]", (long long)n_local_cols, (long long)n_in);
    return GCN_ERANGE;
  }
  if (!Y || ldy < F) {
    set_error("Y must be non-NULL with ldy >= F");
    return GCN_EINVAL;
  }
  if (n_local_cols > 0 && (!X_local || ldx < F)) {
    set_error("X_local must be non-NULL with ldx >= F when n_local_cols > 0");
    return GCN_EINVAL;
  }
  if (n_local_cols < n_in && (!Q_halo || !halo_min || !halo_scale || ldq < F)) {
    set_error("Q_halo, halo_min, halo_scale must be non-NULL with ldq >= F when halo rows exist");
    return GCN_EINVAL;
  }
  const int Fi = (int)F;
  const bool vec4 = aligned(Y, 16) && ldy % 4 == 0 && (n_local_cols == 0 ||
                    (aligned(X_local, 16) && ldx % 4 == 0)) &&
                    (n_local_cols == n_in || (aligned(Q_halo, 4) && ldq % 4 == 0));
  return dispatch<SrcQ8>(m, vec4, Fi, Y, ldy, (hipStream_t)stream, [&](auto t) {
    t.x = X_local;
    t.ldx = ldx;
    t.n_local = n_local_cols;
    t.q = Q_halo;
    t.ldq = ldq;
    t.zmin = halo_min;
    t.scale = halo_scale;
    t.F = Fi;
    return t;
  });
}
