// Aggregation kernels: Y = A_hat X, dX = A_hat^T G, and the variant whose
// halo input rows are 8-bit or 2-bit codes dequantized on read.
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
//  * Rows are binned by length (see build.hip), and within the bins of 3 or
//    more entries ordered by decreasing length:
//      empty rows           -> zero fill
//      1 or 2 entries       -> one row per slot, several row groups per
//                              wavefront with all their loads issued first
//      3..medium_max        -> one row per slot, E rows of about the same
//                              length per wavefront (k_short)
//      longer rows, on matrices of 2^20 or more columns
//                           -> cut where their columns cross one of 64 column
//                              blocks and into pieces of at most 256 entries;
//                              one piece per slot, launched block by block so
//                              the wavefronts in flight gather from one column
//                              range (k_pieces); every piece writes a partial
//                              row
//      longer rows, on smaller matrices
//                           -> one 256-thread workgroup per chunk of entries,
//                              slots reduced in fixed order through LDS; a row
//                              with several chunks writes partial rows
//                              (k_chunk)
//    A last kernel sums each cut row's partial rows in a fixed order
//    (k_reduce_parts).
//  * Every output element is summed in an order fixed by the graph and F:
//    no atomics, identical bits on every run.
//  * Source rows are gathered with 16-byte loads; the (column, value) pair
//    of an entry is one 8-byte load; outputs use nontemporal stores so the
//    L2 and the Infinity Cache keep the gathered rows.

#include <algorithm>
#include <mutex>

#include "common.h"

namespace gcn {

namespace {

typedef float f4 __attribute__((ext_vector_type(4)));
typedef float f2 __attribute__((ext_vector_type(2)));
typedef uint16_t us4 __attribute__((ext_vector_type(4)));

constexpr int kBlock = 256;
constexpr int kWavesPerBlock = kBlock / 64;

// ---- gather policies ----------------------------------------------------------

// Every policy splits a gather into fetch (issue the loads of features
// [f0, f0 + VEC) of input row j into raw registers) and decode (turn the raw
// registers into fp32 values). A loop issues the fetches of a whole group of
// entries before it decodes any of them, so no load waits on the arithmetic
// of another. TAIL = false promises F % VEC == 0: every fetch is then one
// unguarded vector load, and clamp() moves a lane's f0 past the row end back
// into the row, so a loop may fetch on every lane and discard the values of
// lanes or entries it does not use (no divergent branches around the loads).
// TAIL = true guards each feature against F instead.

template <int VEC, bool TAIL>
struct SrcF32 {
  const float* __restrict__ x;
  uint32_t ld;  // row strides fit 32 bits (checked on the host): one 32 x 32 -> 64-bit multiply
  int F;
  struct Raw {
    float v[VEC];
  };
  __device__ inline int clamp(int f0) const { return TAIL || f0 <= F - VEC ? f0 : F - VEC; }
  __device__ inline void fetch(int32_t j, int f0, Raw& r) const {
    const float* p = x + (uint64_t)(uint32_t)j * ld + f0;
    if constexpr (VEC == 4) {
      if (!TAIL || f0 + 4 <= F) {
        const f4 v = *reinterpret_cast<const f4*>(p);
        r.v[0] = v.x; r.v[1] = v.y; r.v[2] = v.z; r.v[3] = v.w;
      } else {
#pragma unroll
        for (int v = 0; v < 4; ++v) r.v[v] = (f0 + v < F) ? p[v] : 0.f;
      }
    } else {
      r.v[0] = p[0];
    }
  }
  __device__ inline void decode(const Raw& r, int32_t, float* out) const {
#pragma unroll
    for (int v = 0; v < VEC; ++v) out[v] = r.v[v];
  }
};

__device__ inline float bf16_to_f32(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }

template <int VEC, bool TAIL>
struct SrcBF16 {
  const uint16_t* __restrict__ x;
  uint32_t ld;
  int F;
  struct Raw {
    uint16_t v[VEC];
  };
  __device__ inline int clamp(int f0) const { return TAIL || f0 <= F - VEC ? f0 : F - VEC; }
  __device__ inline void fetch(int32_t j, int f0, Raw& r) const {
    const uint16_t* p = x + (uint64_t)(uint32_t)j * ld + f0;
    if constexpr (VEC == 4) {
      if (!TAIL || f0 + 4 <= F) {
        const us4 v = *reinterpret_cast<const us4*>(p);
        r.v[0] = v.x; r.v[1] = v.y; r.v[2] = v.z; r.v[3] = v.w;
      } else {
#pragma unroll
        for (int v = 0; v < 4; ++v) r.v[v] = (f0 + v < F) ? p[v] : (uint16_t)0;
      }
    } else {
      r.v[0] = p[0];
    }
  }
  __device__ inline void decode(const Raw& r, int32_t, float* out) const {
#pragma unroll
    for (int v = 0; v < VEC; ++v) out[v] = bf16_to_f32(r.v[v]);
  }
};

// Input rows j < n_local are fp32; rows j >= n_local are BITS-bit codes (8:
// one byte per feature; 2: four per byte) with a per-row zero point and
// scale: x = fmaf(q, S, Z), exactly one rounding. A halo row's raw registers
// hold the packed codes, Z and S in the slots a local row uses for its
// features, so both kinds cost the same registers (separate registers cost
// occupancy and time).
template <int VEC, int BITS, bool TAIL>
struct SrcQ {
  const float* __restrict__ x;
  uint32_t ldx;
  uint32_t n_local;
  const uint8_t* __restrict__ q;
  uint32_t ldq;
  const float* __restrict__ zmin;
  const float* __restrict__ scale;
  uint32_t ldp;
  int F;
  struct Raw {
    float v[VEC < 3 ? 3 : VEC];  // local: features; halo: {codes, Z, S}
  };
  __device__ inline int clamp(int f0) const { return TAIL || f0 <= F - VEC ? f0 : F - VEC; }
  __device__ inline void fetch(int32_t j, int f0, Raw& r) const {
    if ((uint32_t)j < n_local) {
      typename SrcF32<VEC, TAIL>::Raw fr;
      SrcF32<VEC, TAIL>{x, ldx, F}.fetch(j, f0, fr);
#pragma unroll
      for (int v = 0; v < VEC; ++v) r.v[v] = fr.v[v];
      return;
    }
    const uint32_t h = (uint32_t)j - n_local;
    const uint8_t* qrow = q + (uint64_t)h * ldq;
    const uint64_t po = (uint64_t)h * ldp;
    const uint8_t* p = qrow + f0;
    r.v[1] = zmin[po];
    r.v[2] = scale[po];
    uint32_t c;
    if constexpr (BITS == 2) {
      // byte f0 / 4 holds the codes of features f0 .. f0 + 3 (VEC = 4: f0 % 4 == 0)
      const uint32_t byte = qrow[f0 >> 2];
      c = VEC == 4 ? byte : (byte >> (2 * (f0 & 3))) & 3u;
    } else if constexpr (VEC == 4) {
      if (!TAIL || f0 + 4 <= F) {
        c = *reinterpret_cast<const uint32_t*>(p);
      } else {
        c = 0;
#pragma unroll
        for (int v = 0; v < 4; ++v)
          if (f0 + v < F) c |= (uint32_t)p[v] << (8 * v);
      }
    } else {
      c = p[0];
    }
    r.v[0] = __uint_as_float(c);
  }
  __device__ inline void decode(const Raw& r, int32_t j, float* out) const {
    if ((uint32_t)j >= n_local) {
      const uint32_t c = __float_as_uint(r.v[0]);
      constexpr int w = BITS;
      constexpr uint32_t m = (1u << BITS) - 1u;
#pragma unroll
      for (int v = 0; v < VEC; ++v)
        out[v] = __builtin_fmaf((float)((c >> (w * v)) & m), r.v[2], r.v[1]);
    } else {
#pragma unroll
      for (int v = 0; v < VEC; ++v) out[v] = r.v[v];
    }
  }
};

template <int VEC, bool TAIL>
using SrcQ8 = SrcQ<VEC, 8, TAIL>;
template <int VEC, bool TAIL>
using SrcQ2 = SrcQ<VEC, 2, TAIL>;

// ---- helpers -------------------------------------------------------------------

// Store a finished output row tile; relu clamps it at 0 (the activation of a
// layer fused into the aggregation that produces it).
template <int VEC, bool RELU = false>
__device__ inline void store_row(float* __restrict__ y, int f0, int F, const float* acc_in) {
  float acc[VEC];
#pragma unroll
  for (int v = 0; v < VEC; ++v) acc[v] = RELU ? fmaxf(acc_in[v], 0.f) : acc_in[v];
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

// Gathers in flight per lane in the entry loops.
#ifndef GCN_AGG_UNROLL
#define GCN_AGG_UNROLL 3
#endif
// Unroll factor of the loop over gather groups inside a 64-entry block (1
// keeps the register count, and so the occupancy, of one group).
#ifndef GCN_GROUP_UNROLL
#define GCN_GROUP_UNROLL 1
#endif
// Row groups per wavefront of the one-entry and two-entry row kernels.
#ifndef GCN_TINY_GROUPS1
#define GCN_TINY_GROUPS1 4
#endif
#ifndef GCN_TINY_GROUPS2
#define GCN_TINY_GROUPS2 2
#endif
// Waves per SIMD the entry-loop kernels must fit (caps their registers).
#ifndef GCN_MIN_WAVES
#define GCN_MIN_WAVES 8
#endif
#ifndef GCN_PIECE_MIN_WAVES
#define GCN_PIECE_MIN_WAVES GCN_MIN_WAVES
#endif
// Gathers in flight per lane in the one-run-per-slot loops of k_short and
// k_pieces.
#ifndef GCN_SLOT_UNROLL
#define GCN_SLOT_UNROLL 4
#endif
#ifndef GCN_PIECE_UNROLL
#define GCN_PIECE_UNROLL GCN_SLOT_UNROLL
#endif
#define GCN_PRAGMA(x) _Pragma(#x)
#define GCN_UNROLL_N(n) GCN_PRAGMA(unroll n)

// One (column, value) pair, loaded without keeping it in the caches: the
// entry stream is read once per pass, so L2 and the Infinity Cache are left
// to the gathered feature rows, which hub columns reuse.
__device__ inline Ent load_ent(const Ent* p) {
  const uint64_t raw = __builtin_nontemporal_load(reinterpret_cast<const uint64_t*>(p));
  Ent e;
  e.col = (int32_t)(uint32_t)raw;
  e.val = __uint_as_float((uint32_t)(raw >> 32));
  return e;
}

// One wavefront adds val[k] * x[col[k]] for the entries k of [beg, end) in
// 64-entry blocks starting at beg + 64 * (first + j * stride), j = 0, 1, ...
// The 64 lanes load a block's (column, value) pairs with one coalesced
// access, and the next block's load is issued before this block's gathers;
// slot s takes block positions s, s + E, s + 2E, ... through lane shuffles,
// with U row gathers in flight per lane. A slot's terms are added in
// increasing entry order.
template <int VEC, int G, int U, class Src>
__device__ inline void accumulate_blocks(const Ent* __restrict__ ent, int64_t beg, int64_t end,
                                         int64_t first, int64_t stride, const Src& src, int f0,
                                         bool active, float* acc) {
  constexpr int E = 64 / G;
  constexpr int UU = U < G ? U : G;
  const int lane = threadIdx.x & 63;
  const int slot = lane / G;
  const int fs = src.clamp(f0);
  int64_t base = beg + first * 64;
  const int64_t step = stride * 64;
  Ent cur = {0, 0.f};
  if (base + lane < end) cur = load_ent(ent + base + lane);
  while (base < end) {
    const int64_t nbase = base + step;
    Ent nxt = {0, 0.f};
    const int n = (int)((end - base) < 64 ? (end - base) : 64);
    GCN_UNROLL_N(GCN_GROUP_UNROLL)
    for (int p0 = 0; p0 < G; p0 += UU) {
      if (p0 * E >= n) break;
      float w[UU];
      int32_t col[UU];
      typename Src::Raw raw[UU];
#pragma unroll
      for (int u = 0; u < UU; ++u) {  // positions past n read row 0 (see accumulate_slot)
        const int pos = (p0 + u) * E + slot;
        col[u] = __shfl(cur.col, pos, 64);
        w[u] = __shfl(cur.val, pos, 64);
        src.fetch(col[u], fs, raw[u]);
      }
      // the next block's pairs travel with the first group's gathers
      if (p0 == 0 && nbase + lane < end) nxt = load_ent(ent + nbase + lane);
#pragma unroll
      for (int u = 0; u < UU; ++u) {
        float xv[VEC];
        src.decode(raw[u], col[u], xv);
        const bool ok = (p0 + u) * E + slot < n && active;
#pragma unroll
        for (int v = 0; v < VEC; ++v) {
          const float t = __builtin_fmaf(w[u], xv[v], acc[v]);
          acc[v] = ok ? t : acc[v];
        }
      }
    }
    cur = nxt;
    base = nbase;
  }
}

// Slot s of a wavefront (lanes sG .. sG + G - 1) sums the len entries of
// the run starting at entry b; acc receives the slot's features f0 .. f0 +
// VEC - 1. The G lanes load the pairs G at a time with one coalesced access
// (the next G travel with the current gathers) and share them by lane
// shuffles; the loop bound is the wavefront's longest run, so every lane runs
// the same iterations (all lanes of the wavefront must call this). Every
// lane fetches on every iteration, positions past its run reading row 0
// (a valid row whenever the matrix has entries) and lanes past F a clamped
// feature offset, and a select drops those terms, so the loads are never
// split by divergent branches. Terms are added in entry order.
template <int VEC, int G, int U, class Src>
__device__ inline void accumulate_slot(const Ent* __restrict__ ent, int64_t b, int len,
                                       const Src& src, int f0, bool active, float* acc) {
  const int lane = threadIdx.x & 63;
  const int slot = lane / G, gl = lane % G;
  const int fs = src.clamp(f0);
#pragma unroll
  for (int v = 0; v < VEC; ++v) acc[v] = 0.f;
  int hi = len;  // the wavefront's longest run
#pragma unroll
  for (int off = G; off < 64; off <<= 1) hi = max(hi, __shfl_xor(hi, off, 64));
  Ent me = {0, 0.f};
  if (gl < len) me = load_ent(ent + b + gl);
  for (int p0 = 0; p0 < hi; p0 += G) {
    Ent nx = {0, 0.f};
    if (p0 + G + gl < len) nx = load_ent(ent + b + p0 + G + gl);
    const int np = (hi - p0) < G ? (hi - p0) : G;
    const int nv = active ? len - p0 : 0;  // this slot's terms in the block (may be <= 0)
    for (int p = 0; p < np; p += U) {
      float w[U];
      int32_t col[U];
      typename Src::Raw raw[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int pos = (p + u) < G ? (p + u) : (G - 1);
        col[u] = __shfl(me.col, slot * G + pos, 64);
        w[u] = __shfl(me.val, slot * G + pos, 64);
        src.fetch(col[u], fs, raw[u]);
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        float xv[VEC];
        src.decode(raw[u], col[u], xv);
        const bool ok = p + u < nv;
#pragma unroll
        for (int v = 0; v < VEC; ++v) {
          const float t = __builtin_fmaf(w[u], xv[v], acc[v]);
          acc[v] = ok ? t : acc[v];
        }
      }
    }
    me = nx;
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

// Classes run one row per lane group by k_short: kFirstShort .. kMedium (the
// one- and two-entry classes get no wavefronts there).
constexpr int kSlotClasses = kMedium - kFirstShort + 1;
struct ShortArgs {
  int64_t row_off[kSlotClasses + 1];   // rows of class kFirstShort + k start at row_off[k]
  int64_t wave_off[kSlotClasses + 1];  // first wavefront of each class; [kSlotClasses] = total
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

// Rows with exactly L entries (L = 1 or 2): one row per slot and R groups of
// E rows per wavefront, every load of the R groups issued before any
// arithmetic. Such rows have no other work to hide their chain of dependent
// loads (row id and start, entries, feature rows) behind, so the wavefront
// keeps R * L gathers per lane in flight instead of L; the plan stores their
// starts next to their ids (beg[i] for rows[i]). The terms of a row are added
// in entry order, as in k_short.
template <int VEC, int G, class Src, bool RELU, int L, int R>
__global__ __launch_bounds__(kBlock, GCN_MIN_WAVES) void k_tiny(const int64_t* __restrict__ beg,
                                                  const Ent* __restrict__ ent,
                                                  const int32_t* __restrict__ rows, int64_t n,
                                                  Src src, float* __restrict__ y, int64_t ldy,
                                                  int F) {
  constexpr int E = 64 / G;
  const int lane = threadIdx.x & 63;
  const int slot = lane / G;
  const int64_t wave = (int64_t)blockIdx.x * kWavesPerBlock + (threadIdx.x >> 6);
  const int f0 = (int)blockIdx.y * G * VEC + (lane % G) * VEC;
  const bool fa = f0 < F;
  const int fs = src.clamp(f0);
  // slots past the last row repeat it and lanes past F read a clamped offset
  // (see accumulate_slot), so every load is issued unconditionally
  int32_t r[R];
  int64_t b[R];
  bool has[R];
#pragma unroll
  for (int g = 0; g < R; ++g) {
    const int64_t i = (wave * R + g) * E + slot;
    has[g] = i < n;
    const int64_t ic = has[g] ? i : n - 1;
    r[g] = rows[ic];
    b[g] = beg[ic];
  }
  Ent e[R][L];
#pragma unroll
  for (int g = 0; g < R; ++g)
#pragma unroll
    for (int k = 0; k < L; ++k) e[g][k] = load_ent(ent + b[g] + k);
  typename Src::Raw raw[R][L];
#pragma unroll
  for (int g = 0; g < R; ++g)
#pragma unroll
    for (int k = 0; k < L; ++k) src.fetch(e[g][k].col, fs, raw[g][k]);
#pragma unroll
  for (int g = 0; g < R; ++g) {
    if (!(has[g] && fa)) continue;
    float acc[VEC];
#pragma unroll
    for (int v = 0; v < VEC; ++v) acc[v] = 0.f;
#pragma unroll
    for (int k = 0; k < L; ++k) {
      float xv[VEC];
      src.decode(raw[g][k], e[g][k].col, xv);
#pragma unroll
      for (int v = 0; v < VEC; ++v) acc[v] = __builtin_fmaf(e[g][k].val, xv[v], acc[v]);
    }
    store_row<VEC, RELU>(y + (int64_t)r[g] * ldy, f0, F, acc);
  }
}

// Rows of 3 .. medium_max entries: one row per slot (accumulate_slot), E rows
// per wavefront, the rows of one wavefront from one length class and, within
// it, of about the same length (the plan orders them by decreasing length).
template <int VEC, int G, class Src, bool RELU>
__global__ __launch_bounds__(kBlock, GCN_MIN_WAVES) void k_short(const int64_t* __restrict__ rbeg,
                                                  const int32_t* __restrict__ rlen,
                                                  const Ent* __restrict__ ent,
                                                  const int32_t* __restrict__ rows, ShortArgs sa,
                                                  Src src, float* __restrict__ y, int64_t ldy,
                                                  int F) {
  constexpr int E = 64 / G;
  constexpr int NS = kSlotClasses;
  const int lane = threadIdx.x & 63;
  const int slot = lane / G, gl = lane % G;
  const int64_t wave = (int64_t)blockIdx.x * kWavesPerBlock + (threadIdx.x >> 6);
  if (wave >= sa.wave_off[NS]) return;  // whole wavefront leaves together
  int c = 0;
#pragma unroll
  for (int k = 1; k < NS; ++k)
    if (wave >= sa.wave_off[k]) c = k;
  const int64_t i = sa.row_off[c] + (wave - sa.wave_off[c]) * E + slot;
  const int f0 = (int)blockIdx.y * G * VEC + gl * VEC;
  const bool has_row = i < sa.row_off[c + 1];
  const bool active = has_row && f0 < F;
  int32_t r = 0;
  int64_t b = 0;
  int len = 0;
  if (has_row) {  // start and length come with the row id (rbeg, rlen follow rows from row_off[0])
    r = rows[i];
    b = rbeg[i - sa.row_off[0]];
    len = rlen[i - sa.row_off[0]];
  }
  float acc[VEC];
  accumulate_slot<VEC, G, GCN_SLOT_UNROLL>(ent, b, len, src, f0, active, acc);
  if (active) store_row<VEC, RELU>(y + (int64_t)r * ldy, f0, F, acc);
}

// One workgroup per chunk of a long row. Wavefront w of the workgroup takes
// the chunk's 64-entry blocks w, w + 4, w + 8, ...; wavefront sums meet in
// LDS and are added in wavefront order. Single-chunk rows write Y, others a
// partial row.
template <int VEC, int G, class Src, bool RELU>
__global__ __launch_bounds__(kBlock, GCN_MIN_WAVES) void k_chunk(const Ent* __restrict__ ent,
                                                  const int32_t* __restrict__ chunk_row,
                                                  const int64_t* __restrict__ chunk_beg,
                                                  const int64_t* __restrict__ chunk_end,
                                                  const int32_t* __restrict__ chunk_part, Src src,
                                                  float* __restrict__ y, int64_t ldy,
                                                  float* __restrict__ parts, int64_t ldp, int F) {
  __shared__ float red[kWavesPerBlock][G * VEC];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int slot = lane / G, gl = lane % G;
  const int64_t c = blockIdx.x;
  const int32_t r = chunk_row[c];
  const int64_t beg = chunk_beg[c];
  const int64_t end = chunk_end[c];
  const int f0 = (int)blockIdx.y * G * VEC + gl * VEC;
  const bool active = f0 < F;
  float acc[VEC];
#pragma unroll
  for (int v = 0; v < VEC; ++v) acc[v] = 0.f;
  accumulate_blocks<VEC, G, GCN_AGG_UNROLL>(ent, beg, end, wave, kWavesPerBlock, src, f0, active,
                                            acc);
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
      store_row<VEC, RELU>(y + (int64_t)r * ldy, f0, F, acc);
    else
      store_row<VEC>(parts + (int64_t)part * ldp, f0, F, acc);
  }
}

// Column-blocked pieces (at most piece_max entries each), one per slot, in
// the plan's launch order (column block by column block, decreasing length
// within a block); each writes its partial row.
template <int VEC, int G, class Src>
__global__ __launch_bounds__(kBlock, GCN_PIECE_MIN_WAVES)
void k_pieces(const int64_t* __restrict__ pbeg, const int32_t* __restrict__ plen,
              const int32_t* __restrict__ ppart, int64_t n, const Ent* __restrict__ ent, Src src,
              float* __restrict__ parts, int64_t ldp, int F) {
  constexpr int E = 64 / G;
  const int lane = threadIdx.x & 63;
  const int slot = lane / G, gl = lane % G;
  const int64_t wave = (int64_t)blockIdx.x * kWavesPerBlock + (threadIdx.x >> 6);
  if (wave * E >= n) return;  // whole wavefront leaves together
  const int64_t i = wave * E + slot;
  const bool has = i < n;
  const int f0 = (int)blockIdx.y * G * VEC + gl * VEC;
  const bool active = has && f0 < F;
  const int64_t b = has ? pbeg[i] : 0;
  const int len = has ? plen[i] : 0;
  float acc[VEC];
  accumulate_slot<VEC, G, GCN_PIECE_UNROLL>(ent, b, len, src, f0, active, acc);
  if (active) store_row<VEC>(parts + (int64_t)ppart[i] * ldp, f0, F, acc);
}

// Features f0 .. f0 + VEC - 1 of a partial row (zeros past F).
template <int VEC>
__device__ inline void load_part(const float* __restrict__ row, int f0, int F, float* out) {
  if constexpr (VEC == 4) {
    if (f0 + 4 <= F) {
      const f4 v4 = *reinterpret_cast<const f4*>(row + f0);
      out[0] = v4.x; out[1] = v4.y; out[2] = v4.z; out[3] = v4.w;
    } else {
#pragma unroll
      for (int v = 0; v < 4; ++v) out[v] = f0 + v < F ? row[f0 + v] : 0.f;
    }
  } else {
    out[0] = row[f0];
  }
}

// Sum the partial rows of each multi-chunk row in chunk order: slot s adds
// partials s, s + E, ...; the slots are then combined by the butterfly.
template <int VEC, int G, bool RELU>
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
    // U partial rows in flight per lane; each slot still adds its partials
    // in increasing slot order
    constexpr int U = 4;
    const int64_t pe = part_off[i + 1];
    int64_t p = part_off[i] + slot;
    for (; p + (U - 1) * E < pe; p += U * E) {
      float v[U][VEC];
#pragma unroll
      for (int u = 0; u < U; ++u) load_part<VEC>(parts + (p + u * E) * ldp, f0, F, v[u]);
#pragma unroll
      for (int u = 0; u < U; ++u)
#pragma unroll
        for (int k = 0; k < VEC; ++k) acc[k] += v[u][k];
    }
    for (; p < pe; p += E) {
      float v[VEC];
      load_part<VEC>(parts + p * ldp, f0, F, v);
#pragma unroll
      for (int k = 0; k < VEC; ++k) acc[k] += v[k];
    }
  }
  reduce_slots<VEC, G>(acc);
  if (slot == 0 && active) store_row<VEC, RELU>(y + (int64_t)giant_row[i] * ldy, f0, F, acc);
}

// ---- launch ------------------------------------------------------------------------

inline unsigned blocks_for_waves(int64_t waves) {
  return (unsigned)std::max<int64_t>(1, ceil_div(waves, kWavesPerBlock));
}

// ws: caller-provided room for the partial rows (at least parts_floats(m, F)
// floats), or NULL to allocate them stream-ordered for the call.
template <int VEC, int G, bool RELU, class Src>
gcn_status launch_all(const Mat& m, const Src& src, float* y, int64_t ldy, int F,
                      hipStream_t stream, float* ws) {
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
  // rows of exactly one and exactly two entries
  {
    const int64_t n1 = p.class_off[kFirstShort + 1] - p.class_off[kFirstShort];
    const int64_t n2 = p.class_off[kFirstShort + 2] - p.class_off[kFirstShort + 1];
    constexpr int R1 = GCN_TINY_GROUPS1, R2 = GCN_TINY_GROUPS2;
    if (n1 > 0) {
      ProfScope ps("agg_tiny", stream);
      hipLaunchKernelGGL((k_tiny<VEC, G, Src, RELU, 1, R1>),
                         dim3(blocks_for_waves(ceil_div(n1, E * R1)), tiles), dim3(kBlock), 0,
                         stream, (const int64_t*)p.rbeg, (const Ent*)m.ent,
                         (const int32_t*)(p.rows + p.class_off[kFirstShort]), n1, src, y, ldy, F);
      GCN_HIP(hipGetLastError());
    }
    if (n2 > 0) {
      ProfScope ps("agg_tiny", stream);
      hipLaunchKernelGGL((k_tiny<VEC, G, Src, RELU, 2, R2>),
                         dim3(blocks_for_waves(ceil_div(n2, E * R2)), tiles), dim3(kBlock), 0,
                         stream, (const int64_t*)(p.rbeg + n1), (const Ent*)m.ent,
                         (const int32_t*)(p.rows + p.class_off[kFirstShort + 1]), n2, src, y, ldy,
                         F);
      GCN_HIP(hipGetLastError());
    }
  }
  // rows of 3 .. medium_max entries (the classes of one and two entries get no
  // waves here)
  ShortArgs sa;
  int64_t waves = 0;
  for (int c = kFirstShort; c <= kMedium + 1; ++c) {
    sa.row_off[c - kFirstShort] = p.class_off[c];
    sa.wave_off[c - kFirstShort] = waves;
    if (c >= kFirstShort + 2 && c <= kMedium)
      waves += ceil_div(p.class_off[c + 1] - p.class_off[c], E);
  }
  if (waves > 0) {
    ProfScope ps("agg_short", stream);
    hipLaunchKernelGGL((k_short<VEC, G, Src, RELU>), dim3(blocks_for_waves(waves), tiles),
                       dim3(kBlock), 0, stream, (const int64_t*)p.rbeg, (const int32_t*)p.rlen,
                       (const Ent*)m.ent, (const int32_t*)p.rows, sa, src, y, ldy, F);
    GCN_HIP(hipGetLastError());
  }
  // long rows: chunk table, then column-blocked pieces, then the partial sums
  if (p.n_chunks > 0 || p.n_pieces > 0) {
    float* parts = ws;
    const int64_t ldp = (F + 3) & ~3;
    if (p.n_parts > 0 && !ws) GCN_CHECK(talloc(&parts, p.n_parts * ldp, stream, "partial rows"));
    // a workspace the caller owns is never released here
    auto release = [&]() {
      if (!ws) tfree(parts, stream);
    };
    if (p.n_chunks > 0) {
      ProfScope ps("agg_chunk", stream);
      hipLaunchKernelGGL((k_chunk<VEC, G, Src, RELU>), dim3((unsigned)p.n_chunks, tiles),
                         dim3(kBlock), 0, stream, (const Ent*)m.ent, (const int32_t*)p.chunk_row,
                         (const int64_t*)p.chunk_beg, (const int64_t*)p.chunk_end,
                         (const int32_t*)p.chunk_part, src, y, ldy, parts, ldp, F);
      hipError_t e = hipGetLastError();
      if (e != hipSuccess) {
        release();
        return hip_fail(e, "k_chunk", __FILE__, __LINE__);
      }
    }
    if (p.n_pieces > 0) {
      ProfScope ps("agg_pieces", stream);
      hipLaunchKernelGGL((k_pieces<VEC, G, Src>),
                         dim3(blocks_for_waves(ceil_div(p.n_pieces, E)), tiles),
                         dim3(kBlock), 0, stream, (const int64_t*)p.piece_beg,
                         (const int32_t*)p.piece_len, (const int32_t*)p.piece_part, p.n_pieces,
                         (const Ent*)m.ent, src, parts, ldp, F);
      hipError_t e = hipGetLastError();
      if (e != hipSuccess) {
        release();
        return hip_fail(e, "k_pieces", __FILE__, __LINE__);
      }
    }
    if (p.n_giant > 0) {
      ProfScope ps("agg_reduce_parts", stream);
      hipLaunchKernelGGL((k_reduce_parts<VEC, G, RELU>), dim3(blocks_for_waves(p.n_giant), tiles),
                         dim3(kBlock), 0, stream, (const int32_t*)p.giant_row,
                         (const int32_t*)p.giant_part_off, p.n_giant, (const float*)parts, ldp, y,
                         ldy, F);
      hipError_t e = hipGetLastError();
      if (e != hipSuccess) {
        release();
        return hip_fail(e, "k_reduce_parts", __FILE__, __LINE__);
      }
    }
    release();
  }
  return GCN_OK;
}

// Floats of partial rows one aggregation with the plan of m needs at width F.
int64_t parts_floats(const Mat& m, int64_t F) { return m.plan.n_parts * ((F + 3) & ~int64_t(3)); }

// Lanes per slot: smallest power of two covering min(F, 128) features with
// 4-float lanes (at least 4 lanes); wider rows run as 128-feature tiles
// (blockIdx.y), which beats one slot of 64 lanes per wavefront (F = 256:
// 5% on the product-shaped graph, 16 lanes for F = 128 lose 9%); the scalar
// path always uses 64 lanes.
int lanes_for(int F, bool vec4) {
  if (!vec4) return 64;
  const int need = (std::min(F, 128) + 3) / 4;
  int g = 4;
  while (g < need) g <<= 1;
  return g;
}

template <class Src, bool RELU>
gcn_status launch_vec4(const Mat& m, const Src& src, float* y, int64_t ldy, int F,
                       hipStream_t stream, float* ws) {
  switch (lanes_for(F, true)) {
    case 4: return launch_all<4, 4, RELU>(m, src, y, ldy, F, stream, ws);
    case 8: return launch_all<4, 8, RELU>(m, src, y, ldy, F, stream, ws);
    case 16: return launch_all<4, 16, RELU>(m, src, y, ldy, F, stream, ws);
    default: return launch_all<4, 32, RELU>(m, src, y, ldy, F, stream, ws);
  }
}

// pad_ok: every input row may be read up to a multiple of 4 features (its
// stride leaves room), so an odd F still takes the unguarded 16-byte loads;
// the extra features are never stored.
template <template <int, bool> class SrcT, bool RELU = false, class Make>
gcn_status dispatch(const Mat& m, bool vec4, int F, float* y, int64_t ldy, hipStream_t stream,
                    Make make, bool pad_ok = false, float* ws = nullptr) {
  if (!vec4) return launch_all<1, 64, RELU>(m, make(SrcT<1, false>{}), y, ldy, F, stream, ws);
  if (F % 4 != 0 && !pad_ok)
    return launch_vec4<SrcT<4, true>, RELU>(m, make(SrcT<4, true>{}), y, ldy, F, stream, ws);
  auto src = make(SrcT<4, false>{});
  src.F = (F + 3) & ~3;  // the width the loads may cover; F bounds the stores
  return launch_vec4<SrcT<4, false>, RELU>(m, src, y, ldy, F, stream, ws);
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

// Argument checks of the plain aggregation calls (before any work is enqueued).
gcn_status check_plain(const void* X, int64_t ldx, int dtype, const float* Y, int64_t ldy,
                       int64_t F) {
  if (!X || !Y) {
    set_error("input and output pointers must be non-NULL");
    return GCN_EINVAL;
  }
  if (ldx > (int64_t)UINT32_MAX) {
    set_error("ldx=%lld does not fit 32 bits", (long long)ldx);
    return GCN_ERANGE;
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
  return GCN_OK;
}

gcn_status aggregate(const Mat& m, const void* X, int64_t ldx, int dtype, float* Y, int64_t ldy,
                     int64_t F, void* stream, float* ws = nullptr) {
  GCN_CHECK(check_plain(X, ldx, dtype, Y, ldy, F));
  const int Fi = (int)F;
  hipStream_t s = (hipStream_t)stream;
  const bool yvec = aligned(Y, 16) && ldy % 4 == 0;
  if (dtype == GCN_DT_F32) {
    const bool vec4 = yvec && aligned(X, 16) && ldx % 4 == 0;
    return dispatch<SrcF32>(m, vec4, Fi, Y, ldy, s, [&](auto t) {
      t.x = (const float*)X;
      t.ld = (uint32_t)ldx;
      t.F = Fi;
      return t;
    }, false, ws);
  }
  const bool vec4 = yvec && aligned(X, 8) && ldx % 4 == 0;
  return dispatch<SrcBF16>(m, vec4, Fi, Y, ldy, s, [&](auto t) {
    t.x = (const uint16_t*)X;
    t.ld = (uint32_t)ldx;
    t.F = Fi;
    return t;
  }, false, ws);
}

}  // namespace

gcn_status aggregate_f32(const Mat& m, const float* X, int64_t ldx, float* Y, int64_t ldy,
                         int64_t F, bool relu, hipStream_t stream) {
  const int Fi = (int)F;
  const bool vec4 = aligned(Y, 16) && ldy % 4 == 0 && aligned(X, 16) && ldx % 4 == 0;
  auto make = [&](auto t) {
    t.x = X;
    t.ld = (uint32_t)ldx;
    t.F = Fi;
    return t;
  };
  // the training steps keep their feature rows at strides of a multiple of 4
  const bool pad_ok = ldx >= ((F + 3) & ~int64_t(3));
  return relu ? dispatch<SrcF32, true>(m, vec4, Fi, Y, ldy, stream, make, pad_ok)
              : dispatch<SrcF32, false>(m, vec4, Fi, Y, ldy, stream, make, pad_ok);
}

}  // namespace gcn

using namespace gcn;

extern "C" gcn_status gcn_aggregate_fwd(const gcn_graph* g, const void* X, int64_t ldx, int dtype,
                                        float* Y, int64_t ldy, int64_t F, void* stream) {
  clear_error();
  GCN_CHECK(check_common(g, F));
  return aggregate(g->csr, X, ldx, dtype, Y, ldy, F, stream);
}

extern "C" gcn_status gcn_aggregate_bwd(const gcn_graph* g, const void* G, int64_t ldg, int dtype,
                                        float* dX, int64_t lddx, int64_t F, void* stream) {
  clear_error();
  GCN_CHECK(check_common(g, F));
  return aggregate(g->csc, G, ldg, dtype, dX, lddx, F, stream);
}

extern "C" gcn_status gcn_aggregate_fwd_q8halo(const gcn_graph* g, int64_t n_local_cols,
                                               const float* X_local, int64_t ldx,
                                               const uint8_t* Q_halo, int64_t ldq,
                                               const float* halo_min, const float* halo_scale,
                                               int64_t ldp, float* Y, int64_t ldy, int64_t F,
                                               uint32_t flags, void* stream) {
  clear_error();
  GCN_CHECK(check_common(g, F));
  if (flags & ~(uint32_t)(GCN_Q8_USE_CSC | GCN_Q_CODES_2BIT)) {
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
  if (ldx > (int64_t)UINT32_MAX || ldq > (int64_t)UINT32_MAX || ldp > (int64_t)UINT32_MAX) {
    set_error("ldx, ldq and ldp must fit 32 bits");
    return GCN_ERANGE;
  }
  const bool two_bit = (flags & GCN_Q_CODES_2BIT) != 0;
  const int64_t qbytes = two_bit ? (F + 3) / 4 : F;
  if (n_local_cols < n_in && (!Q_halo || !halo_min || !halo_scale || ldq < qbytes || ldp < 1)) {
    set_error("Q_halo, halo_min, halo_scale must be non-NULL with ldq >= code bytes per row and "
              "ldp >= 1 when halo rows exist");
    return GCN_EINVAL;
  }
  const int Fi = (int)F;
  const bool vec4 = aligned(Y, 16) && ldy % 4 == 0 && (n_local_cols == 0 ||
                    (aligned(X_local, 16) && ldx % 4 == 0)) &&
                    (n_local_cols == n_in || two_bit || (aligned(Q_halo, 4) && ldq % 4 == 0));
  auto make = [&](auto t) {
    t.x = X_local;
    t.ldx = (uint32_t)ldx;
    t.n_local = (uint32_t)n_local_cols;
    t.q = Q_halo;
    t.ldq = (uint32_t)ldq;
    t.zmin = halo_min;
    t.scale = halo_scale;
    t.ldp = (uint32_t)ldp;
    t.F = Fi;
    return t;
  };
  if (two_bit) return dispatch<SrcQ2>(m, vec4, Fi, Y, ldy, (hipStream_t)stream, make);
  return dispatch<SrcQ8>(m, vec4, Fi, Y, ldy, (hipStream_t)stream, make);
}

// ---- the aggregation without allocation -------------------------------------

namespace gcn {
namespace {

// Room for the partial rows of gcn_aggregate_fwd_noalloc: 64 MiB per device,
// held by every device the library runs on until the process ends. In host
// code the name stands for no device address; the address comes from
// hipGetSymbolAddress, once per device.
constexpr int64_t kScratchFloats = int64_t(1) << 24;
__device__ __align__(256) float scratch[kScratchFloats];

std::mutex g_scratch_mu;
float* g_scratch_ptr[64] = {};

// Device address of this device's scratch array (looked up on the first call
// on the device, with the device current).
gcn_status scratch_for_current_device(float** out) {
  int dev = 0;
  GCN_HIP(hipGetDevice(&dev));
  if (dev < 0 || dev >= 64) {
    set_error("device %d out of range for the scratch table", dev);
    return GCN_EINVAL;
  }
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
      return hip_fail(e != hipSuccess ? e : hipErrorInvalidSymbol,
                      "hipGetSymbolAddress(scratch)", __FILE__, __LINE__);
    g_scratch_ptr[dev] = static_cast<float*>(p);
  }
  *out = g_scratch_ptr[dev];
  return GCN_OK;
}

}  // namespace
}  // namespace gcn

extern "C" gcn_status gcn_aggregate_fwd_noalloc(const gcn_graph* g, const void* X, int64_t ldx,
                                                int dtype, float* Y, int64_t ldy, int64_t F,
                                                void* stream) {
  clear_error();
  GCN_CHECK(check_common(g, F));
  GCN_CHECK(check_plain(X, ldx, dtype, Y, ldy, F));
  const int64_t need = parts_floats(g->csr, F);
  if (need > kScratchFloats) {
    set_error("the graph's plan needs %lld floats of partial rows at F=%lld; the no-allocation "
              "call holds %lld (use gcn_aggregate_fwd)", (long long)need, (long long)F,
              (long long)kScratchFloats);
    return GCN_ERANGE;
  }
  float* ws = nullptr;
  GCN_CHECK(scratch_for_current_device(&ws));
  return aggregate(g->csr, X, ldx, dtype, Y, ldy, F, stream, ws);
}
