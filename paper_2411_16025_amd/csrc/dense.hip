// Dense side of a GCN layer (the UPDATE of SuperGCN, arXiv 2411.16025,
// Section 2.1: after aggregation, a linear transform): fp32 GEMMs on the
// gfx950 matrix cores, ReLU, and softmax cross-entropy.
//
// GEMM shapes of full-batch GCN training are tall and skinny: the node count
// is in the millions, feature and class counts are at most a few hundred.
//  * C = A op(B) with M = nodes (NN, NT): one 256-thread workgroup computes a
//    64 x BN tile of C (BN = 64, 128 or 256) over all of K, staging 32-deep
//    slices of A and B in LDS while the next slice is loaded into registers;
//    each wavefront owns 16 rows and issues v_mfma_f32_16x16x4_f32 on BN / 16
//    blocks of 16 x 16. The tile leaves through LDS as row-contiguous
//    16-byte stores, with an optional ReLU or ReLU-backward mask.
//  * Products whose B fits in LDS (weights: K x 48 for the classes, K x 256
//    slices for the hidden layer) take a resident-B kernel: B is staged once
//    per CU and every wavefront streams its own rows of A into the
//    matrix-core registers, several chunks ahead.
//  * C = A^T B with K = nodes (the weight gradients): K is split into fixed
//    chunks; every chunk writes a partial C tile and a second kernel adds the
//    partials in chunk order, so the result is the same on every run.
//
// v_mfma_f32_16x16x4_f32 operand layout (lane l of the wavefront): a holds
// A[l % 16][k0 + l / 16], b holds B[k0 + l / 16][l % 16], and result element
// i holds C[4 * (l / 16) + i][l % 16].

#include <algorithm>
#include <mutex>
#include <type_traits>

#include "common.h"

namespace gcn {
namespace {

typedef float f4 __attribute__((ext_vector_type(4)));
typedef float f2 __attribute__((ext_vector_type(2)));

constexpr int kThreads = 256;
constexpr int kTile = 64;  // C tile is kTile x kTile
constexpr int kKc = 32;    // K slice staged in LDS
constexpr int kPad = 1;    // LDS row padding against bank conflicts
constexpr int64_t kSplitRows = 8192;  // K chunk of the A^T B kernel
#ifndef GCN_TN_MIN_BLOCKS
#define GCN_TN_MIN_BLOCKS 4096
#endif
#ifndef GCN_TN_MIN_SPLIT
#define GCN_TN_MIN_SPLIT 1024
#endif
constexpr int64_t kSplitRowsMin = GCN_TN_MIN_SPLIT;
constexpr int64_t kTnMinBlocks = GCN_TN_MIN_BLOCKS;  // workgroups the A^T B grid aims for

enum Op { kNN = 0, kNT = 1 };

// C[M x N] = A[M x K] * B[K x N] (NN) or A[M x K] * B[N x K]^T (NT).
template <int OP>
__global__ __launch_bounds__(kThreads) void k_gemm_tall(int64_t M, int64_t N, int64_t K,
                                                        const float* __restrict__ A, int64_t lda,
                                                        const float* __restrict__ B, int64_t ldb,
                                                        float* __restrict__ C, int64_t ldc) {
  __shared__ float As[kTile][kKc + kPad];  // As[m][k]
  __shared__ float Bs[kKc][kTile + kPad];  // Bs[k][n]
  const int t = threadIdx.x, lane = t & 63, w = t >> 6;
  const int64_t m0 = (int64_t)blockIdx.x * kTile;
  const int64_t n0 = (int64_t)blockIdx.y * kTile;
  f4 acc[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) acc[j] = f4{0.f, 0.f, 0.f, 0.f};
  for (int64_t k0 = 0; k0 < K; k0 += kKc) {
    // A slice: 64 rows x 32 k, 8 consecutive k per thread
    {
      const int r = t >> 2, c = (t & 3) * 8;
      const int64_t gm = m0 + r;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int64_t gk = k0 + c + e;
        As[r][c + e] = (gm < M && gk < K) ? A[gm * lda + gk] : 0.f;
      }
    }
    if (OP == kNN) {  // B slice: 32 k x 64 n, 8 consecutive n per thread
      const int r = t >> 3, c = (t & 7) * 8;
      const int64_t gk = k0 + r;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int64_t gn = n0 + c + e;
        Bs[r][c + e] = (gk < K && gn < N) ? B[gk * ldb + gn] : 0.f;
      }
    } else {  // B stored N x K: rows n, 8 consecutive k per thread, transposed into Bs
      const int r = t >> 2, c = (t & 3) * 8;
      const int64_t gn = n0 + r;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int64_t gk = k0 + c + e;
        Bs[c + e][r] = (gn < N && gk < K) ? B[gn * ldb + gk] : 0.f;
      }
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < kKc; kk += 4) {
      const float a = As[16 * w + (lane & 15)][kk + (lane >> 4)];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const float b = Bs[kk + (lane >> 4)][16 * j + (lane & 15)];
        acc[j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, acc[j], 0, 0, 0);
      }
    }
    __syncthreads();
  }
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int64_t gn = n0 + 16 * j + (lane & 15);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int64_t gm = m0 + 16 * w + 4 * (lane >> 4) + i;
      if (gm < M && gn < N) C[gm * ldc + gn] = acc[j][i];
    }
  }
}

// Partial C tiles of C = A^T B over rows [chunk * split, ...) of A and B.
// A is [K x M], B is [K x N]; part holds [n_chunks][M][N].
__global__ __launch_bounds__(kThreads) void k_gemm_tn_partial(int64_t M, int64_t N, int64_t K,
                                                              int64_t split,
                                                              const float* __restrict__ A,
                                                              int64_t lda,
                                                              const float* __restrict__ B,
                                                              int64_t ldb,
                                                              float* __restrict__ part) {
  __shared__ float As[kKc][kTile + kPad];  // As[k][m]
  __shared__ float Bs[kKc][kTile + kPad];  // Bs[k][n]
  const int t = threadIdx.x, lane = t & 63, w = t >> 6;
  const int64_t m0 = (int64_t)blockIdx.x * kTile;
  const int64_t n0 = (int64_t)blockIdx.y * kTile;
  const int64_t chunk = blockIdx.z;
  const int64_t kb = chunk * split;
  const int64_t ke = std::min(K, kb + split);
  f4 acc[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) acc[j] = f4{0.f, 0.f, 0.f, 0.f};
  for (int64_t k0 = kb; k0 < ke; k0 += kKc) {
    const int r = t >> 3, c = (t & 7) * 8;
    const int64_t gk = k0 + r;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int64_t gm = m0 + c + e, gn = n0 + c + e;
      As[r][c + e] = (gk < ke && gm < M) ? A[gk * lda + gm] : 0.f;
      Bs[r][c + e] = (gk < ke && gn < N) ? B[gk * ldb + gn] : 0.f;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < kKc; kk += 4) {
      const float a = As[kk + (lane >> 4)][16 * w + (lane & 15)];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const float b = Bs[kk + (lane >> 4)][16 * j + (lane & 15)];
        acc[j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, acc[j], 0, 0, 0);
      }
    }
    __syncthreads();
  }
  float* out = part + chunk * M * N;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int64_t gn = n0 + 16 * j + (lane & 15);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int64_t gm = m0 + 16 * w + 4 * (lane >> 4) + i;
      if (gm < M && gn < N) out[gm * N + gn] = acc[j][i];
    }
  }
}

// Features [c, c + 4) of row `row` of a row-major matrix with `cols` columns,
// zero outside it: one 16-byte load when the four are inside (the caller
// guarantees 16-byte alignment of every row start and of c), else per element.
__device__ inline f4 load4(const float* __restrict__ p, int64_t row, int64_t rows, int64_t ld,
                           int64_t c, int64_t cols) {
  f4 v = {0.f, 0.f, 0.f, 0.f};
  if (row >= rows) return v;
  const float* q = p + row * ld + c;
  if (c + 4 <= cols) return *reinterpret_cast<const f4*>(q);
#pragma unroll
  for (int e = 0; e < 4; ++e)
    if (c + e < cols) v[e] = q[e];
  return v;
}

// Wide-tile C = A op(B) for 16-byte aligned operands: a 64 x BN tile per
// 256-thread workgroup (BN up to 256, so the tall operand is read once per
// BN columns), 32-deep K slices in LDS, software-pipelined: the next slice's
// A and B tiles are loaded into registers while the current slice is
// multiplied from LDS, so the loads' latency overlaps the matrix-core work.
// B is kept k-major for NN and n-major for NT (both written with 16-byte
// LDS stores). With mask, C = 0 where mask <= 0 (a ReLU backward); with
// relu, C = max(C, 0) (a ReLU forward).
#ifndef GCN_GEMM_MIN_BLOCKS
#define GCN_GEMM_MIN_BLOCKS 2
#endif
// From this depth on, the 256-column NN tile takes two 16-row blocks per
// wavefront (128 x 256 per workgroup, each B fragment feeding two MFMAs):
// 3% faster at K = 516, slower at K <= 204.
constexpr int64_t kDeepK = 384;
// Workgroups per CU the 64- and 128-column tiles must fit (fewer registers,
// more waves to overlap LDS and global latency).
#ifndef GCN_GEMM_MIN_BLOCKS_NARROW
#define GCN_GEMM_MIN_BLOCKS_NARROW 4
#endif
#ifndef GCN_GEMM_KK_UNROLL
#define GCN_GEMM_KK_UNROLL 8
#endif
#define GCN_GEMM_PRAGMA(x) _Pragma(#x)
#define GCN_GEMM_UNROLL(n) GCN_GEMM_PRAGMA(unroll n)

// LDS row stride for rows read along n: 16 mod 32 floats, so the operand
// reads of a half-wavefront (16 columns x 2 rows) hit 32 distinct banks.
constexpr int stride_n(int bn) { return bn + (48 - bn % 32) % 32; }

template <int OP, int BN, int RB>
__global__ __launch_bounds__(kThreads,
                             BN == 256 ? GCN_GEMM_MIN_BLOCKS : GCN_GEMM_MIN_BLOCKS_NARROW)
void k_gemm_tall_v(int64_t M, int64_t N, int64_t K, const float* __restrict__ A, int64_t lda,
                   const float* __restrict__ B, int64_t ldb, float* __restrict__ C, int64_t ldc,
                   const float* __restrict__ mask, int64_t ldm, bool relu, bool cvec) {
  // RB 16-row blocks per wavefront: a BM x BN tile per workgroup
  constexpr int BM = kTile * RB;
  constexpr int NB = BN / 16;
  constexpr int BQ = 8 * BN;                          // 16-byte pieces of a B slice
  constexpr int BL = (BQ + kThreads - 1) / kThreads;  // per thread (the last may be idle)
  constexpr int AL = 2 * RB;                          // 16-byte A loads per thread per slice
  // LDS strides chosen so that the operand reads of a half-wavefront (16
  // rows or columns x 2 k values) hit 32 distinct banks: rows read along k
  // (A, and B of NT) have a stride of 2 mod 32 floats and are written with
  // 8-byte stores; rows read along n (B of NN) have a stride of 16 mod 32
  constexpr int AS = kKc + 2;
  constexpr int BR = OP == kNN ? kKc : BN;
  constexpr int BC = OP == kNN ? stride_n(BN) : kKc + 2;
  // the output tile is staged through the same LDS, CW columns at a time
  constexpr int CW = BN < 128 ? BN : 128;
  constexpr int kOperands = BM * AS + BR * BC;
  constexpr int kStage = BM * (CW + 4);
  __shared__ __align__(16) float smem[kOperands > kStage ? kOperands : kStage];
  auto& As = *reinterpret_cast<float (*)[BM][AS]>(smem);
  auto& Bs = *reinterpret_cast<float (*)[BR][BC]>(smem + BM * AS);
  const int t = threadIdx.x, lane = t & 63, w = t >> 6;
  const int64_t m0 = (int64_t)blockIdx.x * BM;
  const int64_t n0 = (int64_t)blockIdx.y * BN;
  f4 acc[RB][NB];
#pragma unroll
  for (int r = 0; r < RB; ++r)
#pragma unroll
    for (int j = 0; j < NB; ++j) acc[r][j] = f4{0.f, 0.f, 0.f, 0.f};
  f4 ra[AL], rb[BL];
  auto load_slice = [&](int64_t k0) {
#pragma unroll
    for (int j = 0; j < AL; ++j) {  // A: BM x 32 floats
      const int idx = t + kThreads * j, r = idx >> 3, c = (idx & 7) * 4;
      ra[j] = load4(A, m0 + r, M, lda, k0 + c, K);
    }
#pragma unroll
    for (int j = 0; j < BL; ++j) {
      const int idx = t + kThreads * j;
      if (BQ % kThreads != 0 && idx >= BQ) continue;
      if (OP == kNN) {  // B rows k0 .. k0 + 31, columns n0 .. n0 + BN - 1
        const int r = idx / (BN / 4), c = (idx % (BN / 4)) * 4;
        rb[j] = load4(B, k0 + r, K, ldb, n0 + c, N);
      } else {  // B stored N x K: rows n0 .. n0 + BN - 1, columns k0 .. k0 + 31
        const int r = idx >> 3, c = (idx & 7) * 4;
        rb[j] = load4(B, n0 + r, N, ldb, k0 + c, K);
      }
    }
  };
  auto store_slice = [&]() {
#pragma unroll
    for (int j = 0; j < AL; ++j) {
      const int idx = t + kThreads * j, r = idx >> 3, c = (idx & 7) * 4;
      *reinterpret_cast<f2*>(&As[r][c]) = f2{ra[j].x, ra[j].y};
      *reinterpret_cast<f2*>(&As[r][c + 2]) = f2{ra[j].z, ra[j].w};
    }
#pragma unroll
    for (int j = 0; j < BL; ++j) {
      const int idx = t + kThreads * j;
      if (BQ % kThreads != 0 && idx >= BQ) continue;
      if (OP == kNN) {
        const int r = idx / (BN / 4), c = (idx % (BN / 4)) * 4;
        *reinterpret_cast<f4*>(&Bs[r][c]) = rb[j];
      } else {
        const int r = idx >> 3, c = (idx & 7) * 4;
        *reinterpret_cast<f2*>(&Bs[r][c]) = f2{rb[j].x, rb[j].y};
        *reinterpret_cast<f2*>(&Bs[r][c + 2]) = f2{rb[j].z, rb[j].w};
      }
    }
  };
  load_slice(0);
  store_slice();
  __syncthreads();
  for (int64_t k0 = 0; k0 < K; k0 += kKc) {
    const bool more = k0 + kKc < K;
    if (more) load_slice(k0 + kKc);
    // the steps of a last, partial slice past K would only add zero products
    // (kn is the same for the whole workgroup)
    const int kn = more ? kKc : (int)(K - k0);
    GCN_GEMM_UNROLL(GCN_GEMM_KK_UNROLL)
    for (int kk = 0; kk < kKc; kk += 4) {
      if (kk >= kn) break;
      float a[RB];
#pragma unroll
      for (int r = 0; r < RB; ++r) a[r] = As[16 * (RB * w + r) + (lane & 15)][kk + (lane >> 4)];
#pragma unroll
      for (int j = 0; j < NB; ++j) {
        const float b = OP == kNN ? Bs[kk + (lane >> 4)][16 * j + (lane & 15)]
                                  : Bs[16 * j + (lane & 15)][kk + (lane >> 4)];
#pragma unroll
        for (int r = 0; r < RB; ++r)
          acc[r][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[r], b, acc[r][j], 0, 0, 0);
      }
    }
    __syncthreads();
    if (more) {
      store_slice();
      __syncthreads();
    }
  }
  if (cvec) {
    // CW columns at a time: the wave writes its 16 x CW block to LDS in the
    // matrix-core layout, then stores it row by row with 16-byte accesses (the
    // mask is read the same way)
    float (*st)[CW + 4] = reinterpret_cast<float (*)[CW + 4]>(smem);
    constexpr int LPR = CW / 4;                     // lanes per row
    constexpr int RPI = 64 / LPR;                   // rows per store instruction
    constexpr int NIT = (16 * RB + RPI - 1) / RPI;  // store instructions per column block
#pragma unroll
    for (int c0 = 0; c0 < BN; c0 += CW) {
      // the mask values this lane applies, loaded before the staging so
      // their latency overlaps it (one 16-byte load per store)
      f4 mk[NIT];
      if (mask) {
#pragma unroll
        for (int it = 0; it < NIT; ++it) {
          mk[it] = f4{1.f, 1.f, 1.f, 1.f};
          if (64 % LPR != 0 && (lane / LPR >= RPI || it * RPI + lane / LPR >= 16 * RB)) continue;
          const int64_t gm = m0 + 16 * RB * w + it * RPI + lane / LPR;
          const int64_t gn = n0 + c0 + 4 * (lane % LPR);
          if (gm < M && gn + 4 <= N) mk[it] = *reinterpret_cast<const f4*>(mask + gm * ldm + gn);
        }
      }
      __syncthreads();  // the operands (or the previous columns) are no longer read
#pragma unroll
      for (int r = 0; r < RB; ++r)
#pragma unroll
        for (int j = c0 / 16; j < (c0 + CW) / 16; ++j)
#pragma unroll
          for (int i = 0; i < 4; ++i)
            st[16 * (RB * w + r) + 4 * (lane >> 4) + i][16 * j - c0 + (lane & 15)] = acc[r][j][i];
      __syncthreads();
#pragma unroll
      for (int it = 0; it < NIT; ++it) {
        // with 48 columns (12 lanes a row) lanes 60 .. 63 have no row
        if (64 % LPR != 0 && (lane / LPR >= RPI || it * RPI + lane / LPR >= 16 * RB)) continue;
        const int rl = 16 * RB * w + it * RPI + lane / LPR;
        const int cl = 4 * (lane % LPR);
        const int64_t gm = m0 + rl, gn = n0 + c0 + cl;
        if (gm >= M || gn >= N) continue;
        f4 v = *reinterpret_cast<const f4*>(&st[rl][cl]);
        if (gn + 4 <= N) {
          if (mask) {
#pragma unroll
            for (int e = 0; e < 4; ++e)
              if (!(mk[it][e] > 0.f)) v[e] = 0.f;
          }
          if (relu) {
#pragma unroll
            for (int e = 0; e < 4; ++e) v[e] = fmaxf(v[e], 0.f);
          }
          *reinterpret_cast<f4*>(C + gm * ldc + gn) = v;
        } else {
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            if (gn + e >= N) break;
            float x = (mask && !(mask[gm * ldm + gn + e] > 0.f)) ? 0.f : v[e];
            if (relu) x = fmaxf(x, 0.f);
            C[gm * ldc + gn + e] = x;
          }
        }
      }
    }
    return;
  }
#pragma unroll
  for (int r = 0; r < RB; ++r)
#pragma unroll
  for (int j = 0; j < NB; ++j) {
    const int64_t gn = n0 + 16 * j + (lane & 15);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int64_t gm = m0 + 16 * (RB * w + r) + 4 * (lane >> 4) + i;
      if (gm < M && gn < N) {
        float v = (mask && !(mask[gm * ldm + gn] > 0.f)) ? 0.f : acc[r][j][i];
        if (relu) v = fmaxf(v, 0.f);
        C[gm * ldc + gn] = v;
      }
    }
  }
}

// Resident-B C = A op(B) for products whose B (a weight matrix) fits in LDS:
// each workgroup (one per CU) stages its BN-column slice of B in LDS once and
// then stays on its CU; every wavefront walks its own 16 * RB-row tiles of C
// with no further barriers. A is streamed straight from memory into the
// matrix-core operand registers, D slots of CPS 16-deep K chunks ahead
// (across tile boundaries), so the loads of one wavefront overlap the MFMAs
// of the others. Narrow outputs (the 47 classes) are bound by the stream of
// A, which the staged-tile kernel reads one 32-deep slice per barrier pair;
// wide ones with a short K by the stores of C.
//
// Operand order inside a chunk: for a full chunk of 16 k, lane (g = l / 16,
// r = l % 16) holds A[r][16 j + 4 g .. + 3] as one 16-byte load and matrix-core
// step i takes element i, so step i contracts over k = 16 j + 4 g + i for the
// four lane groups g; the last, partial chunk (K % 16 != 0) takes
// k = 16 j + 4 i + g instead, element by element, so that its steps stop at
// ceil((K - 16 j) / 4). B is stored in LDS in the same order, one float4 per
// (chunk, 16-column block, lane), and read with one 16-byte LDS load per block
// and chunk. The sum over k is the same; only its order differs from the
// staged-tile kernel.
//
// Stores: the four results of a lane (rows 4 g .. 4 g + 3 of one column) are
// transposed within each quad of lanes with DPP moves, so that every lane
// writes 4 consecutive columns of one row as one 16-byte store.

__device__ inline float dpp_quad(float v, int ctrl_sel) {
  // 0x4E: quad_perm [2, 3, 0, 1]; 0xB1: quad_perm [1, 0, 3, 2]
  const int x = __float_as_int(v);
  const int y = ctrl_sel == 0 ? __builtin_amdgcn_mov_dpp(x, 0x4E, 0xF, 0xF, false)
                              : __builtin_amdgcn_mov_dpp(x, 0xB1, 0xF, 0xF, false);
  return __int_as_float(y);
}

// In each quad of lanes (q = lane & 3) element i of lane q is M[i][q] on
// entry and M[q][i] on return: the 2 x 2 blocks are swapped across lanes two
// apart, then each 2 x 2 block is transposed across neighbouring lanes.
__device__ inline f4 quad_transpose(f4 v, int q) {
  const bool lo = q < 2;
  float x = lo ? v[2] : v[0], y = lo ? v[3] : v[1];
  x = dpp_quad(x, 0);
  y = dpp_quad(y, 0);
  if (lo) { v[2] = x; v[3] = y; } else { v[0] = x; v[1] = y; }
  const bool ev = (q & 1) == 0;
  x = ev ? v[1] : v[0];
  y = ev ? v[3] : v[2];
  x = dpp_quad(x, 1);
  y = dpp_quad(y, 1);
  if (ev) { v[1] = x; v[3] = y; } else { v[0] = x; v[2] = y; }
  return v;
}

template <int OP, int NBLK, int RB, int D, int CPS, int WAVES>
__global__ __launch_bounds__(64 * WAVES) void k_gemm_bres(
    int64_t M, int64_t N, int64_t K, const float* __restrict__ A, int64_t lda,
    const float* __restrict__ B, int64_t ldb, float* __restrict__ C, int64_t ldc,
    const float* __restrict__ mask, int64_t ldm, bool relu, bool cvec) {
  extern __shared__ __align__(16) float bres_lds[];
  const f4* Bs = reinterpret_cast<const f4*>(bres_lds);
  constexpr int BN = 16 * NBLK;
  const int64_t NC = K / 16;          // full chunks (a multiple of D * CPS)
  const int kt = (int)(K - 16 * NC);  // k of the partial chunk (0: none)
  const int64_t n0 = (int64_t)blockIdx.y * BN;
  const int t = threadIdx.x, lane = t & 63;
  // stage B: slot (chunk j, block nb, lane l, element i) holds
  // B[k][n0 + 16 nb + l % 16] with k as described above (zero past K or N);
  // n runs fastest over the threads so the reads of an NN B row are
  // contiguous; 8 loads are in flight per thread
  {
    const int64_t total = (NC + (kt > 0)) * NBLK * 256;
    constexpr int U = 8, kThr = 64 * WAVES;
    for (int64_t base = 0; base < total; base += (int64_t)U * kThr) {
      float v[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int64_t idx = base + (int64_t)u * kThr + t;
        const int n = (int)(idx & 15);
        const int i = (int)((idx >> 4) & 3);
        const int g = (int)((idx >> 6) & 3);
        const int64_t jb = idx >> 8;  // j * NBLK + nb
        const int nb = (int)(jb % NBLK);
        const int64_t j = jb / NBLK;
        const int64_t k = j < NC ? 16 * j + 4 * g + i : 16 * j + 4 * i + g;
        const int64_t col = n0 + 16 * nb + n;
        v[u] = 0.f;
        if (idx < total && k < K && col < N) v[u] = OP == kNN ? B[k * ldb + col] : B[col * ldb + k];
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int64_t idx = base + (int64_t)u * kThr + t;
        if (idx < total) {
          const int n = (int)(idx & 15);
          const int i = (int)((idx >> 4) & 3);
          const int g = (int)((idx >> 6) & 3);
          bres_lds[((idx >> 8) * 64 + 16 * g + n) * 4 + i] = v[u];
        }
      }
    }
  }
  __syncthreads();
  constexpr int TR = 16 * RB;  // rows per tile
  const int64_t T = (M + TR - 1) / TR;
  const int64_t TW = (int64_t)gridDim.x * WAVES;
  const int64_t first = (int64_t)blockIdx.x * WAVES +
                        __builtin_amdgcn_readfirstlane(t >> 6);
  if (first >= T) return;
  const int g = lane >> 4, r = lane & 15, q = lane & 3;
  // This lane's A elements of a tile: row tile * TR + 16 rb + r (rows past M
  // read row M - 1, never stored), from column 4 g on.
  auto rowptr = [&](int64_t tile, int rb) {
    return A + min(min(tile, T - 1) * TR + 16 * rb + r, M - 1) * lda + 4 * g;
  };
  auto load_b = [&](int64_t j, f4 (&b)[NBLK]) {
    const f4* bp = Bs + j * NBLK * 64 + lane;
#pragma unroll
    for (int nb = 0; nb < NBLK; ++nb) b[nb] = bp[nb * 64];
  };
  f4 acc[RB][NBLK];
  auto mma = [&](const f4 (&a)[RB], const f4 (&b)[NBLK], int steps) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      if (i >= steps) break;
#pragma unroll
      for (int nb = 0; nb < NBLK; ++nb)
#pragma unroll
        for (int rb = 0; rb < RB; ++rb)
          acc[rb][nb] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[rb][i], b[nb][i], acc[rb][nb], 0, 0, 0);
    }
  };
  // the partial chunk: element i of lane group g is k = 16 NC + 4 i + g
  // (clamped to K - 1 here, zeroed after the load has landed)
  auto issue_tail = [&](const float* const (&p)[RB], f4 (&dst)[RB]) {
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
      const float* row = p[rb] - 4 * g + 16 * NC;
#pragma unroll
      for (int i = 0; i < 4; ++i) dst[rb][i] = row[min(4 * i + g, kt - 1)];
    }
  };
  // The chunk stream of a wavefront: its tiles first, first + TW, ..., NC
  // chunks each. A ring slot holds CPS consecutive chunks (their loads go
  // out back to back: 64 CPS contiguous bytes of each row), D slots are in
  // flight, and D * CPS divides NC. Each slot is refilled right after its
  // MFMAs with the slot D ahead (of this tile or, in the last group, of the
  // next one; past the last tile a valid row is reloaded and never used), so
  // every group issues the same loads and a wait covers one slot. The next
  // chunk's B fragments are read from LDS before the current chunk's MFMAs.
  // The first group of a tile is peeled: the stores of the previous tile
  // make its first wait a full one (loads and stores share one counter); the
  // groups after it wait for one slot at a time.
  constexpr int SPG = D * CPS;  // chunks per group
  const int64_t NG = NC / SPG;
  const float* pc[RB];  // rows of the current tile
  const float* pn[RB];  // rows of the next tile
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    pc[rb] = rowptr(first, rb);
    pn[rb] = rowptr(first + TW, rb);
  }
  f4 buf[D][RB][CPS], tb[RB], tbn[RB];
#pragma unroll
  for (int d = 0; d < D; ++d)
#pragma unroll
    for (int rb = 0; rb < RB; ++rb)
#pragma unroll
      for (int c = 0; c < CPS; ++c)
        buf[d][rb][c] = *reinterpret_cast<const f4*>(pc[rb] + 16 * (d * CPS + c));
  if (kt > 0) issue_tail(pc, tb);
  auto group = [&](int64_t gi) {
    const bool last = gi + 1 == NG;
    const float* src[RB];
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) src[rb] = last ? pn[rb] : pc[rb] + 16 * SPG * (gi + 1);
    f4 b[2][NBLK];
    load_b(gi * SPG, b[0]);
#pragma unroll
    for (int d = 0; d < D; ++d) {
#pragma unroll
      for (int c = 0; c < CPS; ++c) {
        const int jj = d * CPS + c;
        if (jj + 1 < SPG) load_b(gi * SPG + jj + 1, b[(jj + 1) & 1]);
        f4 a[RB];
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) a[rb] = buf[d][rb][c];
        mma(a, b[jj & 1], 4);
      }
#pragma unroll
      for (int rb = 0; rb < RB; ++rb)
#pragma unroll
        for (int c = 0; c < CPS; ++c)
          buf[d][rb][c] = *reinterpret_cast<const f4*>(src[rb] + 16 * (d * CPS + c));
      // keep the slots in order: without this the scheduler hoists every
      // slot's LDS reads to the top of the group and sinks the refills to
      // its end, which costs registers and the staggering of the loads
      __builtin_amdgcn_sched_barrier(0);
    }
  };
  for (int64_t tile = first; tile < T; tile += TW) {
#pragma unroll
    for (int rb = 0; rb < RB; ++rb)
#pragma unroll
      for (int nb = 0; nb < NBLK; ++nb) acc[rb][nb] = f4{0.f, 0.f, 0.f, 0.f};
    group(0);
    // the next tile's partial chunk goes out after the first (full) wait
    if (kt > 0) issue_tail(pn, tbn);
    for (int64_t gi = 1; gi < NG; ++gi) group(gi);
    if (kt > 0) {
#pragma unroll
      for (int rb = 0; rb < RB; ++rb)
#pragma unroll
        for (int i = 0; i < 4; ++i)
          if (4 * i + g >= kt) tb[rb][i] = 0.f;
      f4 b[NBLK];
      load_b(NC, b);
      mma(tb, b, (kt + 3) / 4);
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) tb[rb] = tbn[rb];
    }
    // the tile leaves: C (with the ReLU-backward mask or the ReLU applied)
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
      const int64_t rbase = tile * TR + 16 * rb;
#pragma unroll
      for (int nb = 0; nb < NBLK; ++nb) {
        if (cvec) {
          // after the transpose: row 4 g + q, columns 4 ((lane >> 2) & 3) .. + 3
          f4 v = quad_transpose(acc[rb][nb], q);
          const int64_t gm = rbase + 4 * g + q;
          const int64_t gn = n0 + 16 * nb + 4 * ((lane >> 2) & 3);
          if (gm < M && gn < N) {
            if (gn + 4 <= N) {
              if (mask) {
                const f4 mk = *reinterpret_cast<const f4*>(mask + gm * ldm + gn);
#pragma unroll
                for (int e = 0; e < 4; ++e)
                  if (!(mk[e] > 0.f)) v[e] = 0.f;
              }
              if (relu) {
#pragma unroll
                for (int e = 0; e < 4; ++e) v[e] = fmaxf(v[e], 0.f);
              }
              // plain stores: nontemporal ones left the 64-byte row pieces
              // to reach memory as partial lines (Z2 0.75 -> 0.71 ms)
              *reinterpret_cast<f4*>(C + gm * ldc + gn) = v;
            } else {
#pragma unroll
              for (int e = 0; e < 4; ++e) {
                if (gn + e >= N) break;
                float x = (mask && !(mask[gm * ldm + gn + e] > 0.f)) ? 0.f : v[e];
                if (relu) x = fmaxf(x, 0.f);
                C[gm * ldc + gn + e] = x;
              }
            }
          }
        } else {
          const int64_t gn = n0 + 16 * nb + r;
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int64_t gm = rbase + 4 * g + i;
            if (gm < M && gn < N) {
              float x = (mask && !(mask[gm * ldm + gn] > 0.f)) ? 0.f : acc[rb][nb][i];
              if (relu) x = fmaxf(x, 0.f);
              C[gm * ldc + gn] = x;
            }
          }
        }
      }
    }
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
      pc[rb] = pn[rb];
      pn[rb] = rowptr(tile + 2 * TW, rb);
    }
  }
}

// Wide-tile partial C = A^T B over one K chunk for 16-byte aligned operands:
// a (16 * WAVES) x BN tile per workgroup, so for C up to 128 x 256 each row
// of A and B is read once per chunk.
template <int WAVES, int BN>
__global__ __launch_bounds__(WAVES * 64) void k_gemm_tn_v(int64_t M, int64_t N, int64_t K,
                                                          int64_t split,
                                                          const float* __restrict__ A, int64_t lda,
                                                          const float* __restrict__ B, int64_t ldb,
                                                          float* __restrict__ part) {
  constexpr int BM = 16 * WAVES, NT = 64 * WAVES, NB = BN / 16;
  // row strides of 16 mod 32 floats: a half-wavefront's reads (16 columns x
  // 2 rows) hit 32 distinct banks
  __shared__ __align__(16) float As[kKc][stride_n(BM)];
  __shared__ __align__(16) float Bs[kKc][stride_n(BN)];
  const int t = threadIdx.x, lane = t & 63, w = t >> 6;
  const int64_t m0 = (int64_t)blockIdx.x * BM;
  const int64_t n0 = (int64_t)blockIdx.y * BN;
  const int64_t chunk = blockIdx.z;
  const int64_t kb = chunk * split;
  const int64_t ke = std::min(K, kb + split);
  f4 acc[NB];
#pragma unroll
  for (int j = 0; j < NB; ++j) acc[j] = f4{0.f, 0.f, 0.f, 0.f};
  for (int64_t k0 = kb; k0 < ke; k0 += kKc) {
#pragma unroll
    for (int j = 0; j < kKc * BM / 4 / NT; ++j) {
      const int idx = t + NT * j, r = idx / (BM / 4), c = (idx % (BM / 4)) * 4;
      *reinterpret_cast<f4*>(&As[r][c]) = load4(A, k0 + r, ke, lda, m0 + c, M);
    }
    constexpr int BQ = kKc * BN / 4;  // 16-byte pieces of a B slice
#pragma unroll
    for (int j = 0; j < (BQ + NT - 1) / NT; ++j) {
      const int idx = t + NT * j, r = idx / (BN / 4), c = (idx % (BN / 4)) * 4;
      if (BQ % NT != 0 && idx >= BQ) continue;
      *reinterpret_cast<f4*>(&Bs[r][c]) = load4(B, k0 + r, ke, ldb, n0 + c, N);
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < kKc; kk += 4) {
      const float a = As[kk + (lane >> 4)][16 * w + (lane & 15)];
#pragma unroll
      for (int j = 0; j < NB; ++j) {
        const float b = Bs[kk + (lane >> 4)][16 * j + (lane & 15)];
        acc[j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, acc[j], 0, 0, 0);
      }
    }
    __syncthreads();
  }
  float* out = part + chunk * M * N;
#pragma unroll
  for (int j = 0; j < NB; ++j) {
    const int64_t gn = n0 + 16 * j + (lane & 15);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int64_t gm = m0 + 16 * w + 4 * (lane >> 4) + i;
      if (gm < M && gn < N) out[gm * N + gn] = acc[j][i];
    }
  }
}

// Streaming partial C = A^T B (the weight gradients: K = nodes, C at most a
// few hundred square) without LDS or barriers. A wavefront owns a 64 x 16 NB
// tile of C and one K chunk. Lane (g = l / 16, x = l % 16) loads, for rows
// k0 + g (k0 a multiple of 4):
//  * one 16-byte piece of A: A[k0 + g][m0 + 4 x .. + 3]; its element c is the
//    matrix-core operand of output row m0 + 4 x + c, so one load feeds four
//    16-row blocks (block c holds the rows m0 + 4 x + c, x = 0 .. 15);
//  * NB words of B: B[k0 + g][n0 + 16 j + x] for the 16-column blocks j.
// Each 4-row step is 4 NB matrix-core operations contracting over the four
// rows. The loads run D slots of CPS steps ahead of the matrix cores (no
// stores inside the loop, so every wait covers exactly one slot); the chunk
// partials are added in chunk order by k_sum_partials, so the result is the
// same on every run. Columns past M or N read a valid column of the row and
// only reach outputs that are not stored; rows past the chunk are zeroed.
template <int NB, int D, int CPS>
__global__ __launch_bounds__(512) void k_gemm_tn_s(int64_t M, int64_t N, int64_t K,
                                                   int64_t split, const float* __restrict__ A,
                                                   int64_t lda, const float* __restrict__ B,
                                                   int64_t ldb, float* __restrict__ part,
                                                   int m_tiles, int n_tiles) {
  const int lane = threadIdx.x & 63;
  const int tile = (int)blockIdx.y * (int)(blockDim.x >> 6) +
                   __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
  if (tile >= m_tiles * n_tiles) return;
  const int64_t m0 = (int64_t)(tile % m_tiles) * 64;
  const int64_t n0 = (int64_t)(tile / m_tiles) * (16 * NB);
  const int64_t chunk = blockIdx.x;
  const int64_t kb = chunk * split;
  const int64_t ke = min(K, kb + split);
  const int g = lane >> 4, x = lane & 15;
  // this lane's pointers at the chunk's first rows (columns clamped into the
  // row); step s adds 4 s rows, clamped to the chunk's last whole step, a
  // wave-uniform offset
  const float* pa = A + (kb + g) * lda + min(m0 + 4 * x, (M - 1) / 4 * 4);
  const float* pb[NB];
#pragma unroll
  for (int j = 0; j < NB; ++j) pb[j] = B + (kb + g) * ldb + min(n0 + 16 * j + x, N - 1);
  const int64_t ns = (ke - kb) / 4;  // full 4-row steps
  f4 acc[4][NB];
#pragma unroll
  for (int c = 0; c < 4; ++c)
#pragma unroll
    for (int j = 0; j < NB; ++j) acc[c][j] = f4{0.f, 0.f, 0.f, 0.f};
  // operands of step s: rows kb + 4 s + g (s clamped to the last whole step)
  auto load = [&](int64_t s, f4& ra, f4& rb) {
    const int64_t r4 = 4 * min(s, ns - 1);
    ra = *reinterpret_cast<const f4*>(pa + r4 * lda);
#pragma unroll
    for (int j = 0; j < NB; ++j) rb[j] = pb[j][r4 * ldb];
  };
  auto mma = [&](const f4& ra, const f4& rb) {
#pragma unroll
    for (int c = 0; c < 4; ++c)
#pragma unroll
      for (int j = 0; j < NB; ++j)
        acc[c][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(ra[c], rb[j], acc[c][j], 0, 0, 0);
  };
  constexpr int SPG = D * CPS;  // steps per group
  const int64_t NG = ns / SPG;
  f4 ra[D][CPS], rb[D][CPS];  // B words in the first NB elements
  auto group = [&](int64_t gi) {
#pragma unroll
    for (int d = 0; d < D; ++d) {
#pragma unroll
      for (int c = 0; c < CPS; ++c) mma(ra[d][c], rb[d][c]);
#pragma unroll
      for (int c = 0; c < CPS; ++c) load((gi + 1) * SPG + d * CPS + c, ra[d][c], rb[d][c]);
      // keep the slots in order (the scheduler would sink the refills)
      __builtin_amdgcn_sched_barrier(0);
    }
  };
  if (NG > 0) {
#pragma unroll
    for (int d = 0; d < D; ++d)
#pragma unroll
      for (int c = 0; c < CPS; ++c) load(d * CPS + c, ra[d][c], rb[d][c]);
    // the first group is peeled (the wait analysis of the loop then keeps
    // one slot's wait per slot)
    group(0);
    for (int64_t gi = 1; gi < NG; ++gi) group(gi);
  }
  // the steps after the last whole group, then the rows of a partial step
  for (int64_t s = NG * SPG; s < ns; ++s) {
    f4 a, bv;
    load(s, a, bv);
    mma(a, bv);
  }
  if (kb + 4 * ns < ke) {
    // rows kb + 4 ns + g, those past the chunk clamped to its last row
    f4 a, bv = f4{0.f, 0.f, 0.f, 0.f};
    const int64_t row = min(kb + 4 * ns + g, ke - 1) - (kb + g);
    a = *reinterpret_cast<const f4*>(pa + row * lda);
#pragma unroll
    for (int j = 0; j < NB; ++j) bv[j] = pb[j][row * ldb];
    if (kb + 4 * ns + g >= ke) a = bv = f4{0.f, 0.f, 0.f, 0.f};
    mma(a, bv);
  }
  // element i of block (c, j): row m0 + 4 (4 g + i) + c, column n0 + 16 j + x
  float* out = part + chunk * M * N;
#pragma unroll
  for (int c = 0; c < 4; ++c)
#pragma unroll
    for (int j = 0; j < NB; ++j)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int64_t gm = m0 + 16 * g + 4 * i + c, gn = n0 + 16 * j + x;
        if (gm < M && gn < N) out[gm * N + gn] = acc[c][j][i];
      }
}

// C[m][n] = sum over chunks of part[chunk][m][n] in a fixed order: a
// workgroup takes 64 consecutive elements; its wavefront g adds chunks g,
// g + 4, g + 8, ... in turn (16 loads in flight), and the four sums are added
// in wavefront order.
__global__ __launch_bounds__(kThreads) void k_sum_partials(int64_t M, int64_t N, int64_t n_chunks,
                                                           const float* __restrict__ part,
                                                           float* __restrict__ C, int64_t ldc) {
  __shared__ float red[kThreads / 64][64];
  constexpr int kW = kThreads / 64, U = 16;
  const int lane = threadIdx.x & 63, g = threadIdx.x >> 6;
  const int64_t e = (int64_t)blockIdx.x * 64 + lane;
  const int64_t MN = M * N;
  float s = 0.f;
  if (e < MN) {
    int64_t c = g;
    for (; c + (U - 1) * kW < n_chunks; c += U * kW) {
      float v[U];
#pragma unroll
      for (int u = 0; u < U; ++u) v[u] = part[(c + u * kW) * MN + e];
#pragma unroll
      for (int u = 0; u < U; ++u) s += v[u];
    }
    for (; c < n_chunks; c += kW) s += part[c * MN + e];
  }
  red[g][lane] = s;
  __syncthreads();
  if (g == 0 && e < MN) {
    float t = red[0][lane];
#pragma unroll
    for (int w = 1; w < kW; ++w) t += red[w][lane];
    C[(e / N) * ldc + (e % N)] = t;
  }
}

// Backward of GCN layer 1 when it aggregates first (H1 = relu(P W1),
// P = A_hat X, Z2 = H1 W2), fused over one chunk of rows:
//   dZ1 = (dZ2 W2^T) masked by H1 > 0,   dW1 += P^T dZ1,   dW2 += H1^T dZ2.
// dZ1 never leaves the registers: of the three separate products (dZ1 stored,
// then read back by P^T dZ1 beside a second pass over H1 for H1^T dZ2) only
// the operand reads remain.
//
// Workgroup (chunk, hidden slice of 128 columns), one wavefront per SIMD
// (the accumulators and two sets of operands take about 450 VGPRs and
// AGPRs); wavefront w owns the two 16-column blocks hs + 16 hb (hb = 0, 1,
// hs = 128 slice + 32 w) of the hidden layer and walks the chunk in groups of
// 16 rows r0 ... r0 + 15. Lane (g = l / 16, x = l % 16), per group:
//  * dH1 block hb = dZ2[r0 .. r0 + 15] W2^T: the A operand is a 16-byte piece
//    dZ2[r0 + x][16 j + 4 g .. + 3] (step i of chunk j contracts over class
//    16 j + 4 g + i), the B operand W2[col][16 j + 4 g + i] is kept in
//    registers for the whole kernel; classes past C are zero on both sides.
//    Result element i is dH1[r0 + 4 g + i][col], col = hs + 16 hb + x.
//  * dZ1 = that element where H1[r0 + 4 g + i][col] > 0, else 0.
//  * The result layout is the B operand layout of a product contracting
//    over the rows r0 + 4 g + i (g = 0 .. 3) at step i: dZ1 element i is the
//    B operand of P^T dZ1 (A operand P[r0 + 4 g + i][16 b + x], one per
//    16-row block b of dW1), and the H1 value read for the mask is the A
//    operand of H1^T dZ2 (B operand dZ2[r0 + 4 g + i][16 c + x]).
// The next group's operands are loaded while the current one is multiplied
// (two register sets in turn).
// Columns past f_in, hidden or C read a valid column of their row and reach
// only outputs that are not stored; rows past the chunk are zero. Chunk
// partials go to part1 [chunks][f_in][hidden] and part2 [chunks][hidden][C],
// summed in chunk order by k_sum_partials.
#ifndef GCN_LAYER1_FUSED
#define GCN_LAYER1_FUSED 1
#endif
struct Bwd1Args {
  int64_t n, split;
  int f_in, hidden, C;
  const float* P;
  int64_t ldp;
  const float* H1;
  int64_t ldh;
  const float* dZ2;
  int64_t ldc;
  const float* W2;  // [hidden][ldw], 16-byte aligned rows
  int64_t ldw;
  float* part1;
  float* part2;
};

template <int MB, int CB>
struct Bwd1Ops {
  f4 az[CB];      // dZ2[r0 + x][16 j + 4 g ...]
  float h[2][4];  // H1[r0 + 4 g + i][col(hb)]
  float p[MB][4]; // P[r0 + 4 g + i][16 b + x]
  float z[CB][4]; // dZ2[r0 + 4 g + i][16 c + x]
};

constexpr int kBwd1Waves = 4;

template <int MB, int CB>
__global__ __launch_bounds__(64 * kBwd1Waves) void k_gcn_bwd1(Bwd1Args a) {
  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
  const int hs = (int)blockIdx.y * (32 * kBwd1Waves) + 32 * w;
  if (hs >= a.hidden) return;
  const int g = lane >> 4, x = lane & 15;
  const int64_t kb = (int64_t)blockIdx.x * a.split;
  const int64_t ke = min(a.n, kb + a.split);
  int hcol[2];
#pragma unroll
  for (int hb = 0; hb < 2; ++hb) hcol[hb] = min(hs + 16 * hb + x, a.hidden - 1);
  // W2^T operands: class 16 j + 4 g + i of hidden unit hcol[hb] (classes
  // past C read an in-row piece and are zeroed)
  f4 wt[2][CB];
#pragma unroll
  for (int hb = 0; hb < 2; ++hb)
#pragma unroll
    for (int j = 0; j < CB; ++j) {
      const int k0 = 16 * j + 4 * g;
      f4 v = *reinterpret_cast<const f4*>(a.W2 + (int64_t)hcol[hb] * a.ldw +
                                          min(k0, (int)a.ldw - 4));
#pragma unroll
      for (int e = 0; e < 4; ++e) v[e] = k0 + e < a.C ? v[e] : 0.f;
      wt[hb][j] = v;
    }
  int pcol[MB], zcol[CB], acol[CB];
#pragma unroll
  for (int b = 0; b < MB; ++b) pcol[b] = min(16 * b + x, a.f_in - 1);
#pragma unroll
  for (int c = 0; c < CB; ++c) zcol[c] = min(16 * c + x, a.C - 1);
#pragma unroll
  for (int j = 0; j < CB; ++j) acol[j] = min(16 * j + 4 * g, (int)a.ldc - 4);
  // lane byte offsets from a group's first row r0, the same for every whole
  // group: rows r0 + 4 g + i start at the wave-uniform row r0 + i (32-bit
  // offsets on a wave-uniform base: one register per load)
  uint32_t oh[2], op[MB], oz[CB], oa[CB];
#pragma unroll
  for (int hb = 0; hb < 2; ++hb) oh[hb] = (uint32_t)(4 * (4 * g * a.ldh + hcol[hb]));
#pragma unroll
  for (int b = 0; b < MB; ++b) op[b] = (uint32_t)(4 * (4 * g * a.ldp + pcol[b]));
#pragma unroll
  for (int c = 0; c < CB; ++c) oz[c] = (uint32_t)(4 * (4 * g * a.ldc + zcol[c]));
#pragma unroll
  for (int j = 0; j < CB; ++j) oa[j] = (uint32_t)(4 * (x * a.ldc + acol[j]));
  auto at = [](const float* base, uint32_t off) __attribute__((always_inline)) {
    return reinterpret_cast<const char*>(base) + off;
  };
  // operands of the 16 rows from r0; without FULL, rows at or past ke are
  // zero (the chunk's last, partial group)
  auto load = [&](auto full_t, int64_t r0, Bwd1Ops<MB, CB>& o) __attribute__((always_inline)) {
    constexpr bool FULL = decltype(full_t)::value;
    // the pieces of dZ2 are stored as loaded: their classes past C are
    // zeroed where they are used (a select here would wait for the load)
    if constexpr (FULL) {
      const float* za = a.dZ2 + r0 * a.ldc;
#pragma unroll
      for (int j = 0; j < CB; ++j) o.az[j] = *reinterpret_cast<const f4*>(at(za, oa[j]));
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float* hr = a.H1 + (r0 + i) * a.ldh;
        const float* pr = a.P + (r0 + i) * a.ldp;
        const float* zr = a.dZ2 + (r0 + i) * a.ldc;
#pragma unroll
        for (int hb = 0; hb < 2; ++hb) o.h[hb][i] = *reinterpret_cast<const float*>(at(hr, oh[hb]));
#pragma unroll
        for (int b = 0; b < MB; ++b) o.p[b][i] = *reinterpret_cast<const float*>(at(pr, op[b]));
#pragma unroll
        for (int c = 0; c < CB; ++c) o.z[c][i] = *reinterpret_cast<const float*>(at(zr, oz[c]));
      }
    } else {
      // rows past the chunk: a zero piece (whose classes are then all
      // dropped) and zero operands
      const int64_t ra = min(r0 + x, ke - 1);
      const bool live_a = r0 + x < ke;
#pragma unroll
      for (int j = 0; j < CB; ++j) {
        const f4 v = *reinterpret_cast<const f4*>(a.dZ2 + ra * a.ldc + acol[j]);
        o.az[j] = live_a ? v : f4{0.f, 0.f, 0.f, 0.f};
      }
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int64_t r = min(r0 + 4 * g + i, ke - 1);
        const bool live = r0 + 4 * g + i < ke;
#pragma unroll
        for (int hb = 0; hb < 2; ++hb) {
          const float v = a.H1[r * a.ldh + hcol[hb]];
          o.h[hb][i] = live ? v : 0.f;
        }
#pragma unroll
        for (int b = 0; b < MB; ++b) {
          const float v = a.P[r * a.ldp + pcol[b]];
          o.p[b][i] = live ? v : 0.f;
        }
#pragma unroll
        for (int c = 0; c < CB; ++c) {
          const float v = a.dZ2[r * a.ldc + zcol[c]];
          o.z[c][i] = live ? v : 0.f;
        }
      }
    }
  };
  f4 acc1[MB][2], acc2[2][CB];
#pragma unroll
  for (int b = 0; b < MB; ++b)
#pragma unroll
    for (int hb = 0; hb < 2; ++hb) acc1[b][hb] = f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int hb = 0; hb < 2; ++hb)
#pragma unroll
    for (int c = 0; c < CB; ++c) acc2[hb][c] = f4{0.f, 0.f, 0.f, 0.f};
  auto mma = [&](const Bwd1Ops<MB, CB>& o) __attribute__((always_inline)) {
    // classes past C are zero on both sides of dZ2 W2^T (dZ2's padding may
    // hold anything)
    f4 azc[CB];
#pragma unroll
    for (int j = 0; j < CB; ++j)
#pragma unroll
      for (int e = 0; e < 4; ++e) azc[j][e] = 16 * j + 4 * g + e < a.C ? o.az[j][e] : 0.f;
    float dz[2][4];
#pragma unroll
    for (int hb = 0; hb < 2; ++hb) {
      f4 d = f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int j = 0; j < CB; ++j)
#pragma unroll
        for (int i = 0; i < 4; ++i)
          d = __builtin_amdgcn_mfma_f32_16x16x4f32(azc[j][i], wt[hb][j][i], d, 0, 0, 0);
#pragma unroll
      for (int i = 0; i < 4; ++i) dz[hb][i] = o.h[hb][i] > 0.f ? d[i] : 0.f;
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
#pragma unroll
      for (int b = 0; b < MB; ++b)
#pragma unroll
        for (int hb = 0; hb < 2; ++hb)
          acc1[b][hb] = __builtin_amdgcn_mfma_f32_16x16x4f32(o.p[b][i], dz[hb][i], acc1[b][hb],
                                                             0, 0, 0);
#pragma unroll
      for (int hb = 0; hb < 2; ++hb)
#pragma unroll
        for (int c = 0; c < CB; ++c)
          acc2[hb][c] = __builtin_amdgcn_mfma_f32_16x16x4f32(o.h[hb][i], o.z[c][i], acc2[hb][c],
                                                             0, 0, 0);
    }
  };
  // the next set's loads issued one per matrix-core operation over the
  // first part of the current set's products (in a phase of their own before
  // the products the step's kernel took 2.33 instead of 2.28 ms)
  auto interleave = [&]() __attribute__((always_inline)) {
    constexpr int kLoads = CB + 4 * (2 + MB + CB);
#pragma unroll
    for (int k = 0; k < kLoads; ++k) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
    }
    __builtin_amdgcn_sched_barrier(0);
  };
  using Full = std::integral_constant<bool, true>;
  using Part = std::integral_constant<bool, false>;
  const int64_t nf = (ke - kb) / 16;  // whole groups
  if (nf > 0) {
    // two operand sets in turn: while one group is multiplied the next one's
    // operands load (the last group again where none is left: loaded, unused)
    Bwd1Ops<MB, CB> o0, o1;
    load(Full{}, kb, o0);
    int64_t t = 0;
    for (; t + 2 <= nf; t += 2) {
      load(Full{}, kb + 16 * (t + 1), o1);
      mma(o0);
      interleave();
      load(Full{}, kb + 16 * min(t + 2, nf - 1), o0);
      mma(o1);
      interleave();
    }
    if (t < nf) mma(o0);
  }
  if (kb + 16 * nf < ke) {
    Bwd1Ops<MB, CB> o;
    load(Part{}, kb + 16 * nf, o);
    mma(o);
  }
  // element i of acc1[b][hb]: dW1[16 b + 4 g + i][hs + 16 hb + x];
  // element i of acc2[hb][c]: dW2[hs + 16 hb + 4 g + i][16 c + x]
  float* o1 = a.part1 + (int64_t)blockIdx.x * a.f_in * a.hidden;
  float* o2 = a.part2 + (int64_t)blockIdx.x * a.hidden * a.C;
#pragma unroll
  for (int hb = 0; hb < 2; ++hb) {
    const int col = hs + 16 * hb + x;
#pragma unroll
    for (int b = 0; b < MB; ++b)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int m = 16 * b + 4 * g + i;
        if (m < a.f_in && col < a.hidden) o1[(int64_t)m * a.hidden + col] = acc1[b][hb][i];
      }
#pragma unroll
    for (int c = 0; c < CB; ++c)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int m = hs + 16 * hb + 4 * g + i, cls = 16 * c + x;
        if (m < a.hidden && cls < a.C) o2[(int64_t)m * a.C + cls] = acc2[hb][c][i];
      }
  }
}

// Forward of a GCN first layer that aggregates first, fused over groups of
// 16 rows: H1 = relu(P W1) is stored and Z2 = H1 W2 computed from it while it
// is still in registers (the separate Z2 product re-read H1).
//
// The weights sit in LDS in matrix-core operand order, filled once per
// workgroup: W1^T as [hidden block hb][step s][lane] = W1[4 s + l / 16][16 hb +
// l % 16] and W2 as [hb][class block c][i][lane] = W2[16 hb + 4 (l / 16) + i]
// [16 c + l % 16], zero outside f_in, hidden and C. Every wavefront then takes
// its own row groups r0 ... r0 + 15 (no barriers, no exchange between
// wavefronts). Lane (g = l / 16, x = l % 16), per hidden block hb:
//  * H1^T block = W1^T P^T over the steps s (input features 4 s + g): the B
//    operand is P[r0 + x][4 s + g], loaded for the whole group (the next
//    group's while this one is multiplied). Result element i is
//    H1[r0 + x][16 hb + 4 g + i]: after the ReLU one 16-byte store of H1.
//  * Those four elements are the A operand of H1 W2 at the steps that
//    contract over hidden units 16 hb + 4 g + i: Z2 accumulates in registers
//    over the hidden blocks and is stored once per group.
// Steps s >= ceil(f_in / 4) of the fixed step count S are multiplied by zero
// operands (their LDS reads are clamped into the table).
struct Fwd1Args {
  int64_t n;
  int f_in, hidden, C;
  const float* P;  // [n][ldp]
  int64_t ldp;
  const float* W1;  // [f_in][ldw1]
  int64_t ldw1;
  const float* W2;  // [hidden][ldw2]
  int64_t ldw2;
  float* H1;  // [n][ldh], 16-byte aligned rows
  int64_t ldh;
  float* Z2;  // [n][ldz]
  int64_t ldz;
};

constexpr int kFwd1Waves = 16;

template <int S, int CB>
__global__ __launch_bounds__(64 * kFwd1Waves) void k_gcn_fwd1(Fwd1Args a) {
  extern __shared__ __align__(16) float lds[];
  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
  const int g = lane >> 4, x = lane & 15;
  const int hbn = (a.hidden + 15) / 16;  // hidden blocks
  const int sn = (a.f_in + 3) / 4;       // steps with data (<= S)
  float* lw1 = lds;                      // [hbn][sn][64]
  float* lw2 = lds + hbn * sn * 64;      // [hbn][CB][4][64]
  for (int e = threadIdx.x; e < hbn * sn * 64; e += blockDim.x) {
    const int l = e & 63, st = (e >> 6) % sn, hb = (e >> 6) / sn;
    const int k = 4 * st + (l >> 4), col = 16 * hb + (l & 15);
    lw1[e] = k < a.f_in && col < a.hidden ? a.W1[(int64_t)k * a.ldw1 + col] : 0.f;
  }
  for (int e = threadIdx.x; e < hbn * CB * 4 * 64; e += blockDim.x) {
    const int l = e & 63, i = (e >> 6) & 3, c = (e >> 8) % CB, hb = (e >> 8) / CB;
    const int u = 16 * hb + 4 * (l >> 4) + i, cls = 16 * c + (l & 15);
    lw2[e] = u < a.hidden && cls < a.C ? a.W2[(int64_t)u * a.ldw2 + cls] : 0.f;
  }
  __syncthreads();
  const int64_t ng = (a.n + 15) / 16;
  const int64_t stride = (int64_t)gridDim.x * (blockDim.x >> 6);
  int64_t grp = (int64_t)blockIdx.x * (blockDim.x >> 6) + w;
  if (grp >= ng) return;
  // P operands of a group: P[r0 + x][4 s + g] (ldp >= 4 sn keeps them in the
  // row); rows past n read the last row and reach only rows of H1 and Z2
  // that are not stored; steps past sn read step sn - 1 and are zeroed where
  // used, as are features past f_in (the row's padding may hold anything)
  auto load = [&](int64_t gi, float (&pv)[S]) __attribute__((always_inline)) {
    const float* row = a.P + min(16 * gi + x, a.n - 1) * a.ldp + g;
#pragma unroll
    for (int st = 0; st < S; ++st) pv[st] = row[4 * min(st, sn - 1)];
  };
  auto compute = [&](int64_t gi, float (&pz)[S]) __attribute__((always_inline)) {
    const int64_t r0 = 16 * gi;
    const bool live = r0 + x < a.n;
#pragma unroll
    for (int st = 0; st < S; ++st) pz[st] = 4 * st + g < a.f_in ? pz[st] : 0.f;
    f4 z[CB];
#pragma unroll
    for (int c = 0; c < CB; ++c) z[c] = f4{0.f, 0.f, 0.f, 0.f};
    const float* w1 = lw1 + lane;
    const float* w2 = lw2 + lane;
    for (int hb = 0; hb < hbn; ++hb) {
      // W1 operands from LDS: 8 reads ahead, then one read per product (read
      // next to its product, each read's latency was exposed)
      float wa[S];
#pragma unroll
      for (int st = 0; st < S; ++st) wa[st] = w1[64 * min(st, sn - 1)];
      f4 h = f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int st = 0; st < S; ++st)
        h = __builtin_amdgcn_mfma_f32_16x16x4f32(wa[st], pz[st], h, 0, 0, 0);
      constexpr int kAhead = S < 8 ? S : 8;
#pragma unroll
      for (int k = 0; k < kAhead; ++k) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
#pragma unroll
      for (int k = 0; k < S - kAhead; ++k) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
      }
      __builtin_amdgcn_sched_group_barrier(0x008, kAhead, 0);
      w1 += 64 * sn;
#pragma unroll
      for (int i = 0; i < 4; ++i) h[i] = fmaxf(h[i], 0.f);
      const int c0 = 16 * hb + 4 * g;
      if (live) {
        float* dst = a.H1 + (r0 + x) * a.ldh + c0;
        if (c0 + 4 <= a.hidden)
          *reinterpret_cast<f4*>(dst) = h;
        else
          for (int e = 0; e < 4 && c0 + e < a.hidden; ++e) dst[e] = h[e];
      }
      float wb[CB][4];
#pragma unroll
      for (int c = 0; c < CB; ++c)
#pragma unroll
        for (int i = 0; i < 4; ++i) wb[c][i] = w2[64 * (4 * c + i)];
#pragma unroll
      for (int c = 0; c < CB; ++c)
#pragma unroll
        for (int i = 0; i < 4; ++i)
          z[c] = __builtin_amdgcn_mfma_f32_16x16x4f32(h[i], wb[c][i], z[c], 0, 0, 0);
      w2 += 64 * 4 * CB;
    }
    // element i of z[c]: Z2[r0 + 4 g + i][16 c + x]
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int64_t row = r0 + 4 * g + i;
      if (row < a.n)
#pragma unroll
        for (int c = 0; c < CB; ++c)
          if (16 * c + x < a.C) a.Z2[row * a.ldz + 16 * c + x] = z[c][i];
    }
  };
  // two sets of P operands in turn; the group after the last is the last again
  float p0[S], p1[S];
  load(grp, p0);
  for (;;) {
    const int64_t g1 = grp + stride;
    load(min(g1, ng - 1), p1);
    compute(grp, p0);
    if (g1 >= ng) break;
    const int64_t g2 = g1 + stride;
    load(min(g2, ng - 1), p0);
    compute(g1, p1);
    if (g2 >= ng) break;
    grp = g2;
  }
}

// Backward of a GraphSAGE layer that aggregates Y W_neigh (its output is
// narrower than its input), fused with the LayerNorm backward of its input:
//   dY = DG [W_self | W_neigh]^T,  DG = [dO | G]  (K = 2 fop columns),
//   dX = rstd (dY - mean(dY) - Y mean(dY Y)) where mask > 0, else 0,
// with mask the ReLU output of the layer below, overwritten by dX. dY never
// leaves the registers (the separate product stored it and the LayerNorm
// backward read it back).
//
// [W_self | W_neigh] sits in LDS in matrix-core operand order, [b][s][lane] =
// B[16 b + l % 16][4 s + l / 16] for the 16-column blocks b of dY and the
// 4-deep steps s; each wavefront stages its own 16 x K tile of DG in LDS as
// [s][lane] = DG[r0 + l % 16][4 s + l / 16] and walks its own row groups.
// Result element i of block b in lane (g, x) is dY[r0 + 4 g + i][16 b + x]:
// the row sums of the LayerNorm backward add the lane's NB blocks, then the
// 16 lanes x of the row (DPP, in double, as the separate kernel sums in
// double).
struct TfBwdArgs {
  int64_t n;
  int F, K;         // F = 16 NB, K a multiple of 4
  const float* dg;  // [n][ldg], 16-byte aligned rows
  int64_t ldg;
  const float* bw;  // [F][ldb]
  int64_t ldb;
  const float* y;  // [n][ldy]
  int64_t ldy;
  const float* rstd;
  float* dx;  // [n][ldx]: the mask on entry, dX on return
  int64_t ldx;
};

constexpr int kTfWaves = 8;

template <int OFF>
__device__ inline double row16_partner_d(double v) {
  constexpr int kCtrl = OFF == 1 ? 0xB1 : OFF == 2 ? 0x4E : OFF == 4 ? 0x141 : 0x140;
  const int lo = __builtin_amdgcn_mov_dpp(__double2loint(v), kCtrl, 0xF, 0xF, false);
  const int hi = __builtin_amdgcn_mov_dpp(__double2hiint(v), kCtrl, 0xF, 0xF, false);
  return __hiloint2double(hi, lo);
}

__device__ inline double row16_sum_d(double v) {
  v += row16_partner_d<1>(v);
  v += row16_partner_d<2>(v);
  v += row16_partner_d<4>(v);
  return v + row16_partner_d<8>(v);
}

template <int NB>
__global__ __launch_bounds__(64 * kTfWaves) void k_sage_tf_bwd(TfBwdArgs a) {
  extern __shared__ __align__(16) float lds[];
  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
  const int g = lane >> 4, x = lane & 15;
  const int ks = a.K / 4;
  float* tb = lds;                                 // [NB][ks][64]
  float* ds = lds + (NB + w) * ks * 64;            // this wavefront's [ks][64]
  for (int e = threadIdx.x; e < NB * ks * 64; e += blockDim.x) {
    const int l = e & 63, st = (e >> 6) % ks, b = (e >> 6) / ks;
    tb[e] = a.bw[(int64_t)(16 * b + (l & 15)) * a.ldb + 4 * st + (l >> 4)];
  }
  __syncthreads();
  const int64_t ng = (a.n + 15) / 16;
  const int64_t stride = (int64_t)gridDim.x * kTfWaves;
  for (int64_t grp = (int64_t)blockIdx.x * kTfWaves + w; grp < ng; grp += stride) {
    const int64_t r0 = 16 * grp;
    // the DG tile: piece p (row p / ks, columns 4 (p % ks) .. + 3); rows
    // past n are zero
    for (int p = lane; p < 16 * ks; p += 64) {
      const int r = p / ks, st = p % ks;
      float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
      if (r0 + r < a.n) v = *reinterpret_cast<const float4*>(a.dg + (r0 + r) * a.ldg + 4 * st);
      ds[st * 64 + r] = v.x;
      ds[st * 64 + 16 + r] = v.y;
      ds[st * 64 + 32 + r] = v.z;
      ds[st * 64 + 48 + r] = v.w;
    }
    __builtin_amdgcn_wave_barrier();
    // Y of the group's rows, loaded while the products run (rows past n read
    // the last row and are not stored)
    float yv[NB][4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int64_t row = min(r0 + 4 * g + i, a.n - 1);
#pragma unroll
      for (int b = 0; b < NB; ++b) yv[b][i] = a.y[row * a.ldy + 16 * b + x];
    }
    f4 acc[NB];
#pragma unroll
    for (int b = 0; b < NB; ++b) acc[b] = f4{0.f, 0.f, 0.f, 0.f};
    for (int st = 0; st < ks; ++st) {
      const float av = ds[st * 64 + lane];
      float bv[NB];
#pragma unroll
      for (int b = 0; b < NB; ++b) bv[b] = tb[(b * ks + st) * 64 + lane];
#pragma unroll
      for (int b = 0; b < NB; ++b)
        acc[b] = __builtin_amdgcn_mfma_f32_16x16x4f32(av, bv[b], acc[b], 0, 0, 0);
    }
    // the tile's operand reads are done before the next group's writes
    __builtin_amdgcn_wave_barrier();
    double s1[4], s2[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      s1[i] = 0.0;
      s2[i] = 0.0;
    }
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int b = 0; b < NB; ++b) {
        s1[i] += (double)acc[b][i];
        s2[i] += (double)acc[b][i] * (double)yv[b][i];
      }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int64_t row = r0 + 4 * g + i;
      const double m1 = row16_sum_d(s1[i]) / (double)a.F;
      const double m2 = row16_sum_d(s2[i]) / (double)a.F;
      if (row >= a.n) continue;
      const double r = (double)a.rstd[row];
      float* out = a.dx + row * a.ldx;
#pragma unroll
      for (int b = 0; b < NB; ++b) {
        const float mk = out[16 * b + x];
        const float d = (float)(r * ((double)acc[b][i] - m1 - (double)yv[b][i] * m2));
        out[16 * b + x] = mk > 0.f ? d : 0.f;
      }
    }
  }
}

// one wavefront per row
__global__ __launch_bounds__(kThreads) void k_relu(int64_t n, int64_t F, float* __restrict__ h,
                                                   int64_t ld) {
  const int64_t i = (int64_t)blockIdx.x * (kThreads / 64) + (threadIdx.x >> 6);
  if (i >= n) return;
  float* row = h + i * ld;
  for (int64_t f = threadIdx.x & 63; f < F; f += 64) row[f] = fmaxf(row[f], 0.f);
}

// dh[i, f] = 0 where h[i, f] <= 0 (h = relu(a), so h > 0 exactly where a > 0)
__global__ __launch_bounds__(kThreads) void k_relu_bwd(int64_t n, int64_t F,
                                                       const float* __restrict__ h, int64_t ldh,
                                                       float* __restrict__ dh, int64_t ld) {
  const int64_t i = (int64_t)blockIdx.x * (kThreads / 64) + (threadIdx.x >> 6);
  if (i >= n) return;
  for (int64_t f = threadIdx.x & 63; f < F; f += 64)
    if (!(h[i * ldh + f] > 0.f)) dh[i * ld + f] = 0.f;
}

constexpr int kSoftmaxRowsPerWave = 16;

__global__ void k_zero_count(unsigned long long* __restrict__ cnt) {
  if (threadIdx.x == 0) *cnt = 0ull;
}

// Rows that count in the loss: those with skip[i] == 0 (all rows without a
// skip array). cnt receives their number (integer atomics: exact).
__global__ __launch_bounds__(kThreads) void k_count_kept(int64_t n, const uint8_t* __restrict__ skip,
                                                         unsigned long long* __restrict__ cnt) {
  const int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  const bool keep = i < n && skip[i] == 0;
  const unsigned long long b = __ballot(keep);
  if ((threadIdx.x & 63) == 0 && b) atomicAdd(cnt, (unsigned long long)__popcll(b));
}

// Partner of a lane at distance 1, 2, 4 or 8 within its row of 16 lanes:
// quad permutations, then the mirrors of the half row and of the row. After
// the earlier steps of a butterfly every lane of a quad (half row) holds the
// same value, so the mirror partner carries the operand of lane ^ 4 (^ 8).
template <int OFF>
__device__ inline float row16_partner(float v) {
  const int x = __float_as_int(v);
  constexpr int kCtrl = OFF == 1 ? 0xB1 : OFF == 2 ? 0x4E : OFF == 4 ? 0x141 : 0x140;
  return __int_as_float(__builtin_amdgcn_mov_dpp(x, kCtrl, 0xF, 0xF, false));
}

__device__ inline float row16_max(float v) {
  v = fmaxf(v, row16_partner<1>(v));
  v = fmaxf(v, row16_partner<2>(v));
  v = fmaxf(v, row16_partner<4>(v));
  return fmaxf(v, row16_partner<8>(v));
}

__device__ inline float row16_sum(float v) {
  v += row16_partner<1>(v);
  v += row16_partner<2>(v);
  v += row16_partner<4>(v);
  return v + row16_partner<8>(v);
}

// Softmax cross-entropy over C <= 16 NS classes. A row of 16 lanes holds one
// row of logits (lane l: classes l, l + 16, ...), so a wavefront works on 4
// rows at a time and its 16 rows in 4 steps, with every load of the 16 rows
// issued before any arithmetic. Per row: log-softmax with the row maximum
// subtracted, the loss lse - z[y] (z[y] read directly), and
// dz = (softmax - onehot(y)) / m, where m is the number of rows in the loss
// (n, or *n_kept when skip is given; skipped rows get dz = 0 and add
// nothing). The row losses of a wavefront are added in row order in double,
// the wavefront sums in wavefront order.
template <int NS>
__global__ __launch_bounds__(kThreads) void k_softmax_xent(int64_t n, int C,
                                                           const float* __restrict__ z, int64_t ldz,
                                                           const int32_t* __restrict__ y,
                                                           float* __restrict__ dz, int64_t ldd,
                                                           double* __restrict__ block_loss,
                                                           const uint8_t* __restrict__ skip,
                                                           const unsigned long long* __restrict__ n_kept) {
  constexpr int kSteps = kSoftmaxRowsPerWave / 4;
  __shared__ double wl[kThreads / 64];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int grp = lane >> 4, l = lane & 15;
  const int64_t base = ((int64_t)blockIdx.x * (kThreads / 64) + w) * kSoftmaxRowsPerWave;
  float v[kSteps][NS], zy[kSteps];
  int32_t yl[kSteps];
  bool use[kSteps];
#pragma unroll
  for (int st = 0; st < kSteps; ++st) {
    const int64_t i = base + 4 * st + grp;
    const bool live = i < n;
    use[st] = live && !(skip && skip[i]);
    yl[st] = live ? y[i] : 0;  // labels lie in [0, C)
#pragma unroll
    for (int k = 0; k < NS; ++k) {
      const int c = l + 16 * k;
      v[st][k] = live && c < C ? z[i * ldz + c] : -INFINITY;
    }
  }
  // z[y] of each row; the index is clamped to the row so that a label outside
  // [0, C) (a broken precondition) gives a wrong loss, never a read outside z
#pragma unroll
  for (int st = 0; st < kSteps; ++st)
    zy[st] = use[st] ? z[(base + 4 * st + grp) * ldz + min(max(yl[st], 0), C - 1)] : 0.f;
  const float m_rows = skip ? (float)*n_kept : (float)n;
  double rl[kSteps];
#pragma unroll
  for (int st = 0; st < kSteps; ++st) {
    const int64_t i = base + 4 * st + grp;
    float m = v[st][0];
#pragma unroll
    for (int k = 1; k < NS; ++k) m = fmaxf(m, v[st][k]);
    m = row16_max(m);
    float ex[NS], s = 0.f;
#pragma unroll
    for (int k = 0; k < NS; ++k) {
      ex[k] = l + 16 * k < C ? expf(v[st][k] - m) : 0.f;
      s += ex[k];
    }
    s = row16_sum(s);
    rl[st] = use[st] ? (double)(m + logf(s) - zy[st]) : 0.0;
    if (i < n) {
#pragma unroll
      for (int k = 0; k < NS; ++k) {
        const int c = l + 16 * k;
        if (c < C) dz[i * ldd + c] = use[st] ? (ex[k] / s - (c == yl[st] ? 1.f : 0.f)) / m_rows : 0.f;
      }
    }
  }
  // row 4 st + g of the wavefront sits in lane row g at step st
  double wave_loss = 0.0;
#pragma unroll
  for (int st = 0; st < kSteps; ++st)
#pragma unroll
    for (int g = 0; g < 4; ++g) wave_loss += __shfl(rl[st], 16 * g, 64);
  if (lane == 0) wl[w] = wave_loss;
  __syncthreads();
  if (threadIdx.x == 0) {
    double t = 0.0;
    for (int k = 0; k < kThreads / 64; ++k) t += wl[k];
    block_loss[blockIdx.x] = t;
  }
}

// loss = (sum of the block losses) / n by one workgroup in a fixed order:
// thread t adds blocks t, t + 256, ... in turn, then a fixed tree combines
// the 256 sums.
__global__ __launch_bounds__(kThreads) void k_loss_total(int64_t nb, int64_t n,
                                                         const double* __restrict__ block_loss,
                                                         double* __restrict__ loss,
                                                         const unsigned long long* __restrict__ n_kept) {
  __shared__ double part[kThreads];
  double s = 0.0;
  for (int64_t b = threadIdx.x; b < nb; b += kThreads) s += block_loss[b];
  part[threadIdx.x] = s;
  __syncthreads();
  for (int off = kThreads / 2; off > 0; off >>= 1) {
    if ((int)threadIdx.x < off) part[threadIdx.x] += part[threadIdx.x + off];
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    const double m = n_kept ? (double)*n_kept : (double)n;
    *loss = m > 0 ? part[0] / m : 0.0;
  }
}

}  // namespace

namespace {

bool aligned16(const void* p, int64_t ld) { return ((uintptr_t)p % 16) == 0 && ld % 4 == 0; }

// widest tile of 64, 128 or 256 columns that is not mostly padding
// Output tile widths. C = A B: 256 columns once N > 128 (A is read once per
// tile column). C = A B^T and C = A^T B: at most 128 (more workgroups at 4
// per CU, and less padding of odd widths, outweigh the extra reads of A).
// Outputs of at most 48 columns (the class count of the training steps, 47)
// take a 48-column tile: 3 instead of 4 matrix-core blocks per 16 rows.
int tile_n(int64_t N) { return N <= 48 ? 48 : (N <= 64 ? 64 : (N <= 128 ? 128 : 256)); }
int tile_n_narrow(int64_t N) { return N <= 48 ? 48 : (N <= 64 ? 64 : 128); }

// Compute units of the current device (cached per device).
int cu_count() {
  static std::mutex mu;
  static int cached[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  std::lock_guard<std::mutex> lk(mu);
  if (cached[dev] == 0) {
    int v = 0;
    if (hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        v <= 0)
      v = 256;
    cached[dev] = v;
  }
  return cached[dev];
}

#ifndef GCN_GEMM_RESIDENT
#define GCN_GEMM_RESIDENT 1
#endif
constexpr int64_t kResMinRows = 65536;       // below this the staged tile is used
constexpr int64_t kResMaxLds = 120 * 1024;   // LDS bytes for the resident B slice

template <int OP, int NBLK, int RB, int D, int CPS, int WAVES>
hipError_t launch_bres(int64_t M, int64_t N, int64_t K, const float* A, int64_t lda,
                       const float* B, int64_t ldb, float* C, int64_t ldc, const float* mask,
                       int64_t ldm, bool relu, bool cvec, hipStream_t stream) {
  const size_t lds = (size_t)((K + 15) / 16) * 16 * (16 * NBLK) * sizeof(float);
  auto kern = k_gemm_bres<OP, NBLK, RB, D, CPS, WAVES>;
  hipError_t e = hipFuncSetAttribute((const void*)kern,
                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  // one workgroup per CU (the B slice takes most of the LDS), at most one
  // tile per wavefront
  const int64_t tiles = ceil_div(M, (int64_t)16 * RB);
  const int64_t wg = std::min<int64_t>(cu_count(), ceil_div(tiles, (int64_t)WAVES));
  const dim3 grid((unsigned)wg, (unsigned)ceil_div(N, (int64_t)16 * NBLK));
  hipLaunchKernelGGL(kern, grid, dim3(64 * WAVES), lds, stream, M, N, K, A, lda, B, ldb, C, ldc,
                     mask, ldm, relu, cvec);
  return hipGetLastError();
}

// The resident-B kernel takes tall products whose B slice fits in LDS: 48
// columns (the class count, 47) or 256-column slices of outputs wider than
// 128 (the hidden layer). A ReLU-backward mask stays with the staged tile,
// which loads the mask values before it stages the output (in the resident
// kernel each tile would wait for them: the GCN step's dH1 took 1.46 ms
// against 1.17).
int resident_blocks(int64_t M, int64_t N, int64_t K, bool masked) {
  if (!GCN_GEMM_RESIDENT || M < kResMinRows || K < 16 || masked) return 0;
  const int nblk = N <= 48 ? 3 : (N > 128 ? 16 : 0);
  if (nblk == 0) return 0;
  const int64_t lds = ceil_div(K, (int64_t)16) * 16 * 16 * nblk * (int64_t)sizeof(float);
  return lds <= kResMaxLds ? nblk : 0;
}

template <int OP>
hipError_t launch_tall(int64_t M, int64_t N, int64_t K, const float* A, int64_t lda, const float* B,
                 int64_t ldb, float* C, int64_t ldc, const float* mask, int64_t ldm,
                 bool relu, hipStream_t stream) {
  const int bn = OP == kNN ? tile_n(N) : tile_n_narrow(N);
  // staged 16-byte stores need 16-byte aligned rows of C (and of the mask)
  const bool cvec = aligned16(C, ldc) && (!mask || aligned16(mask, ldm));
  const int nblk = resident_blocks(M, N, K, mask != nullptr);
  // ring: D slots of CPS chunks (D * CPS must divide the chunk count)
  const int64_t nc = K / 16;
#define GCN_BRES(D_, CPS_)                                                                 \
  return launch_bres<OP, 3, 2, D_, CPS_, 8>(M, N, K, A, lda, B, ldb, C, ldc, mask, ldm, relu, \
                                            cvec, stream)
  if (nblk == 3) {
    if (nc % 8 == 0) GCN_BRES(2, 4);
    if (nc % 4 == 0) GCN_BRES(2, 2);
    if (nc % 2 == 0) GCN_BRES(2, 1);
    GCN_BRES(1, 1);
  }
#undef GCN_BRES
  // 256 columns: one 16-row block per wavefront (64 accumulator registers),
  // one chunk per slot
#define GCN_BRES16(D_)                                                                      \
  return launch_bres<OP, 16, 1, D_, 1, 8>(M, N, K, A, lda, B, ldb, C, ldc, mask, ldm, relu, \
                                          cvec, stream)
  if (nblk == 16) {
    if (nc % 4 == 0) GCN_BRES16(4);
    if (nc % 3 == 0) GCN_BRES16(3);
    if (nc % 2 == 0) GCN_BRES16(2);
    GCN_BRES16(1);
  }
#undef GCN_BRES16
  const dim3 grid((unsigned)ceil_div(M, kTile), (unsigned)ceil_div(N, bn));
  if (bn == 48) {  // two 16-row blocks per wavefront (each B fragment feeds two MFMAs)
    const dim3 grid2((unsigned)ceil_div(M, (int64_t)kTile * 2), (unsigned)ceil_div(N, bn));
    hipLaunchKernelGGL((k_gemm_tall_v<OP, 48, 2>), grid2, dim3(kThreads), 0, stream, M, N, K, A,
                       lda, B, ldb, C, ldc, mask, ldm, relu, cvec);
  }
  else if (bn == 64)
    hipLaunchKernelGGL((k_gemm_tall_v<OP, 64, 1>), grid, dim3(kThreads), 0, stream, M, N, K, A,
                       lda, B, ldb, C, ldc, mask, ldm, relu, cvec);
  else if (OP != kNN || bn == 128)
    hipLaunchKernelGGL((k_gemm_tall_v<OP, 128, 1>), grid, dim3(kThreads), 0, stream, M, N, K, A,
                       lda, B, ldb, C, ldc, mask, ldm, relu, cvec);
  else if constexpr (OP == kNN) {
    if (K >= kDeepK) {  // deep products: 128 x 256 tiles
      const dim3 grid_w((unsigned)ceil_div(M, (int64_t)kTile * 2), (unsigned)ceil_div(N, bn));
      hipLaunchKernelGGL((k_gemm_tall_v<OP, 256, 2>), grid_w, dim3(kThreads), 0, stream, M, N,
                         K, A, lda, B, ldb, C, ldc, mask, ldm, relu, cvec);
    } else {
      hipLaunchKernelGGL((k_gemm_tall_v<OP, 256, 1>), grid, dim3(kThreads), 0, stream, M, N, K,
                         A, lda, B, ldb, C, ldc, mask, ldm, relu, cvec);
    }
  }
  return hipGetLastError();
}


// Output tiles of at most 128 rows; the wavefront count (16 rows each) is
// chosen so that the ceil(M / 128) tiles cover M with the least padding
// (M = 200: two tiles of 112 rows instead of 128; M = 47: one of 48).
void launch_tn(int64_t M, int64_t N, int64_t K, int64_t split, int64_t n_chunks, const float* A,
               int64_t lda, const float* B, int64_t ldb, float* part, hipStream_t stream) {
  const int64_t mb = ceil_div(M, (int64_t)16);
  const int waves = (int)ceil_div(mb, ceil_div(mb, (int64_t)8));
  const int bn = tile_n_narrow(N);
  const dim3 grid((unsigned)ceil_div(M, (int64_t)16 * waves), (unsigned)ceil_div(N, bn),
                  (unsigned)n_chunks);
  auto go = [&](auto kern) {
    hipLaunchKernelGGL(kern, grid, dim3(64 * waves), 0, stream, M, N, K, split, A, lda, B, ldb,
                       part);
  };
#define GCN_TNV(W_)                                        \
  case W_:                                                 \
    if (bn == 48)                                          \
      go(k_gemm_tn_v<W_, 48>);                             \
    else if (bn == 64)                                     \
      go(k_gemm_tn_v<W_, 64>);                             \
    else                                                   \
      go(k_gemm_tn_v<W_, 128>);                            \
    break
  switch (waves) {
    GCN_TNV(1); GCN_TNV(2); GCN_TNV(3); GCN_TNV(4);
    GCN_TNV(5); GCN_TNV(6); GCN_TNV(7);
    default: GCN_TNV(8);
  }
#undef GCN_TNV
}

// The streaming A^T B kernel: C tiles of 64 x 16 NB (N <= 64), at most 16 of
// them (one wavefront each, up to 8 per workgroup), K cut into chunks so that
// the chip holds about 8 wavefronts per CU; chunks are whole 32-row groups.
#ifndef GCN_GEMM_TN_STREAM
#define GCN_GEMM_TN_STREAM 1
#endif
constexpr int kTnsD = 4, kTnsCps = 2;
constexpr int64_t kTnsMinK = 65536;

struct TnsPlan {
  int nb = 0, m_tiles = 0, n_tiles = 0, wpw = 0, gy = 0;
  int64_t split = 0, n_chunks = 0;
};

TnsPlan tns_plan(int64_t M, int64_t N, int64_t K) {
  TnsPlan p;
  // outputs of at most 64 columns (the class layer): dW2 0.85 -> 0.63 ms;
  // for 256 columns (dW1) the staged tile was as fast
  if (!GCN_GEMM_TN_STREAM || K < kTnsMinK || N > 64) return p;
  const int nb = (int)ceil_div(N, (int64_t)16);
  const int64_t mt = ceil_div(M, (int64_t)64), nt = ceil_div(N, (int64_t)16 * nb);
  if (mt * nt > 16) return p;
  p.nb = nb;
  p.m_tiles = (int)mt;
  p.n_tiles = (int)nt;
  const int tiles = p.m_tiles * p.n_tiles;
  p.wpw = std::min(tiles, 8);
  p.gy = (int)ceil_div(tiles, p.wpw);
  const int64_t rows = 4 * kTnsD * kTnsCps;
  const int64_t want = std::max<int64_t>(1, (int64_t)cu_count() * 8 / tiles);
  p.split = ceil_div(ceil_div(K, want), rows) * rows;
  p.n_chunks = ceil_div(K, p.split);
  return p;
}

void launch_tns(const TnsPlan& p, int64_t M, int64_t N, int64_t K, const float* A, int64_t lda,
                const float* B, int64_t ldb, float* part, hipStream_t stream) {
  const dim3 grid((unsigned)p.n_chunks, (unsigned)p.gy), block(64 * p.wpw);
#define GCN_TNS(NB_)                                                                          \
  hipLaunchKernelGGL((k_gemm_tn_s<NB_, kTnsD, kTnsCps>), grid, block, 0, stream, M, N, K,    \
                     p.split, A, lda, B, ldb, part, p.m_tiles, p.n_tiles)
  switch (p.nb) {
    case 1: GCN_TNS(1); break;
    case 2: GCN_TNS(2); break;
    case 3: GCN_TNS(3); break;
    default: GCN_TNS(4); break;
  }
#undef GCN_TNS
}

}  // namespace

gcn_status gemm_f32(int op, int64_t M, int64_t N, int64_t K, const float* A, int64_t lda,
                    const float* B, int64_t ldb, float* C, int64_t ldc, hipStream_t stream,
                    const float* mask, int64_t ldm, bool relu) {
  if (M == 0 || N == 0) return GCN_OK;
  const bool vec = aligned16(A, lda) && aligned16(B, ldb);
  if (op == GCN_GEMM_TN) {
    // chunk length: kSplitRows, shrunk (down to kSplitRowsMin) when the output
    // has few tiles so the grid still fills the chip, and grown so the chunk
    // count fits the grid's z range
    const int64_t tiles = ceil_div(M, (int64_t)128) * ceil_div(N, (int64_t)tile_n_narrow(N));
    int64_t split = kSplitRows;
    while (split > kSplitRowsMin && tiles * ceil_div(K, split) < kTnMinBlocks) split /= 2;
    split = std::max<int64_t>(split, ceil_div(ceil_div(K, 65535), kKc) * kKc);
    int64_t n_chunks = std::max<int64_t>(1, ceil_div(K, split));
    // small outputs (up to 16 tiles of 64 x 64) stream both operands
    const TnsPlan tp = vec ? tns_plan(M, N, K) : TnsPlan();
    if (tp.nb) n_chunks = tp.n_chunks;
    float* part = nullptr;
    GCN_CHECK(talloc(&part, n_chunks * M * N, stream, "GEMM partials"));
    {
      ProfScope ps("gemm_tn_partial", stream);
      if (tp.nb)
        launch_tns(tp, M, N, K, A, lda, B, ldb, part, stream);
      else if (vec)
        launch_tn(M, N, K, split, n_chunks, A, lda, B, ldb, part, stream);
      else
        hipLaunchKernelGGL(k_gemm_tn_partial, dim3((unsigned)ceil_div(M, kTile),
                                                   (unsigned)ceil_div(N, kTile),
                                                   (unsigned)n_chunks),
                           dim3(kThreads), 0, stream, M, N, K, split, A, lda, B, ldb, part);
      hipError_t e = hipGetLastError();
      if (e != hipSuccess) {
        tfree(part, stream);
        return hip_fail(e, "k_gemm_tn_partial", __FILE__, __LINE__);
      }
    }
    {
      ProfScope ps("gemm_sum_partials", stream);
      hipLaunchKernelGGL(k_sum_partials, dim3((unsigned)ceil_div(M * N, (int64_t)64)), dim3(kThreads),
                         0, stream, M, N, n_chunks, (const float*)part, C, ldc);
      hipError_t e = hipGetLastError();
      tfree(part, stream);
      if (e != hipSuccess) return hip_fail(e, "k_sum_partials", __FILE__, __LINE__);
    }
    if (mask) GCN_CHECK(relu_bwd(M, N, mask, ldm, C, ldc, stream));
    if (relu) GCN_CHECK(relu_fwd(M, N, C, ldc, stream));
    return GCN_OK;
  }
  const dim3 grid((unsigned)ceil_div(M, kTile), (unsigned)ceil_div(N, kTile));
  ProfScope ps(op == GCN_GEMM_NN ? "gemm_nn" : "gemm_nt", stream);
  if (vec && op == GCN_GEMM_NN)
    GCN_HIP(launch_tall<kNN>(M, N, K, A, lda, B, ldb, C, ldc, mask, ldm, relu, stream));
  else if (vec)
    GCN_HIP(launch_tall<kNT>(M, N, K, A, lda, B, ldb, C, ldc, mask, ldm, relu, stream));
  else if (op == GCN_GEMM_NN)
    hipLaunchKernelGGL(k_gemm_tall<kNN>, grid, dim3(kThreads), 0, stream, M, N, K, A, lda, B, ldb,
                       C, ldc);
  else
    hipLaunchKernelGGL(k_gemm_tall<kNT>, grid, dim3(kThreads), 0, stream, M, N, K, A, lda, B, ldb,
                       C, ldc);
  GCN_HIP(hipGetLastError());
  if (mask && !vec) GCN_CHECK(relu_bwd(M, N, mask, ldm, C, ldc, stream));
  if (relu && !vec) GCN_CHECK(relu_fwd(M, N, C, ldc, stream));
  return GCN_OK;
}


// Workgroups of the fused layer-1 backward (chunks x hidden slices): one per
// CU (its registers fill the CU), a fixed count so that the summation order
// does not depend on the device.
constexpr int64_t kBwd1Blocks = 256;

bool layer1_bwd_fusable(int64_t f_in, int64_t hidden, int64_t C, const float* dZ2, int64_t ldc,
                        const float* W2, int64_t ldw) {
  return GCN_LAYER1_FUSED && f_in >= 1 && f_in <= 112 && hidden >= 1 && C >= 1 && C <= 48 &&
         ldc >= C && ldw >= C && aligned16(dZ2, ldc) && aligned16(W2, ldw);
}

gcn_status layer1_bwd_fused(int64_t n, int64_t f_in, int64_t hidden, int64_t C, const float* P,
                            int64_t ldp, const float* H1, int64_t ldh, const float* dZ2,
                            int64_t ldc, const float* W2, int64_t ldw, float* dW1, float* dW2,
                            hipStream_t stream) {
  if (!layer1_bwd_fusable(f_in, hidden, C, dZ2, ldc, W2, ldw)) {
    set_error("fused layer-1 backward: unsupported shape or alignment");
    return GCN_EINVAL;
  }
  const int64_t slices = ceil_div(hidden, (int64_t)32 * kBwd1Waves);
  const int64_t want = std::max<int64_t>(1, kBwd1Blocks / slices);
  const int64_t split = std::max<int64_t>(16, ceil_div(ceil_div(n, want), (int64_t)16) * 16);
  const int64_t chunks = ceil_div(n, split);  // 0 without rows: the sums write zeros
  const int waves = (int)std::min<int64_t>(kBwd1Waves, ceil_div(hidden, (int64_t)32));
  float* part = nullptr;
  GCN_CHECK(talloc(&part, std::max<int64_t>(1, chunks) * (f_in * hidden + hidden * C), stream,
                   "layer-1 partials"));
  Bwd1Args a{n, split, (int)f_in, (int)hidden, (int)C, P, ldp, H1, ldh, dZ2, ldc, W2, ldw,
             part, part + chunks * f_in * hidden};
  {
    ProfScope ps("gemm_layer1_bwd_fused", stream);
    const dim3 grid((unsigned)std::max<int64_t>(1, chunks), (unsigned)slices), block(64 * waves);
    const int mb = f_in <= 32 ? 2 : (f_in <= 64 ? 4 : 7);
    const int cb = (int)ceil_div(C, (int64_t)16);
#define GCN_BWD1(MB_, CB_) \
  if (mb == MB_ && cb == CB_) hipLaunchKernelGGL((k_gcn_bwd1<MB_, CB_>), grid, block, 0, stream, a)
    GCN_BWD1(2, 1); GCN_BWD1(2, 2); GCN_BWD1(2, 3);
    GCN_BWD1(4, 1); GCN_BWD1(4, 2); GCN_BWD1(4, 3);
    GCN_BWD1(7, 1); GCN_BWD1(7, 2); GCN_BWD1(7, 3);
#undef GCN_BWD1
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) {
      tfree(part, stream);
      return hip_fail(e, "k_gcn_bwd1", __FILE__, __LINE__);
    }
  }
  {
    ProfScope ps("gemm_sum_partials", stream);
    hipLaunchKernelGGL(k_sum_partials, dim3((unsigned)ceil_div(f_in * hidden, (int64_t)64)),
                       dim3(kThreads), 0, stream, f_in, hidden, chunks, (const float*)part, dW1,
                       hidden);
    hipLaunchKernelGGL(k_sum_partials, dim3((unsigned)ceil_div(hidden * C, (int64_t)64)),
                       dim3(kThreads), 0, stream, hidden, C, chunks,
                       (const float*)(part + chunks * f_in * hidden), dW2, C);
    hipError_t e = hipGetLastError();
    tfree(part, stream);
    if (e != hipSuccess) return hip_fail(e, "k_sum_partials", __FILE__, __LINE__);
  }
  return GCN_OK;
}

// LDS bytes of the fused forward's weight tables
int64_t fwd1_lds(int64_t f_in, int64_t hidden, int64_t C) {
  const int64_t hbn = ceil_div(hidden, (int64_t)16), sn = ceil_div(f_in, (int64_t)4);
  return (hbn * sn * 64 + hbn * ceil_div(C, (int64_t)16) * 4 * 64) * (int64_t)sizeof(float);
}
constexpr int64_t kMaxDynLds = 160 * 1024;

bool layer1_fwd_fusable(int64_t f_in, int64_t hidden, int64_t C, const float* P, int64_t ldp,
                        const float* H1, int64_t ldh) {
  (void)P;  // read element by element: any alignment
  return GCN_LAYER1_FUSED && f_in >= 1 && f_in <= 112 && hidden >= 1 && C >= 1 && C <= 48 &&
         ldp >= 4 * ceil_div(f_in, (int64_t)4) && ldh >= hidden && aligned16(H1, ldh) &&
         fwd1_lds(f_in, hidden, C) <= kMaxDynLds;
}

gcn_status layer1_fwd_fused(int64_t n, int64_t f_in, int64_t hidden, int64_t C, const float* P,
                            int64_t ldp, const float* W1, int64_t ldw1, const float* W2,
                            int64_t ldw2, float* H1, int64_t ldh, float* Z2, int64_t ldz,
                            hipStream_t stream) {
  if (!layer1_fwd_fusable(f_in, hidden, C, P, ldp, H1, ldh)) {
    set_error("fused layer-1 forward: unsupported shape or alignment");
    return GCN_EINVAL;
  }
  if (n == 0) return GCN_OK;
  ProfScope ps("gemm_layer1_fwd_fused", stream);
  const Fwd1Args a{n, (int)f_in, (int)hidden, (int)C, P, ldp, W1, ldw1, W2, ldw2, H1, ldh, Z2, ldz};
  const int sn = (int)ceil_div(f_in, (int64_t)4);
  const int smax = sn <= 8 ? 8 : (sn <= 16 ? 16 : (sn <= 25 ? 25 : 28));
  const int cb = (int)ceil_div(C, (int64_t)16);
  const size_t lds = (size_t)fwd1_lds(f_in, hidden, C);
  const int64_t groups = ceil_div(n, (int64_t)16);
  hipError_t e = hipSuccess;
  // one workgroup per CU (the weight tables take most of its LDS), wavefronts
  // on their own row groups
  auto launch = [&](auto kern) {
    e = hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize,
                            (int)lds);
    if (e != hipSuccess) return;
    const int64_t wg = std::min<int64_t>(cu_count(), ceil_div(groups, (int64_t)kFwd1Waves));
    hipLaunchKernelGGL(kern, dim3((unsigned)wg), dim3(64 * kFwd1Waves), lds, stream, a);
    e = hipGetLastError();
  };
#define GCN_FWD1(S_, CB_) \
  if (smax == S_ && cb == CB_) launch(k_gcn_fwd1<S_, CB_>)
  GCN_FWD1(8, 1); GCN_FWD1(8, 2); GCN_FWD1(8, 3);
  GCN_FWD1(16, 1); GCN_FWD1(16, 2); GCN_FWD1(16, 3);
  GCN_FWD1(25, 1); GCN_FWD1(25, 2); GCN_FWD1(25, 3);
  GCN_FWD1(28, 1); GCN_FWD1(28, 2); GCN_FWD1(28, 3);
#undef GCN_FWD1
  if (e != hipSuccess) return hip_fail(e, "k_gcn_fwd1", __FILE__, __LINE__);
  return GCN_OK;
}

// LDS bytes of the fused GraphSAGE backward: the weight table and 8 staged
// DG tiles
int64_t tf_bwd_lds(int64_t F, int64_t K) {
  return (F / 16 + kTfWaves) * (K / 4) * 64 * (int64_t)sizeof(float);
}

bool sage_tf_bwd_fusable(int64_t F, int64_t K, const float* dg, int64_t ldg) {
  const int64_t nb = F / 16;
  return GCN_LAYER1_FUSED && F % 16 == 0 &&
         (nb == 1 || nb == 2 || nb == 3 || nb == 4 || nb == 8 || nb == 16) && K >= 4 &&
         K % 4 == 0 && ldg >= K && aligned16(dg, ldg) && tf_bwd_lds(F, K) <= kMaxDynLds;
}

gcn_status sage_tf_bwd_fused(int64_t n, int64_t F, int64_t K, const float* dg, int64_t ldg,
                             const float* bw, int64_t ldb, const float* y, int64_t ldy,
                             const float* rstd, float* dx, int64_t ldx, hipStream_t stream) {
  if (!sage_tf_bwd_fusable(F, K, dg, ldg)) {
    set_error("fused GraphSAGE backward: unsupported shape or alignment");
    return GCN_EINVAL;
  }
  if (n == 0) return GCN_OK;
  ProfScope ps("gemm_sage_tf_bwd_fused", stream);
  const TfBwdArgs a{n, (int)F, (int)K, dg, ldg, bw, ldb, y, ldy, rstd, dx, ldx};
  const size_t lds = (size_t)tf_bwd_lds(F, K);
  const int64_t wg = std::min<int64_t>(cu_count(), ceil_div(ceil_div(n, (int64_t)16), (int64_t)kTfWaves));
  hipError_t e = hipSuccess;
  auto launch = [&](auto kern) {
    e = hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize,
                            (int)lds);
    if (e != hipSuccess) return;
    hipLaunchKernelGGL(kern, dim3((unsigned)wg), dim3(64 * kTfWaves), lds, stream, a);
    e = hipGetLastError();
  };
  switch (F / 16) {
    case 1: launch(k_sage_tf_bwd<1>); break;
    case 2: launch(k_sage_tf_bwd<2>); break;
    case 3: launch(k_sage_tf_bwd<3>); break;
    case 4: launch(k_sage_tf_bwd<4>); break;
    case 8: launch(k_sage_tf_bwd<8>); break;
    default: launch(k_sage_tf_bwd<16>); break;
  }
  if (e != hipSuccess) return hip_fail(e, "k_sage_tf_bwd", __FILE__, __LINE__);
  return GCN_OK;
}

gcn_status relu_fwd(int64_t n, int64_t F, float* H, int64_t ld, hipStream_t stream) {
  if (n * F == 0) return GCN_OK;
  ProfScope ps("relu", stream);
  hipLaunchKernelGGL(k_relu, dim3((unsigned)ceil_div(n, kThreads / 64)), dim3(kThreads), 0, stream,
                     n, F, H, ld);
  GCN_HIP(hipGetLastError());
  return GCN_OK;
}

gcn_status relu_bwd(int64_t n, int64_t F, const float* H, int64_t ldh, float* dH, int64_t ld,
                    hipStream_t stream) {
  if (n * F == 0) return GCN_OK;
  ProfScope ps("relu_bwd", stream);
  hipLaunchKernelGGL(k_relu_bwd, dim3((unsigned)ceil_div(n, kThreads / 64)), dim3(kThreads), 0,
                     stream, n, F, H, ldh, dH, ld);
  GCN_HIP(hipGetLastError());
  return GCN_OK;
}

gcn_status softmax_xent(int64_t n, int C, const float* z, int64_t ldz, const int32_t* y,
                        float* dz, int64_t ldd, double* loss, hipStream_t stream,
                        const uint8_t* skip) {
  const int64_t nb = std::max<int64_t>(1, ceil_div(n, (kThreads / 64) * kSoftmaxRowsPerWave));
  double* bl = nullptr;
  unsigned long long* cnt = nullptr;
  GCN_CHECK(talloc(&bl, nb, stream, "block losses"));
  hipError_t e = hipSuccess;
  if (skip) {
    gcn_status st = talloc(&cnt, 1, stream, "loss row count");
    if (st != GCN_OK) {
      tfree(bl, stream);
      return st;
    }
    // a kernel, not a memset node, clears the counter (safe under stream capture)
    hipLaunchKernelGGL(k_zero_count, dim3(1), dim3(64), 0, stream, cnt);
    e = hipGetLastError();
    if (e == hipSuccess) {
      hipLaunchKernelGGL(k_count_kept, dim3((unsigned)std::max<int64_t>(1, ceil_div(n, kThreads))),
                         dim3(kThreads), 0, stream, n, skip, cnt);
      e = hipGetLastError();
    }
  }
  if (e == hipSuccess) {
    ProfScope ps("softmax_xent", stream);
    const dim3 grid((unsigned)nb);
    const unsigned long long* kept = cnt;
    if (C <= 16)
      hipLaunchKernelGGL(k_softmax_xent<1>, grid, dim3(kThreads), 0, stream, n, C, z, ldz, y, dz,
                         ldd, bl, skip, kept);
    else if (C <= 32)
      hipLaunchKernelGGL(k_softmax_xent<2>, grid, dim3(kThreads), 0, stream, n, C, z, ldz, y, dz,
                         ldd, bl, skip, kept);
    else if (C <= 48)
      hipLaunchKernelGGL(k_softmax_xent<3>, grid, dim3(kThreads), 0, stream, n, C, z, ldz, y, dz,
                         ldd, bl, skip, kept);
    else
      hipLaunchKernelGGL(k_softmax_xent<4>, grid, dim3(kThreads), 0, stream, n, C, z, ldz, y, dz,
                         ldd, bl, skip, kept);
    e = hipGetLastError();
  }
  if (e == hipSuccess) {
    ProfScope ps("loss_total", stream);
    hipLaunchKernelGGL(k_loss_total, dim3(1), dim3(kThreads), 0, stream, nb, n, (const double*)bl,
                       loss, (const unsigned long long*)cnt);
    e = hipGetLastError();
  }
  tfree(cnt, stream);
  tfree(bl, stream);
  if (e != hipSuccess) return hip_fail(e, "softmax_xent", __FILE__, __LINE__);
  return GCN_OK;
}

}  // namespace gcn

using namespace gcn;

extern "C" gcn_status gcn_gemm_f32(int op, int64_t M, int64_t N, int64_t K, const float* A,
                                   int64_t lda, const float* B, int64_t ldb, float* C, int64_t ldc,
                                   void* stream) {
  clear_error();
  if (op != GCN_GEMM_NN && op != GCN_GEMM_NT && op != GCN_GEMM_TN) {
    set_error("unknown GEMM op %d", op);
    return GCN_EINVAL;
  }
  if (M < 0 || N < 0 || K < 0 || (M > 0 && N > 0 && (!A || !B || !C)) || ldc < N) {
    set_error("invalid GEMM sizes or pointers");
    return GCN_EINVAL;
  }
  const int64_t a_cols = op == GCN_GEMM_TN ? M : K;
  const int64_t b_cols = op == GCN_GEMM_NT ? K : N;
  if (lda < a_cols || ldb < b_cols) {
    set_error("leading dimensions too small (lda=%lld ldb=%lld)", (long long)lda, (long long)ldb);
    return GCN_EINVAL;
  }
  if (op == GCN_GEMM_TN && (M * N >= (1ll << 31))) {
    set_error("A^T B output too large");
    return GCN_ERANGE;
  }
  return gemm_f32(op, M, N, K, A, lda, B, ldb, C, ldc, (hipStream_t)stream);
}

extern "C" gcn_status gcn_relu(int64_t n, int64_t F, float* H, int64_t ld, void* stream) {
  clear_error();
  if (n < 0 || F < 0 || (n * F > 0 && !H) || ld < F) {
    set_error("invalid ReLU arguments");
    return GCN_EINVAL;
  }
  return relu_fwd(n, F, H, ld, (hipStream_t)stream);
}

extern "C" gcn_status gcn_relu_bwd(int64_t n, int64_t F, const float* H, int64_t ldh, float* dH,
                                   int64_t ld, void* stream) {
  clear_error();
  if (n < 0 || F < 0 || (n * F > 0 && (!H || !dH)) || ldh < F || ld < F) {
    set_error("invalid ReLU backward arguments");
    return GCN_EINVAL;
  }
  return relu_bwd(n, F, H, ldh, dH, ld, (hipStream_t)stream);
}

extern "C" gcn_status gcn_softmax_xent(int64_t n, int64_t C, const float* logits, int64_t ld,
                                       const int32_t* labels, float* dlogits, int64_t ldd,
                                       double* loss, void* stream) {
  clear_error();
  if (n <= 0 || C <= 0 || C > 64 || !logits || !labels || !dlogits || !loss || ld < C ||
      ldd < C) {
    set_error("invalid softmax cross-entropy arguments (1 <= C <= 64)");
    return GCN_EINVAL;
  }
  return softmax_xent(n, (int)C, logits, ld, labels, dlogits, ldd, loss, (hipStream_t)stream);
}
