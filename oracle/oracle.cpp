// CPU ORACLE for the GCN aggregation path -- TEST INFRASTRUCTURE ONLY.
//
// Plain, slow, obviously correct reference used by the test suite, by the
// GPU smoke check and by the benchmark's CPU-baseline leg. The GPU library
// never links, loads or calls this file, and this file shares no code with
// the GPU library.
//
// What it computes (SuperGCN, Chen et al., arXiv 2411.16025):
//  * structure   -- Section 4, "clustering and sorting": the index array is
//                   sorted and the source rows feeding one destination row
//                   are grouped together. Written as its plain definition:
//                   collect (row, col) pairs, std::sort, std::unique, count
//                   rows. Edge s->d is the entry (row d, col s): rows of
//                   `src` are added into `dst` (Index_add, Section 4).
//  * normalize   -- GCN propagation matrix D~^-1/2 (A+I) D~^-1/2 (Section
//                   2.1 cites GCN; Lemma 2 writes the layer as A H W). The
//                   degree d~ = deg + 1 counts the single self-loop.
//  * spmm        -- Section 4: Index_add / SpMM, Y[r,:] = sum_k val[k] *
//                   X[col[k],:], accumulated in double in CSR order.
//  * quantize / dequantize -- Section 2.4: Z = min(h), S = (max-min)/(2^b-1),
//                   q = round((h-Z)/S), h' = q*S + Z, with b = 8 per row.
//                   Round-to-nearest-even replaces the stochastic rounding
//                   (Section 7.3 removes the random number generation);
//                   dequantization is a single fused multiply-add.
//  * spmm_q8     -- the one-GPU share of Section 6.1 step 3: halo columns
//                   (col >= n_local_cols) are dequantized on read.
//
// Every floating-point result is accumulated in double; the only roundings
// are those the definitions above fix (fp32 val, fp32 dequantized value).

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstring>
#include <utility>
#include <vector>

#include <omp.h>
#include <parallel/algorithm>

namespace {

constexpr uint32_t kSymmetrize = 1u;
constexpr uint32_t kAddSelfLoops = 2u;

// Visit every (row, col) entry the edge list defines before sorting and
// deduplication: edge e gives (dst[e], src[e]); with SYMMETRIZE also
// (src[e], dst[e]); with ADD_SELF_LOOPS drawn self pairs are dropped (the
// self-loops are added separately, one per node). Returns false if an id is
// out of range.
template <class Fn>
bool for_each_edge_pair(int64_t n_rows, int64_t n_cols, int64_t e_begin, int64_t e_end,
                        const int32_t* src, const int32_t* dst, uint32_t flags, Fn&& fn) {
  bool ok = true;
  for (int64_t e = e_begin; e < e_end; ++e) {
    const int64_t s = src[e], d = dst[e];
    if (s < 0 || s >= n_cols || d < 0 || d >= n_rows) {
      ok = false;
      continue;
    }
    if ((flags & kAddSelfLoops) && s == d) continue;
    fn(d, s);
    if (flags & kSymmetrize) fn(s, d);
  }
  return ok;
}

inline uint64_t pack(int64_t major, int64_t minor) {
  return ((uint64_t)major << 32) | (uint64_t)(uint32_t)minor;
}

void sort_keys(std::vector<uint64_t>& keys) {
  if (keys.size() > (1u << 20))
    __gnu_parallel::sort(keys.begin(), keys.end());
  else
    std::sort(keys.begin(), keys.end());
}

}  // namespace

extern "C" {

// Sorted, deduplicated structure of A (transpose == 0: CSR, rows = dst) or
// of A^T (transpose == 1: CSC, rows = src ids). ptr has n_major + 1 entries
// (n_major = n_rows, or n_cols when transposed); idx receives at most cap
// entries. Returns nnz, -1 if cap is too small, -2 for an id out of range,
// -3 for SYMMETRIZE on a rectangular shape.
int64_t orc_structure(int64_t n_rows, int64_t n_cols, int64_t n_edges, const int32_t* src,
                      const int32_t* dst, uint32_t flags, int transpose, int64_t cap,
                      int64_t* ptr, int32_t* idx) {
  if ((flags & kSymmetrize) && n_rows != n_cols) return -3;
  std::vector<uint64_t> keys;
  keys.reserve((size_t)(n_edges * ((flags & kSymmetrize) ? 2 : 1) +
                        std::min(n_rows, n_cols)));
  bool ok = for_each_edge_pair(n_rows, n_cols, 0, n_edges, src, dst, flags,
                               [&](int64_t r, int64_t c) {
                                 keys.push_back(transpose ? pack(c, r) : pack(r, c));
                               });
  if (!ok) return -2;
  if (flags & kAddSelfLoops)
    for (int64_t i = 0; i < std::min(n_rows, n_cols); ++i) keys.push_back(pack(i, i));
  sort_keys(keys);
  keys.erase(std::unique(keys.begin(), keys.end()), keys.end());
  const int64_t nnz = (int64_t)keys.size();
  if (nnz > cap) return -1;
  const int64_t n_major = transpose ? n_cols : n_rows;
  std::fill(ptr, ptr + n_major + 1, 0);
  for (int64_t k = 0; k < nnz; ++k) {
    ptr[(keys[k] >> 32) + 1] += 1;
    idx[k] = (int32_t)(keys[k] & 0xFFFFFFFFu);
  }
  for (int64_t i = 0; i < n_major; ++i) ptr[i + 1] += ptr[i];
  return nnz;
}

// Structure of selected major indices only (rows of A, or rows of A^T when
// transposed), computed straight from the edge list without building the
// whole matrix. sel must hold distinct ids. out_ptr has n_sel + 1 entries;
// out_idx at most cap entries. Returns the entry count, -1 if cap is too
// small, -2 for an id out of range, -3 for SYMMETRIZE on a rectangular
// shape, -4 for a repeated selection.
int64_t orc_rows_of(int64_t n_rows, int64_t n_cols, int64_t n_edges, const int32_t* src,
                    const int32_t* dst, uint32_t flags, int transpose, int64_t n_sel,
                    const int32_t* sel, int64_t cap, int64_t* out_ptr, int32_t* out_idx) {
  if ((flags & kSymmetrize) && n_rows != n_cols) return -3;
  const int64_t n_major = transpose ? n_cols : n_rows;
  std::vector<int32_t> slot((size_t)n_major, -1);
  for (int64_t i = 0; i < n_sel; ++i) {
    if (sel[i] < 0 || sel[i] >= n_major) return -2;
    if (slot[sel[i]] >= 0) return -4;
    slot[sel[i]] = (int32_t)i;
  }
  const int nt = omp_get_max_threads();
  std::vector<std::vector<uint64_t>> found((size_t)nt);
  bool ok_all = true;
#pragma omp parallel num_threads(nt) reduction(&& : ok_all)
  {
    const int t = omp_get_thread_num();
    const int64_t lo = n_edges * t / nt, hi = n_edges * (t + 1) / nt;
    auto& mine = found[(size_t)t];
    ok_all = for_each_edge_pair(n_rows, n_cols, lo, hi, src, dst, flags,
                                [&](int64_t r, int64_t c) {
                                  const int64_t major = transpose ? c : r;
                                  const int64_t minor = transpose ? r : c;
                                  const int32_t s = slot[(size_t)major];
                                  if (s >= 0) mine.push_back(pack(s, minor));
                                });
  }
  if (!ok_all) return -2;
  std::vector<uint64_t> keys;
  for (auto& v : found) keys.insert(keys.end(), v.begin(), v.end());
  if (flags & kAddSelfLoops)
    for (int64_t i = 0; i < n_sel; ++i)
      if (sel[i] < std::min(n_rows, n_cols)) keys.push_back(pack(i, sel[i]));
  sort_keys(keys);
  keys.erase(std::unique(keys.begin(), keys.end()), keys.end());
  const int64_t total = (int64_t)keys.size();
  if (total > cap) return -1;
  std::fill(out_ptr, out_ptr + n_sel + 1, 0);
  for (int64_t k = 0; k < total; ++k) {
    out_ptr[(keys[k] >> 32) + 1] += 1;
    out_idx[k] = (int32_t)(keys[k] & 0xFFFFFFFFu);
  }
  for (int64_t i = 0; i < n_sel; ++i) out_ptr[i + 1] += out_ptr[i];
  return total;
}

// deg[r] = number of entries of row r whose column differs from r (the
// degree without the self-loop).
void orc_row_degrees(int64_t n_major, const int64_t* ptr, const int32_t* idx, int32_t* deg) {
  for (int64_t r = 0; r < n_major; ++r) {
    int32_t d = 0;
    for (int64_t k = ptr[r]; k < ptr[r + 1]; ++k) d += (idx[k] != r);
    deg[r] = d;
  }
}

// val of entry (r, c) = 1 / sqrt(d~_r * d~_c), d~ = deg + 1, computed in
// double and rounded once to fp32. deg is indexed by node id in both roles.
void orc_normalize(int64_t n_major, const int64_t* ptr, const int32_t* idx, const int32_t* deg,
                   float* val) {
#pragma omp parallel for schedule(dynamic, 1024)
  for (int64_t r = 0; r < n_major; ++r)
    for (int64_t k = ptr[r]; k < ptr[r + 1]; ++k) {
      const double dr = (double)deg[r] + 1.0;
      const double dc = (double)deg[idx[k]] + 1.0;
      val[k] = (float)(1.0 / std::sqrt(dr * dc));
    }
}

// The same formula entry by entry, for rows held out of their natural
// position (sampled rows): deg_rows[i] is the degree of the i-th listed row,
// deg_cols[k] the degree of the column of entry k.
void orc_normalize_listed(int64_t n_sel, const int64_t* ptr, const int32_t* deg_rows,
                          const int32_t* deg_cols, float* val) {
  for (int64_t i = 0; i < n_sel; ++i)
    for (int64_t k = ptr[i]; k < ptr[i + 1]; ++k) {
      const double dr = (double)deg_rows[i] + 1.0;
      const double dc = (double)deg_cols[k] + 1.0;
      val[k] = (float)(1.0 / std::sqrt(dr * dc));
    }
}

// Y[r, f] = sum_k val[k] * X[idx[k], f] in double, in stored order.
// S[r, f] = sum_k |val[k] * X[idx[k], f]| (the scale for tolerances).
// Y and S are n_major x F with row stride F; S may be null.
void orc_spmm(int64_t n_major, const int64_t* ptr, const int32_t* idx, const float* val,
              const float* X, int64_t ldx, int64_t F, double* Y, double* S) {
#pragma omp parallel for schedule(dynamic, 256)
  for (int64_t r = 0; r < n_major; ++r)
    for (int64_t f = 0; f < F; ++f) {
      double acc = 0.0, mag = 0.0;
      for (int64_t k = ptr[r]; k < ptr[r + 1]; ++k) {
        const double t = (double)val[k] * (double)X[(int64_t)idx[k] * ldx + f];
        acc += t;
        mag += std::fabs(t);
      }
      Y[r * F + f] = acc;
      if (S) S[r * F + f] = mag;
    }
}

// Y = A H for a float64 H (the training step keeps every intermediate in
// double): Y[r, f] = sum_k val[k] * H[idx[k], f] in stored order.
void orc_spmm_f64(int64_t n_major, const int64_t* ptr, const int32_t* idx, const float* val,
                  const double* H, int64_t ldh, int64_t F, double* Y) {
#pragma omp parallel for schedule(dynamic, 256)
  for (int64_t r = 0; r < n_major; ++r) {
    double* y = Y + r * F;
    for (int64_t f = 0; f < F; ++f) y[f] = 0.0;
    for (int64_t k = ptr[r]; k < ptr[r + 1]; ++k) {
      const double w = (double)val[k];
      const double* h = H + (int64_t)idx[k] * ldh;
      for (int64_t f = 0; f < F; ++f) y[f] += w * h[f];
    }
  }
}

// Dequantized value of one code: fmaf(q, S, Z), a single rounding.
float orc_dequant(uint8_t q, float scale, float zero) { return std::fmaf((float)q, scale, zero); }

// Dequantize an n x F code matrix row by row: out[i, f] = fmaf(Q[i, f],
// scale[i], zmin[i]).
void orc_dequant_rows(int64_t n, int64_t F, const uint8_t* Q, int64_t ldq, const float* zmin,
                      const float* scale, float* out, int64_t ldo) {
  for (int64_t i = 0; i < n; ++i)
    for (int64_t f = 0; f < F; ++f) out[i * ldo + f] = orc_dequant(Q[i * ldq + f], scale[i], zmin[i]);
}

// As orc_spmm, with columns >= n_local_cols read from uint8 codes:
// x = fmaf((float)Q[j - n_local_cols, f], scale[j - nlc], zmin[j - nlc]).
void orc_spmm_q8(int64_t n_major, const int64_t* ptr, const int32_t* idx, const float* val,
                 int64_t n_local_cols, const float* X, int64_t ldx, const uint8_t* Q, int64_t ldq,
                 const float* zmin, const float* scale, int64_t F, double* Y, double* S) {
#pragma omp parallel for schedule(dynamic, 256)
  for (int64_t r = 0; r < n_major; ++r)
    for (int64_t f = 0; f < F; ++f) {
      double acc = 0.0, mag = 0.0;
      for (int64_t k = ptr[r]; k < ptr[r + 1]; ++k) {
        const int64_t j = idx[k];
        float x;
        if (j < n_local_cols) {
          x = X[j * ldx + f];
        } else {
          const int64_t h = j - n_local_cols;
          x = orc_dequant(Q[h * ldq + f], scale[h], zmin[h]);
        }
        const double t = (double)val[k] * (double)x;
        acc += t;
        mag += std::fabs(t);
      }
      Y[r * F + f] = acc;
      if (S) S[r * F + f] = mag;
    }
}

// Per-row uint8 quantization: Z = min, S = (max - min) / 255 (fp32),
// q = clamp(nearbyint((x - Z) / S), 0, 255); all codes 0 when S == 0.
void orc_quantize_rows(int64_t n, int64_t F, const float* X, int64_t ldx, uint8_t* Q, int64_t ldq,
                       float* zmin, float* scale) {
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < n; ++i) {
    const float* x = X + i * ldx;
    float mn = x[0], mx = x[0];
    for (int64_t f = 1; f < F; ++f) {
      mn = std::min(mn, x[f]);
      mx = std::max(mx, x[f]);
    }
    const float s = (mx - mn) / 255.0f;
    zmin[i] = mn;
    scale[i] = s;
    for (int64_t f = 0; f < F; ++f) {
      float q = 0.0f;
      if (s != 0.0f) q = std::nearbyint((x[f] - mn) / s);
      q = std::min(255.0f, std::max(0.0f, q));
      Q[i * ldq + f] = (uint8_t)q;
    }
  }
}

// LayerNorm of each row over its F features (Section 6.1, step 2: applied to
// the embedding table before quantization to remove outliers):
// y = (x - mean) / sqrt(var + eps) * gamma + beta with the biased variance,
// all in double, rounded once to fp32. gamma/beta may be null (1 and 0).
void orc_layernorm_rows(int64_t n, int64_t F, const float* X, int64_t ldx, const float* gamma,
                        const float* beta, double eps, float* Y, int64_t ldy) {
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < n; ++i) {
    const float* x = X + i * ldx;
    double mean = 0.0;
    for (int64_t f = 0; f < F; ++f) mean += (double)x[f];
    mean /= (double)F;
    double var = 0.0;
    for (int64_t f = 0; f < F; ++f) var += ((double)x[f] - mean) * ((double)x[f] - mean);
    var /= (double)F;
    const double inv = 1.0 / std::sqrt(var + eps);
    for (int64_t f = 0; f < F; ++f) {
      const double g = gamma ? (double)gamma[f] : 1.0;
      const double b = beta ? (double)beta[f] : 0.0;
      Y[i * ldy + f] = (float)(((double)x[f] - mean) * inv * g + b);
    }
  }
}

// b-bit per-row quantization (Section 2.4), b = 8 or 2:
// Z = min, S = (max - min) / (2^b - 1), q = clamp(nearbyint((x - Z) / S), 0, 2^b - 1)
// in fp32; codes 0 when S == 0. 8-bit codes are bytes; 2-bit codes are packed
// four per byte, feature f of a row in bits [2 (f % 4), 2 (f % 4) + 2) of byte
// f / 4 (pad codes 0). Params at zmin[i * ldp], scale[i * ldp].
void orc_quantize_rows_bits(int64_t n, int64_t F, int bits, const float* X, int64_t ldx,
                            uint8_t* Q, int64_t ldq, float* zmin, float* scale, int64_t ldp) {
  const float levels = (float)((1 << bits) - 1);
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < n; ++i) {
    const float* x = X + i * ldx;
    float mn = x[0], mx = x[0];
    for (int64_t f = 1; f < F; ++f) {
      mn = std::min(mn, x[f]);
      mx = std::max(mx, x[f]);
    }
    const float s = (mx - mn) / levels;
    zmin[i * ldp] = mn;
    scale[i * ldp] = s;
    uint8_t* q = Q + i * ldq;
    if (bits == 2)
      for (int64_t k = 0; k < (F + 3) / 4; ++k) q[k] = 0;
    for (int64_t f = 0; f < F; ++f) {
      float c = 0.0f;
      if (s != 0.0f) c = std::nearbyint((x[f] - mn) / s);
      c = std::min(levels, std::max(0.0f, c));
      if (bits == 8)
        q[f] = (uint8_t)c;
      else
        q[f / 4] |= (uint8_t)((uint32_t)c << (2 * (f % 4)));
    }
  }
}

// Code of feature f of a b-bit row.
static inline uint32_t code_of(const uint8_t* row, int64_t f, int bits) {
  return bits == 8 ? row[f] : (row[f / 4] >> (2 * (f % 4))) & 3u;
}

// Dequantize b-bit rows: out[i, f] = fmaf(q, scale[i * ldp], zmin[i * ldp]).
void orc_dequant_rows_bits(int64_t n, int64_t F, int bits, const uint8_t* Q, int64_t ldq,
                           const float* zmin, const float* scale, int64_t ldp, float* out,
                           int64_t ldo) {
  for (int64_t i = 0; i < n; ++i)
    for (int64_t f = 0; f < F; ++f)
      out[i * ldo + f] =
          std::fmaf((float)code_of(Q + i * ldq, f, bits), scale[i * ldp], zmin[i * ldp]);
}

// orc_spmm_q8 for b-bit halo codes.
void orc_spmm_qbits(int64_t n_major, const int64_t* ptr, const int32_t* idx, const float* val,
                    int64_t n_local_cols, const float* X, int64_t ldx, int bits, const uint8_t* Q,
                    int64_t ldq, const float* zmin, const float* scale, int64_t ldp, int64_t F,
                    double* Y, double* S) {
#pragma omp parallel for schedule(dynamic, 256)
  for (int64_t r = 0; r < n_major; ++r)
    for (int64_t f = 0; f < F; ++f) {
      double acc = 0.0, mag = 0.0;
      for (int64_t k = ptr[r]; k < ptr[r + 1]; ++k) {
        const int64_t j = idx[k];
        float x;
        if (j < n_local_cols) {
          x = X[j * ldx + f];
        } else {
          const int64_t h = j - n_local_cols;
          x = std::fmaf((float)code_of(Q + h * ldq, f, bits), scale[h * ldp], zmin[h * ldp]);
        }
        const double t = (double)val[k] * (double)x;
        acc += t;
        mag += std::fabs(t);
      }
      Y[r * F + f] = acc;
      if (S) S[r * F + f] = mag;
    }
}

// Minimum vertex cover of a bipartite graph (Section 5.3): a maximum matching
// by augmenting paths (Kuhn's method: for each left vertex, search an
// alternating path to a free right vertex), then Koenig's construction: Z =
// vertices reachable from free left vertices along alternating paths (left to
// right on any edge, right to left on matched edges); the cover is
// (left not in Z) plus (right in Z). Edge e joins left eu[e] and right ev[e].
// Returns the matching size, which equals the cover size.
int64_t orc_bipartite_cover(int64_t n_u, int64_t n_v, int64_t n_edges, const int32_t* eu,
                            const int32_t* ev, uint8_t* cover_u, uint8_t* cover_v) {
  std::vector<int64_t> off((size_t)n_u + 1, 0);
  for (int64_t e = 0; e < n_edges; ++e) off[eu[e] + 1] += 1;
  for (int64_t u = 0; u < n_u; ++u) off[u + 1] += off[u];
  std::vector<int32_t> adj((size_t)n_edges);
  std::vector<int64_t> pos(off.begin(), off.end() - 1);
  for (int64_t e = 0; e < n_edges; ++e) adj[pos[eu[e]]++] = ev[e];
  std::vector<int32_t> match_u((size_t)n_u, -1), match_v((size_t)n_v, -1);
  std::vector<int64_t> seen((size_t)n_v, -1);
  std::vector<int32_t> stack_u, stack_v;
  std::vector<int64_t> stack_k;
  int64_t size = 0;
  for (int64_t root = 0; root < n_u; ++root) {
    // depth-first search for an augmenting path from root (explicit stack)
    stack_u.assign(1, (int32_t)root);
    stack_k.assign(1, off[root]);
    stack_v.clear();
    bool found = false;
    while (!stack_u.empty() && !found) {
      const int32_t u = stack_u.back();
      int64_t& k = stack_k.back();
      if (k == off[u + 1]) {
        stack_u.pop_back();
        stack_k.pop_back();
        if (!stack_v.empty()) stack_v.pop_back();
        continue;
      }
      const int32_t v = adj[k++];
      if (seen[v] == root) continue;
      seen[v] = root;
      if (match_v[v] < 0) {
        // augment along the stack: u_0 v_0 u_1 v_1 ... u_last v
        stack_v.push_back(v);
        for (size_t i = 0; i < stack_u.size(); ++i) {
          match_u[stack_u[i]] = stack_v[i];
          match_v[stack_v[i]] = stack_u[i];
        }
        found = true;
      } else {
        stack_v.push_back(v);
        stack_u.push_back(match_v[v]);
        stack_k.push_back(off[match_v[v]]);
      }
    }
    size += found;
  }
  // Koenig: alternating reachability from free left vertices
  std::vector<uint8_t> zu((size_t)n_u, 0), zv((size_t)n_v, 0);
  std::vector<int32_t> queue;
  for (int64_t u = 0; u < n_u; ++u)
    if (match_u[u] < 0) {
      zu[u] = 1;
      queue.push_back((int32_t)u);
    }
  for (size_t qi = 0; qi < queue.size(); ++qi) {
    const int32_t u = queue[qi];
    for (int64_t k = off[u]; k < off[u + 1]; ++k) {
      const int32_t v = adj[k];
      if (zv[v]) continue;
      zv[v] = 1;
      const int32_t w = match_v[v];
      if (w >= 0 && !zu[w]) {
        zu[w] = 1;
        queue.push_back(w);
      }
    }
  }
  for (int64_t u = 0; u < n_u; ++u) cover_u[u] = !zu[u];
  for (int64_t v = 0; v < n_v; ++v) cover_v[v] = zv[v];
  return size;
}

int orc_num_threads(void) { return omp_get_max_threads(); }

// Threads used by later parallel regions (n >= 1); timing only, no arithmetic.
void orc_set_num_threads(int n) { omp_set_num_threads(n < 1 ? 1 : n); }

}  // extern "C"
