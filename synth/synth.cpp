// Seeded synthetic inputs shared by the aggregation library's tests, its
// benchmark and the CPU oracle's tests.
//
// This file holds random-number generation and graph/feature synthesis only.
// It contains none of the aggregation method's arithmetic: no CSR build, no
// degree normalization, no aggregation and no quantization.
//
// Random numbers come from SplitMix64 used as a counter-based generator:
// element i of stream `seed` is mix(seed + (i + 1) * GAMMA), which is exactly
// the i-th output of the SplitMix64 sequence started at state `seed`
// (Steele, Lea and Flood, "Fast splittable pseudorandom number generators",
// OOPSLA 2014). Every output depends only on (seed, counter), so the results
// do not depend on the number of threads.

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstring>
#include <utility>
#include <vector>

#include <omp.h>

namespace {

constexpr uint64_t kGamma = 0x9E3779B97F4A7C15ULL;

inline uint64_t mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
  return z ^ (z >> 31);
}

// i-th output of the SplitMix64 sequence seeded with `seed`.
inline uint64_t sm64(uint64_t seed, uint64_t i) { return mix64(seed + (i + 1) * kGamma); }

// Unbiased-enough bounded integer in [0, n) from 64 random bits (Lemire's
// multiply-high reduction; the bias is below 2^-32 for n < 2^32).
inline uint64_t bounded(uint64_t h, uint64_t n) {
  return (uint64_t)(((unsigned __int128)h * n) >> 64);
}

// RMAT quadrant thresholds on 32-bit uniforms.
struct RmatThresholds {
  uint64_t a, ab, abc;
};

inline RmatThresholds thresholds(double a, double b, double c) {
  const double two32 = 4294967296.0;
  return {(uint64_t)(a * two32), (uint64_t)((a + b) * two32), (uint64_t)((a + b + c) * two32)};
}

// One RMAT vertex pair over [0, 2^scale)^2. Level l (most significant first)
// consumes 32 random bits; quadrant a -> (0,0), b -> (0,1), c -> (1,0),
// d -> (1,1), where the first coordinate is u and the second v.
inline void rmat_pair(uint64_t seed, uint64_t counter_base, int scale, const RmatThresholds& t,
                      uint64_t* u_out, uint64_t* v_out) {
  uint64_t u = 0, v = 0;
  uint64_t word = 0;
  for (int l = 0; l < scale; ++l) {
    if ((l & 1) == 0) word = sm64(seed, counter_base + (uint64_t)(l >> 1));
    const uint64_t r = (l & 1) ? (word >> 32) : (word & 0xFFFFFFFFULL);
    uint64_t bu, bv;
    if (r < t.a) {
      bu = 0; bv = 0;
    } else if (r < t.ab) {
      bu = 0; bv = 1;
    } else if (r < t.abc) {
      bu = 1; bv = 0;
    } else {
      bu = 1; bv = 1;
    }
    u = (u << 1) | bu;
    v = (v << 1) | bv;
  }
  *u_out = u;
  *v_out = v;
}

// Counter layout for RMAT draws: draw d, attempt t, word w.
inline uint64_t rmat_counter(uint64_t d, uint64_t t) { return (d << 24) | (t << 5); }

// Draw number d of an RMAT stream over [0, n) by rejection from [0, 2^scale).
inline void rmat_draw(uint64_t seed, uint64_t d, int scale, uint64_t n, const RmatThresholds& th,
                      uint64_t* u, uint64_t* v) {
  for (uint64_t t = 0;; ++t) {
    rmat_pair(seed, rmat_counter(d, t & 0x7FFFF), scale, th, u, v);
    if (*u < n && *v < n) return;
  }
}

int scale_for(uint64_t n) {
  int s = 0;
  while ((1ULL << s) < n) ++s;
  return s;
}

}  // namespace

extern "C" {

// Raw SplitMix64 outputs: out[i] = element (first + i) of stream `seed`.
void synth_splitmix64(uint64_t seed, uint64_t first, int64_t count, uint64_t* out) {
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < count; ++i) out[i] = sm64(seed, first + (uint64_t)i);
}

// Seeded permutation of [0, n) by Fisher-Yates (Knuth, TAOCP vol. 2,
// Algorithm P), step i drawing its swap partner from element i of the stream.
void synth_permutation(uint64_t seed, int64_t n, int32_t* perm) {
  for (int64_t i = 0; i < n; ++i) perm[i] = (int32_t)i;
  for (int64_t i = n - 1; i > 0; --i) {
    const int64_t j = (int64_t)bounded(sm64(seed, (uint64_t)i), (uint64_t)(i + 1));
    const int32_t tmp = perm[i];
    perm[i] = perm[j];
    perm[j] = tmp;
  }
}

// Erdos-Renyi style edge list: `m` ordered pairs drawn uniformly from
// [0, n)^2. Pair e uses element e of the stream: low 32 bits -> src,
// high 32 bits -> dst.
void synth_er_edges(uint64_t seed, int64_t n, int64_t m, int32_t* src, int32_t* dst) {
#pragma omp parallel for schedule(static)
  for (int64_t e = 0; e < m; ++e) {
    const uint64_t h = sm64(seed, (uint64_t)e);
    src[e] = (int32_t)(((h & 0xFFFFFFFFULL) * (uint64_t)n) >> 32);
    dst[e] = (int32_t)(((h >> 32) * (uint64_t)n) >> 32);
  }
}

// RMAT edge list (Chakrabarti, Zhan and Faloutsos, SDM 2004): `m` draws over
// [0, n) with quadrant probabilities a, b, c (d = 1 - a - b - c), by
// rejection from the next power of two. If perm is non-null, both endpoints
// are relabelled through it (perm must be a permutation of [0, n)).
// Draw e yields (u, v) -> src[e] = v, dst[e] = u.
void synth_rmat_edges(uint64_t seed, int64_t n, int64_t m, double a, double b, double c,
                      const int32_t* perm, int32_t* src, int32_t* dst) {
  const int scale = scale_for((uint64_t)n);
  const RmatThresholds th = thresholds(a, b, c);
#pragma omp parallel for schedule(static, 4096)
  for (int64_t e = 0; e < m; ++e) {
    uint64_t u, v;
    rmat_draw(seed, (uint64_t)e, scale, (uint64_t)n, th, &u, &v);
    int32_t su = (int32_t)u, sv = (int32_t)v;
    if (perm) {
      su = perm[su];
      sv = perm[sv];
    }
    src[e] = sv;
    dst[e] = su;
  }
}

// Marks the first draw of every unordered pair: first[e] = 1 when the pair
// {a[e], b[e]} (a[e] != b[e], ids in [0, n)) occurs in no earlier draw, else
// 0 (self pairs get 0). Returns the number of distinct pairs. Used by recipes
// that fix a count of distinct pairs rather than a count of draws: they take
// draws in order until that count is reached. The draws are dealt into
// buckets by a hash of the pair (keeping draw order within a bucket), and
// each bucket is scanned in order against a hash set of its own.
int64_t synth_first_draws(int64_t m, const int32_t* a, const int32_t* b, int64_t n,
                          uint8_t* first) {
  constexpr int kBucketBits = 10;
  constexpr int kBuckets = 1 << kBucketBits;
  const int nt = omp_get_max_threads();
  std::vector<int64_t> cnt((size_t)nt * kBuckets + 1, 0);
  auto key_of = [&](int64_t e) -> uint64_t {
    const uint64_t lo = (uint64_t)std::min(a[e], b[e]), hi = (uint64_t)std::max(a[e], b[e]);
    return lo * (uint64_t)n + hi;
  };
  auto bucket_of = [](uint64_t key) { return (int)(mix64(key) >> (64 - kBucketBits)); };
#pragma omp parallel num_threads(nt)
  {
    const int t = omp_get_thread_num();
    const int64_t lo = m * t / nt, hi = m * (t + 1) / nt;
    for (int64_t e = lo; e < hi; ++e) {
      first[e] = 0;
      if (a[e] != b[e]) ++cnt[(size_t)bucket_of(key_of(e)) * nt + t];
    }
  }
  // offsets: bucket-major, thread order within a bucket (draw order kept)
  int64_t run = 0;
  for (size_t i = 0; i < (size_t)nt * kBuckets; ++i) {
    const int64_t c = cnt[i];
    cnt[i] = run;
    run += c;
  }
  cnt[(size_t)nt * kBuckets] = run;
  std::vector<uint64_t> keys((size_t)run);
  std::vector<int64_t> draw((size_t)run);
#pragma omp parallel num_threads(nt)
  {
    const int t = omp_get_thread_num();
    const int64_t lo = m * t / nt, hi = m * (t + 1) / nt;
    for (int64_t e = lo; e < hi; ++e) {
      if (a[e] == b[e]) continue;
      const uint64_t k = key_of(e);
      const int64_t o = cnt[(size_t)bucket_of(k) * nt + t]++;
      keys[o] = k;
      draw[o] = e;
    }
  }
  // after the scatter, cnt[b * nt + t] is where slot (b, t + 1) starts; the
  // start of bucket b is cnt[b * nt - 1] (0 for b = 0)
  int64_t distinct = 0;
#pragma omp parallel for schedule(dynamic, 4) reduction(+ : distinct)
  for (int bk = 0; bk < kBuckets; ++bk) {
    const int64_t beg = bk == 0 ? 0 : cnt[(size_t)bk * nt - 1];
    const int64_t end = cnt[(size_t)(bk + 1) * nt - 1];
    size_t cap = 16;
    while (cap < (size_t)(2 * (end - beg))) cap <<= 1;
    std::vector<uint64_t> set(cap, UINT64_MAX);
    for (int64_t i = beg; i < end; ++i) {
      size_t h = (size_t)mix64(keys[i] ^ 0x5bd1e995ULL) & (cap - 1);
      while (set[h] != UINT64_MAX && set[h] != keys[i]) h = (h + 1) & (cap - 1);
      if (set[h] == UINT64_MAX) {
        set[h] = keys[i];
        first[draw[i]] = 1;
        ++distinct;
      }
    }
  }
  return distinct;
}

// Index of the k-th (1-based) nonzero flag, or -1 when there are fewer.
int64_t synth_nth_set(int64_t m, const uint8_t* flags, int64_t k) {
  int64_t seen = 0;
  for (int64_t e = 0; e < m; ++e)
    if (flags[e] && ++seen == k) return e;
  return -1;
}

// One worker's partition of an undirected RMAT graph over [0, n_total), from
// its draws {u[e], v[e]} in draw order (first: synth_first_draws of them).
// A draw emits "v contributes to row u" when u < n_local and "u contributes
// to row v" when v < n_local, so the local-local block stays symmetric; self
// pairs emit nothing. A first draw adds as many distinct entries as it has
// local endpoints. With target >= 0, draws are taken until the distinct
// entries reach exactly `target`, a draw that would pass it being left out;
// take[e] (length m) marks the draws taken. Returns the number of draws
// consumed (one past the last taken), or -1 if the draws cannot reach the
// target.
int64_t synth_partition_select(int64_t m, const int32_t* u, const int32_t* v,
                               const uint8_t* first, int64_t n_local, int64_t target,
                               uint8_t* take) {
  int64_t total = 0;
  for (int64_t e = 0; e < m; ++e) {
    const int64_t add = first[e] ? (int64_t)(u[e] < n_local) + (v[e] < n_local) : 0;
    take[e] = 0;
    if (target >= 0 && total + add > target) continue;
    take[e] = u[e] != v[e];
    total += add;
    if (target >= 0 && total == target) return e + 1;
  }
  return target < 0 ? m : -1;
}

// The entries of the taken draws (see synth_partition_select), "src
// contributes to row dst", in draw order (duplicates included); returns their
// count (at most 2 m). raw_count[x] (length n_total, zeroed here) receives
// the number of taken draws touching x, a stand-in for the vertex's degree in
// the whole (unpartitioned) graph.
int64_t synth_partition_emit(int64_t m, const int32_t* u, const int32_t* v, const uint8_t* take,
                             int64_t n_local, int64_t n_total, int32_t* src, int32_t* dst,
                             int64_t* raw_count) {
  const int nt = omp_get_max_threads();
  std::vector<int64_t> counts((size_t)nt + 1, 0);
#pragma omp parallel num_threads(nt)
  {
    const int tid = omp_get_thread_num();
    const int64_t lo = m * tid / nt, hi = m * (tid + 1) / nt;
    int64_t c = 0;
    for (int64_t e = lo; e < hi; ++e)
      if (take[e]) c += (u[e] < n_local) + (v[e] < n_local);
    counts[tid + 1] = c;
  }
  for (int t = 0; t < nt; ++t) counts[t + 1] += counts[t];
#pragma omp parallel num_threads(nt)
  {
    const int tid = omp_get_thread_num();
    const int64_t lo = m * tid / nt, hi = m * (tid + 1) / nt;
    int64_t o = counts[tid];
    for (int64_t e = lo; e < hi; ++e) {
      if (!take[e]) continue;
      if (u[e] < n_local) { src[o] = v[e]; dst[o] = u[e]; ++o; }
      if (v[e] < n_local) { src[o] = u[e]; dst[o] = v[e]; ++o; }
    }
  }
  std::memset(raw_count, 0, sizeof(int64_t) * (size_t)n_total);
  for (int64_t e = 0; e < m; ++e) {
    if (!take[e]) continue;
    raw_count[u[e]] += 1;
    raw_count[v[e]] += 1;
  }
  return counts[nt];
}

// Uniform[-1, 1) features: x = (h >> 40) * 2^-23 - 1, exact in fp32.
// Element (i, j) of the n x f matrix (row stride ld) uses counter i*f + j.
void synth_uniform(uint64_t seed, int64_t n, int64_t f, int64_t ld, float* x) {
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < n; ++i)
    for (int64_t j = 0; j < f; ++j) {
      const uint64_t h = sm64(seed, (uint64_t)(i * f + j));
      x[i * ld + j] = (float)(int32_t)(h >> 40) * 0x1p-23f - 1.0f;
    }
}

// Standard normal features by the Box-Muller transform in double, rounded
// to fp32. Element k = i*f + j uses counters 2k and 2k+1.
void synth_normal(uint64_t seed, int64_t n, int64_t f, int64_t ld, float* x) {
  const double two_pi = 6.283185307179586476925286766559;
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < n; ++i)
    for (int64_t j = 0; j < f; ++j) {
      const uint64_t k = (uint64_t)(i * f + j);
      const double u1 = (double)((sm64(seed, 2 * k) >> 11) + 1) * 0x1p-53;  // (0, 1]
      const double u2 = (double)(sm64(seed, 2 * k + 1) >> 11) * 0x1p-53;    // [0, 1)
      x[i * ld + j] = (float)(std::sqrt(-2.0 * std::log(u1)) * std::cos(two_pi * u2));
    }
}

// Glorot-uniform weights U(-L, L), L = sqrt(6 / (fan_in + fan_out)), for a
// fan_in x fan_out row-major matrix; element k uses counter k.
void synth_glorot(uint64_t seed, int64_t fan_in, int64_t fan_out, float* w) {
  const double lim = std::sqrt(6.0 / (double)(fan_in + fan_out));
  const int64_t total = fan_in * fan_out;
#pragma omp parallel for schedule(static)
  for (int64_t k = 0; k < total; ++k) {
    const uint64_t h = sm64(seed, (uint64_t)k);
    const double u = (double)(h >> 11) * 0x1p-53;  // [0, 1)
    w[k] = (float)((2.0 * u - 1.0) * lim);
  }
}

// Class labels uniform in [0, n_classes).
void synth_labels(uint64_t seed, int64_t n, int32_t n_classes, int32_t* y) {
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < n; ++i)
    y[i] = (int32_t)(((sm64(seed, (uint64_t)i) >> 32) * (uint64_t)n_classes) >> 32);
}

// Uniform random bytes in [0, 255] (code matrices for tests that exercise
// the halo path with arbitrary codes).
void synth_bytes(uint64_t seed, int64_t n, int64_t f, int64_t ld, uint8_t* q) {
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < n; ++i)
    for (int64_t j = 0; j < f; ++j) q[i * ld + j] = (uint8_t)(sm64(seed, (uint64_t)(i * f + j)) >> 56);
}

int synth_num_threads(void) { return omp_get_max_threads(); }

}  // extern "C"
