// Hybrid pre/post-aggregation split of a remote graph (Algorithm 1, Section
// 5.2) with the minimum vertex cover of Section 5.3, on the host.
//
// The cut edges between a sending and a receiving worker form a bipartite
// graph (sources on the sender, destinations on the receiver). Sending a
// source row serves all of its cut edges (post-aggregation on the receiver);
// sending a pre-aggregated destination row serves all of its cut edges
// (pre-aggregation on the sender). The fewest rows that serve every edge form a
// minimum vertex cover (Eq. 1), which for a bipartite graph has the size of a
// maximum matching (Koenig). Each connected component is solved on its own,
// components in parallel: Hopcroft-Karp for the matching, then Koenig's
// alternating-path construction for the cover.

#include <algorithm>
#include <atomic>
#include <cstdint>
#include <cstdlib>
#include <new>
#include <numeric>
#include <thread>
#include <vector>

#include "common.h"

namespace gcn {
namespace {

constexpr int32_t kInf = INT32_MAX;

// Disjoint sets over sources [0, n_src) and destinations n_src + [0, n_dst).
struct Dsu {
  std::vector<int32_t> parent;
  explicit Dsu(int64_t n) : parent((size_t)n) { std::iota(parent.begin(), parent.end(), 0); }
  int32_t find(int32_t x) {
    while (parent[x] != x) {
      parent[x] = parent[parent[x]];
      x = parent[x];
    }
    return x;
  }
  void unite(int32_t a, int32_t b) {
    a = find(a);
    b = find(b);
    if (a != b) parent[std::max(a, b)] = std::min(a, b);
  }
};

// One connected component with local ids: left = sources, right = destinations.
struct Component {
  std::vector<int32_t> left, right;  // global ids, increasing
  std::vector<int64_t> off;          // left adjacency (local right ids)
  std::vector<int32_t> adj;
};

// Maximum matching by Hopcroft-Karp phases: a breadth-first search layers the
// left vertices by alternating distance from the free ones, then depth-first
// searches along the layers find a maximal set of disjoint shortest augmenting
// paths. Returns match_l (local right id or -1) and match_r.
void hopcroft_karp(const Component& c, std::vector<int32_t>& match_l, std::vector<int32_t>& match_r) {
  const int32_t nl = (int32_t)c.left.size(), nr = (int32_t)c.right.size();
  match_l.assign(nl, -1);
  match_r.assign(nr, -1);
  // greedy start: match each left vertex to its first free neighbour
  for (int32_t u = 0; u < nl; ++u)
    for (int64_t k = c.off[u]; k < c.off[u + 1]; ++k)
      if (match_r[c.adj[k]] < 0) {
        match_l[u] = c.adj[k];
        match_r[c.adj[k]] = u;
        break;
      }
  std::vector<int32_t> dist(nl), queue, stack, via;
  std::vector<int64_t> it(nl);
  queue.reserve(nl);
  for (;;) {
    queue.clear();
    for (int32_t u = 0; u < nl; ++u) {
      dist[u] = match_l[u] < 0 ? 0 : kInf;
      if (match_l[u] < 0) queue.push_back(u);
    }
    int32_t free_layer = kInf;  // layer at which a free right vertex is reached
    for (size_t qi = 0; qi < queue.size(); ++qi) {
      const int32_t u = queue[qi];
      if (dist[u] >= free_layer) break;
      for (int64_t k = c.off[u]; k < c.off[u + 1]; ++k) {
        const int32_t w = match_r[c.adj[k]];
        if (w < 0) {
          free_layer = std::min(free_layer, dist[u] + 1);
        } else if (dist[w] == kInf) {
          dist[w] = dist[u] + 1;
          queue.push_back(w);
        }
      }
    }
    if (free_layer == kInf) return;
    for (int32_t u = 0; u < nl; ++u) it[u] = c.off[u];
    for (int32_t root = 0; root < nl; ++root) {
      if (match_l[root] >= 0) continue;
      stack.assign(1, root);
      via.clear();
      while (!stack.empty()) {
        const int32_t x = stack.back();
        if (it[x] == c.off[x + 1]) {  // dead end: drop x from this phase
          dist[x] = kInf;
          stack.pop_back();
          if (!via.empty()) via.pop_back();
          continue;
        }
        const int32_t v = c.adj[it[x]++];
        const int32_t w = match_r[v];
        if (w < 0) {
          if (dist[x] + 1 != free_layer) continue;  // only shortest paths
          via.push_back(v);
          for (size_t i = 0; i < stack.size(); ++i) {
            match_l[stack[i]] = via[i];
            match_r[via[i]] = stack[i];
          }
          break;
        }
        if (dist[w] == dist[x] + 1) {
          via.push_back(v);
          stack.push_back(w);
        }
      }
    }
  }
}

// Koenig's construction from a maximum matching: Z = vertices reachable from
// free left vertices by alternating paths; cover = (left \ Z) + (right in Z).
void koenig_cover(const Component& c, const std::vector<int32_t>& match_l,
                  const std::vector<int32_t>& match_r, std::vector<uint8_t>& in_l,
                  std::vector<uint8_t>& in_r) {
  const int32_t nl = (int32_t)c.left.size(), nr = (int32_t)c.right.size();
  std::vector<uint8_t> zl(nl, 0), zr(nr, 0);
  std::vector<int32_t> queue;
  for (int32_t u = 0; u < nl; ++u)
    if (match_l[u] < 0) {
      zl[u] = 1;
      queue.push_back(u);
    }
  for (size_t qi = 0; qi < queue.size(); ++qi) {
    const int32_t u = queue[qi];
    for (int64_t k = c.off[u]; k < c.off[u + 1]; ++k) {
      const int32_t v = c.adj[k];
      if (zr[v]) continue;
      zr[v] = 1;
      const int32_t w = match_r[v];
      if (w >= 0 && !zl[w]) {
        zl[w] = 1;
        queue.push_back(w);
      }
    }
  }
  in_l.resize(nl);
  in_r.resize(nr);
  for (int32_t u = 0; u < nl; ++u) in_l[u] = !zl[u];
  for (int32_t v = 0; v < nr; ++v) in_r[v] = zr[v];
}

int worker_threads() {
  int n = (int)std::thread::hardware_concurrency();
  if (const char* s = std::getenv("OMP_NUM_THREADS")) {
    const int v = std::atoi(s);
    if (v > 0) n = std::min(n > 0 ? n : v, v);
  }
  return std::max(1, std::min(n, 64));
}

gcn_status split(int64_t n_src, int64_t n_dst, int64_t n_edges, const int32_t* src,
                 const int32_t* dst, uint8_t* is_post, int32_t* src_slot, int32_t* dst_slot,
                 int64_t* volume) {
  // per-source adjacency (counting sort), duplicates removed
  std::vector<int64_t> off((size_t)n_src + 1, 0);
  for (int64_t e = 0; e < n_edges; ++e) off[(size_t)src[e] + 1] += 1;
  for (int64_t u = 0; u < n_src; ++u) off[u + 1] += off[u];
  std::vector<int32_t> adj((size_t)n_edges);
  {
    std::vector<int64_t> pos(off.begin(), off.end() - 1);
    for (int64_t e = 0; e < n_edges; ++e) adj[(size_t)pos[src[e]]++] = dst[e];
  }
  int64_t w = 0;
  for (int64_t u = 0; u < n_src; ++u) {
    const int64_t a = off[u], b = off[u + 1];
    std::sort(adj.begin() + a, adj.begin() + b);
    const int64_t start = w;
    for (int64_t k = a; k < b; ++k)
      if (k == a || adj[k] != adj[k - 1]) adj[w++] = adj[k];
    off[u] = start;
  }
  off[n_src] = w;
  // connected components
  Dsu dsu(n_src + n_dst);
  for (int64_t u = 0; u < n_src; ++u)
    for (int64_t k = off[u]; k < off[u + 1]; ++k) dsu.unite((int32_t)u, (int32_t)(n_src + adj[k]));
  std::vector<int32_t> comp_of((size_t)(n_src + n_dst), -1);
  std::vector<Component> comps;
  std::vector<int32_t> local((size_t)(n_src + n_dst), -1);
  for (int64_t u = 0; u < n_src; ++u) {
    if (off[u] == off[u + 1]) continue;
    const int32_t r = dsu.find((int32_t)u);
    if (comp_of[r] < 0) {
      comp_of[r] = (int32_t)comps.size();
      comps.emplace_back();
    }
    Component& c = comps[comp_of[r]];
    local[u] = (int32_t)c.left.size();
    c.left.push_back((int32_t)u);
  }
  for (int64_t v = 0; v < n_dst; ++v) {
    const int32_t r = dsu.find((int32_t)(n_src + v));
    if (comp_of[r] < 0) continue;  // destination without cut edges
    Component& c = comps[comp_of[r]];
    local[n_src + v] = (int32_t)c.right.size();
    c.right.push_back((int32_t)v);
  }
  for (Component& c : comps) {
    c.off.assign(c.left.size() + 1, 0);
    for (size_t i = 0; i < c.left.size(); ++i) c.off[i + 1] = c.off[i] + (off[c.left[i] + 1] - off[c.left[i]]);
    c.adj.resize((size_t)c.off.back());
    for (size_t i = 0; i < c.left.size(); ++i) {
      const int32_t u = c.left[i];
      for (int64_t k = off[u]; k < off[u + 1]; ++k)
        c.adj[(size_t)(c.off[i] + k - off[u])] = local[n_src + adj[k]];
    }
  }
  // largest components first, spread over a pool of threads
  std::vector<int32_t> order(comps.size());
  std::iota(order.begin(), order.end(), 0);
  std::stable_sort(order.begin(), order.end(), [&](int32_t a, int32_t b) {
    return comps[a].adj.size() > comps[b].adj.size();
  });
  std::vector<uint8_t> cover_l((size_t)n_src, 0), cover_r((size_t)n_dst, 0);
  std::atomic<size_t> next{0};
  std::atomic<int64_t> matched{0};
  std::atomic<bool> failed{false};
  auto work = [&]() {
    try {
      std::vector<int32_t> ml, mr;
      std::vector<uint8_t> il, ir;
      int64_t local_matched = 0;
      for (size_t i; (i = next.fetch_add(1)) < order.size();) {
        const Component& c = comps[order[i]];
        hopcroft_karp(c, ml, mr);
        for (int32_t m : ml) local_matched += m >= 0;
        koenig_cover(c, ml, mr, il, ir);
        // components own disjoint vertices: no two threads write one flag
        for (size_t u = 0; u < c.left.size(); ++u) cover_l[c.left[u]] = il[u];
        for (size_t v = 0; v < c.right.size(); ++v) cover_r[c.right[v]] = ir[v];
      }
      matched += local_matched;
    } catch (...) {
      failed = true;
    }
  };
  const int nt = (int)std::min<size_t>((size_t)worker_threads(), std::max<size_t>(1, comps.size()));
  std::vector<std::thread> pool;
  for (int t = 1; t < nt; ++t) pool.emplace_back(work);
  work();
  for (auto& t : pool) t.join();
  if (failed) {
    set_error("out of host memory in the vertex-cover search");
    return GCN_ENOMEM;
  }
  int64_t n_cover = 0;
  if (src_slot) {
    int32_t k = 0;
    for (int64_t u = 0; u < n_src; ++u) src_slot[u] = cover_l[u] ? k++ : -1;
  }
  if (dst_slot) {
    int32_t k = 0;
    for (int64_t v = 0; v < n_dst; ++v) dst_slot[v] = cover_r[v] ? k++ : -1;
  }
  for (int64_t u = 0; u < n_src; ++u) n_cover += cover_l[u];
  for (int64_t v = 0; v < n_dst; ++v) n_cover += cover_r[v];
  if (n_cover != matched.load()) {
    set_error("internal error: cover size differs from the matching size");
    return GCN_ESTATE;
  }
  if (is_post)
    for (int64_t e = 0; e < n_edges; ++e) is_post[e] = cover_l[src[e]];
  if (volume) *volume = n_cover;
  return GCN_OK;
}

// Post-aggregation combine on the receiver: Y[idx[j], :] += P[j, :], one
// wavefront per received partial row.
constexpr int kAddWaves = 4;

__global__ __launch_bounds__(64 * kAddWaves) void k_add_rows(int64_t n, int64_t F,
                                                             const float* __restrict__ P,
                                                             int64_t ldp,
                                                             const int32_t* __restrict__ idx,
                                                             int64_t n_y, float* __restrict__ Y,
                                                             int64_t ldy, bool vec4) {
  const int64_t j = (int64_t)blockIdx.x * kAddWaves + threadIdx.x / 64;
  if (j >= n) return;
  const int64_t r = idx[j];
  if (r < 0 || r >= n_y) return;
  const float* p = P + j * ldp;
  float* y = Y + r * ldy;
  const int lane = threadIdx.x & 63;
  if (vec4) {
    for (int64_t f = 4 * lane; f < F; f += 256) {
      const float4 a = *reinterpret_cast<const float4*>(p + f);
      float4 b = *reinterpret_cast<const float4*>(y + f);
      b.x += a.x;
      b.y += a.y;
      b.z += a.z;
      b.w += a.w;
      *reinterpret_cast<float4*>(y + f) = b;
    }
  } else {
    for (int64_t f = lane; f < F; f += 64) y[f] += p[f];
  }
}

// The same combine for partial sums that arrive quantized (Section 6.1 step
// 3 applied to the pre-aggregated rows): Y[idx[j], f] += fmaf(q[j, f], S[j],
// Z[j]), codes of BITS bits (8: a byte per feature; 2: four per byte, feature
// f in bits 2 (f % 4) of byte f / 4). One wavefront per received row; with
// vec4 a lane takes four features (one 4-byte or one 1-byte code load).
template <int BITS>
__global__ __launch_bounds__(64 * kAddWaves) void k_add_rows_q(
    int64_t n, int64_t F, const uint8_t* __restrict__ Q, int64_t ldq,
    const float* __restrict__ zmin, const float* __restrict__ scale, int64_t ldp,
    const int32_t* __restrict__ idx, int64_t n_y, float* __restrict__ Y, int64_t ldy,
    bool vec4) {
  const int64_t j = (int64_t)blockIdx.x * kAddWaves + threadIdx.x / 64;
  if (j >= n) return;
  const int64_t r = idx[j];
  if (r < 0 || r >= n_y) return;
  const uint8_t* q = Q + j * ldq;
  const float z = zmin[j * ldp], sc = scale[j * ldp];
  float* y = Y + r * ldy;
  const int lane = threadIdx.x & 63;
  constexpr uint32_t mask = (1u << BITS) - 1u;
  if (vec4) {
    for (int64_t f = 4 * lane; f < F; f += 256) {
      const uint32_t c = BITS == 8 ? *reinterpret_cast<const uint32_t*>(q + f) : (uint32_t)q[f >> 2];
      float4 b = *reinterpret_cast<const float4*>(y + f);
      b.x += __builtin_fmaf((float)(c & mask), sc, z);
      b.y += __builtin_fmaf((float)((c >> BITS) & mask), sc, z);
      b.z += __builtin_fmaf((float)((c >> (2 * BITS)) & mask), sc, z);
      b.w += __builtin_fmaf((float)((c >> (3 * BITS)) & mask), sc, z);
      *reinterpret_cast<float4*>(y + f) = b;
    }
  } else {
    for (int64_t f = lane; f < F; f += 64) {
      const uint32_t c = BITS == 8 ? (uint32_t)q[f] : ((uint32_t)q[f >> 2] >> (2 * (f & 3))) & mask;
      y[f] += __builtin_fmaf((float)c, sc, z);
    }
  }
}

}  // namespace
}  // namespace gcn

using namespace gcn;

extern "C" gcn_status gcn_add_rows_q(int64_t n, int64_t F, int bits, const uint8_t* Q, int64_t ldq,
                                     const float* zmin, const float* scale, int64_t ldp,
                                     const int32_t* idx, int64_t n_y, float* Y, int64_t ldy,
                                     void* stream_) {
  clear_error();
  if (bits != 8 && bits != 2) {
    set_error("bits must be 8 or 2 (got %d)", bits);
    return GCN_EINVAL;
  }
  const int64_t qbytes = bits == 8 ? F : (F + 3) / 4;
  if (n < 0 || F < 1 || n_y < 0 || ldq < qbytes || ldp < 1 || ldy < F) {
    set_error("need n >= 0, n_y >= 0, F >= 1, ldq >= code bytes per row, ldp >= 1 and ldy >= F");
    return GCN_EINVAL;
  }
  if (n == 0) return GCN_OK;
  if (!Q || !zmin || !scale || !idx || !Y) {
    set_error("Q, zmin, scale, idx and Y must not be NULL");
    return GCN_EINVAL;
  }
  hipStream_t stream = (hipStream_t)stream_;
  const bool vec4 = F % 4 == 0 && ldy % 4 == 0 && reinterpret_cast<uintptr_t>(Y) % 16 == 0 &&
                    (bits == 2 || (ldq % 4 == 0 && reinterpret_cast<uintptr_t>(Q) % 4 == 0));
  ProfScope ps("add_rows_q", stream);
  const dim3 grid((unsigned)((n + kAddWaves - 1) / kAddWaves)), block(64 * kAddWaves);
  if (bits == 8)
    hipLaunchKernelGGL(k_add_rows_q<8>, grid, block, 0, stream, n, F, Q, ldq, zmin, scale, ldp,
                       idx, n_y, Y, ldy, vec4);
  else
    hipLaunchKernelGGL(k_add_rows_q<2>, grid, block, 0, stream, n, F, Q, ldq, zmin, scale, ldp,
                       idx, n_y, Y, ldy, vec4);
  GCN_HIP(hipGetLastError());
  return GCN_OK;
}

extern "C" gcn_status gcn_add_rows(int64_t n, int64_t F, const float* P, int64_t ldp,
                                   const int32_t* idx, int64_t n_y, float* Y, int64_t ldy,
                                   void* stream_) {
  clear_error();
  if (n < 0 || F < 1 || n_y < 0 || ldp < F || ldy < F) {
    set_error("need n >= 0, n_y >= 0, F >= 1, ldp >= F and ldy >= F");
    return GCN_EINVAL;
  }
  if (n == 0) return GCN_OK;
  if (!P || !idx || !Y) {
    set_error("P, idx and Y must not be NULL");
    return GCN_EINVAL;
  }
  hipStream_t stream = (hipStream_t)stream_;
  const bool vec4 = F % 4 == 0 && ldp % 4 == 0 && ldy % 4 == 0 &&
                    reinterpret_cast<uintptr_t>(P) % 16 == 0 && reinterpret_cast<uintptr_t>(Y) % 16 == 0;
  ProfScope ps("add_rows", stream);
  hipLaunchKernelGGL(k_add_rows, dim3((unsigned)((n + kAddWaves - 1) / kAddWaves)),
                     dim3(64 * kAddWaves), 0, stream, n, F, P, ldp, idx, n_y, Y, ldy, vec4);
  GCN_HIP(hipGetLastError());
  return GCN_OK;
}

extern "C" gcn_status gcn_prepost_split(int64_t n_src, int64_t n_dst, int64_t n_edges,
                                        const int32_t* src, const int32_t* dst, uint8_t* is_post,
                                        int32_t* src_slot, int32_t* dst_slot, int64_t* volume) {
  clear_error();
  if (n_src < 0 || n_dst < 0 || n_edges < 0 || n_src + n_dst > INT32_MAX) {
    set_error("n_src, n_dst and n_edges must be >= 0 and n_src + n_dst < 2^31");
    return GCN_EINVAL;
  }
  if (n_edges > 0 && (!src || !dst)) {
    set_error("src and dst must not be NULL when n_edges > 0");
    return GCN_EINVAL;
  }
  for (int64_t e = 0; e < n_edges; ++e)
    if (src[e] < 0 || src[e] >= n_src || dst[e] < 0 || dst[e] >= n_dst) {
      set_error("an edge endpoint lies outside [0, n_src) x [0, n_dst)");
      return GCN_ERANGE;
    }
  try {
    return split(n_src, n_dst, n_edges, src, dst, is_post, src_slot, dst_slot, volume);
  } catch (const std::bad_alloc&) {
    set_error("out of host memory in the vertex-cover search");
    return GCN_ENOMEM;
  }
}
