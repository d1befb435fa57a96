// Error reporting, device allocation helpers and per-kernel event profiling.

#include <cstdarg>
#include <deque>
#include <map>
#include <mutex>
#include <string>
#include <vector>

#include "common.h"

namespace gcn {

namespace {
thread_local std::string g_last_error;

std::mutex g_prof_mu;
bool g_prof_on = false;
struct Pending {
  const char* name;
  hipEvent_t start, stop;
};
std::vector<Pending> g_pending;
struct Totals {
  int64_t launches = 0;
  double ms = 0.0;
};
std::map<std::string, Totals> g_totals;
std::deque<std::string> g_names;  // stable storage for names handed out (no reallocation)
}  // namespace

void set_error(const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = buf;
}

void clear_error() { g_last_error.clear(); }

gcn_status hip_fail(hipError_t e, const char* what, const char* file, int line) {
  set_error("%s failed: %s (%s:%d)", what, hipGetErrorString(e), file, line);
  (void)hipGetLastError();  // clear the sticky launch error where possible
  return (e == hipErrorOutOfMemory || e == hipErrorMemoryAllocation) ? GCN_ENOMEM : GCN_EHIP;
}

gcn_status dmalloc(void** p, size_t bytes, const char* what) {
  *p = nullptr;
  hipError_t e = hipMalloc(p, bytes);
  if (e != hipSuccess) {
    *p = nullptr;
    (void)hipGetLastError();
    set_error("device allocation of %zu bytes for %s failed: %s", bytes, what,
              hipGetErrorString(e));
    return GCN_ENOMEM;
  }
  return GCN_OK;
}

void dfree(void* p) {
  if (p) (void)hipFree(p);
}

// Stream-ordered temporaries come from the device's default memory pool. By
// default the pool hands freed blocks back to the driver at every
// synchronization, which makes each call pay for mapping its temporaries
// again; once per device the pool is told to keep them instead.
namespace {
std::mutex g_pool_mu;
uint64_t g_pool_done = 0;  // bit d set once device d's pool is configured

void keep_pool_memory() {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return;
  std::lock_guard<std::mutex> lk(g_pool_mu);
  if (g_pool_done & (1ull << dev)) return;
  hipMemPool_t pool;
  if (hipDeviceGetDefaultMemPool(&pool, dev) == hipSuccess) {
    uint64_t keep = UINT64_MAX;
    (void)hipMemPoolSetAttribute(pool, hipMemPoolAttrReleaseThreshold, &keep);
  }
  (void)hipGetLastError();
  g_pool_done |= 1ull << dev;
}
}  // namespace

namespace {
std::mutex g_side_mu;
hipStream_t g_side[64] = {};
}  // namespace

gcn_status SideWork::init(hipStream_t m) {
  main = m;
  int dev = 0;
  GCN_HIP(hipGetDevice(&dev));
  if (dev < 0 || dev >= 64) {
    set_error("device %d out of range for the side stream", dev);
    return GCN_EINVAL;
  }
  {
    std::lock_guard<std::mutex> lk(g_side_mu);
    if (!g_side[dev]) GCN_HIP(hipStreamCreateWithFlags(&g_side[dev], hipStreamNonBlocking));
    side = g_side[dev];
  }
  GCN_HIP(hipEventCreateWithFlags(&ev_fork, hipEventDisableTiming));
  GCN_HIP(hipEventCreateWithFlags(&ev_join, hipEventDisableTiming));
  return GCN_OK;
}

gcn_status SideWork::fork() {
  GCN_HIP(hipEventRecord(ev_fork, main));
  GCN_HIP(hipStreamWaitEvent(side, ev_fork, 0));
  pending = true;
  return GCN_OK;
}

gcn_status SideWork::join() {
  if (!pending) return GCN_OK;
  pending = false;
  GCN_HIP(hipEventRecord(ev_join, side));
  GCN_HIP(hipStreamWaitEvent(main, ev_join, 0));
  return GCN_OK;
}

SideWork::~SideWork() {
  (void)join();
  if (ev_fork) (void)hipEventDestroy(ev_fork);
  if (ev_join) (void)hipEventDestroy(ev_join);
}

gcn_status tmalloc(void** p, size_t bytes, hipStream_t stream, const char* what) {
  *p = nullptr;
  keep_pool_memory();
  hipError_t e = hipMallocAsync(p, bytes, stream);
  if (e != hipSuccess) {
    *p = nullptr;
    (void)hipGetLastError();
    set_error("stream-ordered allocation of %zu bytes for %s failed: %s", bytes, what,
              hipGetErrorString(e));
    return GCN_ENOMEM;
  }
  return GCN_OK;
}

void tfree(void* p, hipStream_t stream) {
  if (p) (void)hipFreeAsync(p, stream);
}

gcn_status check_graph(const gcn_graph* g) {
  if (!g) {
    set_error("graph handle is NULL");
    return GCN_EINVAL;
  }
  if (g->magic != kMagic) {
    set_error("graph handle is freed or corrupted");
    return GCN_ESTATE;
  }
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev != g->device) {
    set_error("the graph lives on device %d, the current device is %d", g->device, dev);
    return GCN_ESTATE;
  }
  return GCN_OK;
}

bool profiling() { return g_prof_on; }

ProfScope::ProfScope(const char* n, hipStream_t s) : name(n), stream(s) {
  if (!g_prof_on) return;
  if (hipEventCreate(&start) != hipSuccess) {
    start = nullptr;
    return;
  }
  (void)hipEventRecord(start, stream);
}

ProfScope::~ProfScope() {
  if (!start) return;
  hipEvent_t stop = nullptr;
  if (hipEventCreate(&stop) != hipSuccess) {
    (void)hipEventDestroy(start);
    return;
  }
  (void)hipEventRecord(stop, stream);
  std::lock_guard<std::mutex> lk(g_prof_mu);
  g_pending.push_back({name, start, stop});
}

}  // namespace gcn

using namespace gcn;

extern "C" const char* gcn_last_error(void) { return g_last_error.c_str(); }

extern "C" gcn_status gcn_profile_enable(int on) {
  std::lock_guard<std::mutex> lk(g_prof_mu);
  for (auto& p : g_pending) {
    (void)hipEventSynchronize(p.stop);
    (void)hipEventDestroy(p.start);
    (void)hipEventDestroy(p.stop);
  }
  g_pending.clear();
  g_totals.clear();
  g_prof_on = on != 0;
  return GCN_OK;
}

extern "C" gcn_status gcn_profile_read(const char** names, int64_t* launches, double* total_ms,
                                       int cap, int* n_kernels) {
  std::lock_guard<std::mutex> lk(g_prof_mu);
  for (auto& p : g_pending) {
    float ms = 0.f;
    if (hipEventSynchronize(p.stop) == hipSuccess &&
        hipEventElapsedTime(&ms, p.start, p.stop) == hipSuccess) {
      Totals& t = g_totals[p.name];
      t.launches += 1;
      t.ms += ms;
    }
    (void)hipEventDestroy(p.start);
    (void)hipEventDestroy(p.stop);
  }
  g_pending.clear();
  int i = 0;
  for (auto& kv : g_totals) {
    if (i < cap) {
      bool found = false;
      for (auto& s : g_names)
        if (s == kv.first) found = true;
      if (!found) g_names.push_back(kv.first);
      for (auto& s : g_names)
        if (s == kv.first && names) names[i] = s.c_str();
      if (launches) launches[i] = kv.second.launches;
      if (total_ms) total_ms[i] = kv.second.ms;
    }
    ++i;
  }
  if (n_kernels) *n_kernels = i;
  return GCN_OK;
}
