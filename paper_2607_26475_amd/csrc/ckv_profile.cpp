// ckv_profile.cpp -- event pool and aggregation behind ckv_profile_*().
#include <atomic>
#include <mutex>
#include <vector>

#include "ckv_launch.hpp"
#include "ckv_profile.hpp"

namespace ckv {
namespace {

struct Record {
  int id;
  hipEvent_t start, stop;
};

std::atomic<bool> g_on{false};
std::atomic<uint32_t> g_mask{0};
uint32_t g_every = 1;                 // stamp one launch in g_every per class
uint64_t g_seen[CKV_K_COUNT] = {};    // launches of each class since begin
std::mutex g_mu;
std::vector<Record> g_records;
std::vector<hipEvent_t> g_pool;

hipEvent_t take_event() {
  if (!g_pool.empty()) {
    hipEvent_t e = g_pool.back();
    g_pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

void recycle_all() {
  for (const Record& r : g_records) {
    g_pool.push_back(r.start);
    g_pool.push_back(r.stop);
  }
  g_records.clear();
}

}  // namespace

bool profile_events(int id, hipEvent_t* start, hipEvent_t* stop) {
  if (!g_on.load(std::memory_order_relaxed)) return false;
  if (!((g_mask.load(std::memory_order_relaxed) >> id) & 1u)) return false;
  std::lock_guard<std::mutex> lk(g_mu);
  if (!g_on.load(std::memory_order_relaxed)) return false;
  if (g_seen[id]++ % g_every) return false;
  hipEvent_t a = take_event(), b = take_event();
  if (!a || !b) {
    if (a) g_pool.push_back(a);
    if (b) g_pool.push_back(b);
    return false;
  }
  g_records.push_back({id, a, b});
  *start = a;
  *stop = b;
  return true;
}

#ifdef CKV_DEBUG
std::atomic<int> g_debug{1};
#else
std::atomic<int> g_debug{0};
#endif
thread_local hipError_t g_debug_err = hipSuccess;

bool debug_on() { return g_debug.load(std::memory_order_relaxed) != 0; }

void debug_after_launch(hipStream_t s) {
  hipError_t e = hipGetLastError();
  if (e == hipSuccess) e = hipStreamSynchronize(s);
  if (e != hipSuccess && g_debug_err == hipSuccess) g_debug_err = e;
}

hipError_t launch_status() {
  const hipError_t e = g_debug_err;
  g_debug_err = hipSuccess;
  const hipError_t last = hipGetLastError();
  return e != hipSuccess ? e : last;
}

}  // namespace ckv

extern "C" {

int ckv_set_debug(int on) {
  ckv::g_debug.store(on ? 1 : 0);
  return CKV_OK;
}

const char* ckv_kernel_name(int id) {
  static const char* names[CKV_K_COUNT] = {"zero", "score", "hist", "filter", "finish",
                                           "attn", "combine", "dual", "gather", "miss",
                                           "landmarks", "expand", "reconstruct",
                                           "select_attn", "probe", "critical"};
  return (id >= 0 && id < CKV_K_COUNT) ? names[id] : "";
}

int ckv_profile_begin_sampled(uint32_t kernel_mask, uint32_t every) {
  if (every < 1) return ckv::fail(CKV_EINVAL, "every must be at least 1");
  std::lock_guard<std::mutex> lk(ckv::g_mu);
  ckv::recycle_all();
  ckv::g_every = every;
  for (uint64_t& c : ckv::g_seen) c = 0;
  ckv::g_mask.store(kernel_mask & CKV_K_ALL);
  ckv::g_on.store(true);
  return CKV_OK;
}

int ckv_profile_begin(uint32_t kernel_mask) { return ckv_profile_begin_sampled(kernel_mask, 1); }

int ckv_profile_end(ckv_kernel_stats* stats) {
  if (!stats) return ckv::fail(CKV_EINVAL, "stats is NULL");
  std::lock_guard<std::mutex> lk(ckv::g_mu);
  ckv::g_on.store(false);
  for (int i = 0; i < CKV_K_COUNT; ++i) stats[i] = ckv_kernel_stats{0, 0.0, 0.0};
  int rc = CKV_OK;
  for (const ckv::Record& r : ckv::g_records) {
    float ms = 0.f;
    hipError_t e = hipEventSynchronize(r.stop);
    if (e == hipSuccess) e = hipEventElapsedTime(&ms, r.start, r.stop);
    if (e != hipSuccess) {
      rc = ckv::hip_fail(e, "kernel timing event");
      continue;
    }
    ckv_kernel_stats& s = stats[r.id];
    s.launches += 1;
    s.total_ms += ms;
    if (ms > s.max_ms) s.max_ms = ms;
  }
  ckv::recycle_all();
  return rc;
}

}  // extern "C"
