// Event registry behind msa_profile_enable / _reset / _read / _kernel_name.
// Host code only; guarded by one mutex (the attention path itself never
// touches it unless timing is enabled).
#include <atomic>
#include <cstring>
#include <deque>
#include <mutex>
#include <string>
#include <vector>

#include "msa.h"
#include "msa_profile.h"

namespace {

struct Pair {
  hipEvent_t start;
  hipEvent_t stop;
};

struct Entry {
  std::string name;
  std::vector<Pair> pairs;   // pairs[0 .. used) hold launches since the last reset
  size_t used = 0;
};

std::atomic<bool> g_enabled{false};
std::mutex g_mu;
// a deque never moves its elements when it grows, so the name pointers that
// msa_profile_kernel_name hands out stay valid until the library is unloaded
std::deque<Entry> g_entries;

Entry* find(const char* name) {
  for (auto& e : g_entries)
    if (e.name == name) return &e;
  return nullptr;
}

}  // namespace

namespace msa_prof {

bool enabled() { return g_enabled.load(std::memory_order_relaxed); }

void record(const char* kernel, hipEvent_t* start, hipEvent_t* stop) {
  std::lock_guard<std::mutex> lock(g_mu);
  Entry* e = find(kernel);
  if (!e) {
    g_entries.push_back(Entry{kernel, {}, 0});
    e = &g_entries.back();
  }
  if (e->used == e->pairs.size()) {
    Pair p{nullptr, nullptr};
    if (hipEventCreate(&p.start) != hipSuccess || hipEventCreate(&p.stop) != hipSuccess) return;
    e->pairs.push_back(p);
  }
  *start = e->pairs[e->used].start;
  *stop = e->pairs[e->used].stop;
  ++e->used;
}

}  // namespace msa_prof

extern "C" int msa_profile_enable(int on) {
  g_enabled.store(on != 0);
  return MSA_OK;
}

extern "C" int msa_profile_reset(void) {
  std::lock_guard<std::mutex> lock(g_mu);
  for (auto& e : g_entries) e.used = 0;
  return MSA_OK;
}

extern "C" const char* msa_profile_kernel_name(int i) {
  std::lock_guard<std::mutex> lock(g_mu);
  if (i < 0 || static_cast<size_t>(i) >= g_entries.size()) return nullptr;
  return g_entries[i].name.c_str();
}

extern "C" int msa_profile_read(const char* kernel, int64_t* launches, double* total_ms) {
  if (!kernel || !launches || !total_ms) return MSA_ERR_INVALID;
  std::lock_guard<std::mutex> lock(g_mu);
  *launches = 0;
  *total_ms = 0.0;
  const Entry* e = find(kernel);
  if (!e) return MSA_OK;
  for (size_t i = 0; i < e->used; ++i) {
    if (hipEventSynchronize(e->pairs[i].stop) != hipSuccess) return MSA_ERR_HIP;
    float ms = 0.f;
    if (hipEventElapsedTime(&ms, e->pairs[i].start, e->pairs[i].stop) != hipSuccess) return MSA_ERR_HIP;
    *total_ms += ms;
  }
  *launches = static_cast<int64_t>(e->used);
  return MSA_OK;
}
