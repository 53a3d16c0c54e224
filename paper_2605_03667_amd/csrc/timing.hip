// Per-kernel timing for benchmarking: while enabled, every launch made by an
// entry point is bracketed by two hipEvents recorded on the launch stream.
// Events are created once and reused; nothing is allocated on the device.
#include <stdlib.h>
#include <string.h>

#include <string>
#include <vector>

#include "../../include/elas.h"
#include "internal.h"

namespace elas {

namespace {

struct Record {
  const char* tag;
  hipEvent_t start, stop;
};

struct Entry {
  std::string tag;
  int64_t launches = 0;
  double ms = 0.0;
};

bool g_enabled = false;
std::string g_only;                   // when not empty: the one tag that is timed
std::vector<hipEvent_t> g_pool;       // every event ever created, reused
size_t g_next = 0;                    // next free event in g_pool
std::vector<Record> g_records;
std::vector<Entry> g_entries;

hipEvent_t next_event() {
  if (g_next == g_pool.size()) {
    hipEvent_t e = nullptr;
    if (hipEventCreate(&e) != hipSuccess) return nullptr;
    g_pool.push_back(e);
  }
  return g_pool[g_next++];
}

// ELAS_DEBUG_SYNC: initial state from the environment variable of that name
// (set and not "0"), then whatever elas_debug_sync() last set.
int debug_sync_initial() {
  const char* v = getenv("ELAS_DEBUG_SYNC");
  return v != nullptr && v[0] != '\0' && strcmp(v, "0") != 0;
}
int g_debug_sync = debug_sync_initial();
thread_local hipError_t g_debug_error = hipSuccess;
thread_local const char* g_debug_tag = nullptr;

}  // namespace

bool timing_enabled() { return g_enabled; }

void debug_sync_reset() {
  g_debug_error = hipSuccess;
  g_debug_tag = nullptr;
}

hipError_t debug_sync_error(const char** tag) {
  if (tag) *tag = g_debug_tag;
  return g_debug_error;
}

TimedLaunch::TimedLaunch(const char* tag, hipStream_t stream) : tag_(tag), stream_(stream) {
  if (!g_enabled || (!g_only.empty() && g_only != tag)) return;
  start_ = next_event();
  stop_ = next_event();
  if (start_ && stop_) hipEventRecord(start_, stream_);
}

TimedLaunch::~TimedLaunch() {
  if (g_enabled && start_ && stop_) {
    hipEventRecord(stop_, stream_);
    g_records.push_back({tag_, start_, stop_});
  }
  if (g_debug_sync) {
    // wait for this launch and keep the first failure with its kernel tag
    const hipError_t e = hipStreamSynchronize(stream_);
    if (e != hipSuccess && g_debug_error == hipSuccess) {
      g_debug_error = e;
      g_debug_tag = tag_;
    }
  }
}

}  // namespace elas

extern "C" {

int elas_timing_enable(int enable) {
  elas::g_enabled = enable != 0;
  if (enable) {
    elas::g_records.clear();
    elas::g_entries.clear();
    elas::g_next = 0;
  }
  return ELAS_OK;
}

int elas_debug_sync(int enable) {
  const int prev = elas::g_debug_sync;
  if (enable >= 0) elas::g_debug_sync = enable != 0;
  return prev;
}

int elas_timing_only(const char* tag) {
  elas::g_only = tag ? tag : "";
  return ELAS_OK;
}

int elas_timing_collect(void) {
  elas::g_entries.clear();
  for (const auto& r : elas::g_records) {
    if (hipEventSynchronize(r.stop) != hipSuccess) return -ELAS_ERR_DEVICE;
    float ms = 0.f;
    if (hipEventElapsedTime(&ms, r.start, r.stop) != hipSuccess) return -ELAS_ERR_DEVICE;
    elas::Entry* e = nullptr;
    for (auto& x : elas::g_entries)
      if (x.tag == r.tag) e = &x;
    if (!e) {
      elas::g_entries.push_back({r.tag, 0, 0.0});
      e = &elas::g_entries.back();
    }
    e->launches += 1;
    e->ms += ms;
  }
  return (int)elas::g_entries.size();
}

int elas_timing_entry(int i, char* name, int name_cap, int64_t* launches, double* total_ms) {
  if (i < 0 || i >= (int)elas::g_entries.size()) return ELAS_ERR_SHAPE;
  const auto& e = elas::g_entries[i];
  if (name && name_cap > 0) {
    strncpy(name, e.tag.c_str(), (size_t)name_cap - 1);
    name[name_cap - 1] = '\0';
  }
  if (launches) *launches = e.launches;
  if (total_ms) *total_ms = e.ms;
  return ELAS_OK;
}

}  // extern "C"
