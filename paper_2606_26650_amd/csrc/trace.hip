// Launch tracing: when enabled, the library brackets each of its kernel
// launches with a pair of HIP events recorded on the launch stream and keeps
// the kernel tag with its algorithmic work (flops, bytes).  Durations are read
// back on demand, so a caller can time individual kernels inside a running
// workload without an external profiler.  Tracing is process-global and meant
// for one host thread.
#include <cstring>
#include <vector>

#include "kernels.h"

namespace catq {

struct TraceSlot {
  hipEvent_t start, stop;
  catq_trace_rec rec;
};

static std::vector<TraceSlot> g_slots;
static int g_count = 0;
static bool g_on = false;

int trace_begin(hipStream_t stream, const char* tag, double flops, double bytes, int64_t M,
                int64_t N, int64_t K) {
  if (!g_on || g_count >= (int)g_slots.size()) return -1;
  TraceSlot& s = g_slots[g_count];
  std::memset(&s.rec, 0, sizeof(s.rec));
  std::strncpy(s.rec.tag, tag, sizeof(s.rec.tag) - 1);
  s.rec.flops = flops;
  s.rec.bytes = bytes;
  s.rec.M = M;
  s.rec.N = N;
  s.rec.K = K;
  if (hipEventRecord(s.start, stream) != hipSuccess) return -1;
  return g_count++;
}

void trace_end(int slot, hipStream_t stream) {
  if (slot < 0) return;
  (void)hipEventRecord(g_slots[slot].stop, stream);
}

}  // namespace catq

using namespace catq;

extern "C" catq_status catq_trace_enable(int32_t capacity) {
  clear_error();
  CATQ_REQUIRE(capacity > 0 && capacity <= (1 << 20), CATQ_ERR_VALUE, "capacity out of range");
  for (auto& s : g_slots) {
    (void)hipEventDestroy(s.start);
    (void)hipEventDestroy(s.stop);
  }
  g_slots.assign(capacity, TraceSlot{});
  for (auto& s : g_slots) {
    if (hipEventCreate(&s.start) != hipSuccess || hipEventCreate(&s.stop) != hipSuccess) {
      set_error("hipEventCreate failed");
      g_slots.clear();
      return CATQ_ERR_HIP;
    }
  }
  g_count = 0;
  g_on = true;
  return CATQ_OK;
}

extern "C" void catq_trace_pause(int32_t paused) { g_on = !paused && !g_slots.empty(); }

extern "C" void catq_trace_reset(void) { g_count = 0; }

extern "C" int32_t catq_trace_count(void) { return g_count; }

extern "C" catq_status catq_trace_get(int32_t i, catq_trace_rec* out) {
  clear_error();
  CATQ_REQUIRE(out != nullptr, CATQ_ERR_NULL, "out is NULL");
  CATQ_REQUIRE(i >= 0 && i < g_count, CATQ_ERR_VALUE, "record %d of %d", i, g_count);
  TraceSlot& s = g_slots[i];
  if (hipEventSynchronize(s.stop) != hipSuccess) {
    set_error("hipEventSynchronize failed");
    return CATQ_ERR_HIP;
  }
  float ms = 0.f;
  if (hipEventElapsedTime(&ms, s.start, s.stop) != hipSuccess) {
    set_error("hipEventElapsedTime failed");
    return CATQ_ERR_HIP;
  }
  *out = s.rec;
  out->ms = ms;
  return CATQ_OK;
}

extern "C" void catq_trace_disable(void) {
  for (auto& s : g_slots) {
    (void)hipEventDestroy(s.start);
    (void)hipEventDestroy(s.stop);
  }
  g_slots.clear();
  g_count = 0;
  g_on = false;
}
