// Host-side runtime helpers shared by the C-ABI translation units: thread-local error
// text, HIP error mapping, stream-ordered per-call workspace, optional kernel timing.
#pragma once

#include <hip/hip_runtime.h>

#include <string>
#include <vector>

#include "ringattn.h"

namespace ra {

extern thread_local std::string g_err;
int set_err(int code, const char* fmt, ...);

#define RA_HIP(expr)                                                                   \
  do {                                                                                 \
    hipError_t e_ = (expr);                                                            \
    if (e_ != hipSuccess)                                                              \
      return set_err(e_ == hipErrorOutOfMemory ? RA_ENOMEM : RA_EHIP, "%s failed: %s", \
                     #expr, hipGetErrorString(e_));                                    \
  } while (0)

void keep_pool();

// Stream-ordered workspace and events owned by one call; released on every exit path.
struct CallResources {
  hipStream_t stream;
  void* ws = nullptr;
  std::vector<hipEvent_t> events;
  explicit CallResources(hipStream_t s) : stream(s) {}
  ~CallResources() {
    if (ws) (void)hipFreeAsync(ws, stream);
    for (hipEvent_t e : events) (void)hipEventDestroy(e);
  }
  int alloc(size_t bytes) {
    if (bytes == 0) return RA_OK;
    keep_pool();
    RA_HIP(hipMallocAsync(&ws, bytes, stream));
    return RA_OK;
  }
  int event(hipEvent_t* e) {
    RA_HIP(hipEventCreateWithFlags(e, hipEventDisableTiming));
    events.push_back(*e);
    return RA_OK;
  }
};

// Kernel timing (ring_attn_timing_enable): true when launches are to be bracketed.
bool timing_on();
// own_a: the start event belongs to this entry (false when it is the end event of the
// entry before it)
void timing_push(int kind, hipEvent_t a, hipEvent_t b, bool own_a);

// Runs f() (which enqueues kernels on st) between two timing events when timing is on.
// chain, if given, carries the end event of the previous launch of a sequence that has
// nothing else enqueued between its launches: that event then also starts this launch,
// so one event, not two, separates consecutive launches (each costs a few microseconds
// of idle time between the kernels).
template <class F>
hipError_t timed_launch(int kind, hipStream_t st, F&& f, hipEvent_t* chain = nullptr) {
  if (!timing_on()) return f();
  // no system-scope fences: the events only carry timestamps, and the fences of a default
  // event widen the gap between consecutive launches by about 3 us per event
  hipEvent_t a = chain ? *chain : nullptr, b;
  const bool own_a = a == nullptr;
  hipError_t e;
  if (own_a) {
    e = hipEventCreateWithFlags(&a, hipEventDisableSystemFence);
    if (e != hipSuccess) return e;
    (void)hipEventRecord(a, st);
  }
  e = hipEventCreateWithFlags(&b, hipEventDisableSystemFence);
  if (e != hipSuccess) return e;
  e = f();
  (void)hipEventRecord(b, st);
  timing_push(kind, a, b, own_a);
  if (chain) *chain = b;
  return e;
}

}  // namespace ra
