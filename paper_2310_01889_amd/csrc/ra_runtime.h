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
void timing_push(int kind, hipEvent_t a, hipEvent_t b);

template <class F>
hipError_t timed_launch(int kind, hipStream_t st, F&& f) {
  if (!timing_on()) return f();
  hipEvent_t a, b;
  hipError_t e = hipEventCreate(&a);
  if (e != hipSuccess) return e;
  e = hipEventCreate(&b);
  if (e != hipSuccess) return e;
  (void)hipEventRecord(a, st);
  e = f();
  (void)hipEventRecord(b, st);
  timing_push(kind, a, b);
  return e;
}

}  // namespace ra
