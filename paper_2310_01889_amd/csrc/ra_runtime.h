// Host-side runtime helpers shared by the C-ABI translation units: thread-local error
// text, HIP error mapping, stream-ordered per-call workspace, optional kernel timing.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <initializer_list>
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

// Tensors made of rows of elements are read and written with 16-byte vector accesses from
// their start, so they must begin on a 16-byte boundary (rows16); float32 per-row vectors
// such as lse on a 4-byte one (vec4).  A null pointer (an absent optional argument) passes.
inline int check_aligned(std::initializer_list<const void*> rows16, std::initializer_list<const void*> vec4 = {}) {
  for (const void* p : rows16)
    if (reinterpret_cast<uintptr_t>(p) & 15u) return set_err(RA_EINVAL, "tensor pointer %p is not 16-byte aligned", p);
  for (const void* p : vec4)
    if (reinterpret_cast<uintptr_t>(p) & 3u) return set_err(RA_EINVAL, "pointer %p is not 4-byte aligned", p);
  return RA_OK;
}

// The current device's workspace pool: a stream-ordered memory pool owned by the library
// (created on first use, release threshold unlimited, so workspace freed at the end of a
// call is reused by the next call instead of being unmapped and mapped again).  The
// device's default pool is left as it is.
int workspace_pool(hipMemPool_t* out);

// Stream-ordered workspace and events owned by one call; released on every exit path.
// side: the library's side stream when the call enqueued work on it.  Before the workspace
// goes back to the pool the caller stream waits for everything enqueued on the side stream
// so far -- also on an error return in the middle of a call, where the call's own final
// join was never enqueued -- so that no copy still queued there can write into memory a
// later call has been given.
struct CallResources {
  hipStream_t stream;
  hipStream_t side = nullptr;
  void* ws = nullptr;
  std::vector<hipEvent_t> events;
  explicit CallResources(hipStream_t s) : stream(s) {}
  ~CallResources() {
    if (ws && side && side != stream) {
      hipEvent_t e;
      if (hipEventCreateWithFlags(&e, hipEventDisableTiming) == hipSuccess) {
        (void)hipEventRecord(e, side);
        (void)hipStreamWaitEvent(stream, e, 0);
        (void)hipEventDestroy(e);
      } else {
        (void)hipStreamSynchronize(side);
      }
    }
    if (ws) (void)hipFreeAsync(ws, stream);
    for (hipEvent_t e : events) (void)hipEventDestroy(e);
  }
  int alloc(size_t bytes) {
    if (bytes == 0) return RA_OK;
    hipMemPool_t pool;
    int rc = workspace_pool(&pool);
    if (rc) return rc;
    RA_HIP(hipMallocFromPoolAsync(&ws, bytes, pool, stream));
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
