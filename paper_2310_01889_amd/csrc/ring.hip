// Virtual-ring scheduler and the C ABI of the attention entry points.
//
// The ring of Section 3 is emulated on one device.  Every host's query block and every
// key/value block live in device memory.  A call runs n_hosts steps; at step t, host i
// folds in key/value block order(i, t) -- (i - t) mod n_hosts for the ring -- and every
// host with work at that step is one slot of a single kernel launch.  Step 0 reads each
// host's block where it lies (a host's own block needs no transfer).  For t >= 1 the
// block comes from that host's receive buffer: two slots used alternately (the
// double buffer of the paper's memory accounting: current and receiving key/value
// blocks).  The slot for step t+1 is filled while step t computes (the ppermute of the
// paper's code, overlapped with the blockwise computation): by the step-t kernels
// themselves when a bf16 call covers the whole ring in ring order, otherwise by copies on
// a library-owned side stream, with events ordering every copy after the last reader of
// its slot and every step after its copy (see run_ring).
#include <stdarg.h>
#include <stdio.h>
#include <stdlib.h>

#include <algorithm>
#include <mutex>
#include <string>
#include <vector>

#include "ra_common.h"
#include "ra_kernels.h"
#include "ra_runtime.h"
#include "ringattn.h"

namespace ra {

thread_local std::string g_err;

int set_err(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}


// ---------------------------------------------------------------------------------
// Per-device side stream (created once, default priority) and memory-pool setting.
// ---------------------------------------------------------------------------------
namespace {
std::mutex g_mu;
hipStream_t g_side[64];
}  // namespace

int side_stream(hipStream_t* out) {
  int dev = 0;
  RA_HIP(hipGetDevice(&dev));
  if (dev < 0 || dev >= 64) return set_err(RA_EHIP, "device index %d out of range", dev);
  std::lock_guard<std::mutex> lk(g_mu);
  if (!g_side[dev]) RA_HIP(hipStreamCreateWithFlags(&g_side[dev], hipStreamNonBlocking));
  *out = g_side[dev];
  return RA_OK;
}

namespace {
hipMemPool_t g_pool[64];
}  // namespace

int workspace_pool(hipMemPool_t* out) {
  int dev = 0;
  RA_HIP(hipGetDevice(&dev));
  if (dev < 0 || dev >= 64) return set_err(RA_EHIP, "device index %d out of range", dev);
  std::lock_guard<std::mutex> lk(g_mu);
  if (!g_pool[dev]) {
    hipMemPoolProps props{};
    props.allocType = hipMemAllocationTypePinned;
    props.handleTypes = hipMemHandleTypeNone;
    props.location.type = hipMemLocationTypeDevice;
    props.location.id = dev;
    hipMemPool_t pool;
    RA_HIP(hipMemPoolCreate(&pool, &props));
    uint64_t thr = ~0ull;
    hipError_t e = hipMemPoolSetAttribute(pool, hipMemPoolAttrReleaseThreshold, &thr);
    if (e != hipSuccess) {
      (void)hipMemPoolDestroy(pool);
      return set_err(RA_EHIP, "hipMemPoolSetAttribute failed: %s", hipGetErrorString(e));
    }
    g_pool[dev] = pool;
  }
  *out = g_pool[dev];
  return RA_OK;
}

// ---------------------------------------------------------------------------------
// Optional per-kernel timing (benchmarks): when enabled, every step-kernel launch is
// bracketed by timing events on the stream it is launched on.
// ---------------------------------------------------------------------------------
namespace {
std::mutex g_tmu;
bool g_timing = false;
struct TimedLaunch { int kind; hipEvent_t a, b; bool own_a; };
std::vector<TimedLaunch> g_timed;
}  // namespace

bool timing_on() {
  std::lock_guard<std::mutex> lk(g_tmu);
  return g_timing;
}

void timing_push(int kind, hipEvent_t a, hipEvent_t b, bool own_a) {
  std::lock_guard<std::mutex> lk(g_tmu);
  g_timed.push_back({kind, a, b, own_a});
}

static bool env_flag(const char* name) {
  const char* v = getenv(name);
  return v && v[0] && v[0] != '0';
}


// ---------------------------------------------------------------------------------
// Ring plan shared by forward and backward.
// ---------------------------------------------------------------------------------
struct RingProblem {
  const void *q, *k, *v;
  int B, H, S, D, N, causal, elt;   // elt: bytes per element (2 = bf16, 4 = float32)
  int Sq;                           // rows of q / o / lse: S (all hosts) or c (one host)
  std::vector<int> hosts;           // hosts evaluated by this call
  std::vector<int> order;           // order[i * N + t] (empty: ring order (i - t) mod N)
  int c() const { return S / N; }
  int blk(int i, int t) const { return order.empty() ? ((i - t) % N + N) % N : order[i * N + t]; }
  bool active(int i, int j) const { return !causal || j <= i; }  // block j not fully masked
  int q_row0(int i) const { return Sq == S ? i * c() : 0; }
};

// Receive buffers: slot s (0/1) of host-slot hslot, for k and v.
struct RecvBuffers {
  char* base = nullptr;
  size_t blk_bytes = 0;
  int nh = 0;
  char* k(int s, int hslot) const { return base + ((size_t)(s * nh + hslot)) * blk_bytes; }
  char* v(int s, int hslot) const { return base + ((size_t)((2 + s) * nh + hslot)) * blk_bytes; }
  static size_t bytes(size_t blk_bytes, int nh) { return 4 * (size_t)nh * blk_bytes; }
};

static int copy_block(const RingProblem& P, const void* src_all, char* dst, int j, hipStream_t st) {
  const size_t rowb = (size_t)P.H * P.D * P.elt;
  const size_t blkb = (size_t)P.c() * rowb;
  const char* src = (const char*)src_all + (size_t)j * blkb;
  if (P.B == 1) {
    RA_HIP(hipMemcpyAsync(dst, src, blkb, hipMemcpyDeviceToDevice, st));
  } else {
    RA_HIP(hipMemcpy2DAsync(dst, blkb, src, (size_t)P.S * rowb, blkb, P.B, hipMemcpyDeviceToDevice, st));
  }
  return RA_OK;
}

// Enqueue the whole ring: `launch(t, hosts_of_step, ..., forward, contiguous)` is called once
// per step with, for every active host, (host, block, kv pointers, batch stride, first/last
// flags); `contiguous` says that nothing was enqueued on the stream since the previous step.
//
// The block a host needs at step t+1 is the one its predecessor holds at step t.  In bf16,
// when the call covers every host of the ring in ring order, the step-t kernels write that
// block into the successor's receive slot themselves (the forward kernel's workgroups as
// they finish, the backward's dK/dV kernel from the rows it loads anyway) -- the send half
// of the ring's exchange, with no separate copy and no wait between the steps.  Otherwise
// (one host's share; a custom order; float32; or RINGATTN_SERIAL_COPY set) each step's
// blocks are copied from their home rows into the receive slots by device-to-device
// copies, on a side stream two steps ahead (or serially on the caller stream).
template <class Launch>
static int run_ring(const RingProblem& P, hipStream_t stream, CallResources& R, char* recv_base, Launch&& launch) {
  const int N = P.N;
  const int nh = (int)P.hosts.size();
  RecvBuffers rb;
  rb.base = recv_base;
  rb.blk_bytes = (size_t)P.B * P.c() * P.H * P.D * P.elt;
  rb.nh = nh;

  // first / last active step of every host
  std::vector<int> first(nh, -1), last(nh, -1);
  for (int t = 0; t < N; ++t)
    for (int s = 0; s < nh; ++s)
      if (P.active(P.hosts[s], P.blk(P.hosts[s], t))) {
        if (first[s] < 0) first[s] = t;
        last[s] = t;
      }

  const bool serial = env_flag("RINGATTN_SERIAL_COPY");
  const bool poison = env_flag("RINGATTN_POISON");
  bool forward = N > 1 && !serial && P.elt == 2 && nh == N && P.order.empty();
  for (int s = 0; forward && s < nh; ++s) forward = P.hosts[s] == s;
  hipStream_t side = stream;
  if (!serial && !forward && N > 1) {
    int rc = side_stream(&side);
    if (rc) return rc;
    R.side = side;
  }
  std::vector<hipEvent_t> ev_copy(N + 1, nullptr);
  hipEvent_t ev_entry = nullptr;
  if (side != stream) {
    int rc = R.event(&ev_entry);
    if (rc) return rc;
    RA_HIP(hipEventRecord(ev_entry, stream));
    RA_HIP(hipStreamWaitEvent(side, ev_entry, 0));
  }
  auto enqueue_copies = [&](int t) -> int {
    for (int s = 0; s < nh; ++s) {
      const int i = P.hosts[s], j = P.blk(i, t);
      if (!P.active(i, j)) continue;
      if (poison) {  // a step that read its slot before this copy landed would see NaN
        RA_HIP(hipMemsetAsync(rb.k(t & 1, s), 0xFF, rb.blk_bytes, side));
        RA_HIP(hipMemsetAsync(rb.v(t & 1, s), 0xFF, rb.blk_bytes, side));
      }
      int rc = copy_block(P, P.k, rb.k(t & 1, s), j, side);
      if (!rc) rc = copy_block(P, P.v, rb.v(t & 1, s), j, side);
      if (rc) return rc;
    }
    if (side != stream) {
      int rc = R.event(&ev_copy[t]);
      if (rc) return rc;
      RA_HIP(hipEventRecord(ev_copy[t], side));
    }
    return RA_OK;
  };
  if (N > 1 && !serial && !forward) {
    int rc = enqueue_copies(1);
    if (!rc && N > 2) rc = enqueue_copies(2);
    if (rc) return rc;
  }

  const size_t rowe = (size_t)P.H * P.D;
  for (int t = 0; t < N; ++t) {
    if (t >= 1 && !forward) {
      if (serial) {
        int rc = enqueue_copies(t);
        if (rc) return rc;
      } else {
        RA_HIP(hipStreamWaitEvent(stream, ev_copy[t], 0));
      }
    }
    std::vector<StepHost> hs;
    std::vector<int> host_ids, blk_ids;
    for (int s = 0; s < nh; ++s) {
      const int i = P.hosts[s], j = P.blk(i, t);
      if (!P.active(i, j)) continue;
      StepHost h{};
      if (t == 0) {
        h.k = (const char*)P.k + (size_t)j * P.c() * rowe * P.elt;
        h.v = (const char*)P.v + (size_t)j * P.c() * rowe * P.elt;
        h.kv_bstride = (long long)P.S * rowe;
      } else {
        h.k = rb.k(t & 1, s);
        h.v = rb.v(t & 1, s);
        h.kv_bstride = (long long)P.c() * rowe;
      }
      h.q_row0 = P.q_row0(i);
      h.q_pos0 = i * P.c();
      h.k_pos0 = j * P.c();
      h.flags = (t == first[s] ? kFirst : 0) | (t == last[s] ? kLast : 0);
      hs.push_back(h);
      host_ids.push_back(i);
      blk_ids.push_back(j);
    }
    StepForward fw{};  // zero: no forwarding
    if (forward && t + 1 < N) {
      const int nxt = (t + 1) & 1;
      fw.k0 = rb.k(nxt, 0);
      fw.v0 = rb.v(nxt, 0);
      fw.blk_bytes = (long long)rb.blk_bytes;
      for (size_t n = 0; n < hs.size(); ++n) {
        const int succ = (host_ids[n] + 1) % N;  // holds block blk_ids[n] at step t+1
        if (P.active(succ, blk_ids[n])) fw.to[n] = (signed char)(succ + 1);
      }
      if (poison) {  // a receive slot the step-t kernels leave unwritten would read NaN
        RA_HIP(hipMemsetAsync(rb.k(nxt, 0), 0xFF, rb.blk_bytes * nh, stream));
        RA_HIP(hipMemsetAsync(rb.v(nxt, 0), 0xFF, rb.blk_bytes * nh, stream));
      }
    }
    // contiguous: nothing has been enqueued on the stream since the previous step's launch
    const bool contiguous = t > 0 && forward && !poison;
    int rc = launch(t, hs, host_ids, blk_ids, fw, contiguous);
    if (rc) return rc;
    if (!serial && !forward && t >= 1 && t + 2 < N) {
      hipEvent_t done;
      rc = R.event(&done);
      if (rc) return rc;
      RA_HIP(hipEventRecord(done, stream));
      RA_HIP(hipStreamWaitEvent(side, done, 0));
      rc = enqueue_copies(t + 2);
      if (rc) return rc;
    }
  }
  if (side != stream) {
    hipEvent_t tail;
    int rc = R.event(&tail);
    if (rc) return rc;
    RA_HIP(hipEventRecord(tail, side));
    RA_HIP(hipStreamWaitEvent(stream, tail, 0));
  }
  return RA_OK;
}

// ---------------------------------------------------------------------------------
// Forward
// ---------------------------------------------------------------------------------
static int run_fwd(const RingProblem& P, void* o, float* lse, hipStream_t stream) {
  const int nh = (int)P.hosts.size();
  const size_t recv = P.N > 1 ? RecvBuffers::bytes((size_t)P.B * P.c() * P.H * P.D * P.elt, nh) : 0;
  const size_t nrow = (size_t)P.B * P.H * P.Sq;
  const bool need_state = P.N > 1;
  const size_t state = need_state ? nrow * (P.D + 2) * sizeof(float) : 0;
  CallResources R(stream);
  int rc = R.alloc(recv + state);
  if (rc) return rc;
  char* base = (char*)R.ws;
  float* acc = need_state ? (float*)(base + recv) : nullptr;
  float* m = need_state ? acc + nrow * P.D : nullptr;
  float* l = need_state ? m + nrow : nullptr;

  FwdStep st{};
  st.q = P.q;
  st.o = o;
  st.lse = lse;
  st.acc = acc;
  st.m = m;
  st.l = l;
  st.q_bstride = (long long)P.Sq * P.H * P.D;
  st.B = P.B;
  st.H = P.H;
  st.Sq = P.Sq;
  st.c = P.c();
  st.causal = P.causal;
  st.scale = 1.0f / sqrtf((float)P.D);
  hipEvent_t chain = nullptr;  // end event of the previous step's launch (timing)
  return run_ring(P, stream, R, base, [&](int, const std::vector<StepHost>& hs, const std::vector<int>&,
                                         const std::vector<int>&, const StepForward& fw, bool contiguous) -> int {
    st.n_slots = (int)hs.size();
    for (size_t s = 0; s < hs.size(); ++s) st.host[s] = hs[s];
    st.fwd = fw;
    if (!contiguous) chain = nullptr;
    RA_HIP(timed_launch(RA_KERNEL_ATTN_FWD, stream, [&] {
      return P.elt == 2 ? launch_fwd_bf16(st, P.D, stream) : launch_fwd_f32(st, P.D, stream);
    }, &chain));
    return RA_OK;
  });
}

// ---------------------------------------------------------------------------------
// Backward
// ---------------------------------------------------------------------------------
static int run_bwd(const RingProblem& P, const void* o, const float* lse, const void* dO, void* dq,
                   void* dk, void* dv, hipStream_t stream) {
  const int nh = (int)P.hosts.size();
  const size_t recv = P.N > 1 ? RecvBuffers::bytes((size_t)P.B * P.c() * P.H * P.D * P.elt, nh) : 0;
  const size_t nrow = (size_t)P.B * P.H * P.Sq;
  const size_t telems = (size_t)P.B * P.S * P.H * P.D;
  const bool f32 = P.elt == 4;  // float32 gradients accumulate straight into the outputs
  const size_t grads = f32 ? 0 : 3 * telems * sizeof(float);
  CallResources R(stream);
  int rc = R.alloc(recv + 2 * nrow * sizeof(float) + grads);
  if (rc) return rc;
  char* base = (char*)R.ws;
  float* delta = (float*)(base + recv);
  float* lse2 = delta + nrow;  // bf16 path: -lse sqrt(D), in units of q.k
  float* gq = f32 ? (float*)dq : lse2 + nrow;
  float* gk = f32 ? (float*)dk : gq + telems;
  float* gv = f32 ? (float*)dv : gk + telems;
  // bf16: the call covers every host, so it holds every contribution to each gradient
  // row: the first one is written and the last one goes out in bf16 (no zero fill, no
  // cast).  float32: the outputs are zeroed and accumulated into.
  std::vector<int> blk_first(P.N, -1), blk_last(P.N, -1);  // steps that touch block j
  if (f32) {
    RA_HIP(launch_zero_f32(gq, (long long)telems, stream));
    RA_HIP(launch_zero_f32(gk, (long long)telems, stream));
    RA_HIP(launch_zero_f32(gv, (long long)telems, stream));
  } else {
    for (int t = 0; t < P.N; ++t)
      for (int i : P.hosts) {
        const int j = P.blk(i, t);
        if (!P.active(i, j)) continue;
        if (blk_first[j] < 0) blk_first[j] = t;
        blk_last[j] = t;
      }
  }
  if (f32)
    RA_HIP(launch_bwd_pre_f32((const float*)o, (const float*)dO, delta, P.B, P.Sq, P.H, P.D, stream));
  else
    RA_HIP(launch_bwd_pre_bf16(o, dO, lse, delta, lse2, P.B, P.Sq, P.H, P.D, stream));

  BwdStep st{};
  st.q = P.q;
  st.dO = dO;
  st.lse = f32 ? lse : lse2;
  st.delta = delta;
  st.dq = gq;
  st.dk = gk;
  st.dv = gv;
  st.q_bstride = (long long)P.Sq * P.H * P.D;
  st.dkv_bstride = (long long)P.S * P.H * P.D;
  st.B = P.B;
  st.H = P.H;
  st.Sq = P.Sq;
  st.c = P.c();
  st.causal = P.causal;
  st.scale = 1.0f / sqrtf((float)P.D);
  if (!f32) {
    st.dq_out = dq;
    st.dk_out = dk;
    st.dv_out = dv;
  }
  hipEvent_t chain = nullptr;  // end event of the previous step's launch (timing)
  rc = run_ring(P, stream, R, base, [&](int t, const std::vector<StepHost>& hs, const std::vector<int>&,
                                       const std::vector<int>& blks, const StepForward& fw, bool contiguous) -> int {
    st.n_slots = (int)hs.size();
    st.fwd = fw;
    for (size_t s = 0; s < hs.size(); ++s) {
      st.host[s] = hs[s];
      st.dkv_row0[s] = blks[s] * P.c();
      st.dkv_flags[s] = f32 ? 0
                            : (unsigned char)((t == blk_first[blks[s]] ? kFirst : 0) |
                                              (t == blk_last[blks[s]] ? kLast : 0));
    }
    if (!contiguous) chain = nullptr;
    RA_HIP(timed_launch(RA_KERNEL_ATTN_BWD, stream, [&] {
      return f32 ? launch_bwd_f32(st, P.D, stream) : launch_bwd_bf16(st, P.D, stream);
    }, &chain));
    return RA_OK;
  });
  return rc;
}

// ---------------------------------------------------------------------------------
// Backward, one host's share: the key/value blocks arrive in ring order together with the
// float32 dK/dV they carry; this host adds its contribution and passes them on.
// ---------------------------------------------------------------------------------
static int copy_rows(void* dst, size_t dpitch, const void* src, size_t spitch, size_t width, int height,
                     hipStream_t st) {
  if (height == 1 || (dpitch == width && spitch == width)) {
    RA_HIP(hipMemcpyAsync(dst, src, width * height, hipMemcpyDeviceToDevice, st));
  } else {
    RA_HIP(hipMemcpy2DAsync(dst, dpitch, src, spitch, width, height, hipMemcpyDeviceToDevice, st));
  }
  return RA_OK;
}

static int run_bwd_host(const void* q_blk, const void* k_all, const void* v_all, const void* o_blk,
                        const float* lse_blk, const void* dO_blk, void* dq_blk, float* dk_acc, float* dv_acc,
                        int B, int H, int S, int D, int N, int host, int causal, hipStream_t stream) {
  const int c = S / N;
  const size_t rowe = (size_t)H * D;           // elements per token row
  const size_t blk = (size_t)c * rowe;         // elements of one block (per batch)
  const size_t nrow = (size_t)B * H * c;
  const size_t qel = (size_t)B * blk;
  // workspace: K/V slots (bf16) and dK/dV slots (float32), 2 each; Delta, lse2; dq (float32,
  // written by the host's first active step, rounded into dq_blk by its last)
  const size_t kv_slot = qel * 2, g_slot = qel * 4;
  CallResources R(stream);
  int rc = R.alloc(4 * kv_slot + 4 * g_slot + 2 * nrow * 4 + qel * 4);
  if (rc) return rc;
  char* base = (char*)R.ws;
  auto kslot = [&](int s) { return base + s * kv_slot; };
  auto vslot = [&](int s) { return base + (2 + s) * kv_slot; };
  auto dkslot = [&](int s) { return (float*)(base + 4 * kv_slot + s * g_slot); };
  auto dvslot = [&](int s) { return (float*)(base + 4 * kv_slot + (2 + s) * g_slot); };
  float* delta = (float*)(base + 4 * kv_slot + 4 * g_slot);
  float* lse2 = delta + nrow;
  float* dq32 = lse2 + nrow;
  RA_HIP(launch_bwd_pre_bf16(o_blk, dO_blk, lse_blk, delta, lse2, B, c, H, D, stream));

  auto blk_of = [&](int t) { return ((host - t) % N + N) % N; };
  auto active = [&](int t) { return !causal || blk_of(t) <= host; };
  int t_last = 0;  // the host's last active step (step 0, its own block, is always active)
  for (int t = 0; t < N; ++t)
    if (active(t)) t_last = t;
  hipStream_t side = stream;
  rc = side_stream(&side);
  if (rc) return rc;
  R.side = side;
  hipEvent_t ev;
  if ((rc = R.event(&ev))) return rc;
  RA_HIP(hipEventRecord(ev, stream));
  RA_HIP(hipStreamWaitEvent(side, ev, 0));
  std::vector<hipEvent_t> ev_recv(N + 2, nullptr);
  // receive block blk_of(t) with its carried gradients into slot t & 1
  auto receive = [&](int t) -> int {
    if (t >= N || !active(t)) return RA_OK;
    const int j = blk_of(t), s2 = t & 1;
    const size_t off = (size_t)j * blk;
    int r = copy_rows(kslot(s2), blk * 2, (const char*)k_all + off * 2, (size_t)S * rowe * 2, blk * 2, B, side);
    if (!r) r = copy_rows(vslot(s2), blk * 2, (const char*)v_all + off * 2, (size_t)S * rowe * 2, blk * 2, B, side);
    if (!r) r = copy_rows(dkslot(s2), blk * 4, dk_acc + off, (size_t)S * rowe * 4, blk * 4, B, side);
    if (!r) r = copy_rows(dvslot(s2), blk * 4, dv_acc + off, (size_t)S * rowe * 4, blk * 4, B, side);
    if (r) return r;
    if ((r = R.event(&ev_recv[t]))) return r;
    RA_HIP(hipEventRecord(ev_recv[t], side));
    return RA_OK;
  };
  // pass block blk_of(t) on: its carried gradients leave slot t & 1
  auto send = [&](int t) -> int {
    const int j = blk_of(t), s2 = t & 1;
    const size_t off = (size_t)j * blk;
    int r = copy_rows(dk_acc + off, (size_t)S * rowe * 4, dkslot(s2), blk * 4, blk * 4, B, side);
    if (!r) r = copy_rows(dv_acc + off, (size_t)S * rowe * 4, dvslot(s2), blk * 4, blk * 4, B, side);
    return r;
  };
  if ((rc = receive(1)) || (rc = receive(2))) return rc;

  BwdStep st{};
  st.q = q_blk;
  st.dO = dO_blk;
  st.lse = lse2;
  st.delta = delta;
  st.dq = dq32;
  st.dq_out = dq_blk;
  st.q_bstride = (long long)blk;
  st.B = B;
  st.H = H;
  st.Sq = c;
  st.c = c;
  st.causal = causal;
  st.scale = 1.0f / sqrtf((float)D);
  st.n_slots = 1;
  for (int t = 0; t < N; ++t) {
    if (!active(t)) continue;
    const int j = blk_of(t);
    StepHost& h = st.host[0];
    h = StepHost{};
    if (t == 0) {  // the host's own block and the gradients it carries: in place
      h.k = (const char*)k_all + (size_t)j * blk * 2;
      h.v = (const char*)v_all + (size_t)j * blk * 2;
      h.kv_bstride = (long long)S * rowe;
      st.dk = dk_acc + (size_t)j * blk;
      st.dv = dv_acc + (size_t)j * blk;
      st.dkv_bstride = (long long)S * rowe;
    } else {
      RA_HIP(hipStreamWaitEvent(stream, ev_recv[t], 0));
      h.k = kslot(t & 1);
      h.v = vslot(t & 1);
      h.kv_bstride = (long long)blk;
      st.dk = dkslot(t & 1);
      st.dv = dvslot(t & 1);
      st.dkv_bstride = (long long)blk;
    }
    h.q_row0 = 0;
    h.q_pos0 = host * c;
    h.k_pos0 = j * c;
    h.flags = (t == 0 ? kFirst : 0) | (t == t_last ? kLast : 0);
    st.dkv_row0[0] = 0;
    RA_HIP(timed_launch(RA_KERNEL_ATTN_BWD, stream, [&] { return launch_bwd_bf16(st, D, stream); }));
    if (t >= 1) {
      hipEvent_t done;
      if ((rc = R.event(&done))) return rc;
      RA_HIP(hipEventRecord(done, stream));
      RA_HIP(hipStreamWaitEvent(side, done, 0));
      if ((rc = send(t)) || (rc = receive(t + 2))) return rc;
    }
  }
  hipEvent_t tail;
  if ((rc = R.event(&tail))) return rc;
  RA_HIP(hipEventRecord(tail, side));
  RA_HIP(hipStreamWaitEvent(stream, tail, 0));
  return RA_OK;
}

// ---------------------------------------------------------------------------------
// Argument validation
// ---------------------------------------------------------------------------------
static int validate(int B, int H, int S, int D, int N, int causal, int tile) {
  if (B <= 0 || H <= 0 || S <= 0 || D <= 0 || N <= 0)
    return set_err(RA_EINVAL, "sizes must be positive (B=%d H=%d S=%d D=%d n_hosts=%d)", B, H, S, D, N);
  if (causal != 0 && causal != 1) return set_err(RA_EINVAL, "causal must be 0 or 1 (got %d)", causal);
  if (D != 64 && D != 128) return set_err(RA_EUNSUPPORTED, "head dim D=%d not supported (64 or 128)", D);
  if (N > kMaxSlots) return set_err(RA_EUNSUPPORTED, "n_hosts=%d exceeds %d", N, kMaxSlots);
  if (S % N) return set_err(RA_EUNSUPPORTED, "S=%d is not a multiple of n_hosts=%d", S, N);
  if ((S / N) % tile)
    return set_err(RA_EUNSUPPORTED, "block S/n_hosts=%d is not a multiple of %d", S / N, tile);
  if ((long long)B * S * H * D >= (1ll << 31))
    return set_err(RA_EUNSUPPORTED, "B*S*H*D = %lld elements exceeds 2^31-1", (long long)B * S * H * D);
  return RA_OK;
}

static RingProblem all_hosts(const void* q, const void* k, const void* v, int B, int H, int S, int D, int N,
                             int causal, int elt) {
  RingProblem P{q, k, v, B, H, S, D, N, causal, elt, S, {}, {}};
  for (int i = 0; i < N; ++i) P.hosts.push_back(i);
  return P;
}

}  // namespace ra

using namespace ra;

// ---------------------------------------------------------------------------------
// Ragged causal lengths.  The sequence is cut into n_hosts blocks of c tokens, c the
// smallest multiple of 128 with n_hosts * c >= S, so the trailing blocks are short or
// empty; the tensors are staged into zero-padded workspace copies of length n_hosts * c.
// Under the causal mask no real query sees a padded key (its position is >= S), and a
// padded query row adds exactly zero to dK and dV (its o and dO are zero, so Delta = 0,
// dP = 0 and dS = 0), so the real rows come out as for the unpadded sequence.
// ---------------------------------------------------------------------------------
namespace {

__global__ void pad_zero_kernel(uint32_t* base, long long pitch_w, long long off_w, long long len_w,
                                long long rows) {
  const long long n = rows * len_w;
  for (long long i = blockIdx.x * (long long)blockDim.x + threadIdx.x; i < n;
       i += (long long)gridDim.x * blockDim.x)
    base[(i / len_w) * pitch_w + off_w + i % len_w] = 0u;
}

// dst [outer][n_dst units] <- src [outer][n_src units], n_src <= n_dst, the tail of each
// row zeroed; unit bytes a multiple of 4
int pad_copy(void* dst, const void* src, long long outer, long long n_src, long long n_dst, long long unit,
             hipStream_t st) {
  RA_HIP(hipMemcpy2DAsync(dst, (size_t)(n_dst * unit), src, (size_t)(n_src * unit), (size_t)(n_src * unit),
                          (size_t)outer, hipMemcpyDeviceToDevice, st));
  const long long pad_w = (n_dst - n_src) * unit / 4;
  if (pad_w > 0) {
    const long long n = outer * pad_w;
    const int blocks = (int)std::min<long long>((n + 255) / 256, 4096);
    pad_zero_kernel<<<blocks, 256, 0, st>>>((uint32_t*)dst, n_dst * unit / 4, n_src * unit / 4, pad_w, outer);
    RA_HIP(hipGetLastError());
  }
  return RA_OK;
}

// dst [outer][n_dst units] <- the first n_dst units of each row of src [outer][n_src units]
int unpad_copy(void* dst, const void* src, long long outer, long long n_dst, long long n_src, long long unit,
               hipStream_t st) {
  RA_HIP(hipMemcpy2DAsync(dst, (size_t)(n_dst * unit), src, (size_t)(n_src * unit), (size_t)(n_dst * unit),
                          (size_t)outer, hipMemcpyDeviceToDevice, st));
  return RA_OK;
}

// *Sp = n_hosts * c
int padded_len(int S, int N, long long* Sp) {
  if (S <= 0 || N <= 0) return set_err(RA_EINVAL, "sizes must be positive (S=%d n_hosts=%d)", S, N);
  const long long c = (((long long)S + N - 1) / N + 127) / 128 * 128;
  if (c * N > 0x7fffffffll) return set_err(RA_EUNSUPPORTED, "padded length %lld exceeds 2^31-1", c * N);
  *Sp = c * N;
  return RA_OK;
}

}  // namespace


extern "C" {

const char* ring_attn_last_error(void) { return g_err.c_str(); }

int ring_attn_release_workspace(void) {
  g_err.clear();
  hipMemPool_t pool;
  int rc = workspace_pool(&pool);
  if (rc) return rc;
  RA_HIP(hipMemPoolTrimTo(pool, 0));
  return RA_OK;
}

void ring_attn_timing_enable(int on) {
  std::lock_guard<std::mutex> lk(g_tmu);
  g_timing = on != 0;
}

int ring_attn_timing_read(int kind, double* total_ms, int* launches) {
  g_err.clear();
  if (!total_ms || !launches) return set_err(RA_EINVAL, "null pointer argument");
  std::vector<TimedLaunch> mine, rest;
  {
    std::lock_guard<std::mutex> lk(g_tmu);
    for (const TimedLaunch& t : g_timed) (t.kind == kind ? mine : rest).push_back(t);
    g_timed.swap(rest);
  }
  double sum = 0;
  int rc = RA_OK;
  for (const TimedLaunch& t : mine) {
    float ms = 0.f;
    if (rc == RA_OK) {
      hipError_t e = hipEventSynchronize(t.b);
      if (e == hipSuccess) e = hipEventElapsedTime(&ms, t.a, t.b);
      if (e != hipSuccess) rc = set_err(RA_EHIP, "timing event: %s", hipGetErrorString(e));
    }
    sum += ms;
  }
  // an entry's start event may be the end event of the entry before it: destroy once all
  // durations are read
  for (const TimedLaunch& t : mine) {
    if (t.own_a) (void)hipEventDestroy(t.a);
    (void)hipEventDestroy(t.b);
  }
  *total_ms = sum;
  *launches = (int)mine.size();
  return rc;
}

int ring_attn_fwd(const void* q, const void* k, const void* v, void* o, float* lse, int B, int H, int S, int D,
                  int n_hosts, int causal, hipStream_t stream) {
  g_err.clear();
  if (!q || !k || !v || !o || !lse) return set_err(RA_EINVAL, "null pointer argument");
  if (int e = check_aligned({q, k, v, o}, {lse})) return e;
  int rc = validate(B, H, S, D, n_hosts, causal, 128);
  if (rc) return rc;
  return run_fwd(all_hosts(q, k, v, B, H, S, D, n_hosts, causal, 2), o, lse, stream);
}

int ring_attn_fwd_f32(const float* q, const float* k, const float* v, float* o, float* lse, int B, int H, int S,
                      int D, int n_hosts, int causal, hipStream_t stream) {
  g_err.clear();
  if (!q || !k || !v || !o || !lse) return set_err(RA_EINVAL, "null pointer argument");
  if (int e = check_aligned({q, k, v, o}, {lse})) return e;
  int rc = validate(B, H, S, D, n_hosts, causal, 64);
  if (rc) return rc;
  return run_fwd(all_hosts(q, k, v, B, H, S, D, n_hosts, causal, 4), o, lse, stream);
}

int ring_attn_fwd_host(const void* q_blk, const void* k_all, const void* v_all, void* o_blk, float* lse_blk, int B,
                       int H, int S, int D, int n_hosts, int host_idx, int causal, hipStream_t stream) {
  g_err.clear();
  if (!q_blk || !k_all || !v_all || !o_blk || !lse_blk) return set_err(RA_EINVAL, "null pointer argument");
  if (int e = check_aligned({q_blk, k_all, v_all, o_blk}, {lse_blk})) return e;
  int rc = validate(B, H, S, D, n_hosts, causal, 128);
  if (rc) return rc;
  if (host_idx < 0 || host_idx >= n_hosts)
    return set_err(RA_EINVAL, "host_idx=%d outside [0, n_hosts=%d)", host_idx, n_hosts);
  RingProblem P{q_blk, k_all, v_all, B, H, S, D, n_hosts, causal, 2, S / n_hosts, {host_idx}, {}};
  return run_fwd(P, o_blk, lse_blk, stream);
}

int ring_attn_fwd_ordered(const void* q, const void* k, const void* v, void* o, float* lse, int B, int H, int S,
                          int D, int n_hosts, int causal, const int* kv_order, hipStream_t stream) {
  g_err.clear();
  if (!q || !k || !v || !o || !lse || !kv_order) return set_err(RA_EINVAL, "null pointer argument");
  if (int e = check_aligned({q, k, v, o}, {lse, kv_order})) return e;
  int rc = validate(B, H, S, D, n_hosts, causal, 128);
  if (rc) return rc;
  RingProblem P = all_hosts(q, k, v, B, H, S, D, n_hosts, causal, 2);
  P.order.assign(kv_order, kv_order + (size_t)n_hosts * n_hosts);
  for (int i = 0; i < n_hosts; ++i) {
    std::vector<int> seen(n_hosts, 0);
    for (int t = 0; t < n_hosts; ++t) {
      const int j = P.order[i * n_hosts + t];
      if (j < 0 || j >= n_hosts || seen[j]++)
        return set_err(RA_EINVAL, "kv_order row %d is not a permutation of 0..%d", i, n_hosts - 1);
    }
  }
  return run_fwd(P, o, lse, stream);
}

int ring_attn_bwd_host(const void* q_blk, const void* k_all, const void* v_all, const void* o_blk,
                       const float* lse_blk, const void* dO_blk, void* dq_blk, float* dk_acc, float* dv_acc, int B,
                       int H, int S, int D, int n_hosts, int host_idx, int causal, hipStream_t stream) {
  g_err.clear();
  if (!q_blk || !k_all || !v_all || !o_blk || !lse_blk || !dO_blk || !dq_blk || !dk_acc || !dv_acc)
    return set_err(RA_EINVAL, "null pointer argument");
  if (int e = check_aligned({q_blk, k_all, v_all, o_blk, dO_blk, dq_blk, dk_acc, dv_acc}, {lse_blk})) return e;
  int rc = validate(B, H, S, D, n_hosts, causal, 128);
  if (rc) return rc;
  if (host_idx < 0 || host_idx >= n_hosts)
    return set_err(RA_EINVAL, "host_idx=%d outside [0, n_hosts=%d)", host_idx, n_hosts);
  return run_bwd_host(q_blk, k_all, v_all, o_blk, lse_blk, dO_blk, dq_blk, dk_acc, dv_acc, B, H, S, D, n_hosts,
                      host_idx, causal, stream);
}

int ring_attn_bwd(const void* q, const void* k, const void* v, const void* o, const float* lse, const void* dO,
                  void* dq, void* dk, void* dv, int B, int H, int S, int D, int n_hosts, int causal,
                  hipStream_t stream) {
  g_err.clear();
  if (!q || !k || !v || !o || !lse || !dO || !dq || !dk || !dv) return set_err(RA_EINVAL, "null pointer argument");
  if (int e = check_aligned({q, k, v, o, dO, dq, dk, dv}, {lse})) return e;
  int rc = validate(B, H, S, D, n_hosts, causal, 128);
  if (rc) return rc;
  return run_bwd(all_hosts(q, k, v, B, H, S, D, n_hosts, causal, 2), o, lse, dO, dq, dk, dv, stream);
}

int ring_attn_bwd_f32(const float* q, const float* k, const float* v, const float* o, const float* lse,
                      const float* dO, float* dq, float* dk, float* dv, int B, int H, int S, int D, int n_hosts,
                      int causal, hipStream_t stream) {
  g_err.clear();
  if (!q || !k || !v || !o || !lse || !dO || !dq || !dk || !dv) return set_err(RA_EINVAL, "null pointer argument");
  if (int e = check_aligned({q, k, v, o, dO, dq, dk, dv}, {lse})) return e;
  int rc = validate(B, H, S, D, n_hosts, causal, 64);
  if (rc) return rc;
  return run_bwd(all_hosts(q, k, v, B, H, S, D, n_hosts, causal, 4), o, lse, dO, dq, dk, dv, stream);
}

int ring_attn_fwd_varlen(const void* q, const void* k, const void* v, void* o, float* lse, int B, int H, int S,
                         int D, int n_hosts, hipStream_t stream) {
  g_err.clear();
  if (!q || !k || !v || !o || !lse) return set_err(RA_EINVAL, "null pointer argument");
  if (int e = check_aligned({q, k, v, o}, {lse})) return e;
  long long Sp = 0;
  int rc = padded_len(S, n_hosts, &Sp);
  if (rc) return rc;
  rc = validate(B, H, (int)Sp, D, n_hosts, 1, 128);
  if (rc) return rc;
  if (Sp == S) return run_fwd(all_hosts(q, k, v, B, H, S, D, n_hosts, 1, 2), o, lse, stream);
  const long long row = (long long)H * D * 2, t = B * Sp * row;
  CallResources R(stream);
  if ((rc = R.alloc((size_t)(4 * t + (long long)B * H * Sp * 4)))) return rc;
  char* w = (char*)R.ws;
  char *qp = w, *kp = w + t, *vp = w + 2 * t, *op = w + 3 * t;
  float* lp = (float*)(w + 4 * t);
  if ((rc = pad_copy(qp, q, B, S, Sp, row, stream)) || (rc = pad_copy(kp, k, B, S, Sp, row, stream)) ||
      (rc = pad_copy(vp, v, B, S, Sp, row, stream)))
    return rc;
  if ((rc = run_fwd(all_hosts(qp, kp, vp, B, H, (int)Sp, D, n_hosts, 1, 2), op, lp, stream))) return rc;
  if ((rc = unpad_copy(o, op, B, S, Sp, row, stream))) return rc;
  return unpad_copy(lse, lp, (long long)B * H, S, Sp, 4, stream);
}

int ring_attn_bwd_varlen(const void* q, const void* k, const void* v, const void* o, const float* lse,
                         const void* dO, void* dq, void* dk, void* dv, int B, int H, int S, int D, int n_hosts,
                         hipStream_t stream) {
  g_err.clear();
  if (!q || !k || !v || !o || !lse || !dO || !dq || !dk || !dv) return set_err(RA_EINVAL, "null pointer argument");
  if (int e = check_aligned({q, k, v, o, dO, dq, dk, dv}, {lse})) return e;
  long long Sp = 0;
  int rc = padded_len(S, n_hosts, &Sp);
  if (rc) return rc;
  rc = validate(B, H, (int)Sp, D, n_hosts, 1, 128);
  if (rc) return rc;
  if (Sp == S) return run_bwd(all_hosts(q, k, v, B, H, S, D, n_hosts, 1, 2), o, lse, dO, dq, dk, dv, stream);
  const long long row = (long long)H * D * 2, t = B * Sp * row;
  CallResources R(stream);
  if ((rc = R.alloc((size_t)(8 * t + (long long)B * H * Sp * 4)))) return rc;
  char* w = (char*)R.ws;
  char* p[8];
  for (int i = 0; i < 8; ++i) p[i] = w + i * t;  // q k v o dO dq dk dv
  float* lp = (float*)(w + 8 * t);
  const void* src[5] = {q, k, v, o, dO};
  for (int i = 0; i < 5; ++i)
    if ((rc = pad_copy(p[i], src[i], B, S, Sp, row, stream))) return rc;
  if ((rc = pad_copy(lp, lse, (long long)B * H, S, Sp, 4, stream))) return rc;
  if ((rc = run_bwd(all_hosts(p[0], p[1], p[2], B, H, (int)Sp, D, n_hosts, 1, 2), p[3], lp, p[4], p[5], p[6], p[7],
                    stream)))
    return rc;
  if ((rc = unpad_copy(dq, p[5], B, S, Sp, row, stream)) || (rc = unpad_copy(dk, p[6], B, S, Sp, row, stream)))
    return rc;
  return unpad_copy(dv, p[7], B, S, Sp, row, stream);
}

}  // extern "C"
