// Step descriptors passed by value to the kernels, and the launchers the ring
// scheduler calls.  One kernel launch covers every virtual host that has work in one
// ring step; each host contributes one "slot".
#pragma once

#include <hip/hip_runtime.h>

namespace ra {

constexpr int kMaxSlots = 64;        // hosts per launch (= maximum ring size)
constexpr int kFirst = 1;            // host's first active step: start from m=-inf, l=0, acc=0
constexpr int kLast = 2;             // host's last active step: finalize o = acc / l, lse

// Forwarding of the key/value block a host holds to the host that needs it at the next
// ring step (host i at step t holds block j = (i - t) mod N, which host i+1 holds at step
// t+1).  The bf16 step kernels copy the block's rows into that host's receive slot for the
// next step (the backward's dK/dV kernel from the rows it has in hand; the forward kernel
// after its own work, each workgroup its 128-row slice): slot s of the next step's half of
// the receive buffers starts at k0 + s * blk_bytes (v0 for values), in the layout
// [B, c, H, D].  to[n] is 1 + the destination slot of launch slot n, or 0 for none, so
// that a zero-initialised descriptor forwards nothing.
struct StepForward {
  const void* k0;
  const void* v0;
  long long blk_bytes;
  signed char to[kMaxSlots];
};

// One host's work in one ring step.
struct StepHost {
  const void* k;          // key block, row 0 (batch 0, head 0)
  const void* v;          // value block, row 0
  long long kv_bstride;   // elements between consecutive batches of k / v
  int q_row0;             // first row of the host's queries in q / o / lse / state rows
  int q_pos0;             // global position of that row (causal mask)
  int k_pos0;             // global position of the key block's first row
  int flags;              // kFirst | kLast
};

// Forward step: fold one key/value block into every listed host's running state.
struct FwdStep {
  StepHost host[kMaxSlots];
  const void* q;          // [B, Sq, H, D]
  void* o;                // [B, Sq, H, D]
  float* lse;             // [B, H, Sq]
  float* acc;             // running numerator, float32, B*H*Sq*D
  float* m;               // running max (log2 units of the scaled scores), [B, H, Sq]
  float* l;               // running denominator, [B, H, Sq]
  long long q_bstride;    // Sq * H * D
  int n_slots, B, H, Sq, c, causal;
  float scale;            // 1 / sqrt(D)
  StepForward fwd;        // bf16 kernel only: forward each slot's block to the next host
};

// Backward step: one key/value block per host; dq accumulates per host, dk/dv per block.
struct BwdStep {
  StepHost host[kMaxSlots];
  const void* q;          // [B, Sq, H, D]
  const void* dO;         // [B, Sq, H, D]
  const float* lse;       // [B, H, Sq]  lse, natural log (float32 kernels); -lse sqrt(D) (bf16)
  const float* delta;     // [B, H, Sq]  rowsum(dO * o) (float32 kernels); its negative (bf16)
  float* dq;              // float32 [B, Sq, H, D]
  float* dk;              // float32 [B, Skv, H, D]: gradient of the block each host holds
  float* dv;              //   (home position of that block: see dkv_row0)
  int dkv_row0[kMaxSlots];// first row of the host's current block in dk / dv
  long long q_bstride;    // Sq * H * D
  long long dkv_bstride;  // Skv * H * D
  int n_slots, B, H, Sq, c, causal;
  float scale;
  StepForward fwd;        // bf16 dK/dV kernel only: forward each slot's block (the keys a
                          // workgroup holds) to the next host
  // bf16 kernels, when the call holds every contribution to the gradients: the block a slot
  // holds is touched for the first time (kFirst: write dk / dv instead of adding into them)
  // or the last time (kLast: write the final sum, rounded, to dk_out / dv_out instead).
  // 0 = add into dk / dv.
  unsigned char dkv_flags[kMaxSlots];
  void* dk_out;           // bf16 [B, Skv, H, D] results (rows at the block's home position)
  void* dv_out;
  void* dq_out;           // bf16 [B, Sq, H, D]; when set, dq follows the host's kFirst / kLast
                          // flags the same way (null: always add into dq)
};

hipError_t launch_fwd_bf16(const FwdStep& s, int D, hipStream_t st);
hipError_t launch_fwd_f32(const FwdStep& s, int D, hipStream_t st);
// -Delta = -rowsum(dO * o) and -lse * sqrt(D), both [B, H, S] (for the bf16 step kernels)
hipError_t launch_bwd_pre_bf16(const void* o, const void* dO, const float* lse, float* ndelta, float* nlse_s,
                               int B, int S, int H, int D, hipStream_t st);
hipError_t launch_bwd_pre_f32(const float* o, const float* dO, float* delta, int B, int S, int H,
                              int D, hipStream_t st);
hipError_t launch_bwd_bf16(const BwdStep& s, int D, hipStream_t st);
hipError_t launch_bwd_f32(const BwdStep& s, int D, hipStream_t st);
hipError_t launch_cast_f32_bf16(const float* src, void* dst, long long n, hipStream_t st);
hipError_t launch_zero_f32(float* p, long long n, hipStream_t st);

}  // namespace ra
