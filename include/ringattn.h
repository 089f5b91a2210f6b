/*
 * ringattn.h -- C ABI of the MI355X (gfx950) ring-attention library.
 *
 * Ring Attention with Blockwise Transformers (Liu, Zaharia, Abbeel; arXiv 2310.01889):
 * one host's share of exact blockwise self-attention.  The sequence of length S is split
 * into n_hosts equal blocks of c = S / n_hosts tokens; host i keeps query block i
 * resident while key/value blocks reach it in ring order, block (i - t) mod n_hosts at
 * step t (Section 3, "Ring-Based Blockwise Attention"; Appendix A forward code).  Each
 * block is folded into the output with running row maximum, running denominator and a
 * rescaled output accumulator.  The backward pass (Appendix A backward code) accumulates
 * dQ on the host and dK/dV with the rotating block.  A blockwise feed-forward network
 * (Section 2 equation; Algorithm 1) follows the attention of the same query block.
 *
 * On one GPU the ring is virtual: all hosts' blocks live in device memory; each call
 * runs n_hosts ring steps, each one kernel launch covering every host that has work at
 * that step, and the block each host needs at the next step reaches its per-host receive
 * buffer (double buffer) during the current step: in bf16 calls over the whole ring the
 * step kernels write it there themselves (each host sends the block it holds to the next
 * host); otherwise (one host's share, float32) device-to-device copies on a
 * library-owned side stream bring it in, overlapping the compute of the current step.
 *
 * Conventions shared by every entry point
 *   - Pointers are DEVICE pointers unless stated.  The caller allocates and owns every
 *     input and output and keeps them alive until `stream` has finished the call.  The
 *     library keeps no pointer after returning.
 *   - Tensors are dense row-major.  q, k, v, o, dO, dq, dk, dv: [B, S, H, D] (batch,
 *     position, head, dim per head; the layout of the paper's code).  lse: float32
 *     [B, H, S], holding max + ln(denominator) of the scaled scores (natural log).
 *   - Every tensor except lse (and the optional per-row rstd of rms_norm_fwd) starts on a
 *     16-byte boundary; lse and rstd on a 4-byte one.  Other pointers give RA_EINVAL.
 *   - "bf16" tensors hold IEEE bfloat16 (hip_bfloat16 / torch.bfloat16).  Products are
 *     taken in bf16 with float32 accumulation (the paper's float32-logits option);
 *     softmax statistics, accumulators and weight gradients are float32; outputs are
 *     rounded to bf16 with round-to-nearest-even.
 *   - Scores are scaled by 1/sqrt(D) (Section 2 equation).  With causal != 0, query at
 *     global position p sees key at global position p' iff p' <= p; masked keys
 *     contribute exactly zero and fully masked blocks are skipped.
 *   - Calls are asynchronous and stream-ordered on `stream` (a hipStream_t; NULL means
 *     the legacy default stream).  Work on a side stream is joined back to `stream`
 *     by events, so callers see single-stream semantics.  Distinct streams may be used
 *     from distinct threads concurrently.
 *   - Workspace (receive buffers, float32 accumulators) is allocated stream-ordered on
 *     `stream` from a memory pool the library owns on each device, and freed back to that
 *     pool at the end of the call (stream-ordered).  The pool keeps freed memory cached for
 *     later calls until the process ends or ring_attn_release_workspace() is called; the
 *     device's default memory pool and its settings are not touched.
 *   - Return value: RA_OK or an ra_status error code.  Arguments are validated before
 *     anything is enqueued: on error nothing is enqueued and outputs are untouched.
 *     ring_attn_last_error() describes the last error on the calling thread.  NaN or
 *     Inf inputs are not checked; they propagate.
 *
 * Supported shapes: D in {64, 128}; 1 <= n_hosts <= 64; S % n_hosts == 0; the block
 * c = S / n_hosts a multiple of 128 (bf16 attention) or 64 (float32 attention); B, H >= 1;
 * B * S * H * D < 2^31 elements per tensor.  ring_attn_fwd_varlen / ring_attn_bwd_varlen
 * (causal, bf16) take any S >= 1; the limits then hold for the padded length.
 */
#ifndef RINGATTN_H
#define RINGATTN_H

#include <hip/hip_runtime.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  RA_OK = 0,
  RA_EINVAL = 1,        /* null pointer, non-positive size, bad enum value         */
  RA_EUNSUPPORTED = 2,  /* shape outside the supported set listed above            */
  RA_EHIP = 3,          /* a HIP launch, copy or event call failed                 */
  RA_ENOMEM = 4         /* workspace allocation failed                             */
} ra_status;

/* Activation of the feed-forward network. */
typedef enum { RA_ACT_GELU_ERF = 0, RA_ACT_RELU = 1, RA_ACT_GELU_TANH = 2 } ra_act;

/*
 * Ring attention forward (Section 3; Appendix A forward code), bf16.
 *   q, k, v  in   bf16 [B, S, H, D]
 *   o        out  bf16 [B, S, H, D]      softmax(q k^T / sqrt(D)) v, row by row
 *   lse      out  f32  [B, H, S]         log-sum-exp of each query's scaled scores
 *   n_hosts       number of virtual hosts of the ring; block c = S / n_hosts
 *   causal        0 or 1
 */
int ring_attn_fwd(const void* q, const void* k, const void* v, void* o, float* lse,
                  int B, int H, int S, int D, int n_hosts, int causal, hipStream_t stream);

/*
 * Ring attention backward (Appendix A backward code), bf16.
 *   q, k, v, o, lse   the forward inputs and outputs (o, lse as written by ring_attn_fwd)
 *   dO        in   bf16 [B, S, H, D]   upstream gradient of o
 *   dq, dk, dv out bf16 [B, S, H, D]   gradients of sum(dO * o); accumulated in float32
 *                                      (dq on the host, dk/dv with their rotating block)
 *                                      and rounded once at the end.
 */
int ring_attn_bwd(const void* q, const void* k, const void* v, const void* o, const float* lse,
                  const void* dO, void* dq, void* dk, void* dv,
                  int B, int H, int S, int D, int n_hosts, int causal, hipStream_t stream);

/*
 * Causal ring attention for any sequence length S >= 1 (Section 3: the sequence is cut into
 * one block per host; here the last blocks may be short or empty), bf16.  The block is
 * c = the smallest multiple of 128 with n_hosts * c >= S; the library stages q, k, v (and
 * o, lse, dO) into zero-padded workspace copies of length n_hosts * c, runs the ring on
 * them and copies the first S rows out.  Padded keys lie after every real query, so the
 * causal mask hides them; padded query rows add exactly zero to dK and dV.  Arguments,
 * layouts and outputs as ring_attn_fwd / ring_attn_bwd with causal = 1; S need not be a
 * multiple of n_hosts or of 128 (when n_hosts * c == S no copies are made).  Workspace:
 * 4 (forward) or 8 (backward) bf16 tensors [B, n_hosts * c, H, D] plus one float32
 * [B, H, n_hosts * c], stream-ordered.  Errors: RA_EINVAL for null pointers or
 * non-positive sizes, RA_EUNSUPPORTED when the padded shape is outside the supported set.
 */
int ring_attn_fwd_varlen(const void* q, const void* k, const void* v, void* o, float* lse,
                         int B, int H, int S, int D, int n_hosts, hipStream_t stream);
int ring_attn_bwd_varlen(const void* q, const void* k, const void* v, const void* o,
                         const float* lse, const void* dO, void* dq, void* dk, void* dv,
                         int B, int H, int S, int D, int n_hosts, hipStream_t stream);

/* float32 twins of ring_attn_fwd / ring_attn_bwd: every tensor is float32, products and
 * accumulation are float32 (no bf16 rounding anywhere). */
int ring_attn_fwd_f32(const float* q, const float* k, const float* v, float* o, float* lse,
                      int B, int H, int S, int D, int n_hosts, int causal, hipStream_t stream);
int ring_attn_bwd_f32(const float* q, const float* k, const float* v, const float* o,
                      const float* lse, const float* dO, float* dq, float* dk, float* dv,
                      int B, int H, int S, int D, int n_hosts, int causal, hipStream_t stream);

/*
 * One host's share of the ring (Section 3; the per-host view of Figure 2 and of the
 * Appendix A scan), bf16: query block `host_idx` against every key/value block, the
 * blocks arriving in ring order (host_idx - t) mod n_hosts, step 0 being the host's own
 * block, each later block prefetched into the host's receive buffer on the side stream.
 *   q_blk     in   bf16 [B, c, H, D]    query block host_idx (global positions host_idx*c + r)
 *   k_all, v_all in bf16 [B, S, H, D]   all key/value blocks, S = n_hosts * c
 *   o_blk     out  bf16 [B, c, H, D]
 *   lse_blk   out  f32  [B, H, c]
 */
int ring_attn_fwd_host(const void* q_blk, const void* k_all, const void* v_all, void* o_blk,
                       float* lse_blk, int B, int H, int S, int D, int n_hosts, int host_idx,
                       int causal, hipStream_t stream);

/*
 * One host's share of the ring backward (Appendix A backward code seen from host
 * host_idx), bf16: dq of query block host_idx, and this host's contribution to the float32
 * dK_j, dV_j that travel with every key/value block j.  Blocks arrive in ring order
 * (host_idx - t) mod n_hosts; from step 1 on, K_j, V_j and the gradients dK_j, dV_j they carry
 * are received into the host's double buffer on the side stream, the host adds its
 * contribution, and the gradients are passed on (copied out) -- three times the bytes of
 * the forward rotation.
 *   q_blk, o_blk, dO_blk  in  bf16 [B, c, H, D];  lse_blk in f32 [B, H, c] (ring_attn_fwd_host)
 *   k_all, v_all          in  bf16 [B, S, H, D]
 *   dq_blk                out bf16 [B, c, H, D]
 *   dk_acc, dv_acc        in/out f32 [B, S, H, D]: the gradients the blocks carry when they
 *                         reach this host; this host's contributions are added.
 */
int ring_attn_bwd_host(const void* q_blk, const void* k_all, const void* v_all, const void* o_blk,
                       const float* lse_blk, const void* dO_blk, void* dq_blk, float* dk_acc,
                       float* dv_acc, int B, int H, int S, int D, int n_hosts, int host_idx,
                       int causal, hipStream_t stream);

/*
 * Ring attention forward with an explicit block order, bf16 (checks the permutation
 * invariance that Section 3 relies on: blocks may be folded in any order).
 *   kv_order  HOST pointer, int[n_hosts * n_hosts]; row i is the sequence of key/value
 *             blocks host i folds in, a permutation of 0..n_hosts-1.  Copied before return.
 * Otherwise as ring_attn_fwd.  Returns RA_EINVAL if a row is not a permutation.
 */
int ring_attn_fwd_ordered(const void* q, const void* k, const void* v, void* o, float* lse,
                          int B, int H, int S, int D, int n_hosts, int causal,
                          const int* kv_order, hipStream_t stream);

/*
 * Ring decode (the paper's appendix on the inference requirement), bf16: the Tq newest
 * tokens attend to a key/value cache of S tokens that stays split in n_hosts blocks of
 * c = S / n_hosts over the ring.  The queries sit at global positions S - Tq .. S - 1
 * (their own keys and values are the last Tq rows of the cache) on the last host, and the
 * blocks are folded into their running maximum / numerator / denominator in ring order,
 * block n_hosts-1 first, then n_hosts-2, ..., 0 (Section 3), with the online-softmax
 * recurrence of Section 2.  With causal != 0 query t sees cache positions <= S - Tq + t;
 * otherwise the whole cache.  On one GPU all blocks are resident: one launch computes the
 * partial state of every block (each split in chunks, one wave per chunk; the step reads
 * the whole cache once and is bound by HBM bandwidth) and a second folds them in ring
 * order.
 *   q        in   bf16 [B, Tq, H, D]
 *   k_cache, v_cache in bf16 [B, S, H, D]
 *   o        out  bf16 [B, Tq, H, D]
 *   lse      out  f32  [B, H, Tq]      max + ln(denominator) of each query's scaled scores
 *   1 <= Tq <= min(32, S); D in {64, 128}; S % n_hosts == 0 and c a multiple of 32;
 *   n_hosts <= 64.  Workspace: B * H * (S / chunk) * Tq * (D + 2) floats, stream-ordered.
 */
int ring_attn_decode(const void* q, const void* k_cache, const void* v_cache, void* o, float* lse,
                     int B, int H, int S, int D, int Tq, int n_hosts, int causal,
                     hipStream_t stream);

/*
 * ring_attn_decode for callers that cannot allocate device memory: code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation.  Same arguments, same
 * kernels and the same result as ring_attn_decode, bit for bit, but no allocation of any
 * kind: the chunk partial states live in a fixed 32 MiB device array (8388608 floats) that
 * the library holds on every device it runs on until the process ends.  The call needs
 * B * H * nch * Tq * (D + 2) floats of it, with nch = S / kch chunks, kch = the block
 * S / n_hosts halved while B * H * nch < 4096 and the half stays a multiple of 32 (e.g.
 * B = 1, H = 32, D = 128, S = 262144 over 8 hosts: nch = 128, Tq <= 15); larger shapes
 * return RA_EUNSUPPORTED before anything is enqueued.  Every call on a device uses that
 * device's one array (nothing in it has to start at zero: each call writes every entry it
 * reads), so calls that overlap on one device -- on different streams, or from different
 * threads without ordering -- race and give wrong results; order them on one stream.
 */
int ring_attn_decode_noalloc(const void* q, const void* k_cache, const void* v_cache, void* o,
                             float* lse, int B, int H, int S, int D, int Tq, int n_hosts,
                             int causal, hipStream_t stream);

/*
 * Blockwise feed-forward network (Section 2 equation and "Blockwise Parallel
 * Transformers"; Algorithm 1's feed-forward step), bf16:
 *   y = act(x W1 + b1) W2 + b2, computed `block` rows at a time, so the [rows, d_ff]
 *   intermediate exists for one block only.
 *   x  in bf16 [T, d_model];  w1 in bf16 [d_model, d_ff];  b1 in bf16 [d_ff] or NULL
 *   w2 in bf16 [d_ff, d_model];  b2 in bf16 [d_model] or NULL;  y out bf16 [T, d_model]
 *   act: an ra_act value.   T % block == 0, block % 256 == 0, d_model % 256 == 0,
 *   d_ff % 256 == 0.
 */
int blockwise_ffn(const void* x, const void* w1, const void* b1, const void* w2, const void* b2,
                  void* y, int T, int d_model, int d_ff, int block, int act, hipStream_t stream);

/*
 * Backward of blockwise_ffn for upstream dy (bf16 [T, d_model]).  The pre-activation
 * x W1 + b1 is recomputed block by block (gradient checkpointing, Section 4 setting).
 *   dx  out bf16 [T, d_model]
 *   dw1 out f32 [d_model, d_ff], db1 out f32 [d_ff] (may be NULL),
 *   dw2 out f32 [d_ff, d_model], db2 out f32 [d_model] (may be NULL).
 * Weight and bias gradients are overwritten (not accumulated into) and kept in float32.
 */
int blockwise_ffn_bwd(const void* x, const void* w1, const void* b1, const void* w2,
                      const void* dy, void* dx, float* dw1, float* db1, float* dw2, float* db2,
                      int T, int d_model, int d_ff, int block, int act, hipStream_t stream);

/*
 * Per-block projection used by Algorithm 1 (query/key/value of each input block and the
 * output projection), bf16:  y = x W (+ residual).
 *   x in bf16 [T, d_in]; w in bf16 [d_in, d_out]; residual in bf16 [T, d_out] or NULL;
 *   y out bf16 [T, d_out].  T % block == 0, block % 256 == 0, d_in, d_out % 256 == 0.
 */
int blockwise_linear(const void* x, const void* w, const void* residual, void* y, int T,
                     int d_in, int d_out, int block, hipStream_t stream);

/* Backward of blockwise_linear without residual: dx = dy W^T (bf16 [T, d_in], may be
 * NULL), dw = x^T dy (f32 [d_in, d_out], overwritten). */
int blockwise_linear_bwd(const void* x, const void* w, const void* dy, void* dx, float* dw,
                         int T, int d_in, int d_out, int block, hipStream_t stream);

/*
 * One transformer layer as Algorithm 1 composes it, bf16, batch 1: the query, key and value
 * of each host's input block, ring attention over the n_hosts hosts, the output projection
 * with residual, and the blockwise feed-forward network on each host's block with residual:
 *     Q, K, V = X Wq, X Wk, X Wv;  A = RingAttention(Q, K, V);  Y = X + A Wo;
 *     Z = Y + act(Y W1) W2          (no biases, no normalisation, no positional encoding)
 *   x  in bf16 [S, d_model];  wq, wk, wv, wo in bf16 [d_model, d_model];
 *   w1 in bf16 [d_model, d_ff]; w2 in bf16 [d_ff, d_model];  z out bf16 [S, d_model]
 *   Heads: d_model = n_heads * D with D in {64, 128}; head h owns columns [h D, (h+1) D).
 *   The host block c = S / n_hosts (a multiple of 256) is also the projection / FFN block.
 */
int ring_layer_fwd(const void* x, const void* wq, const void* wk, const void* wv, const void* wo,
                   const void* w1, const void* w2, void* z, int S, int d_model, int n_heads,
                   int d_ff, int n_hosts, int causal, int act, hipStream_t stream);

/*
 * Backward of ring_layer_fwd for upstream dz (bf16 [S, d_model]).  Every activation is
 * recomputed from x (full gradient checkpointing, the paper's training setting).
 *   dx out bf16 [S, d_model]; dwq, dwk, dwv, dwo out f32 [d_model, d_model];
 *   dw1 out f32 [d_model, d_ff]; dw2 out f32 [d_ff, d_model] (overwritten).
 */
int ring_layer_bwd(const void* x, const void* wq, const void* wk, const void* wv, const void* wo,
                   const void* w1, const void* w2, const void* dz, void* dx, float* dwq, float* dwk,
                   float* dwv, float* dwo, float* dw1, float* dw2, int S, int d_model, int n_heads,
                   int d_ff, int n_hosts, int causal, int act, hipStream_t stream);

/*
 * LLaMA-style layer (the architecture the paper trains, Section 4 model configuration)
 * and its pieces.  The pieces are not defined by the paper; these entry points implement
 * the usual definitions, stated here:
 *   RMSNorm   y = x / sqrt(mean(x^2) + 1e-6) * g   (row-wise; gain g bf16 [d])
 *   RoPE      in each head, pair (2i, 2i+1) at global position p rotated by the angle
 *             p * 10000^(-2i/D)
 *   SwiGLU    (silu(x W1) * (x W3)) W2,  silu(u) = u / (1 + e^-u)
 *   layer     n1 = RMSNorm(x; g1);  h = x + Attn(RoPE(n1 Wq), RoPE(n1 Wk), n1 Wv) Wo;
 *             z = h + SwiGLU(RMSNorm(h; g2))
 * with Attn the ring attention of this library (causal by global position).
 */

/* RMSNorm forward.  x in bf16 [T, d]; g in bf16 [d]; y out bf16 [T, d]; rstd out f32 [T]
 * (1 / sqrt(mean(x^2) + eps)) or NULL.  d % 8 == 0, d <= 8192. */
int rms_norm_fwd(const void* x, const void* g, void* y, float* rstd, int T, int d, hipStream_t stream);

/* RMSNorm backward for upstream dy (f32 [T, d]): dx out bf16 [T, d] = dres + dx_norm (dres
 * bf16 [T, d] or NULL: a residual gradient added before the one rounding); dg out f32 [d]
 * (overwritten; summed over rows in a fixed order). */
int rms_norm_bwd(const void* x, const void* g, const float* dy, const void* dres, void* dx, float* dg,
                 int T, int d, hipStream_t stream);

/* Rotary position embedding in place on x bf16 [S, H, D] (rows at global positions
 * pos0 .. pos0 + S - 1); inverse = 1 applies the transpose (rotation by minus the angle),
 * which is the backward pass.  D % 4 == 0.  Angles are formed in double precision. */
int rope_apply(void* x, int S, int H, int D, int pos0, int inverse, hipStream_t stream);

/* SwiGLU feed-forward over row blocks of `block`:
 *   y = (silu(x W1) * (x W3)) W2 (+ residual)
 *   x in bf16 [T, d_model]; w1, w3 in bf16 [d_model, d_ff]; w2 in bf16 [d_ff, d_model];
 *   residual bf16 [T, d_model] or NULL; y out bf16 [T, d_model].  Shapes as blockwise_ffn. */
int swiglu_ffn(const void* x, const void* w1, const void* w3, const void* w2, const void* residual,
               void* y, int T, int d_model, int d_ff, int block, hipStream_t stream);

/* Backward of swiglu_ffn (no residual) for upstream dy bf16 [T, d_model], recomputing
 * x W1 and x W3 block by block: dx out bf16 [T, d_model]; dw1, dw3 out f32 [d_model, d_ff],
 * dw2 out f32 [d_ff, d_model] (overwritten). */
int swiglu_ffn_bwd(const void* x, const void* w1, const void* w3, const void* w2, const void* dy,
                   void* dx, float* dw1, float* dw3, float* dw2, int T, int d_model, int d_ff,
                   int block, hipStream_t stream);

/*
 * One LLaMA-style layer, forward (batch 1).
 *   x       in  bf16 [S, d_model]
 *   params  HOST array of 9 device pointers, in this order:
 *           g1 [d_model], wq, wk, wv, wo [d_model, d_model], g2 [d_model],
 *           w1, w3 [d_model, d_ff], w2 [d_ff, d_model]       (all bf16)
 *   z       out bf16 [S, d_model]
 * d_model = n_heads * D with D in {64, 128}, d_model <= 8192; S % n_hosts == 0; the host
 * block S / n_hosts (the projection and feed-forward block) and d_model, d_ff multiples of 256.
 */
int llama_layer_fwd(const void* x, const void* const* params, void* z, int S, int d_model,
                    int n_heads, int d_ff, int n_hosts, int causal, hipStream_t stream);

/*
 * Backward of llama_layer_fwd for upstream dz (bf16 [S, d_model]); the forward is
 * recomputed from x (full gradient checkpointing, the paper's training setting).
 *   dx     out bf16 [S, d_model]
 *   grads  HOST array of 9 device pointers (f32, overwritten) matching params:
 *          dg1, dwq, dwk, dwv, dwo, dg2, dw1, dw3, dw2
 */
int llama_layer_bwd(const void* x, const void* const* params, const void* dz, void* dx,
                    float* const* grads, int S, int d_model, int n_heads, int d_ff, int n_hosts,
                    int causal, hipStream_t stream);

/*
 * One training step of a stack of n_layers LLaMA-style layers: the forward pass keeps only
 * each layer's input, the backward pass runs the layers last to first, each recomputing
 * its own forward (the paper's full recomputation of attention and feed-forward).
 *   x       in  bf16 [S, d_model]
 *   params  HOST array of 9 * n_layers device pointers (layer l at params + 9 l, as above)
 *   dz      in  bf16 [S, d_model]: gradient of the loss with respect to the stack output
 *   z       out bf16 [S, d_model]: the stack output
 *   dx      out bf16 [S, d_model]
 *   grads   HOST array of 9 * n_layers device pointers (f32, overwritten)
 */
int llama_stack_train_step(const void* x, const void* const* params, const void* dz, void* z,
                           void* dx, float* const* grads, int n_layers, int S, int d_model,
                           int n_heads, int d_ff, int n_hosts, int causal, hipStream_t stream);

/* Description of the last error returned on the calling thread ("" if none).  Valid
 * until the next library call on that thread. */
const char* ring_attn_last_error(void);

/*
 * Return the cached workspace of the current device's library pool to the driver
 * (hipMemPoolTrimTo to zero bytes).  Memory still in use by calls whose stream has not
 * reached the end of the call stays allocated.  Not part of the method.  Returns RA_OK,
 * or RA_EHIP if the pool cannot be created or trimmed.
 */
int ring_attn_release_workspace(void);

/*
 * Kernel timing for benchmarks and profiling (not part of the method).
 * ring_attn_timing_enable(1) makes every later launch of the library's hot kernels be
 * bracketed by timing events on the stream it runs on; ring_attn_timing_read(kind, ...)
 * waits for the recorded launches of that kind, returns their summed duration in
 * milliseconds and their number, and forgets them.  Kinds:
 */
enum { RA_KERNEL_ATTN_FWD = 0, RA_KERNEL_ATTN_BWD = 1, RA_KERNEL_GEMM = 2, RA_KERNEL_DECODE = 3 };
void ring_attn_timing_enable(int on);
int ring_attn_timing_read(int kind, double* total_ms, int* launches);

/*
 * Matrix-core calibration for benchmarks (not part of the method): launches 512
 * workgroups of 256 threads (two waves per SIMD on 256 compute units); every wave issues
 * iters x 32 bf16 32x32x16 matrix products (4 independent accumulator chains) and writes
 * one float to sink[wave].  The caller times the launch on `stream`: the work is
 * 2048 * iters * 32 * 32768 flop.
 *   iters            in [1, 2^20] (else RA_EINVAL)
 *   random_operands  0: the same two operands in every product (the headline rate);
 *                    1: random signs and mantissas (magnitudes in [0.5, 8)) that change
 *                    from one product to the next, as real data does (else RA_EINVAL)
 *   sink             device float[2048], overwritten
 */
int ring_attn_mfma_probe(int iters, int random_operands, float* sink, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* RINGATTN_H */
