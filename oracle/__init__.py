"""CPU oracle for the ring-attention hot path: TEST INFRASTRUCTURE ONLY.

A plain, slow, float64 implementation (NumPy, and plain PyTorch CPU operations where the
work is large) of what the HIP library computes, written
from the paper (Liu, Zaharia, Abbeel, "Ring Attention with Blockwise Transformers for
Near-Infinite Context", arXiv 2310.01889).  Only the test suite, the smoke check in
``__graft_entry__.py`` and the ``cpu_baseline`` leg of ``bench.py`` may import it; the
product path (``paper_2310_01889_amd``) never does, and shares no code with it.

Modules
  attention  -- exact softmax attention from its definition (Section 2 equation),
                forward and backward, materialising the score matrix (row-chunked).
  ring       -- the ring schedule of Section 3 / Appendix A: N virtual hosts, each
                holding one query block; key/value blocks (and, in the backward pass,
                their gradients) are physically rotated host i -> host i+1 after
                every step, and each block is folded in with running max /
                numerator / denominator statistics, tile by tile.
  brute      -- scalar triple loops (no BLAS) for tiny shapes.
  ffn        -- position-wise feed-forward network (Section 2 equation) with the
                activations used here (GeLU-erf, ReLU, GeLU-tanh), its blockwise
                form (Section 2, "Blockwise Parallel Transformers"), and the
                projection ``y = x w (+ residual)``; forward and backward.
  decode     -- ring decode (the paper's appendix on inference): a few query tokens
                at the end of a long key/value cache that is split in host blocks; the
                blocks circulate past the queries in ring order and are folded into
                their running softmax state.
  llama      -- the LLaMA-style layer the paper trains (RMSNorm, rotary position
                embedding, SwiGLU feed-forward, pre-norm residuals) around the same
                attention, its backward, and a stack of layers trained with full
                recomputation.
  layer      -- one transformer layer as Algorithm 1 composes it: projections,
                ring attention, output projection with residual, blockwise FFN with
                residual; forward and backward.
  overlap    -- Section 3's arithmetic intensity between hosts: the block size at which
                a ring step's attention work hides the key/value transfer (c >= F/B) and
                the minimal sequence per host (6c).

Every function takes and returns float64 arrays.  Inputs in bf16 are passed in already
rounded (the exact values the GPU sees), then upcast.

Parity status: attention forward/backward, ring bookkeeping, ring decode, FFN and the overlap
condition (against the paper's printed table, tests/golden/) are pinned by the
tests in tests/test_oracle_*.py (closed forms, invariants, brute force, finite
differences, library routines).  The two layer compositions (``layer``: the paper fixes
neither norms, biases nor the activation of that layer; ``llama``: the LLaMA architecture
around the attention) are readings of the paper: the code is pinned to each reading by a
restatement in torch library routines with autograd for every gradient and by finite
differences, ``layer`` also by the closed form of zero query and key weights, and each of
their parts has its own pins.
"""
