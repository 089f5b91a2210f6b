"""Arithmetic intensity between hosts (oracle; test infrastructure only).

Section 3 ("Arithmetic Intensity Between Hosts", "Memory Requirement") sizes the ring's
block so that a step's attention work hides the transfer of the next key/value block:

  * one step of host i against one block of c tokens (hidden size d) costs 2 d c^2
    flops for the scores q k^T and 2 d c^2 for the weighted sum with v: 4 d c^2;
  * the key and value blocks it passes on are c x d bf16 values each, 2 c d bytes
    apiece: 4 c d bytes;
  * the transfer hides under the work when 4 d c^2 / F >= 4 c d / B for a host with F
    flop/s and a link of B bytes/s one way, i.e. c >= F / B (independent of d);
  * a host stores six blocks (query, key, value, the two receive blocks, output), so the
    smallest sequence per host is s = 6 c.

The HIP library does not compute these; they fix the block size a multi-GPU ring would
use, and the tests pin them to the paper's table of minimal block size and sequence
length per device (tests/golden/min_block_size_table.txt).
"""


def step_flops(c, d):
    """Flops of one ring step of one host against one block: 4 d c^2."""
    return 4.0 * d * c * c


def step_bytes(c, d):
    """Bytes of the key and value blocks a host passes on per step (bf16): 4 c d."""
    return 4.0 * c * d


def min_block_size(flops, bandwidth):
    """Smallest block c (tokens) with step_flops(c, d) / flops >= step_bytes(c, d) / bandwidth."""
    return flops / bandwidth


def min_seq_len(flops, bandwidth):
    """Smallest sequence per host: six blocks of the minimal size."""
    return 6.0 * min_block_size(flops, bandwidth)
