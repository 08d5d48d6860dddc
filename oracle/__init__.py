"""Plain fp64 CPU oracle for fused RoPE + masked attention (AttnFuse, arXiv 2609.13612).

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import, call or
execute anything in this package: only ``tests/``, ``__graft_entry__.smoke()``
and the ``cpu_baseline`` leg of ``bench.py`` use it.  It shares no code, header,
table or constant generator with the HIP path; it consumes plain numpy arrays
and imports nothing but numpy.

What it computes is the plain definition of the method, written out in fp64
with the full score matrix materialised per (batch, head):

    O = softmax(mask(scale * R(Q) R(K)^T + bias)) V,     LSE = m + ln(l)

* The online-softmax recurrence the kernels use is exact (Section 2,
  "FlashAttention and online softmax"), so the definition is the oracle.
* RoPE is the pre-matmul rotation (Section 2 "Rotary Position Embeddings",
  Section 4.1 "Fused RoPE").
* Masks, ALiBi and a dense additive bias are the post-matmul modifications
  (Section 3.1, the list of ten combinators); relu attention replaces the
  softmax (the same list).
* The backward follows the FlashAttention-2 equations; the forward keeps one
  scalar per row, L = m + log l (Section 4.4 "Backward Pass").
* Decode (one query per sequence against a key/value cache, Section 4.2 "Flash
  Decoding") is the same definition for that single row: ``decode_forward``.

Every function is pinned by ``tests/test_oracle_*.py`` against invariants,
closed forms, an independent brute force, finite differences and library
special cases.  No function here is "parity unpinned".
"""
from .rope import (
    ROPE_NONE,
    ROPE_NEOX,
    ROPE_INTERLEAVED,
    ROPE_KINDS,
    rope_frequencies,
    rope_pair_indices,
    rope_rotate,
)
from .attention import (
    MASK_NONE,
    MASK_CAUSAL,
    MASK_SLIDING_WINDOW,
    MASK_KINDS,
    NORM_SOFTMAX,
    NORM_RELU,
    NORM_KINDS,
    visibility,
    block_visible,
    attention_scores,
    attention_probs,
    attention_forward,
    attention_backward,
    attention_forward_rows,
)
from .decode import decode_forward

__all__ = [
    "ROPE_NONE", "ROPE_NEOX", "ROPE_INTERLEAVED", "ROPE_KINDS",
    "rope_frequencies", "rope_pair_indices", "rope_rotate",
    "MASK_NONE", "MASK_CAUSAL", "MASK_SLIDING_WINDOW", "MASK_KINDS",
    "visibility", "block_visible", "attention_scores", "attention_probs",
    "attention_forward", "attention_backward", "attention_forward_rows",
    "decode_forward",
]
