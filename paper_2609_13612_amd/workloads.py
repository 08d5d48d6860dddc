"""Named workload shapes and their algorithmic FLOP / byte counts.

The five prefill workloads are the parity and benchmark shapes of the build,
the three decode workloads are the cache geometries of the paper's decode
table (batch 1, which the table leaves unstated), and the block-sparse
workload is the paper's BigBird case (N = 4096) on the GPT-2-small heads of
its Ampere comparisons; inputs are seeded N(0, 1) tensors (see ``inputs``).  FLOPs count only visible
(query, key) pairs: 4*D per pair for the forward (Q K^T and P V) and 10*D for
the backward (five matmuls: S, dV, dP, dQ, dK), the FlashAttention convention.
The separate rotation moves 4 bytes per bf16 element of Q and K (read + write).
"""
from dataclasses import dataclass, field


@dataclass(frozen=True)
class Workload:
    name: str
    B: int
    H: int
    Hkv: int
    S: int
    D: int
    rope: str = "neox"
    theta: float = 10000.0
    mask: str = "causal"
    window: int = 0
    alibi: bool = False
    dtype: str = "bf16"
    backward: bool = False
    notes: str = field(default="", compare=False)

    def visible_pairs(self, S=None):
        """Visible (query, key) pairs per (batch, head)."""
        S = self.S if S is None else S
        if self.mask == "none":
            return S * S
        if self.mask == "causal":
            return S * (S + 1) // 2
        W = self.window
        # rows i < W see i+1 keys, the rest see W keys
        w = min(W, S)
        return w * (w + 1) // 2 + (S - w) * W

    def fwd_flops(self, S=None):
        return 4 * self.D * self.B * self.H * self.visible_pairs(S)

    def bwd_flops(self, S=None):
        return 10 * self.D * self.B * self.H * self.visible_pairs(S)

    def rope_bytes(self, S=None):
        S = self.S if S is None else S
        return 4 * self.B * (self.H + self.Hkv) * S * self.D


WORKLOADS = {
    "rope_causal_tiny": Workload("rope_causal_tiny", 1, 2, 2, 128, 64, rope="interleaved",
                                 notes="fp32 and bf16 parity case; interleaved pairs"),
    "rope_causal_b8h16s2048d64": Workload("rope_causal_b8h16s2048d64", 8, 16, 16, 2048, 64,
                                          notes="fused and separate-RoPE forward"),
    "rope_swa1024_b4h32kv8s8192d128": Workload("rope_swa1024_b4h32kv8s8192d128", 4, 32, 8, 8192, 128,
                                               mask="sliding_window", window=1024, notes="GQA, forward only"),
    "alibi_causal_b4h16s4096d128": Workload("alibi_causal_b4h16s4096d128", 4, 16, 16, 4096, 128, rope="none",
                                            alibi=True, notes="post-matmul modification only"),
    "llama3_8b_b1h32kv8s8192d128": Workload("llama3_8b_b1h32kv8s8192d128", 1, 32, 8, 8192, 128, theta=500000.0,
                                            backward=True, notes="Llama-3-8B attention layer, fwd + bwd"),
}

LLAMA_SWEEP_S = (1024, 1536, 2048, 2560, 3072, 4096, 6144, 8192, 16384)


@dataclass(frozen=True)
class DecodeWorkload:
    """One query per sequence against a key/value cache of S_kv tokens
    (the paper's decode table: Q.N = 1, large cache)."""
    name: str
    B: int
    H: int
    Hkv: int
    S_kv: int
    D: int
    rope: str = "neox"
    theta: float = 10000.0
    notes: str = field(default="", compare=False)

    def cache_bytes(self):
        """K and V cache bytes read once (bf16), the kernel's algorithmic traffic
        with the query, output and LSE (negligible) left out."""
        return 2 * 2 * self.B * self.Hkv * self.S_kv * self.D

    def flops(self):
        """4*D per (query head, cached key), as for the forward."""
        return 4 * self.D * self.B * self.H * self.S_kv


DECODE_WORKLOADS = {
    "decode_llama3_8b_h32kv8_cache4096": DecodeWorkload("decode_llama3_8b_h32kv8_cache4096", 1, 32, 8, 4096, 128,
                                                        theta=500000.0, notes="Llama-3-8B geometry"),
    "decode_llama3_70b_h64kv8_cache32768": DecodeWorkload("decode_llama3_70b_h64kv8_cache32768", 1, 64, 8, 32768,
                                                          128, theta=500000.0, notes="Llama-3-70B geometry"),
    "decode_mistral_7b_h32kv8_cache16384": DecodeWorkload("decode_mistral_7b_h32kv8_cache16384", 1, 32, 8, 16384,
                                                          128, notes="Mistral-7B geometry"),
}


@dataclass(frozen=True)
class SparseWorkload:
    """Block-sparse attention with a BigBird-style block mask (64-position
    blocks: a band of ``window`` blocks, ``n_global`` global blocks and
    ``n_random`` random blocks per block row, drawn with ``mask_seed``)."""
    name: str
    B: int
    H: int
    Hkv: int
    S: int
    D: int
    window: int = 3
    n_global: int = 1
    n_random: int = 1
    mask_seed: int = 0
    notes: str = field(default="", compare=False)

    def active(self):
        from . import inputs
        return inputs.bigbird_blocks((self.S + 63) // 64, window=self.window, n_global=self.n_global,
                                     n_random=self.n_random, seed=self.mask_seed)

    def visible_pairs(self, active=None):
        """Visible (query, key) pairs per (batch, head): every active block
        contributes its rows times its columns (the last block may be short)."""
        import numpy as np
        active = self.active() if active is None else active
        nb = active.shape[0]
        size = np.full(nb, 64)
        size[-1] = self.S - 64 * (nb - 1)
        return int((size[:, None] * size[None, :] * active).sum())

    def fwd_flops(self, active=None):
        return 4 * self.D * self.B * self.H * self.visible_pairs(active)

    def bwd_flops(self, active=None):
        return 10 * self.D * self.B * self.H * self.visible_pairs(active)


SPARSE_WORKLOADS = {
    "bigbird_b4h12s4096d64": SparseWorkload("bigbird_b4h12s4096d64", 4, 12, 12, 4096, 64,
                                            notes="BigBird-style mask at N = 4096, GPT-2-small heads, no RoPE"),
}
