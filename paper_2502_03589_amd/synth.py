"""Seeded synthetic inputs shared by the tests, the benchmark and the oracle checks.

This module holds no arithmetic of the method: it only draws fp16 tensors,
sequence lengths and page tables from named, seeded NumPy streams, and
describes the five synthetic workloads (shapes, bit-widths, partition sizes).
Every consumer (HIP path, oracle) receives the same arrays.

The workloads stand in for the paper's datasets (Sec. 7.1, dataset table):
prompt lengths of 256 (short prompts), 4K/8K (arXiv-like) and 1K..32K
(Cocktail-like), plus a 128K long-context case; N(0,1) fp16 values stand in
for real activations because no trained weights are used.
"""
from __future__ import annotations

import dataclasses
from typing import Optional

import numpy as np

# Sub-stream identifiers: each named quantity gets its own SeedSequence child so
# that changing one shape never changes another quantity's values.
_STREAMS = {
    "q": 1, "k": 2, "v": 3, "lens": 4, "outlier": 5,
    "step_k": 6, "step_v": 7, "pages": 8, "p_codes": 9, "misc": 10,
}


def rng_for(seed: int, name: str, sub: int = 0) -> np.random.Generator:
    """Generator for the named sub-stream `name` (optionally indexed by `sub`)."""
    return np.random.default_rng(np.random.SeedSequence(seed, spawn_key=(_STREAMS[name], sub)))


def normal_f16(seed: int, name: str, shape, sub: int = 0) -> np.ndarray:
    """N(0,1) drawn in float32 and rounded to float16."""
    g = rng_for(seed, name, sub)
    return g.standard_normal(shape, dtype=np.float32).astype(np.float16)


def outlier_channels(seed: int, head_dim: int, count: int) -> np.ndarray:
    """`count` distinct K channels (drawn once, shared by every batch/head/token)."""
    g = rng_for(seed, "outlier")
    return np.sort(g.choice(head_dim, size=count, replace=False))


def scale_channels_f16(x: np.ndarray, channels: np.ndarray, factor: float) -> np.ndarray:
    """Multiply the given last-axis channels by `factor` (done in float32, rounded to fp16)."""
    y = x.astype(np.float32)
    y[..., channels] *= np.float32(factor)
    return y.astype(np.float16)


def uniform_lengths(seed: int, batch: int, lo: int, hi: int) -> np.ndarray:
    """Per-request context lengths drawn uniformly from the integers [lo, hi]."""
    g = rng_for(seed, "lens")
    return g.integers(lo, hi + 1, size=batch, dtype=np.int64).astype(np.int32)


def page_table(seed: int, lens: np.ndarray, page_tokens: int, spare_pages: int = 0):
    """Block table for a paged cache: each sequence gets ceil(len/page) pages
    (plus `spare_pages` for appends) taken from a seeded permutation of the pool.

    Returns (block_table int32 [B][max_blocks], num_pages)."""
    need = [(int(n) + spare_pages * page_tokens + page_tokens - 1) // page_tokens for n in lens]
    need = [max(1, x) for x in need]
    total = int(sum(need))
    perm = rng_for(seed, "pages").permutation(total).astype(np.int32)
    maxb = max(need)
    table = np.full((len(lens), maxb), -1, dtype=np.int32)
    pos = 0
    for b, nb in enumerate(need):
        table[b, :nb] = perm[pos:pos + nb]
        pos += nb
    return table, total


@dataclasses.dataclass(frozen=True)
class Workload:
    """One synthetic configuration (shapes and quantization parameters)."""
    name: str
    batch: int
    q_heads: int
    kv_heads: int
    head_dim: int
    kv_bits: int
    partition: int
    qp_bits: int = 8
    context: int = 0                 # uniform context length (decode) / prompt length (prefill)
    len_range: Optional[tuple] = None  # (lo, hi) for ragged contexts
    page_tokens: int = 0             # 0 = contiguous cache
    outlier_channels: int = 0
    outlier_factor: float = 1.0
    causal: bool = False
    steps: int = 0                   # appended tokens (quantize-on-write workload)
    seed: int = 0

    @property
    def group(self) -> int:
        return self.q_heads // self.kv_heads


WORKLOADS = {
    # single decode step: 1 q head, 1 kv head, d=128, L=256, 2-bit KV, partition 32
    "decode_tiny_l256": Workload("decode_tiny_l256", 1, 1, 1, 128, 2, 32, context=256, seed=1001),
    # Llama-3-8B-shaped decode: B=16, 32/8 heads, L=4096, 4 outlier K channels x10, 2-bit, partition 32
    "decode_llama8b_l4096": Workload("decode_llama8b_l4096", 16, 32, 8, 128, 2, 32, context=4096,
                                     outlier_channels=4, outlier_factor=10.0, seed=1002),
    # causal prefill: B=1, 32/8 heads, L=8192, 4-bit K/V, partition 64, 8-bit Q/P
    "prefill_l8192": Workload("prefill_l8192", 1, 32, 8, 128, 4, 64, context=8192, causal=True, seed=1003),
    # 70B-shaped one-GPU share: B=64, 64/8 heads, L ~ U[1024, 32768], 256-token pages
    "decode_70b_ragged": Workload("decode_70b_ragged", 64, 64, 8, 128, 2, 32, len_range=(1024, 32768),
                                  page_tokens=256, seed=1004),
    # long context: B=4, 32/8 heads, L=131072, append 1 token/step for 64 steps
    "decode_long_l131072": Workload("decode_long_l131072", 4, 32, 8, 128, 2, 32, context=131072,
                                    steps=64, seed=1005),
}
