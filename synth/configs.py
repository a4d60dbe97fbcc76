"""Workload shapes for the link step, one entry per evaluated configuration.

The shapes stand in for the paper's workloads (Sec. 5.2): documents or
few-shot examples become immutable chunks, the user query becomes the mutable
suffix; Sec. 5.6 fixes 512-token chunks for the long-context sweep and Sec. 5.5
uses LegoLink-16 with vLLM's 16-token KV blocks.  The datasets themselves are
not used: all values are i.i.d. normal draws (see ``gen``).
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Optional

SEED_BASE = 2410153320


@dataclass(frozen=True)
class AttnWorkload:
    """One attention layer of the link step (q, k, v of the recomputed rows are given)."""

    name: str
    seed: int
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    block_size: int
    # requests: each is a list of chunk ids (into the chunk pool) plus a suffix length
    requests: List[List[int]]
    chunk_lens: List[int]            # length of every chunk in the pool
    suffix_lens: List[int]           # per request
    k: int                           # LegoLink-k; k < 0 = recompute every token (FR)
    value_scale: float = 1.0         # values are N(0,1) * value_scale
    qk_scale: float = 1.0            # queries and keys additionally scaled by this

    @property
    def batch(self) -> int:
        return len(self.requests)

    def linked_len(self, r: int) -> int:
        return sum(self.chunk_lens[c] for c in self.requests[r]) + self.suffix_lens[r]


@dataclass(frozen=True)
class ModelWorkload:
    """Full decoder stack (Llama-style) link step on one request."""

    name: str
    seed: int
    n_layers: int
    hidden: int
    ffn: int
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    block_size: int
    rope_theta: float
    rms_eps: float
    chunk_lens: List[int]
    suffix_len: int
    k: int

    @property
    def linked_len(self) -> int:
        return sum(self.chunk_lens) + self.suffix_len


def _pool_requests(seed: int, n_req: int, per_req: int, pool: int) -> List[List[int]]:
    import numpy as np

    rng = np.random.default_rng([seed, 7])
    return [list(map(int, rng.permutation(pool)[:per_req])) for _ in range(n_req)]


def c1() -> AttnWorkload:
    """4 chunks x 128 tokens, MHA 8 heads, d=64, k=4, 16 suffix tokens, values N(0,1)*0.5."""
    return AttnWorkload("c1_mha8_d64_4x128_k4", SEED_BASE + 0, 8, 8, 64, 16,
                        [[0, 1, 2, 3]], [128] * 4, [16], 4, 0.5)


def c2() -> AttnWorkload:
    """One Llama-3-8B-shaped attention layer: 10 chunks x 512, GQA 32/8, d=128, k=16, 64 suffix."""
    return AttnWorkload("c2_gqa32x8_d128_10x512_k16", SEED_BASE + 1, 32, 8, 128, 16,
                        [list(range(10))], [512] * 10, [64], 16)


def c3(n_layers: int = 32, n_chunks: int = 20, chunk_len: int = 1024, k: int = 32,
       suffix: int = 128, hidden: int = 4096, ffn: int = 14336, hq: int = 32, hkv: int = 8,
       d: int = 128) -> ModelWorkload:
    """Llama-3-8B-shaped 32-layer link step: 20 chunks x 1024 compiled at 0..1023, k=32, 128 suffix."""
    name = f"c3_llama8b_L{n_layers}_{n_chunks}x{chunk_len}_k{k}_q{suffix}"
    return ModelWorkload(name, SEED_BASE + 2, n_layers, hidden, ffn, hq, hkv, d, 16,
                         500000.0, 1e-5, [chunk_len] * n_chunks, suffix, k)


def c4() -> AttnWorkload:
    """32 requests x 8 distinct chunks of 2000 from a pool of 64, k=32, 128 suffix, GQA 32/8."""
    seed = SEED_BASE + 3
    return AttnWorkload("c4_serving_32req_8x2000_pool64_k32", seed, 32, 8, 128, 16,
                        _pool_requests(seed, 32, 8, 64), [2000] * 64, [128] * 32, 32)


def c5(k: int = 32) -> AttnWorkload:
    """64 chunks x 2048 = 131072 linked tokens + 256 suffix, GQA 32/8, d=128; k in {0,4,32,-1}."""
    tag = "all" if k < 0 else str(k)
    return AttnWorkload(f"c5_long_64x2048_k{tag}", SEED_BASE + 4, 32, 8, 128, 16,
                        [list(range(64))], [2048] * 64, [256], k)


CONFIGS = {"c1": c1, "c2": c2, "c3": c3, "c4": c4, "c5": c5}


def get_config(name: str, **kw):
    return CONFIGS[name](**kw)
