"""Seeded random draws for the link-step workloads.

Every array is a pure function of (seed, identity of the thing drawn), so the
oracle and the GPU harness can each ask for exactly the rows they need and get
identical values.  Values are drawn in float32 from N(0, 1), multiplied by a
scale, and rounded to bfloat16 with round-to-nearest-even; arrays of bfloat16
are carried as uint16 bit patterns.

Identities:
  * chunk cache   : (seed, "chunk", layer, chunk id)  -> K then V, [L, Hkv, D]
  * recomputed row: (seed, "row", request, linked position) -> q [Hq, D], k, v [Hkv, D]
  * token         : (seed, "tok", kind, owner, index) -> embedding [hidden] (fp32)
                    kind 0 = token ``index`` of chunk ``owner``,
                    kind 1 = suffix token ``index`` of request ``owner``,
                    kind 2 = the dummy token (owner 0, index 0)
  * weights       : (seed, "w", layer, tensor id)
"""
from __future__ import annotations

from concurrent.futures import ThreadPoolExecutor
from typing import Dict, Sequence, Tuple

import numpy as np

_CHUNK, _ROW, _TOK, _W, _MAT = 1, 2, 3, 4, 5


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 to bfloat16 (nearest, ties to even); returns uint16 bit patterns."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    r = (u + (np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1)))) >> np.uint32(16)
    return r.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """Exact widening of bfloat16 bit patterns to float32."""
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def _normal_bf16(rng: np.random.Generator, shape, scale: float) -> np.ndarray:
    x = rng.standard_normal(size=shape, dtype=np.float32)
    if scale != 1.0:
        x *= np.float32(scale)
    return f32_to_bf16_bits(x)


def chunk_cache(seed: int, chunk_id: int, length: int, hkv: int, d: int,
                scale: float = 1.0, layer: int = 0, qk_scale: float = 1.0) -> Tuple[np.ndarray, np.ndarray]:
    """Cached K and V of one immutable chunk, bf16 bits [length, hkv, d] each.
    K is N(0, 1) * scale * qk_scale, V is N(0, 1) * scale."""
    rng = np.random.default_rng([seed, _CHUNK, layer, chunk_id])
    k = _normal_bf16(rng, (length, hkv, d), scale * qk_scale)
    v = _normal_bf16(rng, (length, hkv, d), scale)
    return k, v


def row_qkv(seed: int, request: int, positions: Sequence[int], hq: int, hkv: int, d: int,
            scale: float = 1.0, qk_scale: float = 1.0) -> Tuple[np.ndarray, np.ndarray, np.ndarray]:
    """q [n, hq, d], k [n, hkv, d], v [n, hkv, d] (bf16 bits) for the given linked positions;
    q and k are N(0, 1) * scale * qk_scale, v is N(0, 1) * scale."""
    n = len(positions)
    q = np.empty((n, hq, d), np.uint16)
    k = np.empty((n, hkv, d), np.uint16)
    v = np.empty((n, hkv, d), np.uint16)
    for i, p in enumerate(positions):
        rng = np.random.default_rng([seed, _ROW, request, int(p)])
        q[i] = _normal_bf16(rng, (hq, d), scale * qk_scale)
        k[i] = _normal_bf16(rng, (hkv, d), scale * qk_scale)
        v[i] = _normal_bf16(rng, (hkv, d), scale)
    return q, k, v


def token_embeddings(seed: int, kind: int, owner: int, indices: Sequence[int], hidden: int) -> np.ndarray:
    """fp32 [n, hidden] embeddings, N(0, 1); kind 0 = chunk token, kind 1 = suffix token."""
    out = np.empty((len(indices), hidden), np.float32)
    for i, t in enumerate(indices):
        rng = np.random.default_rng([seed, _TOK, kind, owner, int(t)])
        out[i] = rng.standard_normal(size=hidden, dtype=np.float32)
    return out


def dummy_embeddings(seed: int, n_dummy: int, hidden: int) -> np.ndarray:
    """fp32 [n_dummy, hidden]: n_dummy copies of one dummy token's embedding (a
    begin-of-sequence-like token prepended to every chunk at compile)."""
    if n_dummy <= 0:
        return np.zeros((0, hidden), np.float32)
    return np.repeat(token_embeddings(seed, 2, 0, [0], hidden), n_dummy, axis=0)


# tensor ids inside one layer
W_ATTN_NORM, W_QKV, W_O, W_MLP_NORM, W_GATE_UP, W_DOWN, W_FINAL_NORM = range(7)


_SLAB_ROWS = 512      # linear weights are drawn in slabs of this many rows, one stream each


def _weight_slab(seed: int, layer: int, tid: int, shape, fan_in: int, slab: int) -> np.ndarray:
    rng = np.random.default_rng([seed, _W, layer, tid, slab])
    rows = min(_SLAB_ROWS, shape[0] - slab * _SLAB_ROWS)
    return _normal_bf16(rng, (rows, shape[1]), 0.5 / np.sqrt(fan_in))


def _norm_weight(seed: int, layer: int, tid: int, n: int) -> np.ndarray:
    rng = np.random.default_rng([seed, _W, layer, tid])
    x = np.float32(1.0) + np.float32(0.1) * rng.standard_normal(size=n, dtype=np.float32)
    return f32_to_bf16_bits(x)


def model_weights(seed: int, layer: int, hidden: int, ffn: int, hq: int, hkv: int, d: int,
                  threads: int = 1) -> Dict[str, np.ndarray]:
    """bf16-bit weights of one decoder layer in [out, in] layout.

    wqkv rows: [Hq*d query | Hkv*d key | Hkv*d value]; w_gate_up rows: [ffn gate | ffn up].
    Linear weights are N(0, (0.5/sqrt(fan_in))^2), drawn in slabs of 512 rows with one
    random stream per slab (so they can be drawn in parallel); norm weights 1 + 0.1*N(0, 1).
    """
    linear = {"wqkv": (W_QKV, ((hq + 2 * hkv) * d, hidden), hidden),
              "wo": (W_O, (hidden, hq * d), hq * d),
              "w_gate_up": (W_GATE_UP, (2 * ffn, hidden), hidden),
              "w_down": (W_DOWN, (hidden, ffn), ffn)}
    out = {"attn_norm": _norm_weight(seed, layer, W_ATTN_NORM, hidden),
           "mlp_norm": _norm_weight(seed, layer, W_MLP_NORM, hidden)}
    for name, (_, shape, _) in linear.items():
        out[name] = np.empty(shape, np.uint16)
    jobs = [(name, slab) for name, (_, shape, _) in linear.items()
            for slab in range(-(-shape[0] // _SLAB_ROWS))]

    def fill(job):
        name, slab = job
        tid, shape, fan_in = linear[name]
        out[name][slab * _SLAB_ROWS:(slab + 1) * _SLAB_ROWS] = _weight_slab(seed, layer, tid, shape, fan_in, slab)

    if threads <= 1:
        for job in jobs:
            fill(job)
    else:
        with ThreadPoolExecutor(threads) as ex:
            list(ex.map(fill, jobs))
    return {k: out[k] for k in ("attn_norm", "wqkv", "wo", "mlp_norm", "w_gate_up", "w_down")}


def final_norm_weight(seed: int, hidden: int) -> np.ndarray:
    return _norm_weight(seed, 1 << 20, W_FINAL_NORM, hidden)


def matrix_bf16(seed: int, tag: int, shape, scale: float = 1.0) -> np.ndarray:
    """A seeded N(0, 1) * scale matrix as bf16 bits (operands of stand-alone projection cases)."""
    rng = np.random.default_rng([seed, _MAT, tag])
    return _normal_bf16(rng, shape, scale)


def matrix_f32(seed: int, tag: int, shape, scale: float = 1.0) -> np.ndarray:
    """A seeded N(0, 1) * scale float32 matrix (e.g. a residual stream fed to a projection)."""
    rng = np.random.default_rng([seed, _MAT, tag])
    x = rng.standard_normal(size=shape, dtype=np.float32)
    return x * np.float32(scale)
