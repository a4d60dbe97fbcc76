"""Model-level link step and compile step, for Llama-style decoders.

Sec. 4.2 gives the per-layer recipe for the selected rows: project the k'
hidden rows to Q, K, V, place K and V among the cached vectors of the other
tokens, attend with the causal MASK, and apply W_O.  The rest of the layer is
the model's own (Sec. 5.1 evaluates Llama / Mistral / Yi decoders), which the
paper does not restate; this oracle uses the standard Llama layer: pre-norm
RMSNorm, rotary embedding with the "rotate half" pairing (i, i + d/2) and
inverse frequencies theta^(-2i/d), grouped-query attention, SwiGLU MLP, final
RMSNorm.  No LM head (the link step ends at the last hidden state).

The compile step (Sec. 2.2) runs one chunk alone through the same model with
positions 0..L-1 and keeps each layer's K and V; LegoLink-0 (Sec. 5.4) runs
dummy tokens plus the chunk and keeps the chunk's K and V only.

Precision reading: weights, KV caches and the activations fed to a weight
matrix are bf16; everything else is float64 here.  With ``bf16_storage`` the
oracle rounds (round-to-nearest-even, via float32) exactly where a value is
stored as bf16: the normalised activations entering a projection, q/k/v after
the rotation, the attention output entering W_O and the SwiGLU product
entering W_down.  The residual stream is never rounded.
"""
from __future__ import annotations

from typing import Dict, List, Sequence, Tuple

import numpy as np

from .link import _round_bf16, expand_kv, legolink_positions, masked_attention, rerotate_cached, rope  # noqa: F401


def _bf16_to_f64(bits: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bit patterns to float64 (a multi-threaded library cast)."""
    import torch

    b = np.ascontiguousarray(bits, dtype=np.uint16).view(np.int16)
    return torch.from_numpy(b).view(torch.bfloat16).to(torch.float64).numpy()


def rmsnorm(x: np.ndarray, w: np.ndarray, eps: float) -> np.ndarray:
    """x / sqrt(mean(x^2) + eps) * w, row-wise."""
    return x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps) * w


def _silu(x: np.ndarray) -> np.ndarray:
    return x / (1.0 + np.exp(-x))


def projection(a: np.ndarray, w: np.ndarray, epilogue: str, c_in: np.ndarray = None) -> np.ndarray:
    """The row-set projections of a layer (Sec. 4.2: Q = E W_Q, ...; O = A V_exp W_O;
    the model's SwiGLU MLP) as plain definitions on float64 inputs:
    "store"    a @ w.T
    "residual" c_in + a @ w.T
    "swiglu"   silu(g) * u with [g | u] = a @ w.T split in halves (gate rows first)."""
    y = a @ w.T
    if epilogue == "store":
        return y
    if epilogue == "residual":
        return c_in + y
    if epilogue == "swiglu":
        f = w.shape[0] // 2
        return _silu(y[:, :f]) * y[:, f:]
    raise ValueError(epilogue)


class _Cfg:
    def __init__(self, hidden, ffn, hq, hkv, d, theta, eps):
        self.hidden, self.ffn, self.hq, self.hkv, self.d = hidden, ffn, hq, hkv, d
        self.theta, self.eps = theta, eps


def _layer(h: np.ndarray, s_pos: np.ndarray, w: Dict[str, np.ndarray], cfg: _Cfg,
           cached_k: Sequence[np.ndarray], cached_v: Sequence[np.ndarray], n_total: int,
           bf16_storage: bool):
    """One decoder layer for the selected rows h [nS, hidden] (float64, updated copy returned)."""
    rnd = _round_bf16 if bf16_storage else (lambda a: a)
    hq, hkv, d = cfg.hq, cfg.hkv, cfg.d
    n = h.shape[0]
    x = rnd(rmsnorm(h, _bf16_to_f64(w["attn_norm"]), cfg.eps))
    qkv = x @ _bf16_to_f64(w["wqkv"]).T                                     # Q = E W_Q, K = E W_K, V = E W_V
    q = qkv[:, : hq * d].reshape(n, hq, d)
    k = qkv[:, hq * d: (hq + hkv) * d].reshape(n, hkv, d)
    v = qkv[:, (hq + hkv) * d:].reshape(n, hkv, d)
    q = rnd(rope(q, s_pos, cfg.theta))
    k = rnd(rope(k, s_pos, cfg.theta))
    v = rnd(v)
    K_exp, V_exp = expand_kv(cached_k, cached_v, s_pos, k, v, n_total)    # recomputed rows at their positions
    o, _ = masked_attention(q, K_exp, V_exp, s_pos)                          # Eq. (1)
    o = rnd(o.reshape(n, hq * d))
    h = h + o @ _bf16_to_f64(w["wo"]).T                                     # O = A V_exp W_O, residual
    x2 = rnd(rmsnorm(h, _bf16_to_f64(w["mlp_norm"]), cfg.eps))
    gu = x2 @ _bf16_to_f64(w["w_gate_up"]).T
    a = rnd(_silu(gu[:, : cfg.ffn]) * gu[:, cfg.ffn:])
    h = h + a @ _bf16_to_f64(w["w_down"]).T
    return h, k, v


def decoder_layer(h: np.ndarray, s_pos: np.ndarray, weights: Dict[str, np.ndarray],
                  cached_k: Sequence[np.ndarray], cached_v: Sequence[np.ndarray], n_total: int,
                  hidden: int, ffn: int, hq: int, hkv: int, d: int, theta: float, eps: float,
                  bf16_storage: bool = True):
    """One decoder layer of the link step for the selected rows (Sec. 4.2 per-layer
    recipe inside the Llama block), on its own: h [nS, hidden] is the layer's input
    hidden rows of S at linked positions s_pos; cached_k / cached_v the layer's chunk
    caches as compiled.  Returns (h after the layer, recomputed k [nS, Hkv, d], v).
    This is exactly the step link_model repeats per layer."""
    cfg = _Cfg(hidden, ffn, hq, hkv, d, theta, eps)
    return _layer(np.asarray(h, dtype=np.float64), np.asarray(s_pos), weights, cfg, cached_k, cached_v,
                  n_total, bf16_storage)


def link_model(emb_s: np.ndarray, chunk_lens: Sequence[int], suffix_len: int, k: int,
               weights: Sequence[Dict[str, np.ndarray]], final_norm: np.ndarray,
               caches: Sequence[Tuple[Sequence[np.ndarray], Sequence[np.ndarray]]],
               hidden: int, ffn: int, hq: int, hkv: int, d: int, theta: float, eps: float,
               bf16_storage: bool = True, rerotate: bool = False):
    """Full-model link step for one request.

    emb_s [nS, hidden]: layer-0 hidden rows of S (embeddings of those tokens),
    in ascending position order.  caches[l] = (chunk K list, chunk V list) of
    layer l, each [L_j, Hkv, d] as compiled (float64 values of bf16 data).
    rerotate: cached K of chunks j > 0 is first moved to its linked positions
    (re-rotation variant, see link.rerotate_cached; not for k < 0).
    Returns (s_pos, out [nS, hidden] after the final norm, per-layer recomputed
    (k, v) of S).
    """
    cfg = _Cfg(hidden, ffn, hq, hkv, d, theta, eps)
    s_pos = legolink_positions(chunk_lens, suffix_len, k)
    if len(s_pos) != emb_s.shape[0]:
        raise ValueError(f"|S| = {len(s_pos)} but {emb_s.shape[0]} embedding rows were given")
    n_total = sum(int(x) for x in chunk_lens) + suffix_len
    h = np.asarray(emb_s, dtype=np.float64)
    new_kv = []
    for layer, w in enumerate(weights):
        ck, cv = caches[layer] if caches else ([], [])
        if rerotate and k >= 0:
            ck = rerotate_cached(ck, chunk_lens, theta, bf16_storage)
        h, ks, vs = _layer(h, s_pos, w, cfg, ck, cv, n_total, bf16_storage)
        new_kv.append((ks, vs))
    out = rmsnorm(h, _bf16_to_f64(final_norm), eps)
    return s_pos, out, new_kv


def compile_chunk(emb_chunk: np.ndarray, weights: Sequence[Dict[str, np.ndarray]],
                  final_norm: np.ndarray, hidden: int, ffn: int, hq: int, hkv: int, d: int,
                  theta: float, eps: float, bf16_storage: bool = True, dummy_emb: np.ndarray = None):
    """Compile step (Sec. 2.2): prefill one chunk alone at positions 0..L-1.

    This is the link step of a request with no cached chunks whose tokens are
    all new, so every token is computed.  Returns (hidden out, per-layer (K, V)).

    dummy_emb [n_dummy, hidden]: LegoLink-0's compile (Sec. 5.4).  The dummy
    tokens are placed before the chunk, the n_dummy + L tokens are prefilled
    together at positions 0..n_dummy+L-1, and the dummies' rows are then
    dropped: the returned hidden states and K/V are the chunk's L rows only,
    their K rotated at positions n_dummy..n_dummy+L-1.
    """
    nd = 0 if dummy_emb is None else int(np.asarray(dummy_emb).shape[0])
    rows = emb_chunk if nd == 0 else np.concatenate([np.asarray(dummy_emb, np.float64),
                                                     np.asarray(emb_chunk, np.float64)])
    n = rows.shape[0]
    _, out, kv = link_model(rows, [], n, 0, weights, final_norm, [([], [])] * len(weights),
                            hidden, ffn, hq, hkv, d, theta, eps, bf16_storage)
    return out[nd:], [(k[nd:], v[nd:]) for k, v in kv]
