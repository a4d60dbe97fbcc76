"""Attention-level link step, written from Sec. 4.2 and Eq. (1) of the paper.

Notation follows Sec. 4.2: the k' selected tokens are recomputed, K_exp / V_exp
(N rows) hold the cached KV of the N - k' unselected tokens plus the
recomputed rows, each at its own linked position, and A = softmax(Q K_exp^T . MASK) with
MASK letting each selected token attend only to tokens at or before it.

Readings where the paper is silent (each one is a choice):
  * the logits are scaled by 1/sqrt(d) (standard attention; needed for
    recompute-everything to equal an ordinary prefill);
  * MASK is additive -inf (a masked key gets zero weight), and a token attends
    to itself (key position <= query position);
  * cached K keeps the rotary phase it was compiled with (no re-rotation); the
    re-rotation variant (``rerotate_theta``) instead rotates chunk j's cached K
    by its linked offset, stored again as bf16;
  * k larger than a chunk recomputes the whole chunk; k = 0 recomputes only the
    suffix (the Naive scheme of Sec. 2.3); k < 0 means recompute every token
    including the first chunk (FR, Sec. 2.3);
  * GQA: query head h reads KV head floor(h / G), G = Hq / Hkv.
"""
from __future__ import annotations

from typing import List, Sequence, Tuple

import numpy as np


def _round_bf16(x: np.ndarray) -> np.ndarray:
    """float64 -> float32 -> bf16 (nearest, ties to even) -> float64."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    u = (u + (np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1)))) & np.uint32(0xFFFF0000)
    return u.view(np.float32).astype(np.float64)


def rope(x: np.ndarray, pos: np.ndarray, theta: float) -> np.ndarray:
    """Rotate [n, H, d] by linked positions pos [n]; pairs (i, i + d/2), angle pos * theta^(-2i/d)."""
    d = x.shape[-1]
    half = d // 2
    inv_freq = theta ** (-np.arange(half, dtype=np.float64) * 2.0 / d)
    ang = np.asarray(pos, dtype=np.float64)[:, None] * inv_freq[None, :]      # [n, d/2]
    cos = np.cos(ang)[:, None, :]
    sin = np.sin(ang)[:, None, :]
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * cos - x2 * sin, x2 * cos + x1 * sin], axis=-1)


def rerotate_cached(cached_k: Sequence[np.ndarray], chunk_lens: Sequence[int], theta: float,
                    bf16_storage: bool = True) -> List[np.ndarray]:
    """Re-rotation variant of the cached K: chunk j's rows were rotated at their own
    positions t, so rotating them by the chunk's linked offset off_j puts them at
    off_j + t (rotations compose).  Chunk 0 (offset 0) is unchanged.  With
    bf16_storage the rotated rows are rounded to bf16, as a stored cache is."""
    out = []
    for j, (ck, off) in enumerate(zip(cached_k, chunk_offsets(chunk_lens))):
        if j == 0 or off == 0:
            out.append(ck)
            continue
        r = rope(np.asarray(ck, np.float64), np.full(ck.shape[0], off), theta)
        out.append(_round_bf16(r) if bf16_storage else r)
    return out


def chunk_offsets(chunk_lens: Sequence[int]) -> List[int]:
    """Linked position of each chunk's first token: the chunks are concatenated in order."""
    offs, acc = [], 0
    for length in chunk_lens:
        offs.append(acc)
        acc += int(length)
    return offs


def legolink_positions(chunk_lens: Sequence[int], suffix_len: int, k: int) -> np.ndarray:
    """Linked positions of the selected set S (Sec. 4.2), ascending.

    LegoLink-k selects the first k tokens of every chunk except the first, plus
    every mutable (query) token, which sit after all chunks.  k < 0 selects all
    tokens (FR).
    """
    offs = chunk_offsets(chunk_lens)
    n_chunk_tokens = sum(int(x) for x in chunk_lens)
    if k < 0:
        return np.arange(n_chunk_tokens + suffix_len, dtype=np.int64)
    sel = []
    for j, (off, length) in enumerate(zip(offs, chunk_lens)):
        if j == 0:
            continue  # the first chunk is never recomputed
        sel.extend(range(off, off + min(k, int(length))))
    sel.extend(range(n_chunk_tokens, n_chunk_tokens + suffix_len))
    return np.asarray(sel, dtype=np.int64)


def expand_kv(cached_k: Sequence[np.ndarray], cached_v: Sequence[np.ndarray],
              s_pos: np.ndarray, k_s: np.ndarray, v_s: np.ndarray,
              n_total: int) -> Tuple[np.ndarray, np.ndarray]:
    """Build K_exp and V_exp [N, Hkv, d] (Sec. 4.2, third step).

    cached_k[j], cached_v[j] are chunk j's cache [L_j, Hkv, d] exactly as the
    compile step stored it.  Rows of S take the recomputed k_s / v_s; every
    other row takes the cached vector of the chunk that holds that position.
    """
    hkv, d = k_s.shape[1], k_s.shape[2]
    K = np.full((n_total, hkv, d), np.nan)
    V = np.full((n_total, hkv, d), np.nan)
    pos = 0
    for ck, cv in zip(cached_k, cached_v):
        K[pos:pos + ck.shape[0]] = ck
        V[pos:pos + cv.shape[0]] = cv
        pos += ck.shape[0]
    K[s_pos] = k_s
    V[s_pos] = v_s
    if np.isnan(K).any() or np.isnan(V).any():
        raise ValueError("a linked position has neither a cached nor a recomputed vector")
    return K, V


def masked_attention(q: np.ndarray, K_exp: np.ndarray, V_exp: np.ndarray, s_pos: np.ndarray,
                     scale: float | None = None, rows: Sequence[int] | None = None,
                     row_group: int = 256) -> Tuple[np.ndarray, np.ndarray]:
    """Eq. (1): per selected row r at linked position p and head h,
    A = softmax over keys i <= p of scale * <q[r,h], K_exp[i, h // G]>,
    O = A . V_exp[:, h // G].  Returns out [n, Hq, d] and the natural-log
    normaliser lse [n, Hq] (log of the softmax denominator, max included).

    ``rows`` restricts the computation to some rows of S (each row is
    independent); rows are processed ``row_group`` at a time to bound memory.
    The steps run as float64 PyTorch CPU operations (multi-threaded library
    matmul, exp and sums; nothing fused or reordered).
    """
    import torch

    n_s, hq, d = q.shape
    hkv = K_exp.shape[1]
    G = hq // hkv
    if scale is None:
        scale = 1.0 / np.sqrt(d)
    rows = np.arange(n_s) if rows is None else np.asarray(rows, dtype=np.int64)
    out = np.zeros((len(rows), hq, d))
    lse = np.zeros((len(rows), hq))
    qt = torch.from_numpy(np.ascontiguousarray(q, dtype=np.float64))
    n_max = int(np.asarray(s_pos)[rows].max()) + 1 if len(rows) else 0
    Kg = [torch.from_numpy(np.ascontiguousarray(K_exp[:n_max, g, :], dtype=np.float64)) for g in range(hkv)]
    Vg = [torch.from_numpy(np.ascontiguousarray(V_exp[:n_max, g, :], dtype=np.float64)) for g in range(hkv)]
    for g0 in range(0, len(rows), row_group):
        rr = rows[g0:g0 + row_group]
        p = torch.from_numpy(np.asarray(s_pos)[rr].astype(np.int64))
        n_keys = int(p.max()) + 1
        masked = torch.arange(n_keys)[None, :] > p[:, None]    # key after the query: excluded
        rt = torch.from_numpy(rr)
        for h in range(hq):
            g = h // G
            logits = scale * (qt[rt, h, :] @ Kg[g][:n_keys].T)
            logits.masked_fill_(masked, -np.inf)
            m = logits.amax(dim=1, keepdim=True)
            e = torch.exp(logits - m)
            denom = e.sum(dim=1, keepdim=True)
            out[g0:g0 + len(rr), h, :] = ((e @ Vg[g][:n_keys]) / denom).numpy()
            lse[g0:g0 + len(rr), h] = (m + torch.log(denom))[:, 0].numpy()
    return out, lse


def link_attention(chunk_lens: Sequence[int], suffix_len: int, k: int,
                   cached_k: Sequence[np.ndarray], cached_v: Sequence[np.ndarray],
                   q_s: np.ndarray, k_s: np.ndarray, v_s: np.ndarray,
                   scale: float | None = None, rows: Sequence[int] | None = None,
                   rerotate_theta: float | None = None):
    """One attention layer of the link step for one request.

    q_s, k_s, v_s are the recomputed rows of S in ascending position order
    (already projected and rotated).  rerotate_theta: the re-rotation variant
    (cached K moved to its linked positions, rotary base theta; not for k < 0).
    Returns (s_pos, out, lse, K_exp, V_exp).
    """
    if rerotate_theta is not None and k >= 0:
        cached_k = rerotate_cached(cached_k, chunk_lens, rerotate_theta)
    s_pos = legolink_positions(chunk_lens, suffix_len, k)
    if len(s_pos) != q_s.shape[0]:
        raise ValueError(f"|S| = {len(s_pos)} but {q_s.shape[0]} query rows were given")
    n_total = sum(int(x) for x in chunk_lens) + suffix_len
    K_exp, V_exp = expand_kv(cached_k, cached_v, s_pos, k_s, v_s, n_total)
    out, lse = masked_attention(q_s, K_exp, V_exp, s_pos, scale, rows)
    return s_pos, out, lse, K_exp, V_exp


def decode_attention(chunk_lens: Sequence[int], suffix_len: int, k: int,
                     cached_k: Sequence[np.ndarray], cached_v: Sequence[np.ndarray],
                     k_s: np.ndarray, v_s: np.ndarray,
                     new_q: np.ndarray, new_k: np.ndarray, new_v: np.ndarray,
                     scale: float | None = None):
    """Decode after the link step, for one request: t new tokens appended after the
    N = sum(chunk_lens) + suffix_len linked tokens attend, causally, over the linked
    sequence (K_exp / V_exp of the link step, Sec. 4.2) extended by themselves.

    k_s, v_s: the link step's recomputed rows of S (ascending); new_q / new_k /
    new_v: [t, H, d] rows of the new tokens at positions N .. N + t - 1.
    Returns (new_pos, out, lse, K_exp, V_exp) with K_exp / V_exp [N + t, Hkv, d].
    """
    s_pos = legolink_positions(chunk_lens, suffix_len, k)
    n_total = sum(int(x) for x in chunk_lens) + suffix_len
    t = new_q.shape[0]
    new_pos = np.arange(n_total, n_total + t, dtype=np.int64)
    K_exp, V_exp = expand_kv(cached_k, cached_v, np.concatenate([s_pos, new_pos]),
                             np.concatenate([k_s, new_k]), np.concatenate([v_s, new_v]), n_total + t)
    out, lse = masked_attention(new_q, K_exp, V_exp, new_pos, scale)
    return new_pos, out, lse, K_exp, V_exp
