"""Pins for the CPU oracle: each check ties it to something other than itself.

* the worked selection examples in tests/golden (Sec. 4.2, by hand);
* library causal attention (torch SDPA, float64) for recompute-everything (FR,
  Sec. 2.3) and for the Naive scheme (k = 0, Sec. 2.3);
* closed forms of softmax attention (constant V, zero query, a lone key,
  one-hot V, one-hot K);
* the HuggingFace Llama forward for the compile step (Sec. 2.2) and, through
  prefix-caching / recompute-all identities, for the model-level link step.
"""
import os

import numpy as np
import pytest
import torch

import oracle
from synth import bf16_bits_to_f32, chunk_cache, final_norm_weight, model_weights, row_qkv

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "selection_examples.txt")


def _read_golden():
    cases = []
    with open(GOLDEN) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            lens, suf, k, s = [x.strip() for x in line.split("|")]
            cases.append(([int(x) for x in lens.split(",")], int(suf), int(k),
                          [int(x) for x in s.split(",")] if s else []))
    return cases


@pytest.mark.parametrize("case", _read_golden())
def test_selection_golden(case):
    lens, suf, k, expect = case
    assert oracle.legolink_positions(lens, suf, k).tolist() == expect


def test_selection_size_closed_form():
    rng = np.random.default_rng(1)
    for _ in range(50):
        lens = rng.integers(1, 40, size=rng.integers(1, 8)).tolist()
        suf, k = int(rng.integers(0, 20)), int(rng.integers(0, 50))
        s = oracle.legolink_positions(lens, suf, k)
        assert len(s) == sum(min(k, L) for L in lens[1:]) + suf
        assert np.all(np.diff(s) > 0)


# ---------------------------------------------------------------- attention level

def _f(x):
    return bf16_bits_to_f32(x).astype(np.float64)


def _case(lens, suf, k, hq, hkv, d, seed=5):
    """Chunk caches and the recomputed rows of S for one request (float64 values of bf16 data)."""
    ck, cv = [], []
    for j, L in enumerate(lens):
        a, b = chunk_cache(seed, j, L, hkv, d)
        ck.append(_f(a)); cv.append(_f(b))
    s_pos = oracle.legolink_positions(lens, suf, k)
    q, kk, vv = row_qkv(seed, 0, s_pos, hq, hkv, d)
    return ck, cv, _f(q), _f(kk), _f(vv)


def _sdpa(q, K, V, mask):
    """Library attention in float64: q [n, Hq, d], K/V [N, Hkv, d] (GQA by h // G), mask [n, N] bool."""
    G = q.shape[1] // K.shape[1]
    qt = torch.from_numpy(q).permute(1, 0, 2)[None]
    Kt = torch.from_numpy(K).permute(1, 0, 2).repeat_interleave(G, dim=0)[None]
    Vt = torch.from_numpy(V).permute(1, 0, 2).repeat_interleave(G, dim=0)[None]
    o = torch.nn.functional.scaled_dot_product_attention(qt, Kt, Vt, attn_mask=torch.from_numpy(mask))
    return o[0].permute(1, 0, 2).numpy()


@pytest.mark.parametrize("hq,hkv,d", [(4, 4, 16), (8, 2, 32)])
def test_fr_equals_causal_prefill(hq, hkv, d):
    """S = all tokens (FR): the link step is ordinary causal self-attention."""
    lens, suf = [9, 13, 6], 5
    ck, cv, q, k, v = _case(lens, suf, -1, hq, hkv, d)
    s_pos, out, _, _, _ = oracle.link_attention(lens, suf, -1, ck, cv, q, k, v)
    qt = torch.from_numpy(q).permute(1, 0, 2)[None]
    G = hq // hkv
    Kt = torch.from_numpy(k).permute(1, 0, 2).repeat_interleave(G, dim=0)[None]
    Vt = torch.from_numpy(v).permute(1, 0, 2).repeat_interleave(G, dim=0)[None]
    ref = torch.nn.functional.scaled_dot_product_attention(qt, Kt, Vt, is_causal=True)[0].permute(1, 0, 2)
    np.testing.assert_allclose(out, ref.numpy(), rtol=0, atol=1e-12)


def test_k0_equals_naive_concatenation():
    """k = 0: only the suffix is computed; it attends to the caches concatenated as stored."""
    lens, suf, hq, hkv, d = [7, 12, 5, 9], 6, 8, 4, 16
    ck, cv, q, k, v = _case(lens, suf, 0, hq, hkv, d)
    s_pos, out, _, _, _ = oracle.link_attention(lens, suf, 0, ck, cv, q, k, v)
    K = np.concatenate(ck + [k], axis=0)
    V = np.concatenate(cv + [v], axis=0)
    n_c = sum(lens)
    mask = np.arange(n_c + suf)[None, :] <= (n_c + np.arange(suf))[:, None]
    np.testing.assert_allclose(out, _sdpa(q, K, V, mask), rtol=0, atol=1e-12)


def test_placement_cached_equals_fresh():
    """If every cached vector equals the recomputed one, LegoLink-k gives FR's rows of S.

    Fails if a recomputed row, or a chunk's cache, is put at the wrong linked position.
    """
    lens, suf, hq, hkv, d, seed = [11, 17, 4, 20], 3, 4, 2, 16, 9
    n = sum(lens) + suf
    allq, allk, allv = (_f(a) for a in row_qkv(seed, 0, range(n), hq, hkv, d))
    offs = oracle.chunk_offsets(lens)
    ck = [allk[o:o + L] for o, L in zip(offs, lens)]
    cv = [allv[o:o + L] for o, L in zip(offs, lens)]
    mask = np.tril(np.ones((n, n), bool))
    full = _sdpa(allq, allk, allv, mask)
    for k in (0, 1, 3, 5, 100):
        s = oracle.legolink_positions(lens, suf, k)
        _, out, _, _, _ = oracle.link_attention(lens, suf, k, ck, cv, allq[s], allk[s], allv[s])
        np.testing.assert_allclose(out, full[s], rtol=0, atol=1e-12)


def test_one_hot_v_marks_recomputed_positions():
    """V_exp = e_i for recomputed rows and 0 for cached rows: out's support is S up to the row."""
    lens, suf, hq, hkv, k = [6, 5, 7], 4, 2, 1, 2
    n = sum(lens) + suf
    d = 32
    ck, _, q, kk, _ = _case(lens, suf, k, hq, hkv, d)
    cv = [np.zeros((L, hkv, d)) for L in lens]
    s = oracle.legolink_positions(lens, suf, k)
    vs = np.zeros((len(s), hkv, d))
    vs[np.arange(len(s)), :, s] = 1.0
    _, out, _, _, _ = oracle.link_attention(lens, suf, k, ck, cv, q, kk, vs)
    for r, p in enumerate(s):
        support = set(np.nonzero(out[r, 0] > 0)[0].tolist())
        assert support == set(x for x in s.tolist() if x <= p)
    # all-one-hot V (cached too): out is the attention row itself, masked entries exactly 0
    cv = []
    for o, L in zip(oracle.chunk_offsets(lens), lens):
        z = np.zeros((L, hkv, d)); z[np.arange(L), :, o + np.arange(L)] = 1.0; cv.append(z)
    _, out, _, _, _ = oracle.link_attention(lens, suf, k, ck, cv, q, kk, vs)
    for r, p in enumerate(s):
        assert np.all(out[r, :, p + 1: n] == 0.0)
        np.testing.assert_allclose(out[r].sum(axis=-1), 1.0, atol=1e-13)


def test_closed_forms():
    lens, suf, hq, hkv, d, k = [5, 8], 4, 4, 2, 16, 3
    ck, cv, q, kk, vv = _case(lens, suf, k, hq, hkv, d)
    s = oracle.legolink_positions(lens, suf, k)
    # constant V -> constant output
    cvc = [np.full_like(x, 0.75) for x in cv]
    _, out, _, _, _ = oracle.link_attention(lens, suf, k, ck, cvc, q, kk, np.full_like(vv, 0.75))
    np.testing.assert_allclose(out, 0.75, atol=1e-14)
    # zero query -> uniform weights: mean of V_exp[0..p], lse = log(p + 1)
    _, out, lse, _, V = oracle.link_attention(lens, suf, k, ck, cv, np.zeros_like(q), kk, vv)
    for r, p in enumerate(s):
        for h in range(hq):
            np.testing.assert_allclose(out[r, h], V[: p + 1, h // (hq // hkv)].mean(axis=0), atol=1e-13)
        np.testing.assert_allclose(lse[r], np.log(p + 1), atol=1e-13)


def test_position_zero_and_one_hot_keys():
    """FR row at position 0 sees only itself; one-hot keys give a closed-form normaliser."""
    lens, suf, hq, hkv, d = [4, 3], 2, 2, 2, 16
    ck, cv, q, kk, vv = _case(lens, suf, -1, hq, hkv, d)
    _, out, lse, _, _ = oracle.link_attention(lens, suf, -1, ck, cv, q, kk, vv)
    np.testing.assert_allclose(out[0], vv[0], atol=1e-15)
    np.testing.assert_allclose(lse[0], (q[0] * kk[0]).sum(-1) / np.sqrt(d), atol=1e-13)
    # keys c * e_i, query e_j: row at p >= j has lse = log(p + exp(c / sqrt(d)))
    n, c, j = sum(lens) + suf, 3.0, 2
    kk1 = np.zeros_like(kk)
    kk1[np.arange(n), :, np.arange(n)] = c
    q1 = np.zeros_like(q)
    q1[:, :, j] = 1.0
    _, _, lse, _, _ = oracle.link_attention(lens, suf, -1, ck, cv, q1, kk1, vv)
    for p in range(j, n):
        np.testing.assert_allclose(lse[p], np.log(p + np.exp(c / np.sqrt(d))), atol=1e-13)


def test_gqa_equals_replicated_mha():
    lens, suf, k, d = [6, 9], 3, 2, 16
    ck, cv, q, kk, vv = _case(lens, suf, k, 8, 2, d)
    _, out_gqa, lse_gqa, _, _ = oracle.link_attention(lens, suf, k, ck, cv, q, kk, vv)
    rep = lambda a: np.repeat(a, 4, axis=1)  # noqa: E731
    _, out_mha, lse_mha, _, _ = oracle.link_attention(lens, suf, k, [rep(x) for x in ck],
                                                      [rep(x) for x in cv], q, rep(kk), rep(vv))
    np.testing.assert_allclose(out_gqa, out_mha, atol=1e-15)
    np.testing.assert_allclose(lse_gqa, lse_mha, atol=1e-15)


def test_lse_is_log_normaliser():
    """exp(scale * q.k - lse) over allowed keys sums to 1 and reproduces out."""
    lens, suf, k, hq, hkv, d = [10, 7, 12], 5, 4, 4, 2, 16
    ck, cv, q, kk, vv = _case(lens, suf, k, hq, hkv, d)
    s, out, lse, K, V = oracle.link_attention(lens, suf, k, ck, cv, q, kk, vv)
    for r, p in enumerate(s):
        for h in range(hq):
            w = np.exp(K[: p + 1, h // 2] @ q[r, h] / np.sqrt(d) - lse[r, h])
            np.testing.assert_allclose(w.sum(), 1.0, atol=1e-12)
            np.testing.assert_allclose(w @ V[: p + 1, h // 2], out[r, h], atol=1e-12)


# ---------------------------------------------------------------- model level

TINY = dict(hidden=64, ffn=96, hq=4, hkv=2, d=16, theta=500000.0, eps=1e-5)


def _tiny_weights(n_layers, seed=11):
    ws = [model_weights(seed, l, TINY["hidden"], TINY["ffn"], TINY["hq"], TINY["hkv"], TINY["d"])
          for l in range(n_layers)]
    return ws, final_norm_weight(seed, TINY["hidden"])


def _hf_model(ws, fn):
    from transformers import LlamaConfig, LlamaModel

    t = TINY
    cfg = LlamaConfig(vocab_size=8, hidden_size=t["hidden"], intermediate_size=t["ffn"],
                      num_hidden_layers=len(ws), num_attention_heads=t["hq"],
                      num_key_value_heads=t["hkv"], head_dim=t["d"], rope_theta=t["theta"],
                      rms_norm_eps=t["eps"], max_position_embeddings=4096,
                      attention_bias=False, mlp_bias=False)
    cfg._attn_implementation = "eager"
    m = LlamaModel(cfg).double().eval()
    f = lambda b: torch.from_numpy(_f(b))  # noqa: E731
    qd, kd = t["hq"] * t["d"], t["hkv"] * t["d"]
    with torch.no_grad():
        for layer, w in zip(m.layers, ws):
            wqkv = f(w["wqkv"])
            layer.self_attn.q_proj.weight.copy_(wqkv[:qd])
            layer.self_attn.k_proj.weight.copy_(wqkv[qd:qd + kd])
            layer.self_attn.v_proj.weight.copy_(wqkv[qd + kd:])
            layer.self_attn.o_proj.weight.copy_(f(w["wo"]))
            gu = f(w["w_gate_up"])
            layer.mlp.gate_proj.weight.copy_(gu[: t["ffn"]])
            layer.mlp.up_proj.weight.copy_(gu[t["ffn"]:])
            layer.mlp.down_proj.weight.copy_(f(w["w_down"]))
            layer.input_layernorm.weight.copy_(f(w["attn_norm"]))
            layer.post_attention_layernorm.weight.copy_(f(w["mlp_norm"]))
        m.norm.weight.copy_(f(fn))
    return m


def test_compile_matches_hf_llama():
    """Compile step = ordinary Llama prefill of one chunk at positions 0..L-1 (Sec. 2.2)."""
    ws, fn = _tiny_weights(3)
    L = 23
    emb = np.random.default_rng(3).standard_normal((L, TINY["hidden"]))
    out, kv = oracle.compile_chunk(emb, ws, fn, bf16_storage=False, **TINY)
    m = _hf_model(ws, fn)
    with torch.no_grad():
        r = m(inputs_embeds=torch.from_numpy(emb)[None], position_ids=torch.arange(L)[None], use_cache=True)
    # the HF RMSNorm computes in float32, hence the tolerance
    np.testing.assert_allclose(out, r.last_hidden_state[0].numpy(), atol=2e-5, rtol=0)
    for layer, (k, v) in enumerate(kv):
        hk = r.past_key_values.layers[layer].keys[0].permute(1, 0, 2).numpy()
        hv = r.past_key_values.layers[layer].values[0].permute(1, 0, 2).numpy()
        np.testing.assert_allclose(k, hk, atol=2e-5, rtol=0)
        np.testing.assert_allclose(v, hv, atol=2e-5, rtol=0)


def _tok_emb(n_tokens, seed=4):
    return np.random.default_rng(seed).standard_normal((n_tokens, TINY["hidden"]))


def _compile_all(ws, fn, lens, emb, bf16):
    caches_k = [[] for _ in ws]
    caches_v = [[] for _ in ws]
    for o, L in zip(oracle.chunk_offsets(lens), lens):
        _, kv = oracle.compile_chunk(emb[o:o + L], ws, fn, bf16_storage=bf16, **TINY)
        for layer, (k, v) in enumerate(kv):
            caches_k[layer].append(k)
            caches_v[layer].append(v)
    return list(zip(caches_k, caches_v))


@pytest.mark.parametrize("k", [0, 2, 7])
def test_single_chunk_link_equals_prefill(k):
    """One cached chunk + suffix: chunk 0 is never recomputed and its cache is exact
    (it has no prefix), so the link step equals a full prefill of chunk + suffix."""
    ws, fn = _tiny_weights(2)
    lens, suf = [19], 6
    emb = _tok_emb(sum(lens) + suf)
    caches = _compile_all(ws, fn, lens, emb, bf16=False)
    s, out, _ = oracle.link_model(emb[19:], lens, suf, k, ws, fn, caches, bf16_storage=False, **TINY)
    full, _ = oracle.compile_chunk(emb, ws, fn, bf16_storage=False, **TINY)
    np.testing.assert_allclose(out, full[s], atol=1e-10, rtol=0)


def test_recompute_whole_chunks_equals_prefill():
    """k >= every chunk length recomputes all chunks but the first, whose cache is exact:
    the link step equals the full prefill (FR) on every selected row."""
    ws, fn = _tiny_weights(2)
    lens, suf = [9, 6, 11], 4
    emb = _tok_emb(sum(lens) + suf, seed=8)
    caches = _compile_all(ws, fn, lens, emb, bf16=False)
    s = oracle.legolink_positions(lens, suf, 11)
    _, out, kv = oracle.link_model(emb[s], lens, suf, 11, ws, fn, caches, bf16_storage=False, **TINY)
    full, fkv = oracle.compile_chunk(emb, ws, fn, bf16_storage=False, **TINY)
    np.testing.assert_allclose(out, full[s], atol=1e-10, rtol=0)
    for (k1, v1), (k2, v2) in zip(kv, fkv):
        np.testing.assert_allclose(k1, k2[s], atol=1e-10, rtol=0)
        np.testing.assert_allclose(v1, v2[s], atol=1e-10, rtol=0)


def test_link_differs_from_prefill_when_caches_are_position_independent():
    """With several chunks and small k the link step is an approximation: the cached
    rows of later chunks were compiled at positions from 0, so the result differs
    from FR (guards against an oracle that silently recomputes everything)."""
    ws, fn = _tiny_weights(2)
    lens, suf = [9, 6, 11], 4
    emb = _tok_emb(sum(lens) + suf, seed=8)
    caches = _compile_all(ws, fn, lens, emb, bf16=False)
    s = oracle.legolink_positions(lens, suf, 1)
    _, out, _ = oracle.link_model(emb[s], lens, suf, 1, ws, fn, caches, bf16_storage=False, **TINY)
    full, _ = oracle.compile_chunk(emb, ws, fn, bf16_storage=False, **TINY)
    assert np.abs(out - full[s]).max() > 1e-3


def test_bf16_storage_stays_close():
    """Rounding at the bf16 storage points moves the result by about bf16 precision only."""
    ws, fn = _tiny_weights(2)
    lens, suf, k = [9, 6, 11], 4, 3
    emb = _tok_emb(sum(lens) + suf, seed=8)
    s = oracle.legolink_positions(lens, suf, k)
    c64 = _compile_all(ws, fn, lens, emb, bf16=False)
    c16 = _compile_all(ws, fn, lens, emb, bf16=True)
    _, o64, _ = oracle.link_model(emb[s], lens, suf, k, ws, fn, c64, bf16_storage=False, **TINY)
    _, o16, _ = oracle.link_model(emb[s], lens, suf, k, ws, fn, c16, bf16_storage=True, **TINY)
    assert np.abs(o64 - o16).max() < 5e-2


def test_round_bf16_matches_library_cast():
    """The oracle's bf16 storage rounding (float64 -> float32 -> bf16, nearest, ties to
    even) against torch's float32 -> bfloat16 conversion: random values over many
    binades, exact ties with even and odd kept halves, near ties either side,
    carries into the next binade, signed zeros, subnormals and overflow to inf."""
    from oracle.link import _round_bf16
    rng = np.random.default_rng(11)
    vals = [rng.standard_normal(200000) * np.exp2(rng.integers(-30, 30, 200000))]
    hi = rng.integers(0, 1 << 16, 50000, dtype=np.uint32) << np.uint32(16)
    for low in (0x8000, 0x7FFF, 0x8001, 0x0001, 0xFFFF, 0x0000):     # ties, near ties, extremes
        f = (hi | np.uint32(low)).view(np.float32)
        vals.append(f[np.isfinite(f)].astype(np.float64))          # NaN patterns are not a rounding question
    vals.append(np.array([0.0, -0.0, 1.0 + 2.0 ** -8, 1.0 + 3 * 2.0 ** -8, -(1.0 + 2.0 ** -8),
                          np.float32(np.finfo(np.float32).max), 2.0 ** -140, 2.0 ** -149, 3.0 * 2.0 ** -134]))
    x = np.concatenate(vals)
    ref = torch.from_numpy(x.astype(np.float32)).to(torch.bfloat16).to(torch.float64).numpy()
    got = _round_bf16(x)
    assert np.array_equal(np.signbit(got), np.signbit(ref))
    assert np.array_equal(got, ref)
    # hand-worked cases (bf16 keeps 8 significant bits: the spacing at 1 is 2^-7)
    r = _round_bf16(np.array([1.0 + 2.0 ** -8, 1.0 + 3 * 2.0 ** -8, 1.0 + 2.0 ** -8 + 2.0 ** -20, -1.5 - 2.0 ** -9]))
    assert r.tolist() == [1.0, 1.0 + 2.0 ** -6, 1.0 + 2.0 ** -7, -1.5]


def test_masked_attention_row_subset_equals_full():
    """Computing some rows of S (any order of groups, any group size) gives those rows
    of the full result: rows are independent, so sampled parity checks are sound."""
    rng = np.random.default_rng(12)
    n_total, hkv, hq, d = 300, 2, 4, 16
    K = rng.standard_normal((n_total, hkv, d))
    V = rng.standard_normal((n_total, hkv, d))
    s_pos = np.sort(rng.choice(n_total, 57, replace=False))
    q = rng.standard_normal((57, hq, d))
    out, lse = oracle.masked_attention(q, K, V, s_pos)
    for rows, group in (([0, 56], 256), (rng.choice(57, 20, replace=False), 3), (np.arange(57), 7)):
        o2, l2 = oracle.masked_attention(q, K, V, s_pos, rows=rows, row_group=group)
        np.testing.assert_allclose(o2, out[rows], rtol=0, atol=1e-12)
        np.testing.assert_allclose(l2, lse[rows], rtol=0, atol=1e-12)


def test_rope_properties():
    rng = np.random.default_rng(2)
    x = rng.standard_normal((5, 3, 16))
    pos = np.array([0, 1, 7, 1000, 131071])
    y = oracle.rope(x, pos, 500000.0)
    np.testing.assert_allclose(y[0], x[0], atol=0)                     # position 0: identity
    np.testing.assert_allclose(np.linalg.norm(y, axis=-1), np.linalg.norm(x, axis=-1), rtol=1e-13)
    # relative position: <R(a) q, R(b) k> depends on a - b only
    q, k = rng.standard_normal((1, 1, 16)), rng.standard_normal((1, 1, 16))
    d1 = (oracle.rope(q, np.array([50]), 1e4) * oracle.rope(k, np.array([20]), 1e4)).sum()
    d2 = (oracle.rope(q, np.array([130]), 1e4) * oracle.rope(k, np.array([100]), 1e4)).sum()
    np.testing.assert_allclose(d1, d2, rtol=1e-12)


def test_projection_brute_force():
    """The projection oracle against explicit sums on tiny inputs (a dropped term,
    a transposed operand or a swapped gate/up half changes these values)."""
    import math
    rng = np.random.default_rng(5)
    m, n, k = 3, 6, 5
    a = rng.standard_normal((m, k))
    w = rng.standard_normal((n, k))
    c0 = rng.standard_normal((m, n))
    dot = [[sum(a[i, t] * w[j, t] for t in range(k)) for j in range(n)] for i in range(m)]
    assert np.allclose(oracle.projection(a, w, "store"), dot, rtol=0, atol=1e-12)
    assert np.allclose(oracle.projection(a, w, "residual", c0), np.asarray(dot) + c0, rtol=0, atol=1e-12)
    f = n // 2
    sw = [[dot[i][j] / (1.0 + math.exp(-dot[i][j])) * dot[i][j + f] for j in range(f)] for i in range(m)]
    assert np.allclose(oracle.projection(a, w, "swiglu"), sw, rtol=0, atol=1e-12)
    # identity weights: the store epilogue returns the rows themselves
    assert np.array_equal(oracle.projection(a, np.eye(k), "store"), a)


def test_decode_equals_link_of_the_grown_request():
    """Decoding t tokens after a link step gives the rows the link step of the grown
    request (its suffix t tokens longer, those t rows recomputed like every suffix
    row) computes for them; and decoding 2 + 3 tokens in two steps gives the same as
    5 at once (causal attention: earlier rows never see later keys)."""
    rng = np.random.default_rng(11)
    lens, suffix, k, hq, hkv, d = [9, 14, 7], 5, 3, 4, 2, 8
    ck = [rng.standard_normal((L, hkv, d)) for L in lens]
    cv = [rng.standard_normal((L, hkv, d)) for L in lens]
    n_s = len(oracle.legolink_positions(lens, suffix, k))
    t = 5
    q = rng.standard_normal((n_s + t, hq, d))
    kk = rng.standard_normal((n_s + t, hkv, d))
    vv = rng.standard_normal((n_s + t, hkv, d))
    pos, out, lse, K, V = oracle.decode_attention(lens, suffix, k, ck, cv, kk[:n_s], vv[:n_s],
                                                  q[n_s:], kk[n_s:], vv[n_s:])
    s_grown, out_g, lse_g, K_g, V_g = oracle.link_attention(lens, suffix + t, k, ck, cv, q, kk, vv)
    assert np.array_equal(pos, s_grown[n_s:])
    assert np.allclose(out, out_g[n_s:], rtol=0, atol=1e-12) and np.allclose(lse, lse_g[n_s:], rtol=0, atol=1e-12)
    assert np.array_equal(K, K_g) and np.array_equal(V, V_g)
    # two steps: 2 tokens, then 3 more after them
    _, o1, _, _, _ = oracle.decode_attention(lens, suffix, k, ck, cv, kk[:n_s], vv[:n_s],
                                             q[n_s:n_s + 2], kk[n_s:n_s + 2], vv[n_s:n_s + 2])
    _, o2, _, _, _ = oracle.decode_attention(lens, suffix + 2, k, ck, cv, kk[:n_s + 2], vv[:n_s + 2],
                                             q[n_s + 2:], kk[n_s + 2:], vv[n_s + 2:])
    assert np.allclose(np.concatenate([o1, o2]), out, rtol=0, atol=1e-12)


def test_dummy_compile_matches_hf_llama():
    """LegoLink-0's compile (Sec. 5.4): the dummy tokens and the chunk are one
    ordinary Llama prefill at positions 0..n_dummy+L-1 whose first n_dummy rows
    are dropped; hidden states and K/V of the chunk rows match the HuggingFace
    forward of the whole sequence."""
    ws, fn = _tiny_weights(2)
    nd, L = 4, 21
    rng = np.random.default_rng(13)
    bos = rng.standard_normal(TINY["hidden"])
    dummy = np.tile(bos, (nd, 1))
    emb = rng.standard_normal((L, TINY["hidden"]))
    out, kv = oracle.compile_chunk(emb, ws, fn, bf16_storage=False, dummy_emb=dummy, **TINY)
    assert out.shape[0] == L and all(k.shape[0] == L and v.shape[0] == L for k, v in kv)
    m = _hf_model(ws, fn)
    seq = np.concatenate([dummy, emb])
    with torch.no_grad():
        r = m(inputs_embeds=torch.from_numpy(seq)[None], position_ids=torch.arange(nd + L)[None], use_cache=True)
    np.testing.assert_allclose(out, r.last_hidden_state[0].numpy()[nd:], atol=2e-5, rtol=0)
    for layer, (k, v) in enumerate(kv):
        hk = r.past_key_values.layers[layer].keys[0].permute(1, 0, 2).numpy()[nd:]
        hv = r.past_key_values.layers[layer].values[0].permute(1, 0, 2).numpy()[nd:]
        np.testing.assert_allclose(k, hk, atol=2e-5, rtol=0)
        np.testing.assert_allclose(v, hv, atol=2e-5, rtol=0)


def test_dummy_compile_equals_link_after_cached_dummies():
    """The dummies form an exact prefix: compiling them alone as chunk 0 and linking
    the chunk as a suffix (k = 0, so nothing of chunk 0 is recomputed) gives the
    dummy compile's K/V and hidden states; and the dummies change the cache (the
    result differs from the plain compile)."""
    ws, fn = _tiny_weights(2)
    nd, L = 4, 13
    rng = np.random.default_rng(17)
    dummy = np.tile(rng.standard_normal(TINY["hidden"]), (nd, 1))
    emb = rng.standard_normal((L, TINY["hidden"]))
    out, kv = oracle.compile_chunk(emb, ws, fn, bf16_storage=False, dummy_emb=dummy, **TINY)
    caches = _compile_all(ws, fn, [nd], dummy, bf16=False)
    s, out_l, kv_l = oracle.link_model(emb, [nd], L, 0, ws, fn, caches, bf16_storage=False, **TINY)
    assert s.tolist() == list(range(nd, nd + L))
    np.testing.assert_allclose(out, out_l, atol=1e-10, rtol=0)
    for (k1, v1), (k2, v2) in zip(kv, kv_l):
        np.testing.assert_allclose(k1, k2, atol=1e-10, rtol=0)
        np.testing.assert_allclose(v1, v2, atol=1e-10, rtol=0)
    _, kv0 = oracle.compile_chunk(emb, ws, fn, bf16_storage=False, **TINY)
    assert np.abs(kv0[0][0] - kv[0][0]).max() > 1e-3


def test_rerotated_naive_equals_causal_attention_at_linked_positions():
    """Re-rotation variant: chunk caches hold K rotated at the chunk's own positions
    0..L-1.  Rotating chunk j's rows by its linked offset must give K rotated at the
    linked positions (so the rotations compose), and the k = 0 link step over them is
    then ordinary causal attention with every key at its linked position (torch
    SDPA).  Without re-rotation the same inputs give a different result."""
    rng = np.random.default_rng(21)
    lens, suf, hq, hkv, d, theta = [9, 13, 6], 5, 4, 2, 16, 10000.0
    n = sum(lens) + suf
    k_raw = rng.standard_normal((n, hkv, d))
    v = rng.standard_normal((n, hkv, d))
    q_raw = rng.standard_normal((n, hq, d))
    offs = oracle.chunk_offsets(lens)
    ck = [oracle.rope(k_raw[o:o + L], np.arange(L), theta) for o, L in zip(offs, lens)]
    cv = [v[o:o + L] for o, L in zip(offs, lens)]
    rot = oracle.rerotate_cached(ck, lens, theta, bf16_storage=False)
    for o, L, r in zip(offs, lens, rot):
        np.testing.assert_allclose(r, oracle.rope(k_raw[o:o + L], np.arange(o, o + L), theta), rtol=0, atol=1e-12)
    k_lin = oracle.rope(k_raw, np.arange(n), theta)
    q_lin = oracle.rope(q_raw, np.arange(n), theta)
    s = np.arange(sum(lens), n)
    # the rounding step of the stored variant is the only difference from the exact one
    s_pos, out, _, K, _ = oracle.link_attention(lens, suf, 0, ck, cv, q_lin[s], k_lin[s], v[s],
                                                rerotate_theta=theta)
    assert np.abs(K[:sum(lens)] - k_lin[:sum(lens)]).max() < 2e-2
    _, out_exact, _, _, _ = oracle.link_attention(lens, suf, 0, rot, cv, q_lin[s], k_lin[s], v[s])
    G = hq // hkv
    qt = torch.from_numpy(q_lin).permute(1, 0, 2)[None]
    Kt = torch.from_numpy(k_lin).permute(1, 0, 2).repeat_interleave(G, dim=0)[None]
    Vt = torch.from_numpy(v).permute(1, 0, 2).repeat_interleave(G, dim=0)[None]
    ref = torch.nn.functional.scaled_dot_product_attention(qt, Kt, Vt, is_causal=True)[0].permute(1, 0, 2).numpy()
    np.testing.assert_allclose(out_exact, ref[s], rtol=0, atol=1e-12)
    assert np.abs(out - ref[s]).max() < 2e-2
    _, out_plain, _, _, _ = oracle.link_attention(lens, suf, 0, ck, cv, q_lin[s], k_lin[s], v[s])
    assert np.abs(out_plain - ref[s]).max() > 1e-2


def test_rerotated_cache_equals_compile_at_linked_positions():
    """Model level: a chunk compiled alone at positions off..off+L-1 has the same hidden
    states as at 0..L-1 (rotary attention sees relative positions only) and K rotated
    by off more; the HuggingFace forward at shifted position ids gives exactly the
    re-rotated cache.  And the model-level link step with re-rotation and k = 0 runs
    the suffix over those caches."""
    ws, fn = _tiny_weights(2)
    lens, suf = [7, 10], 3
    emb = _tok_emb(sum(lens) + suf, seed=23)
    caches = _compile_all(ws, fn, lens, emb, bf16=False)
    m = _hf_model(ws, fn)
    off = lens[0]
    with torch.no_grad():
        r = m(inputs_embeds=torch.from_numpy(emb[off:off + lens[1]])[None],
              position_ids=torch.arange(off, off + lens[1])[None], use_cache=True)
    for layer in range(2):
        rot = oracle.rerotate_cached(caches[layer][0], lens, TINY["theta"], bf16_storage=False)
        hk = r.past_key_values.layers[layer].keys[0].permute(1, 0, 2).numpy()
        np.testing.assert_allclose(rot[1], hk, atol=2e-5, rtol=0)
        np.testing.assert_array_equal(rot[0], caches[layer][0][0])
    # with re-rotated caches every key sits at its linked position; the suffix rows of
    # the k = 0 link step then equal a link over caches compiled at the linked positions
    rot_caches = [(oracle.rerotate_cached(ck, lens, TINY["theta"], bf16_storage=False), cv) for ck, cv in caches]
    s, out_r, _ = oracle.link_model(emb[17:], lens, suf, 0, ws, fn, caches, bf16_storage=False, rerotate=True,
                                    **TINY)
    _, out_e, _ = oracle.link_model(emb[17:], lens, suf, 0, ws, fn, rot_caches, bf16_storage=False, **TINY)
    np.testing.assert_allclose(out_r, out_e, atol=1e-12, rtol=0)
