"""GPU parity of the model-level link step (decoder layers for the selected rows).

The oracle runs the same seeded weights and embeddings in float64, rounding to
bf16 where the data format is bf16 (see oracle/model.py).  Caches are either
compiled by each side on its own (small models: compile + link end to end) or
seeded synthetic caches shared by both (full Llama-3-8B width).  Bars: final
hidden state max |err| <= 2e-2 (values ~N(0, 1) after the final RMSNorm); the
recomputed K/V written into the linked cache max |err| <= 2e-2 (bf16 data).
"""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

import oracle  # noqa: E402
import synth  # noqa: E402
from synth.configs import ModelWorkload, get_config  # noqa: E402

pytestmark = pytest.mark.gpu

ATOL = 2e-2


def _stage(wl, **kw):
    from paper_2410_15332_amd import harness
    print(f"[gpu-test] staging model {wl.name} {kw}", flush=True)
    return harness.stage_model(wl, **kw)


def _f64(bits):
    return synth.bf16_bits_to_f32(bits).astype(np.float64)


def _bits(t):
    return t.detach().cpu().view(torch.int16).numpy().view(np.uint16)


def _oracle_inputs(wl, n_layers):
    ws = [synth.model_weights(wl.seed, l, wl.hidden, wl.ffn, wl.num_q_heads, wl.num_kv_heads, wl.head_dim)
          for l in range(n_layers)]
    fn = synth.final_norm_weight(wl.seed, wl.hidden)
    return ws, fn


def _dims(wl):
    return dict(hidden=wl.hidden, ffn=wl.ffn, hq=wl.num_q_heads, hkv=wl.num_kv_heads, d=wl.head_dim,
                theta=wl.rope_theta, eps=wl.rms_eps)


def _s_embeddings(wl, s_pos):
    offs = oracle.chunk_offsets(wl.chunk_lens)
    n_c = sum(wl.chunk_lens)
    rows = []
    for p in s_pos:
        if p >= n_c:
            rows.append(synth.token_embeddings(wl.seed, 1, 0, [p - n_c], wl.hidden)[0])
        else:
            j = max(i for i, o in enumerate(offs) if o <= p)
            rows.append(synth.token_embeddings(wl.seed, 0, j, [p - offs[j]], wl.hidden)[0])
    return np.asarray(rows, dtype=np.float64)


def _linked_rows(st, layer, s_pos):
    """Recomputed K/V rows of S read back from the GPU's linked cache (token-major)."""
    from paper_2410_15332_amd import epic_link as el
    kc, vc = _bits(st.k_caches[layer]), _bits(st.v_caches[layer])
    K, V = el.read_linked_kv(kc, vc, st.views, 0)
    return _f64(K[s_pos]), _f64(V[s_pos])


def _check(st, n_layers, caches_ref, rerotate=False):
    wl = st.wl
    torch.cuda.synchronize()
    s_pos = oracle.legolink_positions(wl.chunk_lens, wl.suffix_len, wl.k)
    assert np.array_equal(st.views["s_pos"], s_pos), "planner selection differs from the oracle"
    ws, fn = _oracle_inputs(wl, n_layers)
    emb = _s_embeddings(wl, s_pos)
    _, out_ref, kv_ref = oracle.link_model(emb, wl.chunk_lens, wl.suffix_len, wl.k, ws, fn, caches_ref,
                                           bf16_storage=True, rerotate=rerotate, **_dims(wl))
    out = st.out.double().cpu().numpy()
    assert np.all(np.isfinite(out))
    err = np.abs(out - out_ref).max()
    print(f"[gpu-test] {wl.name}: final hidden max|err| {err:.3e} mean {np.abs(out - out_ref).mean():.2e}",
          flush=True)
    assert err <= ATOL, f"final hidden max |err| {err}"
    for layer in range(n_layers):
        gk, gv = _linked_rows(st, layer, s_pos)
        ek = np.abs(gk - kv_ref[layer][0]).max()
        evv = np.abs(gv - kv_ref[layer][1]).max()
        assert ek <= ATOL and evv <= ATOL, f"layer {layer}: recomputed K/V err {ek}, {evv}"
    return err


def _oracle_compiled_caches(wl, n_layers, n_dummy=0, outs=None):
    ws, fn = _oracle_inputs(wl, n_layers)
    dummy = synth.dummy_embeddings(wl.seed, n_dummy, wl.hidden).astype(np.float64) if n_dummy else None
    ck = [[] for _ in range(n_layers)]
    cv = [[] for _ in range(n_layers)]
    for j, L in enumerate(wl.chunk_lens):
        emb = synth.token_embeddings(wl.seed, 0, j, range(L), wl.hidden).astype(np.float64)
        out, kv = oracle.compile_chunk(emb, ws, fn, bf16_storage=True, dummy_emb=dummy, **_dims(wl))
        if outs is not None:
            outs.append(out)
        for layer, (k, v) in enumerate(kv):
            ck[layer].append(k)
            cv[layer].append(v)
    return list(zip(ck, cv))


def _check_chunk_caches(st, ref):
    """The chunk blocks hold each chunk's compiled K/V, token t at slot t."""
    wl = st.wl
    for layer in range(wl.n_layers):
        kc, vc = _bits(st.k_caches[layer]), _bits(st.v_caches[layer])
        for j, blocks in enumerate(st.chunk_block_ids):
            L = wl.chunk_lens[j]
            kb = kc[blocks].transpose(0, 2, 1, 3).reshape(-1, wl.num_kv_heads, wl.head_dim)
            vb = vc[blocks].transpose(0, 3, 1, 2).reshape(-1, wl.num_kv_heads, wl.head_dim)
            ek = np.abs(_f64(kb[:L]) - ref[layer][0][j]).max()
            ev = np.abs(_f64(vb[:L]) - ref[layer][1][j]).max()
            assert ek <= ATOL and ev <= ATOL, f"layer {layer} chunk {j}: compiled K/V err {ek}, {ev}"
            # slots past the chunk's end are zero (nothing of the dummies or a neighbour leaks in)
            assert not kb[L:].any() and not vb[L:].any(), f"layer {layer} chunk {j}: stray rows"


def _small(name, lens, suffix, k, hidden=512, ffn=1024, hq=8, hkv=2, d=64, layers=3, seed=31):
    return ModelWorkload(name, seed, layers, hidden, ffn, hq, hkv, d, 16, 500000.0, 1e-5, lens, suffix, k)


SMALL = [
    _small("ragged_d64_g4", [37, 100, 16, 51], 23, 5),
    _small("d128_g2", [64, 45, 80], 30, 16, hidden=512, ffn=1536, hq=4, hkv=2, d=128),
    _small("mha_k0", [50, 70], 12, 0, hidden=256, ffn=512, hq=4, hkv=4, d=64),
]


@pytest.mark.parametrize("wl", SMALL, ids=[w.name for w in SMALL])
def test_compile_and_link_small(wl):
    """Compile on each side independently, then link: end-to-end parity."""
    st = _stage(wl, caches="compile")
    st.run()
    torch.cuda.synchronize()
    # the GPU-compiled chunk caches against the oracle's compile (bf16 data, tolerance)
    ref = _oracle_compiled_caches(wl, wl.n_layers)
    _check_chunk_caches(st, ref)
    _check(st, wl.n_layers, ref)


LEGO0 = [
    (_small("lego0_ragged_d64", [37, 100, 16, 51, 12], 23, 0), 4),
    (_small("lego0_d128_g2", [64, 45, 80], 30, 0, hidden=512, ffn=1536, hq=4, hkv=2, d=128), 4),
    (_small("dummy_block_k3", [20, 28], 9, 3, layers=2), 16),
]


@pytest.mark.parametrize("wl,nd", LEGO0, ids=[f"{w.name}_nd{n}" for w, n in LEGO0])
def test_dummy_compile_then_link(wl, nd):
    """LegoLink-0 (Sec. 5.4): each side compiles every chunk after nd dummy tokens
    and drops their K/V; the GPU's chunk caches and compiled hidden rows match the
    oracle's, then the link step over those caches (k = 0: only the suffix is
    computed) matches end to end."""
    st = _stage(wl, caches="compile", n_dummy=nd, keep_compile=True)
    outs = []
    ref = _oracle_compiled_caches(wl, wl.n_layers, nd, outs)
    _check_chunk_caches(st, ref)
    cst = st.compile_stage
    got = cst.out.double().cpu().numpy()
    for j, L in enumerate(wl.chunk_lens):
        a = int(cst.views["s_off"][j])
        err = np.abs(got[a + nd:a + nd + L] - outs[j]).max()
        assert err <= ATOL, f"chunk {j}: compiled hidden max |err| {err}"
    st.run()
    err = _check(st, wl.n_layers, ref)
    print(f"[gpu-test] {wl.name} nd={nd}: linked final hidden max|err| {err:.3e}", flush=True)


def test_recompute_all_equals_full_prefill():
    """k < 0 (FR): the link step is an ordinary prefill of the whole linked sequence."""
    wl = _small("fr", [40, 33], 9, -1, layers=2)
    st = _stage(wl, caches="compile")
    st.run()
    torch.cuda.synchronize()
    ws, fn = _oracle_inputs(wl, 2)
    emb = _s_embeddings(wl, np.arange(sum(wl.chunk_lens) + wl.suffix_len))
    full, _ = oracle.compile_chunk(emb, ws, fn, bf16_storage=True, **_dims(wl))
    err = np.abs(st.out.double().cpu().numpy() - full).max()
    assert err <= ATOL, err


def test_llama8b_width_two_layers_synthetic_caches():
    """Llama-3-8B layer shapes (hidden 4096, FFN 14336, GQA 32/8, d 128), the
    20 x 1024-token chunks and 128-token suffix of the 32-layer configuration,
    LegoLink-32, two layers, seeded synthetic caches shared with the oracle."""
    wl = get_config("c3", n_layers=2)
    st = _stage(wl, caches="synthetic")
    st.run()
    caches = []
    for layer in range(2):
        ck, cv = [], []
        for j, L in enumerate(wl.chunk_lens):
            kb, vb = synth.chunk_cache(wl.seed, j, L, wl.num_kv_heads, wl.head_dim, 0.5, layer=layer)
            ck.append(_f64(kb))
            cv.append(_f64(vb))
        caches.append((ck, cv))
    assert st.sizes.n_s == 19 * 32 + 128
    _check(st, 2, caches)


def test_model_rejects_unsupported_width():
    from paper_2410_15332_amd import epic_link as el
    cfg = el.epic_model_cfg(el.attn_cfg(8, 2, 64), 500, 1024, 1, 5e5, 1e-5)
    s = el.epic_plan_sizes()
    assert el.epic_model_workspace_bytes(cfg, s) == 0


def test_recompute_all_wide_output_tiles():
    """A recompute-all link of 4100 rows at hidden 1024: enough row tiles that every
    projection (W_O and W_down included) runs on 128-column output tiles, where the
    short link steps above run their narrow outputs on 64-column tiles."""
    wl = _small("fr_wide", [2000, 2000], 100, -1, hidden=1024, ffn=2048, hq=8, hkv=2, d=128, layers=1)
    st = _stage(wl, caches="synthetic")
    st.run()
    torch.cuda.synchronize()
    assert st.sizes.n_s == 4100
    ws, fn = _oracle_inputs(wl, 1)
    emb = _s_embeddings(wl, np.arange(4100))
    full, _ = oracle.compile_chunk(emb, ws, fn, bf16_storage=True, **_dims(wl))
    err = np.abs(st.out.double().cpu().numpy() - full).max()
    print(f"[gpu-test] fr_wide: final hidden max|err| {err:.3e}", flush=True)
    assert err <= ATOL, err


@pytest.mark.parametrize("wl", [_small("rr_ragged_d64", [37, 100, 16, 51], 23, 5),
                                _small("rr_k0_d128", [64, 45, 80], 30, 0, hidden=512, ffn=1536, hq=4, hkv=2, d=128)],
                         ids=["rr_ragged_d64", "rr_k0_d128"])
def test_compile_and_link_with_rerotation(wl):
    """Re-rotation variant at model level: each side compiles the chunks, then links
    with the cached K of chunks 1.. moved to its linked positions (the model's rotary
    base); end-to-end parity, and the re-rotated linked cache of every layer within a
    bf16 step of the oracle's."""
    st = _stage(wl, caches="compile", rerotate=True)
    st.run()
    torch.cuda.synchronize()
    ref = _oracle_compiled_caches(wl, wl.n_layers)
    err = _check(st, wl.n_layers, ref, rerotate=True)
    from paper_2410_15332_amd import epic_link as el
    offs = oracle.chunk_offsets(wl.chunk_lens)
    s_pos = oracle.legolink_positions(wl.chunk_lens, wl.suffix_len, wl.k)
    for layer in range(wl.n_layers):
        K, _ = el.read_linked_kv(_bits(st.k_caches[layer]), _bits(st.v_caches[layer]), st.views, 0)
        rot = oracle.rerotate_cached(ref[layer][0], wl.chunk_lens, wl.rope_theta)
        for j in range(1, len(wl.chunk_lens)):
            rows = [t for t in range(wl.chunk_lens[j]) if offs[j] + t not in set(s_pos.tolist())]
            got = _f64(K[[offs[j] + t for t in rows]])
            assert np.abs(got - rot[j][rows]).max() <= ATOL, f"layer {layer} chunk {j}: re-rotated K"
    print(f"[gpu-test] {wl.name} re-rotated: final hidden max|err| {err:.3e}", flush=True)
