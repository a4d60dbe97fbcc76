"""GPU parity of decode after the link step: epic_plan_decode + epic_link_attention
against oracle.decode_attention (new tokens attending over the linked sequence of
the link step, extended by themselves).

Each case runs the link step, then several decode steps that append tokens to each
request (filling the last private block, opening new ones from the free list).
Bars as for the link step: linked cache bit-exact after every step (the link
step's recomputed rows and the earlier decoded rows stay, the new rows land at
their positions, shared chunk blocks untouched); attention output max |err|
<= 2e-2; |exp(lse_gpu - lse_ref) - 1| <= 1e-3.
"""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

import oracle  # noqa: E402
import synth  # noqa: E402
from synth.configs import get_config  # noqa: E402

pytestmark = pytest.mark.gpu


def _bits(t):
    return t.detach().cpu().view(torch.int16).numpy().view(np.uint16)


def _f64(bits):
    return synth.bf16_bits_to_f32(bits).astype(np.float64)


def _run_decode(wl, steps, spare_blocks=64, tile_rows=0):
    from paper_2410_15332_amd import epic_link as el, harness
    print(f"[gpu-test] decode after {wl.name} k={wl.k}: steps {[sum(s) for s in steps]} tokens, "
          f"tile rows {tile_rows or 'auto'}", flush=True)
    st = harness.stage_attention(wl, spare_blocks=spare_blocks, tile_rows=tile_rows)
    st.run()
    hq, hkv, d = wl.num_q_heads, wl.num_kv_heads, wl.head_dim
    per = []
    for r, chunks in enumerate(wl.requests):
        lens = [wl.chunk_lens[c] for c in chunks]
        s_ref = oracle.legolink_positions(lens, wl.suffix_lens[r], wl.k)
        ck, cv = [], []
        for c in chunks:
            kb, vb = synth.chunk_cache(wl.seed, c, wl.chunk_lens[c], hkv, d, wl.value_scale, qk_scale=wl.qk_scale)
            ck.append(_f64(kb))
            cv.append(_f64(vb))
        _, k, v = synth.row_qkv(wl.seed, r, s_ref, hq, hkv, d, wl.value_scale, wl.qk_scale)
        per.append(dict(lens=lens, suffix=wl.suffix_lens[r], ck=ck, cv=cv, k=_f64(k), v=_f64(v)))
    prev_sizes, prev_host, spare = st.sizes, st.dplan.host, st.spare
    worst = 0.0
    for new in steps:
        ds = harness.stage_decode(wl, st.cfg, prev_sizes, prev_host, spare, st.num_blocks, new)
        if tile_rows:
            assert ds.sizes.tile_rows == tile_rows
        elif max(new) <= 16 // (wl.num_q_heads // wl.num_kv_heads) and sum(new) > 0:
            assert ds.sizes.tile_rows == 16, "decode-shaped plan without 16-row tiles"
        ds.run(st.k_cache, st.v_cache)
        torch.cuda.synchronize()
        out, lse = ds.out.float().cpu().numpy(), ds.lse.cpu().numpy()
        kc, vc = _bits(st.k_cache), _bits(st.v_cache)
        for r, t in enumerate(new):
            p = per[r]
            a, b = int(ds.views["s_off"][r]), int(ds.views["s_off"][r + 1])
            assert b - a == t
            pos = ds.views["s_pos"][a:b]
            q_new, k_new, v_new = (_f64(x) for x in synth.row_qkv(wl.seed, r, pos, hq, hkv, d, wl.value_scale,
                                                                  wl.qk_scale))
            ref_pos, o_ref, l_ref, K_exp, V_exp = oracle.decode_attention(
                p["lens"], p["suffix"], wl.k, p["ck"], p["cv"], p["k"], p["v"], q_new, k_new, v_new)
            assert np.array_equal(pos, ref_pos), f"request {r}: decode positions differ"
            if t:
                err = np.abs(out[a:b] - o_ref).max() / max(1.0, wl.value_scale)
                worst = max(worst, err)
                assert err <= 2e-2, f"request {r}: max |out err| {err}"
                assert np.all(np.abs(np.exp(lse[a:b].astype(np.float64) - l_ref) - 1.0) <= 1e-3)
            gk, gv = el.read_linked_kv(kc, vc, ds.views, r)
            assert np.array_equal(_f64(gk), K_exp), f"request {r}: linked K differs after decode"
            assert np.array_equal(_f64(gv), V_exp), f"request {r}: linked V differs after decode"
            p["k"] = np.concatenate([p["k"], k_new])
            p["v"] = np.concatenate([p["v"], v_new])
            p["suffix"] += t
        prev_sizes, prev_host, spare = ds.sizes, ds.dplan.host, ds.spare
    for c, ids in st.chunk_block_ids.items():
        kr, vr = synth.chunk_cache(wl.seed, c, wl.chunk_lens[c], hkv, d, wl.value_scale, qk_scale=wl.qk_scale)
        kb, vb = el.pack_blocks(kr, vr)
        assert np.array_equal(kc[ids], kb) and np.array_equal(vc[ids], vb), f"chunk {c} blocks modified"
    print(f"[gpu-test]   max |out err| {worst:.3e}", flush=True)


def test_decode_after_c1():
    """4 x 128 chunks + 16 suffix tokens (one full block): the first token opens a block."""
    _run_decode(get_config("c1"), [[1], [3], [16], [0], [1]])


@pytest.mark.parametrize("tile_rows", [0, 16, 128])
def test_decode_after_c2_gqa(tile_rows):
    """Auto: 16-row tiles (the decode kernel) for 1-token steps, 128-row tiles for 17
    and 5 tokens at G = 4.  Forced 16: the link step itself and every decode step on
    the decode kernel (several 16-row tiles per request).  Forced 128: the prefill
    kernel throughout."""
    _run_decode(get_config("c2"), [[1], [1], [17], [5]], tile_rows=tile_rows)


def test_decode_batched_c4():
    """32 requests of 8 shared chunks each; uneven token counts per request and step."""
    wl = get_config("c4")
    rng = np.random.default_rng(4)
    steps = [[1] * wl.batch, [int(x) for x in rng.integers(0, 18, size=wl.batch)]]
    _run_decode(wl, steps, spare_blocks=128)


def test_decode_after_c5_long_context():
    """One request of 131 328 linked tokens (LegoLink-32): a token, then four more."""
    _run_decode(get_config("c5", k=32), [[1], [4]])
