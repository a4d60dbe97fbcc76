"""The link step captured in a HIP graph: the library launches only kernels on the
caller's stream, allocates nothing and never synchronises, so one call can be
captured and replayed.  Each replay must give exactly the eager result (the
kernels are deterministic: fixed summation orders, no atomics on values), also
with eager work and host synchronisation between the replays, and after the
outputs were overwritten."""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

from synth.configs import ModelWorkload, get_config  # noqa: E402

pytestmark = pytest.mark.gpu


def _bits(t):
    return t.detach().cpu().view(torch.int16).numpy().view(np.uint16) if t.dtype == torch.bfloat16 \
        else t.detach().cpu().numpy()


def _replays(st, outs, reset, n=3):
    from paper_2410_15332_amd import harness
    st.run()
    torch.cuda.synchronize()
    ref = [_bits(x).copy() for x in outs()]
    g = harness.capture_graph(st.run)
    for i in range(n):
        reset()                                   # eager work between replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for r, x in zip(ref, outs()):
            assert np.array_equal(r, _bits(x)), f"replay {i} differs from the eager step"
        st.run()                                  # an eager step between replays
        torch.cuda.synchronize()
    return ref


def test_attention_step_graph_replays():
    from paper_2410_15332_amd import harness
    print("[gpu-test] graph: c2 attention step", flush=True)
    st = harness.stage_attention(get_config("c2"))
    _replays(st, lambda: [st.out, st.lse, st.k_cache, st.v_cache],
             lambda: (st.out.zero_(), st.lse.fill_(-1.0)))


def test_attention_step_graph_replays_split_kv():
    from paper_2410_15332_amd import harness
    print("[gpu-test] graph: c5 k=0 (split-KV partials and combine)", flush=True)
    st = harness.stage_attention(get_config("c5", k=0))
    assert st.sizes.n_partials > 0
    _replays(st, lambda: [st.out, st.lse], lambda: (st.out.zero_(), st.lse.zero_()))


def test_model_step_graph_replays():
    """Model level: the 128-row projections cut tiles along K, so this also replays the
    GEMM's partial sums and arrival counters (cleared by a kernel each call)."""
    from paper_2410_15332_amd import harness
    print("[gpu-test] graph: small model link step", flush=True)
    wl = ModelWorkload("graph_small", 41, 2, 512, 1024, 8, 2, 64, 16, 500000.0, 1e-5, [37, 100, 51], 23, 5)
    st = harness.stage_model(wl, caches="compile")
    _replays(st, lambda: [st.out, st.k_caches[1]], lambda: st.out.zero_())


def test_decode_step_graph_replays():
    """Decode after the link step (16-row tiles, split-KV partials and the combine)."""
    import types

    from paper_2410_15332_amd import harness
    print("[gpu-test] graph: c2 decode step", flush=True)
    wl = get_config("c2")
    st = harness.stage_attention(wl, spare_blocks=4 * wl.batch)
    st.run()
    ds = harness.stage_decode(wl, st.cfg, st.sizes, st.dplan.host, st.spare, st.num_blocks, [1] * wl.batch)
    assert ds.sizes.tile_rows == 16 and ds.sizes.n_partials > 0
    step = types.SimpleNamespace(run=lambda: ds.run(st.k_cache, st.v_cache))
    _replays(step, lambda: [ds.out, ds.lse, st.k_cache, st.v_cache], lambda: (ds.out.zero_(), ds.lse.zero_()))
