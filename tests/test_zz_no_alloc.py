"""The no-allocation attention entry point (epic_link_attention_noalloc) against
epic_link_attention with a caller workspace: two calls in a row on the library's
fixed scratch array, the second with a smaller plan, each bit-identical to the
workspace entry point on the same inputs (same kernels, same plan), including
the linked cache; and a plan whose partials exceed the array is rejected on the
host before anything is enqueued."""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

from synth.configs import AttnWorkload, get_config  # noqa: E402

pytestmark = pytest.mark.gpu


def _stage(wl, **kw):
    from paper_2410_15332_amd import harness
    print(f"[gpu-test] staging {wl.name} k={wl.k} {kw}", flush=True)
    return harness.stage_attention(wl, **kw)


def _run_both(st):
    """Workspace entry point first, then the no-allocation one on fresh outputs and a
    fresh copy of the caches; returns both results."""
    from paper_2410_15332_amd import epic_link as el
    k0, v0 = st.k_cache.clone(), st.v_cache.clone()
    st.run()
    torch.cuda.synchronize()
    ref = (st.out.clone(), st.lse.clone(), st.k_cache.clone(), st.v_cache.clone())
    st.k_cache.copy_(k0)
    st.v_cache.copy_(v0)
    st.out.fill_(float("nan"))
    st.lse.fill_(float("nan"))
    el.epic_link_attention_noalloc(st.cfg, st.dplan, st.q_s, st.k_s, st.v_s, st.k_cache, st.v_cache, st.out,
                                   st.lse)
    torch.cuda.synchronize()
    return ref, (st.out, st.lse, st.k_cache, st.v_cache)


def test_noalloc_matches_workspace_entry_point_twice():
    from paper_2410_15332_amd import epic_link as el
    big = _stage(get_config("c5", k=32))
    small = _stage(get_config("c2"))
    need_big = el.epic_link_workspace_bytes(big.cfg, big.sizes)
    need_small = el.epic_link_workspace_bytes(small.cfg, small.sizes)
    assert 0 < need_small < need_big <= el.NOALLOC_SCRATCH_BYTES, (need_small, need_big)
    for st in (big, small):
        ref, got = _run_both(st)
        for name, a, b in zip(("out", "lse", "k_cache", "v_cache"), ref, got):
            assert torch.equal(a, b), f"{st.wl.name}: {name} differs from the workspace entry point"
        print(f"[gpu-test] {st.wl.name}: no-allocation entry point bit-identical "
              f"({el.epic_link_workspace_bytes(st.cfg, st.sizes) / 2**20:.1f} MiB of partials)", flush=True)


def test_noalloc_rejects_plans_beyond_the_scratch_array():
    from paper_2410_15332_amd import epic_link as el
    wl = AttnWorkload("many_partials", 5, 32, 8, 128, 16, [list(range(64))], [2048] * 64, [256], 32)
    st = _stage(wl, split_blocks=4)
    assert el.epic_link_workspace_bytes(st.cfg, st.sizes) > el.NOALLOC_SCRATCH_BYTES
    before = st.out.clone()
    with pytest.raises(el.EpicError) as e:
        el.epic_link_attention_noalloc(st.cfg, st.dplan, st.q_s, st.k_s, st.v_s, st.k_cache, st.v_cache, st.out,
                                       st.lse)
    assert e.value.status == 4 and "scratch" in str(e.value)
    torch.cuda.synchronize()
    assert torch.equal(before, st.out)
