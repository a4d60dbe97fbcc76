"""GPU parity of the projection GEMM (epic_gemm) against the oracle's plain
definitions (oracle.projection, float64 on the bf16 operands).

Cases: the four projections of the 32-layer link step (736 rows: whole 192 x 256 and
96 x 128 tiles, 256 x 128 tiles cut along K across workgroups), whole 192-row tiles with row
and column tails, whole 96- and 128-row tiles with row tails, the same projections at a
compile-sized row count (whole-tile rounds plus cut tiles; checked on sampled
rows), row and column tails, tiny shapes, tiles cut into up to 56 parts, the
fallback finish of cut tiles (bit-identical to the polled one), and m = 0.  Bars: fp32 outputs
max |err| <= 1e-4 * s, s = sqrt(K) * sigma_a * sigma_w (the spread of an output;
fp32 accumulation of bf16 products leaves ~1e-6 s); SwiGLU (bf16 output)
|err| <= 2^-8 |ref| + 1e-4 s.
"""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

import oracle  # noqa: E402
import synth  # noqa: E402

pytestmark = pytest.mark.gpu

SEED = 2410153399
EPI = {"store": 0, "residual": 1, "swiglu": 2}


def _dev_bits(bits):
    return torch.from_numpy(bits.view(np.int16)).cuda().view(torch.bfloat16)


def _f64(bits):
    return synth.bf16_bits_to_f32(bits).astype(np.float64)


def _run(m, n, k, epi, tag, sample=None):
    from paper_2410_15332_amd import epic_link as el
    print(f"[gpu-test] gemm m={m} n={n} k={k} {epi}", flush=True)
    sa, sw = 1.0, 1.0 / np.sqrt(k)
    a = synth.matrix_bf16(SEED, 3 * tag, (m, k), sa)
    w = synth.matrix_bf16(SEED, 3 * tag + 1, (n, k), sw)
    ws = torch.empty(el.epic_gemm_workspace_bytes(), dtype=torch.uint8, device="cuda")
    ws.fill_(0xAB)                                      # stale contents must not matter
    da, dw = _dev_bits(a), _dev_bits(w)
    c0 = None
    if epi == "swiglu":
        out = torch.full((m, n // 2), float("nan"), dtype=torch.bfloat16, device="cuda")
        el.epic_gemm(el.GEMM_SWIGLU, da, dw, act=out, workspace=ws)
    else:
        if epi == "residual":
            c0 = synth.matrix_f32(SEED, 3 * tag + 2, (m, n))
            out = torch.from_numpy(c0.copy()).cuda()
        else:
            out = torch.full((m, n), float("nan"), dtype=torch.float32, device="cuda")
        el.epic_gemm(EPI[epi], da, dw, c=out, workspace=ws)
    torch.cuda.synchronize()
    if epi == "swiglu":
        got = synth.bf16_bits_to_f32(out.view(torch.int16).cpu().numpy().view(np.uint16)).astype(np.float64)
    else:
        got = out.cpu().numpy().astype(np.float64)
    rows = np.arange(m) if sample is None else np.asarray(sample)
    ref = oracle.projection(_f64(a[rows]), _f64(w), epi, None if c0 is None else c0[rows].astype(np.float64))
    got = got[rows]
    assert np.all(np.isfinite(got)), "unwritten or non-finite outputs"
    s = np.sqrt(k) * sa * sw
    err = np.abs(got - ref)
    bound = (2.0 ** -8) * np.abs(ref) + 1e-4 * s if epi == "swiglu" else 1e-4 * s
    print(f"[gpu-test]   max|err| {err.max():.3e} (scale {s:.3f})", flush=True)
    assert np.all(err <= bound), f"max err {err.max()} at {np.unravel_index(err.argmax(), err.shape)}"
    return got


LINK = [  # the projections of the Llama-3-8B-shaped link step, 736 S rows
    (736, 6144, 4096, "store"),
    (736, 4096, 4096, "residual"),
    (736, 28672, 4096, "swiglu"),
    (736, 4096, 14336, "residual"),
]


@pytest.mark.parametrize("m,n,k,epi", LINK, ids=[f"{c[3]}_{c[1]}x{c[2]}" for c in LINK])
def test_link_step_projections(m, n, k, epi):
    _run(m, n, k, epi, tag=LINK.index((m, n, k, epi)))


BIG = [  # whole-tile rounds (compile-sized row counts), sampled rows
    (4096, 28672, 4096, "swiglu"),
    (4100, 4224, 1024, "residual"),     # row tail and a column tail inside a 256-wide tile
    (20480, 6144, 4096, "store"),
]


@pytest.mark.parametrize("m,n,k,epi", BIG, ids=[f"{c[3]}_{c[0]}x{c[1]}x{c[2]}" for c in BIG])
def test_large_row_counts_sampled(m, n, k, epi):
    rng = np.random.default_rng(7)
    sample = sorted(set([0, 1, 255, 256, 257, m - 257, m - 256, m - 1] + rng.integers(0, m, 56).tolist()))
    _run(m, n, k, epi, tag=10 + BIG.index((m, n, k, epi)), sample=sample)


TALL = [  # whole tiles of 192 x 256 (fewer rounds x rows than 256 x 256): row and column tails
    (550, 32768, 256, "store"),         # 3 x 128 tiles in 2 rounds of 192; last row tile 166 rows
    (600, 24448, 512, "residual"),      # 4 x 96 tiles, last row tile 24 rows, last tile 128 columns
]


@pytest.mark.parametrize("m,n,k,epi", TALL, ids=[f"{c[3]}_{c[0]}x{c[1]}x{c[2]}" for c in TALL])
def test_192_row_tiles(m, n, k, epi):
    _run(m, n, k, epi, tag=60 + TALL.index((m, n, k, epi)))


WHOLE_NARROW = [  # one round of whole 96 x 128 or 128 x 128 tiles (short K): row tails (n % 128 == 0)
    (760, 4096, 2048, "store"),         # 8 x 32 tiles of 96 rows, last row tile 88 rows
    (700, 4096, 1024, "swiglu"),        # ffn 2048: 8 x 32 tiles of 96 x 64 outputs, last row tile 28 rows
    (800, 4096, 2048, "store"),         # 9 x 32 tiles of 96 rows would be 288: 7 x 32 of 128, last 32 rows
    (200, 14336, 1024, "swiglu"),       # ffn 7168: 2 x 112 tiles of 128 x 64 outputs, last row tile 72 rows
]


@pytest.mark.parametrize("m,n,k,epi", WHOLE_NARROW, ids=[f"{c[3]}_{c[0]}x{c[1]}x{c[2]}" for c in WHOLE_NARROW])
def test_whole_narrow_tiles(m, n, k, epi):
    _run(m, n, k, epi, tag=70 + WHOLE_NARROW.index((m, n, k, epi)))


SMALL = [
    (1, 128, 64, "store"),
    (28, 384, 256, "residual"),
    (200, 768, 512, "store"),
    (255, 384, 640, "swiglu"),          # ffn = 192: 64-column SwiGLU tiles
    (257, 1024, 512, "swiglu"),
    (513, 640, 1536, "residual"),
]


@pytest.mark.parametrize("m,n,k,epi", SMALL, ids=[f"{c[3]}_{c[0]}x{c[1]}x{c[2]}" for c in SMALL])
def test_small_and_ragged(m, n, k, epi):
    _run(m, n, k, epi, tag=20 + SMALL.index((m, n, k, epi)))


MANY = [  # few tiles, long K: a tile cut into 16-56 parts (the last-stage owner waits for all)
    (64, 128, 14336, "residual"),       # 1 tile, 224 K stages over 56 workgroups
    (16, 256, 8192, "store"),           # 2 tiles, 32 parts each
    (1, 128, 4096, "swiglu"),           # one row, one 64-column SwiGLU tile in 16 parts
    (200, 384, 1024, "swiglu"),         # 3 tiles of 4 parts
]


@pytest.mark.parametrize("m,n,k,epi", MANY, ids=[f"{c[3]}_{c[0]}x{c[1]}x{c[2]}" for c in MANY])
def test_tiles_cut_into_many_parts(m, n, k, epi):
    _run(m, n, k, epi, tag=50 + MANY.index((m, n, k, epi)))


CUT = [(736, 6144, 4096, "store"), (736, 4096, 14336, "residual"), (300, 1024, 512, "store"),
       (64, 128, 14336, "residual")]


@pytest.mark.parametrize("m,n,k,epi", CUT, ids=[f"{c[3]}_{c[0]}x{c[1]}x{c[2]}" for c in CUT])
def test_cut_tile_fallback_matches_fast_path(m, n, k, epi, monkeypatch):
    """A cut tile's last-stage owner finishes from its registers once the other parts
    have arrived; with no polls allowed (EPIC_GEMM_FINISH_POLLS=0) it always falls back
    to writing its partial and letting the last to arrive finish.  Both paths sum the
    same partials in the same K order: bit-identical outputs, each within the bar."""
    fast = _run(m, n, k, epi, tag=40 + CUT.index((m, n, k, epi)))
    monkeypatch.setenv("EPIC_GEMM_FINISH_POLLS", "0")
    slow = _run(m, n, k, epi, tag=40 + CUT.index((m, n, k, epi)))
    assert np.array_equal(fast, slow)


def test_repeated_calls_reuse_workspace():
    """Back-to-back calls on one workspace: the split-tile counters are reset."""
    for _ in range(2):
        _run(736, 6144, 4096, "residual", tag=30)     # 256 x 128 tiles cut along K
        _run(300, 1024, 512, "store", tag=31)


def test_empty_and_rejected_shapes():
    from paper_2410_15332_amd import epic_link as el
    ws = torch.empty(el.epic_gemm_workspace_bytes(), dtype=torch.uint8, device="cuda")
    a = torch.zeros((0, 64), dtype=torch.bfloat16, device="cuda")
    w = torch.zeros((128, 64), dtype=torch.bfloat16, device="cuda")
    c = torch.zeros((0, 128), dtype=torch.float32, device="cuda")
    el.epic_gemm(el.GEMM_STORE, a, w, c=c, workspace=ws)          # m = 0: nothing to do
    a = torch.zeros((4, 48), dtype=torch.bfloat16, device="cuda")
    w = torch.zeros((128, 48), dtype=torch.bfloat16, device="cuda")
    with pytest.raises(el.EpicError) as e:                         # k % 64 != 0
        el.epic_gemm(el.GEMM_STORE, a, w, c=torch.zeros((4, 128), device="cuda"), workspace=ws)
    assert e.value.status == 2
    with pytest.raises(el.EpicError) as e:                         # k % 64 != 0
        el.epic_gemm(el.GEMM_STORE, a[:, :32].contiguous(), w[:, :32].contiguous(),
                     c=torch.zeros((4, 128), device="cuda"), workspace=ws)
    assert e.value.status == 2
    a = torch.zeros((4, 64), dtype=torch.bfloat16, device="cuda")
    w = torch.zeros((128, 64), dtype=torch.bfloat16, device="cuda")
    with pytest.raises(el.EpicError) as e:                         # workspace too small
        el.epic_gemm(el.GEMM_STORE, a, w, c=torch.zeros((4, 128), device="cuda"), workspace=ws[:1024])
    assert e.value.status == 4
