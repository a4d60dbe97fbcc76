"""The measurement probes bench.py reports beside its roofline (not part of the link
step): the streaming-read probe reads every 16-byte word of its buffer exactly once (the
XOR of its per-workgroup outputs equals the XOR of the buffer's words, which fails if a
word is skipped or read twice), and the MFMA probes run to completion with finite sums."""
import ctypes
import os

import numpy as np
import pytest

torch = pytest.importorskip("torch")

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _lib():
    lib = ctypes.CDLL(os.path.join(ROOT, "paper_2410_15332_amd", "probe", "libepic_probe.so"))
    lib.epic_probe_hbm_read.restype = ctypes.c_int
    lib.epic_probe_hbm_read.argtypes = [ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p, ctypes.c_int,
                                        ctypes.c_void_p]
    for name in ("epic_probe_mfma_bf16", "epic_probe_mfma_bf16_varied"):
        fn = getattr(lib, name)
        fn.restype = ctypes.c_int
        fn.argtypes = [ctypes.c_void_p, ctypes.c_int, ctypes.c_int, ctypes.c_void_p]
    return lib


@pytest.mark.parametrize("words16,blocks", [(1, 1), (1000, 7), (65536 + 13, 64), (1 << 22, 4096)])
def test_hbm_read_probe_reads_every_word_once(words16, blocks):
    print(f"[gpu-test] hbm read probe: {words16} x 16 B, {blocks} workgroups", flush=True)
    lib = _lib()
    data = np.random.default_rng(words16).integers(0, 2**31, size=4 * words16, dtype=np.int64).astype(np.int32)
    src = torch.from_numpy(data).cuda()
    out = torch.zeros(blocks, dtype=torch.int32, device="cuda")
    rc = lib.epic_probe_hbm_read(src.data_ptr(), 16 * words16, out.data_ptr(), blocks,
                                 torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    assert rc == 0
    got = np.bitwise_xor.reduce(out.cpu().numpy().view(np.uint32))
    assert got == np.bitwise_xor.reduce(data.view(np.uint32))


@pytest.mark.parametrize("varied", [False, True])
def test_mfma_probe_runs(varied):
    print(f"[gpu-test] mfma probe varied={varied}", flush=True)
    lib = _lib()
    out = torch.full((4 * 512,), float("nan"), dtype=torch.float32, device="cuda")
    fn = lib.epic_probe_mfma_bf16_varied if varied else lib.epic_probe_mfma_bf16
    rc = fn(out.data_ptr(), 4, 64, torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    assert rc == 0
    assert torch.isfinite(out).all()
