"""The C-ABI library loads without a GPU and exports every entry point the header declares."""
import ctypes
import os
import re

from paper_2410_15332_amd import epic_link as el

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    names = []
    for fn in os.listdir(os.path.join(ROOT, "include")):
        if fn.endswith(".h"):
            text = open(os.path.join(ROOT, "include", fn)).read()
            text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
            names += re.findall(r"^[A-Za-z_][\w\s\*]*?\b(epic_\w+)\s*\(", text, flags=re.M)
    return sorted(set(names))


def test_header_declares_entry_points():
    d = _declared()
    for name in ("epic_plan_link", "epic_link_attention", "epic_link_layer", "epic_link_model"):
        assert name in d


def test_library_exports_every_declared_symbol():
    lib = ctypes.CDLL(el._LIB_PATH)
    missing = [n for n in _declared() if not hasattr(lib, n)]
    assert not missing, missing
    assert sorted(el.EXPORTED) == _declared()


def test_status_strings_and_version():
    assert el.epic_status_string(0) == "ok"
    assert "workspace" in el.epic_status_string(4)
    assert "gfx950" in el.epic_version()


def test_workspace_bytes_scale_with_partials():
    cfg = el.attn_cfg(32, 8, 128, 0.0, 8)
    reqs = [el.Request([512] * 4, [list(range(32 * j, 32 * j + 32)) for j in range(4)], 64, 16)]
    s = el.epic_plan_sizes_get(reqs, cfg, 1000)
    assert s.n_partials > 0
    assert el.epic_link_workspace_bytes(cfg, s) >= s.n_partials * 8 * 128 * (128 + 1) * 4


def test_probe_library_exports_what_bench_calls():
    """The measurement probes (built beside the product library, never linked into
    it) load without a GPU, export the entry points bench.py binds, and reject bad
    arguments on the host before any launch."""
    lib = ctypes.CDLL(os.path.join(ROOT, "paper_2410_15332_amd", "probe", "libepic_probe.so"))
    for name in ("epic_probe_mfma_bf16", "epic_probe_mfma_bf16_varied", "epic_probe_mfma_bf16_flops",
                 "epic_probe_hbm_read", "epic_probe_coexec", "epic_probe_coexec_iters", "epic_probe_load_path",
                 "epic_probe_load_path_stage_bytes"):
        assert hasattr(lib, name), name
    lib.epic_probe_coexec.restype = ctypes.c_int
    lib.epic_probe_coexec.argtypes = [ctypes.c_int] * 4 + [ctypes.c_void_p] * 3
    assert lib.epic_probe_coexec(1, 32, 1, 256, None, None, None) != 0       # no buffers
    assert lib.epic_probe_coexec(1, 24, 1, 256, 16, 16, None) != 0           # not a built variant
    lib.epic_probe_mfma_bf16_flops.restype = ctypes.c_double
    lib.epic_probe_mfma_bf16_flops.argtypes = [ctypes.c_int, ctypes.c_int]
    assert lib.epic_probe_mfma_bf16_flops(2, 3) == 2 * 8 * 3 * 4 * 2.0 * 32 * 32 * 16
    lib.epic_probe_mfma_bf16_varied.restype = ctypes.c_int
    lib.epic_probe_mfma_bf16_varied.argtypes = [ctypes.c_void_p, ctypes.c_int, ctypes.c_int, ctypes.c_void_p]
    assert lib.epic_probe_mfma_bf16_varied(None, 1, 8, None) != 0          # no output buffer
    lib.epic_probe_hbm_read.restype = ctypes.c_int
    lib.epic_probe_hbm_read.argtypes = [ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p, ctypes.c_int,
                                        ctypes.c_void_p]
    assert lib.epic_probe_hbm_read(None, 16, None, 1, None) != 0            # no buffers
    lib.epic_probe_load_path.restype = ctypes.c_int
    lib.epic_probe_load_path.argtypes = [ctypes.c_int, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int, ctypes.c_int,
                                         ctypes.c_void_p, ctypes.c_void_p]
    assert lib.epic_probe_load_path_stage_bytes(1) == 32768
    assert lib.epic_probe_load_path_stage_bytes(10) == -1                  # no such variant
    assert lib.epic_probe_load_path(0, None, 1 << 30, 4, 256, 16, None) != 0       # no source
    assert lib.epic_probe_load_path(0, 16, 1 << 30, 4, 254, 16, None) != 0         # steps not a multiple of 4
    assert lib.epic_probe_load_path(0, 16, 64 << 20, 4, 256, 16, None) != 0        # source smaller than 32 regions
    assert lib.epic_probe_load_path(11, 16, 1 << 30, 4, 256, 16, None) != 0        # no such variant
