"""Run the load-path probe (load_path.hip in the probe library) and print, per
access shape, prefetch depth and region sharing, the bytes per second each CU
pulls through buffer loads.

    python -m paper_2410_15332_amd.probe.load_path
"""
import ctypes
import os

SHAPES = {0: "LDS 4 x 32 KB, 16 rows x 64 B", 1: "LDS 4 x 32 KB, 8 rows x 128 B", 2: "LDS 4 x 32 KB, 1 KB contiguous",
          3: "LDS 4 x 32 KB, 16 rows x 64 B in line pairs", 4: "VGPR 4 x 32 KB, 16 rows x 64 B",
          5: "VGPR 4 x 32 KB, 8 rows x 128 B", 6: "LDS 2 x 16 KB, 8 rows x 128 B", 7: "LDS 2 x 32 KB, 8 rows x 128 B",
          8: "LDS 2 x 64 KB, 8 rows x 128 B", 9: "LDS 1 x 64 KB (drained), 8 rows x 128 B"}
SHARING = {4: "4 regions per XCD (8 CUs of an XCD per region)", -4: "4 regions, each read on all 8 XCDs",
           -32: "32 regions, each on 8 XCDs, 1 CU per XCD", 32: "256 regions, one per CU"}
PASS_BYTES = 8 << 20        # bytes each workgroup streams per measured launch


def main():
    import torch

    lib = ctypes.CDLL(os.path.join(os.path.dirname(os.path.abspath(__file__)), "libepic_probe.so"))
    lib.epic_probe_load_path.restype = ctypes.c_int
    lib.epic_probe_load_path.argtypes = [ctypes.c_int, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int, ctypes.c_int,
                                         ctypes.c_void_p, ctypes.c_void_p]
    src = torch.randn(256 << 20, device="cuda")          # 1 GB: 256 regions of 4 MB
    sink = torch.zeros(256, device="cuda")
    stream = torch.cuda.current_stream().cuda_stream
    cases = [(v, 4) for v in range(10)] + [(v, r) for r in (-4, -32, 32) for v in (0, 1)]
    for variant, regions in cases:
        stage = lib.epic_probe_load_path_stage_bytes(variant)
        steps = PASS_BYTES // stage
        for _ in range(2):                               # warm-up, then 5 timed launches
            if lib.epic_probe_load_path(variant, src.data_ptr(), src.numel() * 4, regions, steps,
                                        sink.data_ptr(), stream) != 0:
                raise RuntimeError("load-path probe rejected its arguments")
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(5):
            lib.epic_probe_load_path(variant, src.data_ptr(), src.numel() * 4, regions, steps, sink.data_ptr(), stream)
        e1.record()
        torch.cuda.synchronize()
        us = e0.elapsed_time(e1) / 5 * 1e3
        per_cu = steps * stage / us / 1e3
        print(f"{SHAPES[variant]:44s} | {SHARING[regions]:46s} | {us:7.1f} us | {per_cu:6.1f} GB/s per CU | "
              f"{per_cu * 256 / 1e3:5.1f} TB/s", flush=True)


if __name__ == "__main__":
    main()
