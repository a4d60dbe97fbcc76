"""Run the co-execution probe (coexec.hip in the probe library) and print, per
variant, the shader cycles per iteration of 8 MFMA slots and the engine clock.
Modes: accumulators in AGPRs or VGPRs, and 4, 2 or 1 independent accumulator chains.

    python -m paper_2410_15332_amd.probe.coexec
"""
import ctypes
import os

VARIANTS = [(1, 0, 0), (0, 32, 0), (0, 32, 1), (0, 32, 2),
            (1, 16, 0), (1, 32, 0), (1, 48, 0), (1, 64, 0), (1, 8, 1), (1, 16, 1), (1, 32, 1), (1, 16, 2), (1, 32, 2),
            (2, 0, 0), (2, 32, 0), (2, 48, 0), (2, 16, 1), (2, 32, 1),
            (3, 0, 0), (3, 32, 0), (4, 0, 0), (4, 32, 0)]
KINDS = {0: "fma", 1: "exp", 2: "max"}
MODES = {0: "no mfma              ", 1: "8 mfma (AGPR acc, 4) ", 2: "8 mfma (VGPR acc, 4) ",
         3: "8 mfma (AGPR acc, 2) ", 4: "8 mfma (AGPR acc, 1) "}


def main():
    import torch

    lib = ctypes.CDLL(os.path.join(os.path.dirname(os.path.abspath(__file__)), "libepic_probe.so"))
    lib.epic_probe_coexec.restype = ctypes.c_int
    lib.epic_probe_coexec.argtypes = [ctypes.c_int] * 4 + [ctypes.c_void_p] * 3
    iters = lib.epic_probe_coexec_iters()
    n_cu = torch.cuda.get_device_properties(0).multi_processor_count
    for per_simd in (1, 2):
        blocks = n_cu * per_simd
        out = torch.empty(blocks * 256, dtype=torch.float32, device="cuda")
        cyc = torch.zeros(blocks * 8, dtype=torch.int64, device="cuda")
        for mfma, nv, kind in VARIANTS:
            for _ in range(2):                      # warm-up launch, then the measured one
                rc = lib.epic_probe_coexec(mfma, nv, kind, blocks, out.data_ptr(), cyc.data_ptr(),
                                           torch.cuda.current_stream().cuda_stream)
                if rc != 0:
                    raise RuntimeError(f"co-execution probe failed: {rc}")
            torch.cuda.synchronize()
            c = cyc.view(-1, 2).double()
            cycles, ticks = c[:, 0].mean().item(), c[:, 1].mean().item()
            label = f"{MODES[mfma]}+ {nv:2d} {KINDS[kind]}"
            print(f"{label}  waves/SIMD={per_simd}: {cycles / iters:7.1f} cycles/iter "
                  f"({cycles / iters / 8:5.1f} per MFMA slot)  clock {cycles / (ticks * 10.0):.2f} GHz", flush=True)


if __name__ == "__main__":
    main()
