"""MI355X (gfx950) link step of LegoLink position-independent caching (EPIC, arXiv 2410.15332).

The compute path is libepic_link.so (C ABI in include/epic_link.h): a host
planner in C++ and HIP kernels for gfx950.  ``epic_link`` is its ctypes binding
(same names as the C entry points); ``build`` compiles the library;
``harness`` stages seeded synthetic workloads in device memory for the tests and
the benchmark.  Import ``paper_2410_15332_amd.epic_link`` explicitly: it raises
ImportError when the library is not built.
"""

__all__ = ["epic_link", "build", "harness"]
