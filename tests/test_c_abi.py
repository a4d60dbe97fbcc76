"""The boundary is a C ABI: the header compiles as C99 and C++17, and a C program
linked against libepic_link plans a request through the host entry points (no GPU
needed) and gets the selection the paper defines (Sec. 4.2: the first k tokens of
every chunk but the first, plus the suffix)."""
import os
import shutil
import subprocess

import pytest

import oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
INCLUDE = os.path.join(ROOT, "include")
LIBDIR = os.path.join(ROOT, "paper_2410_15332_amd")

needs_gcc = pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc not available")


@needs_gcc
@pytest.mark.parametrize("lang,std", [("c", "c99"), ("c++", "c++17")])
def test_header_compiles(lang, std):
    cc = "gcc" if lang == "c" else "g++"
    r = subprocess.run([cc, f"-std={std}", "-Wall", "-Wextra", "-Werror", "-fsyntax-only", "-x", lang,
                        os.path.join(INCLUDE, "epic_link.h")], capture_output=True, text=True)
    assert r.returncode == 0, r.stderr


@needs_gcc
def test_plan_from_c(tmp_path):
    exe = str(tmp_path / "plan_from_c")
    r = subprocess.run(["gcc", "-std=c99", "-Wall", "-Werror", f"-I{INCLUDE}",
                        os.path.join(ROOT, "tests", "c", "plan_from_c.c"), f"-L{LIBDIR}", "-lepic_link",
                        f"-Wl,-rpath,{LIBDIR}", "-o", exe], capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    r = subprocess.run([exe], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stderr
    lines = r.stdout.strip().split("\n")
    s_pos = [int(x) for x in lines[1].split()]
    assert s_pos == oracle.legolink_positions([20, 18, 5], 3, 2).tolist()
    assert lines[0] == f"n_s {len(s_pos)} n_private 3"
    # chunk 1's first block keeps cached rows (copied from block 2), chunk 2's single
    # block keeps 3 cached rows (from block 4), the suffix block is fresh
    assert lines[2].split() == ["5:2", "6:4", "7:-1"]
    assert lines[3].startswith("bad 1 ")
