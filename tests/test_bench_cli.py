"""bench.py's command-line contract on the CPU: more than one GPU is refused with a
message (bench.py measures one GPU), and every workload name it offers is one the
configuration table knows."""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=300)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def test_workloads_resolve_to_configs():
    sys.path.insert(0, ROOT)
    import bench
    from synth.configs import get_config

    for name, (cfg, kw) in bench.WORKLOADS.items():
        wl = get_config(cfg, **kw)
        assert wl.name, name
