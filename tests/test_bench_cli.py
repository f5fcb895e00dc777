"""Host-side checks of bench.py's command line (no GPU is touched): more than
one GPU is refused with a message, and the workload table it reports from
matches the useful-FLOP formula 2 B C_out C_in N_B^2 d_f^k d_out^k."""
import os
import subprocess
import sys

import workloads as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120, cwd=ROOT)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""


def test_useful_flops_formula():
    for w in W.WORKLOADS.values():
        for s in w.layers:
            nb = 1 << s.k
            d_out = s.d_image - s.d_filter + 1
            expect = 2 * s.B * s.C_out * s.C_in * nb * nb * s.d_filter ** s.k * d_out ** s.k
            assert s.useful_flops() == expect, (w.name, s)
