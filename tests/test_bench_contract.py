"""Host-side checks of bench.py's contract that need no GPU: more than one GPU
is refused with a message, and the algorithmic flop counts it prices the
edge kernel with follow their closed forms."""
import os
import subprocess
import sys

import bench

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout.strip() == ""


def test_edge_kernel_flops_closed_form():
    # per edge: projection 2RdC, the harmonics/radial products 2Rd + 17R and
    # the Hadamard multiply-add RC; per node: the output factor 2dRC
    N, E, d, C, R = 3200, 151118, 25, 128, 128
    per_edge = 2 * R * d * C + 2 * R * d + 17 * R + R * C
    assert bench.edge_kernel_flops(N, E, d, C, R) == E * per_edge + N * 2 * d * R * C
    assert bench.forward_flops(N, E, d, C, R) == bench.edge_kernel_flops(N, E, d, C, R) + N * 2 * d * C * C
