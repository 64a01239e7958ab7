"""bench.py's command-line contract without a GPU: more than one GPU is
refused with a message (the library measures one GPU), and the byte counts
that the roofline uses are the algorithmic ones of the 7B shape."""
import os
import subprocess
import sys

import jf_inputs

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""


def test_roofline_bytes_are_algorithmic():
    sys.path.insert(0, ROOT)
    import bench
    shape = jf_inputs.MODEL_SHAPES["7b"]
    # gate/up: both 18944 x 3584 bf16 matrices once, 16 x 3584 activations
    # in and 16 x 18944 SwiGLU outputs, each at bf16 size (the second bf16
    # plane of the activations is 0.04% more and not counted)
    assert bench.gateup_bytes(shape, 16) == 2 * 18944 * 3584 * 2 + 16 * 3584 * 2 + 16 * 18944 * 2
    assert bench.gateup_bytes(shape, 16) == 272302080
