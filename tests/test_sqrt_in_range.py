"""The short square root of the BF16-state commit, checked on the CPU (no
GPU): for every binary32 input in [2^-96, +inf) and each hardware root the
one-ulp accuracy of v_sqrt_f32 allows there, the residual selection gives the
correctly rounded root (tests/native/sqrt_in_range.c).  The one-ulp bound
itself is a measured property of gfx950; the GPU tests check the commit's
outputs bit for bit against the oracle on both sides of the range."""
import os
import subprocess


def test_selection_is_exact_for_every_input_and_every_allowed_hardware_root(tmp_path):
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    exe = tmp_path / "sqrt_in_range"
    subprocess.run(["gcc", "-O2", "-std=c11", "-fopenmp", "-ffp-contract=off", "-mfma", "-o", str(exe),
                    os.path.join(root, "tests", "native", "sqrt_in_range.c"), "-lm"], check=True)
    r = subprocess.run([str(exe)], capture_output=True, text=True, timeout=600)
    checked, bad = (int(x) for x in r.stdout.split())
    assert checked == 0x7F800000 - 0x0F800000
    assert bad == 0 and r.returncode == 0
