"""The short first mixing round of the digests of 16-bit words (the BF16
state and the bf16 working copy), checked on the CPU (no GPU): for every
value of index bits 16..31 that passes its two carry conditions and every
16-bit word, the short form gives the definition's first round, and exactly
four values of those bits fail the conditions (tests/native/index_lo16.c).
The GPU tests check the kernels' digests bit for bit against the oracle on
tiles of every index form."""
import os
import subprocess


def test_short_round_matches_the_definition_for_every_word(tmp_path):
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    exe = tmp_path / "index_lo16"
    subprocess.run(["gcc", "-O2", "-std=c11", "-fopenmp", "-o", str(exe),
                    os.path.join(root, "tests", "native", "index_lo16.c")], check=True)
    r = subprocess.run([str(exe)], capture_output=True, text=True, timeout=600)
    checked, bad, failing = (int(x) for x in r.stdout.split())
    assert failing == 4
    assert checked == (65536 - 4) * (65536 + 64 * 4)
    assert bad == 0 and r.returncode == 0
