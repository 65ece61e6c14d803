"""The C ABI driven from plain C: tests/native/c_caller allocates device
memory and a stream with the HIP runtime, commits a seeded warm shard twice
through pact_adamw_commit, takes pact_shard_digest and pact_bf16_digest, and
compares every output bit for bit with the CPU oracle linked into the same
program (no Python, no torch on its side).  Each case runs it as a child
process."""
import os
import subprocess

import pytest

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PROG = os.path.join(ROOT, "tests", "native", "c_caller")


@pytest.mark.parametrize("n,offset,step,seed", [
    (100_003, 6_795_022_080, 5, 3),        # several tiles, ragged tail, indices beyond 2^32
    (1, 0, 1, 1),                          # one element: the element-wise path only
    (3 * 4096 + 5, (1 << 32) - 5000, 100, 2),  # the index range crosses 2^32 inside a tile
    ((1 << 20), 1_140_000_000, 18, 4),     # whole tiles only
])
def test_c_caller_matches_oracle(n, offset, step, seed):
    assert os.path.exists(PROG), "tests/native/c_caller is not built: run make"
    print(f"c_caller n={n} offset={offset} step={step} seed={seed}", flush=True)
    r = subprocess.run([PROG, str(n), str(offset), str(step), str(seed)], capture_output=True, text=True,
                       timeout=120)
    assert r.returncode == 0, f"rc={r.returncode}\nstdout: {r.stdout}\nstderr: {r.stderr}"
    assert r.stdout.startswith("c_caller ok:"), r.stdout
