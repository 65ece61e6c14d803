"""The recovery protocol with the ranks' shards on the GPU: four rank
processes on cuda:0, each committing its shard through libpactshard (the
fused commit that zeroes the gradient, the gradient guard of phase 2 and the
state digest of phase 3), checked against the oracle's uninterrupted run of
the whole flat vector."""
import os

import pytest

from paper_2609_18178_amd import recovery as rc
from tests.test_recovery import reference_digests

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
M64 = (1 << 64) - 1
NUMEL = 1_000_003  # several tiles and a ragged tail per shard


def _run(tmp_path, shards, faults, updates=4, checkpoint_at=2):
    sv = rc.Supervisor(world=4, shards=shards, layers=32, updates=updates, numel=NUMEL, seed=11,
                       engine="paper_2609_18178_amd.recovery:ShardEngine", checkpoint_at=checkpoint_at,
                       faults=faults, max_restarts=1, deadline=240.0, workdir=str(tmp_path), cwd=ROOT)
    print(f"[gpu-recovery] {shards} shards, faults {faults}", flush=True)
    out = sv.run()
    for c in sv.cohorts:
        print(f"[gpu-recovery] cohort g{c.generation}: exit {c.exit_codes} in {c.seconds:.1f} s", flush=True)
    return sv, out


def _check(sv, out, shards, updates=4):
    ref = reference_digests(shards, NUMEL, 11, updates)
    got = [int(r["state_digest"], 16) for r in out.results]
    for r, d in enumerate(got):
        assert d == ref[r % shards], r
    assert (sum(got[:shards]) & M64) == (sum(ref) & M64)


def test_four_ranks_repair_a_committed_fault_in_memory(tmp_path):
    """Four ranks, one sub-shard each: a fault at the committed boundary of
    update 3 is repaired in place (33 references rebound on the affected
    rank), and the wrapping sum of the four final digests is the oracle's
    digest of the whole vector after the uninterrupted run."""
    sv, out = _run(tmp_path, 4, [{"rank": 1, "site": "committed", "update": 3}])
    assert out.ok and len(sv.cohorts) == 1, (out.exit_codes, sv.log_text(1, 0)[-3000:])
    _check(sv, out, 4)
    for r in out.results:
        assert r["generation"] == 1 and r["replayed_updates"] == 0
        (rep,) = r["repairs"]
        assert rep["rebound_references"] == (33 if r["rank"] == 1 else 0)


def test_torn_commit_on_one_rank_is_rejected_at_agreement(tmp_path):
    """Two shards, two replicas: rank 3's commit of update 3 reaches only half
    of its shard; phase 3 rejects the cohort (every rank exits fenced) and the
    supervisor's restart from the checkpoint ends at the oracle's state."""
    sv, out = _run(tmp_path, 2, [{"rank": 0, "site": "committed", "update": 3},
                                 {"rank": 3, "kind": "torn_commit", "update": 3}])
    first = sv.cohorts[0]
    assert first.exit_codes == [rc.EXIT_FENCED] * 4, [sv.log_text(r, 0)[-1500:] for r in range(4)]
    assert all("torn" in r["why"] for r in first.results)
    assert out.ok and out.generation == 1
    _check(sv, out, 2)


def test_ten_successive_repairs_keep_every_rank_bit_identical(tmp_path):
    """Ten faults at committed boundaries over twelve updates (Sec. IV-G's
    repeated-lifecycle check): ten in-memory repairs with no replay, and
    every rank's final state equals the uninterrupted run's, bit for bit."""
    faults = [{"rank": (3 * k) % 4, "site": "committed", "update": 2 + k} for k in range(10)]
    sv, out = _run(tmp_path, 2, faults, updates=12, checkpoint_at=0)
    assert out.ok and len(sv.cohorts) == 1, (out.exit_codes, sv.log_text(0, 0)[-3000:])
    _check(sv, out, 2, updates=12)
    for r in out.results:
        assert r["generation"] == 10 and r["replayed_updates"] == 0 and len(r["repairs"]) == 10
        assert {x["rebound_references"] for x in r["repairs"]} <= {0, 33}
    # repair-stage times, slowest rank per repair (as the paper reports them)
    for phase in ("guard", "agree", "replace", "rebind", "release"):
        per = [max(r["repairs"][k]["phases_ms"][phase] for r in out.results) for k in range(10)]
        print(f"[gpu-recovery] {phase}: mean {sum(per) / 10:.3f} ms, min {min(per):.3f}, max {max(per):.3f}")
    tot = [max(r["repairs"][k]["total_ms"] for r in out.results) for k in range(10)]
    print(f"[gpu-recovery] guard to release: mean {sum(tot) / 10:.2f} ms, min {min(tot):.2f}, max {max(tot):.2f}")
