"""The in-memory recovery protocol (Sec. III-A, III-C, III-D) over local
processes, without a GPU: ranks hold their shards in host memory and commit
them with the oracle (tests/protocol_engines.py); the control plane and the
replication groups are Gloo on CPU tensors.  Faults are injected in the
data plane (a rank drops out of a collective, so its peers time out) and in
each phase of the protocol."""
import os
import subprocess
import sys
import time

import numpy as np
import pytest

import oracle
import workloads as wl
from paper_2609_18178_amd import recovery as rc

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
ENGINE = "tests.protocol_engines:OracleEngine"
DEADLINES = {"guard": 3.0, "agree": 3.0, "replace": 5.0, "rebind": 2.0, "release": 3.0, "poll": 12.0}
M64 = (1 << 64) - 1


def reference_digests(shards, numel, seed, updates):
    """The uninterrupted run, by the oracle, on the whole flat vector: the
    state digest of each shard after every update is not needed, only the
    final one per shard (shard s covers [s*numel, (s+1)*numel))."""
    n = shards * numel
    p = wl.draw(n, 0, seed, wl.ARRAY_PARAM, 0, wl.NORMAL(0.02))
    m = np.zeros(n, np.float32)
    v = np.zeros(n, np.float32)
    b = np.zeros(n, np.uint16)
    for t in range(1, updates + 1):
        g = wl.draw(n, 0, seed, wl.ARRAY_GRAD, t, wl.NORMAL(1e-3))
        oracle.adamw_commit(p, g, m, v, b, oracle.Hyper(), t)
    return [oracle.state_digest(p[s * numel:(s + 1) * numel], m[s * numel:(s + 1) * numel],
                                v[s * numel:(s + 1) * numel], s * numel) for s in range(shards)]


def supervisor(tmp_path, world=4, shards=2, layers=4, updates=5, numel=3001, faults=(), checkpoint_at=2,
               max_restarts=1, **kw):
    return rc.Supervisor(world=world, shards=shards, layers=layers, updates=updates, numel=numel, seed=11,
                         engine=ENGINE, checkpoint_at=checkpoint_at, faults=list(faults), max_restarts=max_restarts,
                         deadline=120.0, workdir=str(tmp_path), cwd=ROOT, deadlines=dict(DEADLINES),
                         data_timeout=1.0, **kw)


def final_digests(out):
    return [int(r["state_digest"], 16) for r in out.results]


def check_against_reference(sv, out):
    b = sv.base
    ref = reference_digests(b["shards"], b["numel"], b["seed"], b["updates"])
    got = final_digests(out)
    for r, d in enumerate(got):
        assert d == ref[r % b["shards"]], r
    # replicas bit-identical, and the shard digests compose to the whole
    assert (sum(got[:b["shards"]]) & M64) == (sum(ref) & M64)
    for r in out.results:
        assert r["committed_digest"] == r["state_digest"] and r["frontier"] == b["updates"]


# ---------------------------------------------------------------------------
# pieces
# ---------------------------------------------------------------------------

def test_envelope_qualifies_only_committed_failures():
    env = rc.Envelope()
    for phi, act in ((rc.Phi.COMMITTED, rc.Action.L1_PRESERVE), (rc.Phi.FORWARD, rc.Action.L2_RESTART),
                     (rc.Phi.BACKWARD, rc.Action.L2_RESTART)):
        assert env.action(rc.ObservationKey("mi355x-rocm", "hsdp", phi, "continue")) == act
    # a platform-specific entry overrides the wildcard one (Sec. II-C: the
    # same phase can qualify differently on another stack)
    env = rc.Envelope({(rc.ANY, rc.ANY, "committed", rc.ANY): rc.Action.L1_PRESERVE,
                       ("other-stack", rc.ANY, "committed", rc.ANY): rc.Action.L2_RESTART})
    assert env.action(rc.ObservationKey("other-stack", "ddp", rc.Phi.COMMITTED, "x")) == rc.Action.L2_RESTART
    assert env.action(rc.ObservationKey("mi355x-rocm", "ddp", rc.Phi.COMMITTED, "x")) == rc.Action.L1_PRESERVE
    # nothing qualified: fail-stop
    assert rc.Envelope({}).action(rc.ObservationKey("a", "b", rc.Phi.COMMITTED, "c")) == rc.Action.L2_RESTART


def test_rebind_redirects_exactly_the_cached_references():
    old, new, intra, world = object(), object(), object(), object()
    model = rc.build_model(32, old, intra, world)
    t0 = time.perf_counter()
    n = rc.rebind(model, old, new, groups=(intra, world))
    dt = time.perf_counter() - t0
    assert n == 33  # L + 1 (Sec. III-D, 32 layers)
    for w in rc.wrappers(model):
        assert w._inter_node_pg is new
        assert w.process_group is intra and w._handle.process_group is intra
        assert w._exec_order_data.world_group is world
    assert rc.rebind(model, old, new, groups=(intra, world)) == 0  # nothing left to redirect
    assert dt < 0.5
    # a stray reference in nested metadata is found too
    model2 = rc.build_model(2, old, intra, world)
    model2.children[1]._exec_order_data.order.append({"pg": old})
    assert rc.rebind(model2, old, new, groups=(intra, world)) == 4
    assert model2.children[1]._exec_order_data.order[0]["pg"] is new


# ---------------------------------------------------------------------------
# whole cohorts
# ---------------------------------------------------------------------------

def test_fault_free_run_matches_the_oracle(tmp_path):
    sv = supervisor(tmp_path)
    out = sv.run()
    assert out.ok and len(sv.cohorts) == 1, out.exit_codes
    check_against_reference(sv, out)


def test_committed_faults_repair_in_memory_with_no_replay(tmp_path):
    """Three faults at committed boundaries (post-commit metric reduction),
    on different ranks and groups: three in-place repairs, generation 3,
    L + 1 references rebound on the affected ranks, no restart, and the
    final state bit-identical to the uninterrupted run (Sec. IV-G)."""
    faults = [{"rank": 0, "site": "committed", "update": 2}, {"rank": 3, "site": "committed", "update": 3},
              {"rank": 2, "site": "committed", "update": 5}]
    sv = supervisor(tmp_path, faults=faults)
    out = sv.run()
    assert out.ok and len(sv.cohorts) == 1, (out.exit_codes, sv.log_text(0, 0)[-2000:])
    check_against_reference(sv, out)
    for r in out.results:
        assert r["generation"] == 3 and r["replayed_updates"] == 0
        assert [x["frontier"] for x in r["repairs"]] == [2, 3, 5]
        for x, shard in zip(r["repairs"], (0, 1, 0)):
            assert x["affected_shards"] == [shard]
            assert x["rebound_references"] == (5 if r["shard"] == shard else 0)
            assert set(x["phases_ms"]) == {"guard", "agree", "replace", "rebind", "release"}


@pytest.mark.parametrize("site", ["forward", "backward"])
def test_uncommitted_fault_is_rejected_then_restarted_from_checkpoint(tmp_path, site):
    """A failure during forward or backward is outside the qualified
    envelope: every rank exits with the fail-stop rejection, the supervisor
    starts a fresh cohort of the next generation from the checkpoint, which
    replays A = F - C updates and ends bit-identical to the uninterrupted run."""
    sv = supervisor(tmp_path, faults=[{"rank": 1, "site": site, "update": 4}])
    out = sv.run()
    first = sv.cohorts[0]
    assert first.exit_codes == [rc.EXIT_REJECTED] * 4 and not first.killed
    assert out.ok and out.generation == 1
    check_against_reference(sv, out)
    assert all(r["replayed_updates"] == 2 for r in out.results)  # frontier 4, checkpoint 2


@pytest.mark.parametrize("kind", ["raise", "hang"])
@pytest.mark.parametrize("phase", ["guard", "agree", "replace", "rebind", "release"])
def test_failure_in_any_phase_ends_every_rank_within_its_deadline(tmp_path, phase, kind):
    """Safety invariant: an exception or a hang of one rank in phases 2-6
    ends that rank (fail-stop, or its own watchdog), and every peer exits
    non-zero by itself within the deadlines -- nobody resumes alone and the
    supervisor never has to kill a rank."""
    faults = [{"rank": 0, "site": "committed", "update": 2}, {"rank": 1, "phase": phase, "kind": kind}]
    sv = supervisor(tmp_path, world=2, shards=1, updates=3, faults=faults, max_restarts=0)
    out = sv.run()
    assert not out.killed
    assert all(c != rc.EXIT_OK for c in out.exit_codes), out.exit_codes
    assert out.exit_codes[1] == (rc.EXIT_FAILSTOP if kind == "raise" else rc.EXIT_TIMEOUT)
    budget = DEADLINES[phase] + DEADLINES["release"] + DEADLINES["agree"] + 15.0
    assert out.seconds < budget


def test_stale_generation_is_fenced(tmp_path):
    faults = [{"rank": 0, "site": "committed", "update": 2}, {"rank": 3, "kind": "stale_generation"}]
    sv = supervisor(tmp_path, faults=faults, max_restarts=0)
    out = sv.run()
    assert out.exit_codes == [rc.EXIT_FENCED] * 4
    assert all("stale rank fenced" in r["why"] for r in out.results)


def test_frontier_mismatch_aborts(tmp_path):
    faults = [{"rank": 2, "site": "committed", "update": 3}, {"rank": 1, "kind": "frontier_mismatch"}]
    sv = supervisor(tmp_path, faults=faults, max_restarts=0)
    out = sv.run()
    assert out.exit_codes == [rc.EXIT_FENCED] * 4
    assert all("frontier" in r["why"] for r in out.results)


def test_torn_commit_is_rejected_at_agreement_and_restarted(tmp_path):
    """A commit that reached only half of a rank's shard while its host side
    carried on: the rank's state digest no longer equals the digest of its
    commit, phase 3 rejects the cohort, and the restart from the checkpoint
    ends bit-identical to the uninterrupted run."""
    faults = [{"rank": 0, "site": "committed", "update": 3}, {"rank": 3, "kind": "torn_commit", "update": 3}]
    sv = supervisor(tmp_path, faults=faults)
    out = sv.run()
    first = sv.cohorts[0]
    assert first.exit_codes == [rc.EXIT_FENCED] * 4
    assert all("torn" in r["why"] for r in first.results)
    assert out.ok
    check_against_reference(sv, out)


def test_outstanding_gradient_fails_the_guard(tmp_path):
    faults = [{"rank": 0, "site": "committed", "update": 2}, {"rank": 2, "kind": "outstanding_grad"}]
    sv = supervisor(tmp_path, faults=faults, max_restarts=0)
    out = sv.run()
    assert out.exit_codes[2] == rc.EXIT_FAILSTOP and "outstanding" in out.results[2]["why"]
    assert all(c != rc.EXIT_OK for c in out.exit_codes) and not out.killed


def test_a_rank_of_an_old_generation_cannot_join(tmp_path):
    """Generation fencing at the rendezvous: each cohort meets on a control
    plane of its own generation, so a rank started for a generation whose
    cohort is gone never assembles a world and exits non-zero by itself."""
    sv = supervisor(tmp_path, world=2, shards=1, updates=2, checkpoint_at=0, control_timeout=3.0)
    out = sv.run()
    assert out.ok
    spec = os.path.join(str(tmp_path), "spec_g0.json")
    env = dict(os.environ, GLOO_SOCKET_IFNAME="lo")
    t0 = time.monotonic()
    r = subprocess.run([sys.executable, "-m", "paper_2609_18178_amd.recovery", "--spec", spec, "--rank", "1"],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=120)
    assert r.returncode != 0
    assert time.monotonic() - t0 < 100


def test_break_even_model_reproduces_the_papers_worked_example():
    """Pin: eq. (4) of Sec. III-B evaluated on the paper's inputs gives the
    figures it prints for them (tests/golden/break_even_example.txt), each to
    the precision printed."""
    g = {}
    with open(os.path.join(ROOT, "tests", "golden", "break_even_example.txt")) as f:
        for line in f:
            if line.strip() and not line.startswith("#"):
                k, v = line.split()
                g[k] = float(v)
    S = rc.saving_per_recovery(g["age_updates"], g["update_seconds"], g["repair_seconds"])
    assert abs(S - g["saving_seconds"]) < 0.05
    guard = g["guard_overhead"] * g["baseline_seconds"]
    assert abs(guard - g["daily_guard_cost_seconds"]) < 0.05
    days = rc.break_even_interval(S, g["guard_overhead"]) / 86400.0
    assert abs(days - g["break_even_days"]) < 0.1
    for pct, key in ((0.02, "2pct"), (0.10, "10pct")):
        rate = pct * g["interruptions_per_day"]
        assert abs(rate - g[f"eligible_per_day_at_{key}"]) < 0.0006
    # the paper carries the event rates rounded to three decimals
    rate2 = g["eligible_per_day_at_2pct"]
    assert abs(1.0 / (0.02 * g["interruptions_per_day"]) - g["days_per_incident_at_2pct"]) < 0.01
    assert abs(rate2 * S - g["daily_saving_at_2pct_seconds"]) < 0.1
    assert abs(rate2 * S / guard - g["offset_fraction_at_2pct"]) < 0.001
    rate10 = g["eligible_per_day_at_10pct"]
    gross = rc.net_saving(rate10, S, 0, 0, 0, 0)
    assert abs(gross - g["daily_gross_saving_at_10pct_seconds"]) < 0.15
    net = rc.net_saving(rate10, S, 0, 0.1, g["guard_overhead"], g["baseline_seconds"])
    assert abs(net - g["daily_net_saving_at_10pct_seconds"]) < 0.15
    assert abs(net / guard - g["net_over_guard_cost_at_10pct"]) < 0.05
    # rejections cost C each: C < 0.1 s (Sec. III-B) barely moves the balance
    assert rc.net_saving(rate10, S, 5, 0.1, g["guard_overhead"], g["baseline_seconds"]) == pytest.approx(net - 0.5)
