"""Host-side logic of bench.py (no GPU): the one-GPU guard and the counter
records it turns rocprofv3 CSV output into."""
import csv
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402
import workloads as wl  # noqa: E402

N = wl.WORKLOADS["mistral7b_shard16"].numel
FIELDS = ["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value", "Start_Timestamp", "End_Timestamp"]


def _write_csv(path, rows):
    with open(path, "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=FIELDS)
        w.writeheader()
        for r in rows:
            w.writerow(r)


@pytest.fixture()
def sandbox(tmp_path, monkeypatch):
    (tmp_path / "profiles").mkdir()
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    monkeypatch.setattr(bench, "kernel_source_hash", lambda: "feedfacecafebeef")
    return tmp_path


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "4"], capture_output=True, text=True)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""


def test_record_traffic_scales_by_the_probe(sandbox):
    # the probe moves exactly 16 B read and 14 B written per element; the
    # fetch counter is made to read half of that, the write counter 1.25x
    probe_f, probe_w = 16.0 * N / 2 / 1024, 14.0 * N * 1.25 / 1024
    commit_f, commit_w = 16.5 * N / 2 / 1024, 14.0 * N * 1.25 / 1024
    fetch = [{"Dispatch_Id": i, "Kernel_Name": name, "Counter_Name": "FETCH_SIZE", "Counter_Value": val,
              "Start_Timestamp": 0, "End_Timestamp": 1}
             for i, (name, val) in enumerate([("void pact::tile_kernel<(pact::Mode)0>(x)", commit_f),
                                              ("pact::probe_kernel(float const*)", probe_f),
                                              ("void pact::tile_kernel<(pact::Mode)0>(x)", commit_f)])]
    write = [dict(r, Counter_Name="WRITE_SIZE", Counter_Value=(commit_w if "Mode" in r["Kernel_Name"] else probe_w))
             for r in fetch]
    _write_csv(sandbox / "f.csv", fetch)
    _write_csv(sandbox / "w.csv", write)
    rec = bench.record_traffic("mistral7b_shard16", str(sandbox / "f.csv"), str(sandbox / "w.csv"))
    assert rec["fetch_scale"] == pytest.approx(2.0)
    assert rec["write_scale"] == pytest.approx(0.8)
    assert rec["fetch_bytes_per_launch"] == pytest.approx(16.5 * N)
    assert rec["write_bytes_per_launch"] == pytest.approx(14.0 * N)
    assert rec["commit_dispatches"] == [2, 2]
    stored = json.load(open(sandbox / "profiles" / "traffic_mistral7b_shard16.json"))
    assert stored["bytes_per_launch"] == pytest.approx(30.5 * N)
    assert bench.stored_traffic("mistral7b_shard16", "feedfacecafebeef")["bytes_per_launch"] == pytest.approx(30.5 * N)
    assert bench.stored_traffic("mistral7b_shard16", "0000000000000000") is None


def test_record_clock(sandbox):
    rows = []
    # two commit dispatches of 2 ms at 1.5 GHz on each of the 8 XCDs, 108 VALU
    # instructions per element; one probe dispatch at 2.4 GHz
    for d, (name, dur_ns, ghz, per_elem) in enumerate([("void pact::tile_kernel<(pact::Mode)0>(a)", 2_000_000, 1.5, 108),
                                                       ("void pact::tile_kernel<(pact::Mode)0>(a)", 2_000_000, 1.5, 108),
                                                       ("pact::probe_kernel(float const*)", 2_000_000, 2.4, 2)]):
        cycles = ghz * dur_ns
        valu = per_elem * N / 64
        for cname, val in (("GRBM_GUI_ACTIVE", cycles * 8), ("SQ_INSTS_VALU", valu), ("SQ_ACTIVE_INST_VALU", valu)):
            rows.append({"Dispatch_Id": d, "Kernel_Name": name, "Counter_Name": cname, "Counter_Value": val,
                         "Start_Timestamp": 1000, "End_Timestamp": 1000 + dur_ns})
    _write_csv(sandbox / "c.csv", rows)
    rec = bench.record_clock("mistral7b_shard16", str(sandbox / "c.csv"))
    c = rec["kernels"]["commit"]
    assert c["dispatches"] == 2
    assert c["us"] == pytest.approx(2000.0)
    assert c["clock_ghz"] == pytest.approx(1.5)
    assert c["valu_instr_per_element"] == pytest.approx(108.0)
    assert c["valu_issue_per_cu_cycle"] == pytest.approx(108 * N / 64 / 256 / 3.0e6)
    assert c["valu_busy_pct"] == pytest.approx(100 * c["valu_issue_per_cu_cycle"])
    assert c["gbps"] == pytest.approx(30 * N / 2e-3 / 1e9)
    assert rec["kernels"]["probe"]["clock_ghz"] == pytest.approx(2.4)
    assert bench.stored_clock("mistral7b_shard16", "feedfacecafebeef")["kernels"]["commit"]["dispatches"] == 2
    assert bench.stored_clock("mistral7b_shard16", "0123456789abcdef") is None


def test_oracle_replay_matches_a_direct_run_and_sees_a_wrong_digest():
    """The in-run parity replay (chunked, threaded) equals the oracle run as
    one plain sequence over the whole shard, and reports a mismatch."""
    from dataclasses import replace

    import numpy as np

    import oracle

    w = replace(wl.WORKLOADS["decoder1b_shard16"], numel=300_007)
    p, g, m, v = wl.arrays_host(w)
    b = np.zeros(w.numel, np.uint16)
    h = oracle.Hyper(**w.hypers[0])
    for st in (100, 101):
        oracle.adamw_commit(p, g, m, v, b, h, st)
    d = oracle.commit_and_digest(p, g, m, v, b, h, 102, w.global_offset)
    r = bench.oracle_replay(w, [100, 101, 102], d, threads=3, chunk=100_000)
    assert r["match"] and r["oracle_digest"] == f"{d:#018x}"
    assert not bench.oracle_replay(w, [100, 101, 102], d ^ 1, threads=2, chunk=70_001)["match"]
    assert not bench.oracle_replay(w, [100, 101], d, threads=2)["match"]
