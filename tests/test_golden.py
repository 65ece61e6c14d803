"""Fixtures under tests/golden/: published test vectors (each file cites its
source) and digests of small seeded workloads written by
tests/golden/make_digests.py from the oracle alone.  No GPU."""
import json
import os

import numpy as np

import oracle
import workloads as wl

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _rows(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return [line.split() for line in f if line.strip() and not line.startswith("#")]


def test_splitmix64_fixture():
    rows = _rows("splitmix64_vectors.txt")
    assert len(rows) == 6
    for x, out in rows:
        assert oracle.splitmix64(int(x, 16)) == int(out)


def test_philox_fixture():
    rows = _rows("philox4x32_10_kat.txt")
    assert len(rows) == 3
    for r in rows:
        ctr, key, want = r[0:4], r[4:6], r[6:10]
        got = wl.philox4x32_10([int(x, 16) for x in ctr], [int(x, 16) for x in key])
        assert got == tuple(int(x, 16) for x in want)


def golden_cases():
    with open(os.path.join(GOLDEN, "oracle_digests.json")) as f:
        return json.load(f)


def test_oracle_still_reproduces_its_stored_digests():
    """A regression guard on the oracle and the generator: the stored digests
    were written by the oracle; any later change to either that moves a bit
    shows up here."""
    for c in golden_cases():
        if c["workload"] == "shrunken_mistral":
            w = wl.shrunken_mistral()
            p, g, m, v = wl.arrays_host(w)
            b = np.zeros(p.size, np.uint16)
            per, total = oracle.commit_segments(p, g, m, v, b, w.segments, [oracle.Hyper(**h) for h in w.hypers],
                                                c["step"], w.global_offset)
            assert [f"{x:#018x}" for x in per] == c["segment_digests"]
            bf = sum(oracle.bf16_digest(b[o:o + ln], w.global_offset + o) for o, ln, _ in w.segments)
        else:
            w = wl.WORKLOADS[c["workload"]]
            p, g, m, v = wl.arrays_host(w, c["start"], c["count"])
            b = np.zeros(p.size, np.uint16)
            total = oracle.commit_and_digest(p, g, m, v, b, oracle.Hyper(**w.hypers[0]), c["step"],
                                             w.global_offset + c["start"])
            bf = oracle.bf16_digest(b, w.global_offset + c["start"])
        assert f"{total:#018x}" == c["state_digest"], c["name"]
        assert f"{bf & oracle.MASK64:#018x}" == c["bf16_digest"], c["name"]
