"""Writes tests/golden/oracle_digests.json: digests of small seeded workloads
computed by the oracle alone (no GPU code involved).  The CPU suite checks
that the oracle still reproduces them; the GPU suite compares the library's
digests against them as well as against a live oracle run.

Run: python tests/golden/make_digests.py
"""
import json
import os
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402

import oracle  # noqa: E402
import workloads as wl  # noqa: E402


def cases():
    out = []
    w = wl.WORKLOADS["tiny"]
    p, g, m, v = wl.arrays_host(w)
    b = np.zeros(p.size, np.uint16)
    d = oracle.commit_and_digest(p, g, m, v, b, oracle.Hyper(**w.hypers[0]), w.first_step, w.global_offset)
    out.append(dict(name="tiny", workload="tiny", start=0, count=w.numel, step=w.first_step,
                    state_digest=d, bf16_digest=oracle.bf16_digest(b, w.global_offset)))
    for name in ("decoder1b_shard16", "mistral7b_shard16", "mistral7b_shard4"):
        w = wl.WORKLOADS[name]
        count = 1 << 20
        p, g, m, v = wl.arrays_host(w, 0, count)
        b = np.zeros(count, np.uint16)
        d = oracle.commit_and_digest(p, g, m, v, b, oracle.Hyper(**w.hypers[0]), w.first_step, w.global_offset)
        out.append(dict(name=f"{name}_first_2^20", workload=name, start=0, count=count, step=w.first_step,
                        state_digest=d, bf16_digest=oracle.bf16_digest(b, w.global_offset)))
    w = wl.shrunken_mistral()
    p, g, m, v = wl.arrays_host(w)
    b = np.zeros(p.size, np.uint16)
    per, total = oracle.commit_segments(p, g, m, v, b, w.segments, [oracle.Hyper(**h) for h in w.hypers],
                                        w.first_step, w.global_offset)
    # padding is not digested: the bf16 digest is the sum over segments
    bf = sum(oracle.bf16_digest(b[o:o + ln], w.global_offset + o) for o, ln, _ in w.segments) & oracle.MASK64
    out.append(dict(name="mistral_shrunk", workload="shrunken_mistral", start=0, count=w.numel,
                    step=w.first_step, segment_digests=per, state_digest=total, bf16_digest=bf))
    return out


if __name__ == "__main__":
    recs = cases()
    for r in recs:
        for k in ("state_digest", "bf16_digest"):
            r[k] = f"{r[k]:#018x}"
        if "segment_digests" in r:
            r["segment_digests"] = [f"{x:#018x}" for x in r["segment_digests"]]
    with open(os.path.join(HERE, "oracle_digests.json"), "w") as f:
        json.dump(recs, f, indent=1)
        f.write("\n")
    print(f"wrote {len(recs)} cases")
