"""Shared test plumbing: device shards from workloads, the oracle over host
threads, and comparisons.  Imports the oracle (tests may) and the GPU binding;
the two never meet except here, where their results are compared."""
from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

import oracle
import workloads as wl

M64 = (1 << 64) - 1


def host_threads() -> int:
    return max(1, min(16, os.cpu_count() or 1))


def o_hyper(d: dict) -> oracle.Hyper:
    return oracle.Hyper(**d)


def g_hyper(d: dict):
    import paper_2609_18178_amd as pk

    return pk.Hyper(**d)


def oracle_commit_parallel(p, g, m, v, b, hyper: oracle.Hyper, step: int, first_index: int,
                           parts: int | None = None) -> int:
    """The oracle over disjoint slices in host threads; the digest of the
    whole is the wrapping sum of the slices' digests (partition invariance,
    pinned in the oracle tests).  Each slice runs the unmodified oracle."""
    n = p.size
    parts = parts or host_threads()
    cuts = [n * k // parts for k in range(parts + 1)]

    def one(k):
        a, z = cuts[k], cuts[k + 1]
        return oracle.commit_and_digest(p[a:z], g[a:z], m[a:z], v[a:z], b[a:z], hyper, step, first_index + a)

    with ThreadPoolExecutor(parts) as ex:
        return sum(ex.map(one, range(parts))) & M64


def oracle_digest_parallel(p, m, v, first_index: int, parts: int | None = None) -> int:
    n = p.size
    parts = parts or host_threads()
    cuts = [n * k // parts for k in range(parts + 1)]

    def one(k):
        a, z = cuts[k], cuts[k + 1]
        return oracle.state_digest(p[a:z], m[a:z], v[a:z], first_index + a)

    with ThreadPoolExecutor(parts) as ex:
        return sum(ex.map(one, range(parts))) & M64


def to_device(*arrays, device="cuda"):
    import torch

    return [torch.from_numpy(a).to(device) for a in arrays]


def make_shard(p, g, m, v, global_offset, device="cuda", segments=None, hypers=None):
    """Device copies of host arrays and the Shard over them."""
    import torch
    import paper_2609_18178_amd as pk

    tp, tg, tm, tv = to_device(p, g, m, v, device=device)
    tb = torch.zeros(p.size, dtype=torch.int16, device=device)
    sh = pk.Shard(tp, tg, tm, tv, tb, global_offset=global_offset, segments=segments,
                  hypers=[g_hyper(h) for h in hypers] if hypers else None)
    return sh


def host(t) -> np.ndarray:
    return t.detach().cpu().numpy()


def bits(a: np.ndarray) -> np.ndarray:
    return a.view(np.uint32) if a.dtype == np.float32 else a.view(np.uint16)


def assert_bitwise(name, got: np.ndarray, want: np.ndarray) -> None:
    gb, wb = bits(got), bits(want)
    if not np.array_equal(gb, wb):
        bad = np.flatnonzero(gb != wb)
        i = int(bad[0])
        raise AssertionError(f"{name}: {bad.size} of {gb.size} elements differ; first at {i}: "
                             f"got {int(gb[i]):#x} want {int(wb[i]):#x}")


def oracle_stream_segments(w, step: int, hypers, chunk: int = 1 << 26, check=None):
    """The oracle over a workload's segments, chunk by chunk: each chunk's
    inputs are drawn on the host (same generator, same global indices as the
    device arrays), committed by the oracle cut over host threads, and its
    state and bf16 digests added to its segment.  Memory stays at one chunk.
    ``check(start, p, m, v, b)``, if given, sees each committed chunk."""
    segs = w.segments if w.segments is not None else ((0, w.numel, 0),)
    per, per_b = [], []
    threads = host_threads()
    for off, length, hi in segs:
        d = db = 0
        for a in range(off, off + length, chunk):
            cnt = min(chunk, off + length - a)
            p, g, m, v = wl.arrays_host(w, a, cnt)
            if step != w.first_step:
                g = wl.grad_host(w, step, a, cnt)
            b = np.zeros(cnt, np.uint16)
            d += oracle_commit_parallel(p, g, m, v, b, hypers[hi], step, w.global_offset + a,
                                        parts=threads if cnt >= (1 << 20) else 1)
            db += oracle.bf16_digest(b, w.global_offset + a)
            if check is not None:
                check(a, p, m, v, b)
        per.append(d & M64)
        per_b.append(db & M64)
    return per, per_b


def device_workload(w, device="cuda"):
    """Device arrays of a workload filled chunk by chunk from the host
    generator, and the Shard over them."""
    import torch
    import paper_2609_18178_amd as pk

    n = w.numel
    ts = [torch.empty(n, dtype=torch.float32, device=device) for _ in range(4)]
    for t, aid, step, dist in zip(ts, (wl.ARRAY_PARAM, wl.ARRAY_GRAD, wl.ARRAY_EXP_AVG, wl.ARRAY_EXP_AVG_SQ),
                                  (0, w.first_step, 0, 0), (w.param, w.grad, w.exp_avg, w.exp_avg_sq)):
        wl.fill_device(t, w.global_offset, w.seed, aid, step, dist)
    b = torch.zeros(n, dtype=torch.int16, device=device)
    segs = list(w.segments) if w.segments is not None else None
    hyp = [g_hyper(h) for h in w.hypers] if segs is not None else None
    return pk.Shard(*ts, b, global_offset=w.global_offset, segments=segs, hypers=hyp)
