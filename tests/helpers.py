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
