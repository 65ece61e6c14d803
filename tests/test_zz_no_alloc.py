"""The commit entry point that allocates nothing (pact_adamw_commit_static),
through the C ABI, against the commit with a caller workspace
(pact_adamw_commit_ex) on the same inputs: every output and every digest
slot bit for bit, on calls in a row whose sizes shrink (the static scratch
keeps what the last call left), with and without gradient zeroing, and the
oracle on the last state.  Also: its argument errors come back before
anything is enqueued."""
import ctypes

import numpy as np
import pytest

import oracle
import workloads as wl
from tests.helpers import M64, assert_bitwise, host, make_shard, o_hyper

pytestmark = pytest.mark.gpu

H = wl.DEFAULT_HYPER


@pytest.fixture(scope="module", autouse=True)
def gpu():
    import torch

    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2609_18178_amd as pk

    pk._lib()
    yield


def _pk():
    import paper_2609_18178_amd as pk

    return pk


def _table(seed, nseg, max_len):
    """A seeded segment table with padding gaps and three hyper sets."""
    rng = np.random.default_rng(seed)
    hypers = [dict(H), dict(H, lr=1.5e-4, weight_decay=0.0), dict(H, beta2=0.99, eps=1e-6)]
    segs, off = [], int(rng.integers(0, 5))
    for _ in range(nseg):
        ln = int(rng.choice([0, 1, 5, 4096, 4097, int(rng.integers(1, max_len))]))
        segs.append((off, ln, int(rng.integers(0, 3))))
        off += ln + int(rng.choice([0, 1, 3, 128]))
    return segs, off + int(rng.integers(0, 4)), hypers


def _pair(n, goff, segs=None, hypers=None, seed_start=0):
    """Two device shards holding the same seeded inputs, and the host copy."""
    w = wl.WORKLOADS["mistral7b_shard16"]
    p, g, m, v = wl.arrays_host(w, seed_start, n)
    a = make_shard(p, g, m, v, goff, segments=segs, hypers=hypers)
    b = make_shard(p, g, m, v, goff, segments=segs, hypers=hypers)
    return a, b, (p, g, m, v)


def _same(a, b, what):
    for name in ("param", "grad", "exp_avg", "exp_avg_sq", "param_bf16"):
        assert_bitwise(f"{what} {name}", host(getattr(b, name)), host(getattr(a, name)))


# Calls in a row on one GPU, each smaller than the one before: the static
# scratch of the first (many segments, many tiles) is what the next finds.
CALLS = [
    ("300 segments", dict(segs_seed=5, nseg=300, max_len=30000), 7, False),
    ("40 segments", dict(segs_seed=6, nseg=40, max_len=9000), 8, True),
    ("flat, ragged, beyond 2^32", dict(n=100_003, goff=(5 << 32) - 777), 9, False),
    ("flat, one element", dict(n=1, goff=123), 10, True),
]


def test_static_commit_equals_workspace_commit_on_shrinking_calls():
    pk = _pk()
    lib = pk._lib()
    for what, shape, step, zero in CALLS:
        print(f"[no-alloc] {what}, step {step}, zero_grad={zero}", flush=True)
        if "segs_seed" in shape:
            segs, n, hyp = _table(shape["segs_seed"], shape["nseg"], shape["max_len"])
            goff = 1 << 34
        else:
            segs, hyp, n, goff = None, None, shape["n"], shape["goff"]
        ref, sta, (p, g, m, v) = _pair(n, goff, segs, hyp)
        hyper = None if segs else pk.Hyper(**H)
        flags = pk.PACT_COMMIT_ZERO_GRAD if zero else 0
        ch = ctypes.byref(hyper._c()) if hyper else None
        rc = lib.pact_adamw_commit_ex(ctypes.byref(ref._c()), step, ch, flags)
        assert rc == pk.PACT_OK
        rc = lib.pact_adamw_commit_static(ctypes.byref(sta._c(workspace=False)), step, ch, flags)
        assert rc == pk.PACT_OK, pk._strerror(rc)
        d_ref, d_sta = pk.to_u64(ref.digest), pk.to_u64(sta.digest)
        assert d_sta == d_ref, what
        _same(ref, sta, what)
        # the oracle on the same inputs
        b = np.zeros(n, np.uint16)
        if segs:
            per, total = oracle.commit_segments(p, g, m, v, b, segs, [o_hyper(h) for h in hyp], step, goff)
            assert d_sta == per + [total]
        else:
            assert d_sta == [oracle.commit_and_digest(p, g, m, v, b, o_hyper(H), step, goff)]
        assert_bitwise("oracle param", host(sta.param), p)
        assert_bitwise("oracle bf16", host(sta.param_bf16).view(np.uint16), b)
        if zero:
            # every committed gradient element is +0.0; padding keeps its bits
            gz = host(sta.grad).view(np.uint32)
            covered = np.zeros(n, bool)
            for o, ln, _ in (segs or [(0, n, 0)]):
                covered[o:o + ln] = True
            assert not gz[covered].any()
            assert np.array_equal(gz[~covered], g[~covered].view(np.uint32))
        del ref, sta


def test_binding_static_commit_repeats_like_the_workspace_commit():
    """Ten successive commits through each entry point give the same digest
    sequence (the static scratch is cleared by every call)."""
    pk = _pk()
    segs, n, hyp = _table(11, 60, 20000)
    ref, sta, _ = _pair(n, 1 << 33, segs, hyp)
    for step in range(100, 110):
        a = pk.to_u64(pk.adamw_commit(ref, step))
        b = pk.to_u64(pk.adamw_commit_static(sta, step))
        assert a == b, step
    _same(ref, sta, "after ten commits")


def test_static_commit_argument_errors_leave_state_untouched():
    pk = _pk()
    lib = pk._lib()
    hyp = [dict(H)]
    too_many = [(k * 8, 4, 0) for k in range(pk.PACT_STATIC_MAX_SEGMENTS + 1)]
    n = 8 * len(too_many)
    ref, sta, (p, g, m, v) = _pair(n, 0, too_many, hyp)
    before = [host(getattr(sta, k)).copy() for k in ("param", "exp_avg", "exp_avg_sq")]
    rc = lib.pact_adamw_commit_static(ctypes.byref(sta._c(workspace=False)), 3, None, 0)
    assert rc == pk.PACT_ESCRATCH
    # a caller workspace, or a flag other than zero-grad, is an argument error
    rc = lib.pact_adamw_commit_static(ctypes.byref(sta._c(workspace=True)), 3, None, 0)
    assert rc == pk.PACT_EINVAL
    rc = lib.pact_adamw_commit_static(ctypes.byref(sta._c(workspace=False)), 3, None,
                                      pk.PACT_COMMIT_WORKSPACE_CLEAN)
    assert rc == pk.PACT_EINVAL
    rc = lib.pact_adamw_commit_static(ctypes.byref(sta._c(workspace=False)), 0, None, 0)
    assert rc == pk.PACT_EINVAL
    after = [host(getattr(sta, k)) for k in ("param", "exp_avg", "exp_avg_sq")]
    for x, y in zip(before, after):
        assert np.array_equal(x.view(np.uint32), y.view(np.uint32))
    # at the limit the call runs and agrees with the workspace commit
    at_limit = too_many[:pk.PACT_STATIC_MAX_SEGMENTS]
    ref2, sta2, _ = _pair(n, 77, at_limit, hyp)
    a = pk.to_u64(pk.adamw_commit(ref2, 3))
    b = pk.to_u64(pk.adamw_commit_static(sta2, 3))
    assert a == b and len(b) == pk.PACT_STATIC_MAX_SEGMENTS + 1
    assert b[-1] == sum(b[:-1]) & M64


def test_static_commit_replays_from_a_hip_graph():
    """The use the allocation-free commit is for: captured into a HIP graph
    (the scratch is cleared by a kernel inside the graph, not a memset) and
    replayed three times with eager work in between, each replay equal to
    one more eager commit at the captured step, digests and state bit for
    bit.  An eager call on the device comes first (it looks up the scratch
    address)."""
    import torch

    pk = _pk()
    segs, n, hyp = _table(21, 12, 9000)
    eager, graphed, _ = _pair(n, 1 << 33, segs, hyp)
    want = [pk.to_u64(pk.adamw_commit_static(eager, 9)) for _ in range(3)]
    p_before = host(graphed.param).copy()
    graph = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        with torch.cuda.graph(graph, stream=side):
            pk.adamw_commit_static(graphed, 9)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    assert_bitwise("param before replay", host(graphed.param), p_before)
    for k in range(3):
        graph.replay()
        torch.cuda.synchronize()
        assert pk.to_u64(graphed.digest) == want[k], k
        _ = (torch.ones(1024, device="cuda") * 2).sum().item()  # unrelated eager work in between
    _same(eager, graphed, "after three replays")
