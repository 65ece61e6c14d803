"""GPU path vs the CPU oracle, element by element, through the C ABI.

The library is built in exact mode (no contraction, IEEE sqrt/div, fp32
denormals kept), so the contract is bit-exact for every output: p', m', v',
the bf16 copy and every digest slot.
"""
import numpy as np
import pytest

import oracle
import workloads as wl
from tests.helpers import (M64, assert_bitwise, host, make_shard, o_hyper, g_hyper, oracle_commit_parallel,
                           oracle_digest_parallel)

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


def _compare_full(sh, p, m, v, b, what=""):
    assert_bitwise(what + "param", host(sh.param), p)
    assert_bitwise(what + "exp_avg", host(sh.exp_avg), m)
    assert_bitwise(what + "exp_avg_sq", host(sh.exp_avg_sq), v)
    assert_bitwise(what + "bf16", host(sh.param_bf16).view(np.uint16), b)


def _commit_both(w, start=0, count=None, hyper=H, step=None):
    """Inputs of workload w (slice), committed on the GPU and by the oracle."""
    pk = _pk()
    p, g, m, v = wl.arrays_host(w, start, count)
    sh = make_shard(p, g, m, v, w.global_offset + start)
    step = step or w.first_step
    d_gpu = pk.to_u64(pk.adamw_commit(sh, step, g_hyper(hyper)))[0]
    b = np.zeros(p.size, np.uint16)
    d_ref = oracle_commit_parallel(p, g, m, v, b, o_hyper(hyper), step, w.global_offset + start)
    return sh, (p, g, m, v, b), d_gpu, d_ref


def test_tiny_full_parity():
    """1,048,576 elements, step 1 from m = v = 0: every output bitwise."""
    pk = _pk()
    w = wl.WORKLOADS["tiny"]
    sh, (p, g, m, v, b), d_gpu, d_ref = _commit_both(w)
    _compare_full(sh, p, m, v, b)
    assert d_gpu == d_ref
    # the standalone digest of the committed state equals the fused one
    assert pk.to_u64(pk.shard_digest(sh))[0] == d_ref
    assert pk.to_u64(pk.bf16_digest(sh))[0] == oracle.bf16_digest(b, w.global_offset)


@pytest.mark.parametrize("n", [1, 2, 3, 4, 5, 63, 64, 65, 2047, 2048, 2049, 4093, 10007, 100003])
@pytest.mark.parametrize("shift", [0, 1, 2, 3])
def test_ragged_and_unaligned(n, shift):
    """Ragged tails and views starting 1-3 elements past a 16-byte boundary
    (element-wise path) give the oracle's bits."""
    import torch

    pk = _pk()
    w = wl.WORKLOADS["decoder1b_shard16"]
    p, g, m, v = wl.arrays_host(w, 0, n)
    full = [torch.zeros(n + 8, dtype=torch.float32, device="cuda") for _ in range(4)]
    views = []
    for t, a in zip(full, (p, g, m, v)):
        t[shift:shift + n] = torch.from_numpy(a).cuda()
        views.append(t[shift:shift + n])
    bfull = torch.zeros(n + 8, dtype=torch.int16, device="cuda")
    sh = pk.Shard(*views, bfull[shift:shift + n], global_offset=w.global_offset)
    d_gpu = pk.to_u64(pk.adamw_commit(sh, 100, g_hyper(H)))[0]
    b = np.zeros(n, np.uint16)
    d_ref = oracle.commit_and_digest(p, g, m, v, b, o_hyper(H), 100, w.global_offset)
    assert d_gpu == d_ref
    _compare_full(sh, p, m, v, b)
    # guard elements around the view are untouched
    for t in full + [bfull]:
        h = host(t)
        assert not h[:shift].any() and not h[shift + n:].any()


@pytest.mark.parametrize("segmented", [False, True])
def test_without_workspace(segmented):
    """workspace == NULL: partial sums go straight to the result slots; the
    results are the same bits."""
    import torch

    pk = _pk()
    w = wl.shrunken_mistral() if segmented else wl.WORKLOADS["tiny"]
    p, g, m, v = wl.arrays_host(w)
    segs = w.segments if segmented else None
    hyp = [pk.Hyper(**h) for h in w.hypers] if segmented else None
    t = [torch.from_numpy(a).cuda() for a in (p, g, m, v)]
    sh = pk.Shard(*t, torch.zeros(p.size, dtype=torch.int16, device="cuda"), w.global_offset,
                  segments=segs, hypers=hyp, use_workspace=False)
    assert sh.workspace is None
    got = pk.to_u64(pk.adamw_commit(sh, w.first_step, None if segmented else g_hyper(H)))
    b = np.zeros(p.size, np.uint16)
    if segmented:
        per, total = oracle.commit_segments(p, g, m, v, b, w.segments, [o_hyper(h) for h in w.hypers],
                                            w.first_step, w.global_offset)
        assert got == per + [total]
    else:
        assert got == [oracle.commit_and_digest(p, g, m, v, b, o_hyper(H), w.first_step, w.global_offset)]
    _compare_full(sh, p, m, v, b)


def test_empty_shard():
    """n = 0: the digest is 0 and nothing is read or written."""
    import torch

    pk = _pk()
    e = torch.zeros(0, dtype=torch.float32, device="cuda")
    sh = pk.Shard(e, e.clone(), e.clone(), e.clone(), torch.zeros(0, dtype=torch.int16, device="cuda"), 5)
    sh.digest.fill_(123)
    assert pk.to_u64(pk.adamw_commit(sh, 1, g_hyper(H))) == [0]
    sh.digest.fill_(7)
    assert pk.to_u64(pk.shard_digest(sh)) == [0]


def test_decoder1b_shard_ten_commits():
    """76,000,000-element shard (rank 15 of a 1.216B decoder at 16 ranks), warm
    state from step 100, ten commits with a fresh gradient each: every per-step
    digest and, at the end, every output bitwise."""
    import torch

    pk = _pk()
    w = wl.WORKLOADS["decoder1b_shard16"]
    p, g, m, v = wl.arrays_host(w)
    sh = make_shard(p, g, m, v, w.global_offset)
    b = np.zeros(p.size, np.uint16)
    for step in range(w.first_step, w.first_step + w.commits):
        if step != w.first_step:
            g = wl.grad_host(w, step)
            sh.grad.copy_(torch.from_numpy(g))
        d_gpu = pk.to_u64(pk.adamw_commit(sh, step, g_hyper(H)))[0]
        d_ref = oracle_commit_parallel(p, g, m, v, b, o_hyper(H), step, w.global_offset)
        assert d_gpu == d_ref, f"step {step}"
    _compare_full(sh, p, m, v, b)


def test_repeated_sequences_are_bit_identical():
    """Ten repetitions of a ten-commit sequence give identical digest vectors
    (the ten-repair bitwise check of Sec. IV-G, as digests), equal to the
    oracle's vector."""
    import torch

    pk = _pk()
    w = wl.WORKLOADS["decoder1b_shard16"]
    n = 1 << 22
    p0, g0, m0, v0 = wl.arrays_host(w, 0, n)
    grads = [wl.grad_host(w, s, 0, n) for s in range(100, 110)]
    vectors = []
    for rep in range(10):
        sh = make_shard(p0, g0, m0, v0, w.global_offset)
        vec = []
        for k, step in enumerate(range(100, 110)):
            sh.grad.copy_(torch.from_numpy(grads[k]))
            vec.append(pk.to_u64(pk.adamw_commit(sh, step, g_hyper(H)))[0])
        vectors.append(vec)
    assert all(vec == vectors[0] for vec in vectors)
    p, m, v = p0.copy(), m0.copy(), v0.copy()
    b = np.zeros(n, np.uint16)
    ref = [oracle.commit_and_digest(p, grads[k], m, v, b, o_hyper(H), 100 + k, w.global_offset) for k in range(10)]
    assert vectors[0] == ref


@pytest.mark.parametrize("goff", [2 ** 32 - 1000, 2 ** 56 - 5001])
def test_global_index_edges(goff):
    """Indices crossing 2^32, and the last indices below the tag bits."""
    pk = _pk()
    w = wl.WORKLOADS["decoder1b_shard16"]
    n = 5001
    p, g, m, v = wl.arrays_host(w, 0, n)
    sh = make_shard(p, g, m, v, goff)
    d_gpu = pk.to_u64(pk.adamw_commit(sh, 3, g_hyper(H)))[0]
    b = np.zeros(n, np.uint16)
    assert d_gpu == oracle.commit_and_digest(p, g, m, v, b, o_hyper(H), 3, goff)
    _compare_full(sh, p, m, v, b)
    sh.global_offset = 2 ** 56 - n + 1
    with pytest.raises(pk.PactError) as e:
        pk.adamw_commit(sh, 4, g_hyper(H))
    assert e.value.code == pk.PACT_ERANGE


@pytest.mark.parametrize("goff", [0, 2 ** 32 - 5096, 2 ** 33 - 7000, 2 ** 56 - 3 * 4096 - 123])
def test_every_digest_across_index_halves(goff):
    """Each digesting kernel (commit, state digest, bf16 digest, BF16-state
    commit and digest) on whole tiles that sit below, across and above a
    multiple of 2^32, and at the top of the index range: the vector path
    hashes a tile whose indices share their upper 32 bits in a shorter form
    than one that crosses such a multiple, and both must give the oracle's
    digest."""
    import torch

    pk = _pk()
    w = wl.WORKLOADS["mistral7b_shard16"]
    n = 3 * 4096 + 123  # three whole tiles and a ragged tail
    p, g, m, v = wl.arrays_host(w, 0, n)
    sh = make_shard(p, g, m, v, goff)
    d_gpu = pk.to_u64(pk.adamw_commit(sh, 5, g_hyper(H)))[0]
    b = np.zeros(n, np.uint16)
    assert d_gpu == oracle.commit_and_digest(p, g, m, v, b, o_hyper(H), 5, goff)
    _compare_full(sh, p, m, v, b)
    assert pk.to_u64(pk.shard_digest(sh))[0] == oracle.state_digest(p, m, v, goff)
    assert pk.to_u64(pk.bf16_digest(sh))[0] == oracle.bf16_digest(b, goff)
    pb, gb, mb, vb = _bf16_arrays(w, 0, n)
    t = [torch.from_numpy(a.view(np.int16).copy()).cuda() for a in (pb, gb, mb, vb)]
    sh16 = pk.ShardBf16(*t, global_offset=goff)
    got = pk.to_u64(pk.adamw_commit_bf16(sh16, 5, g_hyper(H)))[0]
    assert got == oracle.commit_and_digest_bf16(pb, gb, mb, vb, o_hyper(H), 5, goff)
    for name, tt, ref in (("param", sh16.param, pb), ("exp_avg", sh16.exp_avg, mb), ("exp_avg_sq", sh16.exp_avg_sq, vb)):
        assert_bitwise(name, host(tt).view(np.uint16), ref)
    assert pk.to_u64(pk.shard_digest_bf16(sh16))[0] == oracle.state_digest_bf16(pb, mb, vb, goff)


@pytest.mark.parametrize("goff", [0x12340000 + 4096, 2 ** 16 - 1000, 0x80B50000 - 4096, (5 << 32) + 0x40B50000,
                                  (7 << 32) + 0xC0B50000 - 2048, 0x00B50000, (3 << 40) + 0xFFFF0000 - 4096])
def test_sixteen_bit_digests_at_every_index_form(goff):
    """The digests of 16-bit words (BF16-state commit and digest, the bf16
    copy's digest) take a short first mixing round on tiles whose indices
    share bits 16..63, unless the low halves of those indices start at
    0x00B50000, 0x40B50000, 0x80B50000 or 0xC0B50000 (where the short round's
    carry assumptions fail).  Tiles of each kind -- short form, across a
    multiple of 2^16, at each excluded start -- must give the oracle's
    digests and state."""
    import torch

    pk = _pk()
    w = wl.WORKLOADS["mistral7b_shard16"]
    n = 3 * 4096 + 123
    p, g, m, v = wl.arrays_host(w, 0, n)
    sh = make_shard(p, g, m, v, goff)
    b = np.zeros(n, np.uint16)
    assert pk.to_u64(pk.adamw_commit(sh, 5, g_hyper(H)))[0] == oracle.commit_and_digest(
        p, g, m, v, b, o_hyper(H), 5, goff)
    assert_bitwise("bf16", host(sh.param_bf16).view(np.uint16), b)
    assert pk.to_u64(pk.bf16_digest(sh))[0] == oracle.bf16_digest(b, goff)
    pb, gb, mb, vb = _bf16_arrays(w, 0, n)
    t = [torch.from_numpy(a.view(np.int16).copy()).cuda() for a in (pb, gb, mb, vb)]
    sh16 = pk.ShardBf16(*t, global_offset=goff)
    assert pk.to_u64(pk.shard_digest_bf16(sh16))[0] == oracle.state_digest_bf16(pb, mb, vb, goff)
    got = pk.to_u64(pk.adamw_commit_bf16(sh16, 5, g_hyper(H)))[0]
    assert got == oracle.commit_and_digest_bf16(pb, gb, mb, vb, o_hyper(H), 5, goff)
    for name, tt, ref in (("param", sh16.param, pb), ("exp_avg", sh16.exp_avg, mb), ("exp_avg_sq", sh16.exp_avg_sq, vb)):
        assert_bitwise(name, host(tt).view(np.uint16), ref)
    assert pk.to_u64(pk.shard_digest_bf16(sh16))[0] == oracle.state_digest_bf16(pb, mb, vb, goff)


def test_multi_segment_shrunken_mistral():
    """Real Mistral tensor roles at a small size with padding, four hyper
    sets (norms without decay, lm_head with its own beta2): per-segment
    digests, their sum, every output, and untouched padding."""
    import torch

    pk = _pk()
    w = wl.shrunken_mistral()
    p, g, m, v = wl.arrays_host(w)
    sh = make_shard(p, g, m, v, w.global_offset, segments=w.segments, hypers=w.hypers)
    sh.param_bf16.fill_(0x5A5A)
    got = pk.to_u64(pk.adamw_commit(sh, 5))
    b = np.full(p.size, 0x5A5A, np.uint16)
    per, total = oracle.commit_segments(p, g, m, v, b, w.segments, [o_hyper(h) for h in w.hypers], 5,
                                        w.global_offset)
    assert got == per + [total]
    _compare_full(sh, p, m, v, b)
    assert pk.to_u64(pk.shard_digest(sh)) == per + [total]
    bd = pk.to_u64(pk.bf16_digest(sh))
    want = [oracle.bf16_digest(b[o:o + ln], w.global_offset + o) for o, ln, _ in w.segments]
    assert bd == want + [sum(want) & M64]
    del torch


def _random_segment_table(seed):
    """(segments, numel, global offset, hyper dicts) drawn from `seed`."""
    rng = np.random.default_rng(seed)
    hypers = [dict(H), dict(H, lr=1.5e-4, weight_decay=0.0), dict(H, beta2=0.99, eps=1e-6)]
    nseg = int(rng.integers(1, 80))
    segs, off = [], int(rng.integers(0, 9))
    for _ in range(nseg):
        ln = int(rng.choice([0, 1, 3, 7, 128, 4095, 4096, 4097, 8192, int(rng.integers(1, 20000))]))
        segs.append((off, ln, int(rng.integers(0, 3))))
        off += ln + int(rng.choice([0, 0, 1, 2, 5, 128, 4096]))
    n = off + int(rng.integers(0, 7))
    return segs, n, int(rng.integers(0, 1 << 40)), hypers


@pytest.mark.parametrize("seed", range(6))
def test_random_segment_tables(seed):
    """Seeded random segment tables: lengths from empty to several tiles (one
    element, unaligned, exact multiples of a tile), gaps of padding between
    segments, random hyper indices over three hyper sets, a random global
    offset below 2^40, sometimes more segments than one launch carries.  The
    commit (every per-segment digest, the total and every output, padding
    untouched), the standalone digest and the zero-grad commit with the
    guard all match the oracle."""
    pk = _pk()
    segs, n, goff, hypers = _random_segment_table(1000 + seed)
    w = wl.WORKLOADS["mistral7b_shard16"]
    p, g, m, v = wl.arrays_host(w, 0, n)
    sh = make_shard(p, g, m, v, goff, segments=segs, hypers=hypers)
    sh.param_bf16.fill_(0x3C3C)
    p0, m0, v0 = p.copy(), m.copy(), v.copy()
    got = pk.to_u64(pk.adamw_commit(sh, 7))
    b = np.full(n, 0x3C3C, np.uint16)
    per, total = oracle.commit_segments(p, g, m, v, b, segs, [o_hyper(h) for h in hypers], 7, goff)
    assert got == per + [total]
    _compare_full(sh, p, m, v, b)
    covered = np.zeros(n, bool)
    for o, ln, _ in segs:
        covered[o:o + ln] = True
    assert np.array_equal(p[~covered].view(np.uint32), p0[~covered].view(np.uint32))
    assert np.array_equal(m[~covered].view(np.uint32), m0[~covered].view(np.uint32))
    assert np.array_equal(v[~covered].view(np.uint32), v0[~covered].view(np.uint32))
    sd_per, sd_total = oracle.segment_digests(p, m, v, segs, goff)
    assert pk.to_u64(pk.shard_digest(sh)) == sd_per + [sd_total]
    got_z = pk.to_u64(pk.adamw_commit(sh, 8, zero_grad=True))
    per_z, total_z = oracle.commit_segments(p, g, m, v, b, segs, [o_hyper(h) for h in hypers], 8, goff)
    assert got_z == per_z + [total_z]
    _compare_full(sh, p, m, v, b, "zero-grad ")
    g_after = host(sh.grad)
    want_g = g.copy()
    want_g[covered] = 0.0
    assert np.array_equal(g_after.view(np.uint32), want_g.view(np.uint32))
    guard = pk.to_u64(pk.grad_guard(sh))
    assert guard == [0] * (len(segs) + 1)


def test_many_segments_span_several_launches():
    """More segments than one launch carries (32), with empty, one-element,
    unaligned and ragged segments and gaps between them."""
    pk = _pk()
    rng = np.random.default_rng(21)
    segs, off = [], 3
    for k in range(100):
        ln = int(rng.choice([0, 1, 5, 2048, 3001, 4096, 9999]))
        segs.append((off, ln, k % 3))
        off += ln + int(rng.integers(0, 9))
    n = off + 17
    hypers = [H, dict(H, weight_decay=0.0), dict(H, lr=1e-3, beta2=0.99)]
    w = wl.WORKLOADS["decoder1b_shard16"]
    p, g, m, v = wl.arrays_host(w, 0, n)
    sh = make_shard(p, g, m, v, 777, segments=segs, hypers=hypers)
    got = pk.to_u64(pk.adamw_commit(sh, 9))
    b = np.zeros(n, np.uint16)
    per, total = oracle.commit_segments(p, g, m, v, b, segs, [o_hyper(h) for h in hypers], 9, 777)
    assert got == per + [total]
    _compare_full(sh, p, m, v, b)


def test_special_values_lr_zero_keeps_every_pattern():
    """lr = 0, g = 0, m = v = 0: p' == p for every non-NaN binary32 pattern
    (denormals, -0, infinities), so the bf16 copy is the RNE of each pattern:
    all 65,536 upper halves crossed with the rounding-boundary lower halves."""
    import torch

    pk = _pk()
    hi = np.arange(1 << 16, dtype=np.uint32) << 16
    lows = np.array([0x0000, 0x0001, 0x7FFF, 0x8000, 0x8001, 0xFFFF, 0x1234, 0xC000], dtype=np.uint32)
    pat = (hi[:, None] | lows[None, :]).reshape(-1)
    pat = pat[(pat & 0x7FFFFFFF) <= 0x7F800000]
    n = pat.size
    p = pat.view(np.float32).copy()
    z = np.zeros(n, np.float32)
    sh = make_shard(p, z, z, z, 0)
    pk.adamw_commit(sh, 1, pk.Hyper(lr=0.0, weight_decay=0.0))
    assert_bitwise("param", host(sh.param), p)
    assert_bitwise("bf16", host(sh.param_bf16).view(np.uint16), oracle.bf16_rne_bits(pat))
    b = np.zeros(n, np.uint16)
    pp, mm, vv = p.copy(), z.copy(), z.copy()
    d = oracle.commit_and_digest(pp, z.copy(), mm, vv, b, oracle.Hyper(lr=0.0, weight_decay=0.0), 1, 0)
    assert pk.to_u64(sh.digest)[0] == d
    del torch


def _nan32(a):
    u = np.asarray(a).view(np.uint32)
    return (u & 0x7FFFFFFF) > 0x7F800000


def _nan16(a):
    u = np.asarray(a).view(np.uint16).astype(np.uint32)
    return (u & 0x7FFF) > 0x7F80


def _assert_same_or_both_nan(what, got, want, isnan):
    """Bitwise where the oracle's result is a number; NaN where it is NaN (the
    payload of a NaN made by an invalid operation is not part of the contract:
    x86 makes 0xFFC00000, the GPU another pattern)."""
    wn, gn = isnan(want), isnan(got)
    assert np.array_equal(wn, gn), f"{what}: NaN at {np.flatnonzero(wn != gn)[:8]}"
    keep = ~wn
    assert_bitwise(what, np.asarray(got)[keep], np.asarray(want)[keep])


@pytest.mark.parametrize("shift", [0, 1])
def test_special_values_through_the_update(shift):
    """Infinities, NaNs, overflowing and denormal gradients, infinite moments
    and weights, planted in a realistic shard and sent through a full update
    (lr > 0): every output bitwise where the oracle gives a number, NaN where
    it gives NaN; the digest equals the oracle's digest of the GPU's own
    outputs (it hashes whatever bits the update produced)."""
    import torch

    pk = _pk()
    rng = np.random.default_rng(12)
    n = 20011
    p = (rng.standard_normal(n) * 0.02).astype(np.float32)
    g = (rng.standard_normal(n) * 1e-3).astype(np.float32)
    m = (rng.standard_normal(n) * 1e-4).astype(np.float32)
    v = np.abs(rng.standard_normal(n) * 3e-4).astype(np.float32) ** 2
    f = lambda bits: np.array([bits], np.uint32).view(np.float32)[0]  # noqa: E731
    specials_g = [np.inf, -np.inf, f(0x7FC00000), f(0x7FC12345), f(0xFFC00000), f(0x7F800001), 3e38, -3e38,
                  1e30, -1e30, 1e20, f(0x00000001), f(0x80000001), -0.0, 0.0, np.finfo(np.float32).max]
    specials_m = [np.inf, -np.inf, f(0x7FC00000), 3e38, -3e38, f(0x00000003)]
    specials_v = [np.inf, f(0x7FC00000), 3e38, f(0x00000001), 0.0]
    specials_p = [np.inf, -np.inf, f(0x7FC00000), np.finfo(np.float32).max, -np.finfo(np.float32).max,
                  f(0x00000001), -0.0]
    # plant each in the full tiles (vector path) and in the ragged tail
    where = [3, 517, 4095, 4096, 9000, 12289, 16383, 20000, 20010]
    for k, pos in enumerate(where):
        for j, x in enumerate(specials_g):
            g[(pos + 37 * j) % n] = x
        for j, x in enumerate(specials_m):
            m[(pos + 11 + 41 * j) % n] = x
        for j, x in enumerate(specials_v):
            v[(pos + 23 + 43 * j) % n] = x
        for j, x in enumerate(specials_p):
            p[(pos + 5 + 47 * j) % n] = x
    # combinations: infinite gradient against an opposite infinite moment
    g[100], m[100] = np.inf, -np.inf
    g[101], v[101] = np.inf, np.inf
    g[102], m[102], v[102] = f(0x7FC00000), np.inf, np.inf
    base = 6_795_022_080
    if shift:
        p, g, m, v = (np.concatenate([np.zeros(shift, np.float32), a]) for a in (p, g, m, v))
    tp, tg, tm, tv = (torch.from_numpy(a.copy()).cuda() for a in (p, g, m, v))
    tb = torch.zeros(p.size, dtype=torch.int16, device="cuda")
    sl = slice(shift, None)
    sh = pk.Shard(tp[sl], tg[sl], tm[sl], tv[sl], tb[sl], global_offset=base)
    hy = dict(lr=3e-4, beta1=0.9, beta2=0.95, eps=1e-8, weight_decay=0.1)
    d = pk.to_u64(pk.adamw_commit(sh, 7, g_hyper(hy)))[0]
    pp, gg, mm, vv = (a[sl].copy() for a in (p, g, m, v))
    b = np.zeros(n, np.uint16)
    oracle.commit_and_digest(pp, gg, mm, vv, b, o_hyper(hy), 7, base)
    got = [host(t[sl]) for t in (tp, tm, tv)]
    for what, gval, want in zip(("param", "exp_avg", "exp_avg_sq"), got, (pp, mm, vv)):
        _assert_same_or_both_nan(what, gval, want, _nan32)
    _assert_same_or_both_nan("bf16", host(tb[sl]).view(np.uint16), b, _nan16)
    assert _nan32(pp).sum() > 20 and np.isinf(pp).sum() > 10  # the plants did reach the outputs
    assert d == oracle.state_digest(*got, base)
    assert pk.to_u64(pk.shard_digest(sh))[0] == d
    assert (host(tg[sl]).view(np.uint32) == g[sl].view(np.uint32)).all()  # the gradient is only read


def test_bias_correction_over_step_sequences():
    """The library carries beta^t over from one call to the next; whatever
    order the steps come in (forward, back to the start, far ahead, repeated)
    every commit must equal the oracle's, which multiplies from 1 each time."""
    pk = _pk()
    rng = np.random.default_rng(21)
    n = 4096 + 17
    p0 = (rng.standard_normal(n) * 0.02).astype(np.float32)
    g0 = (rng.standard_normal(n) * 1e-3).astype(np.float32)
    m0 = (rng.standard_normal(n) * 1e-4).astype(np.float32)
    v0 = (np.abs(rng.standard_normal(n)) * 1e-7).astype(np.float32)
    hypers = [dict(lr=3e-4, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.1),
              dict(lr=1e-4, beta1=0.95, beta2=0.9999, eps=1e-6, weight_decay=0.0)]
    steps = [1, 2, 3, 1000, 1001, 5, 200000, 200001, 7, 2, 3000000, 3000001, 1]
    for hy in hypers:
        for t in steps:
            sh = make_shard(p0, g0, m0, v0, 99)
            d = pk.to_u64(pk.adamw_commit(sh, t, g_hyper(hy)))[0]
            p, g, m, v = p0.copy(), g0.copy(), m0.copy(), v0.copy()
            b = np.zeros(n, np.uint16)
            assert d == oracle.commit_and_digest(p, g, m, v, b, o_hyper(hy), t, 99), (hy, t)
            _compare_full(sh, p, m, v, b, f"t={t} ")


@pytest.mark.parametrize("segmented", [False, True])
def test_workspace_is_left_clear_and_the_clean_flag_skips_clearing(segmented):
    """Every call leaves the workspace lanes at zero, so commits through the
    binding skip clearing them (PACT_COMMIT_WORKSPACE_CLEAN); mixed with the
    digest and the guard, every result still equals the oracle's.  A dirty
    workspace is cleared when the flag is not given, and gives a wrong digest
    when it is (so the flag really skips the clearing)."""
    import torch

    pk = _pk()
    rng = np.random.default_rng(31)
    n = 3 * 4096 + 1000
    p = (rng.standard_normal(n) * 0.02).astype(np.float32)
    g = (rng.standard_normal(n) * 1e-3).astype(np.float32)
    m = (rng.standard_normal(n) * 1e-4).astype(np.float32)
    v = (np.abs(rng.standard_normal(n)) * 1e-7).astype(np.float32)
    segs = [(0, 5000, 0), (5000, 4000, 1), (9100, n - 9100, 0)] if segmented else None
    hys = [dict(H), dict(H, lr=1e-4, weight_decay=0.0)]
    sh = make_shard(p, g, m, v, 4242, segments=segs, hypers=hys if segmented else None)
    assert sh.workspace is not None and sh.workspace_clean

    b = np.zeros(n, np.uint16)

    def expect_commit(step):
        if segmented:
            per, total = oracle.commit_segments(p, g, m, v, b, segs, [o_hyper(h) for h in hys], step, 4242)
            return per + [total]
        return [oracle.commit_and_digest(p, g, m, v, b, o_hyper(H), step, 4242)]

    def expect_digest():
        if segmented:
            per, total = oracle.segment_digests(p, m, v, segs, 4242)
            return per + [total]
        return [oracle.state_digest(p, m, v, 4242)]

    lanes = 16 * (len(segs) if segmented else 1)  # 16 lanes per result slot, one word every 256 bytes

    def workspace_zero():
        words = sh.workspace.view(torch.int64)[::32][:lanes]
        return int(torch.count_nonzero(words).item()) == 0

    hy = None if segmented else g_hyper(H)
    for step in (3, 4):
        assert pk.to_u64(pk.adamw_commit(sh, step, hy)) == expect_commit(step)
        assert workspace_zero()
        assert pk.to_u64(pk.shard_digest(sh)) == expect_digest()
        assert workspace_zero()
        pk.grad_guard(sh)
        assert workspace_zero()
    # dirty workspace, flag not given: the call clears it first
    sh.workspace.copy_(torch.randint(0, 256, sh.workspace.shape, dtype=torch.uint8, device=sh.workspace.device))
    sh.workspace_clean = False
    assert pk.to_u64(pk.adamw_commit(sh, 5, hy)) == expect_commit(5)
    assert workspace_zero() and sh.workspace_clean
    # dirty workspace with the flag: the clearing is skipped, the digest is off
    sh.workspace.copy_(torch.randint(1, 256, sh.workspace.shape, dtype=torch.uint8, device=sh.workspace.device))
    wrong = pk.to_u64(pk.adamw_commit(sh, 6, hy))
    right = expect_commit(6)
    assert wrong[0] != right[0]
    _compare_full(sh, p, m, v, b)  # the state itself is committed correctly
    assert workspace_zero()  # and the call still leaves the workspace clear


def test_commit_replays_from_a_hip_graph():
    """A commit captured into a HIP graph (through torch's graph capture on the
    current stream) replays as the same kernels: each replay equals one more
    eager commit at the captured step, digests and state bit for bit, with
    eager work and synchronisation between the replays."""
    import torch

    pk = _pk()
    rng = np.random.default_rng(41)
    n = 2 * 4096 + 333
    p0 = (rng.standard_normal(n) * 0.02).astype(np.float32)
    g0 = (rng.standard_normal(n) * 1e-3).astype(np.float32)
    m0 = (rng.standard_normal(n) * 1e-4).astype(np.float32)
    v0 = (np.abs(rng.standard_normal(n)) * 1e-7).astype(np.float32)
    hy = g_hyper(H)
    eager = make_shard(p0, g0, m0, v0, 777)
    want = []
    for _ in range(3):
        want.append(pk.to_u64(pk.adamw_commit(eager, 9, hy))[0])
    graphed = make_shard(p0, g0, m0, v0, 777)
    graph = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        with torch.cuda.graph(graph, stream=side):
            pk.adamw_commit(graphed, 9, hy)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    # capture enqueues nothing: the state is untouched until the first replay
    assert_bitwise("param before replay", host(graphed.param), p0)
    for k in range(3):
        graph.replay()
        torch.cuda.synchronize()
        assert pk.to_u64(graphed.digest)[0] == want[k], k
        _ = (torch.ones(1024, device="cuda") * 2).sum().item()  # unrelated eager work in between
    for a, b in ((graphed.param, eager.param), (graphed.exp_avg, eager.exp_avg),
                 (graphed.exp_avg_sq, eager.exp_avg_sq), (graphed.param_bf16, eager.param_bf16)):
        assert torch.equal(a, b)
    p, g, m, v = p0.copy(), g0.copy(), m0.copy(), v0.copy()
    b = np.zeros(n, np.uint16)
    for k in range(3):
        assert oracle.commit_and_digest(p, g, m, v, b, o_hyper(H), 9, 777) == want[k]


def test_denormal_state_is_kept():
    """Denormal moments and weights go through the update without flushing."""
    pk = _pk()
    rng = np.random.default_rng(4)
    n = 65536
    p = (rng.standard_normal(n) * 1e-39).astype(np.float32)
    g = (rng.standard_normal(n) * 1e-40).astype(np.float32)
    m = (rng.standard_normal(n) * 1e-41).astype(np.float32)
    v = np.abs(rng.standard_normal(n) * 1e-42).astype(np.float32)
    hy = dict(lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-30, weight_decay=0.01)
    sh = make_shard(p, g, m, v, 0)
    assert ((m.view(np.uint32) & 0x7F800000) == 0).all()  # every input moment is denormal or 0
    d = pk.to_u64(pk.adamw_commit(sh, 2, g_hyper(hy)))[0]
    b = np.zeros(n, np.uint16)
    assert d == oracle.commit_and_digest(p, g, m, v, b, o_hyper(hy), 2, 0)
    _compare_full(sh, p, m, v, b)
    assert ((m.view(np.uint32) & 0x7F800000) == 0).sum() > n // 2  # and so are most outputs


def test_shard_digest_of_arbitrary_bits():
    """shard_digest is integer work only: any bit patterns, NaNs included."""
    import torch

    pk = _pk()
    rng = np.random.default_rng(6)
    n = 300001
    arr = [rng.integers(0, 2 ** 32, n, dtype=np.uint64).astype(np.uint32).view(np.float32) for _ in range(3)]
    t = [torch.from_numpy(a.copy()).cuda() for a in arr]
    sh = pk.Shard(t[0], None, t[1], t[2], None, global_offset=123456789)
    assert pk.to_u64(pk.shard_digest(sh))[0] == oracle.state_digest(*arr, 123456789)


def test_digest_composes_over_sub_shards():
    """Digests of sub-shard views (with their own offsets) sum to the digest
    of the whole, on the GPU."""
    import torch

    pk = _pk()
    w = wl.WORKLOADS["decoder1b_shard16"]
    n = 1_000_003
    p, g, m, v = wl.arrays_host(w, 0, n)
    tp, tm, tv = (torch.from_numpy(a).cuda() for a in (p, m, v))
    whole = pk.to_u64(pk.shard_digest(pk.Shard(tp, None, tm, tv, None, 99)))[0]
    cuts = [0, 1, 4097, 500000, 999999, n]
    s = 0
    for a, z in zip(cuts[:-1], cuts[1:]):
        s += pk.to_u64(pk.shard_digest(pk.Shard(tp[a:z], None, tm[a:z], tv[a:z], None, 99 + a)))[0]
    assert s & M64 == whole == oracle.state_digest(p, m, v, 99)


def test_state_breaks_are_detected():
    """A commit applied to only part of the shard gives a digest different
    from both the frontier before and after; applying a commit twice differs
    from applying it once."""
    import torch

    pk = _pk()
    w = wl.WORKLOADS["decoder1b_shard16"]
    n = 1 << 20
    p, g, m, v = wl.arrays_host(w, 0, n)
    before = oracle.state_digest(p, m, v, w.global_offset)
    full = make_shard(p, g, m, v, w.global_offset)
    after = pk.to_u64(pk.adamw_commit(full, 100, g_hyper(H)))[0]
    half = make_shard(p, g, m, v, w.global_offset)
    hv = pk.Shard(half.param[: n // 2], half.grad[: n // 2], half.exp_avg[: n // 2], half.exp_avg_sq[: n // 2],
                  half.param_bf16[: n // 2], w.global_offset)
    pk.adamw_commit(hv, 100, g_hyper(H))
    torn = pk.to_u64(pk.shard_digest(half))[0]
    assert len({before, after, torn}) == 3
    twice = pk.to_u64(pk.adamw_commit(full, 100, g_hyper(H)))[0]
    assert twice != after
    del torch


def test_stream_probe_moves_the_bytes():
    import torch

    pk = _pk()
    n = 1 << 20
    a, b_, c, d = (torch.randn(n, device="cuda") for _ in range(4))
    ref = [(a + b_).clone(), c.clone(), d.clone()]
    h = torch.zeros(n, dtype=torch.int16, device="cuda")
    pk.stream_probe(a, b_, c, d, a, c, d, h)
    assert torch.equal(a, ref[0]) and torch.equal(c, ref[1]) and torch.equal(d, ref[2])
    top = (ref[0].view(torch.int32) >> 16).to(torch.int16)
    assert torch.equal(h, top)


def test_binding_checks_result_and_probe_tensors():
    """Destinations for result slots and the probe's tensors are checked
    before anything reaches the library."""
    import torch

    pk = _pk()
    w = wl.WORKLOADS["tiny"]
    p, g, m, v = wl.arrays_host(w, 0, 4096)
    sh = make_shard(p, g, m, v, 0)
    for bad in (torch.zeros(1, dtype=torch.int64),                      # on the host
                torch.zeros(1, dtype=torch.float64, device="cuda"),     # wrong dtype
                torch.zeros(0, dtype=torch.int64, device="cuda"),       # too short
                torch.zeros(4, dtype=torch.int64, device="cuda")[::2]):  # not contiguous
        with pytest.raises((TypeError, ValueError)):
            pk.grad_guard(sh, out=bad)
        with pytest.raises((TypeError, ValueError)):
            pk.bf16_digest(sh, out=bad)
    f = torch.zeros(4096, device="cuda")
    h = torch.zeros(4096, dtype=torch.int16, device="cuda")
    with pytest.raises(ValueError):
        pk.stream_probe(f, f, f, torch.zeros(4092, device="cuda"), f, f, f, h)
    with pytest.raises(TypeError):
        pk.stream_probe(f, f, f, f, f, f, f, torch.zeros(4096, device="cuda"))
    ok = torch.zeros(1, dtype=torch.int64, device="cuda")
    assert pk.grad_guard(sh, out=ok) is ok


def test_shard_arena_layout():
    """The placement-aware arena: five arrays at `spacing` strides in one
    pool, gaps usable through take(), and a commit on it equal to the oracle."""
    import torch

    pk = _pk()
    w = wl.WORKLOADS["decoder1b_shard16"]
    n = 3 * 4096 + 17
    arena = pk.ShardArena(n, "cuda", spacing=64 << 20)
    base = arena.pool.data_ptr()
    ptrs = [t.data_ptr() - base for t in (arena.param, arena.grad, arena.exp_avg, arena.exp_avg_sq, arena.param_bf16)]
    assert ptrs == [k * (64 << 20) for k in range(5)]
    extra = arena.take(1 << 20, torch.float32)
    assert extra.numel() == (1 << 18) and extra.data_ptr() - base >= n * 4
    p, g, m, v = wl.arrays_host(w, 0, n)
    for t, a in zip((arena.param, arena.grad, arena.exp_avg, arena.exp_avg_sq), (p, g, m, v)):
        t.copy_(torch.from_numpy(a))
    extra.fill_(7.0)
    sh = arena.shard(w.global_offset)
    d = pk.to_u64(pk.adamw_commit(sh, 100, g_hyper(H)))[0]
    b = np.zeros(n, np.uint16)
    assert d == oracle.commit_and_digest(p, g, m, v, b, o_hyper(H), 100, w.global_offset)
    _compare_full(sh, p, m, v, b)
    assert bool((extra == 7.0).all())
    with pytest.raises(MemoryError):
        arena.take(1 << 30)


def test_stored_oracle_digests():
    """The library reproduces the digests the oracle stored in tests/golden/."""
    import json
    import os

    pk = _pk()
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "oracle_digests.json")
    for c in json.load(open(path)):
        if c["workload"] == "shrunken_mistral":
            w = wl.shrunken_mistral()
            p, g, m, v = wl.arrays_host(w)
            sh = make_shard(p, g, m, v, w.global_offset, segments=w.segments, hypers=w.hypers)
            got = pk.to_u64(pk.adamw_commit(sh, c["step"]))
            assert [f"{x:#018x}" for x in got[:-1]] == c["segment_digests"]
            total = got[-1]
        else:
            w = wl.WORKLOADS[c["workload"]]
            p, g, m, v = wl.arrays_host(w, c["start"], c["count"])
            sh = make_shard(p, g, m, v, w.global_offset + c["start"])
            total = pk.to_u64(pk.adamw_commit(sh, c["step"], g_hyper(w.hypers[0])))[0]
        assert f"{total:#018x}" == c["state_digest"], c["name"]
        assert f"{pk.to_u64(pk.bf16_digest(sh))[-1]:#018x}" == c["bf16_digest"], c["name"]


@pytest.mark.parametrize("segmented", [False, True])
def test_commit_zero_grad_and_guard(segmented):
    """The commit that also zeroes the gradient leaves the committed boundary
    (update applied, gradients +0.0): every output equals the oracle's, the
    guard counts the outstanding gradients before (as numpy does) and none
    after, per segment; padding in the gradient is untouched."""
    import torch

    pk = _pk()
    w = wl.shrunken_mistral() if segmented else wl.WORKLOADS["decoder1b_shard16"]
    n = w.numel if segmented else 100003
    p, g, m, v = wl.arrays_host(w, 0, n)
    g[::97] = 0.0
    g[1::101] = -0.0
    segs = w.segments if segmented else [(0, n, 0)]
    sh = make_shard(p, g, m, v, w.global_offset, segments=w.segments if segmented else None,
                    hypers=w.hypers if segmented else None)
    before = pk.to_u64(pk.grad_guard(sh))
    want_before = [oracle.count_outstanding(g[o:o + ln].copy()) for o, ln, _ in segs]
    assert before[:len(want_before)] == want_before
    assert before[-1] == sum(want_before)
    hy = None if segmented else g_hyper(H)
    got = pk.to_u64(pk.adamw_commit(sh, w.first_step, hy, zero_grad=True))
    b = np.zeros(n, np.uint16)
    g_ref = g.copy()
    per = []
    for o, ln, hi in segs:
        sl = slice(o, o + ln)
        hyper = o_hyper(w.hypers[hi]) if segmented else o_hyper(H)
        per.append(oracle.commit_and_digest(p[sl], g[sl], m[sl], v[sl], b[sl], hyper, w.first_step,
                                            w.global_offset + o))
        gz = g_ref[sl].copy()
        oracle.zero_grad(gz)
        g_ref[sl] = gz
    want = per + [sum(per) & M64] if segmented else [per[0]]
    assert got == want
    _compare_full(sh, p, m, v, b)
    assert_bitwise("grad", host(sh.grad), g_ref)
    after = pk.to_u64(pk.grad_guard(sh))
    assert after == [0] * len(after)
    del torch


def _bf16_arrays(w, start, count):
    p, g, m, v = wl.arrays_host(w, start, count)
    return [oracle.bf16_rne_bits(a.view(np.uint32)) for a in (p, g, m, v)]


@pytest.mark.parametrize("n,shift", [(1, 0), (7, 3), (4096, 0), (4097, 0), (100003, 5), (1 << 20, 0)])
def test_bf16_state_commit(n, shift):
    """BF16 state (the paper's precision): p', m', v' and the digest bit for
    bit, on ragged sizes and on views off the 16-byte grid."""
    import torch

    pk = _pk()
    w = wl.WORKLOADS["mistral7b_shard16"]
    p, g, m, v = _bf16_arrays(w, 0, n)
    full = [torch.zeros(n + 16, dtype=torch.int16, device="cuda") for _ in range(4)]
    views = []
    for t, a in zip(full, (p, g, m, v)):
        t[shift:shift + n] = torch.from_numpy(a.view(np.int16)).cuda()
        views.append(t[shift:shift + n])
    sh = pk.ShardBf16(*views, global_offset=w.global_offset)
    got = pk.to_u64(pk.adamw_commit_bf16(sh, 5, g_hyper(H)))[0]
    want = oracle.commit_and_digest_bf16(p, g, m, v, o_hyper(H), 5, w.global_offset)
    for name, t, ref in (("param", sh.param, p), ("exp_avg", sh.exp_avg, m), ("exp_avg_sq", sh.exp_avg_sq, v)):
        assert_bitwise(name, host(t).view(np.uint16), ref)
    assert got == want
    assert pk.to_u64(pk.shard_digest_bf16(sh))[0] == want
    for t in full:
        h = host(t)
        assert not h[:shift].any() and not h[shift + n:].any()


def test_bf16_state_segments():
    """BF16 state over the shrunken Mistral layout with per-segment hypers."""
    import torch

    pk = _pk()
    w = wl.shrunken_mistral()
    p, g, m, v = _bf16_arrays(w, 0, w.numel)
    t = [torch.from_numpy(a.view(np.int16).copy()).cuda() for a in (p, g, m, v)]
    sh = pk.ShardBf16(*t, global_offset=w.global_offset, segments=w.segments,
                      hypers=[g_hyper(h) for h in w.hypers])
    got = pk.to_u64(pk.adamw_commit_bf16(sh, 5))
    per = []
    for o, ln, hi in w.segments:
        sl = slice(o, o + ln)
        pp, gg, mm, vv = (a[sl].copy() for a in (p, g, m, v))
        per.append(oracle.commit_and_digest_bf16(pp, gg, mm, vv, o_hyper(w.hypers[hi]), 5, w.global_offset + o))
        p[sl], m[sl], v[sl] = pp, mm, vv
    assert got == per + [sum(per) & M64]
    for name, tt, ref in (("param", sh.param, p), ("exp_avg", sh.exp_avg, m), ("exp_avg_sq", sh.exp_avg_sq, v)):
        assert_bitwise(name, host(tt).view(np.uint16), ref)
@pytest.mark.parametrize("seed", range(3))
def test_bf16_state_random_segment_tables(seed):
    """BF16 state over seeded random segment tables (as for binary32 state):
    per-segment digests, their sum, every output, padding untouched, and the
    standalone digest."""
    import torch

    pk = _pk()
    segs, n, goff, hypers = _random_segment_table(2000 + seed)
    w = wl.WORKLOADS["mistral7b_shard16"]
    p, g, m, v = _bf16_arrays(w, 0, n)
    t = [torch.from_numpy(a.view(np.int16).copy()).cuda() for a in (p, g, m, v)]
    sh = pk.ShardBf16(*t, global_offset=goff, segments=segs, hypers=[g_hyper(h) for h in hypers])
    got = pk.to_u64(pk.adamw_commit_bf16(sh, 9))
    p0, m0, v0 = p.copy(), m.copy(), v.copy()
    per = []
    for o, ln, hi in segs:
        sl = slice(o, o + ln)
        pp, gg, mm, vv = (a[sl].copy() for a in (p, g, m, v))
        per.append(oracle.commit_and_digest_bf16(pp, gg, mm, vv, o_hyper(hypers[hi]), 9, goff + o))
        p[sl], m[sl], v[sl] = pp, mm, vv
    assert got == per + [sum(per) & M64]
    for name, tt, ref in (("param", sh.param, p), ("exp_avg", sh.exp_avg, m), ("exp_avg_sq", sh.exp_avg_sq, v)):
        assert_bitwise(name, host(tt).view(np.uint16), ref)
    covered = np.zeros(n, bool)
    for o, ln, _ in segs:
        covered[o:o + ln] = True
    assert np.array_equal(p[~covered], p0[~covered])
    want = [oracle.state_digest_bf16(p[o:o + ln], m[o:o + ln], v[o:o + ln], goff + o) for o, ln, _ in segs]
    assert pk.to_u64(pk.shard_digest_bf16(sh)) == want + [sum(want) & M64]




def test_bf16_state_edge_operands():
    """Operands of the bias-corrected step at the edges of what training
    produces, through the BF16-state commit.  With beta1 = beta2 = 1/2 and
    g = 0 a planted m or v gives m' = m / 2 and v' = v / 2 exactly: m' =
    2^-63, one bf16 step below it, -2^-63, just below 2, 2, -0 and 0 (one in
    each wave of a tile), v' just below 2^64 and 2^64.  Then eps at 2^-57,
    2^-56, 2^44 and 2^45 (the denominator from the root alone, and from eps
    alone), and beta2 = 1 - 2^-24 at step 1, where rs_bc2 = 2^12, its largest value.
    Every output and the digest bit for bit against the oracle."""
    import torch

    pk = _pk()
    w = wl.WORKLOADS["mistral7b_shard16"]
    n = 16 * 4096
    p0, g0, m0, v0 = _bf16_arrays(w, 0, n)

    def run(p, g, m, v, h, step):
        t = [torch.from_numpy(a.view(np.int16).copy()).cuda() for a in (p, g, m, v)]
        sh = pk.ShardBf16(*t, global_offset=w.global_offset)
        got = pk.to_u64(pk.adamw_commit_bf16(sh, step, g_hyper(h)))[0]
        oracle.adamw_commit_bf16(p, g, m, v, o_hyper(h), step)
        for name, dev, ref in (("param", t[0], p), ("exp_avg", t[2], m), ("exp_avg_sq", t[3], v)):
            assert_bitwise(name, host(dev).view(np.uint16), ref)
        assert got == oracle.state_digest_bf16(p, m, v, w.global_offset)

    p, g, m, v = (a.copy() for a in (p0, g0, m0, v0))
    plant_m = {  # tile: m bits (m' = m / 2)
        4: 0x2080,   # m' = 2^-63, in range
        5: 0x207F,   # m' one step below 2^-63
        6: 0xA080,   # m' = -2^-63
        7: 0x407F,   # m' just below 2
        8: 0x4080,   # m' = 2
        9: 0x8000,   # m' = -0
    }
    for tile, mb in plant_m.items():
        e = tile * 4096 + 1234
        m[e], g[e] = mb, 0
    for tile, vb in ((10, 0x5FFF), (11, 0x6000)):  # v' just below 2^64, and 2^64
        e = tile * 4096 + 77
        v[e], g[e] = vb, 0
    for k in range(4):  # tile 12: m' = 0 in each of its four waves
        e = 12 * 4096 + k * 512 + 9
        m[e], g[e] = 0, 0
    run(p, g, m, v, dict(H, beta1=0.5, beta2=0.5), 3)
    for eps in (2.0 ** -57, 2.0 ** -56, 2.0 ** 44, 2.0 ** 45):
        p, g, m, v = (a.copy() for a in (p0, g0, m0, v0))
        run(p, g, m, v, dict(H, eps=eps), 3)
    p, g, m, v = (a.copy() for a in (p0, g0, m0, v0))
    run(p, g, m, v, dict(H, beta2=float(np.float32(1.0) - np.float32(2.0 ** -24))), 1)
    del torch


def test_bf16_state_square_root_forms():
    """The BF16-state commit takes a short exact square root in waves whose
    second moments all lie in [2^-96, +inf) and the full one in any other
    wave.  Waves planted on both sides of the boundary (v' = 2^-96 exactly,
    one bf16 step below it, a denormal, zero, infinity; a whole tile of
    zeros) and untouched waves: every output and the digest bit for bit
    against the oracle."""
    import torch

    pk = _pk()
    w = wl.WORKLOADS["mistral7b_shard16"]
    n = 16 * 4096
    p, g, m, v = _bf16_arrays(w, 0, n)
    plant = {  # element: (v bits, g bits) with beta2 = 0.5, so v' = v / 2 when g = 0
        4 * 4096 + 5: (0x0000, 0x0000),          # v' = 0
        5 * 4096 + 1000: (0x1000, 0x0000),       # v = 2^-95: v' = 2^-96, in range
        6 * 4096 + 2000: (0x0FFF, 0x0000),       # v' one step below 2^-96
        7 * 4096 + 3000: (0x0001, 0x0000),       # denormal v, v' denormal
        8 * 4096 + 10: (0x7F80, 0x0000),         # v = +inf
    }
    for e, (vb, gb) in plant.items():
        v[e], g[e] = vb, gb
    v[9 * 4096:10 * 4096] = 0  # a whole tile of zero moments and gradients
    g[9 * 4096:10 * 4096] = 0
    m[9 * 4096:10 * 4096] = 0
    for k in range(4):  # tile 10: one element out of range in each of its four waves
        e = 10 * 4096 + k * 512 + 7
        v[e], g[e] = 0x0001, 0x0000
    h = dict(H, beta2=0.5)
    t = [torch.from_numpy(a.view(np.int16).copy()).cuda() for a in (p, g, m, v)]
    sh = pk.ShardBf16(*t, global_offset=w.global_offset)
    got = pk.to_u64(pk.adamw_commit_bf16(sh, 3, g_hyper(h)))[0]
    oracle.adamw_commit_bf16(p, g, m, v, o_hyper(h), 3)
    for name, dev, ref in (("param", t[0], p), ("exp_avg", t[2], m), ("exp_avg_sq", t[3], v)):
        assert_bitwise(name, host(dev).view(np.uint16), ref)
    assert got == oracle.state_digest_bf16(p, m, v, w.global_offset)
