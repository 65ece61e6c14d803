"""Pins of the CPU oracle against facts outside it (no GPU).

Each test names what it is pinned to: a published test vector, a closed form,
an exact error bound, a special case that reduces to a textbook identity, a
library routine, brute force, or an algebraic invariant of the digest.
"""
import os
import random
import subprocess
import tempfile
from fractions import Fraction

import numpy as np
import pytest

import oracle
import workloads as wl

M64 = (1 << 64) - 1
ULP_EXP = 2.0 ** -24  # unit roundoff of binary32


def f32(x):
    return float(np.float32(x))


def ulp(x):
    x = np.abs(np.asarray(x, dtype=np.float32))
    return np.spacing(x).astype(np.float64)


# ---------------------------------------------------------------------------
# splitmix64: published outputs
# ---------------------------------------------------------------------------

def test_splitmix64_published_vectors():
    """Pin: splitmix64 with state 0 first outputs 0xE220A8397B1DCDAF, and the
    published sequence for seed 1234567 (the generator adds gamma each call)."""
    gamma = 0x9E3779B97F4A7C15
    assert oracle.splitmix64(0) == 0xE220A8397B1DCDAF
    seq = [oracle.splitmix64((1234567 + k * gamma) & M64) for k in range(5)]
    assert seq == [
        6457827717110365317,
        3203168211198807973,
        9817491932198370423,
        4593380528125082431,
        16408922859458223821,
    ]


def test_splitmix64_is_injective_on_sample():
    """splitmix64 is a bijection of 2^64 (each step is invertible): no collision
    on a sample that includes words differing in one bit."""
    xs = [random.Random(7).getrandbits(64) for _ in range(2000)]
    xs += [1 << b for b in range(64)] + [0]
    outs = {oracle.splitmix64(x) for x in set(xs)}
    assert len(outs) == len(set(xs))


# ---------------------------------------------------------------------------
# bf16 round-to-nearest-even
# ---------------------------------------------------------------------------

def test_bf16_exhaustive_against_nearest_by_distance(root, tmp_path):
    """Pin: all 2^32 binary32 patterns against an independent nearest-neighbour
    search in double (ties to even, overflow to infinity; NaN stays a quiet NaN
    of the same sign)."""
    exe = tmp_path / "bf16_nearest"
    subprocess.run(
        ["gcc", "-O2", "-fopenmp", "-o", str(exe), os.path.join(root, "tests", "native", "bf16_nearest.c"),
         "-ldl", "-lm"],
        check=True,
    )
    out = subprocess.run(
        [str(exe), os.path.join(root, "oracle", "liboracle.so"), "oracle_bf16_rne"],
        check=True, capture_output=True, text=True,
    ).stdout.split()
    bad, nans = int(out[0]), int(out[1])
    assert nans == 2 * (2 ** 23 - 1)
    assert bad == 0


def test_bf16_hand_points():
    """Textbook RNE points: exact, ties to even in both directions, overflow."""
    cases = {
        0x3F800000: 0x3F80,  # 1.0
        0x3F808000: 0x3F80,  # tie, kept part even -> down
        0x3F818000: 0x3F82,  # tie, kept part odd -> up
        0x3F808001: 0x3F81,  # above the tie -> up
        0x3F807FFF: 0x3F80,  # below the tie -> down
        0x7F7FFFFF: 0x7F80,  # FLT_MAX -> +inf
        0xFF7FFFFF: 0xFF80,  # -FLT_MAX -> -inf
        0x7F800000: 0x7F80,  # +inf
        0x80000000: 0x8000,  # -0
        0x00000001: 0x0000,  # smallest denormal rounds to +0
        0x00008000: 0x0000,  # tie at zero, even -> 0
        0x00018000: 0x0002,  # denormal tie, odd -> up
    }
    got = oracle.bf16_rne_bits(np.array(list(cases), dtype=np.uint32))
    assert [int(x) for x in got] == list(cases.values())
    nan = oracle.bf16_rne_bits(np.array([0x7F800001, 0xFFC00000, 0x7FBFFFFF], dtype=np.uint32))
    for r, sign in zip(nan, (0, 1, 0)):
        r = int(r)
        assert (r & 0x7F80) == 0x7F80 and (r & 0x7F) != 0 and (r >> 15) == sign and (r & 0x40)


def test_bf16_matches_torch_on_finite_values():
    """Library routine: torch's float32 -> bfloat16 conversion rounds to
    nearest even; compare on random finite patterns."""
    import torch

    rng = np.random.default_rng(3)
    bits = rng.integers(0, 2 ** 32, size=1 << 20, dtype=np.uint64).astype(np.uint32)
    bits = bits[(bits & 0x7F800000) != 0x7F800000]
    t = torch.from_numpy(bits.view(np.float32).copy()).to(torch.bfloat16)
    ref = t.view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(oracle.bf16_rne_bits(bits), ref)


# ---------------------------------------------------------------------------
# AdamW: closed forms, exact error bounds, special cases, library routine
# ---------------------------------------------------------------------------

H0 = oracle.Hyper(lr=3e-4, beta1=0.9, beta2=0.95, eps=1e-8, weight_decay=0.1)


def _fresh(n, seed, m_dist=wl.ZERO, v_dist=wl.ZERO, first=0):
    p = wl.draw(n, first, seed, wl.ARRAY_PARAM, 0, wl.NORMAL(0.02))
    g = wl.draw(n, first, seed, wl.ARRAY_GRAD, 1, wl.NORMAL(1e-3))
    m = wl.draw(n, first, seed, wl.ARRAY_EXP_AVG, 0, m_dist)
    v = wl.draw(n, first, seed, wl.ARRAY_EXP_AVG_SQ, 0, v_dist)
    return p, g, m, v


def test_scalars_closed_form():
    """decay, 1-beta, bias corrections: one rounding of the exact real value
    (checked with exact rationals; the double intermediate is exact or within
    one double rounding, which cannot move these binary32 results)."""
    for step in (1, 2, 5, 18, 100):
        sc = oracle.make_scalars(H0, step)
        lr, b1, b2, wd = (Fraction(f32(x)) for x in (H0.lr, H0.beta1, H0.beta2, H0.weight_decay))
        assert sc["decay"] == f32(float(1 - lr * wd))
        assert sc["omb1"] == f32(float(1 - b1)) and sc["omb2"] == f32(float(1 - b2))
        assert sc["beta1"] == f32(H0.beta1) and sc["beta2"] == f32(H0.beta2) and sc["eps"] == f32(H0.eps)
        ss = lr / (1 - b1 ** step)
        assert abs(sc["step_size"] - float(ss)) <= 0.5 * float(np.spacing(np.float32(sc["step_size"]))) * 1.0001
        rs = 1.0 / np.sqrt(float(1 - b2 ** step))
        assert abs(sc["rs_bc2"] - rs) <= 0.5 * float(np.spacing(np.float32(sc["rs_bc2"]))) * 1.0001


def test_scalars_large_step_and_zero_beta():
    """beta^t underflows: bias corrections vanish (step_size == lr, rs == 1).
    beta1 = 0: step_size == lr at any t."""
    sc = oracle.make_scalars(H0, 10 ** 6)
    assert sc["step_size"] == f32(H0.lr) and sc["rs_bc2"] == 1.0
    sc = oracle.make_scalars(oracle.Hyper(lr=1e-3, beta1=0.0, beta2=0.0, eps=1e-8, weight_decay=0.0), 3)
    assert sc["step_size"] == f32(1e-3) and sc["rs_bc2"] == 1.0 and sc["omb1"] == 1.0 and sc["decay"] == 1.0


def test_first_step_closed_form():
    """Pin: at t = 1 from m = v = 0, m' = (1-b1) g and v' = (1-b2) g^2 exactly in
    binary32 (one and two roundings), and p' is within the exact error bound of
    the real closed form  P = p (1 - lr wd) - lr g / (|g| + eps)."""
    n = 1 << 16
    p, g, m, v = _fresh(n, 11)
    p0 = p.copy()
    b = np.empty(n, np.uint16)
    oracle.adamw_commit(p, g, m, v, b, H0, 1)
    omb1, omb2 = np.float32(1 - np.float32(0.9)), np.float32(1 - np.float32(0.95))
    assert float(omb1) == 1.0 - float(np.float32(0.9))  # 1 - beta1 is exact in binary32
    assert np.array_equal(m, omb1 * g)
    assert np.array_equal(v, omb2 * (g * g))

    lr, wd, eps = f32(H0.lr), f32(H0.weight_decay), f32(H0.eps)
    g64, p64 = g.astype(np.float64), p0.astype(np.float64)
    u = lr * g64 / (np.abs(g64) + eps)
    P = p64 * (1.0 - lr * wd) - u
    err = np.abs(p.astype(np.float64) - P)
    bound = 0.5 * ulp(p) + 3 * ULP_EXP * np.abs(p64) + 12 * ULP_EXP * np.abs(u)
    assert np.all(err <= bound), float(np.max(err / bound))
    # the bound is tight enough to see a dropped term: without weight decay
    # or without bias correction the same check fails
    assert not np.all(np.abs(p64 - u - p) <= bound)
    assert not np.all(np.abs(p64 * (1 - lr * wd) - lr * 0.1 * g64 / (np.sqrt(0.05) * np.abs(g64) + eps) - p) <= bound)


@pytest.mark.parametrize("steps", [3, 10])
def test_constant_gradient_closed_form(steps):
    """Pin: with a constant gradient from m = v = 0, the bias-corrected moments
    equal g and g^2 at every step, so each step moves p by exactly
    lr g/(|g|+eps) after decay:  P_t = P_{t-1} (1 - lr wd) - lr g/(|g|+eps).
    Checked after each step against the real recurrence, with a bound that
    accumulates the per-step rounding (m, v each carry t roundings)."""
    n = 1 << 14
    p, g, m, v = _fresh(n, 12)
    b = np.empty(n, np.uint16)
    lr, wd, eps = f32(H0.lr), f32(H0.weight_decay), f32(H0.eps)
    g64 = g.astype(np.float64)
    u = lr * g64 / (np.abs(g64) + eps)
    P = p.astype(np.float64)
    slack = np.zeros(n)
    for t in range(1, steps + 1):
        oracle.adamw_commit(p, g, m, v, b, H0, t)
        P = P * (1.0 - lr * wd) - u
        slack = slack + 0.5 * ulp(p) + 3 * ULP_EXP * np.abs(P) + (8 + 4 * t) * ULP_EXP * np.abs(u)
        assert np.all(np.abs(p - P) <= slack), (t, float(np.max(np.abs(p - P) / slack)))
        # moments against their own closed forms
        b1t, b2t = float(np.float32(0.9)) ** t, float(np.float32(0.95)) ** t
        assert np.all(np.abs(m - (1 - b1t) * g64) <= 2 * t * ULP_EXP * np.abs(g64) * 1.01)
        assert np.all(np.abs(v - (1 - b2t) * g64 * g64) <= 3 * t * ULP_EXP * g64 * g64 * 1.01)


def test_special_cases_reduce_to_identities():
    """lr = 0 leaves p unchanged; wd = 0 gives decay exactly 1; beta1 = 0 makes
    m' == g; beta2 = 0 makes v' == g*g; bf16 is the RNE of p'."""
    n = 4096
    p, g, m, v = _fresh(n, 13, wl.NORMAL(1e-4), wl.ABS_NORMAL(1e-7))
    b = np.empty(n, np.uint16)
    p0 = p.copy()
    oracle.adamw_commit(p, g, m, v, b, oracle.Hyper(lr=0.0, weight_decay=0.1), 7)
    assert np.array_equal(p, p0)
    p, g, m, v = _fresh(n, 13, wl.NORMAL(1e-4), wl.ABS_NORMAL(1e-7))
    oracle.adamw_commit(p, g, m, v, b, oracle.Hyper(beta1=0.0, beta2=0.0, weight_decay=0.0), 4)
    assert np.array_equal(m, g)
    assert np.array_equal(v, g * g)
    assert np.array_equal(b, oracle.bf16_rne_bits(p.view(np.uint32)))
    assert oracle.make_scalars(oracle.Hyper(weight_decay=0.0), 3)["decay"] == 1.0


def test_matches_torch_adamw_within_ulps():
    """Library routine: torch.optim.AdamW (single-tensor, CPU, fp32) computes
    the same update with other rounding (lerp for m, divide by sqrt(bc2));
    ten warm steps agree to a few ulp."""
    import torch

    n = 1 << 15
    p, g, m, v = _fresh(n, 14, wl.NORMAL(1e-4), wl.ABS_NORMAL(1e-7))
    tp = torch.nn.Parameter(torch.from_numpy(p.copy()))
    opt = torch.optim.AdamW([tp], lr=H0.lr, betas=(H0.beta1, H0.beta2), eps=H0.eps,
                            weight_decay=H0.weight_decay, foreach=False, fused=False)
    # warm state as step 100 for both
    opt.state[tp] = {"step": torch.tensor(100.0), "exp_avg": torch.from_numpy(m.copy()),
                     "exp_avg_sq": torch.from_numpy(v.copy())}
    b = np.empty(n, np.uint16)
    for t in range(101, 111):
        gt = wl.draw(n, 0, 14, wl.ARRAY_GRAD, t, wl.NORMAL(1e-3))
        np.copyto(g, gt)
        p_before = p.copy()
        m_prev = m.copy()
        tp.grad = torch.from_numpy(g.copy())
        opt.step()
        oracle.adamw_commit(p, g, m, v, b, H0, t)
        st = opt.state[tp]
        em, ev = st["exp_avg"].numpy(), st["exp_avg_sq"].numpy()
        # m mixes two terms of either sign: bound by the ulps of the terms
        tol_m = 8 * (ulp(em) + ulp(0.9 * m_prev) + ulp(0.1 * g))
        assert np.all(np.abs(m - em) <= tol_m)
        assert np.all(np.abs(v - ev) <= 16 * ulp(ev) + 1e-30)
        tpn = tp.detach().numpy()
        move = np.abs(tpn.astype(np.float64) - p_before)
        # m' can cancel, so scale the update's rounding by its two terms
        sc = oracle.make_scalars(H0, t)
        den = np.sqrt(v.astype(np.float64)) * sc["rs_bc2"] + sc["eps"]
        terms = sc["step_size"] * (0.9 * np.abs(m_prev) + 0.1 * np.abs(g)) / den
        assert np.all(np.abs(p - tpn) <= 4 * ulp(tpn) + 64 * ULP_EXP * (move + terms))
        # keep the two trajectories identical so differences do not compound
        tp.data.copy_(torch.from_numpy(p))
        st["exp_avg"].copy_(torch.from_numpy(m))
        st["exp_avg_sq"].copy_(torch.from_numpy(v))


def test_commit_bf16_and_digest_agree_with_pieces():
    """commit_and_digest == commit, then digest; bf16 == RNE(p')."""
    n = 5000
    a = _fresh(n, 15, wl.NORMAL(1e-4), wl.ABS_NORMAL(1e-7), first=123)
    b1 = [x.copy() for x in a]
    bb1 = np.empty(n, np.uint16)
    d1 = oracle.commit_and_digest(*b1, bb1, H0, 6, 123)
    b2 = [x.copy() for x in a]
    bb2 = np.empty(n, np.uint16)
    oracle.adamw_commit(*b2, bb2, H0, 6)
    assert d1 == oracle.state_digest(b2[0], b2[2], b2[3], 123)
    assert np.array_equal(bb1, oracle.bf16_rne_bits(b1[0].view(np.uint32)))


# ---------------------------------------------------------------------------
# digest: special cases, brute force and invariants
# ---------------------------------------------------------------------------

def _f(x):
    return oracle.splitmix64(x)


def test_digest_special_cases():
    """One element at index i: the digest is f(bits(p) ^ i) + f(bits(m) ^ i ^ 1<<56)
    + f(bits(v) ^ i ^ 2<<56).  Words are zero-extended (a set sign bit does
    not spill into the index bits); the bf16 digest uses tag 3."""
    z = np.zeros(1, np.float32)
    assert oracle.state_digest(z, z, z, 0) == (_f(0) + _f(1 << 56) + _f(2 << 56)) & M64
    neg0 = np.array([-0.0], np.float32)
    assert oracle.state_digest(neg0, z, z, 0) == (_f(0x80000000) + _f(1 << 56) + _f(2 << 56)) & M64
    one = np.array([1.0], np.float32)
    i = 6_795_022_080
    d = oracle.state_digest(one, z, neg0, i)
    assert d == (_f(0x3F800000 ^ i) + _f(i | 1 << 56) + _f((0x80000000 ^ i) | 2 << 56)) & M64
    assert oracle.bf16_digest(np.array([0x3F80], np.uint16), 5) == _f((0x3F80 ^ 5) | 3 << 56)
    assert oracle.state_digest(np.zeros(0, np.float32), np.zeros(0, np.float32),
                               np.zeros(0, np.float32), 99) == 0


@pytest.mark.parametrize("n", [0, 1, 2, 3, 5, 7, 64, 127, 129, 1000])
def test_digest_brute_force(n):
    """Brute force: the digest of n elements is the sum of the digests of the
    n one-element shards at their own indices (each pinned above)."""
    rng = np.random.default_rng(n)
    p = rng.standard_normal(n).astype(np.float32)
    m = rng.standard_normal(n).astype(np.float32)
    v = np.abs(rng.standard_normal(n)).astype(np.float32)
    o = 2 ** 32 - 3
    total = 0
    for i in range(n):
        pi, mi, vi = (int(a[i:i + 1].view(np.uint32)[0]) for a in (p, m, v))
        total += _f(pi ^ (o + i)) + _f(mi ^ ((o + i) | 1 << 56)) + _f(vi ^ ((o + i) | 2 << 56))
    assert oracle.state_digest(p, m, v, o) == total & M64


def test_digest_partition_invariance():
    """Wrap-around addition is associative and commutative: 1..64 random
    (unaligned) cuts, in any order, sum to the whole-shard digest."""
    n = 10007
    o = 6_795_022_080
    rng = np.random.default_rng(5)
    p, m, v = (rng.standard_normal(n).astype(np.float32) for _ in range(3))
    whole = oracle.state_digest(p, m, v, o)
    for parts in list(range(1, 65)):
        cuts = sorted(set(rng.integers(0, n + 1, size=parts - 1).tolist()) | {0, n})
        pieces = list(zip(cuts[:-1], cuts[1:]))
        rng.shuffle(pieces)
        s = 0
        for a, b in pieces:
            s += oracle.state_digest(p[a:b], m[a:b], v[a:b], o + a)
        assert s & M64 == whole


def test_digest_detects_every_single_bit_flip():
    """f is a bijection, so changing one word always changes its term and the
    digest: flip every bit of one element of each array."""
    n = 257
    rng = np.random.default_rng(8)
    arrs = [rng.standard_normal(n).astype(np.float32) for _ in range(3)]
    base = oracle.state_digest(*arrs, 77)
    idx = 131
    for k in range(3):
        for bit in range(32):
            a = [x.copy() for x in arrs]
            a[k].view(np.uint32)[idx] ^= np.uint32(1 << bit)
            assert oracle.state_digest(*a, 77) != base
    # identical shards give identical digests
    assert oracle.state_digest(*[x.copy() for x in arrs], 77) == base


def test_digest_sees_swaps_and_offsets():
    """Swapping p and m at one index, or moving the shard to another offset,
    changes the digest (array tags and the global index enter every word)."""
    n = 100
    rng = np.random.default_rng(9)
    p, m, v = (rng.standard_normal(n).astype(np.float32) for _ in range(3))
    base = oracle.state_digest(p, m, v, 1000)
    p2, m2 = p.copy(), m.copy()
    p2[10], m2[10] = m[10], p[10]
    assert oracle.state_digest(p2, m2, v, 1000) != base
    assert oracle.state_digest(p, m, v, 1001) != base
    assert oracle.state_digest(p[::-1].copy(), m[::-1].copy(), v[::-1].copy(), 1000) != base


def test_segments_sum_and_padding_excluded():
    """Per-segment digests sum to the total; padding slots are neither
    committed nor digested."""
    w = wl.shrunken_mistral()
    hypers = [oracle.Hyper(**h) for h in w.hypers]
    p, g, m, v = wl.arrays_host(w)
    b = np.zeros(w.numel, np.uint16)
    covered = np.zeros(w.numel, bool)
    for off, ln, _ in w.segments:
        covered[off:off + ln] = True
    assert not covered.all(), "layout should contain padding"
    p2 = p.copy()
    p2[~covered] = 12345.0
    g2, m2, v2, b2 = g.copy(), m.copy(), v.copy(), b.copy()
    per, total = oracle.commit_segments(p, g, m, v, b, w.segments, hypers, 5, w.global_offset)
    per2, total2 = oracle.commit_segments(p2, g2, m2, v2, b2, w.segments, hypers, 5, w.global_offset)
    assert per == per2 and total == total2
    assert sum(per) & M64 == total
    assert np.all(p2[~covered] == 12345.0) and np.all(b2[~covered] == 0)
    per3, total3 = oracle.segment_digests(p, m, v, w.segments, w.global_offset)
    assert per3 == per and total3 == total


def _padding_runs(segments, numel):
    """[start, end) runs of the flat layout that no segment covers."""
    runs, at = [], 0
    for off, ln, _ in segments:
        if off > at:
            runs.append((at, off))
        at = off + ln
    if at < numel:
        runs.append((at, numel))
    return runs


def test_segment_walker_uses_each_segments_hypers_and_position():
    """Pin of the multi-segment walker (per-tensor W, M, V of Sec. III-A, eq. 2,
    each tensor with its own AdamW settings) against facts that do not go
    through it.  At t = 1 from m = v = 0 every element of segment s must show
    its own role's closed-form first step: m' = f32(omb1 g) and
    v' = f32(omb2 f32(g g)) bit for bit (lm_head has beta2 0.99, the others
    0.95), and p' inside the exact first-order bound of
    P = p (1 - lr wd) - lr g / (|g| + eps) with the segment's lr and wd
    (embed and lm_head lr 1.5e-4, norms wd 0).  Padding keeps its bits.  The
    digests must satisfy the flat identity: the state digest of the whole
    committed array at the global offset (no walker involved) equals the
    walkers' total plus the digests of the padding runs, for the committing
    and for the read-only walker."""
    w = wl.shrunken_mistral()
    roles = {hi for _, _, hi in w.segments}
    assert roles == set(range(len(w.hypers))), "every role must own a segment"
    goff = 3 * (1 << 32) + 12345  # a rank whose indices start beyond 2^32
    p, g, m, v = wl.arrays_host(w)
    m[:] = 0.0
    v[:] = 0.0
    b = np.zeros(w.numel, np.uint16)
    p0, g0 = p.copy(), g.copy()
    hypers = [oracle.Hyper(**h) for h in w.hypers]
    per, total = oracle.commit_segments(p, g, m, v, b, w.segments, hypers, 1, goff)

    covered = np.zeros(w.numel, bool)
    for off, ln, hi in w.segments:
        sl = slice(off, off + ln)
        covered[sl] = True
        h = w.hypers[hi]
        lr, wd, eps = f32(h["lr"]), f32(h["weight_decay"]), f32(h["eps"])
        omb1 = np.float32(1.0 - f32(h["beta1"]))
        omb2 = np.float32(1.0 - f32(h["beta2"]))
        gs = g0[sl]
        assert np.array_equal(m[sl], omb1 * gs), ("m'", off, hi)
        assert np.array_equal(v[sl], omb2 * (gs * gs)), ("v'", off, hi)
        g64, p64 = gs.astype(np.float64), p0[sl].astype(np.float64)
        u = lr * g64 / (np.abs(g64) + eps)
        P = p64 * (1.0 - lr * wd) - u
        bound = 0.5 * ulp(p[sl]) + 3 * ULP_EXP * np.abs(p64) + 12 * ULP_EXP * np.abs(u)
        assert np.all(np.abs(p[sl].astype(np.float64) - P) <= bound), ("p'", off, hi)
        assert np.array_equal(b[sl], oracle.bf16_rne_bits(p[sl].view(np.uint32))), ("bf16", off, hi)
    # the checks above tell the roles apart: another role's settings fail them
    for off, ln, hi in w.segments:
        other = [k for k in range(len(w.hypers)) if w.hypers[k] != w.hypers[hi]]
        sl = slice(off, off + ln)
        for k in other:
            h = w.hypers[k]
            lr, wd, eps = f32(h["lr"]), f32(h["weight_decay"]), f32(h["eps"])
            g64, p64 = g0[sl].astype(np.float64), p0[sl].astype(np.float64)
            u = lr * g64 / (np.abs(g64) + eps)
            P = p64 * (1.0 - lr * wd) - u
            bound = 0.5 * ulp(p[sl]) + 3 * ULP_EXP * np.abs(p64) + 12 * ULP_EXP * np.abs(u)
            same_p = np.all(np.abs(p[sl].astype(np.float64) - P) <= bound)
            same_v = np.array_equal(v[sl], np.float32(1.0 - f32(h["beta2"])) * (g0[sl] * g0[sl]))
            assert not (same_p and same_v), (off, hi, k)
    pad = ~covered
    assert pad.any(), "the layout should contain padding"
    assert np.array_equal(p[pad].view(np.uint32), p0[pad].view(np.uint32))
    assert not m[pad].view(np.uint32).any() and not v[pad].view(np.uint32).any() and not b[pad].any()

    runs = _padding_runs(w.segments, w.numel)
    pad_digest = sum(oracle.state_digest(p[a:z], m[a:z], v[a:z], goff + a) for a, z in runs) & M64
    whole = oracle.state_digest(p, m, v, goff)
    assert (total + pad_digest) & M64 == whole
    assert sum(per) & M64 == total
    per_r, total_r = oracle.segment_digests(p, m, v, w.segments, goff)
    assert (total_r + pad_digest) & M64 == whole
    # each segment's digest is the sum of its elements' one-element digests
    # (spot check on the smallest segments, the norms)
    for s, (off, ln, hi) in enumerate(w.segments):
        if ln <= 256:
            one = sum(oracle.state_digest(p[i:i + 1], m[i:i + 1], v[i:i + 1], goff + i)
                      for i in range(off, off + ln)) & M64
            assert one == per[s] == per_r[s], (s, off)


# ---------------------------------------------------------------------------
# workload shapes (the paper's model size)
# ---------------------------------------------------------------------------

def test_mistral_shape_arithmetic():
    """Pin: the paper's Mistral-7B parameter count, 7,248,023,552 (Sec. IV-A),
    from the published architecture; 291 tensors; every size a multiple of 128
    so the 512-byte padded layout has no padding."""
    t = wl.mistral_tensors()
    assert len(t) == 291
    assert sum(n for _, n, _ in t) == 7_248_023_552 == wl.MISTRAL_PARAMS
    segs, total = wl.flat_segments(t)
    assert total == 7_248_023_552
    assert wl.MISTRAL_SHARD16 == 453_001_472 and wl.MISTRAL_SHARD16 % 128 == 0
    assert wl.MISTRAL_SHARD4 == 1_812_005_888
    per_layer = sum(n for name, n, _ in t if name.startswith("model.layers.0."))
    assert per_layer == 218_112_000


# ---------------------------------------------------------------------------
# committed boundary: zeroed gradients and the guard
# ---------------------------------------------------------------------------

def test_guard_counts_nonzero_bit_patterns():
    """Library routine: numpy's count_nonzero over the bit patterns; -0.0 and
    denormals count as outstanding, +0.0 does not."""
    rng = np.random.default_rng(10)
    g = rng.standard_normal(100003).astype(np.float32)
    g[rng.integers(0, g.size, 5000)] = 0.0
    g[:7] = [-0.0, 0.0, 1e-45, -1e-45, np.inf, 0.0, -0.0]
    assert oracle.count_outstanding(g) == int(np.count_nonzero(g.view(np.uint32)))
    oracle.zero_grad(g)
    assert not g.view(np.uint32).any() and oracle.count_outstanding(g) == 0
    assert oracle.count_outstanding(np.zeros(0, np.float32)) == 0


# ---------------------------------------------------------------------------
# BF16 state (the paper's precision for weights and moments)
# ---------------------------------------------------------------------------

def _bf16_state(n, seed):
    p, g, m, v = _fresh(n, seed, wl.NORMAL(1e-4), wl.ABS_NORMAL(1e-7))
    return [oracle.bf16_rne_bits(a.view(np.uint32)) for a in (p, g, m, v)]


def _widen(b):
    return (b.astype(np.uint32) << 16).view(np.float32)


def test_bf16_commit_is_the_rounded_binary32_commit():
    """Pin against the pinned binary32 oracle and the pinned RNE rule: on
    widened bf16 inputs, the bf16 commit's p', m', v' are exactly the RNE
    roundings of the binary32 commit's results."""
    n = 1 << 15
    p, g, m, v = _bf16_state(n, 21)
    P, G, Mm, V = (_widen(a).copy() for a in (p, g, m, v))
    junk = np.empty(n, np.uint16)
    oracle.adamw_commit(P, G, Mm, V, junk, H0, 7)
    oracle.adamw_commit_bf16(p, g, m, v, H0, 7)
    assert np.array_equal(p, oracle.bf16_rne_bits(P.view(np.uint32)))
    assert np.array_equal(m, oracle.bf16_rne_bits(Mm.view(np.uint32)))
    assert np.array_equal(v, oracle.bf16_rne_bits(V.view(np.uint32)))


def test_bf16_first_step_closed_form():
    """t = 1 from m = v = 0 on bf16 state: m' = RNE(f32((1-b1) g)), and p'
    within half a bf16 ulp plus the binary32 bound of the real closed form."""
    n = 1 << 14
    p, g, _, _ = _bf16_state(n, 22)
    m = np.zeros(n, np.uint16)
    v = np.zeros(n, np.uint16)
    p0, g64 = _widen(p).astype(np.float64), _widen(g).astype(np.float64)
    oracle.adamw_commit_bf16(p, g, m, v, H0, 1)
    omb1 = np.float32(1 - np.float32(0.9))
    assert np.array_equal(m, oracle.bf16_rne_bits((omb1 * _widen(g)).view(np.uint32)))
    lr, wd, eps = f32(H0.lr), f32(H0.weight_decay), f32(H0.eps)
    u = lr * g64 / (np.abs(g64) + eps)
    P = p0 * (1.0 - lr * wd) - u
    got = _widen(p).astype(np.float64)
    bf_ulp = np.spacing(np.abs(got).astype(np.float32)).astype(np.float64) * 65536.0
    bound = 0.5 * bf_ulp + 0.5 * ulp(got) + 3 * ULP_EXP * np.abs(p0) + 12 * ULP_EXP * np.abs(u)
    assert np.all(np.abs(got - P) <= bound)


def test_bf16_digest_words_and_partitions():
    """16-bit words are zero-extended; tags as for binary32 state; any
    partition sums to the whole."""
    z = np.zeros(1, np.uint16)
    s = np.array([0x8000], np.uint16)
    assert oracle.state_digest_bf16(s, z, z, 9) == (_f(0x8000 ^ 9) + _f(9 | 1 << 56) + _f(9 | 2 << 56)) & M64
    rng = np.random.default_rng(23)
    n = 5003
    p, m, v = (rng.integers(0, 1 << 16, n, dtype=np.uint16) for _ in range(3))
    whole = oracle.state_digest_bf16(p, m, v, 2 ** 40)
    cuts = [0, 1, 2047, 4096, 5000, n]
    parts = sum(oracle.state_digest_bf16(p[a:b], m[a:b], v[a:b], 2 ** 40 + a) for a, b in zip(cuts, cuts[1:]))
    assert parts & M64 == whole
