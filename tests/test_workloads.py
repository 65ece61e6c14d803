"""The seeded input generator: published Philox vectors, reproducibility, and
the value properties the workloads rely on (no GPU)."""
import numpy as np

import workloads as wl


def test_philox4x32_10_known_answers():
    """Pin: the Random123 known-answer vectors for Philox4x32-10."""
    assert wl.philox4x32_10((0, 0, 0, 0), (0, 0)) == (0x6627E8D5, 0xE169C58D, 0xBC57AC4C, 0x9B00DBD8)
    assert wl.philox4x32_10((0xFFFFFFFF,) * 4, (0xFFFFFFFF,) * 2) == (
        0x408F276D, 0x41C83B0E, 0xA20BC7C6, 0x6D5451FD)
    assert wl.philox4x32_10((0x243F6A88, 0x85A308D3, 0x13198A2E, 0x03707344), (0xA4093822, 0x299F31D0)) == (
        0xD16CFE09, 0x94FDCCEB, 0x5001E420, 0x24126EA1)


def test_values_depend_only_on_global_index():
    """Any chunking of the index range draws the same values; a shard at offset
    o equals that slice of the full vector."""
    full = wl.draw(10000, 0, 3, wl.ARRAY_PARAM, 0, wl.NORMAL(0.02))
    parts = np.concatenate([wl.draw(b - a, a, 3, wl.ARRAY_PARAM, 0, wl.NORMAL(0.02))
                            for a, b in ((0, 1), (1, 4097), (4097, 9999), (9999, 10000))])
    assert np.array_equal(full.view(np.uint32), parts.view(np.uint32))
    # offsets past 2^32 use the high counter word
    hi = wl.draw(8, (1 << 32) + 5, 3, wl.ARRAY_PARAM, 0, wl.NORMAL(0.02))
    lo = wl.draw(8, 5, 3, wl.ARRAY_PARAM, 0, wl.NORMAL(0.02))
    assert not np.array_equal(hi, lo)


def test_streams_are_distinct():
    a = wl.draw(1000, 0, 3, wl.ARRAY_PARAM, 0, wl.NORMAL(1.0))
    assert not np.array_equal(a, wl.draw(1000, 0, 3, wl.ARRAY_GRAD, 0, wl.NORMAL(1.0)))
    assert not np.array_equal(a, wl.draw(1000, 0, 3, wl.ARRAY_PARAM, 1, wl.NORMAL(1.0)))
    assert not np.array_equal(a, wl.draw(1000, 0, 4, wl.ARRAY_PARAM, 0, wl.NORMAL(1.0)))


def test_distribution_shape():
    """N(0, sigma): mean ~ 0 and sd ~ sigma; |N|: non-negative; no denormal
    and no negative zero anywhere; zeros are +0."""
    n = 1 << 20
    x = wl.draw(n, 0, 9, wl.ARRAY_GRAD, 1, wl.NORMAL(1e-3)).astype(np.float64)
    assert abs(x.mean()) < 5e-3 * 1e-3
    assert abs(x.std() / 1e-3 - 1) < 5e-3
    a = wl.draw(n, 0, 9, wl.ARRAY_EXP_AVG_SQ, 0, wl.ABS_NORMAL(1e-7))
    assert (a >= 0).all() and not np.signbit(a).any()
    for arr in (x.astype(np.float32), a):
        bits = arr.view(np.uint32)
        assert not (((bits & 0x7F800000) == 0) & ((bits & 0x7FFFFF) != 0)).any()
        assert not (bits == 0x80000000).any()
    z = wl.draw(100, 0, 9, wl.ARRAY_EXP_AVG, 0, wl.ZERO)
    assert (z.view(np.uint32) == 0).all()


def test_workload_table():
    w = wl.WORKLOADS
    assert w["tiny"].numel == 1 << 20 and w["tiny"].first_step == 1
    assert w["decoder1b_shard16"].global_offset == 1_140_000_000
    assert w["mistral7b_shard16"].global_offset == 6_795_022_080 > 2 ** 32
    assert w["mistral7b_shard4"].global_offset == 5_436_017_664
    whole = w["mistral7b_whole"]
    assert whole.numel == 7_248_023_552 and len(whole.segments) == 291
    assert sum(ln for _, ln, _ in whole.segments) == whole.numel
    norms = [s for s in whole.segments if s[2] == wl.ROLE_ORDER.index("norm")]
    assert len(norms) == 65
