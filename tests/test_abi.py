"""The C ABI without a GPU: the library loads, exports every declared symbol,
and rejects bad arguments before touching the device (validation makes no
HIP call, so fake but well-formed addresses suffice)."""
import ctypes
import os
import re

import pytest

import paper_2609_18178_amd as pk
from paper_2609_18178_amd import _CHyper, _CSegment, _CShard

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions():
    text = open(os.path.join(ROOT, "include", "pactshard.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(pact_[a-z0-9_]+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    lib = pk._lib()
    names = declared_functions()
    assert {"pact_adamw_commit", "pact_shard_digest", "pact_bf16_digest", "pact_strerror"} <= set(names)
    for name in names:
        assert hasattr(lib, name), name
    assert lib.pact_version() >= 100


def test_strerror_is_distinct_per_code():
    texts = {code: pk._strerror(code) for code in (0, -1, -2, -3, -4, -5, -6)}
    assert len(set(texts.values())) == 7
    assert pk._strerror(-99) == "unknown error"


BASE = 1 << 40  # fake device addresses, well aligned, far apart
SPAN = 1 << 34


def fake_shard(n=1024, **kw):
    s = _CShard()
    s.param, s.grad, s.exp_avg, s.exp_avg_sq, s.param_bf16 = (BASE + k * SPAN for k in range(5))
    s.digest_dev = BASE + 5 * SPAN
    s.numel = n
    s.global_offset = 0
    for k, v in kw.items():
        setattr(s, k, v)
    return s


GOOD = _CHyper(3e-4, 0.9, 0.95, 1e-8, 0.1)


def commit(s, step=1, h=GOOD):
    return pk._lib().pact_adamw_commit(ctypes.byref(s), step, ctypes.byref(h) if h is not None else None)


def test_null_and_step_errors():
    lib = pk._lib()
    assert lib.pact_adamw_commit(None, 1, ctypes.byref(GOOD)) == pk.PACT_EINVAL
    assert commit(fake_shard(), step=0) == pk.PACT_EINVAL
    assert commit(fake_shard(), h=None) == pk.PACT_EINVAL
    assert commit(fake_shard(param=None)) == pk.PACT_EINVAL
    assert commit(fake_shard(grad=None)) == pk.PACT_EINVAL
    assert commit(fake_shard(param_bf16=None)) == pk.PACT_EINVAL
    assert commit(fake_shard(digest_dev=None)) == pk.PACT_EINVAL
    assert lib.pact_shard_digest(None) == pk.PACT_EINVAL
    assert lib.pact_digest_slots(None) == pk.PACT_EINVAL


@pytest.mark.parametrize("bad", [
    dict(beta1=1.0), dict(beta1=-0.1), dict(beta2=1.0), dict(beta2=-1e-3), dict(eps=0.0), dict(eps=-1e-8),
    dict(eps=float("nan")), dict(lr=-1e-4), dict(lr=float("inf")), dict(weight_decay=-0.1),
    dict(weight_decay=float("nan")),
])
def test_bad_hyperparameters(bad):
    vals = dict(lr=3e-4, beta1=0.9, beta2=0.95, eps=1e-8, weight_decay=0.1)
    vals.update(bad)
    h = _CHyper(vals["lr"], vals["beta1"], vals["beta2"], vals["eps"], vals["weight_decay"])
    assert commit(fake_shard(), h=h) == pk.PACT_EINVAL


def test_alignment_errors():
    assert commit(fake_shard(param=BASE + 2)) == pk.PACT_EALIGN
    assert commit(fake_shard(exp_avg_sq=BASE + 3 * SPAN + 1)) == pk.PACT_EALIGN
    assert commit(fake_shard(param_bf16=BASE + 4 * SPAN + 1)) == pk.PACT_EALIGN
    assert commit(fake_shard(digest_dev=BASE + 5 * SPAN + 4)) == pk.PACT_EALIGN


def test_overlap_errors():
    assert commit(fake_shard(grad=BASE)) == pk.PACT_EOVERLAP
    assert commit(fake_shard(exp_avg=BASE + 4092)) == pk.PACT_EOVERLAP  # last float of param
    assert commit(fake_shard(digest_dev=BASE + 8)) == pk.PACT_EOVERLAP
    assert commit(fake_shard(param_bf16=BASE + 3 * SPAN + 4094)) == pk.PACT_EOVERLAP


def test_range_errors():
    assert commit(fake_shard(n=16, global_offset=(1 << 56) - 15)) == pk.PACT_ERANGE
    assert commit(fake_shard(n=0, global_offset=1 << 56)) == pk.PACT_ERANGE
    assert commit(fake_shard(n=1 << 62)) == pk.PACT_ERANGE
    # one launch grid holds at most (2^32 - 1) // 256 workgroups of one 4096-element tile each
    max_tiles = ((1 << 32) - 1) // 256
    assert commit(fake_shard(n=(max_tiles + 1) * 4096)) == pk.PACT_ERANGE
    # a grid that just fits passes this check and fails later, on the overlapping fake arrays
    assert commit(fake_shard(n=max_tiles * 4096)) == pk.PACT_EOVERLAP


def _with_segs(segs, hypers=(GOOD,), n=1024):
    s = fake_shard(n=n)
    arr = (_CSegment * max(1, len(segs)))(*[_CSegment(*x) for x in segs]) if segs else None
    hs = (_CHyper * len(hypers))(*hypers) if hypers else None
    if segs is not None:
        s.segs = ctypes.cast(arr, ctypes.POINTER(_CSegment)) if arr is not None else ctypes.cast(
            (_CSegment * 1)(), ctypes.POINTER(_CSegment))
        s.num_segs = len(segs)
    if hs is not None:
        s.hypers = ctypes.cast(hs, ctypes.POINTER(_CHyper))
        s.num_hypers = len(hypers)
    s._keep = (arr, hs)
    return s


@pytest.mark.parametrize("segs,hypers", [
    ([], (GOOD,)),                                   # segs given but empty
    ([(0, 100, 0, 0), (50, 100, 0, 0)], (GOOD,)),     # overlapping
    ([(200, 10, 0, 0), (0, 10, 0, 0)], (GOOD,)),      # not increasing
    ([(1000, 100, 0, 0)], (GOOD,)),                   # beyond numel
    ([(0, 10, 1, 0)], (GOOD,)),                       # hyper index out of range
    ([(0, 10, 0, 7)], (GOOD,)),                       # reserved not zero
    ([(0, 10, 0, 0)], (_CHyper(3e-4, 1.5, 0.95, 1e-8, 0.1),)),  # bad hyper in the table
    ([(0, 10, 0, 0)], ()),                            # no hyper table
])
def test_segment_table_errors(segs, hypers):
    s = _with_segs(segs, hypers)
    assert commit(s, h=None) == pk.PACT_EINVAL


def test_digest_slots():
    lib = pk._lib()
    assert lib.pact_digest_slots(ctypes.byref(fake_shard())) == 1
    s = _with_segs([(0, 10, 0, 0), (16, 4, 0, 0), (100, 0, 0, 0)])
    assert lib.pact_digest_slots(ctypes.byref(s)) == 4
    # the slot range must not overlap an array either
    s.digest_dev = BASE + 4 * SPAN + 2048 - 16
    assert commit(s, h=None) == pk.PACT_EOVERLAP


def test_commit_ex_and_guard_validation():
    lib = pk._lib()
    s = fake_shard()
    assert lib.pact_adamw_commit_ex(ctypes.byref(s), 1, ctypes.byref(GOOD), 4) == pk.PACT_EINVAL
    assert lib.pact_adamw_commit_ex(ctypes.byref(s), 1, ctypes.byref(GOOD), 0x80000000) == pk.PACT_EINVAL
    # both known flags pass the flag check (and validation then stops at step 0)
    assert lib.pact_adamw_commit_ex(ctypes.byref(s), 0, ctypes.byref(GOOD), 3) == pk.PACT_EINVAL
    assert lib.pact_adamw_commit_ex(ctypes.byref(s), 0, ctypes.byref(GOOD), 1) == pk.PACT_EINVAL
    assert lib.pact_adamw_commit_ex(ctypes.byref(fake_shard(grad=BASE)), 1, ctypes.byref(GOOD), 1) == \
        pk.PACT_EOVERLAP
    assert lib.pact_grad_guard(None, BASE + 7 * SPAN) == pk.PACT_EINVAL
    assert lib.pact_grad_guard(ctypes.byref(fake_shard(grad=None)), BASE + 7 * SPAN) == pk.PACT_EINVAL
    assert lib.pact_grad_guard(ctypes.byref(fake_shard()), None) == pk.PACT_EINVAL
    assert lib.pact_grad_guard(ctypes.byref(fake_shard()), BASE + 7 * SPAN + 4) == pk.PACT_EALIGN
    assert lib.pact_grad_guard(ctypes.byref(fake_shard()), BASE + SPAN + 8) == pk.PACT_EOVERLAP


def test_bf16_shard_validation():
    from paper_2609_18178_amd import _CShardBf16

    lib = pk._lib()
    s = _CShardBf16()
    s.param, s.grad, s.exp_avg, s.exp_avg_sq = (BASE + k * SPAN for k in range(4))
    s.digest_dev = BASE + 5 * SPAN
    s.numel = 1024
    assert lib.pact_digest_slots_bf16(ctypes.byref(s)) == 1
    assert lib.pact_workspace_bytes_bf16(ctypes.byref(s)) == 16 * 32 * 8
    assert lib.pact_adamw_commit_bf16(ctypes.byref(s), 0, ctypes.byref(GOOD)) == pk.PACT_EINVAL
    s.param = BASE + 1
    assert lib.pact_adamw_commit_bf16(ctypes.byref(s), 1, ctypes.byref(GOOD)) == pk.PACT_EALIGN
    s.param = BASE + SPAN + 2046  # last element overlaps grad's first
    assert lib.pact_adamw_commit_bf16(ctypes.byref(s), 1, ctypes.byref(GOOD)) == pk.PACT_EOVERLAP
    assert lib.pact_shard_digest_bf16(None) == pk.PACT_EINVAL


def test_workspace_contract():
    lib = pk._lib()
    s = fake_shard()
    need = lib.pact_workspace_bytes(ctypes.byref(s))
    assert need == 16 * 32 * 8
    seg = _with_segs([(0, 10, 0, 0), (16, 4, 0, 0), (100, 0, 0, 0)])
    assert lib.pact_workspace_bytes(ctypes.byref(seg)) == 3 * need
    ws = BASE + 6 * SPAN
    assert commit(fake_shard(workspace=ws, workspace_bytes=need - 8)) == pk.PACT_EINVAL
    assert commit(fake_shard(workspace=ws + 4, workspace_bytes=need)) == pk.PACT_EALIGN
    assert commit(fake_shard(workspace=BASE + 2 * SPAN + 1024, workspace_bytes=need)) == pk.PACT_EOVERLAP
    assert commit(fake_shard(workspace=BASE + 5 * SPAN, workspace_bytes=need)) == pk.PACT_EOVERLAP
    assert lib.pact_workspace_bytes(None) == pk.PACT_EINVAL


def test_segment_count_limit():
    s = fake_shard()
    s.segs = ctypes.cast((_CSegment * 1)(), ctypes.POINTER(_CSegment))
    s.num_segs = (1 << 24) + 1
    assert commit(s, h=None) == pk.PACT_EINVAL


def test_probe_errors():
    lib = pk._lib()
    a = [BASE + k * SPAN for k in range(8)]
    assert lib.pact_stream_probe(*a, 1023, None) == pk.PACT_EINVAL
    assert lib.pact_stream_probe(*(a[:7] + [BASE + 7 * SPAN + 4]), 1024, None) == pk.PACT_EALIGN


def test_binding_refuses_cpu_tensors():
    import torch

    t = torch.zeros(16)
    with pytest.raises(TypeError):
        pk.Shard(t, t, t, t, torch.zeros(16, dtype=torch.int16))
    with pytest.raises(TypeError):
        pk.stream_probe(t, t, t, t, t, t, t, torch.zeros(16, dtype=torch.int16))


def test_binding_fails_loudly_without_library(monkeypatch):
    monkeypatch.setattr(pk, "_LIB", None)
    monkeypatch.setattr(pk, "library_path", "/nonexistent/libpactshard.so")
    with pytest.raises(RuntimeError, match="no fallback"):
        pk._lib()


def test_header_is_c99_and_matches_the_binding(tmp_path):
    """pactshard.h compiles as strict C99, and every struct the binding
    mirrors with ctypes has the header's size and field offsets; the error
    codes and flags agree too."""
    import json
    import subprocess

    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    exe = tmp_path / "abi_layout"
    subprocess.run(["gcc", "-std=c99", "-pedantic", "-Wall", "-Wextra", "-Werror", "-I", os.path.join(root, "include"),
                    "-o", str(exe), os.path.join(root, "tests", "native", "abi_layout.c")], check=True)
    c = json.loads(subprocess.run([str(exe)], check=True, capture_output=True, text=True).stdout)
    mirrors = {"pact_hyper": pk._CHyper, "pact_segment": pk._CSegment, "pact_shard": pk._CShard,
               "pact_shard_bf16": pk._CShardBf16, "pact_arena_layout": pk._CArenaLayout}
    for name, cls in mirrors.items():
        assert ctypes.sizeof(cls) == c[name]["sizeof"], name
        py_fields = {f[0]: getattr(cls, f[0]).offset for f in cls._fields_}
        c_fields = c[name]["fields"]
        # the binding names fields as the header does
        assert py_fields == c_fields, (name, py_fields, c_fields)
    for code, value in c["codes"].items():
        assert getattr(pk, code) == value, code


# ---------------------------------------------------------------------------
# Seeded fuzz of the argument validation: a random well-formed shard (fake,
# aligned, disjoint device addresses) with exactly one injected violation of
# a known kind; the call must report exactly that kind.  Every case is
# invalid, so nothing is ever enqueued.
# ---------------------------------------------------------------------------
_VIOLATIONS = {
    # name: (expected code, applies to the state digest call too)
    "null_param": (pk.PACT_EINVAL, True), "null_grad": (pk.PACT_EINVAL, False),
    "null_bf16": (pk.PACT_EINVAL, False), "null_digest": (pk.PACT_EINVAL, True),
    "step0": (pk.PACT_EINVAL, False), "bad_hyper": (pk.PACT_EINVAL, False),
    "no_hyper": (pk.PACT_EINVAL, False), "flags": (pk.PACT_EINVAL, False),
    "range": (pk.PACT_ERANGE, True), "misalign_m": (pk.PACT_EALIGN, True),
    "misalign_bf16": (pk.PACT_EALIGN, False), "misalign_digest": (pk.PACT_EALIGN, True),
    "overlap_arrays": (pk.PACT_EOVERLAP, True), "overlap_digest": (pk.PACT_EOVERLAP, True),
    "ws_small": (pk.PACT_EINVAL, True), "ws_misalign": (pk.PACT_EALIGN, True),
    "ws_overlap": (pk.PACT_EOVERLAP, True), "seg_reserved": (pk.PACT_EINVAL, True),
    "seg_order": (pk.PACT_EINVAL, True), "seg_beyond": (pk.PACT_EINVAL, True),
    "seg_hyper_index": (pk.PACT_EINVAL, False), "seg_bad_hyper": (pk.PACT_EINVAL, False),
    "seg_count0": (pk.PACT_EINVAL, True),
}
_SEG_ONLY = {"seg_reserved", "seg_order", "seg_beyond", "seg_hyper_index", "seg_bad_hyper", "seg_count0"}
_FLAT_ONLY = {"bad_hyper", "no_hyper"}


def _random_hyper(rng):
    return _CHyper(float(rng.uniform(0, 1e-2)), float(rng.uniform(0, 0.999)), float(rng.uniform(0, 0.9999)),
                   float(rng.uniform(1e-12, 1e-3)), float(rng.uniform(0, 0.5)))


def _fuzz_case(rng, violation):
    import numpy as np

    n = int(rng.integers(1, 1 << 20))
    s = _CShard()
    arr = [BASE + k * SPAN + 16 * int(rng.integers(0, 1 << 16)) for k in range(5)]
    s.param, s.grad, s.exp_avg, s.exp_avg_sq, s.param_bf16 = arr
    s.numel = n
    s.global_offset = int(rng.integers(0, (1 << 56) - n))
    s.digest_dev = BASE + 5 * SPAN + 8 * int(rng.integers(0, 1 << 16))
    keep = []
    segmented = violation in _SEG_ONLY or (violation not in _FLAT_ONLY and rng.random() < 0.5)
    if segmented:
        k = int(rng.integers(2, 40))
        cuts = np.sort(rng.integers(0, n + 1, size=2 * k))
        segs = [[int(cuts[2 * i]), int(cuts[2 * i + 1] - cuts[2 * i]), 0, 0] for i in range(k)]
        hyps = [_random_hyper(rng) for _ in range(int(rng.integers(1, 4)))]
        for sg in segs:
            sg[2] = int(rng.integers(0, len(hyps)))
        if violation == "seg_reserved":
            segs[int(rng.integers(0, k))][3] = 1
        elif violation == "seg_order":
            i = int(rng.integers(0, k - 1))
            while segs[i] == segs[i + 1]:  # swapping equal entries changes nothing
                segs[i + 1][0] += 1
                segs[i + 1][1] = max(0, segs[i + 1][1] - 1)
            segs[i], segs[i + 1] = segs[i + 1], segs[i]
        elif violation == "seg_beyond":
            segs[-1][1] = n - segs[-1][0] + int(rng.integers(1, 1000))
        elif violation == "seg_hyper_index":
            segs[int(rng.integers(0, k))][2] = len(hyps)
        elif violation == "seg_bad_hyper":
            hyps[segs[int(rng.integers(0, k))][2]] = _CHyper(3e-4, 1.0, 0.95, 1e-8, 0.1)
        table = (_CSegment * k)(*[_CSegment(*sg) for sg in segs])
        htable = (_CHyper * len(hyps))(*hyps)
        keep += [table, htable]
        s.segs = ctypes.cast(table, ctypes.POINTER(_CSegment))
        s.num_segs = 0 if violation == "seg_count0" else k
        s.hypers = ctypes.cast(htable, ctypes.POINTER(_CHyper))
        s.num_hypers = len(hyps)
        hyper = None
    else:
        hyper = _random_hyper(rng)
        if violation == "bad_hyper":
            bad = [("lr", -1e-3), ("beta1", 1.0), ("beta2", float("nan")), ("eps", 0.0), ("weight_decay", -0.1)]
            name, val = bad[int(rng.integers(0, len(bad)))]
            setattr(hyper, name, val)
    if rng.random() < 0.5 or violation.startswith("ws_"):
        need = pk._lib().pact_workspace_bytes(ctypes.byref(s))
        s.workspace = BASE + 6 * SPAN + 8 * int(rng.integers(0, 1 << 16))
        s.workspace_bytes = need + 8 * int(rng.integers(0, 4))
        if violation == "ws_small":
            s.workspace_bytes = need - 8
        elif violation == "ws_misalign":
            s.workspace += 4
        elif violation == "ws_overlap":
            s.workspace = s.exp_avg + 8 * int(rng.integers(0, n // 2 + 1))
    if violation == "null_param":
        s.param = None
    elif violation == "null_grad":
        s.grad = None
    elif violation == "null_bf16":
        s.param_bf16 = None
    elif violation == "null_digest":
        s.digest_dev = None
    elif violation == "range":
        s.global_offset = (1 << 56) - n + int(rng.integers(1, 1 << 20))
    elif violation == "misalign_m":
        s.exp_avg += int(rng.integers(1, 4))
    elif violation == "misalign_bf16":
        s.param_bf16 += 1
    elif violation == "misalign_digest":
        s.digest_dev += 4
    elif violation == "overlap_arrays":
        s.exp_avg_sq = s.param + 4 * int(rng.integers(0, n))
    elif violation == "overlap_digest":
        s.digest_dev = s.exp_avg + 8 * int(rng.integers(0, n // 2))  # an array both calls read
    step = 0 if violation == "step0" else int(rng.integers(1, 1 << 20))
    flags = (1 << int(rng.integers(2, 32))) if violation == "flags" else int(rng.integers(0, 4))
    if violation == "no_hyper":
        hyper = None
    return s, step, hyper, flags, keep


def test_validation_fuzz():
    """800 seeded cases, each a well-formed shard with one injected
    violation: the commit reports exactly that violation's code, and so does
    the state digest for the violations that concern it."""
    import numpy as np
    import torch

    if torch.cuda.is_available():
        pytest.skip("host-only test: fake device addresses")
    lib = pk._lib()
    rng = np.random.default_rng(4242)
    names = sorted(_VIOLATIONS)
    for case in range(800):
        violation = names[case % len(names)]
        s, step, hyper, flags, keep = _fuzz_case(rng, violation)
        want, digest_too = _VIOLATIONS[violation]
        got = lib.pact_adamw_commit_ex(ctypes.byref(s), step, ctypes.byref(hyper) if hyper is not None else None,
                                       flags)
        assert got == want, (case, violation, got)
        if digest_too:
            assert lib.pact_shard_digest(ctypes.byref(s)) == want, (case, violation)
        del keep


# ---------------------------------------------------------------------------
# the placement rule (pure host arithmetic)
# ---------------------------------------------------------------------------
MIB2 = 2 << 20


@pytest.mark.parametrize("numel", [0, 1, 1000, 1 << 20, 10_000_001, 76_000_000, 453_001_472, 1_812_005_888,
                                   7_248_023_552])
def test_arena_plan_places_every_array_apart_and_in_the_pool(numel):
    pool, spacing, off = pk.arena_plan(numel)
    f32, b16 = numel * 4, numel * 2
    assert spacing % MIB2 == 0 and all(o % MIB2 == 0 for o in off)
    assert off == [k * spacing for k in range(5)]
    assert spacing >= f32 and off[4] + b16 <= pool
    total = 4 * ((f32 + MIB2 - 1) // MIB2 * MIB2) + (b16 + MIB2 - 1) // MIB2 * MIB2
    if total > pk.PACT_ARENA_PACK_BELOW:
        # the measured rule: arrays some tens of GB apart
        assert spacing == max(pk.PACT_ARENA_SPACING, (f32 + MIB2 - 1) // MIB2 * MIB2)
    else:
        # small enough to stay in the on-chip cache: back to back
        assert pool == total
    assert pool < 288 * 10 ** 9  # fits one MI355X


def test_arena_plan_explicit_spacing_and_errors():
    pool, spacing, off = pk.arena_plan(1000, 3 << 20)
    assert spacing == 4 << 20 and off[1] == 4 << 20
    pool, spacing, off = pk.arena_plan(10 << 20, 1)  # never below one array
    assert spacing == 40 << 20
    lib = pk._lib()
    assert lib.pact_arena_plan(10, 0, None) == pk.PACT_EINVAL
    out = pk._CArenaLayout()
    assert lib.pact_arena_plan(1 << 56, 0, ctypes.byref(out)) == pk.PACT_ERANGE
    assert lib.pact_arena_plan(10, 1 << 59, ctypes.byref(out)) == pk.PACT_ERANGE
