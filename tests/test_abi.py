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
    texts = {code: pk._strerror(code) for code in (0, -1, -2, -3, -4, -5)}
    assert len(set(texts.values())) == 6
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
               "pact_shard_bf16": pk._CShardBf16}
    for name, cls in mirrors.items():
        assert ctypes.sizeof(cls) == c[name]["sizeof"], name
        py_fields = {f[0]: getattr(cls, f[0]).offset for f in cls._fields_}
        c_fields = c[name]["fields"]
        # the binding names fields as the header does
        assert py_fields == c_fields, (name, py_fields, c_fields)
    for code, value in c["codes"].items():
        assert getattr(pk, code) == value, code
