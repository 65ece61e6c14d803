"""Oracle: the plain CPU definition of the sharded AdamW commit and state digest.

TEST INFRASTRUCTURE ONLY.  The GPU library never imports, links or calls this
package; only the test suite, the smoke check and the CPU-baseline leg of the
benchmark do.  The arithmetic lives in ``oracle.c`` (single-threaded C,
``-ffp-contract=off``, IEEE binary32); this module only marshals numpy arrays
into it and walks a segment table one segment at a time.

Passages followed: the preserved state W, M, V and the step counter
(Sec. III-A, eq. 2), the committed optimizer boundary (Sec. I; Sec. III-A,
action L1), BF16 working precision (Sec. IV-A) and the bitwise state checks
(abstract; Sec. IV-G).  The paper gives no formula for the update; the reading
fixed for it is stated in ``oracle.h``.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass
from typing import Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
# PACT_ORACLE_LIB lets the mutation tests load a deliberately broken build.
_LIB_PATH = os.environ.get("PACT_ORACLE_LIB") or os.path.join(_HERE, "liboracle.so")

MASK64 = (1 << 64) - 1


class _Hyper(ctypes.Structure):
    _fields_ = [
        ("lr", ctypes.c_float),
        ("beta1", ctypes.c_float),
        ("beta2", ctypes.c_float),
        ("eps", ctypes.c_float),
        ("weight_decay", ctypes.c_float),
    ]


class _Scalars(ctypes.Structure):
    _fields_ = [
        ("beta1", ctypes.c_float),
        ("beta2", ctypes.c_float),
        ("eps", ctypes.c_float),
        ("decay", ctypes.c_float),
        ("omb1", ctypes.c_float),
        ("omb2", ctypes.c_float),
        ("step_size", ctypes.c_float),
        ("rs_bc2", ctypes.c_float),
    ]


@dataclass(frozen=True)
class Hyper:
    """AdamW hyperparameters; each is rounded to binary32 before use."""

    lr: float = 3e-4
    beta1: float = 0.9
    beta2: float = 0.95
    eps: float = 1e-8
    weight_decay: float = 0.1


_lib = None


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            raise RuntimeError(
                f"oracle library missing at {_LIB_PATH}; run __graft_entry__.build() (or make)"
            )
        lib = ctypes.CDLL(_LIB_PATH)
        u64, u32p, u16p, f32p = (
            ctypes.c_uint64,
            ctypes.POINTER(ctypes.c_uint32),
            ctypes.POINTER(ctypes.c_uint16),
            ctypes.POINTER(ctypes.c_float),
        )
        lib.oracle_splitmix64.argtypes = [u64]
        lib.oracle_splitmix64.restype = u64
        lib.oracle_bf16_rne.argtypes = [ctypes.c_uint32]
        lib.oracle_bf16_rne.restype = ctypes.c_uint16
        lib.oracle_bf16_rne_array.argtypes = [u32p, u16p, u64]
        lib.oracle_bf16_rne_array.restype = None
        lib.oracle_make_scalars.argtypes = [ctypes.POINTER(_Hyper), u64, ctypes.POINTER(_Scalars)]
        lib.oracle_make_scalars.restype = None
        lib.oracle_adamw_commit.argtypes = [f32p, f32p, f32p, f32p, u16p, u64, ctypes.POINTER(_Scalars)]
        lib.oracle_adamw_commit.restype = None
        lib.oracle_state_digest.argtypes = [f32p, f32p, f32p, u64, u64]
        lib.oracle_state_digest.restype = u64
        lib.oracle_bf16_digest.argtypes = [u16p, u64, u64]
        lib.oracle_bf16_digest.restype = u64
        lib.oracle_commit_and_digest.argtypes = [
            f32p, f32p, f32p, f32p, u16p, u64, u64, ctypes.POINTER(_Hyper), u64,
        ]
        lib.oracle_commit_and_digest.restype = u64
        lib.oracle_adamw_commit_bf16.argtypes = [u16p, u16p, u16p, u16p, u64, ctypes.POINTER(_Scalars)]
        lib.oracle_adamw_commit_bf16.restype = None
        lib.oracle_state_digest_bf16.argtypes = [u16p, u16p, u16p, u64, u64]
        lib.oracle_state_digest_bf16.restype = u64
        lib.oracle_zero_grad.argtypes = [f32p, u64]
        lib.oracle_zero_grad.restype = None
        lib.oracle_count_outstanding.argtypes = [f32p, u64]
        lib.oracle_count_outstanding.restype = u64
        _lib = lib
    return _lib


def _ptr(a: np.ndarray, ctype):
    return a.ctypes.data_as(ctypes.POINTER(ctype))


def _check(a: np.ndarray, dtype, name: str, n: int | None = None) -> None:
    if not isinstance(a, np.ndarray) or a.dtype != dtype or not a.flags["C_CONTIGUOUS"]:
        raise TypeError(f"{name} must be a C-contiguous numpy array of {np.dtype(dtype)}")
    if n is not None and a.size != n:
        raise ValueError(f"{name} has {a.size} elements, expected {n}")


def _hyper(h: Hyper) -> _Hyper:
    return _Hyper(h.lr, h.beta1, h.beta2, h.eps, h.weight_decay)


# --------------------------------------------------------------------------
# elementary pieces
# --------------------------------------------------------------------------

def splitmix64(x: int) -> int:
    """splitmix64 output for generator state ``x`` (mix of ``x`` + gamma)."""
    return int(_load().oracle_splitmix64(x & MASK64))


def bf16_rne_bits(bits: np.ndarray) -> np.ndarray:
    """RNE binary32 -> bfloat16 over an array of uint32 bit patterns."""
    bits = np.ascontiguousarray(bits, dtype=np.uint32)
    out = np.empty(bits.shape, dtype=np.uint16)
    _load().oracle_bf16_rne_array(_ptr(bits, ctypes.c_uint32), _ptr(out, ctypes.c_uint16), bits.size)
    return out


def make_scalars(h: Hyper, step: int) -> dict:
    """The eight binary32 scalars of one step, as Python floats (exact values)."""
    if step < 1:
        raise ValueError("step counts from 1")
    sc = _Scalars()
    _load().oracle_make_scalars(ctypes.byref(_hyper(h)), step, ctypes.byref(sc))
    return {name: getattr(sc, name) for name, _ in _Scalars._fields_}


# --------------------------------------------------------------------------
# the path
# --------------------------------------------------------------------------

def adamw_commit(p, g, m, v, bf16, h: Hyper, step: int) -> None:
    """One commit in place on numpy float32 p, m, v; writes uint16 bf16."""
    n = p.size
    for a, nm in ((p, "p"), (g, "g"), (m, "m"), (v, "v")):
        _check(a, np.float32, nm, n)
    _check(bf16, np.uint16, "bf16", n)
    if step < 1:
        raise ValueError("step counts from 1")
    lib = _load()
    sc = _Scalars()
    lib.oracle_make_scalars(ctypes.byref(_hyper(h)), step, ctypes.byref(sc))
    lib.oracle_adamw_commit(
        _ptr(p, ctypes.c_float), _ptr(g, ctypes.c_float), _ptr(m, ctypes.c_float),
        _ptr(v, ctypes.c_float), _ptr(bf16, ctypes.c_uint16), n, ctypes.byref(sc),
    )


def state_digest(p, m, v, first_index: int) -> int:
    """Digest of (p, m, v) whose element 0 sits at global flat index ``first_index``."""
    n = p.size
    for a, nm in ((p, "p"), (m, "m"), (v, "v")):
        _check(a, np.float32, nm, n)
    return int(
        _load().oracle_state_digest(
            _ptr(p, ctypes.c_float), _ptr(m, ctypes.c_float), _ptr(v, ctypes.c_float), n, first_index,
        )
    )


def bf16_digest(b, first_index: int) -> int:
    _check(b, np.uint16, "bf16")
    return int(_load().oracle_bf16_digest(_ptr(b, ctypes.c_uint16), b.size, first_index))


def commit_and_digest(p, g, m, v, bf16, h: Hyper, step: int, first_index: int) -> int:
    """The whole hot path on one flat segment: commit, then digest of (p', m', v')."""
    n = p.size
    for a, nm in ((p, "p"), (g, "g"), (m, "m"), (v, "v")):
        _check(a, np.float32, nm, n)
    _check(bf16, np.uint16, "bf16", n)
    if step < 1:
        raise ValueError("step counts from 1")
    return int(
        _load().oracle_commit_and_digest(
            _ptr(p, ctypes.c_float), _ptr(g, ctypes.c_float), _ptr(m, ctypes.c_float),
            _ptr(v, ctypes.c_float), _ptr(bf16, ctypes.c_uint16), n, first_index,
            ctypes.byref(_hyper(h)), step,
        )
    )


def adamw_commit_bf16(p, g, m, v, h: Hyper, step: int) -> None:
    """One commit in place on BF16 state (uint16 bit patterns)."""
    n = p.size
    for a, nm in ((p, "p"), (g, "g"), (m, "m"), (v, "v")):
        _check(a, np.uint16, nm, n)
    if step < 1:
        raise ValueError("step counts from 1")
    lib = _load()
    sc = _Scalars()
    lib.oracle_make_scalars(ctypes.byref(_hyper(h)), step, ctypes.byref(sc))
    lib.oracle_adamw_commit_bf16(_ptr(p, ctypes.c_uint16), _ptr(g, ctypes.c_uint16), _ptr(m, ctypes.c_uint16),
                                 _ptr(v, ctypes.c_uint16), n, ctypes.byref(sc))


def state_digest_bf16(p, m, v, first_index: int) -> int:
    n = p.size
    for a, nm in ((p, "p"), (m, "m"), (v, "v")):
        _check(a, np.uint16, nm, n)
    return int(_load().oracle_state_digest_bf16(_ptr(p, ctypes.c_uint16), _ptr(m, ctypes.c_uint16),
                                                _ptr(v, ctypes.c_uint16), n, first_index))


def commit_and_digest_bf16(p, g, m, v, h: Hyper, step: int, first_index: int) -> int:
    adamw_commit_bf16(p, g, m, v, h, step)
    return state_digest_bf16(p, m, v, first_index)


def zero_grad(g) -> None:
    """The gradient at the committed boundary: every element +0.0."""
    _check(g, np.float32, "g")
    _load().oracle_zero_grad(_ptr(g, ctypes.c_float), g.size)


def count_outstanding(g) -> int:
    """Gradient elements whose bit pattern is not all zero."""
    _check(g, np.float32, "g")
    return int(_load().oracle_count_outstanding(_ptr(g, ctypes.c_float), g.size))


def commit_segments(p, g, m, v, bf16, segments: Sequence[tuple[int, int, int]],
                    hypers: Sequence[Hyper], step: int, global_offset: int):
    """Multi-segment commit over one flat shard.

    ``segments`` lists (offset, length, hyper_index) in shard elements.  The
    flat index of shard element i is ``global_offset + i``; elements that no
    segment covers (padding) are neither committed nor digested.  Returns the
    per-segment digests and their sum mod 2^64.
    """
    per = []
    for off, length, hi in segments:
        sl = slice(off, off + length)
        d = commit_and_digest(p[sl], g[sl], m[sl], v[sl], bf16[sl], hypers[hi], step,
                              global_offset + off)
        per.append(d)
    return per, sum(per) & MASK64


def segment_digests(p, m, v, segments: Sequence[tuple[int, int, int]], global_offset: int):
    """Per-segment state digests of the current (p, m, v) and their sum."""
    per = []
    for off, length, _ in segments:
        sl = slice(off, off + length)
        per.append(state_digest(p[sl], m[sl], v[sl], global_offset + off))
    return per, sum(per) & MASK64
