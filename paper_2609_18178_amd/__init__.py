"""paper_2609_18178_amd -- MI355X (gfx950) sharded AdamW commit and state digest.

A thin ctypes binding over ``libpactshard.so`` (C ABI in ``include/pactshard.h``).
Each call marshals torch tensors into a ``pact_shard`` and enqueues the
library's kernels on torch's current HIP stream; every step of the commit and
of the digest runs in those kernels.  torch supplies device memory and
streams only.  There is no fallback: if the library is missing or the tensors
are not on a GPU, the call raises.

The state these calls act on is a rank's preserved training state: its shard
of the weights W, the AdamW moments M and V and the step counter
(Sec. III-A, eq. 2).  ``adamw_commit`` applies the update after which that
state counts as committed (Sec. I; Sec. III-A, action L1); ``shard_digest``
names it in 64 bits for the bitwise cross-rank state checks of Sec. IV-G.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass
from typing import Optional, Sequence, Tuple

import torch

__all__ = [
    "Hyper", "Shard", "ShardBf16", "ShardArena", "PactError", "adamw_commit", "adamw_commit_static",
    "adamw_commit_bf16", "grad_guard",
    "shard_digest", "shard_digest_bf16", "bf16_digest", "stream_probe",
    "digest_slots", "to_u64", "library_path", "arena_plan",
]

_HERE = os.path.dirname(os.path.abspath(__file__))
library_path = os.path.join(_HERE, "libpactshard.so")

MASK64 = (1 << 64) - 1

PACT_OK, PACT_EINVAL, PACT_EALIGN, PACT_EOVERLAP, PACT_ERANGE, PACT_EHIP, PACT_ESCRATCH = 0, -1, -2, -3, -4, -5, -6
PACT_STATIC_MAX_SEGMENTS = 512


class PactError(RuntimeError):
    def __init__(self, code: int, what: str):
        self.code = code
        super().__init__(f"{what}: {_strerror(code)} (code {code}"
                         + (f", hip error {_lib().pact_last_hip_error()}" if code == PACT_EHIP else "") + ")")


class _CHyper(ctypes.Structure):
    _fields_ = [(n, ctypes.c_float) for n in ("lr", "beta1", "beta2", "eps", "weight_decay")]


class _CSegment(ctypes.Structure):
    _fields_ = [("offset", ctypes.c_uint64), ("length", ctypes.c_uint64),
                ("hyper_index", ctypes.c_uint32), ("reserved", ctypes.c_uint32)]


class _CShard(ctypes.Structure):
    _fields_ = [
        ("param", ctypes.c_void_p), ("grad", ctypes.c_void_p), ("exp_avg", ctypes.c_void_p),
        ("exp_avg_sq", ctypes.c_void_p), ("param_bf16", ctypes.c_void_p),
        ("numel", ctypes.c_uint64), ("global_offset", ctypes.c_uint64),
        ("segs", ctypes.POINTER(_CSegment)), ("num_segs", ctypes.c_uint32), ("num_hypers", ctypes.c_uint32),
        ("hypers", ctypes.POINTER(_CHyper)), ("digest_dev", ctypes.c_void_p),
        ("workspace", ctypes.c_void_p), ("workspace_bytes", ctypes.c_uint64), ("stream", ctypes.c_void_p),
    ]


class _CShardBf16(ctypes.Structure):
    _fields_ = [
        ("param", ctypes.c_void_p), ("grad", ctypes.c_void_p), ("exp_avg", ctypes.c_void_p),
        ("exp_avg_sq", ctypes.c_void_p),
        ("numel", ctypes.c_uint64), ("global_offset", ctypes.c_uint64),
        ("segs", ctypes.POINTER(_CSegment)), ("num_segs", ctypes.c_uint32), ("num_hypers", ctypes.c_uint32),
        ("hypers", ctypes.POINTER(_CHyper)), ("digest_dev", ctypes.c_void_p),
        ("workspace", ctypes.c_void_p), ("workspace_bytes", ctypes.c_uint64), ("stream", ctypes.c_void_p),
    ]


class _CArenaLayout(ctypes.Structure):
    _fields_ = [("pool_bytes", ctypes.c_uint64), ("spacing", ctypes.c_uint64), ("offset", ctypes.c_uint64 * 5)]


_LIB = None


def _lib():
    global _LIB
    if _LIB is None:
        if not os.path.exists(library_path):
            raise RuntimeError(
                f"libpactshard.so not built at {library_path}: run `make` (or __graft_entry__.build()). "
                "There is no fallback implementation."
            )
        lib = ctypes.CDLL(library_path)
        P = ctypes.POINTER(_CShard)
        lib.pact_adamw_commit.argtypes = [P, ctypes.c_uint64, ctypes.POINTER(_CHyper)]
        lib.pact_adamw_commit.restype = ctypes.c_int
        lib.pact_adamw_commit_ex.argtypes = [P, ctypes.c_uint64, ctypes.POINTER(_CHyper), ctypes.c_uint32]
        lib.pact_adamw_commit_ex.restype = ctypes.c_int
        lib.pact_adamw_commit_static.argtypes = [P, ctypes.c_uint64, ctypes.POINTER(_CHyper), ctypes.c_uint32]
        lib.pact_adamw_commit_static.restype = ctypes.c_int
        lib.pact_grad_guard.argtypes = [P, ctypes.c_void_p]
        lib.pact_grad_guard.restype = ctypes.c_int
        PB = ctypes.POINTER(_CShardBf16)
        lib.pact_adamw_commit_bf16.argtypes = [PB, ctypes.c_uint64, ctypes.POINTER(_CHyper)]
        lib.pact_adamw_commit_bf16.restype = ctypes.c_int
        lib.pact_shard_digest_bf16.argtypes = [PB]
        lib.pact_shard_digest_bf16.restype = ctypes.c_int
        lib.pact_digest_slots_bf16.argtypes = [PB]
        lib.pact_digest_slots_bf16.restype = ctypes.c_int64
        lib.pact_workspace_bytes_bf16.argtypes = [PB]
        lib.pact_workspace_bytes_bf16.restype = ctypes.c_int64
        lib.pact_shard_digest.argtypes = [P]
        lib.pact_shard_digest.restype = ctypes.c_int
        lib.pact_bf16_digest.argtypes = [P, ctypes.c_void_p]
        lib.pact_bf16_digest.restype = ctypes.c_int
        lib.pact_digest_slots.argtypes = [P]
        lib.pact_digest_slots.restype = ctypes.c_int64
        lib.pact_workspace_bytes.argtypes = [P]
        lib.pact_workspace_bytes.restype = ctypes.c_int64
        lib.pact_arena_plan.argtypes = [ctypes.c_uint64, ctypes.c_uint64, ctypes.POINTER(_CArenaLayout)]
        lib.pact_arena_plan.restype = ctypes.c_int
        lib.pact_stream_probe.argtypes = [ctypes.c_void_p] * 8 + [ctypes.c_uint64, ctypes.c_void_p]
        lib.pact_stream_probe.restype = ctypes.c_int
        lib.pact_stream_probe_grid.argtypes = [ctypes.c_void_p] * 8 + [ctypes.c_uint64, ctypes.c_uint32,
                                                                       ctypes.c_void_p]
        lib.pact_stream_probe_grid.restype = ctypes.c_int
        lib.pact_strerror.argtypes = [ctypes.c_int]
        lib.pact_strerror.restype = ctypes.c_char_p
        lib.pact_last_hip_error.argtypes = []
        lib.pact_last_hip_error.restype = ctypes.c_int
        lib.pact_version.argtypes = []
        lib.pact_version.restype = ctypes.c_int
        _LIB = lib
    return _LIB


def _strerror(code: int) -> str:
    return _lib().pact_strerror(code).decode()


@dataclass(frozen=True)
class Hyper:
    """AdamW hyperparameters (rounded to binary32 by the library's ABI)."""

    lr: float = 3e-4
    beta1: float = 0.9
    beta2: float = 0.95
    eps: float = 1e-8
    weight_decay: float = 0.1

    def _c(self) -> _CHyper:
        return _CHyper(self.lr, self.beta1, self.beta2, self.eps, self.weight_decay)


def _dev_tensor(t: Optional[torch.Tensor], dtype, name: str, n: int, device: Optional[torch.device] = None):
    if t is None:
        return None
    if not isinstance(t, torch.Tensor) or t.dtype not in dtype:
        raise TypeError(f"{name} must be a torch tensor of {dtype}")
    if t.device.type != "cuda":
        raise TypeError(f"{name} must live on a GPU (got {t.device}); there is no CPU path")
    if device is not None and t.device != device:
        raise ValueError(f"{name} is on {t.device} but param is on {device}: one shard lives on one GPU")
    if not t.is_contiguous() or t.numel() != n:
        raise ValueError(f"{name} must be contiguous with {n} elements")
    return t


class Shard:
    """One rank's flat shard: fp32 param/grad/exp_avg/exp_avg_sq, a bf16 copy,
    and the device slots the digests land in.

    ``segments``: optional [(offset, length, hyper_index)] in shard elements
    with ``hypers`` the per-segment table; without it the shard is one segment.
    ``use_workspace``: allocate the digest workspace (faster on large shards;
    without it the library funnels its partial sums into the result slots).
    """

    def __init__(self, param: torch.Tensor, grad: Optional[torch.Tensor], exp_avg: torch.Tensor,
                 exp_avg_sq: torch.Tensor, param_bf16: Optional[torch.Tensor], global_offset: int = 0,
                 segments: Optional[Sequence[Tuple[int, int, int]]] = None,
                 hypers: Optional[Sequence[Hyper]] = None, use_workspace: bool = True):
        n = param.numel()
        f32 = (torch.float32,)
        self.param = _dev_tensor(param, f32, "param", n)
        self.grad = _dev_tensor(grad, f32, "grad", n, param.device)
        self.exp_avg = _dev_tensor(exp_avg, f32, "exp_avg", n, param.device)
        self.exp_avg_sq = _dev_tensor(exp_avg_sq, f32, "exp_avg_sq", n, param.device)
        self.param_bf16 = _dev_tensor(param_bf16, (torch.bfloat16, torch.int16), "param_bf16", n, param.device)
        self.numel = n
        self.global_offset = int(global_offset)
        self.device = param.device
        self.segments = None if segments is None else [tuple(int(x) for x in s) for s in segments]
        self.hypers = None if hypers is None else list(hypers)
        if self.segments is not None and not self.hypers:
            raise ValueError("a segment table needs a hyper table")
        self.slots = 1 if self.segments is None else len(self.segments) + 1
        self.digest = torch.zeros(self.slots, dtype=torch.int64, device=self.device)
        # the C segment and hyper tables are built once and kept alive here
        if self.segments is not None:
            self._csegs = (_CSegment * len(self.segments))(*[_CSegment(o, l, h, 0) for o, l, h in self.segments])
            self._chypers = (_CHyper * len(self.hypers))(*[h._c() for h in self.hypers])
        else:
            self._csegs = None
            self._chypers = None
        # digest workspace: lets the partial sums spread over several addresses.
        # Allocated zero-filled; every successful call leaves it so, which lets
        # commits skip clearing it (workspace_clean stays true until a launch
        # fails).
        self.workspace = None
        self.workspace_clean = False
        if use_workspace:
            nbytes = int(_lib().pact_workspace_bytes(ctypes.byref(self._c())))
            self.workspace = torch.zeros(nbytes, dtype=torch.uint8, device=self.device)
            self.workspace_clean = True

    def _c(self, digest_out: Optional[torch.Tensor] = None, workspace: bool = True) -> _CShard:
        def ptr(t):
            return None if t is None else t.data_ptr()

        s = _CShard()
        s.param, s.grad = ptr(self.param), ptr(self.grad)
        s.exp_avg, s.exp_avg_sq, s.param_bf16 = ptr(self.exp_avg), ptr(self.exp_avg_sq), ptr(self.param_bf16)
        s.numel, s.global_offset = self.numel, self.global_offset
        if self._csegs is not None:
            s.segs = ctypes.cast(self._csegs, ctypes.POINTER(_CSegment))
            s.num_segs = len(self.segments)
            s.hypers = ctypes.cast(self._chypers, ctypes.POINTER(_CHyper))
            s.num_hypers = len(self.hypers)
        s.digest_dev = (digest_out if digest_out is not None else self.digest).data_ptr()
        ws = getattr(self, "workspace", None) if workspace else None
        if ws is not None:
            s.workspace, s.workspace_bytes = ws.data_ptr(), ws.numel()
        s.stream = torch.cuda.current_stream(self.device).cuda_stream
        return s


class ShardBf16:
    """One rank's flat shard held in BF16 (the paper's precision for weights
    and moments): param, grad, exp_avg, exp_avg_sq as int16/bfloat16 tensors
    of bf16 bit patterns, and the digest slots.  Segments as for Shard."""

    def __init__(self, param: torch.Tensor, grad: Optional[torch.Tensor], exp_avg: torch.Tensor,
                 exp_avg_sq: torch.Tensor, global_offset: int = 0,
                 segments: Optional[Sequence[Tuple[int, int, int]]] = None,
                 hypers: Optional[Sequence[Hyper]] = None, use_workspace: bool = True):
        n = param.numel()
        b16 = (torch.bfloat16, torch.int16)
        self.param = _dev_tensor(param, b16, "param", n)
        self.grad = _dev_tensor(grad, b16, "grad", n, param.device)
        self.exp_avg = _dev_tensor(exp_avg, b16, "exp_avg", n, param.device)
        self.exp_avg_sq = _dev_tensor(exp_avg_sq, b16, "exp_avg_sq", n, param.device)
        self.numel = n
        self.global_offset = int(global_offset)
        self.device = param.device
        self.segments = None if segments is None else [tuple(int(x) for x in s) for s in segments]
        self.hypers = None if hypers is None else list(hypers)
        if self.segments is not None and not self.hypers:
            raise ValueError("a segment table needs a hyper table")
        self.slots = 1 if self.segments is None else len(self.segments) + 1
        self.digest = torch.zeros(self.slots, dtype=torch.int64, device=self.device)
        if self.segments is not None:
            self._csegs = (_CSegment * len(self.segments))(*[_CSegment(o, l, h, 0) for o, l, h in self.segments])
            self._chypers = (_CHyper * len(self.hypers))(*[h._c() for h in self.hypers])
        else:
            self._csegs = None
            self._chypers = None
        self.workspace = None
        if use_workspace:
            nbytes = int(_lib().pact_workspace_bytes_bf16(ctypes.byref(self._c())))
            self.workspace = torch.zeros(nbytes, dtype=torch.uint8, device=self.device)

    def _c(self) -> _CShardBf16:
        def ptr(t):
            return None if t is None else t.data_ptr()

        s = _CShardBf16()
        s.param, s.grad, s.exp_avg, s.exp_avg_sq = (ptr(self.param), ptr(self.grad), ptr(self.exp_avg),
                                                     ptr(self.exp_avg_sq))
        s.numel, s.global_offset = self.numel, self.global_offset
        if self._csegs is not None:
            s.segs = ctypes.cast(self._csegs, ctypes.POINTER(_CSegment))
            s.num_segs = len(self.segments)
            s.hypers = ctypes.cast(self._chypers, ctypes.POINTER(_CHyper))
            s.num_hypers = len(self.hypers)
        s.digest_dev = self.digest.data_ptr()
        ws = getattr(self, "workspace", None)
        if ws is not None:
            s.workspace, s.workspace_bytes = ws.data_ptr(), ws.numel()
        s.stream = torch.cuda.current_stream(self.device).cuda_stream
        return s


# Default distance between the arrays of a ShardArena (the library's
# PACT_ARENA_SPACING), and the size below which the arrays are packed.
ARENA_SPACING = PACT_ARENA_SPACING = 44 << 30
ARENA_PACK_BELOW = PACT_ARENA_PACK_BELOW = 512 << 20


def arena_plan(numel: int, spacing: int = 0):
    """The library's placement rule (``pact_arena_plan``): (pool bytes,
    spacing, byte offsets of param, grad, exp_avg, exp_avg_sq, bf16)."""
    out = _CArenaLayout()
    _call("pact_arena_plan", _lib().pact_arena_plan(int(numel), int(spacing), ctypes.byref(out)))
    return int(out.pool_bytes), int(out.spacing), [int(x) for x in out.offset]


class ShardArena:
    """Device memory for one shard's five arrays, placed by the library's
    rule (``pact_arena_plan``): each array in its own region of HBM.

    On MI355X the commit's eight concurrent streams (reads of p, g, m, v;
    writes of p', m', v' and the bf16 copy) move about 5.6 TB/s when all five
    arrays sit within a few gigabytes of each other, and about 6.4-6.5 TB/s
    when they are spread over four or five regions some tens of gigabytes
    apart (the same bytes, the same kernel; measured with the 30 B/element
    stream probe and with the commit itself).  The arena takes one device
    pool and puts fp32 array k at byte offset k * spacing and the bf16 copy
    at 4 * spacing; the space between the arrays stays usable through
    take().

    spacing: bytes between array starts; 0 (default) takes the library's
    rule: 44 GiB when the five arrays exceed 512 MiB, else back to back.
    Among even spacings of 24-60 GiB, 44, 56, 58 and 60 GiB measured about 1%
    faster than 36-42, 48 and 52 GiB on two MI355X GPUs; 44 GiB is the
    smallest of the fast ones.
    """

    def __init__(self, numel: int, device=None, spacing: Optional[int] = None):
        device = torch.device(device) if device is not None else torch.device("cuda", torch.cuda.current_device())
        if device.type != "cuda":
            raise TypeError("the arena lives on a GPU")
        pool_bytes, self.spacing, offs = arena_plan(numel, spacing or 0)
        self.numel = numel
        self.device = device
        self.pool = torch.empty(pool_bytes, dtype=torch.uint8, device=device)
        views = [self.pool[offs[k]: offs[k] + numel * 4].view(torch.float32) for k in range(4)]
        self.param, self.grad, self.exp_avg, self.exp_avg_sq = views
        self.param_bf16 = self.pool[offs[4]: offs[4] + numel * 2].view(torch.int16)
        # free gaps after each fp32 array: [start, end) in pool bytes
        self._gaps = [[offs[k] + numel * 4, offs[k + 1]] for k in range(4)]

    def take(self, nbytes: int, dtype=torch.uint8, region: Optional[int] = None) -> torch.Tensor:
        """A tensor carved from the space between the arrays (first fit, or
        the gap after array ``region`` in 0..3; 256-byte aligned); raises if
        no gap is large enough."""
        esize = torch.empty((), dtype=dtype).element_size()
        gaps = self._gaps if region is None else [self._gaps[region]]
        for gap in gaps:
            start = (gap[0] + 255) // 256 * 256
            if start + nbytes <= gap[1]:
                gap[0] = start + nbytes
                return self.pool[start:start + nbytes].view(dtype)[: nbytes // esize]
        raise MemoryError(f"no gap of {nbytes} bytes left in the arena")

    def shard(self, global_offset: int = 0, segments=None, hypers=None, use_workspace: bool = True) -> "Shard":
        return Shard(self.param, self.grad, self.exp_avg, self.exp_avg_sq, self.param_bf16, global_offset,
                     segments=segments, hypers=hypers, use_workspace=use_workspace)


def _call(what: str, rc: int) -> None:
    if rc != PACT_OK:
        raise PactError(rc, what)


def digest_slots(shard: Shard) -> int:
    return int(_lib().pact_digest_slots(ctypes.byref(shard._c())))


PACT_COMMIT_ZERO_GRAD = 1
PACT_COMMIT_WORKSPACE_CLEAN = 2


def _note_workspace(shard, rc: int) -> None:
    """After a failed launch the workspace may hold partial sums: stop
    vouching that it is clear (the next commit clears it, and the call after
    that may skip the clearing again)."""
    if rc == PACT_EHIP:
        shard.workspace_clean = False
    elif rc == PACT_OK and getattr(shard, "workspace", None) is not None:
        shard.workspace_clean = True


def adamw_commit(shard: Shard, step: int, hyper: Optional[Hyper] = None, zero_grad: bool = False) -> torch.Tensor:
    """Commit one AdamW step on the shard (in place) and digest the result;
    with ``zero_grad`` the same pass also writes +0.0 into the gradient.

    Returns the device tensor of digest slots (int64 holding uint64 bits); it
    holds the values once the current stream reaches this point.
    """
    if shard.segments is None and hyper is None:
        hyper = Hyper()
    ch = hyper._c() if hyper is not None else None
    flags = PACT_COMMIT_ZERO_GRAD if zero_grad else 0
    if shard.workspace is not None and shard.workspace_clean:
        flags |= PACT_COMMIT_WORKSPACE_CLEAN
    with torch.cuda.device(shard.device):
        rc = _lib().pact_adamw_commit_ex(ctypes.byref(shard._c()), int(step),
                                         ctypes.byref(ch) if ch is not None else None, flags)
    _note_workspace(shard, rc)
    _call("pact_adamw_commit_ex", rc)
    return shard.digest


def adamw_commit_static(shard: Shard, step: int, hyper: Optional[Hyper] = None,
                        zero_grad: bool = False) -> torch.Tensor:
    """``adamw_commit`` through the entry point that allocates nothing: the
    digest partial sums go to the library's static device scratch (at most
    ``PACT_STATIC_MAX_SEGMENTS`` segments) instead of the shard's workspace.
    Calls on one GPU share that scratch, so they must not overlap in time."""
    if shard.segments is None and hyper is None:
        hyper = Hyper()
    ch = hyper._c() if hyper is not None else None
    flags = PACT_COMMIT_ZERO_GRAD if zero_grad else 0
    with torch.cuda.device(shard.device):
        rc = _lib().pact_adamw_commit_static(ctypes.byref(shard._c(workspace=False)), int(step),
                                             ctypes.byref(ch) if ch is not None else None, flags)
    _call("pact_adamw_commit_static", rc)
    return shard.digest


def adamw_commit_bf16(shard: ShardBf16, step: int, hyper: Optional[Hyper] = None) -> torch.Tensor:
    """Commit one AdamW step on BF16 state (in place) and digest the result."""
    if shard.segments is None and hyper is None:
        hyper = Hyper()
    ch = hyper._c() if hyper is not None else None
    with torch.cuda.device(shard.device):
        rc = _lib().pact_adamw_commit_bf16(ctypes.byref(shard._c()), int(step),
                                           ctypes.byref(ch) if ch is not None else None)
    _call("pact_adamw_commit_bf16", rc)
    return shard.digest


def shard_digest_bf16(shard: ShardBf16) -> torch.Tensor:
    """Digest of the current BF16 (param, exp_avg, exp_avg_sq)."""
    with torch.cuda.device(shard.device):
        rc = _lib().pact_shard_digest_bf16(ctypes.byref(shard._c()))
    _call("pact_shard_digest_bf16", rc)
    return shard.digest


def _result_slots(shard, out: Optional[torch.Tensor]) -> torch.Tensor:
    """``out`` checked as a destination for the shard's result slots (int64
    device tensor on the shard's GPU, contiguous, at least ``shard.slots``
    long), or a fresh zeroed one."""
    if out is None:
        return torch.zeros(shard.slots, dtype=torch.int64, device=shard.device)
    if not isinstance(out, torch.Tensor) or out.dtype != torch.int64:
        raise TypeError("out must be an int64 torch tensor")
    if out.device != shard.device:
        raise ValueError(f"out is on {out.device}, the shard on {shard.device}")
    if not out.is_contiguous() or out.numel() < shard.slots:
        raise ValueError(f"out must be contiguous with at least {shard.slots} elements")
    return out


def grad_guard(shard: Shard, out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Count the gradient elements that are not +0.0 (per segment and total)."""
    out = _result_slots(shard, out)
    with torch.cuda.device(shard.device):
        rc = _lib().pact_grad_guard(ctypes.byref(shard._c()), out.data_ptr())
    _note_workspace(shard, rc)
    _call("pact_grad_guard", rc)
    return out


def shard_digest(shard: Shard) -> torch.Tensor:
    """Digest of the shard's current (param, exp_avg, exp_avg_sq)."""
    with torch.cuda.device(shard.device):
        rc = _lib().pact_shard_digest(ctypes.byref(shard._c()))
    _note_workspace(shard, rc)
    _call("pact_shard_digest", rc)
    return shard.digest


def bf16_digest(shard: Shard, out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Digest (tag 3) of the bf16 copy, into ``out`` (allocated if None)."""
    out = _result_slots(shard, out)
    with torch.cuda.device(shard.device):
        rc = _lib().pact_bf16_digest(ctypes.byref(shard._c()), out.data_ptr())
    _note_workspace(shard, rc)
    _call("pact_bf16_digest", rc)
    return out


def stream_probe(i0, i1, i2, i3, o0, o2, o3, oh, workgroups: int = 0) -> None:
    """30-byte/element streaming probe (measurement support): reads the four
    fp32 tensors i0..i3, writes o0, o2, o3 (fp32) and oh (16-bit); all on one
    GPU, contiguous, with the same element count.  Outputs may be the inputs
    (in place).  ``workgroups`` > 0: a persistent grid of that many
    workgroups striding over the tiles instead of one workgroup per tile."""
    if not isinstance(i0, torch.Tensor):
        raise TypeError("i0 must be a torch tensor")
    n = i0.numel()
    for name, t in (("i0", i0), ("i1", i1), ("i2", i2), ("i3", i3), ("o0", o0), ("o2", o2), ("o3", o3)):
        _dev_tensor(t, (torch.float32,), name, n, i0.device)
    _dev_tensor(oh, (torch.int16, torch.bfloat16), "oh", n, i0.device)
    with torch.cuda.device(i0.device):
        rc = _lib().pact_stream_probe_grid(i0.data_ptr(), i1.data_ptr(), i2.data_ptr(), i3.data_ptr(),
                                           o0.data_ptr(), o2.data_ptr(), o3.data_ptr(), oh.data_ptr(), n,
                                           int(workgroups), torch.cuda.current_stream(i0.device).cuda_stream)
    _call("pact_stream_probe_grid", rc)


def to_u64(t: torch.Tensor):
    """Digest slots as Python ints (uint64); synchronizes with the device."""
    return [int(x) & MASK64 for x in t.cpu().tolist()]
