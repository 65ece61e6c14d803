"""Seeded synthetic workloads for the sharded AdamW commit.

Shapes, offsets, value distributions and step numbers of the shards that the
benchmark and the tests run on, and a bit-reproducible host generator for
their contents (``gen.c``: Philox4x32-10 + an Irwin-Hall(8) normal).  This
module holds none of the commit's or digest's arithmetic; the GPU path and the
CPU oracle both read the arrays it draws.

The paper trains full-parameter Mistral-7B (7,248,023,552 parameters) on 16
GPUs in a 4x4 hybrid-sharded layout, and measures checkpoint overheads on a
1,216,448,512-parameter decoder (Sec. II-B, Sec. IV-A).  Neither the weights
nor the training data exist here; the commit's cost depends only on the
element count, layout and value ranges, so synthetic arrays of those shapes
stand in for them.
"""
from __future__ import annotations

import ctypes
import math
import os
from dataclasses import dataclass, field
from typing import List, Optional, Tuple

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "libgen.so")

# array ids in the generator counter
ARRAY_PARAM, ARRAY_GRAD, ARRAY_EXP_AVG, ARRAY_EXP_AVG_SQ = 0, 1, 2, 3

KIND_NORMAL, KIND_ABS_NORMAL, KIND_ZERO = 0, 1, 2

# standard deviation of the centred Irwin-Hall(8) sum of 16-bit uniforms
SUM_SD = math.sqrt(8.0 * (65536.0 * 65536.0 - 1.0) / 12.0)

_lib = None


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            raise RuntimeError(f"generator library missing at {_LIB_PATH}; run make")
        lib = ctypes.CDLL(_LIB_PATH)
        lib.gen_fill.argtypes = [
            ctypes.c_void_p, ctypes.c_uint64, ctypes.c_uint64, ctypes.c_uint64,
            ctypes.c_uint32, ctypes.c_uint64, ctypes.c_int, ctypes.c_float,
        ]
        lib.gen_fill.restype = None
        lib.gen_philox4x32_10.argtypes = [
            ctypes.POINTER(ctypes.c_uint32), ctypes.POINTER(ctypes.c_uint32),
            ctypes.POINTER(ctypes.c_uint32),
        ]
        lib.gen_philox4x32_10.restype = None
        lib.gen_num_threads.argtypes = []
        lib.gen_num_threads.restype = ctypes.c_int
        _lib = lib
    return _lib


def philox4x32_10(ctr, key):
    """One Philox4x32-10 block (exposed for known-answer tests)."""
    c = (ctypes.c_uint32 * 4)(*ctr)
    k = (ctypes.c_uint32 * 2)(*key)
    o = (ctypes.c_uint32 * 4)()
    _load().gen_philox4x32_10(c, k, o)
    return tuple(int(x) for x in o)


def num_threads() -> int:
    return int(_load().gen_num_threads())


@dataclass(frozen=True)
class Dist:
    """Distribution of one array: N(0, sigma), |N(0, sigma)| or all zeros."""

    kind: int
    sigma: float = 0.0

    @property
    def scale(self) -> float:
        return float(np.float32(self.sigma / SUM_SD))


NORMAL = lambda s: Dist(KIND_NORMAL, s)  # noqa: E731
ABS_NORMAL = lambda s: Dist(KIND_ABS_NORMAL, s)  # noqa: E731
ZERO = Dist(KIND_ZERO)


def fill_host(out: np.ndarray, first_index: int, seed: int, array_id: int, step: int, dist: Dist) -> np.ndarray:
    """Fill a float32 numpy array with global indices first_index.. of one array."""
    if out.dtype != np.float32 or not out.flags["C_CONTIGUOUS"]:
        raise TypeError("out must be a C-contiguous float32 array")
    _load().gen_fill(out.ctypes.data, out.size, first_index, seed, array_id, step, dist.kind, dist.scale)
    return out


def draw(n: int, first_index: int, seed: int, array_id: int, step: int, dist: Dist) -> np.ndarray:
    return fill_host(np.empty(n, dtype=np.float32), first_index, seed, array_id, step, dist)


def fill_device(t, first_index: int, seed: int, array_id: int, step: int, dist: Dist,
                chunk: int = 1 << 26) -> None:
    """Fill a float32 torch tensor (any device) in host-generated chunks.

    Each chunk is drawn into pinned host memory and copied; the two staging
    buffers alternate so the copy of one chunk overlaps drawing the next.
    """
    import torch

    n = t.numel()
    flat = t.view(-1)
    if dist.kind == KIND_ZERO:
        flat.zero_()
        return
    if flat.device.type == "cpu":
        fill_host(flat.numpy(), first_index, seed, array_id, step, dist)
        return
    chunk = min(chunk, max(n, 1))
    stage = [torch.empty(chunk, dtype=torch.float32, pin_memory=True) for _ in range(2)]
    done = [None, None]
    stream = torch.cuda.current_stream(flat.device)
    for k, start in enumerate(range(0, n, chunk)):
        cnt = min(chunk, n - start)
        buf = stage[k % 2]
        if done[k % 2] is not None:
            done[k % 2].synchronize()
        fill_host(buf.numpy()[:cnt], first_index + start, seed, array_id, step, dist)
        flat[start:start + cnt].copy_(buf[:cnt], non_blocking=True)
        ev = torch.cuda.Event()
        ev.record(stream)
        done[k % 2] = ev
    torch.cuda.synchronize(flat.device)


# --------------------------------------------------------------------------
# Mistral-7B flat layout (the paper's model: 7,248,023,552 parameters)
# --------------------------------------------------------------------------

MISTRAL_VOCAB = 32768
MISTRAL_HIDDEN = 4096
MISTRAL_LAYERS = 32
MISTRAL_INTERMEDIATE = 14336
MISTRAL_KV_DIM = 1024  # 8 key/value heads x 128
MISTRAL_PARAMS = 7_248_023_552
PAD_ELEMS = 128  # 512 bytes of fp32


def _pad(n: int) -> int:
    return (n + PAD_ELEMS - 1) // PAD_ELEMS * PAD_ELEMS


def mistral_tensors(layers: int = MISTRAL_LAYERS, hidden: int = MISTRAL_HIDDEN,
                    intermediate: int = MISTRAL_INTERMEDIATE, kv_dim: int = MISTRAL_KV_DIM,
                    vocab: int = MISTRAL_VOCAB) -> List[Tuple[str, int, str]]:
    """(name, numel, role) in Hugging Face order; role in {embed, matrix, norm, lm_head}."""
    out = [("model.embed_tokens.weight", vocab * hidden, "embed")]
    for i in range(layers):
        pre = f"model.layers.{i}."
        out += [
            (pre + "self_attn.q_proj.weight", hidden * hidden, "matrix"),
            (pre + "self_attn.k_proj.weight", kv_dim * hidden, "matrix"),
            (pre + "self_attn.v_proj.weight", kv_dim * hidden, "matrix"),
            (pre + "self_attn.o_proj.weight", hidden * hidden, "matrix"),
            (pre + "mlp.gate_proj.weight", intermediate * hidden, "matrix"),
            (pre + "mlp.up_proj.weight", intermediate * hidden, "matrix"),
            (pre + "mlp.down_proj.weight", hidden * intermediate, "matrix"),
            (pre + "input_layernorm.weight", hidden, "norm"),
            (pre + "post_attention_layernorm.weight", hidden, "norm"),
        ]
    out += [("model.norm.weight", hidden, "norm"), ("lm_head.weight", vocab * hidden, "lm_head")]
    return out


def flat_segments(tensors, pad_to: int = PAD_ELEMS):
    """Lay tensors end to end, each padded to ``pad_to`` elements.

    Returns (segments, total) with segments = [(offset, length, role)].
    """
    segs, off = [], 0
    for _, n, role in tensors:
        segs.append((off, n, role))
        off += (n + pad_to - 1) // pad_to * pad_to
    return segs, off


# hyperparameter table of the whole-model layout, indexed by role
ROLE_HYPERS = {
    "matrix": dict(lr=3e-4, beta1=0.9, beta2=0.95, eps=1e-8, weight_decay=0.1),
    "embed": dict(lr=1.5e-4, beta1=0.9, beta2=0.95, eps=1e-8, weight_decay=0.1),
    "lm_head": dict(lr=1.5e-4, beta1=0.9, beta2=0.99, eps=1e-8, weight_decay=0.1),
    "norm": dict(lr=3e-4, beta1=0.9, beta2=0.95, eps=1e-8, weight_decay=0.0),
}
ROLE_ORDER = ("matrix", "embed", "lm_head", "norm")

DEFAULT_HYPER = dict(lr=3e-4, beta1=0.9, beta2=0.95, eps=1e-8, weight_decay=0.1)


# --------------------------------------------------------------------------
# workload configurations
# --------------------------------------------------------------------------

@dataclass(frozen=True)
class Workload:
    name: str
    numel: int            # elements in the shard, padding included
    global_offset: int    # flat index of shard element 0 in the full vector
    first_step: int       # optimizer step of the first commit
    commits: int          # successive commits
    seed: int
    param: Dist
    grad: Dist
    exp_avg: Dist
    exp_avg_sq: Dist
    # multi-segment layout: [(offset, length, hyper_index)] and hyper dicts
    segments: Optional[Tuple[Tuple[int, int, int], ...]] = None
    hypers: Tuple[dict, ...] = field(default_factory=lambda: (DEFAULT_HYPER,))

    def describe(self) -> dict:
        d = dict(workload=self.name, numel=self.numel, global_offset=self.global_offset,
                 first_step=self.first_step, commits=self.commits, seed=self.seed)
        if self.segments is not None:
            d["segments"] = len(self.segments)
        return d


def _warm(name, numel, offset, step, commits, seed, **kw):
    return Workload(name, numel, offset, step, commits, seed,
                    NORMAL(0.02), NORMAL(1e-3), NORMAL(1e-4), ABS_NORMAL(1e-7), **kw)


MISTRAL_SHARD16 = MISTRAL_PARAMS // 16          # 453,001,472
MISTRAL_SHARD4 = MISTRAL_PARAMS // 4            # 1,812,005,888
DECODER_1B_SHARD16 = 76_000_000                 # ~1,216,448,512 / 16


def _whole_model(layers=MISTRAL_LAYERS, hidden=MISTRAL_HIDDEN, intermediate=MISTRAL_INTERMEDIATE,
                 kv_dim=MISTRAL_KV_DIM, vocab=MISTRAL_VOCAB, name="mistral7b_whole", seed=5):
    segs, total = flat_segments(mistral_tensors(layers, hidden, intermediate, kv_dim, vocab))
    table = tuple((off, n, ROLE_ORDER.index(role)) for off, n, role in segs)
    return _warm(name, total, 0, 5, 1, seed, segments=table,
                 hypers=tuple(ROLE_HYPERS[r] for r in ROLE_ORDER))


WORKLOADS = {
    "tiny": Workload("tiny", 1 << 20, 0, 1, 1, 1, NORMAL(0.02), NORMAL(1e-3), ZERO, ZERO),
    "decoder1b_shard16": _warm("decoder1b_shard16", DECODER_1B_SHARD16, 15 * DECODER_1B_SHARD16,
                               100, 10, 2),
    "mistral7b_shard16": _warm("mistral7b_shard16", MISTRAL_SHARD16, 15 * MISTRAL_SHARD16, 5, 1, 3),
    "mistral7b_shard4": _warm("mistral7b_shard4", MISTRAL_SHARD4, 3 * MISTRAL_SHARD4, 18, 10, 4),
    "mistral7b_whole": _whole_model(),
}


def shrunken_mistral(layers=2, hidden=200, intermediate=520, kv_dim=40, vocab=1003, seed=6):
    """Small multi-segment layout with the real tensor roles and odd padded sizes."""
    return _whole_model(layers, hidden, intermediate, kv_dim, vocab, name="mistral_shrunk", seed=seed)


def arrays_host(w: Workload, start: int = 0, count: Optional[int] = None):
    """Host numpy (p, g, m, v) for shard elements [start, start+count) at the first step."""
    if count is None:
        count = w.numel - start
    first = w.global_offset + start
    p = draw(count, first, w.seed, ARRAY_PARAM, 0, w.param)
    g = draw(count, first, w.seed, ARRAY_GRAD, w.first_step, w.grad)
    m = draw(count, first, w.seed, ARRAY_EXP_AVG, 0, w.exp_avg)
    v = draw(count, first, w.seed, ARRAY_EXP_AVG_SQ, 0, w.exp_avg_sq)
    return p, g, m, v


def grad_host(w: Workload, step: int, start: int = 0, count: Optional[int] = None) -> np.ndarray:
    if count is None:
        count = w.numel - start
    return draw(count, w.global_offset + start, w.seed, ARRAY_GRAD, step, w.grad)
