"""In-memory recovery of a sharded training job at a committed optimizer
boundary: the host-side protocol around the commit (Sec. III).

What it models.  A job of W ranks (one process each) in hybrid sharding:
``shards`` shard groups times ``replicas`` replication groups.  Rank r holds
shard ``r % shards`` of the flat state; the ranks holding the same shard form
a replication group (the inter-node group of Sec. II-A) and hold bit-identical
state.  Each update produces a gradient, reduces it over the replication
group, commits AdamW through the rank's engine (the library's fused commit,
which also zeroes the gradient and digests the committed state) and reduces
a metric over the replication group after the commit.

When a replication-group collective fails, the ranks run the six-phase
recovery of Sec. III-C over an out-of-band Gloo control plane that spans all
W ranks (CPU tensors only):

1. observe: the failed collective raises; the failure phase (committed,
   forward, backward) is read from the module states, and the
   qualification envelope (Sec. III-A) maps the observation key to L1
   (preserve in memory) or L2 (fail-stop; restart from a checkpoint);
2. guard and stream sync: the device queue is drained, every module wrapper
   must be IDLE and the gradient guard must count zero outstanding elements;
3. control barrier and frontier agreement: rank 0 broadcasts the committed
   frontier F and the next generation g; every rank must agree exactly.  The
   ranks also agree on the committed state: each rank's digest of its
   current state must equal the digest its last commit produced (a torn or
   altered commit fails here), and replicas of one shard must hold the same
   digest;
4. communicator replacement: the failed replication group is destroyed and
   rebuilt with the same members;
5. reference rebinding: every cached reference to the retired group in the
   rank's module hierarchy is redirected to the new one (the invariant of
   Sec. III-D: exactly the L + 1 references that named it, nothing else);
6. validation and release: an integer all-reduce over the new group must
   return the group size, then a control-plane release barrier.

Safety invariant (Sec. III-C): an exception or a missed deadline in phases
2-6 ends the rank at once with a non-zero status; its peers see the loss on
the control plane (or reach their own deadline) and end too, so the
supervisor restarts the whole cohort from its checkpoint (L2) and no rank
continues alone.  Generations fence stale participants: every repair
advances g, a cohort started by the supervisor gets a control-plane
rendezvous of its own generation, and a rank whose g disagrees is rejected.

Ranks are child processes started by ``Supervisor`` (never an exec of the
supervisor itself); the supervisor makes no GPU call.  The engine that holds
a rank's shard is pluggable: ``ShardEngine`` keeps it on the GPU and runs
every state operation through libpactshard.
"""
from __future__ import annotations

import argparse
import importlib
import json
import os
import subprocess
import sys
import tempfile
import threading
import time
from dataclasses import dataclass, field
from datetime import timedelta
from enum import Enum
from typing import Dict, List, Optional, Tuple

MASK64 = (1 << 64) - 1

# exit statuses of a rank process
EXIT_OK = 0
EXIT_REJECTED = 3   # uncommitted failure: fail-stop rejection, restart from checkpoint (L2)
EXIT_FAILSTOP = 4   # an exception in phases 2-6 (safety invariant)
EXIT_TIMEOUT = 5    # a phase missed its deadline (the rank's own watchdog)
EXIT_FENCED = 6     # disagreement in phase 3: frontier, generation or committed state
EXIT_ERROR = 7      # anything outside the protocol (setup, training)

EXIT_NAMES = {EXIT_OK: "ok", EXIT_REJECTED: "rejected", EXIT_FAILSTOP: "fail-stop", EXIT_TIMEOUT: "timeout",
              EXIT_FENCED: "fenced", EXIT_ERROR: "error"}

PHASES = ("observe", "guard", "agree", "replace", "rebind", "release")


# ---------------------------------------------------------------------------
# state model and qualification contract (Sec. III-A)
# ---------------------------------------------------------------------------

class Phi(str, Enum):
    """Failure phase of an observation."""
    COMMITTED = "committed"
    FORWARD = "forward"
    BACKWARD = "backward"


class Action(int, Enum):
    """Qualified recovery actions: L1 keeps the state in device memory and
    repairs in place; L2 is the fail-stop rejection that hands the job to the
    supervisor's checkpoint restart."""
    L1_PRESERVE = 1
    L2_RESTART = 2


@dataclass(frozen=True)
class ObservationKey:
    """K = <platform, resource profile, failure phase, continuation objective>."""
    platform: str
    resource: str
    phase: Phi
    objective: str


ANY = "*"


class Envelope:
    """Qualified recovery actions by observation key.  Entries may use ``ANY``
    for platform, resource or objective; a key matches the most specific
    entry.  A key no entry qualifies gets L2: in-memory preservation is only
    admitted where it was qualified."""

    def __init__(self, entries: Optional[Dict[Tuple[str, str, str, str], Action]] = None):
        self.entries = dict(entries) if entries is not None else {
            (ANY, ANY, Phi.COMMITTED.value, ANY): Action.L1_PRESERVE,
            (ANY, ANY, Phi.FORWARD.value, ANY): Action.L2_RESTART,
            (ANY, ANY, Phi.BACKWARD.value, ANY): Action.L2_RESTART,
        }

    def action(self, key: ObservationKey) -> Action:
        best, best_score = None, -1
        for (pl, rs, ph, ob), act in self.entries.items():
            if ph != key.phase.value:
                continue
            fields = ((pl, key.platform), (rs, key.resource), (ob, key.objective))
            if any(want != ANY and want != have for want, have in fields):
                continue
            score = sum(want != ANY for want, _ in fields)
            if score > best_score:
                best, best_score = act, score
        return best if best is not None else Action.L2_RESTART


# ---------------------------------------------------------------------------
# break-even model of in-memory recovery (Sec. III-B, eq. (4))
# ---------------------------------------------------------------------------

def saving_per_recovery(age_updates: float, update_seconds: float, repair_seconds: float) -> float:
    """S = A * t_update - T_repair: the replay of A = F - C updates that one
    in-memory recovery avoids, less the repair itself (seconds)."""
    return age_updates * update_seconds - repair_seconds


def net_saving(n_eligible: float, saving: float, n_other: float, reject_cost: float, guard_overhead: float,
               baseline_seconds: float) -> float:
    """Delta T = N_eligible * S - N_other * C - h * T_0 (eq. (4)): the
    cluster time a campaign of baseline length T_0 saves, with N_eligible
    failures at committed boundaries, N_other uncommitted failures that each
    cost C = T_detect + T_reject, and a boundary-guard overhead fraction h."""
    return n_eligible * saving - n_other * reject_cost - guard_overhead * baseline_seconds


def break_even_interval(saving: float, guard_overhead: float) -> float:
    """Training time per eligible failure at which the savings pay for the
    guard exactly (Delta T = 0 with no other failures): S / h seconds."""
    return saving / guard_overhead


class ModState(str, Enum):
    IDLE = "IDLE"
    FORWARD = "FORWARD"
    BACKWARD = "BACKWARD"


# ---------------------------------------------------------------------------
# the module hierarchy and reference rebinding (Sec. II-A, Sec. III-D)
# ---------------------------------------------------------------------------

class ExecMeta:
    """Execution metadata cached by a wrapper (names the world group)."""

    def __init__(self, world):
        self.world_group = world
        self.order = []


class FlatHandle:
    """Flat-parameter handle (names the shard group)."""

    def __init__(self, shard_group):
        self.process_group = shard_group


class Wrapper:
    """A sharded module wrapper: caches the replication group in
    ``_inter_node_pg`` (the reference that must be rebound), the shard group
    in ``process_group`` and in its flat-parameter handle, and the world group
    in its execution metadata (references that must stay)."""

    def __init__(self, name: str, inter, intra, world):
        self.name = name
        self.state = ModState.IDLE
        self._inter_node_pg = inter
        self.process_group = intra
        self._handle = FlatHandle(intra)
        self._exec_order_data = ExecMeta(world)
        self.children: List["Wrapper"] = []


def build_model(layers: int, inter, intra, world) -> Wrapper:
    """A root wrapper over ``layers`` layer wrappers: L + 1 cached references
    to the replication group."""
    root = Wrapper("root", inter, intra, world)
    root.children = [Wrapper(f"layers.{i}", inter, intra, world) for i in range(layers)]
    return root


def wrappers(root: Wrapper) -> List[Wrapper]:
    out, stack = [], [root]
    while stack:
        w = stack.pop()
        out.append(w)
        stack.extend(reversed(w.children))
    return out


class RebindError(RuntimeError):
    pass


def _slots(obj, seen, is_group):
    """(owner, key, value) for every reference reachable from obj through
    instance attributes, lists, tuples-as-lists and dicts.  Group objects are
    leaves."""
    stack = [obj]
    while stack:
        o = stack.pop()
        if id(o) in seen:
            continue
        seen.add(id(o))
        if isinstance(o, dict):
            items = list(o.items())
        elif isinstance(o, list):
            items = list(enumerate(o))
        elif hasattr(o, "__dict__"):
            items = list(vars(o).items())
        else:
            continue
        for k, v in items:
            yield o, k, v
            if v is None or isinstance(v, (str, bytes, int, float, bool, Enum)) or is_group(v):
                continue
            stack.append(v)


def _set(owner, key, value):
    if isinstance(owner, (dict, list)):
        owner[key] = value
    else:
        setattr(owner, key, value)


def rebind(root, old, new, groups=()) -> int:
    """Redirect every reference to ``old`` reachable from ``root`` to ``new``
    and check the rebinding invariant (Sec. III-D): each slot that named
    ``old`` names ``new``, no slot names ``old`` afterwards, and every other
    slot is unchanged.  ``groups`` lists the objects to treat as leaves
    besides old and new.  Returns the number of references redirected."""
    leaves = {id(old), id(new)} | {id(g) for g in groups}
    is_group = lambda v: id(v) in leaves  # noqa: E731
    before = [(o, k, v) for o, k, v in _slots(root, set(), is_group)]
    hits = [(o, k) for o, k, v in before if v is old]
    for o, k in hits:
        _set(o, k, new)
    hit_ids = {(id(o), k if not isinstance(o, list) else int(k)) for o, k in hits}
    after = {(id(o), k if not isinstance(o, list) else int(k)): v for o, k, v in _slots(root, set(), is_group)}
    for o, k, v in before:
        key = (id(o), k if not isinstance(o, list) else int(k))
        now = after.get(key)
        if key in hit_ids:
            if now is not new:
                raise RebindError(f"a reference to the retired group was not redirected ({k})")
        elif now is not v:
            raise RebindError(f"a reference that did not name the retired group changed ({k})")
    if any(v is old for v in after.values()):
        raise RebindError("a reference to the retired group remains")
    return len(hits)


# ---------------------------------------------------------------------------
# the rank's state engine on the GPU
# ---------------------------------------------------------------------------

class ShardEngine:
    """One rank's flat fp32 shard on its GPU: weights, gradient, AdamW
    moments and bf16 copy, committed and digested by libpactshard.

    The gradient of update t stands in for forward and backward: it is drawn
    by the seeded generator from (seed, t) at the shard's global indices, so
    replicas of one shard compute bit-identical updates."""

    def __init__(self, numel: int, global_offset: int, seed: int, hyper: Optional[dict] = None,
                 device: str = "cuda:0"):
        import torch

        import workloads as wl
        from . import Hyper, Shard, _lib

        _lib()  # no library, no engine: there is no fallback
        self.torch, self.wl = torch, wl
        self.numel, self.goff, self.seed = int(numel), int(global_offset), int(seed)
        self.device = torch.device(device)
        torch.cuda.set_device(self.device)
        self.hyper = Hyper(**(hyper or {}))
        t = [torch.empty(self.numel, dtype=torch.float32, device=self.device) for _ in range(4)]
        wl.fill_device(t[0], self.goff, self.seed, wl.ARRAY_PARAM, 0, wl.NORMAL(0.02))
        t[1].zero_()
        t[2].zero_()
        t[3].zero_()
        self.bf16 = torch.zeros(self.numel, dtype=torch.int16, device=self.device)
        self.shard = Shard(t[0], t[1], t[2], t[3], self.bf16, global_offset=self.goff)
        self._Shard = Shard

    def produce_grad(self, step: int) -> None:
        self.wl.fill_device(self.shard.grad, self.goff, self.seed, self.wl.ARRAY_GRAD, step, self.wl.NORMAL(1e-3))

    def commit(self, step: int, torn: bool = False) -> int:
        """The fused commit of update ``step`` (gradient zeroed in the same
        pass); returns the digest the commit produced.  ``torn`` (fault
        injection) models an interrupted commit whose host side carried on:
        the update reaches only the first half of the shard, the whole
        gradient is zeroed, and the digest the partial launch reported is
        returned as the committed one."""
        from . import adamw_commit, to_u64

        if not torn:
            return to_u64(adamw_commit(self.shard, step, self.hyper, zero_grad=True))[0]
        s = self.shard
        half = self._Shard(s.param, s.grad, s.exp_avg, s.exp_avg_sq, s.param_bf16, global_offset=self.goff,
                           segments=[(0, self.numel // 2, 0)], hypers=[self.hyper])
        d = to_u64(adamw_commit(half, step, zero_grad=True))[-1]
        s.grad.zero_()
        return d

    def outstanding(self) -> int:
        from . import grad_guard, to_u64

        return to_u64(grad_guard(self.shard))[0]

    def digest(self) -> int:
        from . import shard_digest, to_u64

        return to_u64(shard_digest(self.shard))[0]

    def synchronize(self) -> None:
        self.torch.cuda.synchronize(self.device)

    def save(self, path: str) -> None:
        import numpy as np

        s = self.shard
        np.savez(path, p=s.param.cpu().numpy(), m=s.exp_avg.cpu().numpy(), v=s.exp_avg_sq.cpu().numpy())

    def load(self, path: str) -> None:
        import numpy as np

        with np.load(path, allow_pickle=False) as z:
            for t, k in ((self.shard.param, "p"), (self.shard.exp_avg, "m"), (self.shard.exp_avg_sq, "v")):
                t.copy_(self.torch.from_numpy(z[k]).to(self.device))
        self.shard.grad.zero_()
        self.synchronize()


def load_engine(spec: str):
    """'module:Class' -> the class."""
    mod, _, cls = spec.partition(":")
    return getattr(importlib.import_module(mod), cls)


# ---------------------------------------------------------------------------
# per-phase deadlines
# ---------------------------------------------------------------------------

class Watchdog:
    """Ends the process with EXIT_TIMEOUT when the current phase outlives its
    deadline (the rank's own bound; its peers see the loss and end too)."""

    def __init__(self, log):
        self._lock = threading.Lock()
        self._phase, self._deadline = None, None
        self._log = log
        t = threading.Thread(target=self._run, daemon=True)
        t.start()

    def _run(self):
        while True:
            time.sleep(0.01)
            with self._lock:
                ph, dl = self._phase, self._deadline
            if dl is not None and time.monotonic() > dl:
                self._log(f"deadline of phase '{ph}' passed")
                _exit(EXIT_TIMEOUT)

    def arm(self, phase: str, seconds: float):
        with self._lock:
            self._phase, self._deadline = phase, time.monotonic() + seconds

    def disarm(self):
        with self._lock:
            self._phase, self._deadline = None, None


def _exit(code: int):
    sys.stdout.flush()
    sys.stderr.flush()
    os._exit(code)


class DataPlaneFault(RuntimeError):
    """A replication-group collective failed (timed out or aborted)."""


class InjectedFault(RuntimeError):
    pass


# ---------------------------------------------------------------------------
# one rank
# ---------------------------------------------------------------------------

@dataclass
class CohortSpec:
    """What the supervisor hands every rank of one cohort."""
    world: int
    shards: int
    layers: int
    updates: int
    numel: int                  # elements per shard
    seed: int
    engine: str
    engine_args: dict
    generation: int
    store: str                  # control-plane rendezvous file of this generation
    workdir: str
    checkpoint_at: int = 0      # update after which every rank saves its state (0: never)
    restart: bool = False       # start from the checkpoint (L2 restart)
    faults: List[dict] = field(default_factory=list)
    control_timeout: float = 20.0
    data_timeout: float = 1.5
    deadlines: Dict[str, float] = field(default_factory=lambda: {
        "guard": 10.0, "agree": 10.0, "replace": 15.0, "rebind": 5.0, "release": 10.0, "poll": 30.0})
    platform: str = "mi355x-rocm"
    resource: str = "hsdp"
    objective: str = "continue"
    envelope: Optional[Dict[str, str]] = None  # "platform|resource|phase|objective" -> "L1" / "L2"
    generation_index: int = 0   # which cohort of the job this is (data-plane faults name the cohort they hit)
    replay_to: int = 0          # frontier the failed cohort reached (a restart replays up to it)


class Rank:
    def __init__(self, spec: CohortSpec, rank: int):
        self.spec, self.rank = spec, rank
        self.shard_idx = rank % spec.shards
        self.replica_idx = rank // spec.shards
        self.result = {"rank": rank, "shard": self.shard_idx, "generation": spec.generation, "repairs": [],
                       "replayed_updates": 0, "exit": None}
        self.repairs = 0
        self.generation = spec.generation
        self.frontier = 0
        self.watch = Watchdog(self.log)
        entries = None
        if spec.envelope is not None:
            entries = {tuple(k.split("|")): (Action.L1_PRESERVE if v == "L1" else Action.L2_RESTART)
                       for k, v in spec.envelope.items()}
        self.envelope = Envelope(entries)

    # -- plumbing ----------------------------------------------------------
    def log(self, msg: str):
        print(f"[rank {self.rank} g{self.generation}] {msg}", file=sys.stderr, flush=True)

    def write_result(self):
        path = os.path.join(self.spec.workdir, f"rank{self.rank}_g{self.spec.generation}.json")
        with open(path + ".tmp", "w") as f:
            json.dump(self.result, f)
        os.replace(path + ".tmp", path)

    def end(self, code: int, why: str):
        self.result["exit"] = code
        self.result["why"] = why
        self.result["frontier"] = self.frontier
        self.result["generation"] = self.generation
        self.log(f"exit {EXIT_NAMES.get(code, code)}: {why}")
        try:
            self.write_result()
        finally:
            _exit(code)

    def faults(self, **match):
        for f in self.spec.faults:
            if f.get("rank") == self.rank and all(f.get(k) == v for k, v in match.items()):
                yield f

    def maybe_fault(self, phase: str):
        for f in self.faults(phase=phase):
            if f.get("repair", 0) != self.repairs:
                continue
            if f["kind"] == "raise":
                raise InjectedFault(f"injected exception in phase {phase}")
            if f["kind"] == "hang":
                self.log(f"injected hang in phase {phase}")
                while True:
                    time.sleep(1.0)

    # -- set-up --------------------------------------------------------------
    def setup(self):
        import torch
        import torch.distributed as dist

        self.torch, self.dist = torch, dist
        sp = self.spec
        dist.init_process_group("gloo", init_method=f"file://{sp.store}", rank=self.rank, world_size=sp.world,
                                timeout=timedelta(seconds=sp.control_timeout))
        self.world = dist.group.WORLD
        self.replicas = sp.world // sp.shards
        # every rank creates every group, in one order (the process-group API
        # requires it); a rank keeps the handles of the groups it belongs to
        self.repl_members = {s: [s + q * sp.shards for q in range(self.replicas)] for s in range(sp.shards)}
        self.repl = {}
        for s in range(sp.shards):
            g = dist.new_group(self.repl_members[s], timeout=timedelta(seconds=sp.data_timeout), backend="gloo")
            if self.rank in self.repl_members[s]:
                self.repl[s] = g
        self.intra = None
        for q in range(self.replicas):
            g = dist.new_group([q * sp.shards + s for s in range(sp.shards)], backend="gloo")
            if q == self.replica_idx:
                self.intra = g
        self.model = build_model(sp.layers, self.repl[self.shard_idx], self.intra, self.world)
        cls = load_engine(sp.engine)
        args = dict(sp.engine_args)
        self.engine = cls(numel=sp.numel, global_offset=self.shard_idx * sp.numel, seed=sp.seed, **args)
        self.committed_digest = 0

    # -- the data plane --------------------------------------------------------
    def _collective(self, site: str, t: int, value: float):
        """A replication-group all-reduce (the gradient reduction, or the
        post-commit metric); an injected fault makes this rank drop out of it,
        so its peers time out as they would on a failed link."""
        for f in self.faults(site=site, update=t):
            if f.get("cohort", 0) == self.spec.generation_index:
                raise DataPlaneFault(f"injected collective timeout at {site} of update {t}")
        x = self.torch.tensor([value], dtype=self.torch.float64)
        try:
            self.dist.all_reduce(x, group=self.repl[self.shard_idx])
        except Exception as e:  # noqa: BLE001 -- any failure of the collective is an observation
            raise DataPlaneFault(f"{site} collective of update {t} failed: {e}") from e
        return float(x.item())

    def set_state(self, st: ModState):
        for w in wrappers(self.model):
            w.state = st

    def update(self, t: int):
        """One optimizer update: forward, backward with the gradient
        reduction, the commit, then the post-commit metric reduction."""
        sp = self.spec
        self.set_state(ModState.FORWARD)
        self.engine.produce_grad(t)
        for f in self.faults(site="forward", update=t):
            if f.get("cohort", 0) == sp.generation_index:
                raise DataPlaneFault(f"injected collective timeout in forward of update {t}")
        self.set_state(ModState.BACKWARD)
        self._collective("backward", t, 1.0)
        torn = any(f.get("cohort", 0) == sp.generation_index for f in self.faults(kind="torn_commit", update=t))
        self.committed_digest = self.engine.commit(t, torn=torn)
        self.frontier = t
        self.set_state(ModState.IDLE)
        if sp.checkpoint_at and t == sp.checkpoint_at and not sp.restart:
            self.engine.save(self.checkpoint_path())
        self._collective("committed", t, float(t))

    def checkpoint_path(self):
        return os.path.join(self.spec.workdir, f"ckpt_rank{self.rank}.npz")

    def phase_now(self) -> Phi:
        states = {w.state for w in wrappers(self.model)}
        if ModState.FORWARD in states:
            return Phi.FORWARD
        if ModState.BACKWARD in states:
            return Phi.BACKWARD
        return Phi.COMMITTED

    # -- the control plane -----------------------------------------------------
    def poll(self, observed: Optional[Action]) -> int:
        """The boundary poll over all W ranks: the largest action code any
        rank observed (0: nothing observed)."""
        x = self.torch.tensor([0 if observed is None else int(observed)], dtype=self.torch.int64)
        self.watch.arm("poll", self.spec.deadlines["poll"])
        self.dist.all_reduce(x, op=self.dist.ReduceOp.MAX)
        self.watch.disarm()
        return int(x.item())

    def run(self):
        sp = self.spec
        t = 1
        if sp.restart:
            self.engine.load(self.checkpoint_path())
            self.frontier = sp.checkpoint_at
            self.committed_digest = self.engine.digest()
            t = sp.checkpoint_at + 1
            self.result["replayed_updates"] = max(0, sp.replay_to - sp.checkpoint_at)
        while t <= sp.updates:
            observed = None
            try:
                self.update(t)
            except DataPlaneFault as e:
                phi = self.phase_now()
                key = ObservationKey(sp.platform, sp.resource, phi, sp.objective)
                observed = self.envelope.action(key)
                self.log(f"observed: {e}; phase {phi.value} -> {observed.name}")
                self.result.setdefault("observed", []).append({"update": t, "phase": phi.value,
                                                               "action": observed.name})
            decision = self.poll(observed)
            if decision == 0:
                t = self.frontier + 1
                continue
            if decision == Action.L2_RESTART:
                self.end(EXIT_REJECTED, "uncommitted failure: fail-stop rejection, checkpoint restart")
            self.recover(affected=observed is not None)
            t = self.frontier + 1
        self.finish()

    def finish(self):
        self.engine.synchronize()
        self.result.update(frontier=self.frontier, generation=self.generation,
                           committed_digest=f"{self.committed_digest:#018x}",
                           state_digest=f"{self.engine.digest():#018x}", exit=EXIT_OK)
        self.write_result()
        # leave together: nobody tears the control plane down under a peer
        self.watch.arm("finish", self.spec.deadlines["release"])
        self.dist.barrier()
        self.watch.disarm()

    # -- phases 2-6 ------------------------------------------------------------
    def recover(self, affected: bool):
        sp = self.spec
        rec = {"generation_from": self.generation, "frontier": self.frontier, "phases_ms": {}}
        t_all = time.perf_counter()

        def phase(name, fn):
            self.watch.arm(name, sp.deadlines[name])
            t0 = time.perf_counter()
            try:
                self.maybe_fault(name)
                out = fn()
            except Fenced as e:
                self.watch.disarm()
                self.end(EXIT_FENCED, f"phase {name}: {e}")
            except BaseException as e:  # noqa: BLE001 -- safety invariant: any error ends the rank
                self.watch.disarm()
                self.end(EXIT_FAILSTOP, f"phase {name}: {type(e).__name__}: {e}")
            self.watch.disarm()
            rec["phases_ms"][name] = (time.perf_counter() - t0) * 1e3
            return out

        phase("guard", self.phase_guard)
        g_new, affected_shards = phase("agree", lambda: self.phase_agree(affected))
        old = phase("replace", lambda: self.phase_replace(affected_shards))
        nref = phase("rebind", lambda: self.phase_rebind(old))
        phase("release", lambda: self.phase_release(affected_shards))
        self.generation = g_new
        self.repairs += 1
        rec.update(generation_to=g_new, rebound_references=nref, affected_shards=affected_shards,
                   total_ms=(time.perf_counter() - t_all) * 1e3, rebind_ms=rec["phases_ms"]["rebind"])
        self.result["repairs"].append(rec)
        self.log(f"repaired at frontier {self.frontier}, generation {g_new}, {nref} references rebound")

    def phase_guard(self):
        """Phase 2: drain the device queue; every wrapper IDLE; zero
        outstanding gradient elements."""
        self.engine.synchronize()
        for f in self.faults(kind="outstanding_grad"):
            if f.get("repair", 0) == self.repairs:
                self.engine.produce_grad(self.frontier + 1)
        busy = [w.name for w in wrappers(self.model) if w.state != ModState.IDLE]
        if busy:
            raise RuntimeError(f"wrappers not IDLE: {busy[:3]}")
        n = self.engine.outstanding()
        if n != 0:
            raise RuntimeError(f"{n} outstanding gradient elements at the boundary")

    def phase_agree(self, affected: bool):
        """Phase 3: control barrier; rank 0's (F, g+1) broadcast; exact
        agreement on the frontier, the generation and the committed state."""
        torch, dist = self.torch, self.dist
        dist.monitored_barrier(timeout=timedelta(seconds=self.spec.deadlines["agree"]))
        gen = self.generation
        for f in self.faults(kind="stale_generation"):
            if f.get("repair", 0) == self.repairs:
                gen -= 1
        frontier = self.frontier
        for f in self.faults(kind="frontier_mismatch"):
            if f.get("repair", 0) == self.repairs:
                frontier -= 1
        prop = torch.tensor([frontier, gen + 1], dtype=torch.int64)
        dist.broadcast(prop, src=0)
        F0, g_new = int(prop[0]), int(prop[1])
        now = self.engine.digest()

        def s64(x):
            return x - (1 << 64) if x >= (1 << 63) else x

        mine = torch.tensor([frontier, gen, s64(self.committed_digest), s64(now), self.shard_idx, int(affected)],
                            dtype=torch.int64)
        rows = [torch.zeros(6, dtype=torch.int64) for _ in range(self.spec.world)]
        dist.all_gather(rows, mine)
        rows = [[int(v) for v in r.tolist()] for r in rows]
        # every rank takes the same decision from the same gathered rows
        for r, (F, g, dc, dn, s, _) in enumerate(rows):
            if F != F0:
                raise Fenced(f"rank {r} holds frontier {F}, rank 0 proposed {F0}")
            if g + 1 != g_new:
                raise Fenced(f"rank {r} holds generation {g}, the cohort moves to {g_new} (stale rank fenced)")
            if dc != dn:
                raise Fenced(f"rank {r}: state digest {dn & MASK64:#018x} differs from its committed digest "
                             f"{dc & MASK64:#018x} (torn or altered commit)")
        by_shard: Dict[int, set] = {}
        for F, g, dc, dn, s, _ in rows:
            by_shard.setdefault(s, set()).add(dc)
        for s, ds in by_shard.items():
            if len(ds) != 1:
                raise Fenced(f"replicas of shard {s} hold different committed states")
        affected_shards = sorted({s for *_, s, a in rows if a})
        return g_new, affected_shards

    def phase_replace(self, affected_shards):
        """Phase 4: retire each affected replication group and build its
        replacement with the same members (every rank takes part in the
        group creation, members only use the result)."""
        dist = self.dist
        old = {}
        for s in affected_shards:
            if s == self.shard_idx:
                old[s] = self.repl[s]
                dist.destroy_process_group(self.repl[s])
            g = dist.new_group(self.repl_members[s], timeout=timedelta(seconds=self.spec.data_timeout),
                               backend="gloo")
            if self.rank in self.repl_members[s]:
                self.repl[s] = g
        return old

    def phase_rebind(self, old):
        """Phase 5: redirect the cached references to the retired group."""
        if self.shard_idx not in old:
            return 0
        new = self.repl[self.shard_idx]
        n = rebind(self.model, old[self.shard_idx], new, groups=(self.intra, self.world))
        if n != self.spec.layers + 1:
            raise RebindError(f"{n} references rebound, expected {self.spec.layers + 1}")
        return n

    def phase_release(self, affected_shards):
        """Phase 6: integer all-reduce over the replacement group, then the
        release barrier over all ranks."""
        torch, dist = self.torch, self.dist
        if self.shard_idx in affected_shards:
            x = torch.ones(1, dtype=torch.int64)
            dist.all_reduce(x, group=self.repl[self.shard_idx])
            if int(x.item()) != len(self.repl_members[self.shard_idx]):
                raise RuntimeError(f"validation all-reduce gave {int(x.item())}")
        dist.monitored_barrier(timeout=timedelta(seconds=self.spec.deadlines["release"]))


class Fenced(RuntimeError):
    """Phase 3 disagreement: the cohort aborts."""


def rank_main(argv=None) -> None:
    ap = argparse.ArgumentParser(description="one rank of a recovery cohort")
    ap.add_argument("--spec", required=True)
    ap.add_argument("--rank", type=int, required=True)
    a = ap.parse_args(argv)
    with open(a.spec) as f:
        spec = CohortSpec(**json.load(f))
    r = Rank(spec, a.rank)
    try:
        r.watch.arm("setup", spec.control_timeout + 30.0)
        r.setup()
        r.watch.disarm()
        r.run()
    except SystemExit:
        raise
    except BaseException as e:  # noqa: BLE001
        r.end(EXIT_ERROR, f"{type(e).__name__}: {e}")
    _exit(EXIT_OK)


# ---------------------------------------------------------------------------
# the supervisor
# ---------------------------------------------------------------------------

@dataclass
class CohortOutcome:
    generation: int
    exit_codes: List[int]
    seconds: float
    killed: List[int]
    results: List[Optional[dict]]

    @property
    def ok(self) -> bool:
        return all(c == EXIT_OK for c in self.exit_codes)


class Supervisor:
    """Starts a cohort of rank processes and, when it fails, a fresh cohort
    from the checkpoint (L2), at most ``max_restarts`` times.  Makes no GPU
    call itself, so it may start GPU ranks."""

    def __init__(self, world: int, shards: int, layers: int, updates: int, numel: int, seed: int = 7,
                 engine: str = "paper_2609_18178_amd.recovery:ShardEngine", engine_args: Optional[dict] = None,
                 checkpoint_at: int = 0, faults: Optional[List[dict]] = None, max_restarts: int = 1,
                 deadline: float = 180.0, workdir: Optional[str] = None, cwd: Optional[str] = None, **extra):
        if world % shards:
            raise ValueError("world must be a multiple of shards")
        self.base = dict(world=world, shards=shards, layers=layers, updates=updates, numel=numel, seed=seed,
                         engine=engine, engine_args=engine_args or {}, checkpoint_at=checkpoint_at,
                         faults=faults or [], **extra)
        self.max_restarts = max_restarts
        self.deadline = deadline
        self.workdir = workdir or tempfile.mkdtemp(prefix="pact_recovery_")
        self.cwd = cwd or os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
        self.cohorts: List[CohortOutcome] = []

    def launch(self, generation: int, index: int, restart: bool, replay_to: int = 0) -> CohortOutcome:
        store = os.path.join(self.workdir, f"store_g{generation}")
        spec = dict(self.base, generation=generation, store=store, workdir=self.workdir, restart=restart,
                    generation_index=index, replay_to=replay_to)
        path = os.path.join(self.workdir, f"spec_g{generation}.json")
        with open(path, "w") as f:
            json.dump(spec, f)
        env = dict(os.environ, GLOO_SOCKET_IFNAME=os.environ.get("GLOO_SOCKET_IFNAME", "lo"),
                   PYTHONUNBUFFERED="1", OMP_NUM_THREADS="1")
        logs, procs = [], []
        t0 = time.monotonic()
        for r in range(spec["world"]):
            log = open(os.path.join(self.workdir, f"rank{r}_g{generation}.log"), "w")
            logs.append(log)
            procs.append(subprocess.Popen([sys.executable, "-m", "paper_2609_18178_amd.recovery", "--spec", path,
                                           "--rank", str(r)], cwd=self.cwd, env=env, stdout=log,
                                          stderr=subprocess.STDOUT, start_new_session=True))
        killed = []
        while any(p.poll() is None for p in procs):
            if time.monotonic() - t0 > self.deadline:
                for r, p in enumerate(procs):
                    if p.poll() is None:
                        p.kill()
                        killed.append(r)
                break
            time.sleep(0.02)
        codes = [p.wait() for p in procs]
        for log in logs:
            log.close()
        results = []
        for r in range(spec["world"]):
            try:
                with open(os.path.join(self.workdir, f"rank{r}_g{generation}.json")) as f:
                    results.append(json.load(f))
            except (OSError, ValueError):
                results.append(None)
        out = CohortOutcome(generation, codes, time.monotonic() - t0, killed, results)
        self.cohorts.append(out)
        return out

    def run(self) -> CohortOutcome:
        gen = 0
        out = self.launch(gen, 0, restart=False)
        restarts = 0
        while not out.ok and restarts < self.max_restarts and self.base["checkpoint_at"]:
            frontier = max((r or {}).get("frontier", 0) for r in out.results)
            gen = max([gen] + [((r or {}).get("generation") or 0) for r in out.results]) + 1
            restarts += 1
            out = self.launch(gen, restarts, restart=True, replay_to=frontier)
        return out

    def log_text(self, rank: int, generation: int) -> str:
        try:
            with open(os.path.join(self.workdir, f"rank{rank}_g{generation}.log")) as f:
                return f.read()
        except OSError:
            return ""


if __name__ == "__main__":
    rank_main()
