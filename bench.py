#!/usr/bin/env python3
"""Benchmark: fused sharded AdamW commit + state digest on one MI355X.

One step = one commit of the whole shard (read p, g, m, v; write p', m', v'
and the bf16 copy; digest of the committed state in the same pass).  Default
workload: the 453,001,472-element 1/16 FSDP shard of Mistral-7B at rank 15
(flat indices beyond 2^32), warm AdamW state at step 5.  Inputs are
synthetic, drawn by the seeded generator in ``workloads`` and resident in HBM
before timing starts.

Prints one JSON line.  ``value`` is elements committed per second;
``roofline`` prices the commit kernel against MI355X's 8 TB/s HBM peak at
30 algorithmic bytes per element; ``cpu_baseline`` times the CPU oracle on a
bounded sample of the same workload.
"""
import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "shard commit+digest elements/s and HBM GB/s (% of MI355X peak), 1 GPU"
PEAK_HBM_GBPS = 8000.0
PREWARM_S = 0.3  # seconds of read-only digest calls before the warm-up commits
SETTLE_S = 0.2   # seconds each neighbouring kernel runs untimed before it is timed
BYTES_PER_ELEM = 30  # read p, g, m, v (16) + write p', m', v' (12) + bf16 (2)
KERNEL_SOURCES = ("paper_2609_18178_amd/csrc/kernels.hip", "paper_2609_18178_amd/csrc/launch.h")


def kernel_source_hash() -> str:
    h = hashlib.sha256()
    for rel in KERNEL_SOURCES:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def parse():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="mistral7b_shard16")
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="target seconds of the pinned single-thread CPU oracle leg (the multi-thread context "
                         "leg takes half)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-probe", action="store_true")
    ap.add_argument("--no-parity", action="store_true", help="skip the in-run oracle replay of the timed commits")
    ap.add_argument("--record-valu-ceiling", action="store_true",
                    help="also write profiles/valu_ceiling_<kernel>.json from this run's cache-resident timings")
    ap.add_argument("--layout", choices=("spread", "packed"), default="spread",
                    help="spread: the five arrays in one ShardArena pool, each in its own region of HBM "
                         "(the library's recommended placement); packed: five separate allocations")
    ap.add_argument("--spacing-gib", type=float, default=0.0,
                    help="spread layout: GiB between the arrays (default 0: the library's placement rule)")
    ap.add_argument("--no-compare-layout", action="store_true",
                    help="skip timing the other layout as well")
    ap.add_argument("--launch-shape", action="store_true",
                    help="only compare launch shapes of the 30 B/element stream probe on the workload's arrays: one "
                         "workgroup per tile against persistent grid-stride grids; writes "
                         "profiles/launch_shape_<workload>.json")
    ap.add_argument("--record-clock", metavar="CLOCK_CSV",
                    help="write profiles/clock_<workload>.json (shader clock, VALU issue and VALU busy per kernel) "
                         "from a rocprofv3 --pmc GRBM_GUI_ACTIVE SQ_INSTS_VALU SQ_ACTIVE_INST_VALU run of bench.py")
    ap.add_argument("--record-traffic", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"),
                    help="turn two rocprofv3 --pmc counter_collection.csv files (FETCH_SIZE, WRITE_SIZE) of a "
                         "bench run into profiles/traffic_<workload>.json and exit")
    return ap.parse_args()


COMMIT_KERNEL = "tile_kernel<(pact::Mode)0>"
PROBE_KERNEL = "probe_kernel("


def _counter_values(path: str, counter: str):
    import csv

    out = {}
    with open(path) as f:
        for row in csv.DictReader(f):
            if row["Counter_Name"] != counter:
                continue
            name = row["Kernel_Name"]
            key = "commit" if COMMIT_KERNEL in name else "probe" if PROBE_KERNEL in name else None
            if key:
                out.setdefault(key, []).append(float(row["Counter_Value"]) * 1024.0)  # KiB -> bytes
    return out


def record_traffic(workload: str, fetch_csv: str, write_csv: str) -> dict:
    """HBM bytes per commit launch from FETCH_SIZE and WRITE_SIZE, each scaled
    by what the same counter reads for the stream probe, whose bytes are known
    exactly (16 fetched and 14 written per element)."""
    import workloads as wl

    n = wl.WORKLOADS[workload].numel
    f = _counter_values(fetch_csv, "FETCH_SIZE")
    w = _counter_values(write_csv, "WRITE_SIZE")
    mean = lambda xs: sum(xs) / len(xs)  # noqa: E731
    f_scale = 16.0 * n / mean(f["probe"])
    w_scale = 14.0 * n / mean(w["probe"])
    fetch = mean(f["commit"]) * f_scale
    write = mean(w["commit"]) * w_scale
    rec = {
        "workload": workload,
        "kernel_source_hash": kernel_source_hash(),
        "bytes_per_launch": fetch + write,
        "fetch_bytes_per_launch": fetch,
        "write_bytes_per_launch": write,
        "algorithmic_bytes_per_launch": BYTES_PER_ELEM * n,
        "fetch_scale": f_scale,
        "write_scale": w_scale,
        "commit_dispatches": [len(f["commit"]), len(w["commit"])],
        "probe_dispatches": [len(f["probe"]), len(w["probe"])],
    }
    path = os.path.join(ROOT, "profiles", f"traffic_{workload}.json")
    with open(path, "w") as fh:
        json.dump(rec, fh, indent=1)
        fh.write("\n")
    return rec


def cpu_baseline(w, seconds: float) -> dict:
    """The oracle, unchanged, on a bounded sample: the first 2^24 elements of
    the same shard (same offset, distributions and step).  The reported
    value: one thread pinned to one host core, repeating commit + digest
    until `seconds` have passed.  Context: the same sample cut into one slice
    per host thread (up to 16), run concurrently."""
    from concurrent.futures import ThreadPoolExecutor

    import numpy as np

    import oracle
    import workloads as wl

    n = min(1 << 24, w.numel)
    p, g, m, v = wl.arrays_host(w, 0, n)
    b = np.zeros(n, np.uint16)
    h = oracle.Hyper(**(w.hypers[0]))

    def leg(threads, budget, pin=None):
        cuts = [n * k // threads for k in range(threads + 1)]

        def one(args):
            k, step = args
            if pin is not None:
                os.sched_setaffinity(0, {pin})  # this thread only
            a, z = cuts[k], cuts[k + 1]
            return oracle.commit_and_digest(p[a:z], g[a:z], m[a:z], v[a:z], b[a:z], h, step, w.global_offset + a)

        done, step, t0 = 0, w.first_step, time.perf_counter()
        with ThreadPoolExecutor(threads) as ex:
            while True:
                list(ex.map(one, [(k, step) for k in range(threads)]))
                done += n
                step += 1
                el = time.perf_counter() - t0
                if el >= budget:
                    return done / el

    host_cpus = os.cpu_count() or 1
    allowed = sorted(os.sched_getaffinity(0))
    threads = max(1, min(16, len(allowed)))
    single = leg(1, seconds, pin=allowed[0])
    multi = leg(threads, seconds / 2)
    return {
        "value": single,
        "unit": "elements/s",
        "cores": 1,
        "kind": "oracle",
        "sample": f"first {n} elements (at most 2^24) of the {w.name} shard (same offset, distributions and step), "
                  f"commit+digest repeated for >= {seconds:g} s, one thread pinned to host core {allowed[0]}",
        "budget_s": seconds,
        "multi_thread": {"value": multi, "threads": threads,
                         "note": f"the same sample cut into {threads} slices run by {threads} threads "
                                 "(context, not the baseline)"},
        "host_cpus": host_cpus,
        "cpu_model": _cpu_model(),
    }


def oracle_replay(w, steps, want_digest: int, threads: int = 16, chunk: int = 1 << 24) -> dict:
    """In-run parity: the oracle replays, on the host, the exact sequence of
    commits the GPU ran (the generated state at the first step, the same
    gradient for every commit, steps `steps`) over the whole shard, chunk by
    chunk (each chunk cut into slices run by host threads; elements are
    independent, so the digest is the wrapping sum), and its final digest
    is compared with the GPU's."""
    from concurrent.futures import ThreadPoolExecutor

    import oracle
    import workloads as wl

    h = oracle.Hyper(**(w.hypers[0]))
    threads = max(1, min(threads, len(os.sched_getaffinity(0))))
    t0 = time.perf_counter()
    total = 0

    def replay(args):
        p, g, m, v, b, first = args
        for st in steps[:-1]:
            oracle.adamw_commit(p, g, m, v, b, h, st)
        return oracle.commit_and_digest(p, g, m, v, b, h, steps[-1], first)

    import numpy as np

    with ThreadPoolExecutor(threads) as ex:
        for a in range(0, w.numel, chunk):
            cnt = min(chunk, w.numel - a)
            p, g, m, v = wl.arrays_host(w, a, cnt)
            b = np.zeros(cnt, np.uint16)
            cuts = [cnt * k // threads for k in range(threads + 1)]
            jobs = [(p[x:y], g[x:y], m[x:y], v[x:y], b[x:y], w.global_offset + a + x)
                    for x, y in zip(cuts[:-1], cuts[1:]) if y > x]
            total += sum(ex.map(replay, jobs))
    total &= (1 << 64) - 1
    return {"checked": f"final digest after the {len(steps)} commits of steps {steps[0]}..{steps[-1]} "
                       "(warm-up and timed), replayed by the oracle over the whole shard",
            "oracle_digest": f"{total:#018x}", "gpu_digest": f"{want_digest:#018x}", "match": total == want_digest,
            "seconds": time.perf_counter() - t0, "threads": threads}


def _cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


# rocprofv3 kernel names -> the names bench.py reports them under
CLOCK_KERNELS = (("tile_kernel<(pact::Mode)0>", "commit", 30), ("probe_kernel(", "probe", 30),
                 ("tile_kernel<(pact::Mode)3>", "commit_zero_grad", 34), ("tile_kernel<(pact::Mode)4>", "grad_guard", 4),
                 ("tile_kernel<(pact::Mode)1>", "shard_digest", 12),
                 ("tile_kernel_bf16<(pact::Mode)5>", "commit_bf16_state", 14))
XCDS = 8      # GRBM_GUI_ACTIVE comes back summed over the eight XCDs
NUM_CUS = 256
# Nominal VALU issue peak: 256 CUs x 4 SIMDs, each SIMD 16 lanes wide, so one
# 64-lane wave-instruction per SIMD every 4 cycles, at 2.4 GHz.  gfx950
# finishes some VALU instructions in fewer cycles, so a kernel can pass it.
VALU_PEAK_WAVE_INSTR_PER_S = NUM_CUS * 4 * 16 / 64 * 2.4e9


def record_clock(workload: str, clock_csv: str) -> dict:
    """Per kernel, from one counter run: duration (dispatch timestamps), shader
    cycles (GRBM_GUI_ACTIVE per XCD), clock, VALU wave-instructions per element
    and per CU per cycle, and rocprofv3's VALUBusy
    (100 * SQ_ACTIVE_INST_VALU / CUs / GRBM_GUI_ACTIVE of one XCD)."""
    import csv

    import workloads as wl

    n = wl.WORKLOADS[workload].numel
    full_grid = -(-n // 4096) * 256  # work-items of one full-shard launch (one 256-thread workgroup per tile)
    disp = {}
    with open(clock_csv) as f:
        for row in csv.DictReader(f):
            hit = [(key, bpe) for pat, key, bpe in CLOCK_KERNELS if pat in row["Kernel_Name"]]
            if not hit or int(row.get("Grid_Size", full_grid)) != full_grid:
                continue  # other kernels, and the sub-shard launches of the VALU-ceiling timing
            d = disp.setdefault(int(row["Dispatch_Id"]), {"key": hit[0][0], "bpe": hit[0][1]})
            d[row["Counter_Name"]] = float(row["Counter_Value"])
            d["dur_s"] = (int(row["End_Timestamp"]) - int(row["Start_Timestamp"])) * 1e-9
    kernels = {}
    for d in disp.values():
        kernels.setdefault(d["key"], []).append(d)
    rec = {"workload": workload, "kernel_source_hash": kernel_source_hash(), "kernels": {}}
    for key, ds in kernels.items():
        k = len(ds)
        dur = sum(d["dur_s"] for d in ds) / k
        cyc = sum(d["GRBM_GUI_ACTIVE"] for d in ds) / k / XCDS
        valu = sum(d["SQ_INSTS_VALU"] for d in ds) / k
        active = (sum(d["SQ_ACTIVE_INST_VALU"] for d in ds) / k) if "SQ_ACTIVE_INST_VALU" in ds[0] else None
        rec["kernels"][key] = {
            "dispatches": k, "us": dur * 1e6, "mcycles": cyc / 1e6, "clock_ghz": cyc / dur / 1e9,
            "bytes_per_element": ds[0]["bpe"], "gbps": ds[0]["bpe"] * n / dur / 1e9,
            "valu_instr_per_element": valu * 64 / n, "valu_issue_per_cu_cycle": valu / NUM_CUS / cyc,
            "valu_busy_pct": None if active is None else 100.0 * active / NUM_CUS / cyc,
        }
    path = os.path.join(ROOT, "profiles", f"clock_{workload}.json")
    with open(path, "w") as fh:
        json.dump(rec, fh, indent=1)
        fh.write("\n")
    return rec


def stored_clock(workload: str, src_hash: str):
    """The clock / VALU record of the current kernel source, if there is one."""
    try:
        with open(os.path.join(ROOT, "profiles", f"clock_{workload}.json")) as f:
            rec = json.load(f)
    except (OSError, ValueError):
        return None
    return rec if rec.get("kernel_source_hash") == src_hash else None


def stored_traffic(workload: str, src_hash: str):
    """HBM bytes per launch from rocprofv3 FETCH_SIZE / WRITE_SIZE runs of the
    current kernel source, if such a record exists."""
    path = os.path.join(ROOT, "profiles", f"traffic_{workload}.json")
    try:
        with open(path) as f:
            rec = json.load(f)
    except (OSError, ValueError):
        return None
    if rec.get("kernel_source_hash") != src_hash:
        return None
    return rec


def launch_shape(w, args) -> dict:
    """The 30 B/element stream probe on the workload's arrays (spread layout,
    zero-filled: the probe's cost does not depend on the values), launched
    with one workgroup per tile (the kernels' shape) and from persistent
    grids of 1-16 workgroups per CU striding over the tiles; median of 20
    launches per shape, four rounds in alternating order, best round kept."""
    import torch

    import paper_2609_18178_amd as pk

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    n = w.numel
    arena = pk.ShardArena(n, dev, spacing=int(args.spacing_gib * (1 << 30)) or None)
    ts = [arena.param, arena.grad, arena.exp_avg, arena.exp_avg_sq]
    for t in ts:
        t.zero_()
    arena.param_bf16.zero_()
    cus = torch.cuda.get_device_properties(dev).multi_processor_count
    shapes = [0] + [cus * k for k in (1, 2, 4, 8, 16)]

    def run(wg):
        pk.stream_probe(ts[0], ts[1], ts[2], ts[3], ts[0], ts[2], ts[3], arena.param_bf16, workgroups=wg)

    def median(wg, reps=20):
        run(wg)
        torch.cuda.synchronize()
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(reps + 1)]
        ev[0].record()
        for r in range(reps):
            run(wg)
            ev[r + 1].record()
        torch.cuda.synchronize()
        xs = sorted(ev[r].elapsed_time(ev[r + 1]) for r in range(reps))
        return xs[reps // 2]

    t_end = time.perf_counter() + PREWARM_S
    while time.perf_counter() < t_end:
        run(0)
    torch.cuda.synchronize()
    res = {wg: [] for wg in shapes}
    for rnd in range(4):
        for wg in (shapes if rnd % 2 == 0 else shapes[::-1]):
            res[wg].append(median(wg))
    best = {wg: min(v) for wg, v in res.items()}
    out = {"workload": w.name, "elements": n, "cus": cus, "kernel_source_hash": kernel_source_hash(),
           "command": f"python bench.py --workload {w.name} --launch-shape",
           "shapes": [{"workgroups": ("one per tile" if wg == 0 else wg),
                       "workgroups_per_cu": (None if wg == 0 else wg // cus),
                       "median_ms": best[wg], "gbps": BYTES_PER_ELEM * n / (best[wg] / 1e3) / 1e9,
                       "vs_one_per_tile": best[0] / best[wg]} for wg in shapes]}
    with open(os.path.join(ROOT, "profiles", f"launch_shape_{w.name}.json"), "w") as fh:
        json.dump(out, fh, indent=1)
        fh.write("\n")
    return out


def main():
    args = parse()
    if args.record_clock:
        print(json.dumps(record_clock(args.workload, args.record_clock)))
        return
    if args.record_traffic:
        print(json.dumps(record_traffic(args.workload, *args.record_traffic)))
        return
    if args.gpus != 1:
        print(f"bench.py: measures one GPU only (asked for --gpus {args.gpus}): the commit of a rank's shard "
              "needs no communication, and the library has no multi-GPU path.", file=sys.stderr)
        sys.exit(2)

    import torch

    import paper_2609_18178_amd as pk
    import workloads as wl

    w = wl.WORKLOADS[args.workload]
    if args.launch_shape:
        print(json.dumps(launch_shape(w, args)))
        return
    if w.segments is not None:
        segments = list(w.segments)
        hypers = [pk.Hyper(**h) for h in w.hypers]
    else:
        segments, hypers = None, None
    hyper = None if segments else pk.Hyper(**w.hypers[0])
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    n = w.numel
    algo_bytes = BYTES_PER_ELEM * n

    def allocate(layout):
        if layout == "spread":
            arena = pk.ShardArena(n, dev, spacing=int(args.spacing_gib * (1 << 30)) or None)
            return arena, [arena.param, arena.grad, arena.exp_avg, arena.exp_avg_sq], arena.param_bf16
        ts = [torch.empty(n, dtype=torch.float32, device=dev) for _ in range(4)]
        return None, ts, torch.empty(n, dtype=torch.int16, device=dev)

    def fill(tensors, bf16):
        for t, aid, st, dist in zip(tensors, (wl.ARRAY_PARAM, wl.ARRAY_GRAD, wl.ARRAY_EXP_AVG, wl.ARRAY_EXP_AVG_SQ),
                                    (0, w.first_step, 0, 0), (w.param, w.grad, w.exp_avg, w.exp_avg_sq)):
            wl.fill_device(t, w.global_offset, w.seed, aid, st, dist)
        bf16.zero_()

    def measure(sh, K, W):
        """Pre-warm, W untimed commits, then K timed ones; hipEvents around each
        call and around the whole timed region, on the stream the library
        launches on.  The pre-warm runs the read-only state digest over the
        shard for PREWARM_S seconds (the state is not changed): after the
        host-side fill the GPU sits at idle clocks, and the first commits run
        up to 10% slower until it has been busy for some tens of ms."""
        t_end = time.perf_counter() + PREWARM_S
        while time.perf_counter() < t_end:
            pk.shard_digest(sh)
            torch.cuda.synchronize()
        step = w.first_step
        for _ in range(W):
            pk.adamw_commit(sh, step, hyper)
            step += 1
        torch.cuda.synchronize()
        ev_s = [torch.cuda.Event(enable_timing=True) for _ in range(K)]
        ev_e = [torch.cuda.Event(enable_timing=True) for _ in range(K)]
        region_s, region_e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        wall0 = time.perf_counter()
        region_s.record()
        for k in range(K):
            ev_s[k].record()
            pk.adamw_commit(sh, step, hyper)
            ev_e[k].record()
            step += 1
        region_e.record()
        torch.cuda.synchronize()
        wall = time.perf_counter() - wall0
        per_launch = [a.elapsed_time(b) for a, b in zip(ev_s, ev_e)]
        return {"ms_per_step": region_s.elapsed_time(region_e) / K, "avg_launch_ms": sum(per_launch) / K,
                "min_launch_ms": min(per_launch), "median_launch_ms": sorted(per_launch)[K // 2],
                "launch_ms": per_launch, "wall_s": wall, "digest": pk.to_u64(sh.digest)[-1]}

    def probe(tensors, bf16, K):
        p_s = [torch.cuda.Event(enable_timing=True) for _ in range(K)]
        p_e = [torch.cuda.Event(enable_timing=True) for _ in range(K)]
        for k in range(K):
            p_s[k].record()
            pk.stream_probe(tensors[0], tensors[1], tensors[2], tensors[3], tensors[0], tensors[2], tensors[3], bf16)
            p_e[k].record()
        torch.cuda.synchronize()
        pms = sum(a.elapsed_time(b) for a, b in zip(p_s, p_e)) / K
        return {"kernel": "stream_probe", "ms": pms, "gbps": algo_bytes / (pms / 1e3) / 1e9,
                "frac_of_peak": algo_bytes / (pms / 1e3) / 1e9 / PEAK_HBM_GBPS}

    t_setup = time.perf_counter()
    arena, tensors, bf16 = allocate(args.layout)
    fill(tensors, bf16)
    sh = pk.Shard(*tensors, bf16, global_offset=w.global_offset, segments=segments, hypers=hypers)
    setup_s = time.perf_counter() - t_setup
    print(f"[bench] {w.name}: {n} elements resident, {args.layout} layout ({setup_s:.1f} s setup)",
          file=sys.stderr, flush=True)

    K = args.steps
    main_m = measure(sh, K, args.warmup)
    ms_per_step = main_m["ms_per_step"]
    avg_launch_ms = main_m["avg_launch_ms"]
    value = n / (ms_per_step / 1e3)
    achieved = algo_bytes / (avg_launch_ms / 1e3) / 1e9
    print("[bench] per commit (ms): " + " ".join(f"{x:.3f}" for x in main_m["launch_ms"]), file=sys.stderr, flush=True)
    print(f"[bench] {K} commits: {ms_per_step:.4f} ms/step, kernel {avg_launch_ms:.4f} ms avg "
          f"(min {main_m['min_launch_ms']:.4f}), {achieved:.1f} GB/s", file=sys.stderr, flush=True)
    last_digest = main_m["digest"]
    wall = main_m["wall_s"]
    timed_steps = [w.first_step + args.warmup, w.first_step + args.warmup + K - 1]

    probe_res = None
    if not args.no_probe and segments is None:
        probe_res = probe(tensors, bf16, K)
        print(f"[bench] stream probe (same 30 B/element, no math): {probe_res['gbps']:.1f} GB/s",
              file=sys.stderr, flush=True)

    # the neighbouring kernels on the same shard (after the timed region):
    # the commit that also zeroes the gradient (34 B/element), the gradient
    # guard (4 B/element) and the standalone state digest (12 B/element)
    extra = {}
    if not args.no_probe:
        def settle(fn, seconds):
            """Run fn back to back for `seconds` before it is timed: the shader
            clock the power manager picks depends on what ran just before
            (after the HBM-heavy commits it sits lower, and a VALU-bound kernel
            timed right after them reads up to 10% slow), so each kernel is
            timed at the clock its own steady run settles to."""
            t_end = time.perf_counter() + seconds
            while time.perf_counter() < t_end:
                for _ in range(4):
                    fn()
                torch.cuda.synchronize()

        def time_call(fn, reps):
            settle(fn, SETTLE_S)
            fn()
            torch.cuda.synchronize()
            s_ev, e_ev = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            s_ev.record()
            for _ in range(reps):
                fn()
            e_ev.record()
            torch.cuda.synchronize()
            return s_ev.elapsed_time(e_ev) / reps

        def median_launch(fn, reps, settle_s=0.0):
            settle(fn, settle_s)
            fn()
            torch.cuda.synchronize()
            ev = [torch.cuda.Event(enable_timing=True) for _ in range(reps + 1)]
            ev[0].record()
            for r in range(reps):
                fn()
                ev[r + 1].record()
            torch.cuda.synchronize()
            ts = sorted(ev[r].elapsed_time(ev[r + 1]) for r in range(reps))
            return ts[reps // 2]

        reps = max(3, K // 2)
        zstep = [w.first_step + args.warmup + K]

        def zcommit():
            pk.adamw_commit(sh, zstep[0], hyper, zero_grad=True)
            zstep[0] += 1

        kernels = [("commit_zero_grad", zcommit, 34), ("grad_guard", lambda: pk.grad_guard(sh), 4),
                   ("shard_digest", lambda: pk.shard_digest(sh), 12)]
        # the same shard held in BF16 (the paper's precision), 14 B/element:
        # its four arrays in four separate regions of the arena when spread
        if segments is None:
            b16 = []
            for k, t in enumerate(tensors):
                try:  # in the gap after fp32 array k when the arena spreads the arrays
                    dst = arena.take(n * 2, torch.int16, region=k) if arena is not None else None
                except MemoryError:  # a packed arena (small shard) has no gaps
                    dst = None
                if dst is None:
                    dst = torch.empty(n, dtype=torch.int16, device=dev)
                dst.view(torch.bfloat16).copy_(t)
                b16.append(dst)
            sh16 = pk.ShardBf16(*b16, global_offset=w.global_offset)
            bstep = [w.first_step]

            def bcommit():
                pk.adamw_commit_bf16(sh16, bstep[0], hyper)
                bstep[0] += 1

            kernels.append(("commit_bf16_state", bcommit, 14))
        # what bounds each one on MI355X (rocprofv3 clock and VALU counters):
        # HBM for the two that move 30+ B or a single array, VALU issue for the
        # BF16-state commit (as much arithmetic as the binary32 commit on half
        # the bytes), both for the digest (three hashes per 12 B)
        bounds = {"commit_zero_grad": "hbm", "grad_guard": "hbm", "shard_digest": "hbm+valu",
                  "commit_bf16_state": "valu"}
        for name, fn, bpe in kernels:
            ms = time_call(fn, reps)
            med = median_launch(fn, reps)
            extra[name] = {"ms": ms, "median_launch_ms": med, "bound": bounds[name], "bytes_per_element": bpe,
                           "gbps": bpe * n / (ms / 1e3) / 1e9,
                           "frac_of_peak": bpe * n / (ms / 1e3) / 1e9 / PEAK_HBM_GBPS}
            print(f"[bench] {name}: {ms:.4f} ms (median {med:.4f}), {extra[name]['gbps']:.1f} GB/s at {bpe} B/element",
                  file=sys.stderr, flush=True)

        # VALU ceilings of the two VALU-heavy kernels: the same kernel on
        # sub-shards small enough to stay in the 256 MB Infinity Cache, at two
        # sizes; the slope of launch time over elements is the kernel's rate
        # when HBM does not limit it (launch and tail costs cancel in the
        # difference).  frac = the full-size time that rate allows / the
        # measured full-size time.
        def subshard_fn(name, m):
            if name == "shard_digest":
                ss = pk.Shard(tensors[0][:m], None, tensors[2][:m], tensors[3][:m], None,
                              global_offset=w.global_offset)
                return lambda: pk.shard_digest(ss)
            ss = pk.ShardBf16(*(t[:m] for t in b16), global_offset=w.global_offset)
            st = [w.first_step]

            def f():
                pk.adamw_commit_bf16(ss, st[0], hyper)
                st[0] += 1
            return f

        sub_sizes = (1 << 22, 2 << 22, 3 << 22, 4 << 22)
        for name, bpe, ws in (("shard_digest", 12, 12), ("commit_bf16_state", 14, 8)):
            if name not in extra or sub_sizes[-1] > n:
                continue
            ts = [median_launch(subshard_fn(name, m), 40, settle_s=SETTLE_S / 2) for m in sub_sizes]
            # least-squares slope of launch time over elements: the fixed
            # launch and tail costs drop out, and four sizes average the noise
            # of any one median
            mx, my = sum(sub_sizes) / len(ts), sum(ts) / len(ts)
            slope = (sum((x - mx) * (y - my) for x, y in zip(sub_sizes, ts))
                     / sum((x - mx) ** 2 for x in sub_sizes))  # ms per element
            rate = 1e3 / slope
            full_ms = extra[name]["median_launch_ms"]
            ceil = {"elements_per_s": rate, "full_size_ms_at_ceiling": n / rate * 1e3,
                    "frac": (n / rate * 1e3) / full_ms,
                    "bytes_per_s_at_ceiling": rate * bpe,
                    "sizes": list(sub_sizes), "median_launch_ms": ts,
                    "working_set_bytes": sub_sizes[-1] * ws,
                    "method": "least-squares slope of the median launch time over four cache-resident "
                              "sub-shards (same kernel, same instruction mix); frac = full-size time at that "
                              "rate / measured full-size median launch time"}
            extra[name]["valu_ceiling"] = ceil
            print(f"[bench] {name}: cache-resident rate {rate:.3e} elem/s -> {n / rate * 1e3:.4f} ms at full size, "
                  f"frac {ceil['frac']:.3f} of that ceiling", file=sys.stderr, flush=True)
            if args.record_valu_ceiling:
                rec = dict(ceil, kernel=name, workload=w.name, full_size_elements=n, full_size_median_ms=full_ms,
                           kernel_source_hash=kernel_source_hash(),
                           command=f"python bench.py --workload {w.name} --record-valu-ceiling")
                with open(os.path.join(ROOT, "profiles", f"valu_ceiling_{name}.json"), "w") as fh:
                    json.dump(rec, fh, indent=1)
                    fh.write("\n")

    other = None
    if not args.no_compare_layout:
        other_layout = "packed" if args.layout == "spread" else "spread"
        del sh
        free, _ = torch.cuda.mem_get_info(dev)
        need = 4 * n * 4 + 2 * n if other_layout == "packed" else pk.arena_plan(n, int(args.spacing_gib * (1 << 30)))[0]
        if free > need + (2 << 30):
            o_arena, o_t, o_b = allocate(other_layout)
            fill(o_t, o_b)
            o_sh = pk.Shard(*o_t, o_b, global_offset=w.global_offset, segments=segments, hypers=hypers)
            om = measure(o_sh, K, args.warmup)
            other = {"layout": other_layout,
                     "note": ("five separate back-to-back allocations: the rate a caller that ignores the library's "
                              "placement rule gets" if other_layout == "packed" else "the library's placement rule"),
                     "ms_per_step": om["ms_per_step"],
                     "value": n / (om["ms_per_step"] / 1e3),
                     "achieved_gbps": algo_bytes / (om["avg_launch_ms"] / 1e3) / 1e9,
                     "frac": algo_bytes / (om["avg_launch_ms"] / 1e3) / 1e9 / PEAK_HBM_GBPS,
                     "same_digest": om["digest"] == last_digest}
            if segments is None and not args.no_probe:
                other["probe_gbps"] = probe(o_t, o_b, K)["gbps"]
            print(f"[bench] {other_layout} layout: {om['ms_per_step']:.4f} ms/step, "
                  f"{other['achieved_gbps']:.1f} GB/s", file=sys.stderr, flush=True)
            del o_sh, o_t, o_b, o_arena
        else:
            print(f"[bench] {other_layout} layout skipped: not enough free device memory", file=sys.stderr)

    src_hash = kernel_source_hash()
    traffic_rec = stored_traffic(w.name, src_hash)
    traffic = None if traffic_rec is None else traffic_rec["bytes_per_launch"]
    clock_rec = stored_clock(w.name, src_hash)
    clock_k = {} if clock_rec is None else clock_rec["kernels"]

    def valu_of(key):
        c = clock_k.get(key)
        if c is None:
            return None
        # busy_pct is rocprofv3's VALUBusy: four cycles per wave-instruction, so
        # on gfx950 (some VALU instructions take fewer) it can pass 100
        return {"busy_pct": c["valu_busy_pct"], "issue_per_cu_per_cycle": c["valu_issue_per_cu_cycle"],
                "instr_per_element": c["valu_instr_per_element"], "clock_ghz": c["clock_ghz"],
                "source": f"profiles/clock_{w.name}.json (rocprofv3 counters of this kernel source)"}

    for name, entry in extra.items():
        entry["valu"] = valu_of(name)
        if entry["valu"] is not None and "valu" in entry["bound"]:
            wave_instr = entry["valu"]["instr_per_element"] * n / 64  # per launch
            achieved_wi = wave_instr / (entry["median_launch_ms"] / 1e3)
            entry["alu_roofline"] = {
                "bound": "alu", "achieved": achieved_wi, "peak": VALU_PEAK_WAVE_INSTR_PER_S,
                "unit": "VALU wave-instructions/s", "frac": achieved_wi / VALU_PEAK_WAVE_INSTR_PER_S,
                "peak_derivation": "256 CUs x 4 SIMDs x 16 lanes per cycle / 64 lanes per wave-instruction x 2.4 GHz",
                "instructions": "SQ_INSTS_VALU per element from the clock record x elements / 64, per launch"}

    parity = None
    all_steps = list(range(w.first_step, w.first_step + args.warmup + K))
    if args.no_parity:
        parity = {"skipped": "--no-parity"}
    elif segments is not None or n * len(all_steps) > 2e10:
        parity = {"skipped": "the in-run replay covers flat shards of up to 2e10 element-commits; "
                             "this workload's parity is in the GPU tests"}
    else:
        print("[bench] oracle replay of the timed commits ...", file=sys.stderr, flush=True)
        parity = oracle_replay(w, all_steps, last_digest)
        print(f"[bench] parity: oracle {parity['oracle_digest']} gpu {parity['gpu_digest']} "
              f"{'match' if parity['match'] else 'MISMATCH'} ({parity['seconds']:.1f} s)", file=sys.stderr, flush=True)

    cpu = None
    if not args.no_cpu_baseline:
        print("[bench] CPU oracle baseline ...", file=sys.stderr, flush=True)
        cpu = cpu_baseline(w, args.cpu_seconds)

    out = {
        "metric": METRIC,
        "value": value,
        "unit": "elements/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic (seeded Philox4x32-10 inputs with the workload's shapes and distributions)",
        "config": dict(w.describe(), parallelism="one rank's shard, no collectives",
                       bytes_per_element=BYTES_PER_ELEM,
                       warmup_commits=args.warmup, timed_steps=timed_steps,
                       state=(f"generated at step {w.first_step}, then evolved by every commit (warm-up commits at "
                              f"steps {w.first_step}..{timed_steps[0] - 1}); the same gradient for every commit"),
                       layout=(f"spread: the five arrays in one ShardArena pool, "
                               f"{pk.arena_plan(n, int(args.spacing_gib * (1 << 30)))[1] / (1 << 30):g} GiB apart"
                               if args.layout == "spread" else "packed: five separate torch allocations")),
        "hbm_gbps_nominal": algo_bytes / (ms_per_step / 1e3) / 1e9,
        "pct_of_peak_hbm": 100.0 * algo_bytes / (ms_per_step / 1e3) / 1e9 / PEAK_HBM_GBPS,
        "roofline": {
            "bound": "hbm",
            "kernel": "tile_kernel<Commit>",
            "achieved": achieved,
            "peak": PEAK_HBM_GBPS,
            "unit": "GB/s",
            "frac": achieved / PEAK_HBM_GBPS,
            "traffic": traffic,
            "algorithmic_bytes_per_launch": algo_bytes,
            "avg_launch_ms": avg_launch_ms,
            "median_launch_ms": main_m["median_launch_ms"],
            "min_launch_ms": main_m["min_launch_ms"],
            "valu": valu_of("commit"),
            # the same 30 B/element pattern with no arithmetic, in the same run:
            # the practical ceiling of the access pattern (context, not the metric)
            "frac_of_probe": (achieved / probe_res["gbps"]) if probe_res else None,
            "timing": "hipEvents around each commit call on the launch stream; a call also runs the "
                      "one-workgroup kernels that clear and sum the digest lanes (a few microseconds)",
        },
        "cpu_baseline": cpu,
        "parity": parity,
        "probe": probe_res,
        "other_layout": other,
        "other_kernels": extra,
        "kernel_source_hash": src_hash,
        "last_digest": f"{last_digest:#018x}",
        "wall_s_timed_region": wall,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
