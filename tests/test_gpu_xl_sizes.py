"""GPU vs oracle at the benchmark workloads' full sizes (marked slow).

The 1/16 and 1/4 Mistral-7B shards are compared element by element after
every commit; the whole 7,248,023,552-element model (291 segments) through
its 292 state digests and 292 bf16 digests, which cover every committed word
(a single differing word changes its segment's digest for certain, since
splitmix64 is a bijection), plus every element of sampled chunks."""
import numpy as np
import pytest

import oracle
import workloads as wl
from tests.helpers import (M64, assert_bitwise, device_workload, g_hyper, host, o_hyper, oracle_commit_parallel,
                           oracle_stream_segments)

pytestmark = [pytest.mark.gpu, pytest.mark.slow]


def _pk():
    import paper_2609_18178_amd as pk

    return pk


def test_mistral7b_shard16_full_size():
    """453,001,472 elements, rank 15 (indices beyond 2^32), warm state at step
    5, in the benchmark's launch configuration: every output bitwise."""
    pk = _pk()
    w = wl.WORKLOADS["mistral7b_shard16"]
    print(f"[{w.name}] drawing", flush=True)
    p, g, m, v = wl.arrays_host(w)
    import torch

    sh = pk.Shard(*(torch.from_numpy(a).cuda() for a in (p, g, m, v)),
                  torch.zeros(w.numel, dtype=torch.int16, device="cuda"), global_offset=w.global_offset)
    print(f"[{w.name}] GPU commit", flush=True)
    d_gpu = pk.to_u64(pk.adamw_commit(sh, w.first_step, g_hyper(w.hypers[0])))[0]
    bd_gpu = pk.to_u64(pk.bf16_digest(sh))[0]
    print(f"[{w.name}] oracle commit", flush=True)
    b = np.zeros(w.numel, np.uint16)
    d_ref = oracle_commit_parallel(p, g, m, v, b, o_hyper(w.hypers[0]), w.first_step, w.global_offset)
    assert d_gpu == d_ref
    assert bd_gpu == oracle.bf16_digest(b, w.global_offset)
    for name, t, ref in (("param", sh.param, p), ("exp_avg", sh.exp_avg, m), ("exp_avg_sq", sh.exp_avg_sq, v)):
        assert_bitwise(name, host(t), ref)
    assert_bitwise("bf16", host(sh.param_bf16).view(np.uint16), b)
    assert pk.to_u64(pk.shard_digest(sh))[0] == d_ref


def test_mistral7b_shard4_ten_commits():
    """The paper's real per-rank state: the 1/4 HSDP shard, 1,812,005,888
    elements at rank 3, warm state at step 18, ten commits with a fresh
    gradient each, per-step digests compared step by step, every output
    bitwise at the end."""
    import torch

    pk = _pk()
    w = wl.WORKLOADS["mistral7b_shard4"]
    hy = w.hypers[0]
    print(f"[{w.name}] drawing", flush=True)
    p, g, m, v = wl.arrays_host(w)
    sh = pk.Shard(*(torch.from_numpy(a).cuda() for a in (p, g, m, v)),
                  torch.zeros(w.numel, dtype=torch.int16, device="cuda"), global_offset=w.global_offset)
    b = np.zeros(w.numel, np.uint16)
    for step in range(w.first_step, w.first_step + w.commits):
        if step != w.first_step:
            g = wl.grad_host(w, step)
            sh.grad.copy_(torch.from_numpy(g))
        d_gpu = pk.to_u64(pk.adamw_commit(sh, step, g_hyper(hy)))[0]
        d_ref = oracle_commit_parallel(p, g, m, v, b, o_hyper(hy), step, w.global_offset)
        print(f"[{w.name}] step {step}: {d_gpu:#018x}", flush=True)
        assert d_gpu == d_ref, f"step {step}"
    for name, t, ref in (("param", sh.param, p), ("exp_avg", sh.exp_avg, m), ("exp_avg_sq", sh.exp_avg_sq, v)):
        assert_bitwise(name, host(t), ref)
    assert_bitwise("bf16", host(sh.param_bf16).view(np.uint16), b)


def test_mistral7b_whole_model_segments():
    """All 7,248,023,552 parameters of Mistral-7B as 291 per-tensor segments
    with per-segment hyperparameters (norms without decay, lm_head with beta2
    0.99): the 291 per-segment digests and their total, the 291 bf16 digests,
    and every element of the sampled chunks."""
    pk = _pk()
    w = wl.WORKLOADS["mistral7b_whole"]
    print(f"[{w.name}] filling the device", flush=True)
    sh = device_workload(w)
    got = pk.to_u64(pk.adamw_commit(sh, w.first_step))
    got_b = pk.to_u64(pk.bf16_digest(sh))
    print(f"[{w.name}] GPU total {got[-1]:#018x}; oracle streaming", flush=True)
    sample_every = 37  # chunks
    counter = {"k": 0, "checked": 0}

    def check(start, p, m, v, b):
        counter["k"] += 1
        if counter["k"] % sample_every:
            return
        sl = slice(start, start + p.size)
        assert_bitwise("param", host(sh.param[sl]), p)
        assert_bitwise("exp_avg", host(sh.exp_avg[sl]), m)
        assert_bitwise("exp_avg_sq", host(sh.exp_avg_sq[sl]), v)
        assert_bitwise("bf16", host(sh.param_bf16[sl]).view(np.uint16), b)
        counter["checked"] += p.size

    per, per_b = oracle_stream_segments(w, w.first_step, [o_hyper(h) for h in w.hypers], check=check)
    assert got[:-1] == per
    assert got[-1] == sum(per) & M64
    assert got_b[:-1] == per_b
    assert counter["checked"] > 0
    print(f"[{w.name}] {counter['checked']} elements compared one by one", flush=True)


def test_every_pattern_through_the_commit():
    """All 2^32 binary32 patterns as weights, with lr = 0, g = 0 and
    m = v = 0, so p' = p * 1 - 0: every non-NaN pattern comes back bit for
    bit (denormals, -0 and infinities included) and every NaN stays a NaN.
    The bf16 copy must be the RNE of the GPU's own p' (NaNs as the commit
    left them, so the check does not depend on how the arithmetic treats NaN
    payloads): compared through the bf16 digest against the oracle's
    conversion of those bits, chunk by chunk."""
    from concurrent.futures import ThreadPoolExecutor

    import torch

    from tests.helpers import host_threads

    pk = _pk()
    chunk = 1 << 30
    hz = pk.Hyper(lr=0.0, weight_decay=0.0)
    threads = host_threads()
    for start in range(0, 1 << 32, chunk):
        print(f"[all patterns] chunk at {start:#x}", flush=True)
        bits = torch.arange(start, start + chunk, dtype=torch.int64, device="cuda").to(torch.int32)
        p_before = bits.clone()
        p = bits.view(torch.float32)
        z = [torch.zeros(chunk, dtype=torch.float32, device="cuda") for _ in range(3)]
        b = torch.zeros(chunk, dtype=torch.int16, device="cuda")
        sh = pk.Shard(p, z[0], z[1], z[2], b, global_offset=start)
        pk.adamw_commit(sh, 1, hz)
        nan = (p_before & 0x7FFFFFFF) > 0x7F800000
        assert torch.equal(p.view(torch.int32)[~nan], p_before[~nan])
        assert bool(torch.isnan(p[nan]).all())
        assert not bool(z[1].view(torch.int32).any()) and not bool(z[2].view(torch.int32).any())
        got = pk.to_u64(pk.bf16_digest(sh))[0]
        hb = p.view(torch.int32).cpu().numpy().view(np.uint32)
        del p_before, nan, z, sh, b, bits, p
        torch.cuda.empty_cache()
        cuts = [chunk * k // threads for k in range(threads + 1)]

        def part(k):
            a, z_ = cuts[k], cuts[k + 1]
            return oracle.bf16_digest(oracle.bf16_rne_bits(hb[a:z_]), start + a)

        with ThreadPoolExecutor(threads) as ex:
            want = sum(ex.map(part, range(threads))) & M64
        assert got == want, f"chunk at {start:#x}"
        del hb
