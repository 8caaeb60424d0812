"""Benchmark: tree-shared decode + verify attention on one MI355X, against its roofline.

    python bench.py [--steps K] [--warmup W] [--workload mixed_serving] [--gpus 1] [--no-cpu]

The default workload is the mixed serving batch (32/8/128; decode and causal verify rows in one
launch, measured after 30% of the candidates were pruned and refilled); it is followed by the
beam-search decode, step-verification and speculative-explosion workloads, reported as sub-records.
(--workload kv_append times the K/V append kernel instead: all K/V writes of the spec_explosion
tree, deduplicated blocks skipped.  --workload cd_sample times one CD branching step of the
spec_explosion decode batch.  --workload verify_sweep and model_step are described below.)

A step is one tkv_decode (or tkv_verify) call over the whole batch: the shared-segment and
private-suffix contractions of every row, the verify rows' causal tiles and the log-sum-exp merge.
The block manager has built the tree, rows are coalesced and the plan is built and uploaded before
timing (host times are reported beside the result).  Inputs are resident in HBM when the timed
region starts; the K/V pool is rotated over several device copies so that no step finds it in the
256 MB Infinity Cache.  Prints one JSON line.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E
MFMA_BF16_PEAK_TFLOPS = 2500.0  # MI355X dense bf16
MALL_BYTES = 256 << 20


ATTN_SOURCES = ("attn.hip", "plan.cpp", "internal.h")


def kernel_sources_digest(files=ATTN_SOURCES):
    """sha256 over the sources that decide what a kernel does (for attention: kernels and planner)."""
    import hashlib
    h = hashlib.sha256()
    for f in files:
        with open(os.path.join(ROOT, "paper_2609_39334_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def measured_traffic(a, key, files):
    """HBM bytes per launch from the committed PMC summary, or None when the kernel's sources have
    changed since the counters were taken."""
    if not (a.traffic and os.path.exists(a.traffic)):
        return None
    with open(a.traffic) as f:
        tr = json.load(f).get(key)
    if tr and tr.get("sources_sha256") == kernel_sources_digest(files):
        return tr.get("bytes_per_launch")
    return None


def _args():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default="mixed_serving")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--no-cpu", action="store_true", help="skip the oracle CPU baseline")
    ap.add_argument("--no-sub-configs", action="store_true",
                    help="time only the headline workload (by default the mixed_serving headline is followed by "
                         "beam_decode, step_verify, spec_explosion and spec_prompts, reported under 'configs')")
    ap.add_argument("--cpu-seconds", type=float, default=15.0, help="target length of the CPU baseline sample")
    ap.add_argument("--no-decode-loop", action="store_true",
                    help="skip the decode-loop planning measurement (host_ms.decode_loop) of decode workloads, whose "
                         "own attention launches would otherwise follow the measured ones (profiling runs)")
    ap.add_argument("--kv-copies", type=int, default=0,
                    help="device copies of the K/V pool rotated over the steps (0: enough to defeat the 256 MB MALL)")
    ap.add_argument("--traffic", default=os.path.join(ROOT, "profiles", "traffic.json"),
                    help="JSON with per-launch HBM bytes of the main kernel from rocprofv3 counters (used only if "
                         "the kernel sources are unchanged since they were taken)")
    ap.add_argument("--plan-options", default=None,
                    help="placement options of the attention plan as JSON (tkv_plan_options fields), e.g. "
                         "'{\"wave_max_rows\": 8}'")
    ap.add_argument("--calib-copy", action="store_true",
                    help="run one plain 256 MiB device-to-device copy first (calibrates HBM byte counters)")
    return ap.parse_args()


def measure_copy_gbs(torch, dev, stream, nbytes=1 << 30, reps=10):
    """Bytes moved per second (read + write) by a plain device-to-device copy of nbytes: the streaming
    rate this machine reaches, reported beside the nominal 8 TB/s."""
    src = torch.empty(nbytes, dtype=torch.uint8, device=dev)
    dst = torch.empty_like(src)
    dst.copy_(src)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record(stream)
    for _ in range(reps):
        dst.copy_(src)
    e1.record(stream)
    torch.cuda.synchronize()
    return 2 * nbytes * reps / (e0.elapsed_time(e1) / 1e3) / 1e9


def measure_gemm_tflops(torch, dev, stream, n=8192, reps=20):
    """Flop rate of a plain n x n x n bf16 matrix product in the vendor library (torch.matmul), timed in
    the same process: the dense MFMA rate a tuned library reaches on this machine at the clock the chip
    sustains under MFMA load, reported beside the nominal 2.5 PFLOP/s."""
    a = torch.randn((n, n), dtype=torch.bfloat16, device=dev)
    b = torch.randn((n, n), dtype=torch.bfloat16, device=dev)
    c = torch.empty((n, n), dtype=torch.bfloat16, device=dev)
    for _ in range(3):
        torch.matmul(a, b, out=c)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record(stream)
    for _ in range(reps):
        torch.matmul(a, b, out=c)
    e1.record(stream)
    torch.cuda.synchronize()
    return 2.0 * n ** 3 * reps / (e0.elapsed_time(e1) / 1e3) / 1e12


def calibration_copy(torch, dev):
    """One plain 256 MiB device-to-device copy: a kernel of known size for the PMC byte counters."""
    src = torch.empty(256 << 20, dtype=torch.uint8, device=dev)
    dst = torch.empty_like(src)
    dst.copy_(src)
    torch.cuda.synchronize()


def bench_kv_append(a):
    """The K/V writes of a whole tree in one tkv_kv_append launch: every token of every extension of
    the spec_explosion script goes to the slot the block manager gave it, tokens of deduplicated
    blocks are skipped.  HBM-bound: each written token moves hkv * d bf16 of K and of V in and out."""
    import torch
    import paper_2609_39334_amd as tkv
    import workloads as W
    dev = torch.device("cuda:0")
    wl = W.spec_explosion(a.seed)
    s = wl.shape
    bm = tkv.BlockManager(wl.num_blocks, s.block_size, wl.max_seqs)
    dsts = []
    t0 = time.perf_counter()
    seq_of = []
    for e in wl.events:                   # replay the script, keeping each extension's slots
        if isinstance(e, W.Extend):
            parent = -1 if e.parent < 0 else seq_of[e.parent]
            seq, blk, hit = bm.extend(parent, e.tokens, e.seal)
            seq_of.append(seq)
            if len(e.tokens):
                dsts.append(tkv.tkv_extend_slots(blk, hit, len(e.tokens), s.block_size))
        elif isinstance(e, W.Prune):
            bm.prune(seq_of[e.handle])
    t_host = time.perf_counter() - t0
    dst = np.concatenate(dsts).astype(np.int32)
    n_tok, n_written = len(dst), int((dst >= 0).sum())
    rng = np.random.default_rng([a.seed, 5])
    new_bits = W.f32_to_bf16_bits(rng.standard_normal((2, n_tok, s.hkv, s.d), dtype=np.float32))

    def to_dev(x):
        return torch.from_numpy(np.ascontiguousarray(x).view(np.int16)).view(torch.bfloat16).to(dev)

    k_new, v_new = to_dev(new_bits[0]), to_dev(new_bits[1])
    d_dst = torch.from_numpy(dst).to(dev)
    k = torch.zeros((wl.num_blocks, s.hkv, s.block_size, s.d), dtype=torch.bfloat16, device=dev)
    v = torch.zeros_like(k)
    stream = torch.cuda.current_stream()
    if a.calib_copy:
        calibration_copy(torch, dev)
    for _ in range(a.warmup):
        tkv.tkv_kv_append(d_dst, k_new, v_new, k, v, stream)
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    ev0.record(stream)
    for _ in range(a.steps):
        tkv.tkv_kv_append(d_dst, k_new, v_new, k, v, stream)
    ev1.record(stream)
    torch.cuda.synchronize()
    ms_step = ev0.elapsed_time(ev1) / a.steps
    row = s.hkv * s.d * 2
    b_alg = n_written * row * 2 * 2 + n_tok * 4      # K and V read and written, plus the slots
    gbs = b_alg / (ms_step / 1e3) / 1e9
    cpu = None
    if not a.no_cpu:
        import oracle
        kh = np.zeros((wl.num_blocks, s.hkv, s.block_size, s.d), dtype=np.uint16)
        vh = np.zeros_like(kh)
        done, t_cpu = 0, 0.0
        while t_cpu < a.cpu_seconds and done < n_tok:
            e = min(n_tok, done + 20000)
            t0 = time.perf_counter()
            oracle.kv_append(kh, vh, dst[done:e], new_bits[0][done:e], new_bits[1][done:e])
            t_cpu += time.perf_counter() - t0
            done = e
        cpu = {"value": round(done / t_cpu, 1), "unit": "tokens/s", "cores": 1, "kind": "oracle",
               "sample": f"the first {done} of {n_tok} tokens, NumPy row scatter, {t_cpu:.1f} s"}
    out = {
        "metric": "kv-append tokens/s and % HBM roofline, tree K/V writes with deduplicated blocks skipped",
        "value": round(n_tok / (ms_step / 1e3), 1), "unit": "tokens/s", "n_gpus": 1, "steps": a.steps,
        "warmup": a.warmup, "ms_per_step": round(ms_step, 5), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic (spec_explosion tree, N(0,1) bf16 rows)",
        "config": {"workload": "kv_append", "tree": "spec_explosion", "hkv": s.hkv, "head_dim": s.d,
                   "block_size": s.block_size, "tokens": n_tok, "written_tokens": n_written,
                   "skipped_tokens": n_tok - n_written},
        "roofline": {"bound": "hbm", "achieved": round(gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(gbs / HBM_PEAK_GBS, 4),
                     "traffic": measured_traffic(a, "kv_append", ("kv_append.hip", "internal.h")), "kernel": "kv_append",
                     "algorithmic_bytes": b_alg, "kernel_us": round(ms_step * 1e3, 2)},
        "cpu_baseline": cpu,
        "host_ms": {"block_manager_and_slots": round(t_host * 1e3, 2)},
    }
    print(json.dumps(out))


def bench_cd_sample(a):
    """One CD branching step: the spec_explosion decode batch's distinct rows, each with its
    multiplicity as potential size, draw from synthetic logits over a 151,936-token vocabulary (the
    Qwen2.5 generators' vocabulary size) and group their draws.  HBM-bound on reading the logits."""
    import torch
    import paper_2609_39334_amd as tkv
    import workloads as W
    dev = torch.device("cuda:0")
    wl = W.spec_explosion(a.seed)
    bm = tkv.BlockManager(wl.num_blocks, wl.shape.block_size, wl.max_seqs)
    got = {}
    W.drive(wl, bm, on_launch=lambda i, l, c: got.setdefault("c", c))
    seqs = [x for x, _ in got["c"]]
    _, first, mult = bm.coalesce(seqs, [1] * len(seqs))
    n_rows, vocab, temperature = len(first), 151936, 0.8
    potential = np.asarray(mult, dtype=np.int64)
    off = np.concatenate([[0], np.cumsum(potential)]).astype(np.int32)
    rng = np.random.default_rng([a.seed, 6])
    logits = torch.empty((n_rows, vocab), dtype=torch.float32, device=dev)
    gen = torch.Generator(device=dev)
    gen.manual_seed(a.seed)
    logits.normal_(0.0, 2.0, generator=gen)
    u = torch.from_numpy(rng.random(int(off[-1]), dtype=np.float32)).to(dev)
    d_off = torch.from_numpy(off).to(dev)
    mp = int(potential.max())
    stream = torch.cuda.current_stream()
    if a.calib_copy:
        calibration_copy(torch, dev)
    for _ in range(a.warmup):
        tkv.tkv_cd_sample(logits, temperature, d_off, u, mp, stream)
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    ev0.record(stream)
    for _ in range(a.steps):
        tkv.tkv_cd_sample(logits, temperature, d_off, u, mp, stream)
    ev1.record(stream)
    torch.cuda.synchronize()
    ms_step = ev0.elapsed_time(ev1) / a.steps
    tok, cnt, ng = tkv.tkv_cd_sample(logits, temperature, d_off, u, mp, stream)
    torch.cuda.synchronize()
    n_groups = int(ng.sum().item())
    b_alg = n_rows * vocab * 4 + int(off[-1]) * (4 + 8) + (n_rows + 1) * 4 + n_rows * 4
    gbs = b_alg / (ms_step / 1e3) / 1e9
    cpu = None
    if not a.no_cpu:
        import oracle
        lg = logits.cpu().numpy()
        uh = u.cpu().numpy()
        done, t_cpu = 0, 0.0
        while t_cpu < a.cpu_seconds and done < n_rows:
            t0 = time.perf_counter()
            oracle.cd_sample.cd_sample(lg[done:done + 1], temperature, potential[done:done + 1], uh[off[done]:off[done + 1]])
            t_cpu += time.perf_counter() - t0
            done += 1
        cpu = {"value": round(done / t_cpu, 1), "unit": "rows/s", "cores": 1, "kind": "oracle",
               "sample": f"the first {done} of {n_rows} rows, NumPy float64 softmax and inverse CDF, {t_cpu:.1f} s"}
    out = {
        "metric": "CD branching rows/s and % HBM roofline (logits read once), one sampling step",
        "value": round(n_rows / (ms_step / 1e3), 1), "unit": "rows/s", "n_gpus": 1, "steps": a.steps,
        "warmup": a.warmup, "ms_per_step": round(ms_step, 5), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "fp32", "data": "synthetic (N(0, 2) fp32 logits, spec_explosion potentials)",
        "config": {"workload": "cd_sample", "rows": n_rows, "draws": int(off[-1]), "vocab": vocab,
                   "temperature": temperature, "max_potential": mp, "groups": n_groups},
        "roofline": {"bound": "hbm", "achieved": round(gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(gbs / HBM_PEAK_GBS, 4),
                     "traffic": measured_traffic(a, "cd_sample", ("cd_sample.hip", "internal.h")), "kernel": "cd_sample",
                     "algorithmic_bytes": b_alg, "kernel_us": round(ms_step * 1e3, 2)},
        "cpu_baseline": cpu,
    }
    print(json.dumps(out))


def bench_verify_sweep(a):
    """Verification throughput against batch size, the shape of the paper's verify-throughput
    microbenchmark (Sec. 4.3, from which it takes its 2,048-token flush threshold), for the attention
    layer of a 28/4/128 verifier (the head layout of a 7B reward model).  A batch is candidate steps
    U{32..256} in sibling groups of 4 under parent steps U{64..256} of a 1,024-token prompt, as lazy
    verification flushes them, filled up to T query tokens; each T is one tkv_verify call."""
    import torch
    import paper_2609_39334_amd as tkv
    import workloads as W
    dev = torch.device("cuda:0")
    hq, hkv, d, bs = 28, 4, 128, 16
    sizes = [256, 512, 1024, 2048, 4096, 8192, 16384]
    rng = np.random.default_rng([a.seed, 8])
    steps, total = [], 0
    while total < sizes[-1]:                      # the largest batch; each smaller one is a prefix of it
        parent = int(rng.integers(64, 257))
        for _ in range(4):
            if total == sizes[-1]:
                break
            edge = min(x for x in sizes if x > total)       # a step ends on every batch size
            n = min(int(rng.integers(32, 257)), edge - total)
            steps.append((len(steps) // 4, parent, n))
            total += n
    prompt = 1024
    nb = -(-prompt // bs) + sum(-(-p // bs) for p in {g: p for g, p, _ in steps}.values()) + \
        sum(-(-n // bs) for _, _, n in steps)
    bm = tkv.BlockManager(nb, bs, len(steps) + 64)
    root = bm.extend(-1, rng.integers(0, 1000, size=prompt).tolist(), True)[0]
    parents, seqs = {}, []
    for g, p, n in steps:
        if g not in parents:
            parents[g] = bm.extend(root, rng.integers(0, 1000, size=p).tolist(), True)[0]
        seqs.append(bm.extend(parents[g], rng.integers(0, 1000, size=n).tolist(), True)[0])
    bl = bm.block_len()
    kbits = W.f32_to_bf16_bits(rng.standard_normal((nb, hkv, bs, d), dtype=np.float32))
    vbits = W.f32_to_bf16_bits(rng.standard_normal((nb, hkv, bs, d), dtype=np.float32))

    def to_dev(x):
        return torch.from_numpy(np.ascontiguousarray(x).view(np.int16)).view(torch.bfloat16).to(dev)

    k0, v0 = to_dev(kbits), to_dev(vbits)
    n_copies = a.kv_copies or max(2, math.ceil(4 * MALL_BYTES / (4 * k0.numel())) + 1)
    ks = [k0] + [k0.clone() for _ in range(n_copies - 1)]
    vs = [v0] + [v0.clone() for _ in range(n_copies - 1)]
    stream = torch.cuda.current_stream()
    sweep, at_threshold = [], None
    for T in sizes:
        rows, acc = [], 0
        for i, (_, _, n) in enumerate(steps):
            if acc == T:
                break
            rows.append((seqs[i], n))
            acc += n
        assert acc == T
        tables = [bm.table(x) for x, _ in rows]
        q_lens = [n for _, n in rows]
        qi = np.concatenate([[0], np.cumsum(q_lens)]).astype(np.int32)
        ki = np.concatenate([[0], np.cumsum([len(t) for t in tables])]).astype(np.int32)
        plan = tkv.Plan((hq, hkv, d, bs, nb), qi, ki, np.concatenate(tables).astype(np.int32), bl, None, device=dev)
        st = plan.stats
        n_qtok = int(qi[-1])
        q = to_dev(W.f32_to_bf16_bits(rng.standard_normal((n_qtok, hq, d), dtype=np.float32)))
        o = torch.empty((n_qtok, hq, d), dtype=torch.bfloat16, device=dev)
        lse = torch.empty((n_qtok, hq), dtype=torch.float32, device=dev)
        reps = max(20, a.steps // 4)
        for i in range(a.warmup):
            plan.verify(q, ks[i % n_copies], vs[i % n_copies], o, lse, stream)
        ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        ev0.record(stream)
        for i in range(reps):
            plan.verify(q, ks[i % n_copies], vs[i % n_copies], o, lse, stream)
        ev1.record(stream)
        torch.cuda.synchronize()
        ms = ev0.elapsed_time(ev1) / reps
        tkv.tkv_plan_profile(plan.h, reps)
        for i in range(reps):
            plan.verify(q, ks[i % n_copies], vs[i % n_copies], o, lse, stream)
        torch.cuda.synchronize()
        n_rec, ms_main, ms_merge = tkv.tkv_plan_profile_read(plan.h)
        tkv.tkv_plan_profile(plan.h, 0)
        t_main = ms_main / max(1, n_rec) / 1e3
        b_uniq = st["uniq_kv_tokens"] * hkv * d * 2 * 2
        entry = {"tokens": n_qtok, "rows": len(rows), "us": round(ms * 1e3, 2), "tokens_per_s": round(n_qtok / (ms / 1e3), 1),
                 "attn_fwd_us": round(t_main * 1e6, 2), "tflops": round(st["flops"] / t_main / 1e12, 1),
                 "flops": st["flops"], "unique_kv_bytes": b_uniq}
        sweep.append(entry)
        if T == 2048:
            at_threshold = (entry, st, tables, q_lens, q, plan)
    best = max(e["tokens_per_s"] for e in sweep)
    saturation = next(e["tokens"] for e in sweep if e["tokens_per_s"] >= 0.9 * best)
    e, st, tables, q_lens, q, _ = at_threshold
    t_main = e["attn_fwd_us"] / 1e6
    mfma_bound = e["flops"] / e["unique_kv_bytes"] > MFMA_BF16_PEAK_TFLOPS * 1e12 / (HBM_PEAK_GBS * 1e9)
    if mfma_bound:
        ach = e["flops"] / t_main / 1e12
        roof = {"bound": "mfma", "achieved": round(ach, 2), "peak": MFMA_BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                "frac": round(ach / MFMA_BF16_PEAK_TFLOPS, 4), "traffic": None, "kernel": "attn_fwd",
                "algorithmic_flops": e["flops"], "kernel_us": e["attn_fwd_us"]}
    else:
        ach = e["unique_kv_bytes"] / t_main / 1e9
        roof = {"bound": "hbm", "achieved": round(ach, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(ach / HBM_PEAK_GBS, 4), "traffic": None, "kernel": "attn_fwd",
                "algorithmic_bytes": e["unique_kv_bytes"], "kernel_us": e["attn_fwd_us"]}
    cpu = None
    if not a.no_cpu:
        import oracle
        kf, vf = W.bf16_bits_to_f32(kbits), W.bf16_bits_to_f32(vbits)
        qf = W.bf16_bits_to_f32(q.view(torch.int16).cpu().numpy().view(np.uint16)).astype(np.float64)
        done_tok, t_cpu, r = 0, 0.0, 0
        while t_cpu < a.cpu_seconds and r < len(tables):
            t0 = time.perf_counter()
            oracle.attention(qf, kf, vf, tables, bl, q_lens, rows=[r])
            t_cpu += time.perf_counter() - t0
            done_tok += q_lens[r]
            r += 1
        cpu = {"value": round(done_tok / t_cpu, 2), "unit": "tokens/s", "cores": len(os.sched_getaffinity(0)),
               "kind": "oracle", "sample": f"the first {r} of {len(tables)} rows of the 2,048-token batch "
                                           f"({done_tok} query tokens), fp64 NumPy gather attention, {t_cpu:.1f} s"}
    out = {
        "metric": "verify tokens/s against batch tokens, attention layer (shape of the verify-throughput microbenchmark)",
        "value": e["tokens_per_s"], "unit": "tokens/s", "n_gpus": 1, "steps": max(20, a.steps // 4),
        "warmup": a.warmup, "ms_per_step": round(e["us"] / 1e3, 5), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic (sibling groups of candidate steps, N(0,1) bf16)",
        "config": {"workload": "verify_sweep", "hq": hq, "hkv": hkv, "head_dim": d, "batch_tokens": 2048,
                   "prompt": prompt, "kv_pool_copies_rotated": n_copies},
        "roofline": roof,
        "cpu_baseline": cpu,
        "sweep": sweep,
        "saturation_tokens": saturation,
    }
    print(json.dumps(out))


def bench_model_step(a):
    """One decode step of a whole model with synthetic weights: the Qwen2.5-7B layer layout (28 layers,
    28/4 heads of 128) over the spec_explosion batch's distinct rows, each with its multiplicity as
    potential size.  Per step: 28 x (GEMMs, K/V append, tree attention) + logits + CD sampling.  Dense
    GEMMs run in hipBLASLt (torch.mm); attention, K/V append and sampling are the library's kernels."""
    import torch
    import paper_2609_39334_amd as tkv
    import workloads as W
    from paper_2609_39334_amd.model import QWEN25_7B, SyntheticDecoder
    dev = torch.device("cuda:0")
    ms_ = QWEN25_7B
    wl = W.spec_explosion(a.seed)
    bs = wl.shape.block_size
    got = {}
    bm = tkv.BlockManager(wl.num_blocks + 4096, bs, wl.max_seqs)
    W.drive(wl, bm, on_launch=lambda i, l, c: got.setdefault("c", c))
    seqs = [x for x, _ in got["c"]]
    _, first, mult = bm.coalesce(seqs, [1] * len(seqs))
    rows = len(first)
    rng = np.random.default_rng([a.seed, 9])
    tokens = rng.integers(0, ms_.vocab, rows)
    dst = np.array([int(bm.append(seqs[f], [int(t)])[0]) for f, t in zip(first, tokens)], dtype=np.int32)
    tables = [bm.table(seqs[f]) for f in first]
    bl = bm.block_len()
    nb = len(bl)
    positions = np.array([int(bl[t].sum()) - 1 for t in tables], dtype=np.int64)
    qi = np.arange(rows + 1, dtype=np.int32)
    ki = np.concatenate([[0], np.cumsum([len(t) for t in tables])]).astype(np.int32)
    t0 = time.perf_counter()
    plan = tkv.Plan((ms_.hq, ms_.hkv, ms_.d, bs, nb), qi, ki, np.concatenate(tables).astype(np.int32), bl, mult,
                    device=dev)
    torch.cuda.synchronize()
    t_plan = time.perf_counter() - t0
    st = plan.stats
    model = SyntheticDecoder(ms_, dev, a.seed)
    g = torch.Generator(device=dev)
    g.manual_seed(a.seed)
    k_pools = [torch.empty((nb, ms_.hkv, bs, ms_.d), dtype=torch.bfloat16, device=dev).normal_(generator=g)
               for _ in range(ms_.layers)]
    v_pools = [torch.empty_like(k_pools[0]).normal_(generator=g) for _ in range(ms_.layers)]
    d_tok = torch.from_numpy(tokens).to(dev)
    d_pos = torch.from_numpy(positions).to(dev)
    d_dst = torch.from_numpy(dst).to(dev)
    off = np.concatenate([[0], np.cumsum(mult)]).astype(np.int32)
    d_off = torch.from_numpy(off).to(dev)
    u = torch.from_numpy(rng.random(int(off[-1]), dtype=np.float32)).to(dev)
    mp = int(max(mult))
    stream = torch.cuda.current_stream()

    def step():
        logits = model.step(d_tok, d_pos, d_dst, plan, k_pools, v_pools, stream)
        return model.sample(logits, 0.8, d_off, u, mp, stream)

    for _ in range(a.warmup):
        step()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    ev0.record(stream)
    for _ in range(a.steps):
        step()
    ev1.record(stream)
    torch.cuda.synchronize()
    ms_step = ev0.elapsed_time(ev1) / a.steps
    # the library's share: attention (plan events around each call), then K/V append and sampling alone
    tkv.tkv_plan_profile(plan.h, ms_.layers * a.steps)
    for _ in range(a.steps):
        step()
    torch.cuda.synchronize()
    n_rec, ms_main, ms_merge = tkv.tkv_plan_profile_read(plan.h)
    tkv.tkv_plan_profile(plan.h, 0)
    attn_ms = (ms_main + ms_merge) / max(1, n_rec) * ms_.layers
    knew = torch.zeros((rows, ms_.hkv, ms_.d), dtype=torch.bfloat16, device=dev)
    logits = torch.zeros((rows, ms_.vocab), dtype=torch.float32, device=dev)
    ev0.record(stream)
    for _ in range(a.steps):
        for li in range(ms_.layers):
            tkv.tkv_kv_append(d_dst, knew, knew, k_pools[li], v_pools[li], stream)
    ev1.record(stream)
    torch.cuda.synchronize()
    append_ms = ev0.elapsed_time(ev1) / a.steps
    ev0.record(stream)
    for _ in range(a.steps):
        model.sample(logits, 0.8, d_off, u, mp, stream)
    ev1.record(stream)
    torch.cuda.synchronize()
    sample_ms = ev0.elapsed_time(ev1) / a.steps
    gemm_flops = 2 * rows * (ms_.layers * (ms_.hidden * (ms_.hq + 2 * ms_.hkv) * ms_.d + ms_.hq * ms_.d * ms_.hidden
                                           + ms_.hidden * 2 * ms_.inter + ms_.inter * ms_.hidden)
                             + ms_.hidden * ms_.vocab)
    flops = gemm_flops + ms_.layers * st["flops"]
    ach = flops / (ms_step / 1e3) / 1e12
    logical = int(off[-1])
    out = {
        "metric": "candidate-tokens/s of a whole decode step (28-layer 7B layout, synthetic weights) and MFMA roofline",
        "value": round(logical / (ms_step / 1e3), 1), "unit": "candidate-tokens/s", "n_gpus": 1, "steps": a.steps,
        "warmup": a.warmup, "ms_per_step": round(ms_step, 4), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic (random-init weights, spec_explosion tree, N(0,1) K/V)",
        "config": {"workload": "model_step", "layers": ms_.layers, "hidden": ms_.hidden, "hq": ms_.hq, "hkv": ms_.hkv,
                   "head_dim": ms_.d, "intermediate": ms_.inter, "vocab": ms_.vocab, "rows": rows,
                   "candidates": logical, "tree": "spec_explosion"},
        "roofline": {"bound": "mfma", "achieved": round(ach, 1), "peak": MFMA_BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                     "frac": round(ach / MFMA_BF16_PEAK_TFLOPS, 4), "traffic": None,
                     "kernel": "whole step (hipBLASLt GEMMs + library kernels)", "algorithmic_flops": flops,
                     "kernel_us": round(ms_step * 1e3, 1)},
        "cpu_baseline": None,
        "breakdown_ms": {"attention (28 calls, library)": round(attn_ms, 3),
                         "kv_append (28 calls, library)": round(append_ms, 3),
                         "cd_sample (library)": round(sample_ms, 3),
                         "rest: GEMMs, norms, RoPE, SiLU": round(ms_step - attn_ms - append_ms - sample_ms, 3)},
        "host_ms": {"plan_and_upload": round(t_plan * 1e3, 2)},
    }
    print(json.dumps(out))


def cpu_baseline(a, qbits, kbits, vbits, tables, bl, q_lens):
    """The oracle (fp64 NumPy gather attention, as it stands) on a bounded, seeded sample of the
    batch's rows, on the host's cores: sub-batches of rows in parallel threads (BLAS one thread
    each), submitted in seeded order until about `a.cpu_seconds` of wall time.  Rows are
    independent, so a sub-batch computes what the whole batch would for its rows."""
    from concurrent.futures import FIRST_COMPLETED, ThreadPoolExecutor, wait
    from threadpoolctl import threadpool_limits
    import oracle
    import workloads as W
    threads = max(1, min(16, len(os.sched_getaffinity(0))))
    kf, vf = W.bf16_bits_to_f32(kbits), W.bf16_bits_to_f32(vbits)
    qoff = np.concatenate([[0], np.cumsum(q_lens)]).astype(np.int64)
    order = np.random.default_rng(0).permutation(len(tables))
    per_sub = 4
    subs = [order[i:i + per_sub].tolist() for i in range(0, len(order), per_sub)]

    def run(sub):
        idx = np.concatenate([np.arange(qoff[r], qoff[r + 1]) for r in sub])
        qs = W.bf16_bits_to_f32(qbits[idx]).astype(np.float64)
        oracle.attention(qs, kf, vf, [tables[r] for r in sub], bl, [q_lens[r] for r in sub])
        return len(idx), len(sub)

    done_tok = done_rows = n_sub = 0
    with threadpool_limits(1):
        with ThreadPoolExecutor(threads) as ex:
            t0, c0 = time.perf_counter(), time.process_time()
            pending = set()
            k = 0
            while True:
                while len(pending) < threads and time.perf_counter() - t0 < a.cpu_seconds:
                    pending.add(ex.submit(run, subs[k % len(subs)]))
                    k += 1
                if not pending:
                    break
                fin, pending = wait(pending, return_when=FIRST_COMPLETED)
                for f in fin:
                    nt, nr = f.result()
                    done_tok += nt
                    done_rows += nr
                    n_sub += 1
            wall, cpu_s = time.perf_counter() - t0, time.process_time() - c0
    return {"value": round(done_tok / wall, 2), "unit": "candidate-tokens/s", "cores": threads, "kind": "oracle",
            "effective_cores": round(cpu_s / wall, 2), "host_cpus": len(os.sched_getaffinity(0)),
            "sample": f"{done_rows} row evaluations ({done_tok} query tokens) of this batch's {len(tables)} rows in "
                      f"seeded order, {n_sub} sub-batches of {per_sub} rows on {threads} threads (BLAS 1 thread "
                      f"each), fp64 NumPy gather attention, {wall:.1f} s wall, {cpu_s:.1f} s CPU"}


def shared_pass_flops(view, s):
    """Algorithmic flops of the shared-prefix pass: the 128-row tile items over shared chunks (item
    kind 0), each query token counted against the chunk keys its causal limit lets it see."""
    items = view["items"].reshape(-1, 8).astype(np.int64)
    toks = view["toks"].reshape(-1, 4).astype(np.int64)
    blen = view["blks"].reshape(-1, 2)[:, 1].astype(np.int64)
    g = s.hq // s.hkv
    cum = np.concatenate([[0], np.cumsum(blen)])
    total = 0
    for kvh, to, nt, bo, nb, pos0, kind, _ in items:
        if kind != 0:
            continue
        keys = cum[bo + nb] - cum[bo]
        vis = np.clip(toks[to:to + nt, 1] - pos0 + 1, 0, keys)
        total += int(vis.sum())
    return total * g * 4 * s.d


def time_plan_updates(wl, steps=48, seed=0, device=None):
    """Cost of a decode loop's planning: the workload's measured launch on a block manager with
    room to grow, then decode steps (one token more for every candidate, a new block when its last
    is full), each followed by tkv_plan_update of one plan.  `steps` steps time the update alone on
    the host; a fresh tkv_plan_create of the same tables is timed every eighth step for comparison.
    With a device, two more passes of `steps` // 2 steps run the loop as a decode loop would: update,
    upload, decode on random K/V, wait; once uploading into the same workspace (after an in-place
    update only the changed descriptor words go), once alternating two workspaces (the whole image
    each time).  Their per-step wall times are reported."""
    import paper_2609_39334_amd as tkv
    import workloads as W
    s = wl.shape
    nb = wl.num_blocks + 16384
    bm = tkv.BlockManager(nb, s.block_size, wl.max_seqs)
    cap = {}
    W.drive(wl, bm, on_launch=lambda i, l, c: cap.__setitem__(i, (l, c)))
    _, cands = cap[len(wl.launches) - 1]
    seqs = [x for x, _ in cands]
    qls = [q for _, q in cands]
    _, first, mult = bm.coalesce(seqs, qls)
    rows = [seqs[c] for c in first]
    qi = np.concatenate([[0], np.cumsum([qls[c] for c in first])]).astype(np.int32)
    shape = (s.hq, s.hkv, s.d, s.block_size, nb)
    rng = np.random.default_rng(seed)

    def grow():
        for x in rows:
            bm.append(x, rng.integers(0, 1 << 15, 1).astype(np.int32))
        t = [bm.table(x) for x in rows]
        return (np.concatenate([[0], np.cumsum([len(x) for x in t])]).astype(np.int32),
                np.concatenate(t).astype(np.int32), bm.block_len())

    h = tkv.tkv_plan_create(shape, qi, *grow(), mult)
    t_upd, in_place, t_create = [], 0, []
    try:
        for k in range(steps):
            ki, kb, bl = grow()
            t0 = time.perf_counter()
            in_place += tkv.tkv_plan_update(h, ki, kb, bl)
            t_upd.append(time.perf_counter() - t0)
            if k % 8 == 0:
                t0 = time.perf_counter()
                h2 = tkv.tkv_plan_create(shape, qi, ki, kb, bl, mult)
                t_create.append(time.perf_counter() - t0)
                tkv.tkv_plan_destroy(h2)
        res = {"decode_steps": steps, "plan_update_median": round(float(np.median(t_upd)) * 1e3, 4),
               "plan_update_mean": round(float(np.mean(t_upd)) * 1e3, 4), "updates_in_place": in_place,
               "plan_create_median_same_tables": round(float(np.median(t_create)) * 1e3, 3)}
        if device is not None:
            import torch
            stream = torch.cuda.current_stream()
            kd = torch.randn((nb, s.hkv, s.block_size, s.d), dtype=torch.bfloat16, device=device)
            vd = torch.randn((nb, s.hkv, s.block_size, s.d), dtype=torch.bfloat16, device=device)
            n_q = int(qi[-1])
            qd = torch.randn((n_q, s.hq, s.d), dtype=torch.bfloat16, device=device)
            od = torch.empty((n_q, s.hq, s.d), dtype=torch.bfloat16, device=device)
            loop = {}
            for mode in ("changed_words", "whole_image"):
                wss = [torch.empty(2 * tkv.tkv_plan_workspace_bytes(h), dtype=torch.uint8, device=device)
                       for _ in range(2)]
                tkv.tkv_plan_upload(h, wss[0], stream)
                t_u, t_l, t_w, n_ip = [], [], [], 0
                for k in range(steps // 2):
                    ki, kb, bl = grow()
                    torch.cuda.synchronize()
                    t0 = time.perf_counter()
                    n_ip += tkv.tkv_plan_update(h, ki, kb, bl)
                    t1 = time.perf_counter()
                    ws = wss[0] if mode == "changed_words" else wss[k % 2]
                    if tkv.tkv_plan_workspace_bytes(h) > ws.numel():
                        break           # a plan made again grew past the workspaces: stop the pass
                    tkv.tkv_plan_upload(h, ws, stream)
                    t2 = time.perf_counter()
                    tkv.tkv_decode(h, qd, kd, vd, od, None, stream)
                    torch.cuda.synchronize()
                    t3 = time.perf_counter()
                    t_u.append(t1 - t0)
                    t_l.append(t2 - t1)
                    t_w.append(t3 - t0)
                loop[mode] = {"steps": len(t_w), "in_place": n_ip, "update_us": round(float(np.median(t_u)) * 1e6, 1),
                              "upload_call_us": round(float(np.median(t_l)) * 1e6, 1),
                              "step_wall_us": round(float(np.median(t_w)) * 1e6, 1)}
            img, _ = tkv.tkv_plan_image(h)
            loop["image_bytes"] = len(img)
            res["loop_update_upload_decode"] = loop
            del kd, vd, qd, od
    finally:
        tkv.tkv_plan_destroy(h)
    return res


def run_attention(a, name, steps, warmup, with_cpu=False, warm=True):
    """Build the workload's tree on the library's block manager, coalesce and plan its measured
    launch, and time `steps` calls after `warmup` ones.  Returns the result fields."""
    import torch
    import paper_2609_39334_amd as tkv
    import workloads as W
    dev = torch.device("cuda:0")
    wl = W.CONFIGS[name](a.seed)
    s = wl.shape
    launch = len(wl.launches) - 1            # the last launch is the measured one (mixed: after prune)

    # ------------------------------------------------------------------ host side: tree, rows, plan
    t0 = time.perf_counter()
    bm = tkv.BlockManager(wl.num_blocks, s.block_size, wl.max_seqs)
    cap = {}
    W.drive(wl, bm, on_launch=lambda i, l, c: cap.__setitem__(i, (l, c)))
    t_bm = time.perf_counter() - t0
    L, cands = cap[launch]
    seqs = [x for x, _ in cands]
    qls = [q for _, q in cands]
    t0 = time.perf_counter()
    _, first, mult = bm.coalesce(seqs, qls)
    t_coal = time.perf_counter() - t0
    tables = [bm.table(seqs[c]) for c in first]
    q_lens = [qls[c] for c in first]
    bl = bm.block_len()
    qi = np.concatenate([[0], np.cumsum(q_lens)]).astype(np.int32)
    ki = np.concatenate([[0], np.cumsum([len(t) for t in tables])]).astype(np.int32)
    kb = np.concatenate(tables).astype(np.int32)
    n_qtok = int(qi[-1])
    t_create = []                              # the host planner alone (what a decode loop pays per step)
    for _ in range(5):
        t0 = time.perf_counter()
        h = tkv.tkv_plan_create_ex((s.hq, s.hkv, s.d, s.block_size, wl.num_blocks), qi, ki, kb, bl, mult,
                                   json.loads(a.plan_options) if a.plan_options else None)
        t_create.append(time.perf_counter() - t0)
        tkv.tkv_plan_destroy(h)
    t0 = time.perf_counter()
    options = json.loads(a.plan_options) if a.plan_options else None
    plan = tkv.Plan((s.hq, s.hkv, s.d, s.block_size, wl.num_blocks), qi, ki, kb, bl, mult, device=dev,
                    options=options)
    torch.cuda.synchronize()
    t_plan = time.perf_counter() - t0
    st = plan.stats
    f_shared = shared_pass_flops(plan.view(), s)

    # ------------------------------------------------------------------ device inputs
    kbits, vbits = wl.kv_values()
    qbits = wl.q_values(launch, n_qtok)

    def to_dev(x):
        return torch.from_numpy(x.view(np.int16)).view(torch.bfloat16).to(dev)

    k0, v0 = to_dev(kbits), to_dev(vbits)
    pool_bytes = 2 * k0.numel() * 2
    n_copies = a.kv_copies or max(2, math.ceil(4 * MALL_BYTES / pool_bytes) + 1)
    ks = [k0] + [k0.clone() for _ in range(n_copies - 1)]
    vs = [v0] + [v0.clone() for _ in range(n_copies - 1)]
    q = to_dev(qbits)
    o = torch.empty((n_qtok, s.hq, s.d), dtype=torch.bfloat16, device=dev)
    lse = torch.empty((n_qtok, s.hq), dtype=torch.float32, device=dev)
    stream = torch.cuda.current_stream()
    call = plan.decode if L.decode else plan.verify

    if a.calib_copy:
        calibration_copy(torch, dev)
    for i in range(warmup):
        call(q, ks[i % n_copies], vs[i % n_copies], o, lse, stream)
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    ev0.record(stream)
    for i in range(steps):                   # the timed steps: nothing else on the stream
        call(q, ks[i % n_copies], vs[i % n_copies], o, lse, stream)
    ev1.record(stream)
    torch.cuda.synchronize()
    ms_step = ev0.elapsed_time(ev1) / steps
    # kernel durations from the library's own events (dispatch-packet timestamps on the launch
    # stream around the attention kernel and around the merge), in a second pass of the same steps
    tkv.tkv_plan_profile(plan.h, steps)
    for i in range(steps):
        call(q, ks[i % n_copies], vs[i % n_copies], o, lse, stream)
    torch.cuda.synchronize()
    n_rec, ms_main, ms_merge = tkv.tkv_plan_profile_read(plan.h)
    tkv.tkv_plan_profile(plan.h, 0)
    t_main = ms_main / max(1, n_rec) / 1e3
    t_merge = ms_merge / max(1, n_rec) / 1e3 if st["n_merge"] else 0.0

    ms_step_warm = None
    if warm:  # the same steps on one pool copy, which then stays in the 256 MB Infinity Cache when it fits
        for _ in range(warmup):
            call(q, ks[0], vs[0], o, lse, stream)
        torch.cuda.synchronize()
        ev0.record(stream)
        for _ in range(steps):
            call(q, ks[0], vs[0], o, lse, stream)
        ev1.record(stream)
        torch.cuda.synchronize()
        ms_step_warm = ev0.elapsed_time(ev1) / steps
    del ks, vs, k0, v0, q, o, lse, plan
    torch.cuda.empty_cache()

    # ------------------------------------------------------------------ accounting
    b_uniq = st["uniq_kv_tokens"] * s.hkv * s.d * 2 * 2            # K and V, bf16
    flops = st["flops"]
    t_call = ms_step / 1e3
    traffic = measured_traffic(a, name, ATTN_SOURCES)
    kernel = "attn_fwd"  # tile items and the wave grid in one launch (attn_tile8 for small verify plans)
    # the bound is the one the work's arithmetic intensity puts it under (ridge: peak flop/s over
    # peak bytes/s); decode is HBM-bound, multi-token verify of long steps is MFMA-bound
    mfma_bound = flops / b_uniq > MFMA_BF16_PEAK_TFLOPS * 1e12 / (HBM_PEAK_GBS * 1e9)
    if mfma_bound:
        achieved = flops / t_main / 1e12
        roof = {"bound": "mfma", "achieved": round(achieved, 2), "peak": MFMA_BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                "frac": round(achieved / MFMA_BF16_PEAK_TFLOPS, 4), "traffic": traffic, "kernel": kernel,
                "algorithmic_flops": flops, "kernel_us": round(t_main * 1e6, 2),
                "frac_whole_call": round(flops / t_call / 1e12 / MFMA_BF16_PEAK_TFLOPS, 4)}
    else:
        achieved = b_uniq / t_main / 1e9
        roof = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": traffic, "kernel": kernel,
                "algorithmic_bytes": b_uniq, "kernel_us": round(t_main * 1e6, 2),
                "frac_whole_call": round(b_uniq / t_call / 1e9 / HBM_PEAK_GBS, 4)}
    shared = {"flops": f_shared, "frac_of_mfma_peak_over_attn_fwd": round(f_shared / t_main / 1e12 / MFMA_BF16_PEAK_TFLOPS, 4)}
    res = {
        "value": round(n_qtok / t_call, 1), "ms_per_step": round(ms_step, 5), "steps": steps, "warmup": warmup,
        "shared_pass": shared,
        "config": {"workload": name, "hq": s.hq, "hkv": s.hkv, "head_dim": s.d, "block_size": s.block_size,
                   "rows": st["n_rows"], "query_tokens": n_qtok, "logical_candidate_tokens": st["logical_qtok"],
                   "decode": bool(L.decode), "unique_kv_bytes": b_uniq,
                   "per_row_kv_bytes": st["path_kv_tokens"] * s.hkv * s.d * 4,
                   "algorithmic_flops": flops, "kv_pool_copies_rotated": n_copies},
        "roofline": roof,
        "hbm_frac_whole_call": round(b_uniq / t_call / 1e9 / HBM_PEAK_GBS, 4),
        "mfma_frac_whole_call": round(flops / t_call / 1e12 / MFMA_BF16_PEAK_TFLOPS, 4),
        "logical_candidate_tokens_per_s": round(st["logical_qtok"] / t_call, 1),
        "kernel_us": {kernel: round(t_main * 1e6, 2), "merge_partials": round(t_merge * 1e6, 2)},
        "plan": {"items": st["n_items"], "shared_items": st["n_items_shared"], "row_items": st["n_items_row"],
                 "wave_items": st["n_items_wave"], "waves": st["n_waves"],
                 "partial_slots": st["n_slots"], "merged_tokens": st["n_merge"], "segments": st["n_segments"],
                 "shared_segments": st["n_shared_segments"]},
        "host_ms": {"block_manager": round(t_bm * 1e3, 2), "coalesce": round(t_coal * 1e3, 3),
                    "plan_create_median": round(sorted(t_create)[2] * 1e3, 3),
                    "first_plan_with_workspace_and_upload": round(t_plan * 1e3, 2)},
    }
    if ms_step_warm is not None:
        res["warm"] = {"ms_per_step": round(ms_step_warm, 5), "value": round(n_qtok / (ms_step_warm / 1e3), 1),
                       "kv_pool_fits_mall": pool_bytes <= MALL_BYTES}
    if L.decode and not a.no_decode_loop:
        res["host_ms"]["decode_loop"] = time_plan_updates(wl, device=dev)
    if with_cpu:
        res["cpu_baseline"] = cpu_baseline(a, qbits, kbits, vbits, tables, bl, q_lens)
    return res


SUB_CONFIGS = ("beam_decode", "step_verify", "spec_explosion", "spec_prompts")


def main():
    a = _args()
    if a.gpus != 1:
        print(json.dumps({"error": "this build runs on one GPU; --gpus N with N > 1 is not supported "
                                   "(the path shards by query tree with no exchange, see DESIGN.md)"}))
        sys.exit(2)
    import torch

    if not torch.cuda.is_available():
        print(json.dumps({"error": "no GPU"}))
        sys.exit(1)
    if a.workload == "kv_append":
        return bench_kv_append(a)
    if a.workload == "cd_sample":
        return bench_cd_sample(a)
    if a.workload == "verify_sweep":
        return bench_verify_sweep(a)
    if a.workload == "model_step":
        return bench_model_step(a)
    import paper_2609_39334_amd as tkv
    tkv.lib()                                  # fails loudly if the HIP library is missing
    head = run_attention(a, a.workload, a.steps, a.warmup, with_cpu=not a.no_cpu)
    torch.cuda.synchronize()
    stream_gbs = measure_copy_gbs(torch, torch.device("cuda:0"), torch.cuda.current_stream())
    gemm_tflops = measure_gemm_tflops(torch, torch.device("cuda:0"), torch.cuda.current_stream())
    out = {
        "metric": "candidate-tokens/s and % HBM roofline (unique KV bytes), tree decode + verify",
        "value": head["value"],
        "unit": "candidate-tokens/s",
        "n_gpus": 1, "steps": a.steps, "warmup": a.warmup,
        "ms_per_step": head["ms_per_step"],
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16", "data": "synthetic (seeded trees, N(0,1) bf16 values)",
        "config": dict(head["config"], **({"plan_options": json.loads(a.plan_options)} if a.plan_options else {})),
        "roofline": head["roofline"],
        "cpu_baseline": head.get("cpu_baseline"),
        "hbm_frac_whole_call": head["hbm_frac_whole_call"],
        "mfma_frac_whole_call": head["mfma_frac_whole_call"],
        "stream_copy_gbs": round(stream_gbs, 1),
        "unique_kv_frac_of_stream_copy": round(head["config"]["unique_kv_bytes"] / (head["kernel_us"]["attn_fwd"] / 1e6)
                                               / 1e9 / stream_gbs, 4),
        "gemm_bf16_tflops": round(gemm_tflops, 1),
        "mfma_achieved_frac_of_gemm": (round(head["roofline"]["achieved"] / gemm_tflops, 4)
                                       if head["roofline"]["bound"] == "mfma" else None),
        "logical_candidate_tokens_per_s": head["logical_candidate_tokens_per_s"],
        "kernel_us": head["kernel_us"], "shared_pass": head["shared_pass"], "plan": head["plan"],
        "host_ms": head["host_ms"],
    }
    if "warm" in head:
        out["warm"] = head["warm"]
    if not a.no_sub_configs and a.workload == "mixed_serving":
        subs = {}
        for name in SUB_CONFIGS:       # the other workloads, each timed the same way (no CPU baseline)
            r = run_attention(a, name, max(a.steps, 100), max(a.warmup, 10), warm=False)
            subs[name] = {"value": r["value"], "ms_per_step": r["ms_per_step"], "steps": r["steps"],
                          "rows": r["config"]["rows"], "query_tokens": r["config"]["query_tokens"],
                          "roofline": {k: r["roofline"][k] for k in ("bound", "achieved", "unit", "frac",
                                                                     "frac_whole_call", "kernel_us", "traffic")},
                          "kernel_us": r["kernel_us"], "shared_pass": r["shared_pass"],
                          "plan_create_ms": r["host_ms"]["plan_create_median"]}
            if "decode_loop" in r["host_ms"]:
                subs[name]["decode_loop_host_ms"] = r["host_ms"]["decode_loop"]
        out["configs"] = subs
    print(json.dumps(out))


if __name__ == "__main__":
    main()
