"""Decode-attention benchmark on the long-tail rollout batch (one MI355X).

One step = the whole hot path for one decode step of the batch: host plan
(length-aware split-K, written to pinned memory that the kernels read in
place) -> attention kernel -> LSE combine. Inputs (q, paged K/V pools, block
table) are resident in HBM before timing. Before its timed steps each leg may
time the plan's group-parity skew candidates (untimed calibration).

    python bench.py [--steps K] [--warmup W] [--gpus 1]

Prints one JSON line. value = algorithmic KV bytes per step / step time.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "decode-attn achieved HBM GB/s (% of peak) + seq-steps/s on long-tail batch"
PEAK_HBM_GBPS = 8000.0
COUNTERS_FILE = os.path.join(ROOT, "profiles", "attn_longtail_counters.json")
KERNEL_SRC = os.path.join(ROOT, "paper_2601_12784_amd", "csrc", "decode_attn.hip")


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def kernel_source_hash(path=None) -> str:
    return hashlib.sha256(open(path or KERNEL_SRC, "rb").read()).hexdigest()[:16]


class Stepper:
    """Runs plan -> upload -> attention (+ merge) for a fixed batch on one stream."""

    def __init__(self, batch, chunk_pages=0, workers_per_cu=0, fp8=None, rotate=1, skew=0):
        """fp8 = (k8, v8, k_scale, v_scale) device tensors: step over that fp8
        cache instead of the batch's bf16 pools. rotate > 1 keeps that many
        device copies of the pools and moves to the next copy every step, so a
        batch smaller than the 256 MB last-level cache is still read from HBM."""
        import torch
        from paper_2601_12784_amd import binding as B
        self.torch = torch
        self.batch = batch
        self.fp8 = None if fp8 is None else (fp8[2], fp8[3])
        k, v = (batch.k_pool.cuda(), batch.v_pool.cuda()) if fp8 is None else (fp8[0], fp8[1])
        self.dev = dict(q=batch.q.cuda(), k=k, v=v, bt=torch.from_numpy(batch.block_table).cuda())
        self.pools = [(k, v)] + [(k.clone(), v.clone()) for _ in range(rotate - 1)]
        self.turn = 0
        self.lens = np.ascontiguousarray(batch.seq_lens, dtype=np.int32)
        self.chunk = chunk_pages or None
        cus = torch.cuda.get_device_properties(0).multi_processor_count
        self.cus = cus
        self.workers_per_cu = workers_per_cu
        self.runner = self.make_runner(skew)
        self.stream = torch.cuda.Stream()  # default priority
        self.out = torch.empty((batch.num_seqs, batch.num_q_heads, batch.head_dim), dtype=torch.float32,
                               device="cuda")
        self.lse = torch.empty((batch.num_seqs, batch.num_q_heads), dtype=torch.float32, device="cuda")
        self.step()
        self.info0 = self.runner.last_info

    def make_runner(self, skew):
        from paper_2601_12784_amd import binding as B
        b = self.batch
        return B.DecodeAttention(b.num_q_heads, b.num_kv_heads, b.head_dim,
                                 opts=B.make_opts(num_cus=self.cus, workers_per_cu=self.workers_per_cu,
                                                  xcd_parity_skew=skew))

    def step(self, ev_attn=None):
        """One decode step; ev_attn = (start, end) events bracketing the attention kernel."""
        d = self.dev
        k, v = self.pools[self.turn]
        self.turn = (self.turn + 1) % len(self.pools)
        self.runner(d["q"], k, v, d["bt"], self.lens, self.batch.scale, out=self.out, lse=self.lse,
                    chunk_pages=self.chunk, stream=self.stream, attn_events=ev_attn, fp8=self.fp8)


EVENT_EVERY = 16  # timing events take the attention kernel of every 16th timed step


def time_steps(stepper, steps, warmup, every=EVENT_EVERY):
    """Times `steps` decode steps after `warmup` untimed ones.
    Returns (wall ms per step, mean and median attention-kernel ms from HIP
    events). The events take the kernel's own start and end times (the
    library launches it with them, so no queue time is counted) on every
    `every`-th timed step only, which keeps whatever a timed dispatch costs
    off the other steps."""
    torch = stepper.torch
    sampled = range(0, steps, max(1, every))
    evs = {i: (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for i in sampled}
    for a, b in evs.values():           # torch creates an event on its first record: not in the timed region
        a.record(stepper.stream)
        b.record(stepper.stream)
    for _ in range(warmup):
        stepper.step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(steps):
        stepper.step(evs.get(i))
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    attn_ms = [a.elapsed_time(b) for a, b in evs.values()]
    return wall / steps * 1e3, float(np.mean(attn_ms)), float(np.median(attn_ms))


SKEW_CANDIDATES = (-40, -20, 0, 20, 40)


def calibrate_skew(stepper, candidates=SKEW_CANDIDATES, rounds=3, steps=200, warmup=100, min_gain=0.0025):
    """Picks the plan's group-parity skew (sf_plan_opts.xcd_parity_skew) for
    this GPU and workload by timing it: one runner per candidate, all on the
    stepper's stream (one hardware queue), in rotated order for `rounds`
    rounds; the score is the median over rounds of each round's median
    attention-kernel time. A candidate is taken only if it beats equal slices
    (0) by at least `min_gain`; the stepper keeps the chosen runner. Which
    sign helps, and how much, differs between GPUs and between the bf16 and
    fp8 kernels, so it is measured rather than fixed."""
    runners = {p: (stepper.runner if p == 0 else stepper.make_runner(p)) for p in candidates}
    times = {p: [] for p in candidates}
    for _ in range(600):                 # out of the idle clocks first
        stepper.step()
    stepper.torch.cuda.synchronize()
    for r in range(rounds):
        order = list(candidates[r % len(candidates):]) + list(candidates[:r % len(candidates)])
        for p in order:
            stepper.runner = runners[p]
            _, _, k_med = time_steps(stepper, steps, warmup)
            times[p].append(k_med * 1e3)
    score = {p: float(np.median(v)) for p, v in times.items()}
    best = min(score, key=score.get)
    chosen = best if score[best] < score[0] * (1.0 - min_gain) else 0
    stepper.runner = runners[chosen]
    return {"chosen": chosen, "kernel_us_median": {str(p): round(s, 2) for p, s in score.items()},
            "what": "plan option xcd_parity_skew (per mille; workers of even launch groups weigh 1000 + p, of odd "
                    "groups 1000 - p) chosen by timing each candidate on this GPU before the timed steps: "
                    f"{rounds} rounds x {steps} steps per candidate, one stream; taken only if it beats equal "
                    f"slices by {100 * min_gain:.2f} %"}


def decode_loop_bench(reps=5, skew=0):
    """The extreme-straggler lengths and caps as a growing-cache decode loop:
    512 sequences, 64 steps, one appended token per active sequence per step.
    Returns seq-steps/s over whole loops, host bookkeeping and planning
    included (median of `reps` timed loops after one untimed loop). Each loop
    starts from the same prompt-time pools and block table; the loops share
    one runner, whose pinned ring and workspace are allocated in the untimed
    loop."""
    import torch
    from paper_2601_12784_amd import binding as B
    from paper_2601_12784_amd.workloads import make_decode_loop
    run = make_decode_loop()
    b = run.base
    k0, v0 = b.k_pool.cuda(), b.v_pool.cuda()
    bt0 = torch.from_numpy(b.block_table).cuda()
    k, v, bt = k0.clone(), v0.clone(), bt0.clone()
    q_all, k_new, v_new = run.q_all.cuda(), run.k_new.cuda(), run.v_new.cuda()
    lens = [run.lengths(t) for t in range(run.steps)]
    kv_read = sum(b.kv_bytes(L) for L in lens)
    out = torch.empty((b.num_seqs, b.num_q_heads, b.head_dim), dtype=torch.float32, device="cuda")
    stream = torch.cuda.Stream()
    attn = B.DecodeAttention(b.num_q_heads, b.num_kv_heads, b.head_dim,   # one runner for every loop
                             opts=B.make_opts(xcd_parity_skew=skew))
    times, issue = [], []
    sink = torch.zeros(64, dtype=torch.uint8, device="cuda")
    for rep in range(reps + 1):
        runner = B.DecodeLoopRunner(b.num_q_heads, b.num_kv_heads, b.head_dim, k, v, bt, b.block_table,
                                    b.seq_lens, b.scale, attn=attn)
        k.copy_(k0)
        v.copy_(v0)
        bt.copy_(bt0)
        # One untimed read of the reset pools: the first kernel to read them
        # after the copies (which stream through 6.8 GB) ran ~30 % slow, a
        # repeat of it at full speed; a decode loop that runs on has been
        # reading its pools all along.
        for pool in (k, v):
            B.sf_debug_stream_read(pool.view(torch.uint8).view(-1), sink, 4096)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for t in range(run.steps):
            runner.step(q_all[t], lens[t], k_new[t] if t else None, v_new[t] if t else None, out=out,
                        stream=stream)
        t1 = time.perf_counter()
        torch.cuda.synchronize()
        if rep:
            times.append(time.perf_counter() - t0)
            issue.append(t1 - t0)
    wall = float(np.median(times))
    seq_steps = run.seq_steps()
    return {"xcd_parity_skew": skew, "workload": f"growing-cache decode loop: {b.num_seqs} sequences (502 x U[1,2048] + 10 x 32768 "
                        f"tokens at step 0), caps +U[0,64], {run.steps} steps, 28 q / 4 kv heads, "
                        "head_dim 128; each step appends one token per active sequence",
            "seq_steps": seq_steps, "loop_ms": round(wall * 1e3, 3),
            "seq_steps_per_s": round(seq_steps / wall, 1),
            "kv_gb_per_s": round(kv_read / wall / 1e9, 2), "kv_bytes_read": int(kv_read),
            "host_issue_ms": round(float(np.median(issue)) * 1e3, 3), "timed_loops": reps}


LLC_BYTES = 256 << 20   # MI355X last-level (Infinity) cache


def config_bench(name, steps, warmup, skew=0):
    """One decode step of a named workload (tiny, gqa7b, gqa32b), timed as the
    long-tail step is: plan -> attention -> combine back to back on one
    stream, wall time per step, attention kernel from HIP events. Batches
    whose pools would fit in the last-level cache rotate over enough device
    copies (at least 4) that every step reads its bytes from HBM. skew=None
    chooses the plan skew for this workload by timing (calibrate_skew)."""
    import torch
    from paper_2601_12784_amd.workloads import make_batch, CONFIGS
    b = make_batch(name, poison=False)
    kv = b.kv_bytes()
    pool_bytes = b.k_pool.numel() * 4
    rotate = 1 if pool_bytes > 2 * LLC_BYTES else max(4, -(-4 * LLC_BYTES // pool_bytes))
    if name == "tiny":
        rotate = 1   # 130 KB: a latency figure, cache-resident by nature
    st = Stepper(b, rotate=rotate, skew=skew or 0)
    cal = calibrate_skew(st) if skew is None else None
    skew = cal["chosen"] if cal else skew
    ms_step, k_mean, k_med = time_steps(st, steps, warmup)
    info = st.runner.last_info
    gbs = kv / (k_mean * 1e-3) / 1e9
    _, bsz, hq, hkv, d = CONFIGS[name]
    res = {"xcd_parity_skew": skew, "workload": f"{name}: {bsz} sequences, {hq} q / {hkv} kv heads, head_dim {d}, page 16",
           "tokens": int(b.seq_lens.sum()), "kv_bytes_per_step": kv, "pool_copies_rotated": rotate,
           "ms_per_step": round(ms_step, 5), "attn_kernel_us": round(k_mean * 1e3, 2),
           "attn_kernel_us_median": round(k_med * 1e3, 2),
           "kv_gb_per_s_step": round(kv / (ms_step * 1e-3) / 1e9, 2),
           "kv_gb_per_s_kernel": round(gbs, 2), "pct_of_peak_hbm_kernel": round(100 * gbs / PEAK_HBM_GBPS, 2),
           "seq_steps_per_s": round(b.num_seqs / (ms_step * 1e-3), 1),
           "workers": info.num_workers, "segments": info.num_work, "cut_pairs": info.num_combine,
           "skew_calibration": cal}
    del st
    torch.cuda.empty_cache()
    return res


def straggler_bench(reps=5, skew=0):
    """The extreme-straggler schedule over its pre-filled pool: 64 decode
    steps, the batch shrinking as sequences reach their caps. Every step's
    queries and compacted block table are uploaded before timing; the timed
    loop is the runner's plan, attention and combine per step, host planning
    included. Returns seq-steps/s over whole loops (median of `reps` after one
    untimed loop) and the attention kernels' summed time from one loop timed
    with HIP events."""
    import torch
    from paper_2601_12784_amd import binding as B
    from paper_2601_12784_amd.workloads import make_straggler
    run = make_straggler(poison=False)
    b = run.base
    k, v = b.k_pool.cuda(), b.v_pool.cuda()
    steps = [run.step_batch(t) for t in range(run.steps)]
    dev = [(s.q.cuda(), torch.from_numpy(s.block_table).cuda(), np.ascontiguousarray(s.seq_lens, np.int32))
           for s in steps]
    kv_read = sum(s.kv_bytes() for s in steps)
    seq_steps = run.seq_steps()
    out = torch.empty((b.num_seqs, b.num_q_heads, b.head_dim), dtype=torch.float32, device="cuda")
    stream = torch.cuda.Stream()
    attn = B.DecodeAttention(b.num_q_heads, b.num_kv_heads, b.head_dim, opts=B.make_opts(xcd_parity_skew=skew))

    def loop(events=None):
        for t, (q, bt, lens) in enumerate(dev):
            attn(q, k, v, bt, lens, b.scale, out=out[: q.shape[0]], stream=stream,
                 attn_events=None if events is None else events[t])

    times = []
    for rep in range(reps + 1):
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        loop()
        torch.cuda.synchronize()
        if rep:
            times.append(time.perf_counter() - t0)
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in dev]
    loop(evs)
    torch.cuda.synchronize()
    kernel_ms = float(sum(a.elapsed_time(z) for a, z in evs))
    wall = float(np.median(times))
    return {"xcd_parity_skew": skew, "workload": f"extreme straggler, pre-filled pool: {b.num_seqs} sequences at step 0 (502 x U[1,2048] "
                        f"+ 10 x 32768 tokens), caps +U[0,64], {run.steps} steps, finished sequences dropped, "
                        "28 q / 4 kv heads, head_dim 128",
            "seq_steps": seq_steps, "loop_ms": round(wall * 1e3, 3),
            "seq_steps_per_s": round(seq_steps / wall, 1),
            "kv_bytes_read": int(kv_read), "kv_gb_per_s": round(kv_read / wall / 1e9, 2),
            "pct_of_peak_hbm": round(100 * kv_read / wall / 1e9 / PEAK_HBM_GBPS, 2),
            "attn_kernels_ms_sum": round(kernel_ms, 3),
            "kv_gb_per_s_kernels": round(kv_read / (kernel_ms * 1e-3) / 1e9, 2),
            "active_at_steps_0_32_63": [int(steps[t].num_seqs) for t in (0, 32, 63)], "timed_loops": reps}


# KV bytes per token of one decode step over all layers of the paper's
# cost-model example model (48 layers x 4 KV heads x head_dim 128, K and V, bf16).
QWEN3_30B_A3B_KV_BYTES_PER_TOKEN = 48 * 4 * 128 * 2 * 2
PAPER_K1_H20 = 7.28e-8   # App. B, coefficient table (seconds per token, reading)


def calibrate_k1(batch_sizes=(64, 96, 128, 192, 256), reps=60):
    """Fits the cost model's attention term, latency = k1 * kv_bytes + c, to
    this library's decode step (plan, upload, attention, merge) on long-tail
    batches of several sizes (every one above the 256 MB last-level cache).
    Each point is the GPU time per step over `reps` back-to-back steps."""
    import torch
    from paper_2601_12784_amd.workloads import build_batch, sample_lengths, config_seed
    points = []
    for bsz in batch_sizes:
        seed = config_seed("longtail") + 50 + bsz
        rng = np.random.Generator(np.random.PCG64(seed))
        lens = sample_lengths("longtail", rng)[:bsz]
        b = build_batch(lens, 28, 4, 128, seed, rng=rng, poison=False)
        st = Stepper(b)
        for _ in range(50):
            st.step()
        torch.cuda.synchronize()
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        with torch.cuda.stream(st.stream):
            ev[0].record()
            for _ in range(reps):
                st.step()
            ev[1].record()
        ev[1].synchronize()
        points.append((b.kv_bytes(), ev[0].elapsed_time(ev[1]) / reps * 1e-3))
        del st, b
        torch.cuda.empty_cache()
    x = np.array([p[0] for p in points], dtype=np.float64)
    y = np.array([p[1] for p in points], dtype=np.float64)
    k1, c = np.polyfit(x, y, 1)
    r2 = 1.0 - float(((y - (k1 * x + c)) ** 2).sum() / ((y - y.mean()) ** 2).sum())
    max_rel = float(np.max(np.abs(k1 * x + c - y) / y))
    return {"fit": "decode-step latency = k1 * kv_bytes + c (App. B.1 attention term)",
            "k1_s_per_byte": float(k1), "c_us": round(float(c) * 1e6, 2), "r2": round(r2, 5),
            "max_rel_err": round(max_rel, 4),
            "points_bytes_us": [[int(a), round(float(t) * 1e6, 2)] for a, t in points],
            "effective_gb_s": round(1e-9 / float(k1), 1),
            "k1_s_per_token_qwen3_30b_a3b": float(k1) * QWEN3_30B_A3B_KV_BYTES_PER_TOKEN,
            "paper_k1_h20_s_per_token": PAPER_K1_H20}


def routing_demo(k1_per_token, mu=0.3, seed=0):
    """The routing strategy (sf_route) on a synthetic 16-instance snapshot and
    600 waiting trajectories, with the fitted k1 and the paper's k2..k4."""
    from paper_2601_12784_amd import binding as B
    rng = np.random.default_rng(seed)

    class I:  # noqa: E742
        def __init__(self, v, n, w, kv):
            self.version, self.running, self.waiting, self.kv = v, n, w, kv

    class T:
        def __init__(self, v, length):
            self.version, self.length = v, length

    budget = 250_000.0   # tokens of KV per instance
    model = B.sf_cost_model(k1_per_token, 1.72e-3, 1.25e-4, 1.07e-2, 1.0, budget)
    insts = [I(int(rng.integers(3, 6)), int(rng.integers(0, 120)), 0, float(rng.uniform(0, 200_000)))
             for _ in range(16)]
    trajs = [T(None if rng.random() < 0.5 else int(rng.integers(3, 6)), float(rng.integers(200, 20_000)))
             for _ in range(600)]
    t0 = time.perf_counter()
    for _ in range(20):
        target, after = B.route(model, mu, 4, insts, trajs)
    us = (time.perf_counter() - t0) / 20 * 1e6
    before = sum(B.cost_throughput(model, B.sf_instance_state(s.version, s.running, s.waiting, 0, s.kv)) for s in insts)
    after_t = sum(B.cost_throughput(model, B.sf_instance_state(s.version, s.running, s.waiting, 0, s.kv)) for s in after)
    return {"instances": 16, "trajectories": 600, "mu": mu, "routed": int(sum(t >= 0 for t in target)),
            "tokens_per_s_before": round(before, 1), "tokens_per_s_after": round(after_t, 1),
            "sf_route_us": round(us, 1)}


EXTEND_KERNEL = "extend_attn_kernel<128>"
EXTEND_SRC = os.path.join(os.path.dirname(os.path.abspath(__file__)), "paper_2601_12784_amd", "csrc",
                          "extend_attn.hip")
PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 matrix peak


def reprefill_bench(reps=20, warmup=5):
    """Extend attention on the 32-sequence full re-prefill: the work list is
    planned and uploaded once, then `reps` attention launches are timed with
    HIP events on their stream. Algorithmic flops count the causal pairs only
    (4 * D per query head and pair)."""
    import torch
    from paper_2601_12784_amd import binding as B
    from paper_2601_12784_amd.workloads import make_reprefill
    eb = make_reprefill(poison=False)
    b = eb.batch
    desc = B.make_desc(b.num_seqs, b.num_q_heads, b.num_kv_heads, b.head_dim, b.block_table.shape[1],
                       b.num_pages, b.scale)
    t0 = time.perf_counter()
    info, work = B.sf_extend_attn_plan(desc, b.seq_lens, eb.q_lens)
    plan_ms = (time.perf_counter() - t0) * 1e3
    work_dev = torch.from_numpy(np.ascontiguousarray(work)).cuda()
    q, kp, vp = eb.q.cuda(), b.k_pool.cuda(), b.v_pool.cuda()
    bt = torch.from_numpy(b.block_table).cuda()
    out = torch.empty((eb.num_rows, b.num_q_heads, b.head_dim), dtype=torch.float32, device="cuda")
    lse = torch.empty((eb.num_rows, b.num_q_heads), dtype=torch.float32, device="cuda")
    stream = torch.cuda.Stream()
    with torch.cuda.stream(stream):
        for _ in range(warmup):
            B.sf_extend_attn(desc, info, None, work_dev, q, kp, vp, bt, out, lse, stream=stream)
        evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(reps)]
        for a, z in evs:
            a.record(stream)
            B.sf_extend_attn(desc, info, None, work_dev, q, kp, vp, bt, out, lse, stream=stream)
            z.record(stream)
    torch.cuda.synchronize()
    ms = [a.elapsed_time(z) for a, z in evs]
    mean_ms = float(np.mean(ms))
    flops = eb.causal_flops()
    tflops = flops / (mean_ms * 1e-3) / 1e12
    return {"workload": "full re-prefill of 32 resumed trajectories: long-tail lengths (lognormal median 2048, "
                        "sigma 1.0, clipped to [256, 16384]), every token new, 28 q / 4 kv heads, head_dim 128, "
                        "page 16, bf16",
            "new_tokens": eb.num_rows, "items": int(info.num_items), "causal_flops": int(flops),
            "kernel_ms": round(mean_ms, 4), "kernel_ms_median": round(float(np.median(ms)), 4),
            "tokens_per_s": round(eb.num_rows / (mean_ms * 1e-3), 1), "host_plan_ms": round(plan_ms, 3),
            "roofline": {"bound": "mfma", "achieved": round(tflops, 2), "peak": PEAK_BF16_TFLOPS,
                         "unit": "TFLOP/s", "frac": round(tflops / PEAK_BF16_TFLOPS, 4), "kernel": EXTEND_KERNEL}}


def fp8_bench(batch, steps, warmup, bf16_kernel_us, skew=None):
    """The same decode step over an fp8 (E4M3) copy of the batch's cache,
    made by the library's quantizer (every page a sequence holds). Bytes per
    step: one byte per cached element plus the K and V scale of every
    (page, KV head) tile read."""
    import torch
    from paper_2601_12784_amd import binding as B
    from paper_2601_12784_amd.workloads import page_fill
    n, hkv, d = batch.num_pages, batch.num_kv_heads, batch.head_dim
    desc = B.make_desc(batch.num_seqs, batch.num_q_heads, hkv, d, batch.block_table.shape[1], n, batch.scale)
    k8 = torch.empty((n, hkv, 16 * d), dtype=torch.uint8, device="cuda")
    v8 = torch.empty((n, hkv, 16 * d), dtype=torch.uint8, device="cuda")
    ks = torch.ones((n, hkv), dtype=torch.float32, device="cuda")
    vs = torch.ones((n, hkv), dtype=torch.float32, device="cuda")
    pages, valid = page_fill(batch)
    kq, vq = batch.k_pool.cuda(), batch.v_pool.cuda()
    pd, vd = torch.from_numpy(pages).cuda(), torch.from_numpy(valid).cuda()
    B.sf_kv_quantize_fp8(desc, kq, vq, pd, vd, k8, v8, ks, vs)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(5):
        B.sf_kv_quantize_fp8(desc, kq, vq, pd, vd, k8, v8, ks, vs)
    e1.record()
    e1.synchronize()
    quant_ms = e0.elapsed_time(e1) / 5
    del kq, vq
    st = Stepper(batch, fp8=(k8, v8, ks, vs), skew=skew or 0)
    cal = calibrate_skew(st) if skew is None else None
    ms_step, k_mean, k_med = time_steps(st, steps, warmup)
    tokens = int(batch.seq_lens.sum())
    tiles = int((-(-batch.seq_lens.astype(np.int64) // 16)).sum()) * hkv
    nbytes = tokens * hkv * d * 2 + tiles * 8
    achieved = nbytes / (k_mean * 1e-3) / 1e9
    del st, k8, v8
    torch.cuda.empty_cache()
    rc = read_ceiling(nbytes)
    rc["attn_kernel_over_ceiling"] = round(achieved / rc["gb_s"], 4)
    return {"kv": "OCP FP8 E4M3 codes, one fp32 scale per (page, KV head) tile for K and for V",
            "read_ceiling": rc,
            "kv_bytes_per_step": nbytes, "ms_per_step": round(ms_step, 5), "attn_kernel_us": round(k_mean * 1e3, 2),
            "seq_steps_per_s": round(batch.num_seqs / (ms_step * 1e-3), 1),
            "kernel_speedup_vs_bf16": round(bf16_kernel_us / (k_mean * 1e3), 3),
            "quantize_ms_whole_cache": round(quant_ms, 3),
            "xcd_parity_skew": cal["chosen"] if cal else skew, "skew_calibration": cal,
            "roofline": {"bound": "hbm", "achieved": round(achieved, 2), "peak": PEAK_HBM_GBPS, "unit": "GB/s",
                         "frac": round(achieved / PEAK_HBM_GBPS, 4), "kernel": "attn_worker_fp8_kernel<128, 8>"}}


def read_ceiling(nbytes, grids=(2048, 4096, 8192), reps=15, warmup=3):
    """Bandwidth of a plain streaming read of nbytes (the library's probe kernel:
    every 16-byte piece loaded once), best of a few grid sizes: the practical
    ceiling for a kernel reading that many bytes. Each launch is timed as the
    attention kernel is, by HIP events handed to its launch, and the launches
    of one grid size are queued back to back, as decode steps are, so the
    events carry the same start latency (median of reps)."""
    import torch
    from paper_2601_12784_amd import binding as B
    nbytes -= nbytes % 16
    buf = torch.full((nbytes,), 0x5A, dtype=torch.uint8, device="cuda")
    sink = torch.zeros(64, dtype=torch.uint8, device="cuda")
    stream = torch.cuda.Stream()
    best = None
    with torch.cuda.stream(stream):
        for blocks in grids:
            evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
                   for _ in range(reps)]
            for a, b in evs:             # create both events (torch does so on a first record)
                a.record(stream)
                b.record(stream)
            for _ in range(warmup):
                B.sf_debug_stream_read(buf, sink, blocks, stream)
            for ev in evs:
                B.sf_debug_stream_read(buf, sink, blocks, stream, events=ev)
            stream.synchronize()
            us = float(np.median([a.elapsed_time(b) * 1e3 for a, b in evs]))
            if best is None or us < best[0]:
                best = (us, blocks)
    del buf
    us, blocks = best
    return {"gb_s": round(nbytes / us / 1e3, 1), "us": round(us, 2), "bytes": nbytes, "blocks": blocks,
            "kernel": "stream_read_kernel",
            "what": "plain streaming read of the step's K+V byte count: each block streams a contiguous "
                    "range, every 16-byte piece loaded once (nontemporal, 8 in flight per lane); launches "
                    "queued back to back, each timed by HIP events handed to its launch, median of "
                    f"{reps}, best of {len(grids)} grid sizes"}


def cpu_baseline(batch, min_s=10.0, max_s=30.0):
    """The fp64 oracle, timed on the host cores over repeated passes of the
    batch (or of a prefix of it, if one pass would exceed max_s)."""
    import tempfile
    import oracle
    from paper_2601_12784_amd.workloads import bf16_bits
    qb, kb, vb = bf16_bits(batch.q), bf16_bits(batch.k_pool), bf16_bits(batch.v_pool)
    native = oracle.load(oracle.build_native(tempfile.mkdtemp(prefix="sf_oracle_")))
    threads = int(native.sf_oracle_max_threads())

    def run(n):
        t = time.perf_counter()
        oracle.decode_attn(qb[:n], kb, vb, batch.block_table[:n], batch.seq_lens[:n], batch.scale, using=native)
        return time.perf_counter() - t

    cum = np.cumsum(batch.seq_lens.astype(np.int64))
    n = min(8, batch.num_seqs)
    per_tok = run(n) / max(1, int(cum[n - 1]))
    n = int(np.searchsorted(cum, max_s / 2 / max(per_tok, 1e-12), side="right"))
    n = max(1, min(batch.num_seqs, n))
    total, passes = 0.0, 0
    while total < min_s and total < max_s - 1.0 and passes < 1000:
        total += run(n)
        passes += 1
    kv = batch.kv_bytes(batch.seq_lens[:n]) * passes
    return {"value": round(kv / total / 1e9, 3), "unit": "GB/s", "cores": threads, "kind": "oracle",
            "sample": f"{passes} passes over the first {n} of {batch.num_seqs} sequences "
                      f"({int(cum[n - 1])} tokens, {kv / passes / 1e9:.3f} GB KV per pass), "
                      f"fp64 C oracle (gcc {' '.join(oracle.NATIVE_FLAGS[:3])}, built on this host) with "
                      f"{threads} OpenMP threads, {total:.1f} s"}


def stored_traffic(kv_bytes_per_launch):
    """HBM bytes per attention launch from committed rocprofv3 counter runs,
    or None if absent or taken on a different kernel source."""
    if not os.path.exists(COUNTERS_FILE):
        return None
    doc = json.load(open(COUNTERS_FILE))
    if doc.get("kernel_source_sha256_16") != kernel_source_hash():
        return None
    return doc.get("traffic_bytes_per_launch")


# the long-tail launch: head_dim 128, no append, 4 waves (workers) per workgroup
ATTN_KERNEL = "attn_worker_kernel<128, false, 4>"
COMBINE_KERNEL = "combine_kernel"
COPY_KERNEL = "__amd_rocclr_copyBuffer"


def _csv_rows(path):
    import csv
    with open(path) as f:
        return list(csv.DictReader(f))


def summarize_counters(fetch_csv, write_csv, copy_mib, kv_bytes, out_path=COUNTERS_FILE, skew=None):
    """Per-launch HBM traffic of the attention kernel from two rocprofv3 --pmc
    runs (FETCH_SIZE, then WRITE_SIZE; KiB per dispatch), each scaled by what
    the same counter reads for a plain device copy of copy_mib MiB."""
    def per_kernel(path, counter):
        vals = {}
        for r in _csv_rows(path):
            if r["Counter_Name"] != counter:
                continue
            vals.setdefault(r["Kernel_Name"], []).append(float(r["Counter_Value"]) * 1024.0)
        return vals

    def pick(vals, name):
        hits = [v for k, v in vals.items() if name in k]
        if not hits:
            raise SystemExit(f"no dispatch of {name} in the counter file")
        return float(np.mean(hits[0])), len(hits[0])

    fetch = per_kernel(fetch_csv, "FETCH_SIZE")
    write = per_kernel(write_csv, "WRITE_SIZE")
    copy_bytes = float(copy_mib) * (1 << 20)
    f_copy, _ = pick(fetch, COPY_KERNEL)
    w_copy, _ = pick(write, COPY_KERNEL)
    f_scale, w_scale = copy_bytes / f_copy, copy_bytes / w_copy
    f_attn, nf = pick(fetch, ATTN_KERNEL)
    w_attn, nw = pick(write, ATTN_KERNEL)
    doc = {
        "kernel": ATTN_KERNEL,
        "workload": "long-tail rollout batch (bench.py default)",
        "kernel_source_sha256_16": kernel_source_hash(),
        "copy_probe_bytes": copy_bytes,
        "fetch_scale": round(f_scale, 5), "write_scale": round(w_scale, 5),
        "fetch_bytes_per_launch": round(f_attn * f_scale), "write_bytes_per_launch": round(w_attn * w_scale),
        "traffic_bytes_per_launch": round(f_attn * f_scale + w_attn * w_scale),
        "algorithmic_kv_bytes_per_launch": kv_bytes,
        "traffic_over_algorithmic": round((f_attn * f_scale + w_attn * w_scale) / kv_bytes, 4),
        "dispatches": {"fetch": nf, "write": nw},
        "raw_counter_bytes_per_launch": {"FETCH_SIZE": round(f_attn), "WRITE_SIZE": round(w_attn),
                                         "copy_FETCH_SIZE": round(f_copy), "copy_WRITE_SIZE": round(w_copy)},
    }
    for name in (COMBINE_KERNEL,):
        try:
            fc, _ = pick(fetch, name)
            wc, _ = pick(write, name)
            doc[name + "_traffic_bytes_per_launch"] = round(fc * f_scale + wc * w_scale)
        except SystemExit:
            pass
    with open(out_path, "w") as f:
        json.dump(doc, f, indent=1)
    md = out_path[:-len(".json")] + ".md"
    cmd = ("cd /tmp && export TMPDIR=/tmp && timeout -s KILL 180 rocprofv3 --pmc {c} --output-format csv "
           "-d $OUT/{d} -o {o} -- python3 $REPO/bench.py --steps 5 --warmup 2 --no-cpu-baseline "
           "--no-skew --no-loop --no-cost --no-reprefill --no-fp8 --no-configs" +
           ("" if skew is None else f" --skew {int(skew)}") + " --copy-probe " + str(int(copy_mib)))
    lines = [f"# HBM traffic of {ATTN_KERNEL} on the long-tail batch (rocprofv3 counters)", "",
             "Two counter passes (one counter each), then the summary:", "", "```",
             cmd.format(c="FETCH_SIZE", d="pmc_fetch", o="f"), cmd.format(c="WRITE_SIZE", d="pmc_write", o="w"),
             "python bench.py --summarize-counters $OUT/pmc_fetch/f_counter_collection.csv "
             f"$OUT/pmc_write/w_counter_collection.csv --copy-probe {int(copy_mib)}" +
             ("" if skew is None else f" --skew {int(skew)}"), "```", "",
             "($REPO: the repository root; $OUT: any directory for the profiler's output.)" +
             ("" if skew is None else f" The plan skew {int(skew)} is the one the default run chose on the same "
                                      "GPU just before (it moves slice boundaries, not the bytes read)."), "",
             f"Kernel source sha256[:16]: `{doc['kernel_source_sha256_16']}`", "",
             "Calibration: a plain device copy (`__amd_rocclr_copyBuffer`) of "
             f"{int(copy_mib)} MiB reads FETCH_SIZE = {doc['raw_counter_bytes_per_launch']['copy_FETCH_SIZE']} B "
             f"and WRITE_SIZE = {doc['raw_counter_bytes_per_launch']['copy_WRITE_SIZE']} B, so the counters are "
             f"scaled by {doc['fetch_scale']} (reads) and {doc['write_scale']} (writes).", "",
             "| per attention launch | bytes |", "|---|---|",
             f"| FETCH_SIZE x scale | {doc['fetch_bytes_per_launch']} |",
             f"| WRITE_SIZE x scale | {doc['write_bytes_per_launch']} |",
             f"| traffic | {doc['traffic_bytes_per_launch']} |",
             f"| algorithmic K+V bytes | {doc['algorithmic_kv_bytes_per_launch']} |",
             f"| traffic / algorithmic | {doc['traffic_over_algorithmic']} |"]
    if COMBINE_KERNEL + "_traffic_bytes_per_launch" in doc:
        lines.append(f"| combine kernel traffic | {doc[COMBINE_KERNEL + '_traffic_bytes_per_launch']} |")
    with open(md, "w") as f:
        f.write("\n".join(lines) + "\n")
    return doc


EXTEND_COUNTERS = {
    "SQ_INSTS_MFMA": "matrix-core instructions (all waves)",
    "SQ_INSTS_VALU": "vector ALU instructions, matrix-core ones included",
    "SQ_INSTS_VALU_TRANS_F32": "transcendental (exp2) instructions",
    "SQ_INSTS_LDS": "LDS instructions",
    "SQ_INSTS_SALU": "scalar ALU instructions",
    "SQ_VALU_MFMA_BUSY_CYCLES": "matrix-core busy cycles, summed over SIMDs",
    "SQ_VALU_MFMA_COEXEC_CYCLES": "cycles with vector ALU and matrix core both busy, summed over SIMDs",
    "SQ_BUSY_CYCLES": "sequencer busy cycles",
    "SQ_WAVE_CYCLES": "wave-cycles (units of 4 cycles)",
    "SQ_ACTIVE_INST_VALU": "wave-cycles issuing vector ALU work (units of 4 cycles)",
    "SQ_ACTIVE_INST_LDS": "wave-cycles issuing LDS work (units of 4 cycles)",
    "SQ_WAIT_INST_ANY": "wave-cycles waiting on a dependency (units of 4 cycles)",
    "SQ_WAIT_INST_LDS": "wave-cycles waiting on LDS (units of 4 cycles)",
    "SQ_LDS_IDX_ACTIVE": "LDS busy cycles",
    "SQ_LDS_BANK_CONFLICT": "LDS bank-conflict cycles",
    "SQ_BUSY_CU_CYCLES": "CU busy cycles",
}


def summarize_extend_counters(csvs, stats_csv, command, out_md, simds=1024, clock_ghz=2.4):
    """Markdown summary of rocprofv3 --pmc passes over the re-prefill leg:
    per-launch means of the counters in EXTEND_COUNTERS and what they say
    about the extend kernel's bound (matrix-core busy share, vector work,
    their overlap)."""
    import collections
    vals = collections.defaultdict(list)
    for path in csvs:
        for r in _csv_rows(path):
            if EXTEND_KERNEL.split("<")[0] in r["Kernel_Name"]:
                vals[r["Counter_Name"]].append(float(r["Counter_Value"]))
    mean = {k: sum(v) / len(v) for k, v in vals.items()}
    kt = [r for r in _csv_rows(stats_csv) if EXTEND_KERNEL.split("<")[0] in r["Name"]]
    us = float(kt[0]["AverageNs"]) / 1e3 if kt else float("nan")
    simd_cycles = us * 1e-6 * clock_ghz * 1e9 * simds
    lines = [f"# Counters: {EXTEND_KERNEL} on the full re-prefill batch", "",
             "Commands (from the repository root; one counter pass per line, then the kernel trace):", "", "```"]
    lines += command.split(" ;; ") + ["```", "",
             "($REPO: the repository root; $OUT: any directory for the profiler's output.)", "",
             f"Kernel source sha256[:16]: `{kernel_source_hash(EXTEND_SRC)}`; mean kernel duration {us:.1f} us "
             f"(rocprofv3 trace); {simds} SIMDs at {clock_ghz} GHz = {simd_cycles:.3e} SIMD-cycles per launch.", "",
             "| counter | per launch | meaning |", "|---|---|---|"]
    for k, what in EXTEND_COUNTERS.items():
        if k in mean:
            lines.append(f"| `{k}` | {mean[k]:.4e} | {what} |")
    if {"SQ_VALU_MFMA_BUSY_CYCLES", "SQ_INSTS_MFMA", "SQ_INSTS_VALU"} <= mean.keys():
        mf = mean["SQ_VALU_MFMA_BUSY_CYCLES"]
        valu = mean["SQ_INSTS_VALU"] - mean["SQ_INSTS_MFMA"]
        trans = mean.get("SQ_INSTS_VALU_TRANS_F32", 0.0)
        co = mean.get("SQ_VALU_MFMA_COEXEC_CYCLES", float("nan"))
        lines += ["", "Derived:", "",
                  f"- matrix-core busy: {mf / simd_cycles:.1%} of SIMD-cycles "
                  f"({mf / mean['SQ_INSTS_MFMA']:.1f} cycles per MFMA instruction)",
                  f"- vector ALU instructions besides MFMA: {valu:.3e}, of which exp2 {trans:.3e}; "
                  f"{valu / mean['SQ_INSTS_MFMA']:.2f} per MFMA",
                  f"- vector ALU and matrix core busy together: {co / simd_cycles:.1%} of SIMD-cycles"]
        if "SQ_WAVE_CYCLES" in mean and "SQ_WAIT_INST_ANY" in mean:
            lines.append(f"- waves waiting on a dependency: {mean['SQ_WAIT_INST_ANY'] / mean['SQ_WAVE_CYCLES']:.1%} "
                         f"of wave time (LDS: {mean.get('SQ_WAIT_INST_LDS', 0) / mean['SQ_WAVE_CYCLES']:.1%})")
    with open(out_md, "w") as f:
        f.write("\n".join(lines) + "\n")


def _events_vs_trace(rows, kernel, event_us):
    """A line comparing the HIP-event mean of a kernel with the trace's."""
    hit = [r for r in rows if kernel in r["Name"]]
    if not hit:
        return []
    tr = float(hit[0]["AverageNs"]) / 1e3
    return [f"- the trace's mean for `{kernel}`: {tr:.2f} us; the events read {event_us - tr:+.2f} us "
            f"({100 * (event_us / tr - 1):+.1f} %) from it (the start event is a marker ahead of the dispatch)"]


def _skew_note(command):
    if "--skew" not in command:
        return []
    return ["The plan skews in the command are the ones a default run (which times the candidates first) chose "
            "on the same GPU just before; fixing them keeps those calibration launches out of the trace.", ""]


def summarize_trace(stats_csv, command, out_md, bench_json=None):
    """Markdown summary of a rocprofv3 --kernel-trace --stats run (the decode
    step, the re-prefill leg when the bench line is an --only-reprefill one,
    or a named workload's step for an --only-config one)."""
    rows = _csv_rows(stats_csv)
    b = json.load(open(bench_json)) if bench_json else None
    if b is not None and "pool_copies_rotated" in b:
        lines = [f"# Kernel trace: the decode step on {b['workload']}", "", "Command (from the repository root):",
                 "", "```", command, "```", ""] + _skew_note(command) + [
                 f"Kernel source sha256[:16]: `{kernel_source_hash()}`", "",
                 "| kernel | calls | average us | min us | max us | share % |", "|---|---|---|---|---|---|"]
        for r in rows:
            lines.append(f"| `{r['Name'][:90]}` | {r['Calls']} | {float(r['AverageNs']) / 1e3:.2f} | "
                         f"{float(r['MinNs']) / 1e3:.2f} | {float(r['MaxNs']) / 1e3:.2f} | {float(r['Percentage']):.2f} |")
        lines += ["", "bench.py line of the same run (HIP events on the kernel's stream):", "",
                  f"- attention kernel mean: {b['attn_kernel_us']} us for {b['kv_bytes_per_step']} bytes of K and V "
                  f"= {b['kv_gb_per_s_kernel']} GB/s ({b['pct_of_peak_hbm_kernel']} % of 8000)",
                  f"- step: {b['ms_per_step'] * 1e3:.1f} us; {b['seq_steps_per_s']} seq-steps/s; "
                  f"{b['pool_copies_rotated']} pool copies rotated"] + _events_vs_trace(rows, ATTN_KERNEL,
                                                                        b['attn_kernel_us'])
        with open(out_md, "w") as f:
            f.write("\n".join(lines) + "\n")
        return
    reprefill = b is not None and "causal_flops" in b
    fp8 = (not reprefill and b is not None and "fp8" in b
           and any("attn_worker_fp8_kernel" in r["Name"] for r in rows))
    title = (f"# Kernel trace: {EXTEND_KERNEL} on the full re-prefill batch" if reprefill
             else "# Kernel trace: the decode step on the long-tail batch, bf16 and fp8 caches" if fp8
             else f"# Kernel trace: {ATTN_KERNEL} on the long-tail batch")
    src = EXTEND_SRC if reprefill else KERNEL_SRC
    lines = [title, "", "Command (from the repository root):", "", "```", command, "```", ""] + _skew_note(command)
    lines += [f"Kernel source sha256[:16]: `{kernel_source_hash(src)}`", "",
             "| kernel | calls | average us | min us | max us | share % |", "|---|---|---|---|---|---|"]
    for r in rows:
        lines.append(f"| `{r['Name'][:90]}` | {r['Calls']} | {float(r['AverageNs']) / 1e3:.2f} | "
                     f"{float(r['MinNs']) / 1e3:.2f} | {float(r['MaxNs']) / 1e3:.2f} | {float(r['Percentage']):.2f} |")
    if reprefill:
        lines += ["", "bench.py line of the same run (HIP events on the kernel's stream):", "",
                  f"- extend kernel mean: {b['kernel_ms'] * 1e3:.1f} us over {b['items']} work items",
                  f"- causal flops per pass: {b['causal_flops']}",
                  f"- roofline achieved: {b['roofline']['achieved']} TFLOP/s "
                  f"({100 * b['roofline']['frac']:.1f}% of {b['roofline']['peak']:.0f})"]
    elif b:
        lines += ["", "bench.py line of the same run (HIP events on the kernel's stream):", "",
                  f"- attention kernel mean: {b['attn_kernel_us']} us",
                  f"- step: {b['ms_per_step'] * 1e3:.1f} us; value {b['value']} GB/s",
                  f"- roofline achieved: {b['roofline']['achieved']} GB/s ({100 * b['roofline']['frac']:.1f}% of 8000)"]
        lines += _events_vs_trace(rows, ATTN_KERNEL, b["attn_kernel_us"])
        if fp8:
            f8 = b["fp8"]
            lines += [f"- fp8 cache: attention kernel mean {f8['attn_kernel_us']} us, step {f8['ms_per_step'] * 1e3:.1f} us, "
                      f"{f8['roofline']['achieved']} GB/s of codes ({100 * f8['roofline']['frac']:.1f}% of 8000), "
                      f"{f8['read_ceiling']['attn_kernel_over_ceiling']} of a plain read of the same bytes"]
    with open(out_md, "w") as f:
        f.write("\n".join(lines) + "\n")


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=500)
    ap.add_argument("--warmup", type=int, default=1000,
                    help="untimed steps first (the GPU leaves its idle clocks during these)")
    ap.add_argument("--chunk-pages", type=int, default=0, help="force the pages per worker")
    ap.add_argument("--workers-per-cu", type=int, default=0, help="planner workers (waves) per CU")
    ap.add_argument("--skew", type=int, default=None,
                    help="plan group-parity skew (per mille) of the long-tail leg; default: chosen by "
                         "timing candidates on this GPU before the timed steps")
    ap.add_argument("--fp8-skew", type=int, default=None, help="the same for the fp8 leg")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-skew", action="store_true", help="skip the equal-bytes uniform batch")
    ap.add_argument("--no-loop", action="store_true", help="skip the growing-cache decode loop")
    ap.add_argument("--no-cost", action="store_true", help="skip the cost-model k1 fit")
    ap.add_argument("--no-reprefill", action="store_true", help="skip the extend (re-prefill) leg")
    ap.add_argument("--no-fp8", action="store_true", help="skip the fp8-cache leg")
    ap.add_argument("--no-configs", action="store_true",
                    help="skip the tiny, 7B-like, 32B-like and pre-filled straggler legs")
    ap.add_argument("--only-reprefill", action="store_true", help="run only the extend leg and print it")
    ap.add_argument("--only-config", default=None, help="run only this named workload's leg and print it")
    ap.add_argument("--summarize-extend-counters", nargs="+", metavar="FILE",
                    help="PMC_CSV... STATS_CSV COMMANDS OUT_MD: counters summary of the re-prefill leg")
    ap.add_argument("--copy-probe", type=int, default=0,
                    help="first run a plain device copy of this many MiB (counter calibration)")
    ap.add_argument("--summarize-counters", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"),
                    help="write the counters summary from two rocprofv3 --pmc runs and exit")
    ap.add_argument("--summarize-trace", nargs=3, metavar=("STATS_CSV", "COMMAND", "OUT_MD"),
                    help="write a markdown summary of a --kernel-trace --stats run and exit")
    ap.add_argument("--bench-json", default=None, help="bench.py output of the traced run")
    args = ap.parse_args()
    if args.summarize_counters:
        from paper_2601_12784_amd.workloads import config_seed, sample_lengths
        lens = sample_lengths("longtail", np.random.Generator(np.random.PCG64(config_seed("longtail"))))
        kv = int(lens.sum()) * 4 * 128 * 2 * 2  # 4 KV heads, head_dim 128, K and V, bf16
        print(json.dumps(summarize_counters(*args.summarize_counters, args.copy_probe or 1024, kv, skew=args.skew),
                         indent=1))
        return
    if args.summarize_trace:
        summarize_trace(*args.summarize_trace, bench_json=args.bench_json)
        return
    if args.summarize_extend_counters:
        *pmc, stats, cmd, out = args.summarize_extend_counters
        summarize_extend_counters(pmc, stats, cmd, out)
        return
    if args.gpus != 1:
        print(json.dumps({"error": "bench.py measures a single GPU (the decode path runs on one device); --gpus must be 1"}))
        log("bench.py runs on exactly one GPU: the decode-attention path here is single-GPU "
            "(sharding is described, not built). Use --gpus 1.")
        sys.exit(2)

    import torch
    from paper_2601_12784_amd import binding as B
    from paper_2601_12784_amd.workloads import make_batch, build_batch, uniform_lengths_like
    B.lib()
    if not torch.cuda.is_available():
        log("no GPU visible")
        sys.exit(1)

    if args.only_reprefill:
        print(json.dumps(reprefill_bench()), flush=True)
        return
    if args.only_config:
        fixed = args.skew if args.skew is not None else (0 if args.only_config == "tiny" else None)
        print(json.dumps(config_bench(args.only_config, args.steps, args.warmup, skew=fixed)), flush=True)
        return

    if args.copy_probe:
        nbytes = args.copy_probe << 20
        src = torch.empty(nbytes, dtype=torch.uint8, device="cuda").fill_(1)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        log(f"copy probe: {nbytes} bytes x3")
        del src, dst

    log("generating long-tail batch")
    batch = make_batch("longtail")
    kv = batch.kv_bytes()
    log(f"  {batch.num_seqs} seqs, {int(batch.seq_lens.sum())} tokens, {kv / 1e9:.3f} GB KV/step")
    st = Stepper(batch, chunk_pages=args.chunk_pages, workers_per_cu=args.workers_per_cu, skew=args.skew or 0)
    calibration = None
    if args.skew is None and not args.chunk_pages:
        log("  choosing the plan's group-parity skew for this GPU (untimed)")
        calibration = calibrate_skew(st)
        log(f"  skew {calibration['chosen']}: {calibration['kernel_us_median']}")
    skew = calibration["chosen"] if calibration else (args.skew or 0)
    ms_step, attn_ms_mean, attn_ms_med = time_steps(st, args.steps, args.warmup)
    info = st.runner.last_info
    log(f"  step {ms_step * 1e3:.1f} us, attention kernel {attn_ms_mean * 1e3:.1f} us (median "
        f"{attn_ms_med * 1e3:.1f}), {info.num_workers} workers x {info.chunk_pages} pages, "
        f"{info.num_work} segments, {info.num_combine} cut pairs")

    desc = B.make_desc(batch.num_seqs, batch.num_q_heads, batch.num_kv_heads, batch.head_dim,
                       batch.block_table.shape[1], batch.num_pages, batch.scale)
    hbuf = np.empty(info.work_bytes // 4, dtype=np.int32)
    t = time.perf_counter()
    for _ in range(50):
        B.sf_decode_attn_plan(desc, st.lens, st.runner.opts, work_host=hbuf)
    plan_us = (time.perf_counter() - t) / 50 * 1e6

    achieved = kv / (attn_ms_mean * 1e-3) / 1e9
    traffic = stored_traffic(kv)
    result = {
        "metric": METRIC,
        "value": round(kv / (ms_step * 1e-3) / 1e9, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": "long-tail rollout batch: 256 sequences, 28 q / 4 kv heads, head_dim 128, "
                               "page 16, KV lengths lognormal(median 2048, sigma 1.0) clipped to [256, 16384], "
                               "bf16 N(0,1), one decode step",
                   "seed": batch.seed, "kv_bytes_per_step": kv, "tokens": int(batch.seq_lens.sum()),
                   "workers": info.num_workers, "pages_per_worker": info.chunk_pages,
                   "xcd_parity_skew": skew,
                   "segments": info.num_work, "cut_pairs": info.num_combine},
        "seq_steps_per_s": round(batch.num_seqs / (ms_step * 1e-3), 1),
        "pct_of_peak_hbm": round(100.0 * kv / (ms_step * 1e-3) / 1e9 / PEAK_HBM_GBPS, 2),
        "attn_kernel_us": round(attn_ms_mean * 1e3, 2),
        "host_plan_us": round(plan_us, 2),
        "skew_calibration": calibration,
        "roofline": {"bound": "hbm", "achieved": round(achieved, 2), "peak": PEAK_HBM_GBPS, "unit": "GB/s",
                     "frac": round(achieved / PEAK_HBM_GBPS, 4),
                     "traffic": traffic},
    }

    log("streaming-read ceiling: a plain kernel reading the same bytes")
    del st
    torch.cuda.empty_cache()
    rc = read_ceiling(kv)
    rc["attn_kernel_over_ceiling"] = round(achieved / rc["gb_s"], 4)
    result["read_ceiling"] = rc
    log(f"  {rc['gb_s']} GB/s ({rc['us']} us); the attention kernel reaches {rc['attn_kernel_over_ceiling']:.3f} of it")

    if not args.no_skew:
        torch.cuda.empty_cache()
        lens_u = uniform_lengths_like(batch.seq_lens.astype(np.int64))
        log("generating equal-token uniform batch")
        ub = build_batch(lens_u, 28, 4, 128, batch.seed + 100, name="uniform")
        su = Stepper(ub, chunk_pages=args.chunk_pages, workers_per_cu=args.workers_per_cu, skew=skew)
        ms_u, attn_u, _ = time_steps(su, args.steps, args.warmup)
        result["skew"] = {"uniform_ms_per_step": round(ms_u, 5), "uniform_kv_bytes": ub.kv_bytes(),
                          "skewed_over_uniform": round(ms_step / ms_u, 4),
                          "uniform_attn_kernel_us": round(attn_u * 1e3, 2)}
        del su

    if not args.no_cost:
        log("cost model: fitting k1 to the decode step on five batch sizes")
        cm = calibrate_k1()
        cm["routing_demo"] = routing_demo(cm["k1_s_per_token_qwen3_30b_a3b"])
        result["cost_model"] = cm
        log(f"  k1 = {cm['k1_s_per_byte']:.3e} s/byte ({cm['effective_gb_s']} GB/s), c = {cm['c_us']} us, "
            f"r2 = {cm['r2']}")

    if not args.no_fp8:
        log("fp8 (E4M3) cache: the same step over the library-quantized cache")
        f8 = fp8_bench(batch, max(100, args.steps // 2), max(100, args.warmup // 2), attn_ms_mean * 1e3,
                       skew=args.fp8_skew)
        result["fp8"] = f8
        log(f"  step {f8['ms_per_step'] * 1e3:.1f} us, kernel {f8['attn_kernel_us']} us "
            f"({f8['roofline']['achieved']} GB/s of fp8 codes, {f8['kernel_speedup_vs_bf16']}x the bf16 kernel; "
            f"{f8['read_ceiling']['attn_kernel_over_ceiling']:.3f} of a plain read of the same bytes)")

    if not args.no_configs:
        legs = {}
        for name in ("tiny", "gqa7b", "gqa32b"):
            log(f"config {name}")
            # the single-step configs choose their own skew (unless --skew fixes it); tiny is latency only
            legs[name] = config_bench(name, args.steps, min(args.warmup, 500),
                                      skew=(skew if args.skew is not None or name == "tiny" else None))
            log(f"  step {legs[name]['ms_per_step'] * 1e3:.1f} us, kernel {legs[name]['attn_kernel_us']} us, "
                f"{legs[name]['kv_gb_per_s_kernel']} GB/s ({legs[name]['pct_of_peak_hbm_kernel']} % of peak), "
                f"{legs[name]['seq_steps_per_s']} seq-steps/s")
        log("config straggler (pre-filled, 64 steps)")
        legs["straggler"] = straggler_bench(skew=skew)
        log(f"  {legs['straggler']['loop_ms']} ms per loop, {legs['straggler']['seq_steps_per_s']} seq-steps/s, "
            f"{legs['straggler']['kv_gb_per_s']} GB/s")
        result["configs"] = legs

    if not args.no_reprefill:
        log("extend attention: full re-prefill of 32 trajectories")
        rp = reprefill_bench()
        result["reprefill"] = rp
        log(f"  {rp['kernel_ms']} ms per pass, {rp['roofline']['achieved']} TFLOP/s "
            f"({100 * rp['roofline']['frac']:.1f} % of bf16 peak), {rp['tokens_per_s']:.0f} tokens/s")

    if not args.no_loop:
        log("growing-cache decode loop (straggler lengths, 64 steps)")
        result["decode_loop"] = decode_loop_bench(skew=skew)
        log(f"  {result['decode_loop']['seq_steps_per_s']} seq-steps/s, "
            f"{result['decode_loop']['loop_ms']} ms per loop")

    if not args.no_cpu_baseline:
        log("timing the oracle on the host")
        result["cpu_baseline"] = cpu_baseline(batch)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
