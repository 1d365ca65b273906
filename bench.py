#!/usr/bin/env python
"""Decode throughput of the paged GQA decode path on one MI355X.

One step is one decode step of the whole path for every active row: the compact
workqueue planner and the split-attention kernel with its last-arriver merge, over a
native paged KV cache (Hq=32, Hkv=8, d=128, fp16, page 16). The default route runs all
of it in one launch (every workgroup derives its tasks from the lengths); --route picks
the planner-kernel + fused-kernel pair, the three-launch ablation or the length-bucket
routes. Before each step, outside the timed region, the step's new token K/V is written
into the pool, seq_lens grows by one, and a 1 GiB streaming read evicts the 256 MB
last-level cache (MALL) so that KV is read from HBM as it would be with the other
layers' KV in between. The eviction reads only, so no dirty lines are left to be
written back during the timed step.

Timing: HIP events on the stream the kernels run on, around each step. Steps are
enqueued back to back behind the cache eviction read, so the events measure device
time (launch overhead included), not Python launch latency; a second pass times the
planner launch with events around it and the decode kernel with events stamped by its
own launch, and a host-synchronized pass gives wall time per step.

value = decode tokens / second = sum of active rows over the timed steps / sum of step
times (event intervals around the step, marker latency included). roofline.achieved =
algorithmic bytes of one decode-kernel launch / its average execution time (start and
stop events stamped by the launch itself, hipExtLaunchKernel, so the interval is the
kernel's own, as rocprofv3 reports it). extra.beta_read_gbs is the streaming-read
bandwidth of the 1 GiB eviction read in the same run (the calibration probe beta).
cpu_baseline = the fp64 numpy oracle on the host over the same steps' inputs.
"""
from __future__ import annotations

import argparse
import dataclasses
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "decode tokens/sec per step + achieved HBM GB/s (% of MI355X peak), B1/B8"
HBM_PEAK_GBS = 8000.0
KERNEL_SRC = os.path.join(ROOT, "paper_2606_26666_amd", "csrc", "pkv_kernels.hip")
PROFILES = os.path.join(ROOT, "profiles")
TASK_BYTES = 20
BUCKET_TOKENS = 16384   # coarse-bucket width: rows grouped by ceil(len / 16384)
ROUTES = ("plan+fused", "one-launch", "two-kernel", "rect", "exact-buckets", "coarse-buckets")


def kernel_hash() -> str:
    return hashlib.sha256(open(KERNEL_SRC, "rb").read()).hexdigest()[:16]


def kv_bytes_per_token(hkv=8, d=128):
    return 2 * hkv * d * 2   # K and V, fp16


def algorithmic_bytes(lens, num_tasks, hq=32, d=128, hkv=8):
    """Bytes one decode-kernel launch must move: K/V of every attended token, Q and out,
    the block-table entries and lengths read, the task list, and each task's partial
    state (fp32 acc[G][d], m[G], l[G]; 2080 B at G=4) written once and read once by the
    merge."""
    from paper_2606_26666_amd.costmodel import slot_bytes
    lens = np.asarray(lens, dtype=np.int64)
    B = lens.size
    kv = kv_bytes_per_token(hkv, d) * int(lens.sum())
    qo = 2 * B * hq * d * 2
    meta = 4 * int(((lens + 15) // 16).sum()) + 4 * B + 4 * (B + 1) + TASK_BYTES * num_tasks
    partial = 2 * slot_bytes(hq // hkv, d) * num_tasks
    return kv + qo + meta + partial, kv


class Runner:
    """Device state of one workload: pools, block table, lengths, buffers."""

    def __init__(self, name, seed, target_tasks, steps, route="plan+fused", policy=0, hkv=8):
        import torch

        import paper_2606_26666_amd as pkv
        from workloads import make_workload
        from workloads.values import device_normal_f16, q_values

        self.torch, self.pkv = torch, pkv
        w = make_workload(name, seed=seed, steps=steps, hkv=hkv)
        if not target_tasks:  # the cost model's rule for the first step's lengths
            from paper_2606_26666_amd import costmodel
            target_tasks = costmodel.default_target(w.lengths_at(0), w.hkv, hq=w.hq)
        self.w = w = dataclasses.replace(w, target_tasks=target_tasks)
        self.dev = torch.device("cuda:0")
        shape = (w.num_pages, w.page_size, w.hkv, w.head_dim)
        self.k = device_normal_f16(shape, seed * 4 + 1, self.dev)
        self.v = device_normal_f16(shape, seed * 4 + 2, self.dev)
        r = np.random.Generator(np.random.PCG64(seed + 7))
        self.q = torch.from_numpy(q_values(w.batch, w.hq, w.head_dim, r)).to(self.dev)
        self.bt = torch.from_numpy(w.block_table).to(self.dev)
        self.lens = torch.from_numpy(w.lengths_at(0)).to(self.dev)
        self.out = torch.empty((w.batch, w.hq, w.head_dim), dtype=torch.float16, device=self.dev)
        self.bufs = pkv.DecodeBuffers(w.batch, w.hq, w.hkv, w.head_dim, w.split_max, self.dev)
        self.params = pkv.make_params(w.hkv, w.split_min, w.split_max, w.target_tasks, w.tile_tokens,
                                      policy=policy)
        self.policy = policy
        self.route = route
        self.fused = route != "two-kernel"
        self.cur_lens = w.lengths_at(0)
        self.last_launches = 0
        self.gen = torch.Generator(device=self.dev)
        self.gen.manual_seed(seed * 4 + 3)
        self.bt_host = w.block_table

    def shape(self, lens):
        """The cost model's account of one step of this route over `lens`."""
        from paper_2606_26666_amd import costmodel
        return costmodel.route_shape(self.route, lens, self.params, self.w.hq, self.w.head_dim,
                                     self.w.max_pages_per_row)

    def rect_splits(self):
        """Split count of the rectangular grid (the cost model's batch rule)."""
        from paper_2606_26666_amd import costmodel
        active = int(np.count_nonzero(np.asarray(self.cur_lens) > 0))
        return costmodel.rect_split_count(active, self.w.hkv, self.params)

    def host_lengths(self, step):
        return self.w.lengths_at(step)

    def prepare(self, steps):
        """Per-step lengths and append positions, staged on the device up front so the
        timed loop never waits on a host copy."""
        torch, w = self.torch, self.w
        lens = np.stack([w.lengths_at(s) for s in range(steps)])
        pos = lens.astype(np.int64) - 1
        pages = self.bt_host[np.arange(w.batch)[None, :], pos // w.page_size].astype(np.int64)
        self.lens_steps = torch.from_numpy(lens).to(self.dev)
        self.pages_steps = torch.from_numpy(pages).to(self.dev)
        self.slots_steps = torch.from_numpy(pos % w.page_size).to(self.dev)
        self.lens_host = lens

    def append(self, step):
        """Write step `step`'s new token K/V at the row's last position and set seq_lens
        (all enqueued on the stream, no host synchronization)."""
        torch, w = self.torch, self.w
        if w.append:
            nk = torch.randn((w.batch, w.hkv, w.head_dim), generator=self.gen, device=self.dev).half()
            nv = torch.randn((w.batch, w.hkv, w.head_dim), generator=self.gen, device=self.dev).half()
            self.k[self.pages_steps[step], self.slots_steps[step]] = nk
            self.v[self.pages_steps[step], self.slots_steps[step]] = nv
        self.lens.copy_(self.lens_steps[step])
        self.cur_lens = self.lens_host[step]
        return self.lens_host[step]

    def plan(self):
        if self.route in ("one-launch", "rect", "exact-buckets", "coarse-buckets"):
            return  # the decode launch plans, or the route's split count comes from the host
        b = self.bufs
        self.pkv.pkv_plan(self.lens, None, self.w.num_pages, self.params, b.tasks, b.split_offsets, b.num_tasks,
                          b.ws, max_pages_per_row=self.w.max_pages_per_row)

    def decode(self, events=None):
        """events: (start, stop) stamped with the decode kernels' execution interval
        (one-launch, plan+fused and two-kernel routes); None for a plain launch."""
        b = self.bufs
        if self.route == "rect":
            self.pkv.pkv_decode_rect(self.q, self.k, self.v, self.bt, self.lens, self.rect_splits(),
                                     self.w.tile_tokens, 1.0, self.out, b.ws)
            return
        if self.route in ("exact-buckets", "coarse-buckets"):
            self.last_launches = self.pkv.pkv_decode_buckets(
                self.q, self.k, self.v, self.bt, self.lens, self.cur_lens,
                0 if self.route == "exact-buckets" else BUCKET_TOKENS, self.params, 1.0, self.out, b.ws)
            return
        if self.route == "one-launch":
            self.pkv.pkv_plan_decode(self.q, self.k, self.v, self.bt, self.lens, self.params, b.tasks,
                                     b.split_offsets, b.num_tasks, 1.0, self.out, b.ws, events=events)
            return
        self.pkv.pkv_decode(self.q, self.k, self.v, self.bt, self.lens, b.tasks, b.split_offsets, b.num_tasks,
                            1.0, self.out, b.ws, fused=self.fused, events=events)


def measure(runner, steps, warmup, flush_bufs):
    torch, pkv = runner.torch, runner.pkv
    Ev = lambda: torch.cuda.Event(enable_timing=True)  # noqa: E731

    def flush():
        if flush_bufs is not None:  # read-only: leaves the cache full of clean lines
            pkv.pkv_stream_read(flush_bufs[0], flush_bufs[1])

    runner.prepare(steps)
    runner.append(0)
    for _ in range(warmup):
        flush()
        runner.plan()
        runner.decode()
    torch.cuda.synchronize()
    ev = []
    ntasks, lens_all = [], []
    for s in range(steps):
        lens_all.append(runner.append(s))
        flush()
        e0, e2 = Ev(), Ev()
        e0.record()
        runner.plan()
        runner.decode()
        e2.record()
        ev.append((e0, e2))
        ntasks.append(runner.bufs.num_tasks.clone() if runner.route in ("one-launch", "plan+fused", "two-kernel")
                      else runner.shape(runner.cur_lens).workgroups)
    torch.cuda.synchronize()
    step_ms = [a.elapsed_time(c) for a, c in ev]
    ntasks = [int(t.item()) if hasattr(t, "item") else int(t) for t in ntasks]
    bits = pkv.pkv_check_device_status(runner.bufs.ws)
    if bits:
        raise RuntimeError(f"device error bits {bits}")
    # per-kernel breakdown on the last step's inputs (kept out of the step timing above):
    # events around the planner launch, and the decode kernels' own execution interval
    # (stamped by the launch itself, the interval rocprofv3 reports); the bucket routes,
    # several launches, take plain events around the decode call
    kernel_stamps = runner.route in ("one-launch", "plan+fused", "two-kernel")
    ev = []
    for s in range(steps):
        flush()
        e0, e1, e2, e3 = Ev(), Ev(), Ev(), Ev()
        e0.record()
        runner.plan()
        e1.record()
        if kernel_stamps:
            runner.decode(events=(e2, e3))
        else:
            e2.record()
            runner.decode()
            e3.record()
        ev.append((e0, e1, e2, e3))
    torch.cuda.synchronize()
    plan_ms = [a.elapsed_time(b) for a, b, c, d in ev]
    dec_ms = [c.elapsed_time(d) for a, b, c, d in ev]
    # marker latency alone: two events with nothing between them
    ev = []
    for s in range(steps):
        e0, e1 = Ev(), Ev()
        e0.record()
        e1.record()
        ev.append((e0, e1))
    torch.cuda.synchronize()
    marker_ms = [a.elapsed_time(b) for a, b in ev]
    # serving-facing wall time: host-synchronized, includes launch overhead
    wall = []
    for s in range(steps):
        flush()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        runner.plan()
        runner.decode()
        torch.cuda.synchronize()
        wall.append((time.perf_counter() - t0) * 1e3)
    return dict(step_ms=step_ms, plan_ms=plan_ms, dec_ms=dec_ms, ntasks=ntasks, lens=lens_all, wall_ms=wall,
                marker_ms=marker_ms)


def read_ceiling(pkv, torch, buf, sink, nbytes, reps=7):
    """Streaming-read bandwidth (GB/s) of the first `nbytes` of the 1 GiB buffer with the
    decode's K/V load policy (non-temporal loads), from the read kernel's own execution
    interval (launch-stamped events), each read after a full pass over the buffer with
    allocating loads, so that the bytes read are not in the 256 MB last-level cache."""
    Ev = lambda: torch.cuda.Event(enable_timing=True)  # noqa: E731
    view = buf[:nbytes - nbytes % 16]
    us = []
    for _ in range(reps):
        pkv.pkv_stream_read(buf, sink)
        e0, e1 = Ev(), Ev()
        pkv.pkv_stream_read_nt_timed(view, sink, events=(e0, e1))
        torch.cuda.synchronize()
        us.append(e0.elapsed_time(e1) * 1e3)
    return view.numel() / float(np.median(us)) / 1e3


def page_read_us(pkv, torch, runner, flush_bufs, reps=7):
    """Read time (us) of the decode's pages in the decode's pattern: the library's
    read-only probe (pkv_stream_read_pages) over the last step's task list, with the
    decode's KV heads per workgroup, each run after the cache-evicting read; median of
    the runs' launch-stamped execution intervals. None for routes without a task list."""
    if runner.route not in ("one-launch", "plan+fused", "two-kernel") or flush_bufs is None:
        return None
    Ev = lambda: torch.cuda.Event(enable_timing=True)  # noqa: E731
    w = runner.w
    hpw = 2 if runner.route == "one-launch" and head_pairs(w.hq, w.hkv, w.target_tasks) else 1
    us = []
    for _ in range(reps):
        pkv.pkv_stream_read(flush_bufs[0], flush_bufs[1])
        e0, e1 = Ev(), Ev()
        pkv.pkv_stream_read_pages(runner.k, runner.v, runner.bt, runner.bufs.tasks, runner.bufs.num_tasks, hpw,
                                  flush_bufs[1], events=(e0, e1))
        torch.cuda.synchronize()
        us.append(e0.elapsed_time(e1) * 1e3)
    return float(np.median(us))


def calibrate(pkv, torch, flush_bufs, reps=10, launches=200):
    """Device constants of the cost model, measured in this run: beta = streaming-read
    bandwidth of a 1 GiB read (GB/s, the read kernel's own execution interval), lambda =
    device time per back-to-back launch of a near-empty kernel (us), from events around
    `launches` 16-byte reads queued behind a backlog of large reads."""
    Ev = lambda: torch.cuda.Event(enable_timing=True)  # noqa: E731
    buf, sink = flush_bufs if flush_bufs is not None else (
        torch.zeros(1 << 30, dtype=torch.uint8, device="cuda"), torch.zeros(1, dtype=torch.int32, device="cuda"))
    pkv.pkv_stream_read(buf, sink)
    beta = read_ceiling(pkv, torch, buf, sink, buf.numel(), reps)
    # launch gap: queue enough 1 GiB reads ahead that the host has enqueued every
    # small launch before the device reaches them, so the interval is device time
    small = buf[:16]
    for _ in range(max(4, launches // 16)):
        pkv.pkv_stream_read(buf, sink)
    e0, e1 = Ev(), Ev()
    e0.record()
    for _ in range(launches):
        pkv.pkv_stream_read(small, sink)
    e1.record()
    torch.cuda.synchronize()
    lam = e0.elapsed_time(e1) * 1e3 / launches
    return {"beta_read_gbs": beta, "launch_gap_us": lam}


def head_pairs(hq, hkv, target):
    """Whether the one-launch kernel runs KV-head pairs: G = 4, even Hkv and at least two
    tasks per resident workgroup (one workgroup per compute unit)."""
    from paper_2606_26666_amd import costmodel
    return costmodel.head_pairs(hq, hkv) and target >= 2 * costmodel.CUS


def split_range(runner, lens):
    """(fewest, most) splits of an active row at the step over `lens`: the planner's
    per-row split counts for the workqueue routes, the launch's S for the rectangular
    grid, the per-group S for the bucket routes."""
    from paper_2606_26666_amd import costmodel
    lens = np.asarray(lens, dtype=np.int64)
    act = lens > 0
    if not act.any():
        return [0, 0]
    if runner.route in ("one-launch", "plan+fused", "two-kernel"):
        _, offs, _ = runner.pkv.pkv_plan_host(lens, runner.params, runner.w.max_pages_per_row, with_tasks=False)
        ns = np.diff(offs)[act]
    elif runner.route == "rect":
        S = runner.rect_splits()
        tiles = -(-lens[act] // runner.w.tile_tokens)
        ns = np.minimum(tiles, S)
    else:
        groups = costmodel.bucket_groups(lens, runner.route == "exact-buckets")
        ns = []
        for rows in groups:
            S = costmodel.rect_split_count(rows.size, runner.w.hkv, runner.params)
            ns += [min(S, -(-int(lens[i]) // runner.w.tile_tokens)) for i in rows if lens[i] > 0]
        ns = np.asarray(ns)
    return [int(ns.min()), int(ns.max())]


def summarize(runner, m):
    w = runner.w
    tokens = w.batch * len(m["step_ms"])
    step_s = sum(m["step_ms"]) / 1e3
    alg, kv = zip(*(algorithmic_bytes(l, t, w.hq, w.head_dim, w.hkv) for l, t in zip(m["lens"], m["ntasks"])))
    marker = float(np.median(m["marker_ms"]))
    # decode-kernel duration: its execution interval as stamped by the launch (the
    # duration rocprofv3 reports); the empty-interval marker latency is reported beside it
    dec_ms = float(np.mean(m["dec_ms"]))
    achieved = float(alg[-1]) / (dec_ms / 1e3) / 1e9  # the breakdown pass ran the last step's inputs
    return {
        "tok_s": tokens / step_s,
        "ms_per_step": float(np.mean(m["step_ms"])),
        "plan_ms": float(np.mean(m["plan_ms"])),
        "event_marker_ms": marker,
        "decode_ms": dec_ms,
        "wall_ms_per_step": float(np.median(m["wall_ms"])),
        "wall_tok_s": w.batch / (float(np.median(m["wall_ms"])) / 1e3),
        "alg_bytes_per_launch": float(np.mean(alg)),
        "alg_bytes_last_step": float(alg[-1]),
        "kv_bytes_per_step": float(np.mean(kv)),
        "decode_gbs": achieved,
        "decode_frac_of_peak": achieved / HBM_PEAK_GBS,
        "step_gbs": float(np.mean(alg)) / (float(np.mean(m["step_ms"])) / 1e3) / 1e9,
        "tasks_per_step": float(np.mean(m["ntasks"])),
        "task_target": int(w.target_tasks),
        "splits_per_row": split_range(runner, m["lens"][-1]),
        "kv_heads_per_workgroup": 2 if runner.route == "one-launch" and head_pairs(w.hq, w.hkv, w.target_tasks)
                                  else 1,
        "launches_per_step": launches_per_step(runner),
        **route_counters(runner, m),
    }


def launches_per_step(runner):
    if runner.route in ("exact-buckets", "coarse-buckets"):
        return runner.last_launches
    return runner.shape(runner.cur_lens).launch_count


def route_counters(runner, m):
    """Scheduler counters of the paper's Tab. 4 for the last timed step (from the cost
    model's route shape): split workgroups per CU, useful KV MiB, partial-state (merge)
    MiB, merge launches."""
    lens = np.asarray(m["lens"][-1], dtype=np.int64)
    sh = runner.shape(lens)
    return {"split_wg_per_cu": sh.workgroups / 256.0,
            "useful_kv_mib": float(lens.sum()) * kv_bytes_per_token(runner.w.hkv, runner.w.head_dim) / 2**20,
            "merge_mib": sh.merge_bytes / 2 / 2**20, "merge_launches": sh.merge_launches}


def read_traffic(workload):
    """HBM bytes per decode launch from the committed rocprofv3 counter summary, if it was
    taken on the current kernel source; else None."""
    path = os.path.join(PROFILES, f"counters_split_kernel_{workload}.md")
    if not os.path.exists(path):
        return None
    kv = {}
    for line in open(path):
        if ":" in line and line.startswith("- "):
            k, v = line[2:].split(":", 1)
            kv[k.strip()] = v.strip()
    if kv.get("kernel_source_sha256") != kernel_hash():
        return None
    try:
        return float(kv["hbm_bytes_per_dispatch"])
    except (KeyError, ValueError):
        return None


def cpu_baseline(runner, steps, min_s=10.0):
    """The fp64 oracle on the host over the same steps' inputs, cycled until about min_s
    seconds of work (a bounded sample of the workload), with the BLAS pool at its default
    size; then one step on one thread, and the tiny 512-token case, both reported beside
    it."""
    from threadpoolctl import threadpool_info, threadpool_limits

    from oracle import ref_decode
    from workloads import make_workload
    from workloads.values import host_normal_f16, q_values
    w = runner.w
    k = runner.k.cpu().numpy()
    v = runner.v.cpu().numpy()
    q = runner.q.cpu().numpy()
    ref_decode(q, k, v, w.block_table, w.lengths_at(0))  # first-touch warmup, untimed
    t0 = time.perf_counter()
    done = 0
    while True:
        ref_decode(q, k, v, w.block_table, w.lengths_at(done % steps))
        done += 1
        if time.perf_counter() - t0 >= min_s:
            break
    dt = time.perf_counter() - t0
    threads = max([x.get("num_threads", 1) for x in threadpool_info()] or [1])
    with threadpool_limits(1):
        t1 = time.perf_counter()
        ref_decode(q, k, v, w.block_table, w.lengths_at(0))
        dt1 = time.perf_counter() - t1
    tw = make_workload("tiny")
    rng = np.random.Generator(np.random.PCG64(11))
    shape = (tw.num_pages, tw.page_size, tw.hkv, tw.head_dim)
    tk, tv = host_normal_f16(shape, rng), host_normal_f16(shape, rng)
    tq = q_values(tw.batch, tw.hq, tw.head_dim, rng)
    t2 = time.perf_counter()
    ref_decode(tq, tk, tv, tw.block_table, tw.lengths_at(0))
    dt_tiny = time.perf_counter() - t2
    return {"value": done * w.batch / dt, "unit": "tokens/s", "cores": int(threads), "kind": "oracle",
            "sample": f"{w.name}: {done} decode steps (its {steps} steps, cycled) of the fp64 numpy oracle, "
                      f"{dt:.1f} s, BLAS threads {threads}, host CPUs {len(os.sched_getaffinity(0))}",
            "one_thread_value": w.batch / dt1,
            "tiny_step_ms": dt_tiny * 1e3}


def oracle_step_tok_s(runner):
    """The oracle's rate on one step of another workload (its first step's inputs, after
    an untimed first-touch call), BLAS pool at its default size."""
    from oracle import ref_decode
    w = runner.w
    k, v, q = runner.k.cpu().numpy(), runner.v.cpu().numpy(), runner.q.cpu().numpy()
    ref_decode(q, k, v, w.block_table, w.lengths_at(0))
    t0 = time.perf_counter()
    ref_decode(q, k, v, w.block_table, w.lengths_at(0))
    return w.batch / (time.perf_counter() - t0)


CALIBRATION = os.path.join(ROOT, "paper_2606_26666_amd", "calibration_mi355x.json")
# (workload, route, policy, task target) steps the cost model is fitted on: the split
# sensitivity sweep of the one-launch workqueue on B1 and B8 bimodal, the one-launch
# route on the other traces, and every route of the bench's routes tables at the task
# target of the cost model's rule (0) (exact buckets are left out: their step time
# includes host launch time whenever the host falls behind)
CAL_RUNS = ([(w, "one-launch", 1, t) for w in ("b1", "b8_bimodal") for t in (128, 256, 512, 1024)]
            + [(w, "one-launch", 1, 0) for w in ("b8_uniform", "b8_zipf", "b4_bimodal")]
            + [(w, r, 1, 0) for w in ("b1", "b8_bimodal", "b8_uniform")
               for r in ("plan+fused", "two-kernel", "rect", "coarse-buckets")])


def dataclass_dict(x):
    import dataclasses
    return dataclasses.asdict(x)


def fit_cost_model(args, flush_bufs, probe, out_path):
    """Time every CAL_RUNS configuration, fit C_min and T_0 with beta and lambda from the
    probes, write the calibration file and return (calibration, rows)."""
    from paper_2606_26666_amd import costmodel
    samples, rows = [], []
    for (wl, route, policy, target) in CAL_RUNS:
        r = Runner(wl, args.seed, target, 50 if wl != "b1" else 20, route=route, policy=policy)
        m = measure(r, args.steps, args.warmup, flush_bufs)
        sh = r.shape(m["lens"][-1])
        us = float(np.mean(m["step_ms"])) * 1e3
        samples.append((sh, us))
        rows.append((wl, route, policy, int(r.w.target_tasks), sh, us, [int(x) for x in m["lens"][-1]]))
        del r
    cal = costmodel.fit(samples, probe["beta_read_gbs"], probe["launch_gap_us"])
    cal.note += f"; written by: python bench.py --calibrate {os.path.relpath(out_path, ROOT)}"
    cal.save(out_path)
    table = [{"workload": wl, "route": route, "policy": pol, "target": t, "measured_us": us,
              "model_us": costmodel.estimate_us(sh, cal), "wg_per_cu": sh.workgroups / 256.0, "lens": lens}
             for (wl, route, pol, t, sh, us, lens) in rows]
    return cal, table


def cost_model_view(runner, measured_us, routes_measured=None):
    """The committed calibration's estimate of every route for the runner's last step,
    the route it would choose and, when every route was timed on this workload
    (`routes_measured`: {route: us per step}), the measured fastest one."""
    from paper_2606_26666_amd import costmodel
    if not os.path.exists(CALIBRATION):
        return None
    cal = costmodel.Calibration.load(CALIBRATION)
    lens = runner.cur_lens
    est = {r: costmodel.estimate_us(costmodel.route_shape(r, lens, runner.params, runner.w.hq, runner.w.head_dim,
                                                         runner.w.max_pages_per_row), cal)
           for r in costmodel.ROUTES}
    out = {"chosen": min(est, key=est.get), "estimate_us": est, "measured_us": measured_us,
           "calibration": {"beta_gbs": cal.beta_gbs, "probe_beta_gbs": cal.probe_beta_gbs,
                           "launch_us": cal.launch_us, "c_min": cal.c_min, "fixed_us": cal.fixed_us,
                           "route_fixed_us": cal.route_fixed_us}}
    if routes_measured:
        out["measured_fastest"] = min(routes_measured, key=routes_measured.get)
        out["routes_measured_us"] = routes_measured
        out["chosen_is_fastest"] = out["chosen"] == out["measured_fastest"]
    return out


def seed_spread(args, workloads, seeds, first, flush_bufs):
    """Per-seed tok/s, step time and decode-kernel bandwidth of each workload on the main
    seed (results already in `first`) and the further held-out seeds, with mean and
    sample std over all of them (the paper reports mean and std over five held-out
    seeds)."""
    keys = ("tok_s", "ms_per_step", "decode_ms", "decode_gbs")
    out = {}
    for name in workloads:
        per = {str(args.seed): {k: first[name][k] for k in keys}}
        for sd in seeds:
            steps = 20 if name == "b1" else 50
            r = Runner(name, sd, args.target_tasks, steps, route=args.route, policy=args.policy, hkv=args.hkv)
            res = summarize(r, measure(r, min(args.steps * 2, steps), args.warmup, flush_bufs))
            per[str(sd)] = {k: res[k] for k in keys}
            del r
        out[name] = {"per_seed": per,
                     **{k + "_mean": float(np.mean([v[k] for v in per.values()])) for k in keys},
                     **{k + "_std": float(np.std([v[k] for v in per.values()], ddof=1)) if len(per) > 1 else 0.0
                        for k in keys}}
    return out


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="b1")
    ap.add_argument("--also", default="b8_bimodal,b8_uniform,b8_zipf,b4_bimodal",
                    help="comma-separated extra workloads, or 'none'")
    ap.add_argument("--seed", type=int, default=20260623)
    ap.add_argument("--seeds", default="20260624,20260625,20260626,20260627",
                    help="further held-out seeds: the main workload and each --also workload are also run "
                         "on these, and extra.seeds reports mean and std over --seed plus these ('none' to skip)")
    ap.add_argument("--target-tasks", type=int, default=0,
                    help="planner task target; 0 = the cost model's rule, max(256, 4 * Hkv * active rows) "
                         "(256 = one task per compute unit)")
    ap.add_argument("--policy", type=int, default=1,
                    help="split policy: 0 one split count from the active batch size, 1 tile quota (smallest "
                         "per-split tile quota whose task count fits --target-tasks)")
    ap.add_argument("--route", default="one-launch", choices=list(ROUTES),
                    help="plan+fused: planner kernel + fused split/merge kernel (2 launches); one-launch: "
                         "planner inside the decode launch; two-kernel: planner, split kernel, merge kernel; "
                         "rect: rectangular (B, Hkv, S) grid + merge kernel; "
                         "exact-buckets / coarse-buckets: host-grouped rows, a rectangular launch pair per group")
    ap.add_argument("--routes-table", default="b1,b8_bimodal,b8_uniform",
                    help="comma-separated workloads on which every route is also timed with its Tab. 4 counters "
                         "('none' to skip)")
    ap.add_argument("--no-flush", action="store_true", help="keep KV warm in the last-level cache")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--hkv", type=int, default=8, choices=(4, 8, 16, 32),
                    help="KV heads (Hq = 32, so G = 32 / hkv: 8 -> G=4, 32 -> G=1, 4 -> G=8)")
    ap.add_argument("--calibrate", metavar="PATH",
                    help="fit the route cost model (C_min, T_0) on the CAL_RUNS steps, write it to PATH, print "
                         "measured against modelled step times as one JSON line, and exit")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one MI355X: this build has no multi-GPU path (run with --gpus 1)",
              file=sys.stderr)
        sys.exit(2)
    import torch
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(2)
    import paper_2606_26666_amd as pkv
    pkv.lib()  # fail loudly when the HIP library is missing

    # a copy of known size (64 MiB read + 64 MiB written), so that rocprofv3 FETCH_SIZE and
    # WRITE_SIZE of this run can be scaled to bytes
    cal = torch.zeros(2 << 26, dtype=torch.uint8, device="cuda")
    pkv.pkv_stream_copy(cal[: 1 << 26], cal[1 << 26:])
    torch.cuda.synchronize()
    del cal
    flush_bufs = None
    if not args.no_flush:
        flush_bufs = (torch.zeros(1 << 30, dtype=torch.uint8, device="cuda"),
                      torch.zeros(1, dtype=torch.int32, device="cuda"))

    cal = calibrate(pkv, torch, flush_bufs)
    if args.calibrate:
        model, table = fit_cost_model(args, flush_bufs, cal, os.path.abspath(args.calibrate))
        print(json.dumps({"calibration": dataclass_dict(model), "steps": table}))
        return
    steps_cfg = max(args.steps, 20 if args.workload == "b1" else 50)
    main_run = Runner(args.workload, args.seed, args.target_tasks, steps_cfg, route=args.route,
                      policy=args.policy, hkv=args.hkv)
    m = measure(main_run, args.steps, args.warmup, flush_bufs)
    s = summarize(main_run, m)
    extra = {args.workload: s, "calibration": cal}
    runs = {args.workload: main_run}

    def with_ceiling(res, runner):
        """Two read ceilings beside the kernel's rate: a contiguous streaming read of the
        step's KV size, and the read-only probe of the decode's own pages and pattern."""
        if flush_bufs is not None:
            nbytes = min(int(res["kv_bytes_per_step"]), flush_bufs[0].numel())
            res["read_ceiling_gbs"] = read_ceiling(pkv, torch, flush_bufs[0], flush_bufs[1], nbytes)
            res["decode_frac_of_read_ceiling"] = res["decode_gbs"] / res["read_ceiling_gbs"]
            pr = page_read_us(pkv, torch, runner, flush_bufs)
            if pr is not None:
                res["page_read_us"] = pr
                res["page_read_gbs"] = res["kv_bytes_per_step"] / pr / 1e3
                res["decode_frac_of_page_read"] = pr / (res["decode_ms"] * 1e3)
        return res

    with_ceiling(s, main_run)
    oracle_also = {}
    also = [x for x in args.also.split(",") if x and x != "none" and x != args.workload]
    for name in also:
        r = Runner(name, args.seed, args.target_tasks, 50, route=args.route, policy=args.policy, hkv=args.hkv)
        extra[name] = with_ceiling(summarize(r, measure(r, min(args.steps * 2, 50), args.warmup, flush_bufs)), r)
        if name == "b8_bimodal" and not args.no_cpu_baseline:
            oracle_also[name] = oracle_step_tok_s(r)
        runs[name] = r
    seeds = [int(x) for x in args.seeds.split(",") if x and x != "none" and int(x) != args.seed]
    if seeds:
        extra["seeds"] = seed_spread(args, [args.workload] + also, seeds,
                                     {args.workload: s, **{n: extra[n] for n in also}}, flush_bufs)
    tables = {}
    for wl in [x for x in args.routes_table.split(",") if x and x != "none"]:
        table = {}
        for route in ROUTES:
            r = Runner(wl, args.seed, args.target_tasks, 50 if wl != "b1" else 20, route=route, policy=args.policy,
                       hkv=args.hkv)
            res = summarize(r, measure(r, min(args.steps * 2, 50 if wl != "b1" else 20), args.warmup, flush_bufs))
            table[route] = {k: res[k] for k in ("tok_s", "ms_per_step", "decode_ms", "launches_per_step",
                                                "split_wg_per_cu", "splits_per_row", "useful_kv_mib", "merge_mib",
                                                "merge_launches")}
            del r
        extra["routes_" + wl] = table
        tables[wl] = {rt: v["ms_per_step"] * 1e3 for rt, v in table.items()}
    # the cost model's route choice for every workload timed above, against the measured
    # fastest route where every route was timed
    for name, r in runs.items():
        extra[name]["cost_model"] = cost_model_view(r, extra[name]["ms_per_step"] * 1e3, tables.get(name))
    extra["cost_model"] = extra[args.workload]["cost_model"]
    traffic = read_traffic(args.workload) if args.hkv == 8 else None  # the summaries cover Hkv = 8
    line = {
        "metric": METRIC,
        "value": s["tok_s"],
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": s["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f16",
        "data": "synthetic",
        "config": {"workload": args.workload, **{k: v for k, v in main_run.w.describe().items() if k != "workload"},
                   "kv_layout": "[num_pages,16,Hkv,d]", "accumulate": "f32",
                   "route": args.route,
                   "split_policy": ["batch split count", "tile quota"][args.policy],
                   # the tile-quota policy does not use split_min; the split counts the
                   # planner gave the active rows at the last timed step:
                   **({"split_min": main_run.w.split_min} if args.policy == 0 else {}),
                   "split_max": main_run.w.split_max,
                   "splits_per_row": s["splits_per_row"],
                   "task_target": s["task_target"],
                   "llc_flushed": not args.no_flush, "parallelism": "single GPU"},
        "roofline": {"bound": "hbm", "achieved": s["decode_gbs"], "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": s["decode_gbs"] / HBM_PEAK_GBS, "traffic": traffic,
                     "kernel": "split_kernel" + (" (planner inside)" if args.route == "one-launch" else ""),
                     "alg_bytes_per_launch": s["alg_bytes_last_step"],
                     "read_ceiling_gbs": s.get("read_ceiling_gbs"), "page_read_gbs": s.get("page_read_gbs"),
                     "kernel_source_sha256": kernel_hash()},
        "cpu_baseline": None if args.no_cpu_baseline else {
            **cpu_baseline(main_run, args.steps),
            **{f"{k}_step_tok_s": val for k, val in oracle_also.items()}},
        "extra": extra,
    }
    print(json.dumps(line))


if __name__ == "__main__":
    main()
