"""Continuous-batching decode harness (Sec. 3.6-3.8, Sec. 4.6).

Requests arrive over decode steps, are admitted into a fixed set of batch slots while
pages last, decode one token per step and leave when their decode length is reached.
Each step runs the attention path of this library over the whole slot batch in one
launch (`pkv_plan_decode`: free slots have length 0 and get no tasks), optionally
followed by a gated-MLP tail of intermediate width 11008 on the active rows (the
model-level proxy of Sec. 4.6, dense fp16 GEMMs through torch).

  PagePool    host free list of physical page ids, handed out in a seeded permuted
              order so that a request's pages are scattered in memory (Sec. 3.7)
  Engine      device state: K/V pools, block table, lengths, Q, workspace, MLP weights
  Scheduler   admission, per-step decode, completion, timing

Timing follows the paper's two clocks: events around the queued device work of a step
(token append + attention, and the MLP tail when enabled), and host wall time per step
with a synchronization, which includes Python-side scheduling and setup.
"""
from __future__ import annotations

import argparse
import dataclasses
import json
import sys
import time

import numpy as np

from . import _binding as _b
from . import costmodel

PAGE = 16


class PagePool:
    """Physical page ids [0, num_pages), handed out from a seeded permutation."""

    def __init__(self, num_pages: int, seed: int = 0):
        if num_pages < 1:
            raise ValueError("num_pages must be positive")
        self.num_pages = int(num_pages)
        order = np.random.Generator(np.random.PCG64(seed)).permutation(self.num_pages)
        self._free = [int(x) for x in order[::-1]]   # pop() returns the permutation in order
        self._used = set()

    @property
    def free_count(self) -> int:
        return len(self._free)

    def alloc(self, n: int) -> list:
        if n > len(self._free):
            raise MemoryError(f"pool exhausted: {n} pages requested, {len(self._free)} free")
        ids = [self._free.pop() for _ in range(n)]
        self._used.update(ids)
        return ids

    def free(self, ids) -> None:
        for i in ids:
            if i not in self._used:
                raise ValueError(f"page {i} is not allocated")
            self._used.remove(i)
            self._free.append(i)


@dataclasses.dataclass
class Active:
    req: object
    slot: int
    pages: list
    length: int        # tokens in the KV cache (prompt + generated so far)
    generated: int = 0


class Engine:
    """Device state of a slot batch. Prompt K/V is synthetic: a request's pages hold the
    pool's seeded values (no prefill is modelled); each decode step writes the new
    token's K/V at the row's next position before attending."""

    def __init__(self, max_batch: int, max_pages_per_row: int, num_pages: int, hq: int = 32, hkv: int = 8,
                 d: int = 128, split=(16, 64), target_tasks: int = 0, policy: int = 1, mlp: bool = False,
                 mlp_width: int = 11008, seed: int = 0, device="cuda"):
        import torch
        self.torch = torch
        self.dev = torch.device(device)
        self.B, self.hq, self.hkv, self.d = max_batch, hq, hkv, d
        self.maxp = max_pages_per_row
        g = torch.Generator(device=self.dev)
        g.manual_seed(seed)
        self.gen = g
        shape = (num_pages, PAGE, hkv, d)
        self.k = torch.randn(shape, generator=g, device=self.dev, dtype=torch.float32).half()
        self.v = torch.randn(shape, generator=g, device=self.dev, dtype=torch.float32).half()
        self.bt_host = np.zeros((max_batch, max_pages_per_row), dtype=np.int32)
        self.bt = torch.zeros((max_batch, max_pages_per_row), dtype=torch.int32, device=self.dev)
        self.lens_host = np.zeros(max_batch, dtype=np.int32)
        self.lens = torch.zeros(max_batch, dtype=torch.int32, device=self.dev)
        self.q = torch.zeros((max_batch, hq, d), dtype=torch.float16, device=self.dev)
        self.out = torch.zeros((max_batch, hq, d), dtype=torch.float16, device=self.dev)
        self.bufs = _b.DecodeBuffers(max_batch, hq, hkv, d, split[1], self.dev)
        # target 0: the cost model's rule, per step, from the active rows
        self.split, self.policy, self.fixed_target = split, policy, target_tasks
        self.params = _b.make_params(hkv, split[0], split[1], target_tasks or costmodel.CUS, policy=policy)
        self.mlp = None
        if mlp:
            h = hq * d
            self.mlp = tuple((torch.randn(shape2, generator=g, device=self.dev, dtype=torch.float32)
                              / np.sqrt(shape2[0])).half()
                             for shape2 in ((h, mlp_width), (h, mlp_width), (mlp_width, h)))

    def admit(self, slot: int, pages, prompt_len: int) -> None:
        row = np.full(self.maxp, 0, dtype=np.int32)
        row[:len(pages)] = pages
        self.bt_host[slot] = row
        self.bt[slot].copy_(self.torch.from_numpy(row))
        self.lens_host[slot] = prompt_len

    def release(self, slot: int) -> None:
        self.lens_host[slot] = 0

    def step(self, active_slots) -> dict:
        """Append one token to every active row, attend, run the MLP tail, wait for the
        device; returns the step's device times (ms: attention, whole step) from events
        on the current stream."""
        torch = self.torch
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
        idx = np.asarray(active_slots, dtype=np.int64)
        pos = self.lens_host[idx].astype(np.int64)                 # the new token's position
        pages = self.bt_host[idx, pos // PAGE].astype(np.int64)
        self.lens_host[idx] += 1
        ev[0].record()
        if idx.size:
            n = idx.size
            pg = torch.from_numpy(pages).to(self.dev, non_blocking=True)
            sl = torch.from_numpy(pos % PAGE).to(self.dev, non_blocking=True)
            self.k[pg, sl] = torch.randn((n, self.hkv, self.d), generator=self.gen, device=self.dev).half()
            self.v[pg, sl] = torch.randn((n, self.hkv, self.d), generator=self.gen, device=self.dev).half()
            self.q.normal_(generator=self.gen)
            self.q.mul_(1.0 / np.sqrt(self.d))
        self.lens.copy_(torch.from_numpy(self.lens_host))
        if not self.fixed_target:
            self.params.target_tasks = costmodel.default_target(self.lens_host[idx], self.hkv, hq=self.hq)
        b = self.bufs
        _b.pkv_plan_decode(self.q, self.k, self.v, self.bt, self.lens, self.params, b.tasks, b.split_offsets,
                           b.num_tasks, 1.0, self.out, b.ws)
        ev[1].record()
        if self.mlp is not None and idx.size:
            x = self.out[torch.from_numpy(idx).to(self.dev)].reshape(idx.size, self.hq * self.d)
            wg, wu, wd = self.mlp
            h = torch.nn.functional.silu(x @ wg) * (x @ wu)
            self.mlp_out = h @ wd
        ev[2].record()
        torch.cuda.synchronize()
        return {"attn_ms": ev[0].elapsed_time(ev[1]), "step_ms": ev[0].elapsed_time(ev[2])}

    def snapshot(self, slots):
        """Host copies of the inputs the last step attended for `slots`: (q, k, v,
        block_table, lens), for checking."""
        self.torch.cuda.synchronize()
        idx = np.asarray(slots, dtype=np.int64)
        return (self.q.cpu().numpy()[idx], self.k.cpu().numpy(), self.v.cpu().numpy(),
                self.bt_host[idx].copy(), self.lens_host[idx].copy())


class Scheduler:
    """Continuous batching over a request trace."""

    def __init__(self, trace, engine: Engine, pool: PagePool, max_batch: int, observer=None):
        """observer(record): called after each step's device work, before finished
        requests release their slots (a checker can still read the step's inputs)."""
        self.observer = observer
        self.pending = sorted(trace, key=lambda q: (q.arrival_step, q.rid))
        self.engine, self.pool, self.B = engine, pool, max_batch
        self.free_slots = list(range(max_batch))[::-1]
        self.active = {}          # slot -> Active
        self.done = []
        self.step_idx = 0
        self.records = []

    def _admit(self) -> None:
        while self.pending and self.free_slots and self.pending[0].arrival_step <= self.step_idx:
            q = self.pending[0]
            need = -(-(q.prompt_len + q.decode_len) // PAGE)   # reserve the whole request
            if need > self.engine.maxp:
                raise ValueError(f"request {q.rid} needs {need} pages, block table holds {self.engine.maxp}")
            if need > self.pool.free_count:
                break                                           # wait for pages
            self.pending.pop(0)
            pages = self.pool.alloc(need)
            slot = self.free_slots.pop()
            self.engine.admit(slot, pages, q.prompt_len)
            self.active[slot] = Active(q, slot, pages, q.prompt_len)

    def step(self, timed: bool = True) -> dict:
        """One decode step; returns its record (active rows, device ms, wall ms)."""
        t0 = time.perf_counter()
        self._admit()
        slots = sorted(self.active)
        res = self.engine.step(slots)          # returns after the device has finished
        wall = (time.perf_counter() - t0) * 1e3
        for s in slots:
            a = self.active[s]
            a.length += 1
            a.generated += 1
        rec = {"step": self.step_idx, "active": len(slots), "attn_ms": res["attn_ms"],
               "step_ms": res["step_ms"], "wall_ms": wall, "slots": slots}
        if self.observer is not None:
            self.observer(rec)
        for s in slots:
            a = self.active[s]
            if a.generated >= a.req.decode_len:
                self.engine.release(s)
                self.pool.free(a.pages)
                del self.active[s]
                self.free_slots.append(s)
                self.done.append(a.req.rid)
        self.step_idx += 1
        self.records.append(rec)
        return rec

    @property
    def finished(self) -> bool:
        return not self.pending and not self.active

    def run(self, max_steps: int, warmup: int = 0) -> dict:
        while not self.finished and self.step_idx < max_steps:
            self.step()
        recs = [r for r in self.records[warmup:] if r["active"] > 0]
        tokens = sum(r["active"] for r in recs)
        dev_ms = sum(r["step_ms"] for r in recs)
        attn_ms = sum(r["attn_ms"] for r in recs)
        wall_ms = sum(r["wall_ms"] for r in recs)
        return {"steps": len(recs), "tokens": tokens, "completed": len(self.done),
                "mean_active": tokens / max(1, len(recs)),
                "device_tok_s": tokens / (dev_ms / 1e3) if dev_ms else 0.0,
                "attention_tok_s": tokens / (attn_ms / 1e3) if attn_ms else 0.0,
                "wall_tok_s": tokens / (wall_ms / 1e3) if wall_ms else 0.0,
                "device_ms_per_step": dev_ms / max(1, len(recs)),
                "wall_ms_per_step": wall_ms / max(1, len(recs))}


def main(argv=None) -> int:
    from workloads.requests import FAMILIES, load_trace, request_trace
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--trace", default="bimodal", help=f"one of {FAMILIES} or a CSV/JSON trace file")
    ap.add_argument("--requests", type=int, default=32)
    ap.add_argument("--max-batch", type=int, default=8)
    ap.add_argument("--steps", type=int, default=400, help="step limit")
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--decode", default="64,256", help="decode length range min,max")
    ap.add_argument("--arrival-gap", type=int, default=0)
    ap.add_argument("--mlp", action="store_true", help="gated-MLP tail (width 11008) after attention")
    ap.add_argument("--target-tasks", type=int, default=0, help="0: the cost model's rule per step")
    ap.add_argument("--seed", type=int, default=20260623)
    args = ap.parse_args(argv)
    import torch
    if not torch.cuda.is_available():
        print("the serving harness needs a GPU", file=sys.stderr)
        return 2
    if args.trace in FAMILIES:
        dmin, dmax = (int(x) for x in args.decode.split(","))
        trace = request_trace(args.trace, args.requests, args.seed, dmin, dmax, args.arrival_gap)
    else:
        trace = load_trace(args.trace)
    maxp = max(-(-(q.prompt_len + q.decode_len) // PAGE) for q in trace)
    num_pages = maxp * args.max_batch + maxp        # the batch's worst case plus one spare row
    engine = Engine(args.max_batch, maxp, num_pages, target_tasks=args.target_tasks, mlp=args.mlp,
                    seed=args.seed)
    sched = Scheduler(trace, engine, PagePool(num_pages, args.seed), args.max_batch)
    stats = sched.run(args.steps, warmup=args.warmup)
    stats.update({"trace": args.trace, "requests": len(trace), "max_batch": args.max_batch, "mlp": args.mlp,
                  "seed": args.seed})
    print(json.dumps(stats))
    return 0


if __name__ == "__main__":
    sys.exit(main())
