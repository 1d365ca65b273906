"""Request lengths and block tables for the synthetic decode workloads.

Page tables follow the paper's generator (Sec. 3.7): request i reserves
L_i = ceil(reserved_i / P) logical pages; with L = sum L_i and hole fraction rho the
physical universe has ceil(L / (1 - rho)) page ids; one seeded permutation of the
universe hands each request a consecutive slice, so logical order is kept inside a
block table while physical ids are scattered.

Length families follow Sec. 3.8 with the concrete distributions of the benchmark
configurations: one 32K row (low-active long context), bimodal (half short
U[256,2048], half long U[16384,32768]), uniform U[1024,32768] and a Zipf-like family
min(32768, 256*k) with k ~ Zipf(1.2).
"""
from __future__ import annotations

import dataclasses
import math

import numpy as np

HQ, HKV, HEAD_DIM, PAGE = 32, 8, 128, 16


def _rngs(seed: int, n: int):
    return [np.random.Generator(np.random.PCG64(s)) for s in np.random.SeedSequence(seed).spawn(n)]


def bimodal_lengths(batch: int, rng: np.random.Generator) -> np.ndarray:
    """Half the rows ~U[256,2048], half ~U[16384,32768] (integers, inclusive), then a
    seeded row permutation so long and short rows interleave."""
    short = rng.integers(256, 2048 + 1, size=batch // 2)
    long = rng.integers(16384, 32768 + 1, size=batch - batch // 2)
    lens = np.concatenate([short, long])
    return lens[rng.permutation(batch)].astype(np.int64)


def uniform_lengths(batch: int, rng: np.random.Generator) -> np.ndarray:
    return rng.integers(1024, 32768 + 1, size=batch).astype(np.int64)


def zipf_lengths(batch: int, rng: np.random.Generator) -> np.ndarray:
    k = rng.zipf(1.2, size=batch)
    return np.minimum(32768, 256 * k).astype(np.int64)


def page_table(reserved: np.ndarray, page_size: int, rho: float, rng: np.random.Generator,
               num_pages: int | None = None):
    """Block table per Sec. 3.7.

    Returns (block_table int32 [B, max_pages_per_row], num_pages). Entries past a row's
    reserved pages are -1 (never a valid page id).
    """
    reserved = np.asarray(reserved, dtype=np.int64)
    lp = -(-reserved // page_size)
    total = int(lp.sum())
    universe = int(math.ceil(total / (1.0 - rho))) if rho > 0 else total
    if num_pages is not None:
        if num_pages < total:
            raise ValueError("pool smaller than the reserved pages")
        universe = int(num_pages)
    perm = rng.permutation(universe)
    maxp = max(1, int(lp.max()) if lp.size else 1)
    bt = np.full((reserved.size, maxp), -1, dtype=np.int32)
    off = 0
    for i, n in enumerate(lp):
        bt[i, :n] = perm[off:off + n]
        off += n
    return bt, universe


@dataclasses.dataclass
class Workload:
    name: str
    seq_lens: np.ndarray          # int32 [B], context length at the first step
    steps: int                    # decode steps
    block_table: np.ndarray       # int32 [B, max_pages_per_row]
    num_pages: int
    split_min: int
    split_max: int
    target_tasks: int
    seed: int
    rho: float
    hq: int = HQ
    hkv: int = HKV
    head_dim: int = HEAD_DIM
    page_size: int = PAGE
    tile_tokens: int = 32
    append: bool = True           # each step appends one token per row before attending

    def lengths_at(self, step: int) -> np.ndarray:
        """Context lengths attended at 0-based decode step `step`: the appended token of
        that step is included, so step 0 of a 32768-token prompt attends 32769 tokens."""
        return (self.seq_lens.astype(np.int64) + (step + 1 if self.append else 0)).astype(np.int32)

    @property
    def batch(self) -> int:
        return int(self.seq_lens.size)

    @property
    def max_pages_per_row(self) -> int:
        return int(self.block_table.shape[1])

    def assigned_pages(self) -> np.ndarray:
        bt = self.block_table
        return np.unique(bt[bt >= 0])

    def describe(self) -> dict:
        return {"workload": self.name, "batch": self.batch, "hq": self.hq, "hkv": self.hkv,
                "head_dim": self.head_dim, "page_size": self.page_size,
                "prompt_lens": [int(x) for x in self.seq_lens], "append": self.append, "steps": self.steps,
                "num_pages": self.num_pages, "rho": self.rho, "seed": self.seed,
                "tile_tokens": self.tile_tokens}


def _build(name, lens, steps, rho, seed, rng_pages, num_pages=None, split=(16, 64),
           target_tasks=256, append=True):
    lens = np.asarray(lens, dtype=np.int64)
    reserved = lens + (steps if append else 0)
    bt, universe = page_table(reserved, PAGE, rho, rng_pages, num_pages=num_pages)
    return Workload(name=name, seq_lens=lens.astype(np.int32), steps=steps, block_table=bt,
                    num_pages=universe, split_min=split[0], split_max=split[1],
                    target_tasks=target_tasks, seed=seed, rho=rho, append=append)


def make_workload(name: str, seed: int = 20260622, steps: int | None = None,
                  target_tasks: int = 256, hkv: int = HKV) -> Workload:
    """The benchmark configurations, as concrete seeded inputs. `hkv` changes the number
    of KV heads (Hq stays 32, so G = 32 / hkv); lengths and page tables do not depend on it.

    tiny        : B=1, 512 tokens (no append), pool of 64 pages, one split
    b1          : B=1, 32768 tokens, 4096-page pool, 20 steps
    b8_bimodal  : 8 rows bimodal, rho=0, 50 steps
    b8_uniform  : 8 rows U[1024,32768], rho=0, 50 steps
    b8_zipf     : 8 rows min(32768, 256 k), k~Zipf(1.2), rho=0, 50 steps
    b4_bimodal  : 4 rows bimodal, rho=0, 50 steps
    """
    w = _make(name, seed, steps, target_tasks)
    return w if hkv == w.hkv else dataclasses.replace(w, hkv=hkv)


def _make(name, seed, steps, target_tasks):
    r_len, r_pages = _rngs(seed, 2)
    if name == "tiny":
        return _build(name, [512], 1 if steps is None else steps, 0.0, seed, r_pages,
                      num_pages=64, split=(1, 1), target_tasks=target_tasks, append=False)
    if name == "b1":
        return _build(name, [32768], 20 if steps is None else steps, 0.5, seed, r_pages,
                      num_pages=4096, target_tasks=target_tasks)
    s = 50 if steps is None else steps
    if name == "b8_bimodal":
        return _build(name, bimodal_lengths(8, r_len), s, 0.0, seed, r_pages, target_tasks=target_tasks)
    if name == "b8_uniform":
        return _build(name, uniform_lengths(8, r_len), s, 0.0, seed, r_pages, target_tasks=target_tasks)
    if name == "b8_zipf":
        return _build(name, zipf_lengths(8, r_len), s, 0.0, seed, r_pages, target_tasks=target_tasks)
    if name == "b4_bimodal":
        return _build(name, bimodal_lengths(4, r_len), s, 0.0, seed, r_pages, target_tasks=target_tasks)
    raise KeyError(name)


WORKLOADS = ("tiny", "b1", "b8_bimodal", "b8_uniform", "b8_zipf", "b4_bimodal")
