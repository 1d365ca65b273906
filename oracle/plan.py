"""Reference compact-workqueue planner (Sec. 3.3-3.4), integers only.

TEST INFRASTRUCTURE: see the package docstring. Parity pins: tests/test_oracle_plan.py.

The paper fixes what a task is and when one exists: a task (row, kv head, split,
t_begin, t_end) is emitted only when its tile interval is non-empty (Sec. 3.4), split
ranges come from the row-local length N*_i = seq_lens[i] (Sec. 3.3), tiles are 32
tokens (Sec. 3.2), and the workqueue's split count depends on the active batch size
and the row's tile count (Sec. 3.5). It leaves the split-count formula and the split
boundaries open; the readings taken here are:

  tiles_i   = ceil(N_i / T)
  policy 0 (batch split count, the default):
    S         = clamp(ceil(target_tasks / max(1, B_act * Hkv)), split_min, split_max),
                B_act = number of rows with N_i > 0
    nsplit_i  = min(S, tiles_i)                    (0 for an empty row)
  policy 1 (tile quota: per-row split counts from the batch's total work, so that
            every task covers about the same number of tiles):
    nsplit_i(Q) = min(split_max, ceil(tiles_i / Q))   (0 for an empty row)
    Q         = the smallest Q >= 1 with Hkv * sum_i nsplit_i(Q) <= target_tasks, or
                max_i tiles_i when no Q meets it (one split per row); split_min is
                not used
  split s of row i owns tiles [b_s, b_{s+1}),  b_s = floor(s * tiles_i / nsplit_i)
  task      = (i, g, s, b_s*T, min(b_{s+1}*T, N_i)),  for s < nsplit_i, g < Hkv
  order     = lexicographic in (row, split, kv head), kv head fastest; the task's index
              is also its partial-state slot
  split_offsets[0] = 0,  split_offsets[i+1] = split_offsets[i] + nsplit_i
"""
from __future__ import annotations

import dataclasses

import numpy as np


@dataclasses.dataclass(frozen=True)
class PlanParams:
    page_size: int = 16
    tile_tokens: int = 32
    num_kv_heads: int = 8
    split_min: int = 16
    split_max: int = 64
    target_tasks: int = 512
    policy: int = 0


def _ceil_div(a: int, b: int) -> int:
    return -(-a // b)


def choose_split_count(seq_lens, p: PlanParams) -> int:
    """Workqueue split count S from the active batch size (Sec. 3.5), policy 0."""
    active = sum(1 for n in seq_lens if int(n) > 0)
    s = _ceil_div(p.target_tasks, max(1, active * p.num_kv_heads))
    return int(min(max(s, p.split_min), p.split_max))


def tile_quota(seq_lens, p: PlanParams) -> int:
    """Tiles per split Q of policy 1: the smallest quota whose task count fits
    target_tasks (plain upward search; the count only falls as Q grows)."""
    tiles = [_ceil_div(int(n), p.tile_tokens) for n in seq_lens]
    tmax = max(tiles, default=0)
    for q in range(1, max(tmax, 1) + 1):
        count = sum(min(p.split_max, _ceil_div(t, q)) for t in tiles)
        if p.num_kv_heads * count <= p.target_tasks:
            return q
    return max(tmax, 1)


def row_split_counts(seq_lens, p: PlanParams):
    """(nsplit per row, the policy's scalar: S for policy 0, Q for policy 1)."""
    tiles = [_ceil_div(int(n), p.tile_tokens) for n in seq_lens]
    if p.policy == 0:
        S = choose_split_count(seq_lens, p)
        return [min(S, t) for t in tiles], S
    Q = tile_quota(seq_lens, p)
    return [min(p.split_max, _ceil_div(t, Q)) for t in tiles], Q


def row_split_bounds(n: int, nsplit_cap: int, tile_tokens: int):
    """Token bounds [(t_begin, t_end)] of the non-empty splits of one row of length n
    cut into min(nsplit_cap, tiles) balanced tile ranges."""
    tiles = _ceil_div(int(n), tile_tokens)
    k = min(int(nsplit_cap), tiles)
    out = []
    for s in range(k):
        b0 = (s * tiles) // k
        b1 = ((s + 1) * tiles) // k
        out.append((b0 * tile_tokens, min(b1 * tile_tokens, int(n))))
    return out


def _validate(seq_lens, p: PlanParams, max_pages_per_row: int | None):
    if p.tile_tokens <= 0 or p.tile_tokens % p.page_size:
        raise ValueError("tile_tokens must be a positive multiple of page_size")
    if not (1 <= p.split_min <= p.split_max):
        raise ValueError("need 1 <= split_min <= split_max")
    if p.policy not in (0, 1):
        raise ValueError("unknown split policy")
    for n in seq_lens:
        if int(n) < 0:
            raise ValueError("negative sequence length")
        if max_pages_per_row is not None and int(n) > max_pages_per_row * p.page_size:
            raise ValueError("sequence length exceeds the block table's capacity")


def ref_plan(seq_lens, p: PlanParams, max_pages_per_row: int | None = None):
    """Returns (tasks int32 [num_tasks, 5], split_offsets int32 [B+1], S or Q)."""
    seq_lens = [int(x) for x in np.asarray(seq_lens).reshape(-1)]
    _validate(seq_lens, p, max_pages_per_row)
    nsplit, S = row_split_counts(seq_lens, p)
    tasks = []
    offsets = [0]
    for i, n in enumerate(seq_lens):
        bounds = row_split_bounds(n, nsplit[i], p.tile_tokens)
        for s, (t0, t1) in enumerate(bounds):
            for g in range(p.num_kv_heads):
                tasks.append((i, g, s, t0, t1))
        offsets.append(offsets[-1] + len(bounds))
    t = np.asarray(tasks, dtype=np.int32).reshape(-1, 5)
    return t, np.asarray(offsets, dtype=np.int32), S
