"""Pins of the reference planner: a hand-worked example, the partition and non-emptiness
properties the workqueue must have (Sec. 3.3-3.4), the closed-form task count, and the
counters the paper prints in Tab. 4."""
import json
import os

import numpy as np
import pytest

from oracle import PlanParams, choose_split_count, ref_plan

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def test_hand_worked_example():
    # T = 32, Hkv = 2, S forced to 2.
    # lengths 0, 1, 33, 100, 64 -> tiles 0, 1, 2, 4, 2 -> nsplit 0, 1, 2, 2, 2
    # row 1: tiles [0,1)            -> tokens [0,1)
    # row 2: tiles [0,1) [1,2)      -> tokens [0,32) [32,33)
    # row 3: tiles [0,2) [2,4)      -> tokens [0,64) [64,100)
    # row 4: tiles [0,1) [1,2)      -> tokens [0,32) [32,64)
    p = PlanParams(num_kv_heads=2, split_min=2, split_max=2)
    tasks, offs, S = ref_plan([0, 1, 33, 100, 64], p)
    assert S == 2
    assert offs.tolist() == [0, 0, 1, 3, 5, 7]
    expect = []
    for (i, s, t0, t1) in [(1, 0, 0, 1), (2, 0, 0, 32), (2, 1, 32, 33), (3, 0, 0, 64),
                           (3, 1, 64, 100), (4, 0, 0, 32), (4, 1, 32, 64)]:
        for g in range(2):
            expect.append([i, g, s, t0, t1])
    assert tasks.tolist() == expect


def test_balanced_bounds_three_splits_of_seven_tiles():
    # 7 tiles over 3 splits: floor(s*7/3) = 0, 2, 4, 7 -> 2, 2, 3 tiles.
    p = PlanParams(num_kv_heads=1, split_min=3, split_max=3)
    tasks, _, _ = ref_plan([7 * 32 - 5], p)
    assert tasks[:, 3:].tolist() == [[0, 64], [64, 128], [128, 219]]


@pytest.mark.parametrize("policy", [0, 1])
@pytest.mark.parametrize("seed", range(6))
def test_partition_properties(seed, policy):
    r = np.random.Generator(np.random.PCG64(seed))
    B = int(r.integers(1, 12))
    lens = r.integers(0, 5000, size=B)
    lens[r.random(B) < 0.2] = 0
    lo = int(r.integers(1, 8))
    p = PlanParams(num_kv_heads=int(r.integers(1, 9)), split_min=lo, split_max=lo + int(r.integers(0, 40)),
                   target_tasks=int(r.integers(1, 3000)), policy=policy)
    tasks, offs, S = ref_plan(lens, p)
    T = p.tile_tokens
    if policy == 0:
        assert p.split_min <= S <= p.split_max
    # brute force over every (row, kv head): the tasks tile [0, N) in split order
    for i, n in enumerate(lens):
        tiles = -(-int(n) // T)
        ns = offs[i + 1] - offs[i]
        if policy == 0:
            assert ns == min(S, tiles)
        else:  # S holds the tile quota Q: no split exceeds it unless split_max binds
            assert ns == min(p.split_max, -(-tiles // S))
            assert ns == 0 or ns == p.split_max or -(-tiles // ns) <= S
        for g in range(p.num_kv_heads):
            mine = [t for t in tasks.tolist() if t[0] == i and t[1] == g]
            assert [t[2] for t in mine] == list(range(ns))
            pos = 0
            sizes = []
            for (_, _, s, t0, t1) in mine:
                assert t0 == pos and t1 > t0 and t0 % T == 0
                assert t1 % T == 0 or t1 == n
                sizes.append(-(-(t1 - t0) // T))
                pos = t1
            assert pos == n
            if sizes:
                assert max(sizes) - min(sizes) <= 1
                assert max(sizes) == -(-tiles // ns)
    # closed-form count and slot order (row, split, kv head) with kv head fastest
    if policy == 0:
        assert len(tasks) == p.num_kv_heads * sum(min(S, -(-int(n) // T)) for n in lens)
    else:  # the quota is the smallest that fits the target (or one split per row)
        def count(q):
            return p.num_kv_heads * sum(min(p.split_max, -(-(-(-int(n) // T)) // q)) for n in lens)
        assert len(tasks) == count(S)
        if S > 1:
            assert count(S - 1) > p.target_tasks
        assert len(tasks) <= p.target_tasks or len(tasks) == p.num_kv_heads * sum(1 for n in lens if n > 0)
    for k, (i, g, s, _, _) in enumerate(tasks.tolist()):
        assert k == (offs[i] + s) * p.num_kv_heads + g


def test_quota_policy_hand_worked():
    # Hkv 2, target 8 -> at most 4 splits summed over rows; tiles 32, 4, 0, 94.
    # Q = 32: splits 1, 1, 0, 3 = 5 (too many); Q = 47: 1, 1, 0, 2 = 4 fits, and every
    # Q in 33..46 still gives ceil(94/Q) = 3 -> Q = 47.
    p = PlanParams(num_kv_heads=2, split_min=2, split_max=64, target_tasks=8, policy=1)
    tasks, offs, Q = ref_plan([1000, 100, 0, 3000], p)
    assert Q == 47 and offs.tolist() == [0, 1, 2, 2, 4]
    # row 3: floor(s*94/2) = 0, 47, 94 tiles
    assert tasks[tasks[:, 0] == 3][::2, 3:].tolist() == [[0, 1504], [1504, 3000]]
    # one 32K row, target 512 over 8 heads: at most 64 splits; split_max = 64 caps the
    # row already at Q = 1, so Q = 1 and the row gets 64 splits
    _, offs, Q = ref_plan([32769], PlanParams(policy=1))
    assert Q == 1 and offs[1] == 64
    # with split_max 100 the cap no longer binds: Q = ceil(1025/64) = 17 -> 61 splits
    _, offs, Q = ref_plan([32769], PlanParams(policy=1, split_max=100))
    assert Q == 17 and offs[1] == 61
    # a target below one split per row: every non-empty row keeps one split
    tasks, offs, Q = ref_plan([40, 900, 0], PlanParams(num_kv_heads=8, target_tasks=8, policy=1))
    assert offs.tolist() == [0, 1, 2, 2] and Q == 29


def test_quota_policy_balances_task_sizes():
    lens = [1000, 30000, 500, 20000, 2000, 17000, 300, 25000]
    p = PlanParams(policy=1)
    tasks, _, Q = ref_plan(lens, p)
    tiles = (tasks[:, 4] - tasks[:, 3] + 31) // 32
    assert tiles.max() <= Q
    # a row with ns = ceil(t / Q) splits has t > Q (ns - 1) tiles, so no piece is smaller
    # than floor(Q (ns - 1) / ns): long rows are cut into pieces close to Q
    for i in (1, 3, 5, 7):
        mine = tiles[tasks[:, 0] == i]
        ns = len(mine) // 8
        assert ns > 10 and mine.min() >= (Q * (ns - 1)) // ns


def test_split_count_rule():
    p = PlanParams()  # Hkv 8, bounds [16, 64], target 512
    assert choose_split_count([32769], p) == 64            # 512 / 8 = 64
    assert choose_split_count([1000] * 8, p) == 16         # 512 / 64 = 8 -> clamped up to 16
    assert choose_split_count([1000] * 3 + [0] * 5, p) == 22  # ceil(512 / 24)
    assert choose_split_count([0, 0], p) == 64             # no active row: 512 / max(1, 0)
    assert choose_split_count([1] * 200, p) == 16


def test_tiny_config_has_eight_tasks():
    tasks, offs, S = ref_plan([512], PlanParams(split_min=1, split_max=1))
    assert S == 1 and len(tasks) == 8 and offs.tolist() == [0, 1]
    assert tasks[:, 3:].tolist() == [[0, 512]] * 8


def test_b1_steps_give_512_tasks_and_a_17_tile_split():
    p = PlanParams()
    for n in range(32769, 32789):
        tasks, _, S = ref_plan([n], p)
        assert S == 64 and len(tasks) == 512
        tiles = (tasks[:, 4] - tasks[:, 3] + 31) // 32
        assert sorted(set(tiles.tolist())) == [16, 17]  # 1025 tiles over 64 splits


def test_tab4_counters():
    g = json.load(open(os.path.join(GOLDEN, "tab4_counters.json")))
    G, d = g["shape"]["hq"] // g["shape"]["hkv"], g["shape"]["head_dim"]
    state_bytes = 4 * (G * d + 2 * G)          # fp32 acc[G][d], m[G], l[G] per task
    assert state_bytes == 2080
    lens = [640, 700, 2000, 17000, 30000, 900, 25000, 32768]  # every row >= 20 tiles
    wq = g["workqueue"]
    tasks, _, S = ref_plan(lens, PlanParams(split_min=wq["split"], split_max=wq["split"]))
    assert round(len(tasks) / g["sms"], 1) == wq["decode_cta_work_per_sm"]
    assert round(len(tasks) * state_bytes / 2**20, 2) == wq["merge_mb"]
    bk = g["buckets"]
    slots = g["shape"]["batch"] * g["shape"]["hkv"] * bk["split"]   # rectangular grid
    assert round(slots / g["sms"], 1) == bk["decode_cta_work_per_sm"]
    assert round(slots * state_bytes / 2**20, 2) == bk["merge_mb"]


def test_invalid_inputs_raise():
    with pytest.raises(ValueError):
        ref_plan([100], PlanParams(), max_pages_per_row=6)   # 6 pages hold 96 tokens
    with pytest.raises(ValueError):
        ref_plan([-1], PlanParams())
    with pytest.raises(ValueError):
        ref_plan([10], PlanParams(tile_tokens=24))
    with pytest.raises(ValueError):
        ref_plan([10], PlanParams(split_min=5, split_max=4))
