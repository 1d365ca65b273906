"""GPU parity of the HIP path (through the C ABI) against the fp64 oracle.

Bars: the task list is bit-exact against ref_plan; outputs are within max abs 2e-3 and
normwise rel 1e-2 of ref_decode; routes that must agree bitwise (fused vs two-kernel
merge, workqueue vs rectangular grid at the same split count, physical page
permutation, one-token context) are compared with torch.equal. Unowned pool pages and
the partial-state workspace are NaN before every call, so a stray read or an
unwritten slot shows up."""
import numpy as np
import pytest
import torch

import paper_2606_26666_amd as pkv
from oracle import PlanParams, ref_decode, ref_decode_rect, ref_plan
from tests.gpu_cases import (Case, assert_close, error_stats, plan_params, read_plan, run_decode, run_plan,
                             run_rect)

pytestmark = pytest.mark.gpu

RAGGED = [1, 15, 16, 17, 31, 32, 33, 100, 517, 1000, 2049, 0, 4000]


def bufs_for(case, split_max=64, rect_splits=0):
    return pkv.DecodeBuffers(case.B, case.hq, case.hkv, case.d, split_max, "cuda", rect_splits=rect_splits)


def oracle_plan(case, p):
    return ref_plan(case.lens, PlanParams(p.page_size, p.tile_tokens, p.num_kv_heads, p.split_min, p.split_max,
                                          p.target_tasks, p.policy), max_pages_per_row=case.bt.shape[1])


@pytest.mark.parametrize("smin,smax,target,policy", [(16, 64, 512, 0), (1, 1, 512, 0), (2, 7, 100, 0),
                                                     (3, 64, 4096, 0), (16, 64, 512, 1), (2, 7, 100, 1)])
def test_plan_bit_exact_ragged(smin, smax, target, policy):
    case = Case(RAGGED, seed=1)
    p = plan_params(8, smin, smax, target, policy=policy)
    bufs = bufs_for(case, smax)
    run_plan(case, bufs, p, check_pages=True)
    tasks, offs = read_plan(bufs)
    rt, ro, _ = oracle_plan(case, p)
    assert np.array_equal(tasks, rt)
    assert np.array_equal(offs, ro)
    assert pkv.pkv_check_device_status(bufs.ws) == 0


@pytest.mark.parametrize("policy", [0, 1])
@pytest.mark.parametrize("seed", range(4))
def test_plan_bit_exact_random_batches(seed, policy):
    r = np.random.Generator(np.random.PCG64(100 + seed))
    B = int(r.integers(1, 1500))
    lens = r.integers(0, 3000, size=B).astype(np.int32)
    lens[r.random(B) < 0.3] = 0
    case = Case(lens, hkv=int(r.choice([1, 2, 4, 8])), hq=8, seed=seed, rho=0.0, values=False)
    p = plan_params(case.hkv, int(r.integers(1, 4)), int(r.integers(4, 40)), int(r.integers(1, 20000)),
                    policy=policy)
    bufs = bufs_for(case, p.split_max)
    run_plan(case, bufs, p)
    tasks, offs = read_plan(bufs)
    rt, ro, _ = oracle_plan(case, p)
    assert np.array_equal(tasks, rt) and np.array_equal(offs, ro)


@pytest.mark.parametrize("policy", [0, 1])
@pytest.mark.parametrize("B", [1, 2, 7, 33, 63, 64])
def test_plan_bit_exact_small_batches(B, policy):
    """Batches of up to 64 rows take the planner's one-wave path (no block-table check)."""
    r = np.random.Generator(np.random.PCG64(300 + B + 1000 * policy))
    lens = r.integers(0, 40000, size=B).astype(np.int32)
    lens[r.random(B) < 0.25] = 0
    if B == 33:
        lens[:] = 0   # nothing active
    case = Case(lens, hkv=8, hq=32, seed=B, rho=0.0, values=False)
    for smin, smax, target in [(16, 64, 512), (1, 1, 512), (2, 9, 37), (1, 300, 100000)]:
        p = plan_params(8, smin, smax, target, policy=policy)
        bufs = bufs_for(case, smax)
        run_plan(case, bufs, p)
        tasks, offs = read_plan(bufs)
        rt, ro, _ = oracle_plan(case, p)
        assert np.array_equal(tasks, rt) and np.array_equal(offs, ro), (smin, smax, target)
        assert pkv.pkv_check_device_status(bufs.ws) == 0


@pytest.mark.parametrize("fused", [True, False])
@pytest.mark.parametrize("hq,hkv", [(32, 8), (8, 8), (16, 8), (32, 4)])
def test_decode_ragged_matches_oracle(fused, hq, hkv):
    case = Case(RAGGED, hq=hq, hkv=hkv, seed=2)
    p = plan_params(hkv, 2, 16, 64)
    bufs = bufs_for(case, 16)
    run_plan(case, bufs, p)
    out = run_decode(case, bufs, fused=fused)
    ref = ref_decode(case.q, case.k, case.v, case.bt, case.lens)
    assert_close(out, ref, f"G={hq // hkv} fused={fused}")
    assert torch.all(out[11] == 0)  # the empty row
    assert pkv.pkv_check_device_status(bufs.ws) == 0


def test_sm_scale_is_applied():
    case = Case([300, 77], seed=3)
    bufs = bufs_for(case)
    run_plan(case, bufs, plan_params(8, 1, 4, 16))
    out = run_decode(case, bufs, sm_scale=0.3)
    assert_close(out, ref_decode(case.q, case.k, case.v, case.bt, case.lens, 0.3), "scale 0.3")


def test_fused_equals_two_kernel_merge_bitwise():
    case = Case(RAGGED, seed=4)
    bufs = bufs_for(case)
    run_plan(case, bufs, plan_params(8, 4, 64, 700))
    a = run_decode(case, bufs, fused=True)
    b = run_decode(case, bufs, fused=False)
    assert torch.equal(a, b)


@pytest.mark.parametrize("S", [1, 3, 16, 64])
def test_workqueue_equals_rectangular_bitwise(S):
    case = Case(RAGGED, seed=5)
    bufs = bufs_for(case, split_max=S, rect_splits=S)
    run_plan(case, bufs, plan_params(8, S, S, 1))
    wq = run_decode(case, bufs, fused=True)
    rect = run_rect(case, bufs, S)
    assert torch.equal(wq, rect)
    assert_close(rect, ref_decode_rect(case.q, case.k, case.v, case.bt, case.lens, S, 32), f"rect S={S}")


def test_physical_page_permutation_is_bitwise_invariant():
    lens = [700, 33, 1600]
    a = Case(lens, seed=6, rho=0.5)
    # same logical K/V, different physical pages
    r = np.random.Generator(np.random.PCG64(60))
    perm = r.permutation(a.num_pages)
    bt2 = np.where(a.bt >= 0, perm[np.maximum(a.bt, 0)], -1).astype(np.int32)
    k2 = np.empty_like(a.k)
    v2 = np.empty_like(a.v)
    k2[perm] = a.k
    v2[perm] = a.v
    b = Case(lens, seed=6, rho=0.5)
    b.bt, b.k, b.v = bt2, k2, v2
    b.bt_dev, b.k_dev, b.v_dev = (torch.from_numpy(x).cuda() for x in (bt2, k2, v2))
    outs = []
    for c in (a, b):
        bufs = bufs_for(c)
        run_plan(c, bufs, plan_params(8))
        outs.append(run_decode(c, bufs))
    assert torch.equal(outs[0], outs[1])


def test_one_token_context_returns_v_exactly():
    case = Case([1, 1, 1, 1], seed=7)
    bufs = bufs_for(case)
    run_plan(case, bufs, plan_params(8))
    out = run_decode(case, bufs).cpu().numpy()
    for i in range(4):
        v0 = case.v[case.bt[i, 0], 0]            # [Hkv, d]
        assert np.array_equal(out[i], np.repeat(v0, 4, axis=0))


def test_all_rows_empty_gives_zeros():
    case = Case([0, 0, 0], seed=8)
    for fused in (True, False):
        bufs = bufs_for(case)
        run_plan(case, bufs, plan_params(8))
        assert int(bufs.num_tasks.item()) == 0
        out = run_decode(case, bufs, fused=fused)
        assert torch.all(out == 0)


def test_repeated_fused_calls_are_identical():
    case = Case([5000, 3000, 40, 9000], seed=9)
    bufs = bufs_for(case)
    run_plan(case, bufs, plan_params(8, 16, 64, 2048))
    first = run_decode(case, bufs, poison_ws=False)
    for _ in range(200):
        again = run_decode(case, bufs, poison_ws=False)
        assert torch.equal(first, again)
    assert_close(first, ref_decode(case.q, case.k, case.v, case.bt, case.lens), "repeat")


def test_sequence_longer_than_block_table_is_flagged_and_zeroed():
    case = Case([100, 50], seed=10)
    lens_bad = case.lens.copy()
    lens_bad[1] = case.bt.shape[1] * 16 + 1
    case.lens_dev = torch.from_numpy(lens_bad).cuda()
    bufs = bufs_for(case)
    run_plan(case, bufs, plan_params(8))
    out = run_decode(case, bufs)
    assert pkv.pkv_check_device_status(bufs.ws) & pkv.PKV_DEVERR_SEQ_LEN
    assert torch.all(out[1] == 0)
    good = ref_decode(case.q[:1], case.k, case.v, case.bt[:1], case.lens[:1])
    assert_close(out[:1], good, "row 0")
    assert pkv.pkv_check_device_status(bufs.ws) == 0  # cleared by the previous read


def test_bad_page_id_is_flagged_and_row_zeroed():
    case = Case([100, 200], seed=11)
    bt_bad = case.bt.copy()
    bt_bad[0, 3] = case.num_pages + 7
    case.bt_dev = torch.from_numpy(bt_bad).cuda()
    for fused in (True, False):
        bufs = bufs_for(case)
        run_plan(case, bufs, plan_params(8))
        out = run_decode(case, bufs, fused=fused)
        assert pkv.pkv_check_device_status(bufs.ws) & pkv.PKV_DEVERR_PAGE_ID
        assert torch.all(out[0] == 0)
        assert_close(out[1:], ref_decode(case.q[1:], case.k, case.v, case.bt[1:], case.lens[1:]), "row 1")
    # the planner's optional page check drops the row up front
    bufs = bufs_for(case)
    run_plan(case, bufs, plan_params(8), check_pages=True)
    tasks, offs = read_plan(bufs)
    assert offs[1] == 0 and np.all(tasks[:, 0] == 1)
    assert pkv.pkv_check_device_status(bufs.ws) & pkv.PKV_DEVERR_PAGE_ID


@pytest.mark.parametrize("policy", [0, 1])
@pytest.mark.parametrize("name", ["tiny", "b1", "b8_bimodal", "b8_uniform", "b8_zipf", "b4_bimodal"])
def test_benchmark_configs_full_size(name, policy):
    """Every output of the first decode step of each benchmark configuration, in the
    launch configuration the benchmark times (planner + fused kernel)."""
    case, w = Case.from_workload(name)
    p = plan_params(w.hkv, w.split_min, w.split_max, w.target_tasks, w.tile_tokens, policy=policy)
    bufs = bufs_for(case, w.split_max)
    run_plan(case, bufs, p)
    tasks, offs = read_plan(bufs)
    rt, ro, _ = oracle_plan(case, p)
    assert np.array_equal(tasks, rt) and np.array_equal(offs, ro)
    out = run_decode(case, bufs)
    ref = ref_decode(case.q, case.k, case.v, case.bt, case.lens)
    assert_close(out, ref, name)
    amax, mean, ulp = error_stats(out, ref)
    print(f"{name} policy {policy}: max|e| {amax:.3e} mean|e| {mean:.3e} within 1 ulp {ulp:.4f}")
    assert ulp > 0.99
    assert pkv.pkv_check_device_status(bufs.ws) == 0


def test_b1_last_step_and_uniform_rect():
    case, w = Case.from_workload("b1", step=19)
    bufs = bufs_for(case, w.split_max)
    run_plan(case, bufs, plan_params(w.hkv, w.split_min, w.split_max, w.target_tasks))
    out = run_decode(case, bufs)
    assert_close(out, ref_decode(case.q, case.k, case.v, case.bt, case.lens), "b1 step 19")
    case, w = Case.from_workload("b8_uniform")
    bufs = bufs_for(case, 16, rect_splits=16)
    run_plan(case, bufs, plan_params(w.hkv, 16, 16, 1))
    wq = run_decode(case, bufs)
    rect = run_rect(case, bufs, 16)
    assert torch.equal(wq, rect)


def run_plan_decode(case, bufs, params, sm_scale=1.0):
    bufs.partial_region().fill_(0xFF)
    out = torch.full((case.B, case.hq, case.d), float("nan"), dtype=torch.float16, device="cuda")
    pkv.pkv_plan_decode(case.q_dev, case.k_dev, case.v_dev, case.bt_dev, case.lens_dev, params, bufs.tasks,
                        bufs.split_offsets, bufs.num_tasks, sm_scale, out, bufs.ws)
    return out


@pytest.mark.parametrize("policy", [0, 1])
def test_plan_decode_one_launch_equals_plan_then_decode(policy):
    case = Case(RAGGED, seed=12)
    p = plan_params(8, 2, 16, 300, policy=policy)
    ref_bufs = bufs_for(case, 16)
    run_plan(case, ref_bufs, p)
    expect = run_decode(case, ref_bufs)
    tasks_ref, offs_ref = read_plan(ref_bufs)
    bufs = bufs_for(case, 16)
    bufs.tasks.fill_(-7)
    got = run_plan_decode(case, bufs, p)
    tasks, offs = read_plan(bufs)
    assert torch.equal(got, expect)
    assert np.array_equal(tasks, tasks_ref) and np.array_equal(offs, offs_ref)
    assert np.array_equal(tasks, oracle_plan(case, p)[0])
    assert pkv.pkv_check_device_status(bufs.ws) == 0


def test_plan_decode_repeated_and_changing_lengths():
    case = Case([3000, 70, 0, 12000], seed=13)
    p = plan_params(8, 16, 64, 512)
    bufs = bufs_for(case)
    first = run_plan_decode(case, bufs, p)
    assert_close(first, ref_decode(case.q, case.k, case.v, case.bt, case.lens), "plan_decode")
    for i in range(100):
        again = run_plan_decode(case, bufs, p)
        assert torch.equal(first, again), i
    # lengths change between calls on the same workspace: the plan follows them
    lens2 = np.array([2990, 1, 10, 11000], dtype=np.int32)  # row 2 owns one page
    case.lens_dev = torch.from_numpy(lens2).cuda()
    out2 = run_plan_decode(case, bufs, p)
    assert_close(out2, ref_decode(case.q, case.k, case.v, case.bt, lens2), "new lengths")
    tasks, _ = read_plan(bufs)
    assert np.array_equal(tasks, ref_plan(lens2, PlanParams(split_min=16, split_max=64, target_tasks=512),
                                          max_pages_per_row=case.bt.shape[1])[0])
    assert pkv.pkv_check_device_status(bufs.ws) == 0


@pytest.mark.parametrize("name", ["b1", "b8_bimodal", "b8_uniform", "b8_zipf", "b4_bimodal"])
def test_plan_decode_benchmark_configs(name):
    case, w = Case.from_workload(name)
    p = plan_params(w.hkv, w.split_min, w.split_max, w.target_tasks, w.tile_tokens)
    bufs = bufs_for(case, w.split_max)
    out = run_plan_decode(case, bufs, p)
    assert_close(out, ref_decode(case.q, case.k, case.v, case.bt, case.lens), name)
    tasks, _ = read_plan(bufs)
    assert np.array_equal(tasks, oracle_plan(case, p)[0])


@pytest.mark.parametrize("name,hkv", [("b1", 32), ("b1", 4), ("b8_bimodal", 32), ("b8_bimodal", 4),
                                      ("b8_uniform", 16), ("b4_bimodal", 32)])
def test_plan_decode_gqa_mappings_full_size(name, hkv):
    """G = 1, 2 and 8 on the benchmark lengths, one launch, with the task target the
    bench uses (the cost model's rule: 1024 tasks for B8 at 32 KV heads, so workgroups
    loop over several tasks after their speculative first one)."""
    from paper_2606_26666_amd import costmodel
    case, w = Case.from_workload(name, hkv=hkv)
    target = costmodel.default_target(case.lens, w.hkv)
    p = plan_params(w.hkv, w.split_min, w.split_max, target, w.tile_tokens, policy=1)
    bufs = bufs_for(case, w.split_max)
    out = run_plan_decode(case, bufs, p)
    assert_close(out, ref_decode(case.q, case.k, case.v, case.bt, case.lens), f"{name} G={32 // hkv}")
    tasks, _ = read_plan(bufs)
    assert np.array_equal(tasks, oracle_plan(case, p)[0])
    again = run_plan_decode(case, bufs, p)  # every first task now starts from its hint
    assert torch.equal(again, out)
    assert pkv.pkv_check_device_status(bufs.ws) == 0


def test_rect_named_rows_reads_and_writes_by_index():
    case = Case(RAGGED, seed=14)
    bufs = bufs_for(case, 16, rect_splits=16)
    ids = [12, 0, 7]
    out = run_rect(case, bufs, 16, row_ids=ids)
    full = run_rect(case, bufs, 16)
    others = [i for i in range(case.B) if i not in ids]
    assert torch.equal(out[ids], full[ids])
    assert torch.all(torch.isnan(out[others].float()))  # rows not named are untouched


def test_exact_length_buckets_match_rectangular_grid():
    case = Case(RAGGED, seed=15)   # every length distinct: one row per bucket, S = 64
    p = plan_params(8, 16, 64, 512)
    bufs = bufs_for(case, 64)
    out = torch.full((case.B, case.hq, case.d), float("nan"), dtype=torch.float16, device="cuda")
    launches = pkv.pkv_decode_buckets(case.q_dev, case.k_dev, case.v_dev, case.bt_dev, case.lens_dev, case.lens,
                                      0, p, 1.0, out, bufs.ws)
    assert launches == 2 * len(set(case.lens.tolist()))
    assert torch.equal(out, run_rect(case, bufs, 64))
    assert_close(out, ref_decode(case.q, case.k, case.v, case.bt, case.lens), "exact buckets")


def test_coarse_buckets_on_benchmark_config():
    case, w = Case.from_workload("b8_bimodal")
    p = plan_params(w.hkv, w.split_min, w.split_max, w.target_tasks)
    bufs = bufs_for(case, w.split_max)
    out = torch.full((case.B, case.hq, case.d), float("nan"), dtype=torch.float16, device="cuda")
    launches = pkv.pkv_decode_buckets(case.q_dev, case.k_dev, case.v_dev, case.bt_dev, case.lens_dev, case.lens,
                                      16384, p, 1.0, out, bufs.ws)
    groups = len({-(-int(n) // 16384) for n in case.lens})
    assert launches == 2 * groups
    assert_close(out, ref_decode(case.q, case.k, case.v, case.bt, case.lens), "coarse buckets")
    assert pkv.pkv_check_device_status(bufs.ws) == 0


def _two_launch(case, p, split_max):
    """Plan kernel, then the fused decode kernel: the route without a speculative start."""
    bufs = bufs_for(case, split_max)
    run_plan(case, bufs, p)
    out = run_decode(case, bufs)
    tasks, offs = read_plan(bufs)
    return out, tasks, offs


@pytest.mark.parametrize("policy,target", [(0, 200), (1, 200), (0, 600), (1, 520)])
def test_plan_decode_hints_never_change_results(policy, target):
    """The one-launch route starts each workgroup on the task that the previous call
    listed at the workgroup's index. Whatever the task buffer holds (garbage, plausible
    but wrong records, the right records at the wrong slots, the exact plan), outputs
    and the task list are bitwise those of the route without that start. Targets of 512
    and more run KV-head pairs, whose hint is the record at twice the index."""
    case = Case([900, 0, 17, 4096, 33, 2500, 1, 700], seed=21)
    p = plan_params(8, 2, 16, target, policy=policy)
    expect, tasks_ref, offs_ref = _two_launch(case, p, 16)
    assert np.array_equal(tasks_ref, oracle_plan(case, p)[0])
    r = np.random.Generator(np.random.PCG64(5))
    bufs = bufs_for(case, 16)
    cap = bufs.tasks.shape[0]
    maxp = case.bt.shape[1]
    garbage = r.integers(-(1 << 30), 1 << 30, size=(cap, 5), dtype=np.int64).astype(np.int32)
    plausible = np.zeros((cap, 5), dtype=np.int32)
    plausible[:, 0] = r.integers(0, case.B, size=cap)
    plausible[:, 1] = r.integers(0, 8, size=cap)
    plausible[:, 3] = 16 * r.integers(0, maxp, size=cap)
    plausible[:, 4] = np.minimum(plausible[:, 3] + r.integers(1, 600, size=cap), maxp * 16)
    shuffled = np.zeros((cap, 5), dtype=np.int32)
    shuffled[:len(tasks_ref)] = tasks_ref[r.permutation(len(tasks_ref))]
    exact = np.zeros((cap, 5), dtype=np.int32)
    exact[:len(tasks_ref)] = tasks_ref
    for label, hint in [("garbage", garbage), ("plausible", plausible), ("shuffled", shuffled), ("exact", exact)]:
        bufs.tasks.copy_(torch.from_numpy(hint).view(bufs.tasks.dtype).reshape(bufs.tasks.shape).cuda())
        got = run_plan_decode(case, bufs, p)
        tasks, offs = read_plan(bufs)
        assert torch.equal(got, expect), label
        assert np.array_equal(tasks, tasks_ref) and np.array_equal(offs, offs_ref), label
        assert pkv.pkv_check_device_status(bufs.ws) == 0, label


@pytest.mark.parametrize("target", [256, 512])
def test_plan_decode_speculation_across_growing_steps(target):
    """Decode steps with every row one token longer than at the previous step (pages and
    tiles fill and new ones start), one workspace throughout: each step's output is bitwise
    that of the two-launch route, and its task list is the oracle's (target 512: KV-head
    pairs)."""
    base = np.array([1000, 15, 4063, 31, 300, 2047, 64, 9000], dtype=np.int32)
    steps = 40
    case = Case(base + steps, seed=22)
    p = plan_params(8, 1, 64, target, policy=1)
    bufs = bufs_for(case, 64)
    for s in range(steps + 1):
        lens = base + s
        case.lens = lens
        case.lens_dev = torch.from_numpy(lens).cuda()
        expect, tasks_ref, _ = _two_launch(case, p, 64)
        got = run_plan_decode(case, bufs, p)
        tasks, _ = read_plan(bufs)
        assert torch.equal(got, expect), s
        assert np.array_equal(tasks, tasks_ref), s
        if s % 13 == 0:
            assert np.array_equal(tasks, oracle_plan(case, p)[0]), s
            assert_close(got, ref_decode(case.q, case.k, case.v, case.bt, lens), f"step {s}")
    assert pkv.pkv_check_device_status(bufs.ws) == 0


def test_plan_decode_batch_above_one_wave():
    """More than 64 rows: the one-launch route plans with the workgroup-wide planner and
    starts no task early. Twice on one workspace."""
    r = np.random.Generator(np.random.PCG64(23))
    lens = r.integers(0, 700, size=80).astype(np.int32)
    lens[::9] = 0
    case = Case(lens, seed=23)
    p = plan_params(8, 1, 4, 600, policy=1)
    ref = ref_decode(case.q, case.k, case.v, case.bt, case.lens)
    bufs = bufs_for(case, 4)
    for rep in range(2):
        out = run_plan_decode(case, bufs, p)
        assert_close(out, ref, f"B=80 call {rep}")
        tasks, offs = read_plan(bufs)
        plan = oracle_plan(case, p)
        assert np.array_equal(tasks, plan[0]) and np.array_equal(offs, plan[1]), rep
    assert pkv.pkv_check_device_status(bufs.ws) == 0


@pytest.mark.parametrize("name,hkv,policy", [("b1", 8, 1), ("b8_bimodal", 8, 1), ("b8_uniform", 8, 0),
                                             ("b8_zipf", 8, 1), ("b4_bimodal", 8, 1), ("b1", 4, 1),
                                             ("b8_bimodal", 4, 1)])
def test_plan_decode_head_pairs_full_size(name, hkv, policy):
    """Task target 512 on the benchmark lengths: at G = 4 the one-launch route runs KV
    heads g and g + 1 of a split in one workgroup (at G = 8 one head, two tasks per
    workgroup). Each head's arithmetic is that of a one-head task, so the output is bitwise
    the plan-kernel + fused-kernel route's at the same plan, and within tolerance of the
    oracle; a repeated call (every workgroup starting from its hint) is bitwise the same."""
    case, w = Case.from_workload(name, hkv=hkv)
    p = plan_params(w.hkv, w.split_min, w.split_max, 512, w.tile_tokens, policy=policy)
    expect, tasks_ref, offs_ref = _two_launch(case, p, w.split_max)
    bufs = bufs_for(case, w.split_max)
    out = run_plan_decode(case, bufs, p)
    tasks, offs = read_plan(bufs)
    assert np.array_equal(tasks, oracle_plan(case, p)[0])
    assert np.array_equal(tasks, tasks_ref) and np.array_equal(offs, offs_ref)
    assert torch.equal(out, expect), name
    assert_close(out, ref_decode(case.q, case.k, case.v, case.bt, case.lens), f"{name} pairs G={32 // hkv}")
    again = run_plan_decode(case, bufs, p)
    assert torch.equal(again, out)
    assert pkv.pkv_check_device_status(bufs.ws) == 0


@pytest.mark.parametrize("lens,target", [([1], 512), ([16, 0, 17], 512), ([0, 5000, 0, 5000, 4000], 4096),
                                         ([31, 32, 33, 3000, 0, 64], 1000)])
def test_plan_decode_head_pairs_small_and_ragged(lens, target):
    """KV-head pairs on short, empty and ragged rows (single-page rows, a row of one
    token, splits of one tile, more tasks than resident workgroups so that workgroups
    loop over several pairs): bitwise the two-launch route, and the oracle within
    tolerance."""
    case = Case(lens, seed=31)
    p = plan_params(8, 1, 64, target, policy=1)
    expect, tasks_ref, _ = _two_launch(case, p, 64)
    bufs = bufs_for(case, 64)
    for rep in range(2):
        out = run_plan_decode(case, bufs, p)
        tasks, _ = read_plan(bufs)
        assert np.array_equal(tasks, tasks_ref), rep
        assert torch.equal(out, expect), rep
    assert_close(out, ref_decode(case.q, case.k, case.v, case.bt, case.lens), f"pairs {lens}")
    assert pkv.pkv_check_device_status(bufs.ws) == 0


@pytest.mark.parametrize("hq,hkv", [(8, 2), (12, 3), (64, 16)])
def test_plan_decode_head_pairs_other_head_counts(hq, hkv):
    """Task target 512 at G = 4 with other KV-head counts: two KV heads (one pair per
    split), an odd count (no pairs: one head per workgroup), and sixteen. Bitwise the
    two-launch route, and the oracle within tolerance."""
    case = Case([3000, 0, 700, 17, 9000], hq=hq, hkv=hkv, seed=33)
    p = plan_params(hkv, 1, 64, 512, policy=1)
    expect, tasks_ref, _ = _two_launch(case, p, 64)
    bufs = bufs_for(case, 64)
    for rep in range(2):
        out = run_plan_decode(case, bufs, p)
        tasks, _ = read_plan(bufs)
        assert np.array_equal(tasks, tasks_ref), rep
        assert torch.equal(out, expect), rep
    assert np.array_equal(tasks, oracle_plan(case, p)[0])
    assert_close(out, ref_decode(case.q, case.k, case.v, case.bt, case.lens), f"pairs hq={hq} hkv={hkv}")
    assert pkv.pkv_check_device_status(bufs.ws) == 0


def _random_config(seed):
    r = np.random.Generator(np.random.PCG64(seed))
    hq, hkv = [(32, 8), (32, 4), (32, 16), (32, 32), (8, 2), (16, 4)][seed % 6]
    B = int(r.integers(1, 41))
    kind = r.integers(0, 4, size=B)  # empty, one page or less, medium, long
    lens = np.where(kind == 0, 0, np.where(kind == 1, r.integers(1, 17, size=B),
                    np.where(kind == 2, r.integers(17, 2000, size=B), r.integers(2000, 9000, size=B))))
    budget = 480000 // hkv  # tokens: keep the pools and the fp64 oracle small
    if lens.sum() > budget:
        lens = (lens * (budget / lens.sum())).astype(np.int64)
    smin = int(r.integers(1, 9))
    smax = int(r.integers(smin, 65))
    target = int(r.choice([64, 256, 512, 700, 2048]))
    return lens.astype(np.int32), hq, hkv, smin, smax, target, int(seed % 2)


@pytest.mark.parametrize("seed", range(12))
def test_plan_decode_random_configurations(seed):
    """Seeded random batches (1-40 rows of empty, single-page, medium and long lengths),
    query/KV head counts G = 1, 2, 4, 8, split bounds, task targets from 64 to 2048 (so
    one or several tasks per workgroup, and KV-head pairs at G = 4 from 512) and both
    split policies: the one-launch route is bitwise the plan + fused route, its task list
    is the oracle's, and its output is within tolerance of the oracle."""
    lens, hq, hkv, smin, smax, target, policy = _random_config(seed)
    case = Case(lens, hq=hq, hkv=hkv, seed=100 + seed)
    p = plan_params(hkv, smin, smax, target, policy=policy)
    expect, tasks_ref, offs_ref = _two_launch(case, p, smax)
    bufs = bufs_for(case, smax)
    out = run_plan_decode(case, bufs, p)
    tasks, offs = read_plan(bufs)
    ref_t, ref_o, _ = oracle_plan(case, p)
    assert np.array_equal(tasks, ref_t) and np.array_equal(offs, ref_o)
    assert np.array_equal(tasks, tasks_ref) and np.array_equal(offs, offs_ref)
    assert torch.equal(out, expect), (seed, hq, hkv, target, policy)
    assert_close(out, ref_decode(case.q, case.k, case.v, case.bt, case.lens), f"random config {seed}")
    assert pkv.pkv_check_device_status(bufs.ws) == 0


@pytest.mark.parametrize("name", ["b1", "b8_bimodal"])
def test_plan_decode_every_step_of_a_benchmark_run(name):
    """Every decode step of a benchmark run at full size, as bench.py runs it (one
    workspace, the task target of the cost model's rule for the first step's lengths,
    lengths growing by one token per step, so every launch after the first starts from
    the previous plan's hint, KV-head pairs on B8): each step bitwise the plan + fused
    route and its task list the oracle's; the first and last steps within tolerance of
    the oracle."""
    from paper_2606_26666_amd import costmodel
    case, w = Case.from_workload(name)
    target = costmodel.default_target(w.lengths_at(0), w.hkv, hq=w.hq)
    p = plan_params(w.hkv, w.split_min, w.split_max, target, w.tile_tokens, policy=1)
    bufs = bufs_for(case, w.split_max)
    for s in range(w.steps):
        lens = w.lengths_at(s)
        case.lens = lens
        case.lens_dev = torch.from_numpy(lens).cuda()
        expect, tasks_ref, _ = _two_launch(case, p, w.split_max)
        out = run_plan_decode(case, bufs, p)
        tasks, _ = read_plan(bufs)
        assert np.array_equal(tasks, tasks_ref), s
        assert torch.equal(out, expect), s
        if s in (0, w.steps - 1):
            assert np.array_equal(tasks, oracle_plan(case, p)[0]), s
            assert_close(out, ref_decode(case.q, case.k, case.v, case.bt, lens), f"{name} step {s}")
    assert pkv.pkv_check_device_status(bufs.ws) == 0


@pytest.mark.parametrize("target", [256, 512])
def test_plan_decode_maximum_batch(target):
    """The largest batch the one-launch route plans in-launch (1024 rows, a tenth of them
    empty, 1-300 tokens each): thousands of tasks, so every workgroup loops over many
    (one head, or KV-head pairs at 512); bitwise the two-launch route, the oracle's task
    list, and the oracle within tolerance."""
    r = np.random.Generator(np.random.PCG64(41))
    lens = r.integers(1, 301, size=1024).astype(np.int32)
    lens[r.permutation(1024)[:102]] = 0
    case = Case(lens, seed=41)
    p = plan_params(8, 1, 4, target, policy=1)
    expect, tasks_ref, offs_ref = _two_launch(case, p, 4)
    bufs = bufs_for(case, 4)
    for rep in range(2):
        out = run_plan_decode(case, bufs, p)
        tasks, offs = read_plan(bufs)
        assert np.array_equal(tasks, tasks_ref) and np.array_equal(offs, offs_ref), rep
        assert torch.equal(out, expect), rep
    assert np.array_equal(tasks, oracle_plan(case, p)[0])
    assert_close(out, ref_decode(case.q, case.k, case.v, case.bt, case.lens), f"B=1024 target {target}")
    assert pkv.pkv_check_device_status(bufs.ws) == 0


@pytest.mark.parametrize("target", [8, 512])
def test_plan_decode_one_split_per_long_row(target):
    """One split per row (bounds (1, 1)) over rows of up to 40000 tokens: a task spans up
    to 2500 pages, so each wave walks several blocks of 64 page ids (one head per
    workgroup at target 8, KV-head pairs at 512). Bitwise the two-launch route and within
    tolerance of the oracle."""
    case = Case([40000, 13, 20001, 0, 5000], seed=43)
    p = plan_params(8, 1, 1, target, policy=1)
    expect, tasks_ref, _ = _two_launch(case, p, 1)
    bufs = bufs_for(case, 1)
    out = run_plan_decode(case, bufs, p)
    tasks, _ = read_plan(bufs)
    assert np.array_equal(tasks, tasks_ref) and np.array_equal(tasks, oracle_plan(case, p)[0])
    assert torch.equal(out, expect)
    assert_close(out, ref_decode(case.q, case.k, case.v, case.bt, case.lens), f"one split, target {target}")
    assert pkv.pkv_check_device_status(bufs.ws) == 0


# merge_group has two paths: column threads over runs of states (at most 64 splits, in
# one round of loads up to 32 splits and two beyond; the full-size and ragged cases above
# take the first round only), and blocks of states staged in LDS after a first pass for
# the maximum (more than 64). Rows of 282 and 375 tiles give every route that merges 33
# to 200 splits, at every G; the fused and two-kernel merges lay the column path out
# differently (512 against 256 threads), so their bitwise equality checks it as well.
MANY = [9000, 12000, 70, 0]


@pytest.mark.parametrize("split_max", [33, 48, 64, 65, 128, 200])
@pytest.mark.parametrize("hq,hkv", [(8, 8), (16, 8), (32, 8), (32, 4)])
def test_merge_of_many_splits(hq, hkv, split_max):
    """Split counts 33 to 200 (policy 0, S = split_max; 33 and 64 bound the column
    path's second round, 65 is the general path's smallest): the fused and two-kernel
    merges are bitwise equal and within tolerance of the oracle, and the one-launch route
    (KV-head pairs at G = 4, whose merge covers both heads' states) is bitwise the same."""
    case = Case(MANY, hq=hq, hkv=hkv, seed=61)
    p = plan_params(hkv, split_max, split_max, 1 << 20)
    bufs = bufs_for(case, split_max)
    run_plan(case, bufs, p)
    tasks, offs = read_plan(bufs)
    assert np.array_equal(np.diff(offs), [split_max, split_max, 3, 0])
    assert np.array_equal(tasks, oracle_plan(case, p)[0])
    fused = run_decode(case, bufs, fused=True)
    two = run_decode(case, bufs, fused=False)
    assert torch.equal(fused, two)
    assert_close(fused, ref_decode(case.q, case.k, case.v, case.bt, case.lens), f"G={hq // hkv} S={split_max}")
    assert pkv.pkv_check_device_status(bufs.ws) == 0
    one_bufs = bufs_for(case, split_max)
    for rep in range(2):
        one = run_plan_decode(case, one_bufs, p)
        assert torch.equal(one, fused), rep
    assert pkv.pkv_check_device_status(one_bufs.ws) == 0


@pytest.mark.parametrize("S", [96, 200])
@pytest.mark.parametrize("hq,hkv", [(8, 8), (16, 8), (32, 8), (32, 4)])
def test_rect_many_columns(hq, hkv, S):
    """A rectangular grid of 96 or 200 columns: the 70-token row fills 3 and merges 93 or
    197 neutral states, the empty row merges only neutral states; bitwise the workqueue at
    the same split count, and within tolerance of the oracle's rectangular merge."""
    case = Case(MANY, hq=hq, hkv=hkv, seed=62)
    bufs = bufs_for(case, split_max=S, rect_splits=S)
    run_plan(case, bufs, plan_params(hkv, S, S, 1))
    wq = run_decode(case, bufs)
    rect = run_rect(case, bufs, S)
    assert torch.equal(wq, rect)
    assert torch.all(rect[3] == 0)
    assert_close(rect, ref_decode_rect(case.q, case.k, case.v, case.bt, case.lens, S, 32), f"rect S={S}")
    assert pkv.pkv_check_device_status(bufs.ws) == 0


@pytest.mark.parametrize("corrupt", ["task rows", "split offsets"])
def test_flagged_decode_leaves_the_workspace_usable(corrupt):
    """A fused decode over a task list or split_offsets that is not a plan of the batch
    skips what it cannot place (PKV_DEVERR_TASK) and may leave completion counters short
    of their split count. The status check that reports it restores them, so the next
    one-launch call on the same workspace is bitwise the fresh two-launch route's."""
    case = Case([3000, 500, 40], seed=63)
    p = plan_params(8, 4, 16, 256)
    expect, _, _ = _two_launch(case, p, 16)
    bufs = bufs_for(case, 16)
    run_plan(case, bufs, p)
    torch.cuda.synchronize()
    if corrupt == "task rows":
        bufs.tasks[::5, 0] = 99            # rows outside the batch; the other tasks count
    else:
        bufs.split_offsets[1] = -5         # rows 0 and 1 get no consistent slot range
    run_decode(case, bufs, fused=True)
    assert pkv.pkv_check_device_status(bufs.ws) & pkv.PKV_DEVERR_TASK
    for rep in range(2):
        got = run_plan_decode(case, bufs, p)
        assert torch.equal(got, expect), rep
    assert pkv.pkv_check_device_status(bufs.ws) == 0
