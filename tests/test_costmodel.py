"""The route cost model (Sec. 3.5): route counts against hand counts and the paper's
Tab. 4 arithmetic, the estimate's closed form, the fit recovering planted constants, and
the calibration file round trip. Host arithmetic only (no GPU)."""
import numpy as np
import pytest

import paper_2606_26666_amd as pkv
from paper_2606_26666_amd import costmodel as cm


def params(target=512, smin=16, smax=64, policy=0, hkv=8):
    return pkv.make_params(hkv, smin, smax, target, policy=policy)


def test_route_counts_by_hand():
    lens = [640, 700, 2000, 17000, 30000, 900, 25000, 32768]   # 8 distinct lengths, all >= 20 tiles
    p = params(target=512, smin=20, smax=20)                     # S = 20 everywhere (Tab. 4 workqueue)
    wq = cm.route_shape("plan+fused", lens, p)
    assert wq.workgroups == 8 * 8 * 20 and wq.launch_count == 2 and wq.merge_launches == 0
    assert wq.merge_bytes == 2 * 1280 * 2080
    ex = cm.route_shape("exact-buckets", lens, params(target=512, smin=32, smax=32))
    assert ex.launch_count == 16 and ex.merge_launches == 8               # Tab. 4: 16 launches
    assert ex.workgroups == 8 * 8 * 32                                     # 2048 slots
    assert round(ex.merge_bytes / 2 / 2**20, 2) == 4.06
    co = cm.route_shape("coarse-buckets", lens, p)                         # keys 1, 1, 1, 2, 2, 1, 2, 2
    assert co.launch_count == 4 and len(co.launches) == 2
    rect = cm.route_shape("rect", lens + [0], p)                           # 9 rows incl. an empty one
    assert rect.workgroups == 9 * 8 * 20 and rect.launch_count == 2
    one = cm.route_shape("one-launch", [32769], params(target=256, policy=1))
    assert one.workgroups == 256 and one.launch_count == 1
    kv = 32769 * 4096
    assert one.launches == [(kv, 256)]


def test_empty_rows_form_a_bucket_launch():
    sh = cm.route_shape("exact-buckets", [0, 0, 100], params())
    assert sh.launch_count == 4 and sh.launches[0][0] == 0


def test_estimate_closed_form():
    cal = cm.Calibration(beta_gbs=5000.0, launch_us=2.0, c_min=2.0, fixed_us=7.0, cus=256)
    sh = cm.RouteShape([(5_000_000, 128), (10_000_000, 1024)], 3, 1_000_000, 1)
    # launch 1: 0.5 WG/CU -> x4; launch 2: 4 WG/CU -> x1
    want = 5_000_000 / 5e6 * 4 + 10_000_000 / 5e6 + 3 * 2.0 + 1_000_000 / 5e6 + 7.0   # 5e6 B/us
    assert cm.estimate_us(sh, cal) == pytest.approx(want)


def test_choose_route_prefers_fewer_launches_at_equal_work():
    cal = cm.Calibration(beta_gbs=6000.0, launch_us=1.5, c_min=1.0, fixed_us=10.0)
    best, est = cm.choose_route([20000] * 8, params(target=256, policy=1), cal,
                                routes=("one-launch", "plan+fused", "two-kernel"))
    assert best == "one-launch"
    assert est["plan+fused"] - est["one-launch"] == pytest.approx(1.5)
    assert est["two-kernel"] - est["plan+fused"] == pytest.approx(1.5)


def test_fit_recovers_planted_constants():
    truth = cm.Calibration(beta_gbs=5400.0, launch_us=1.5, c_min=1.3, fixed_us=9.0,
                           route_fixed_us={"one-launch": 0.0, "planner kernel": 1.25, "rectangular": -2.0},
                           pair_gain=0.06)
    r = np.random.Generator(np.random.PCG64(3))
    samples = []
    for target in (64, 128, 256, 512, 1024):
        for lens in ([32769], list(r.integers(1000, 32768, size=8))):
            for route in ("one-launch", "plan+fused", "rect", "coarse-buckets"):
                sh = cm.route_shape(route, lens, params(target=target, policy=1 if route == "one-launch" else 0))
                samples.append((sh, cm.estimate_us(sh, truth)))
    assert any(sh.pairs for sh, _ in samples) and not all(sh.pairs for sh, _ in samples)
    got = cm.fit(samples, 6000.0, truth.launch_us)          # probe 6000, true effective 0.9 of it
    assert got.beta_gbs == pytest.approx(5400.0) and got.c_min == pytest.approx(1.3)
    assert got.pair_gain == pytest.approx(0.06)
    assert got.fixed_us == pytest.approx(9.0, abs=1e-6) and got.probe_beta_gbs == 6000.0
    for fam, v in truth.route_fixed_us.items():
        assert got.route_fixed_us[fam] == pytest.approx(v, abs=1e-6)


def test_route_terms_in_the_estimate():
    """A family's fixed term is added to every route of that family; the pair gain scales
    only the KV streaming time of a one-launch step that runs KV-head pairs."""
    base = cm.Calibration(beta_gbs=5000.0, launch_us=2.0, c_min=1.0, fixed_us=7.0)
    more = cm.Calibration(beta_gbs=5000.0, launch_us=2.0, c_min=1.0, fixed_us=7.0,
                          route_fixed_us={"rectangular": 3.0}, pair_gain=0.1)
    lens = [20000] * 8
    for route in cm.ROUTES:
        sh = cm.route_shape(route, lens, params(target=512, policy=1))
        d = cm.estimate_us(sh, more) - cm.estimate_us(sh, base)
        if cm.FAMILY[route] == "rectangular":
            assert d == pytest.approx(3.0)
        elif sh.pairs:
            assert route == "one-launch" and d == pytest.approx(-0.1 * 8 * 20000 * 4096 / 5e6)
        else:
            assert d == pytest.approx(0.0)


def test_calibration_roundtrip(tmp_path):
    cal = cm.Calibration(5500.0, 1.54, 1.25, 10.5, 256, 6087.7, {"rectangular": -1.0}, 0.04, note="x")
    path = tmp_path / "cal.json"
    cal.save(str(path))
    assert cm.Calibration.load(str(path)) == cal


def test_committed_calibration_loads():
    import os
    path = os.path.join(os.path.dirname(cm.__file__), "calibration_mi355x.json")
    cal = cm.Calibration.load(path)
    assert 1000 < cal.beta_gbs <= cal.probe_beta_gbs < 8000      # below the 8 TB/s peak
    assert 0 < cal.launch_us < 20 and 0 < cal.c_min < 8 and cal.cus == 256
    best, _ = cm.choose_route([32769], params(target=256, policy=1), cal,
                              routes=("one-launch", "plan+fused", "two-kernel", "rect"))
    assert best == "one-launch"


def test_default_target_rule():
    """One task per compute unit unless the KV heads need room for 4 splits per active
    row (the measured optimum of every G and trace in the split sweep), and two per
    compute unit where KV-head pairs run and the longest row would get at most 24 splits
    per KV head at that target."""
    b1, b4 = [32768], [1500, 20000, 0, 30000]
    b8 = [300, 20000, 1800, 31000, 700, 25000, 1200, 17000]   # longest row 32% of the tokens
    assert cm.default_target(b1, 8) == 256           # B1, G = 4: one row
    assert cm.default_target(b8, 8) == 512           # B8, G = 4: KV-head pairs, two tasks per CU
    assert cm.default_target(b4, 8) == 256           # B4, G = 4: longest row 58% of the tokens
    assert cm.default_target(b8, 4) == 256           # B8, G = 8: one head per workgroup
    assert cm.default_target([1000] * 16, 8) == 512  # 16 even rows, G = 4: 4 splits per row
    assert cm.default_target(b8, 8, hq=8) == 256     # G = 1 body runs one head
    share = [1000] * 8
    share[0] = 4200                                  # 3/8 of the tokens: exactly 24 splits at Hkv = 8
    assert cm.default_target(share, 8) == 512 and cm.default_target([4201] + share[1:], 8) == 256
    assert cm.head_pairs(32, 8) and not cm.head_pairs(32, 4) and not cm.head_pairs(32, 16)
    assert not cm.head_pairs(12, 3)                  # odd KV-head count
    assert cm.default_target(b8, 16) == 512          # B8, G = 2
    assert cm.default_target(b8, 32) == 1024         # B8, G = 1
    assert cm.default_target(b4[:3] + [9000], 32) == 384  # three active rows, G = 1: 4 * 32 * 3
    assert cm.default_target(b1, 32) == 256          # B1, G = 1
    assert cm.default_target([0, 0], 8) == 256       # an idle step still gets a valid target
    # the planner never exceeds the task buffer whatever the target: B * Hkv * split_max
    lens = [20000, 300, 0, 9000]
    p = params(target=cm.default_target(lens, 32), smin=1, smax=64, policy=1, hkv=32)
    _, _, n = pkv.pkv_plan_host(lens, p, 2000, with_tasks=False)
    assert n <= p.target_tasks and n <= len(lens) * 32 * 64


@pytest.mark.parametrize("name,expect", [("b1", 256), ("b8_bimodal", 512), ("b8_uniform", 512),
                                         ("b8_zipf", 512), ("b4_bimodal", 256)])
def test_default_target_on_benchmark_traces(name, expect):
    """The targets the benchmark runs with at its main seed: KV-head pairs (512 tasks) on
    the B8 traces, one head per workgroup (256) for B1 and B4; and the longest row's
    split count at the chosen target stays within the pair limit where pairs run."""
    from oracle.plan import PlanParams, ref_plan
    from workloads import make_workload
    w = make_workload(name, seed=20260623)
    lens = w.lengths_at(0)
    target = cm.default_target(lens, w.hkv, hq=w.hq)
    assert target == expect
    _, offs, _ = ref_plan(lens, PlanParams(split_min=w.split_min, split_max=w.split_max, target_tasks=target,
                                           policy=1, num_kv_heads=w.hkv))
    if target == 512:
        assert int(np.diff(offs).max()) <= cm.PAIR_MAX_SPLITS
