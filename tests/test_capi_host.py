"""The C ABI library loads, exports every function include/pkv.h declares, sizes its
buffers as documented, and rejects bad arguments on the host before enqueuing anything
(no GPU needed: every call below fails validation, so no HIP call is made)."""
import ctypes

import pytest

import paper_2606_26666_amd as pkv
from paper_2606_26666_amd import _binding as b

FAKE = 4096  # a non-null, 16-byte-aligned address that is never dereferenced


def lib():
    try:
        return pkv.lib()
    except RuntimeError as e:  # the build step has not run
        pytest.fail(str(e))


def test_exports_every_header_function():
    L = lib()
    names = pkv.header_functions()
    assert {"pkv_plan", "pkv_decode", "pkv_decode_rect", "pkv_max_tasks", "pkv_workspace_size",
            "pkv_workspace_init", "pkv_check_device_status", "pkv_status_string", "pkv_stream_copy", "pkv_stream_read",
            "pkv_plan_decode", "pkv_decode_buckets"} <= set(names)
    for n in names:
        assert hasattr(L, n), n


def test_sizes():
    assert pkv.pkv_max_tasks(1, 8, 64) == 512
    assert pkv.pkv_max_tasks(8, 8, 64) == 4096
    assert pkv.pkv_max_tasks(0, 8, 64) == -1
    assert pkv.pkv_max_tasks(1 << 20, 1 << 10, 1 << 10) == -1
    # header 256 + counters (8 -> 256) + 512 slots of fp32 {m[4], l[4], acc[4][128]} = 2080 B
    assert pkv.pkv_workspace_size(1, 32, 8, 128, 512) == 256 + 256 + 512 * 2080
    assert pkv.pkv_workspace_size(8, 32, 8, 128, 10) == 256 + 256 + 10 * 2080
    assert pkv.pkv_workspace_size(1, 8, 8, 128, 1) == 512 + 4 * (128 + 4)    # G = 1: padded to 16 B
    assert pkv.pkv_workspace_size(1, 32, 8, 64, 1) == 0      # d != 128
    assert pkv.pkv_workspace_size(1, 30, 8, 128, 1) == 0     # Hq % Hkv
    assert pkv.pkv_workspace_size(1, 64, 4, 128, 1) == 0     # G = 16 has no kernel


def test_status_strings():
    L = lib()
    for st in range(6):
        assert L.pkv_status_string(st)
    assert L.pkv_status_string(99) == b"unknown status"


def plan(L, **kw):
    args = dict(seq_lens=FAKE, bt=0, B=2, maxp=10, num_pages=100,
                params=b.PlanParams(16, 32, 8, 16, 64, 512), tasks=FAKE, max_tasks=2 * 8 * 64,
                offs=FAKE, ntasks=FAKE, ws=FAKE, ws_bytes=1 << 20)
    args.update(kw)
    return L.pkv_plan(args["seq_lens"], args["bt"], args["B"], args["maxp"], args["num_pages"],
                      ctypes.byref(args["params"]), args["tasks"], args["max_tasks"], args["offs"],
                      args["ntasks"], args["ws"], args["ws_bytes"], None)


def test_plan_validation():
    L = lib()
    assert plan(L, seq_lens=0) == pkv.PKV_ERR_INVALID_ARG
    assert plan(L, tasks=0) == pkv.PKV_ERR_INVALID_ARG
    assert plan(L, B=0) == pkv.PKV_ERR_INVALID_ARG
    assert plan(L, B=5000, max_tasks=5000 * 8 * 64) == pkv.PKV_ERR_INVALID_ARG
    assert plan(L, maxp=0) == pkv.PKV_ERR_INVALID_ARG
    assert plan(L, bt=FAKE, num_pages=0) == pkv.PKV_ERR_INVALID_ARG
    assert plan(L, ws=FAKE + 4) == pkv.PKV_ERR_INVALID_ARG
    assert plan(L, params=b.PlanParams(8, 32, 8, 16, 64, 512)) == pkv.PKV_ERR_UNSUPPORTED
    assert plan(L, params=b.PlanParams(16, 24, 8, 16, 64, 512)) == pkv.PKV_ERR_UNSUPPORTED
    assert plan(L, params=b.PlanParams(16, 0, 8, 16, 64, 512)) == pkv.PKV_ERR_UNSUPPORTED
    assert plan(L, params=b.PlanParams(16, 32, 8, 65, 64, 512)) == pkv.PKV_ERR_INVALID_ARG
    assert plan(L, params=b.PlanParams(16, 32, 8, 0, 64, 512)) == pkv.PKV_ERR_INVALID_ARG
    assert plan(L, params=b.PlanParams(16, 32, 0, 16, 64, 512)) == pkv.PKV_ERR_INVALID_ARG
    assert plan(L, params=b.PlanParams(16, 32, 8, 16, 64, 0)) == pkv.PKV_ERR_INVALID_ARG
    assert plan(L, params=b.PlanParams(16, 32, 8, 16, 64, 512, 2)) == pkv.PKV_ERR_INVALID_ARG  # policy
    assert plan(L, params=b.PlanParams(16, 32, 1, 16, 65537, 512)) == pkv.PKV_ERR_INVALID_ARG  # split cap
    assert plan(L, max_tasks=2 * 8 * 64 - 1) == pkv.PKV_ERR_WORKSPACE
    assert plan(L, ws_bytes=511) == pkv.PKV_ERR_WORKSPACE
    assert plan(L, maxp=1 << 28) == pkv.PKV_ERR_INVALID_ARG


def decode(L, **kw):
    a = dict(q=FAKE, k=FAKE, v=FAKE, num_pages=100, bt=FAKE, maxp=10, seq_lens=FAKE, B=2, Hq=32, Hkv=8, d=128,
             tasks=FAKE, offs=FAKE, ntasks=FAKE, max_tasks=1024, scale=1.0, flags=1, out=FAKE, ws=FAKE,
             ws_bytes=1 << 22)
    a.update(kw)
    return L.pkv_decode(a["q"], a["k"], a["v"], a["num_pages"], a["bt"], a["maxp"], a["seq_lens"], a["B"],
                        a["Hq"], a["Hkv"], a["d"], a["tasks"], a["offs"], a["ntasks"], a["max_tasks"],
                        a["scale"], a["flags"], a["out"], a["ws"], a["ws_bytes"], None)


def test_decode_validation():
    L = lib()
    for k in ("q", "k", "v", "bt", "seq_lens", "tasks", "offs", "ntasks", "out", "ws"):
        assert decode(L, **{k: 0}) == pkv.PKV_ERR_INVALID_ARG, k
    assert decode(L, q=FAKE + 2) == pkv.PKV_ERR_INVALID_ARG       # 16-byte alignment
    assert decode(L, out=FAKE + 2) == pkv.PKV_ERR_INVALID_ARG
    assert decode(L, B=0) == pkv.PKV_ERR_INVALID_ARG
    assert decode(L, num_pages=0) == pkv.PKV_ERR_INVALID_ARG
    assert decode(L, Hq=30) == pkv.PKV_ERR_INVALID_ARG
    assert decode(L, d=64) == pkv.PKV_ERR_UNSUPPORTED
    assert decode(L, Hq=64, Hkv=4) == pkv.PKV_ERR_UNSUPPORTED     # G = 16
    assert decode(L, Hq=24, Hkv=8) == pkv.PKV_ERR_UNSUPPORTED     # G = 3
    assert decode(L, flags=3) == pkv.PKV_ERR_INVALID_ARG
    assert decode(L, scale=float("nan")) == pkv.PKV_ERR_INVALID_ARG
    assert decode(L, max_tasks=0) == pkv.PKV_ERR_INVALID_ARG
    assert decode(L, ws_bytes=1000) == pkv.PKV_ERR_WORKSPACE


def test_rect_validation():
    L = lib()

    def rect(**kw):
        a = dict(q=FAKE, S=16, tile=32, ws_bytes=1 << 22, B=2, d=128)
        a.update(kw)
        ids = (ctypes.c_int32 * len(a.get("ids", []) or [0]))(*(a.get("ids") or [0]))
        return L.pkv_decode_rect(a["q"], FAKE, FAKE, 100, FAKE, 10, FAKE, a["B"], 32, 8, a["d"],
                                 ids if a.get("ids") is not None else None, a.get("n", 0), a["S"],
                                 a["tile"], 1.0, FAKE, FAKE, a["ws_bytes"], None)
    assert rect(S=0) == pkv.PKV_ERR_INVALID_ARG
    assert rect(S=65537) == pkv.PKV_ERR_INVALID_ARG
    assert rect(tile=24) == pkv.PKV_ERR_UNSUPPORTED
    assert rect(d=96) == pkv.PKV_ERR_UNSUPPORTED
    assert rect(q=0) == pkv.PKV_ERR_INVALID_ARG
    assert rect(ws_bytes=2 * 8 * 16 * 2080) == pkv.PKV_ERR_WORKSPACE  # header missing
    assert rect(ids=[0, 5], n=2) == pkv.PKV_ERR_INVALID_ARG              # row 5 outside B = 2
    assert rect(ids=[0], n=65) == pkv.PKV_ERR_INVALID_ARG                # more than 64 rows
    assert rect(ids=[1], n=1, S=0) == pkv.PKV_ERR_INVALID_ARG


def test_copy_and_init_validation():
    L = lib()
    assert L.pkv_stream_copy(FAKE, FAKE, 15, None) == pkv.PKV_ERR_INVALID_ARG
    assert L.pkv_stream_copy(0, FAKE, 16, None) == pkv.PKV_ERR_INVALID_ARG
    assert L.pkv_stream_read(FAKE, 17, FAKE, None) == pkv.PKV_ERR_INVALID_ARG
    assert L.pkv_stream_read(FAKE, 16, 0, None) == pkv.PKV_ERR_INVALID_ARG
    assert L.pkv_stream_read_nt_timed(FAKE, 17, FAKE, None, None, None) == pkv.PKV_ERR_INVALID_ARG
    assert L.pkv_stream_read_nt_timed(FAKE, 16, 0, None, None, None) == pkv.PKV_ERR_INVALID_ARG
    assert L.pkv_workspace_init(FAKE, 100, 1, 8, None) == pkv.PKV_ERR_WORKSPACE
    assert L.pkv_workspace_init(0, 1 << 20, 1, 8, None) == pkv.PKV_ERR_INVALID_ARG
    assert L.pkv_check_device_status(0, None, None) == pkv.PKV_ERR_INVALID_ARG


def test_stream_read_pages_validation():
    L = lib()

    def rp(**kw):
        a = dict(k=FAKE, num_pages=100, maxp=10, B=2, hkv=8, d=128, tasks=FAKE, max_tasks=64, hpw=1, sink=FAKE)
        a.update(kw)
        return L.pkv_stream_read_pages(a["k"], FAKE, a["num_pages"], FAKE, a["maxp"], a["B"], a["hkv"], a["d"],
                                       a["tasks"], FAKE, a["max_tasks"], a["hpw"], a["sink"], None, None, None)
    assert rp(k=0) == pkv.PKV_ERR_INVALID_ARG
    assert rp(k=FAKE + 8) == pkv.PKV_ERR_INVALID_ARG          # K not 16-byte aligned
    assert rp(tasks=0) == pkv.PKV_ERR_INVALID_ARG
    assert rp(sink=FAKE + 2) == pkv.PKV_ERR_INVALID_ARG
    assert rp(num_pages=0) == pkv.PKV_ERR_INVALID_ARG
    assert rp(max_tasks=0) == pkv.PKV_ERR_INVALID_ARG
    assert rp(hkv=257) == pkv.PKV_ERR_INVALID_ARG
    assert rp(hpw=3) == pkv.PKV_ERR_INVALID_ARG
    assert rp(hpw=2, hkv=3) == pkv.PKV_ERR_INVALID_ARG         # pairs need an even head count
    assert rp(maxp=1 << 28) == pkv.PKV_ERR_INVALID_ARG         # maxp * 16 beyond int32
    assert rp(d=64) == pkv.PKV_ERR_UNSUPPORTED


def test_plan_decode_validation():
    L = lib()

    def pd(**kw):
        a = dict(B=2, d=128, params=b.PlanParams(16, 32, 8, 16, 64, 512), max_tasks=2 * 8 * 64, ws_bytes=1 << 22)
        a.update(kw)
        return L.pkv_plan_decode(FAKE, FAKE, FAKE, 100, FAKE, 10, FAKE, a["B"], 32, 8, a["d"],
                                 ctypes.byref(a["params"]), FAKE, a["max_tasks"], FAKE, FAKE, 1.0, FAKE, FAKE,
                                 a["ws_bytes"], None)
    assert pd(B=2000, max_tasks=2000 * 8 * 64) == pkv.PKV_ERR_UNSUPPORTED   # planner inside: B <= 1024
    assert pd(d=64) == pkv.PKV_ERR_UNSUPPORTED
    assert pd(params=b.PlanParams(16, 32, 4, 16, 64, 512)) == pkv.PKV_ERR_INVALID_ARG   # Hkv mismatch
    assert pd(max_tasks=100) == pkv.PKV_ERR_WORKSPACE
    assert pd(ws_bytes=4096) == pkv.PKV_ERR_WORKSPACE


def test_plan_decode_noalloc_validation():
    """The entry point without a workspace rejects, before touching any device, what
    pkv_plan_decode rejects, a missing error word, and sizes beyond its scratch: B * Hkv
    above 16384 completion counters, or more slots than 16 MiB - 64 KiB holds."""
    L = lib()

    def pd(**kw):
        a = dict(B=2, hq=32, hkv=8, d=128, params=b.PlanParams(16, 32, 8, 16, 64, 512), max_tasks=2 * 8 * 64,
                 err=FAKE)
        a.update(kw)
        return L.pkv_plan_decode_noalloc(FAKE, FAKE, FAKE, 100, FAKE, 10, FAKE, a["B"], a["hq"], a["hkv"], a["d"],
                                         ctypes.byref(a["params"]), FAKE, a["max_tasks"], FAKE, FAKE, 1.0, FAKE,
                                         a["err"], None)
    assert pd(err=0) == pkv.PKV_ERR_INVALID_ARG
    assert pd(err=FAKE + 2) == pkv.PKV_ERR_INVALID_ARG
    assert pd(B=600, hkv=32, params=b.PlanParams(16, 32, 32, 1, 1, 512),
              max_tasks=600 * 32) == pkv.PKV_ERR_WORKSPACE                    # 19200 counters > 16384
    assert pd(B=1000, max_tasks=1000 * 8 * 64) == pkv.PKV_ERR_WORKSPACE     # 512000 slots > the scratch's
    assert pd(B=1100, params=b.PlanParams(16, 32, 8, 1, 1, 512), max_tasks=1100 * 8) == pkv.PKV_ERR_UNSUPPORTED
    assert pd(d=64) == pkv.PKV_ERR_UNSUPPORTED
    assert pd(params=b.PlanParams(16, 32, 4, 16, 64, 512)) == pkv.PKV_ERR_INVALID_ARG   # Hkv mismatch
    assert pd(max_tasks=100) == pkv.PKV_ERR_WORKSPACE                                  # below the plan's bound
    # the slot limit: 8034 slots of 2080 B fit in 16 MiB - 64 KiB, 8035 do not
    p1 = b.PlanParams(16, 32, 8, 1, 1, 512)
    assert pd(B=1, params=b.PlanParams(16, 32, 8, 1, 1004, 512), max_tasks=8035) == pkv.PKV_ERR_WORKSPACE
    assert pd(B=1, params=p1, max_tasks=8035) == pkv.PKV_ERR_WORKSPACE
    assert pd(B=1, hq=64, hkv=8, params=p1, max_tasks=4018) == pkv.PKV_ERR_WORKSPACE   # G = 8: 4160-B slots


@pytest.mark.parametrize("policy", [0, 1])
def test_host_planner_matches_oracle(policy):
    """pkv_plan_host (C++) against the oracle's ref_plan: bit-exact task lists and offsets."""
    import numpy as np

    from oracle import PlanParams, ref_plan
    lib()
    r = np.random.Generator(np.random.PCG64(7 + policy))
    for trial in range(60):
        B = int(r.integers(1, 300)) if trial % 3 else int(r.integers(1, 9))
        lens = r.integers(0, 70000, size=B).astype(np.int32)
        lens[r.random(B) < 0.2] = 0
        hkv = int(r.choice([1, 2, 4, 8]))
        smin = int(r.integers(1, 17))
        smax = smin + int(r.integers(0, 100))
        target = int(r.integers(1, 5000))
        tile = int(r.choice([16, 32, 64]))
        maxp = int(lens.max()) // 16 + 1
        p = pkv.make_params(hkv, smin, smax, target, tile, policy=policy)
        tasks, offs, n = pkv.pkv_plan_host(lens, p, maxp)
        rt, ro, _ = ref_plan(lens, PlanParams(16, tile, hkv, smin, smax, target, policy), max_pages_per_row=maxp)
        assert n == len(rt) and np.array_equal(tasks, rt) and np.array_equal(offs, ro), (trial, B, policy)


def test_host_planner_validation():
    import numpy as np
    L = lib()
    p = b.PlanParams(16, 32, 8, 16, 64, 512)
    lens = np.array([100, 40], dtype=np.int32)
    n = ctypes.c_int32(-1)
    assert L.pkv_plan_host(lens.ctypes.data, 2, 10, ctypes.byref(p), None, 0, None, ctypes.byref(n)) == pkv.PKV_OK
    assert n.value == 8 * (4 + 2)                         # S = 32 caps nothing: 4 + 2 splits
    assert L.pkv_plan_host(lens.ctypes.data, 2, 6, ctypes.byref(p), None, 0, None, ctypes.byref(n)) \
        == pkv.PKV_ERR_INVALID_ARG                        # 100 tokens > 6 pages
    bad = np.array([-1], dtype=np.int32)
    assert L.pkv_plan_host(bad.ctypes.data, 1, 10, ctypes.byref(p), None, 0, None, ctypes.byref(n)) \
        == pkv.PKV_ERR_INVALID_ARG
    tasks = np.zeros((3, 5), dtype=np.int32)
    assert L.pkv_plan_host(lens.ctypes.data, 2, 10, ctypes.byref(p), tasks.ctypes.data, 3, None,
                           ctypes.byref(n)) == pkv.PKV_ERR_WORKSPACE
    assert L.pkv_plan_host(lens.ctypes.data, 2, 10, ctypes.byref(b.PlanParams(16, 24, 8, 16, 64, 512)), None, 0,
                           None, ctypes.byref(n)) == pkv.PKV_ERR_UNSUPPORTED
    assert L.pkv_plan_host(0, 2, 10, ctypes.byref(p), None, 0, None, ctypes.byref(n)) == pkv.PKV_ERR_INVALID_ARG
