"""pkv_plan_decode_noalloc (the one-launch route with the library's per-device scratch
instead of a caller workspace) against pkv_plan_decode, through the C ABI: two calls in
a row, the second with a smaller batch, each bitwise equal to the workspace entry
point's output and plan, and within tolerance of the oracle."""
import numpy as np
import pytest
import torch

import paper_2606_26666_amd as pkv
from oracle import ref_decode
from tests.gpu_cases import Case, assert_close, plan_params, read_plan

pytestmark = pytest.mark.gpu


def _with_workspace(case, p, split_max):
    bufs = pkv.DecodeBuffers(case.B, case.hq, case.hkv, case.d, split_max, "cuda")
    out = torch.full((case.B, case.hq, case.d), float("nan"), dtype=torch.float16, device="cuda")
    pkv.pkv_plan_decode(case.q_dev, case.k_dev, case.v_dev, case.bt_dev, case.lens_dev, p, bufs.tasks,
                        bufs.split_offsets, bufs.num_tasks, 1.0, out, bufs.ws)
    tasks, offs = read_plan(bufs)
    assert pkv.pkv_check_device_status(bufs.ws) == 0
    return out, tasks, offs


def _without_workspace(case, p, split_max):
    max_tasks = pkv.pkv_max_tasks(case.B, case.hkv, split_max)
    tasks = torch.full((max_tasks, 5), -3, dtype=torch.int32, device="cuda")
    offs = torch.zeros(case.B + 1, dtype=torch.int32, device="cuda")
    ntasks = torch.zeros(1, dtype=torch.int32, device="cuda")
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    out = torch.full((case.B, case.hq, case.d), float("nan"), dtype=torch.float16, device="cuda")
    pkv.pkv_plan_decode_noalloc(case.q_dev, case.k_dev, case.v_dev, case.bt_dev, case.lens_dev, p, tasks, offs,
                                ntasks, 1.0, out, err)
    torch.cuda.synchronize()
    n = int(ntasks.item())
    return out, tasks[:n].cpu().numpy(), offs.cpu().numpy(), int(err.item())


@pytest.mark.parametrize("target", [256, 512])
def test_noalloc_matches_workspace_entry_point(target):
    """Target 512 runs KV-head pairs. The second call has fewer, shorter rows, so it uses
    fewer counters and slots than the first left behind."""
    cases = [Case([9000, 0, 700, 4000, 17, 2500], seed=51), Case([1200, 33], seed=52)]
    for i, case in enumerate(cases):
        p = plan_params(8, 1, 64, target, policy=1)
        expect, tasks_ref, offs_ref = _with_workspace(case, p, 64)
        out, tasks, offs, err = _without_workspace(case, p, 64)
        assert err == 0, (i, err)
        assert np.array_equal(tasks, tasks_ref) and np.array_equal(offs, offs_ref), i
        assert torch.equal(out, expect), i
        assert_close(out, ref_decode(case.q, case.k, case.v, case.bt, case.lens), f"noalloc call {i}")


def test_noalloc_flags_a_bad_length_in_its_error_word():
    """A length beyond the block table: the row is planned empty and written as zeros,
    and the flag lands in the caller's error word; a following good call is clean."""
    case = Case([300, 120], seed=53)
    bad = case.lens.copy()
    bad[1] = case.bt.shape[1] * 16 + 1
    good_lens = case.lens_dev
    case.lens_dev = torch.from_numpy(bad).cuda()
    p = plan_params(8, 1, 16, 256, policy=1)
    out, _, _, err = _without_workspace(case, p, 16)
    assert err & pkv.PKV_DEVERR_SEQ_LEN
    assert torch.all(out[1] == 0)
    assert_close(out[:1], ref_decode(case.q[:1], case.k, case.v, case.bt[:1], case.lens[:1]), "row 0")
    case.lens_dev = good_lens
    expect, _, _ = _with_workspace(case, p, 16)
    out, _, _, err = _without_workspace(case, p, 16)
    assert err == 0 and torch.equal(out, expect)
