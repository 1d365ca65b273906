"""The one-launch decode inside a captured HIP graph (through torch.cuda.CUDAGraph).

A decode step is one kernel with no memset (the kernel itself restores the completion
counters), so it can be captured once and replayed while the caller updates lengths,
queries and pages in place. Each replay is separated by eager work and a
synchronization, and each is compared bitwise with an eager call on the same inputs and
within tolerance with the oracle."""
import numpy as np
import pytest
import torch

import paper_2606_26666_amd as pkv
from oracle import ref_decode
from tests.gpu_cases import Case, assert_close, plan_params, read_plan

pytestmark = pytest.mark.gpu


def test_plan_decode_replays_in_a_graph():
    base = np.array([3000, 0, 517, 9000, 33, 1200], dtype=np.int32)
    steps = 6
    case = Case(base + 40 * steps, seed=31)
    p = plan_params(8, 1, 64, 256, policy=1)
    graph_bufs = pkv.DecodeBuffers(case.B, case.hq, case.hkv, case.d, 64, "cuda")
    eager_bufs = pkv.DecodeBuffers(case.B, case.hq, case.hkv, case.d, 64, "cuda")
    lens_dev = torch.from_numpy(base).cuda()
    q_dev = case.q_dev.clone()
    out = torch.zeros((case.B, case.hq, case.d), dtype=torch.float16, device="cuda")

    def step(bufs, o):
        pkv.pkv_plan_decode(q_dev, case.k_dev, case.v_dev, case.bt_dev, lens_dev, p, bufs.tasks,
                            bufs.split_offsets, bufs.num_tasks, 1.0, o, bufs.ws)

    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):  # warm up on the capture stream
        step(graph_bufs, out)
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step(graph_bufs, out)
    torch.cuda.synchronize()
    rng = np.random.Generator(np.random.PCG64(32))
    for i in range(steps):
        lens = base + 40 * (i + 1)
        lens[1] = 0 if i % 2 == 0 else 16 * i + 3  # a row that empties and refills
        lens_dev.copy_(torch.from_numpy(lens))
        q_host = (rng.standard_normal(case.q.shape) / np.sqrt(case.d)).astype(np.float16)
        q_dev.copy_(torch.from_numpy(q_host))
        torch.cuda.synchronize()
        out.fill_(float("nan"))
        g.replay()
        torch.cuda.synchronize()
        replayed = out.clone()
        eager = torch.full_like(out, float("nan"))
        step(eager_bufs, eager)
        torch.cuda.synchronize()
        assert torch.equal(replayed, eager), i
        assert_close(replayed, ref_decode(q_host, case.k, case.v, case.bt, lens), f"replay {i}")
        tg, og = read_plan(graph_bufs)
        te, oe = read_plan(eager_bufs)
        assert np.array_equal(tg, te) and np.array_equal(og, oe), i
    assert pkv.pkv_check_device_status(graph_bufs.ws) == 0
    assert pkv.pkv_check_device_status(eager_bufs.ws) == 0
