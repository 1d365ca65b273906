"""The read-only probe of the decode kernel's page pattern (pkv_stream_read_pages): it runs
over a plan's task list with one KV head and with head pairs per workgroup, skips records
that no valid plan holds, writes nothing but (practically never) its sink word, and leaves
a decode on the same inputs bitwise unchanged."""
import numpy as np
import pytest
import torch

import paper_2606_26666_amd as pkv
from gpu_cases import Case, plan_params, rng, run_decode, run_plan

pytestmark = pytest.mark.gpu


def _probe(case, bufs, hpw, sink):
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    pkv.pkv_stream_read_pages(case.k_dev, case.v_dev, case.bt_dev, bufs.tasks, bufs.num_tasks, hpw, sink,
                              events=(e0, e1))
    torch.cuda.synchronize()
    return e0.elapsed_time(e1)


def test_page_read_probe_over_a_plan():
    case = Case([3000, 17, 0, 900, 12000, 1], seed=31)
    bufs = pkv.DecodeBuffers(case.B, case.hq, case.hkv, case.d, 64, "cuda")
    run_plan(case, bufs, plan_params(8, target=512, policy=1))
    before = run_decode(case, bufs).clone()
    k0, v0 = case.k_dev.view(torch.int16).clone(), case.v_dev.view(torch.int16).clone()
    sink = torch.zeros(1, dtype=torch.int32, device="cuda")
    for hpw in (1, 2):
        assert _probe(case, bufs, hpw, sink) > 0
    assert torch.equal(case.k_dev.view(torch.int16), k0) and torch.equal(case.v_dev.view(torch.int16), v0)
    assert torch.equal(run_decode(case, bufs), before)


def test_page_read_probe_skips_records_of_no_valid_plan():
    case = Case([700, 2000, 33], seed=32)
    bufs = pkv.DecodeBuffers(case.B, case.hq, case.hkv, case.d, 64, "cuda")
    r = rng(33)
    n = bufs.max_tasks
    maxp = case.bt.shape[1]
    t = np.stack([r.integers(-3, case.B + 3, n), r.integers(-3, case.hkv + 3, n), r.integers(0, 64, n),
                  r.integers(-40, maxp * 16 + 40, n), r.integers(-40, maxp * 16 + 400, n)], axis=1)
    t[::3, 4] = t[::3, 3] + r.integers(1, 200, len(t[::3]))  # some plausible ranges among the garbage
    bufs.tasks.copy_(torch.from_numpy(t.astype(np.int32)))
    bufs.num_tasks.fill_(n)
    sink = torch.zeros(1, dtype=torch.int32, device="cuda")
    for hpw in (1, 2):
        assert _probe(case, bufs, hpw, sink) > 0
    bufs.num_tasks.fill_(1 << 30)  # a count beyond the buffer is capped at max_tasks
    assert _probe(case, bufs, 1, sink) > 0


def test_streaming_reads_both_policies():
    """The contiguous streaming reads (allocating, and non-temporal as the decode's K/V
    loads) read a buffer without changing it, write nothing but their sink word, and the
    non-temporal one stamps its own execution interval."""
    buf = torch.arange(1 << 20, dtype=torch.int32, device="cuda")
    ref = buf.clone()
    sink = torch.zeros(1, dtype=torch.int32, device="cuda")
    pkv.pkv_stream_read(buf, sink)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    pkv.pkv_stream_read_nt_timed(buf, sink, events=(e0, e1))
    pkv.pkv_stream_read_nt_timed(buf[:4], sink)  # one 16-byte load
    torch.cuda.synchronize()
    assert e0.elapsed_time(e1) > 0
    assert torch.equal(buf, ref)
    assert int(sink.item()) == 0  # the data does not hash to the sink's fixed value
