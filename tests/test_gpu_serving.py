"""The continuous-batching harness on the GPU: admitted requests attend over their
pages after each appended token (checked against the fp64 oracle at several steps),
free slots produce zeros, and the MLP tail runs on the active rows."""
import numpy as np
import pytest
import torch

from oracle import ref_decode
from paper_2606_26666_amd.serving import PAGE, Engine, PagePool, Scheduler
from tests.gpu_cases import assert_close
from workloads.requests import Request

pytestmark = pytest.mark.gpu


def test_serving_steps_match_oracle():
    trace = [Request(0, 0, 300, 3), Request(1, 0, 5000, 6), Request(2, 1, 1200, 2), Request(3, 2, 64, 4),
             Request(4, 2, 20000, 3), Request(5, 4, 900, 2)]
    maxp = max(-(-(q.prompt_len + q.decode_len) // PAGE) for q in trace)
    engine = Engine(4, maxp, 4 * maxp, mlp=True, seed=7)
    checked = []

    def check(rec):  # runs before finished requests give their slots back
        slots = rec["slots"]
        q, k, v, bt, lens = engine.snapshot(slots)
        out = engine.out.cpu()
        if slots:
            assert_close(out[slots], ref_decode(q, k, v, bt, lens), f"step {rec['step']}")
            assert engine.mlp_out.shape == (len(slots), 32 * 128)
            assert torch.isfinite(engine.mlp_out).all()
            checked.append(rec["step"])
        idle = [s for s in range(4) if s not in slots]
        assert torch.all(out[idle] == 0)

    sched = Scheduler(trace, engine, PagePool(4 * maxp, seed=7), max_batch=4, observer=check)
    while not sched.finished and sched.step_idx < 30:
        sched.step()
    checked = len(checked)
    assert sched.finished and sorted(sched.done) == list(range(6)) and checked >= 6
    stats = sched.run(30)
    assert stats["tokens"] == sum(q.decode_len for q in trace)
