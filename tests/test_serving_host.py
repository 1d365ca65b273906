"""Host side of the continuous-batching harness: request traces (families, files), the
page pool and the scheduler's admission / completion logic against a recording fake
engine (no GPU)."""
import numpy as np
import pytest

from paper_2606_26666_amd.serving import PAGE, PagePool, Scheduler
from workloads.requests import FAMILIES, Request, load_trace, request_trace, save_trace


@pytest.mark.parametrize("family", FAMILIES)
def test_trace_families(family):
    a = request_trace(family, 40, seed=5, decode_min=3, decode_max=9, arrival_gap=2)
    assert a == request_trace(family, 40, seed=5, decode_min=3, decode_max=9, arrival_gap=2)
    assert [q.arrival_step for q in a] == [2 * i for i in range(40)]
    assert all(3 <= q.decode_len <= 9 for q in a)
    p = np.array([q.prompt_len for q in a])
    if family == "bucketed":
        assert p.tolist()[:8] == [8192, 16384, 32768, 65536] * 2
    elif family == "homogeneous":
        assert (p == 32768).all()
    elif family == "bimodal":
        long = p[3::4]
        short = np.delete(p, np.arange(3, 40, 4))
        assert (long >= 16384).all() and (long <= 32768).all() and (short <= 2048).all() and (short >= 256).all()
    elif family == "uniform":
        assert (p >= 1024).all() and (p <= 32768).all()
    else:
        assert (p % 256 == 0).all() and (p <= 32768).all()


@pytest.mark.parametrize("ext", ["csv", "json"])
def test_trace_file_roundtrip(tmp_path, ext):
    t = request_trace("uniform", 12, seed=1, arrival_gap=3)
    path = str(tmp_path / f"t.{ext}")
    save_trace(t, path)
    assert load_trace(path) == t


def test_trace_file_without_arrivals(tmp_path):
    path = tmp_path / "t.csv"
    path.write_text("prompt_len,decode_len\n100,5\n3000,7\n")
    assert load_trace(str(path)) == [Request(0, 0, 100, 5), Request(1, 0, 3000, 7)]
    bad = tmp_path / "b.json"
    bad.write_text('[{"prompt_len": 10, "decode_len": 0}]')
    with pytest.raises(ValueError):
        load_trace(str(bad))


def test_page_pool():
    pool = PagePool(100, seed=3)
    a = pool.alloc(30)
    b = pool.alloc(70)
    assert len(set(a) | set(b)) == 100 and pool.free_count == 0
    assert a != sorted(a)                      # scattered, not consecutive
    with pytest.raises(MemoryError):
        pool.alloc(1)
    pool.free(a)
    with pytest.raises(ValueError):
        pool.free(a[:1])                       # double free
    assert pool.free_count == 30 and sorted(pool.alloc(30)) == sorted(a)


class FakeEngine:
    def __init__(self, maxp):
        self.maxp = maxp
        self.lens = {}
        self.log = []

    def admit(self, slot, pages, prompt_len):
        assert slot not in self.lens
        self.lens[slot] = prompt_len
        self.log.append(("admit", slot, len(pages)))

    def release(self, slot):
        del self.lens[slot]
        self.log.append(("release", slot))

    def step(self, slots):
        assert sorted(slots) == sorted(self.lens)
        for s in slots:
            self.lens[s] += 1
        return {"attn_ms": 1.0, "step_ms": 2.0}


def test_scheduler_admission_and_completion():
    trace = [Request(0, 0, 100, 3), Request(1, 0, 40, 1), Request(2, 1, 16, 2), Request(3, 5, 10, 1)]
    eng = FakeEngine(maxp=16)
    pool = PagePool(64)
    s = Scheduler(trace, eng, pool, max_batch=2)
    recs = [s.step() for _ in range(4)]
    assert [r["active"] for r in recs] == [2, 2, 2, 0]        # step 3: request 3 has not arrived
    # step 0: rids 0, 1 admitted; rid 1 finishes after one token and frees its slot;
    # step 1: rid 2 takes it; rid 0 ends at step 2, rid 2 at step 2
    assert s.done == [1, 0, 2]
    while not s.finished:
        s.step()
    assert s.done == [1, 0, 2, 3] and pool.free_count == 64 and not s.active
    stats = s.run(100)
    # four steps had active rows (steps 3 and 4 were idle): 7 tokens over 4 x 2 ms
    assert stats["tokens"] == 3 + 1 + 2 + 1 and stats["steps"] == 4
    assert stats["device_tok_s"] == pytest.approx(1000.0 * 7 / (2.0 * 4))


def test_scheduler_waits_for_pages():
    # two requests each reserving ceil(200 / 16) = 13 pages; the pool holds 20
    trace = [Request(0, 0, 190, 10), Request(1, 0, 190, 10)]
    eng = FakeEngine(maxp=16)
    pool = PagePool(20)
    s = Scheduler(trace, eng, pool, max_batch=4)
    s.step()
    assert len(s.active) == 1 and pool.free_count == 20 - 13
    for _ in range(9):
        s.step()
    assert s.done == [0] and len(s.active) == 0
    s.step()
    assert len(s.active) == 1            # admitted once the first released its pages
    assert -(-200 // PAGE) == 13


def test_scheduler_rejects_oversized_request():
    s = Scheduler([Request(0, 0, 1000, 10)], FakeEngine(maxp=8), PagePool(100), max_batch=1)
    with pytest.raises(ValueError):
        s.step()
