"""The seeded inputs have the structure of the paper's workloads (Sec. 3.7-3.8)."""
import math

import numpy as np

from workloads import WORKLOADS, make_workload, page_table
from workloads.values import poison_unassigned_pages, unassigned_pages


def test_page_table_is_consecutive_slices_of_one_permutation():
    r = np.random.Generator(np.random.PCG64(0))
    reserved = np.array([100, 16, 1, 300])
    bt, universe = page_table(reserved, 16, 0.5, r)
    lp = [7, 1, 1, 19]
    assert universe == math.ceil(sum(lp) / 0.5)
    ids = np.concatenate([bt[i, :n] for i, n in enumerate(lp)])
    assert len(set(ids.tolist())) == len(ids) and ids.min() >= 0 and ids.max() < universe
    for i, n in enumerate(lp):
        assert np.all(bt[i, n:] == -1)
    # the same seed gives the same permutation: slices are consecutive pieces of it
    perm = np.random.Generator(np.random.PCG64(0)).permutation(universe)
    assert np.array_equal(ids, perm[:len(ids)])


def test_workload_shapes():
    for name in WORKLOADS:
        w = make_workload(name)
        last = w.lengths_at(w.steps - 1)
        assert np.all(last <= w.max_pages_per_row * w.page_size)
        assert w.block_table.max() < w.num_pages
    b1 = make_workload("b1")
    assert b1.num_pages == 4096 and b1.lengths_at(0)[0] == 32769 and b1.lengths_at(19)[0] == 32788
    assert b1.max_pages_per_row == 2050
    tiny = make_workload("tiny")
    assert tiny.lengths_at(0)[0] == 512 and tiny.max_pages_per_row == 32 and tiny.num_pages == 64
    bi = make_workload("b8_bimodal").seq_lens
    assert np.sum((bi >= 256) & (bi <= 2048)) == 4 and np.sum((bi >= 16384) & (bi <= 32768)) == 4
    z = make_workload("b8_zipf").seq_lens
    assert np.all(z % 256 == 0) and np.all(z <= 32768)


def test_poison_marks_only_unowned_pages():
    w = make_workload("tiny")
    pool = np.zeros((w.num_pages, 16, 1, 2), dtype=np.float16)
    poison_unassigned_pages(pool, w.block_table)
    owned = w.block_table[w.block_table >= 0]
    assert np.all(np.isfinite(pool[owned]))
    assert np.all(np.isnan(pool[unassigned_pages(w.block_table, w.num_pages)]))
