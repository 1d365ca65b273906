"""Pins of the fp64 attention oracle against facts fixed outside it: closed forms,
invariants of Eq. (1), the split/merge identity of Sec. 3.3, and torch's fp64 SDPA as an
independent library routine (the paper's own reference path, Sec. 3.9)."""
import math

import numpy as np
import pytest
import torch

from oracle import PlanParams, ref_decode, ref_decode_rect, ref_decode_split, ref_plan

P = 16


def rng(seed):
    return np.random.Generator(np.random.PCG64(seed))


def scatter_pool(kc, vc, num_pages, r, fill=np.nan):
    """Place contiguous per-row K/V ([n, Hkv, d] each) into a paged NHD pool through a
    random block table, one token at a time (the inverse of a block-table read)."""
    rows = len(kc)
    hkv, d = kc[0].shape[1:]
    need = [-(-k.shape[0] // P) for k in kc]
    perm = r.permutation(num_pages)
    maxp = max(1, max(need))
    bt = np.full((rows, maxp), -1, dtype=np.int32)
    kpool = np.full((num_pages, P, hkv, d), fill, dtype=np.float16)
    vpool = np.full((num_pages, P, hkv, d), fill, dtype=np.float16)
    off = 0
    for i in range(rows):
        bt[i, :need[i]] = perm[off:off + need[i]]
        off += need[i]
        for j in range(kc[i].shape[0]):
            page, slot = bt[i, j // P], j % P
            for g in range(hkv):
                kpool[page, slot, g, :] = kc[i][j, g, :]
                vpool[page, slot, g, :] = vc[i][j, g, :]
    return kpool, vpool, bt


def random_rows(lens, hkv, d, r):
    kc = [r.standard_normal((n, hkv, d)).astype(np.float16) for n in lens]
    vc = [r.standard_normal((n, hkv, d)).astype(np.float16) for n in lens]
    return kc, vc


def sdpa_fp64(q_row, K, V, scale):
    """torch SDPA in fp64 on one row: q [Hq,d], K/V [n,Hkv,d] with KV heads repeated so
    query head h reads KV head h // G."""
    hq = q_row.shape[0]
    hkv = K.shape[1]
    G = hq // hkv
    qt = torch.from_numpy(q_row.astype(np.float64))[None, :, None, :]
    kt = torch.from_numpy(K.astype(np.float64)).permute(1, 0, 2).repeat_interleave(G, dim=0)[None]
    vt = torch.from_numpy(V.astype(np.float64)).permute(1, 0, 2).repeat_interleave(G, dim=0)[None]
    o = torch.nn.functional.scaled_dot_product_attention(qt, kt.contiguous(), vt.contiguous(), scale=scale)
    return o[0, :, 0, :].numpy()


@pytest.mark.parametrize("lens,hq,hkv,scale", [
    ([1, 17, 40, 100], 8, 2, 1.0),
    ([33, 5], 32, 8, 1.0 / math.sqrt(128)),
    ([64, 3, 129], 4, 4, 0.37),
    ([50], 8, 1, 1.3),
])
def test_matches_torch_sdpa_on_contiguous_data(lens, hq, hkv, scale):
    r = rng(1)
    d = 32 if hq != 32 else 128
    kc, vc = random_rows(lens, hkv, d, r)
    kpool, vpool, bt = scatter_pool(kc, vc, sum(-(-n // P) for n in lens) + 5, r)
    q = r.standard_normal((len(lens), hq, d)).astype(np.float16)
    out = ref_decode(q, kpool, vpool, bt, np.array(lens), scale)
    for i in range(len(lens)):
        np.testing.assert_allclose(out[i], sdpa_fp64(q[i], kc[i], vc[i], scale), rtol=1e-12, atol=1e-13)


def test_one_token_context_returns_v_exactly():
    r = rng(2)
    lens = [1, 1, 1]
    kc, vc = random_rows(lens, 4, 16, r)
    kpool, vpool, bt = scatter_pool(kc, vc, 8, r)
    q = r.standard_normal((3, 8, 16)).astype(np.float16)
    out = ref_decode(q, kpool, vpool, bt, np.array(lens))
    for i in range(3):
        for h in range(8):
            assert np.array_equal(out[i, h], vc[i][0, h // 2].astype(np.float64))


def test_constant_v_returns_the_constant():
    r = rng(3)
    lens = [70, 16]
    kc, _ = random_rows(lens, 2, 16, r)
    c = r.standard_normal((2, 16)).astype(np.float16)  # one constant vector per KV head
    vc = [np.broadcast_to(c, (n, 2, 16)).copy() for n in lens]
    kpool, vpool, bt = scatter_pool(kc, vc, 12, r)
    q = r.standard_normal((2, 4, 16)).astype(np.float16)
    out = ref_decode(q, kpool, vpool, bt, np.array(lens))
    for i in range(2):
        for h in range(4):
            np.testing.assert_allclose(out[i, h], c[h // 2].astype(np.float64), rtol=1e-14, atol=1e-15)


def test_zero_query_gives_mean_of_v():
    r = rng(4)
    lens = [45]
    kc, vc = random_rows(lens, 2, 16, r)
    kpool, vpool, bt = scatter_pool(kc, vc, 4, r)
    q = np.zeros((1, 4, 16), dtype=np.float16)
    out = ref_decode(q, kpool, vpool, bt, np.array(lens))
    for h in range(4):
        np.testing.assert_allclose(out[0, h], vc[0][:, h // 2].astype(np.float64).mean(0), rtol=1e-13)


def test_two_token_logistic_closed_form():
    # With two tokens the weights are the logistic function of the score gap:
    # w1 = (1 + tanh((s1 - s2)/2)) / 2, w2 = 1 - w1.
    r = rng(5)
    kc, vc = random_rows([2], 1, 8, r)
    kpool, vpool, bt = scatter_pool(kc, vc, 2, r)
    q = r.standard_normal((1, 1, 8)).astype(np.float16)
    scale = 0.8
    out = ref_decode(q, kpool, vpool, bt, np.array([2]), scale)
    k = kc[0][:, 0].astype(np.float64)
    v = vc[0][:, 0].astype(np.float64)
    qq = q[0, 0].astype(np.float64)
    s1 = scale * sum(qq[t] * k[0, t] for t in range(8))
    s2 = scale * sum(qq[t] * k[1, t] for t in range(8))
    w1 = 0.5 * (1.0 + math.tanh(0.5 * (s1 - s2)))
    np.testing.assert_allclose(out[0, 0], w1 * v[0] + (1.0 - w1) * v[1], rtol=1e-13, atol=1e-15)


def test_hard_attention_limit_without_overflow():
    # Scores of order 1e4: softmax collapses onto the top token; a missing
    # max-subtraction overflows exp and gives NaN.
    r = rng(6)
    kc, vc = random_rows([300], 1, 16, r)
    kpool, vpool, bt = scatter_pool(kc, vc, 20, r)
    q = r.standard_normal((1, 1, 16)).astype(np.float16)
    scale = 2000.0
    s = (kc[0][:, 0].astype(np.float64) @ q[0, 0].astype(np.float64)) * scale
    top = np.argsort(s)[::-1]
    assert s[top[0]] - s[top[1]] > 50  # the seeded draw has a clear winner
    out = ref_decode(q, kpool, vpool, bt, np.array([300]), scale)
    assert np.all(np.isfinite(out))
    np.testing.assert_allclose(out[0, 0], vc[0][top[0], 0].astype(np.float64), rtol=0, atol=1e-15)


def test_gqa_grouping_is_contiguous():
    # V of KV head g is the constant g+1; query head h must see h // G + 1, and changing
    # the keys of any other KV head must not move it.
    r = rng(7)
    hkv, hq, d = 4, 16, 8
    kc, _ = random_rows([20], hkv, d, r)
    vc = [np.stack([np.full((20, d), g + 1.0) for g in range(hkv)], axis=1).astype(np.float16)]
    kpool, vpool, bt = scatter_pool(kc, vc, 4, r)
    q = r.standard_normal((1, hq, d)).astype(np.float16)
    out = ref_decode(q, kpool, vpool, bt, np.array([20]))
    for h in range(hq):
        np.testing.assert_allclose(out[0, h], np.full(d, h // (hq // hkv) + 1.0), rtol=1e-14)
    vc2 = [r.standard_normal((20, hkv, d)).astype(np.float16)]
    kpool, vpool, bt = scatter_pool(kc, vc2, 4, rng(70))
    base = ref_decode(q, kpool, vpool, bt, np.array([20]))
    kc_mod = [kc[0].copy()]
    kc_mod[0][:, 3] = r.standard_normal((20, d)).astype(np.float16)
    kpool2, vpool2, bt2 = scatter_pool(kc_mod, vc2, 4, rng(70))
    mod = ref_decode(q, kpool2, vpool2, bt2, np.array([20]))
    assert np.array_equal(base[0, :12], mod[0, :12])
    assert not np.array_equal(base[0, 12:], mod[0, 12:])


def test_physical_page_permutation_invariance():
    r = rng(8)
    lens = [37, 100, 16]
    kc, vc = random_rows(lens, 2, 16, r)
    a = scatter_pool(kc, vc, 40, rng(80))
    b = scatter_pool(kc, vc, 40, rng(81))
    assert not np.array_equal(a[2], b[2])
    q = r.standard_normal((3, 4, 16)).astype(np.float16)
    oa = ref_decode(q, *a[:2], a[2], np.array(lens))
    ob = ref_decode(q, *b[:2], b[2], np.array(lens))
    assert np.array_equal(oa, ob)


def test_unowned_slots_are_never_read():
    # Pool filled with NaN outside the rows' tokens: a read past seq_len or outside the
    # block table would make the output NaN.
    r = rng(9)
    lens = [1, 15, 17, 33]
    kc, vc = random_rows(lens, 2, 16, r)
    kpool, vpool, bt = scatter_pool(kc, vc, 20, r, fill=np.nan)
    q = r.standard_normal((4, 4, 16)).astype(np.float16)
    assert np.all(np.isfinite(ref_decode(q, kpool, vpool, bt, np.array(lens))))


def test_empty_row_is_zero():
    r = rng(10)
    kc, vc = random_rows([5, 0], 2, 16, r)
    kpool, vpool, bt = scatter_pool(kc, vc, 4, r)
    q = r.standard_normal((2, 4, 16)).astype(np.float16)
    out = ref_decode(q, kpool, vpool, bt, np.array([5, 0]))
    assert np.all(out[1] == 0)


@pytest.mark.parametrize("S", [1, 2, 7, 16, 64])
def test_split_merge_equals_unsplit(S):
    r = rng(11)
    lens = [1, 31, 32, 33, 300, 1000, 0]
    kc, vc = random_rows(lens, 2, 16, r)
    kpool, vpool, bt = scatter_pool(kc, vc, 120, r)
    q = r.standard_normal((len(lens), 8, 16)).astype(np.float16)
    full = ref_decode(q, kpool, vpool, bt, np.array(lens), 0.9)
    p = PlanParams(num_kv_heads=2, split_min=S, split_max=S)
    tasks, offs, _ = ref_plan(lens, p)
    out, m, l, a = ref_decode_split(q, kpool, vpool, bt, np.array(lens), tasks, offs, 0.9)
    np.testing.assert_allclose(out, full, rtol=1e-12, atol=1e-14)
    rect = ref_decode_rect(q, kpool, vpool, bt, np.array(lens), S, 32, 0.9)
    np.testing.assert_allclose(rect, full, rtol=1e-12, atol=1e-14)
    assert np.all(l > 0)  # every emitted task is non-empty


def test_partial_states_match_direct_sums():
    # One task covering tokens [32, 64): its state is (max x, sum e^{x-m}, sum e^{x-m} v).
    r = rng(12)
    kc, vc = random_rows([64], 1, 8, r)
    kpool, vpool, bt = scatter_pool(kc, vc, 4, r)
    q = r.standard_normal((1, 2, 8)).astype(np.float16)
    tasks = np.array([[0, 0, 0, 0, 32], [0, 0, 1, 32, 64]], dtype=np.int32)
    _, m, l, a = ref_decode_split(q, kpool, vpool, bt, np.array([64]), tasks, np.array([0, 2]))
    k = kc[0][32:, 0].astype(np.float64)
    v = vc[0][32:, 0].astype(np.float64)
    for j in range(2):
        x = [sum(float(q[0, j, t]) * k[n, t] for t in range(8)) for n in range(32)]
        mx = max(x)
        assert m[1, j] == pytest.approx(mx, rel=1e-14)
        assert l[1, j] == pytest.approx(sum(math.exp(xi - mx) for xi in x), rel=1e-13)
        ref_a = [sum(math.exp(x[n] - mx) * v[n, t] for n in range(32)) for t in range(8)]
        np.testing.assert_allclose(a[1, j], ref_a, rtol=1e-12, atol=1e-14)
