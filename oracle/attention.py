"""Reference paged GQA decode attention in fp64 (Eq. 1, Sec. 3.1-3.3).

TEST INFRASTRUCTURE: see the package docstring. Parity pins: tests/test_oracle_attention.py.

Layout (the native serving layout taken for this build): K and V pools are
[num_pages, page_size, Hkv, d]; token j of row i is slot j % P of physical page
block_table[i, j // P] (Sec. 3.2). Query head h reads KV head h // G with
G = Hq / Hkv, i.e. heads [g*G, (g+1)*G) share KV head g (Sec. 3.1). All arithmetic is
fp64 on exactly converted fp16 inputs; nothing is rounded back to fp16 here.
"""
from __future__ import annotations

import numpy as np

from .plan import row_split_bounds


def gather_row(cache: np.ndarray, block_table_row: np.ndarray, n: int) -> np.ndarray:
    """The row's first n cached tokens as fp64 [n, Hkv, d], read through its block table."""
    num_pages, page_size, hkv, d = cache.shape
    if n == 0:
        return np.zeros((0, hkv, d), dtype=np.float64)
    npages = -(-n // page_size)
    pages = np.asarray(block_table_row[:npages], dtype=np.int64)
    if pages.size < npages or pages.min() < 0 or pages.max() >= num_pages:
        raise ValueError("block table entry outside the page pool")
    rows = cache[pages].reshape(npages * page_size, hkv, d)[:n]
    return rows.astype(np.float64)


def _check(q, k_cache, v_cache):
    b, hq, d = q.shape
    hkv = k_cache.shape[2]
    if k_cache.shape != v_cache.shape or k_cache.shape[3] != d or hq % hkv:
        raise ValueError("inconsistent shapes")
    return b, hq, hkv, hq // hkv, d


def ref_decode(q, k_cache, v_cache, block_table, seq_lens, sm_scale: float = 1.0) -> np.ndarray:
    """Eq. (1): O[i,h] = sum_j softmax_j(sm_scale * q[i,h].K_i[j]) V_i[j] over the row's
    seq_lens[i] tokens, KV head h // G. Rows of length 0 give 0. Returns fp64 [B, Hq, d]."""
    b, hq, hkv, G, d = _check(q, k_cache, v_cache)
    out = np.zeros((b, hq, d), dtype=np.float64)
    for i in range(b):
        n = int(seq_lens[i])
        if n == 0:
            continue
        K = gather_row(k_cache, block_table[i], n)
        V = gather_row(v_cache, block_table[i], n)
        for h in range(hq):
            g = h // G
            s = sm_scale * (K[:, g, :] @ q[i, h].astype(np.float64))
            w = np.exp(s - s.max())
            out[i, h] = (w @ V[:, g, :]) / w.sum()
    return out


def ref_split_state(q_h: np.ndarray, K: np.ndarray, V: np.ndarray, sm_scale: float):
    """Partial state of one split for one query head (Sec. 3.3):
    m = max_j x_j, l = sum_j exp(x_j - m), a = sum_j exp(x_j - m) v_j, x_j = sm_scale q.k_j.
    An empty split is the neutral state (-inf, 0, 0)."""
    d = q_h.shape[0]
    if K.shape[0] == 0:
        return -np.inf, 0.0, np.zeros(d, dtype=np.float64)
    x = sm_scale * (K @ q_h.astype(np.float64))
    m = x.max()
    e = np.exp(x - m)
    return m, e.sum(), e @ V


def ref_merge(states) -> np.ndarray:
    """Exact merge of split states in the given order (Sec. 3.3):
    m = max m_s, l = sum exp(m_s - m) l_s, a = sum exp(m_s - m) a_s, O = a / l.
    When every state is neutral (l = 0) the output is 0."""
    ms = np.array([s[0] for s in states], dtype=np.float64)
    m = ms.max()
    if m == -np.inf:
        return np.zeros_like(states[0][2])
    l = 0.0
    a = np.zeros_like(states[0][2])
    for ms_, ls_, as_ in states:
        c = np.exp(ms_ - m)
        l += c * ls_
        a = a + c * as_
    return a / l


def ref_decode_split(q, k_cache, v_cache, block_table, seq_lens, tasks, split_offsets,
                     sm_scale: float = 1.0):
    """Workqueue evaluation: a partial state per (task, query head of the task's group),
    then a segmented merge over each (row, kv head)'s split range in split order.

    Returns (out fp64 [B,Hq,d], m [T,G], l [T,G], a [T,G,d]) with T = len(tasks); the
    task's index is its slot, (split_offsets[i] + s) * Hkv + g."""
    b, hq, hkv, G, d = _check(q, k_cache, v_cache)
    T = len(tasks)
    m = np.full((T, G), -np.inf)
    l = np.zeros((T, G))
    a = np.zeros((T, G, d))
    rows = {}
    for t, (i, g, s, t0, t1) in enumerate(np.asarray(tasks).tolist()):
        if (split_offsets[i] + s) * hkv + g != t:
            raise ValueError("task order does not match split_offsets")
        if i not in rows:
            n = int(seq_lens[i])
            rows[i] = (gather_row(k_cache, block_table[i], n), gather_row(v_cache, block_table[i], n))
        K, V = rows[i]
        for j in range(G):
            h = g * G + j
            m[t, j], l[t, j], a[t, j] = ref_split_state(q[i, h], K[t0:t1, g, :], V[t0:t1, g, :], sm_scale)
    out = np.zeros((b, hq, d))
    for i in range(b):
        ns = int(split_offsets[i + 1] - split_offsets[i])
        if ns == 0:
            continue
        for g in range(hkv):
            slots = [(int(split_offsets[i]) + s) * hkv + g for s in range(ns)]
            for j in range(G):
                out[i, g * G + j] = ref_merge([(m[k, j], l[k, j], a[k, j]) for k in slots])
    return out, m, l, a


def ref_decode_rect(q, k_cache, v_cache, block_table, seq_lens, S: int, tile_tokens: int,
                    sm_scale: float = 1.0):
    """Rectangular (B, Hkv, S) split grid (Sec. 3.4): every row gets S split columns;
    column s of row i owns the s-th balanced tile range when s < min(S, tiles_i) and is
    otherwise empty, contributing the neutral state (Sec. 3.3). Merge runs over all S
    columns in order. Returns out fp64 [B, Hq, d]."""
    b, hq, hkv, G, d = _check(q, k_cache, v_cache)
    out = np.zeros((b, hq, d))
    for i in range(b):
        n = int(seq_lens[i])
        K = gather_row(k_cache, block_table[i], n)
        V = gather_row(v_cache, block_table[i], n)
        bounds = row_split_bounds(n, S, tile_tokens)
        bounds = bounds + [(0, 0)] * (S - len(bounds))
        for h in range(hq):
            g = h // G
            states = [ref_split_state(q[i, h], K[t0:t1, g, :], V[t0:t1, g, :], sm_scale)
                      for (t0, t1) in bounds]
            out[i, h] = ref_merge(states)
    return out
