"""Seeded Q/K/V values.

Pool pages hold fp16(N(0,1)) for every slot, including pages no request owns; parity
runs overwrite unowned pages with NaN so a read outside the block table shows up in
the output. Queries are fp16(N(0,1)/sqrt(d)): the 1/sqrt(d) of Eq. (1) is folded into
the stored query, so the softmax scale passed to the attention call is 1.

Host generation (numpy PCG64) serves small and medium cases. Pools of hundreds of MB
are generated on the device with torch's seeded Philox generator; a parity test that
needs them on the host copies the same tensor back.
"""
from __future__ import annotations

import numpy as np


def host_normal_f16(shape, rng: np.random.Generator, scale: float = 1.0) -> np.ndarray:
    x = rng.standard_normal(int(np.prod(shape)), dtype=np.float32)
    if scale != 1.0:
        x *= np.float32(scale)
    return x.astype(np.float16).reshape(shape)


def q_values(batch: int, hq: int, head_dim: int, rng: np.random.Generator) -> np.ndarray:
    return host_normal_f16((batch, hq, head_dim), rng, scale=1.0 / np.sqrt(head_dim))


def unassigned_pages(block_table: np.ndarray, num_pages: int) -> np.ndarray:
    used = np.zeros(num_pages, dtype=bool)
    bt = block_table[block_table >= 0]
    used[bt] = True
    return np.nonzero(~used)[0]


def poison_unassigned_pages(pool, block_table: np.ndarray):
    """Write NaN into every pool page that no block-table entry names (host numpy array
    or torch tensor, shape [num_pages, P, Hkv, d])."""
    idx = unassigned_pages(block_table, pool.shape[0])
    if idx.size:
        try:
            import torch
            if isinstance(pool, torch.Tensor):
                pool[torch.as_tensor(idx, device=pool.device)] = float("nan")
                return pool
        except ImportError:  # pragma: no cover
            pass
        pool[idx] = np.nan
    return pool


def device_normal_f16(shape, seed: int, device):
    """fp16(N(0,1)) of `shape` drawn on `device` from torch's seeded generator."""
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(int(seed))
    return torch.randn(tuple(shape), generator=g, device=device, dtype=torch.float32).to(torch.float16)
