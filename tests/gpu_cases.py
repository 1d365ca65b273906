"""Shared helpers for the GPU parity tests: seeded device inputs, one decode step through
the C ABI, and the tolerance check against the fp64 oracle."""
from __future__ import annotations

import numpy as np
import torch

import paper_2606_26666_amd as pkv
from workloads import make_workload, page_table
from workloads.values import device_normal_f16, host_normal_f16, poison_unassigned_pages, q_values

ABS_TOL = 2e-3   # max |out - ref|
REL_TOL = 1e-2   # max |out - ref| / max |ref| (normwise; elementwise relative error is ill-posed near 0)
MEAN_TOL = 3e-4  # mean |out - ref|, the paper's second correctness statistic (Sec. 3.6)
DEV = "cuda"


def rng(seed):
    return np.random.Generator(np.random.PCG64(seed))


class Case:
    """Inputs of one decode call, on the host (numpy, for the oracle) and the device."""

    def __init__(self, lens, hq=32, hkv=8, seed=0, rho=0.3, poison=True, device_values=False,
                 block_table=None, num_pages=None, values=True):
        r = rng(seed)
        self.lens = np.asarray(lens, dtype=np.int32)
        self.B, self.hq, self.hkv, self.d = len(lens), hq, hkv, 128
        if block_table is None:
            block_table, num_pages = page_table(np.maximum(self.lens, 1), 16, rho, r)
        self.bt = np.ascontiguousarray(block_table, dtype=np.int32)
        self.num_pages = int(num_pages)
        shape = (self.num_pages, 16, hkv, self.d)
        if not values:  # planner-only cases: a one-page pool
            shape = (1, 16, hkv, self.d)
        if device_values:
            self.k_dev = device_normal_f16(shape, seed * 2 + 1, DEV)
            self.v_dev = device_normal_f16(shape, seed * 2 + 2, DEV)
            if poison and values:
                poison_unassigned_pages(self.k_dev, self.bt)
                poison_unassigned_pages(self.v_dev, self.bt)
            self.k = self.k_dev.cpu().numpy()
            self.v = self.v_dev.cpu().numpy()
        else:
            self.k = host_normal_f16(shape, r)
            self.v = host_normal_f16(shape, r)
            if poison and values:
                poison_unassigned_pages(self.k, self.bt)
                poison_unassigned_pages(self.v, self.bt)
            self.k_dev = torch.from_numpy(self.k).to(DEV)
            self.v_dev = torch.from_numpy(self.v).to(DEV)
        self.q = q_values(self.B, hq, self.d, r)
        self.q_dev = torch.from_numpy(self.q).to(DEV)
        self.bt_dev = torch.from_numpy(self.bt).to(DEV)
        self.lens_dev = torch.from_numpy(self.lens).to(DEV)

    @classmethod
    def from_workload(cls, name, step=0, seed=20260622, poison=True, hkv=8):
        w = make_workload(name, seed=seed, hkv=hkv)
        return cls(w.lengths_at(step), hq=w.hq, hkv=w.hkv, seed=seed, poison=poison, device_values=True,
                   block_table=w.block_table, num_pages=w.num_pages), w


def plan_params(hkv, split_min=16, split_max=64, target=512, tile=32, policy=0):
    return pkv.make_params(hkv, split_min, split_max, target, tile_tokens=tile, policy=policy)


def run_plan(case, bufs, params, check_pages=False):
    pkv.pkv_plan(case.lens_dev, case.bt_dev if check_pages else None, case.num_pages, params, bufs.tasks,
                 bufs.split_offsets, bufs.num_tasks, bufs.ws, max_pages_per_row=case.bt.shape[1])


def read_plan(bufs):
    torch.cuda.synchronize()
    n = int(bufs.num_tasks.item())
    return bufs.tasks[:n].cpu().numpy(), bufs.split_offsets.cpu().numpy()


def run_decode(case, bufs, fused=True, sm_scale=1.0, poison_ws=True):
    if poison_ws:
        bufs.partial_region().fill_(0xFF)  # every partial slot starts as NaN
    out = torch.full((case.B, case.hq, case.d), float("nan"), dtype=torch.float16, device=DEV)
    pkv.pkv_decode(case.q_dev, case.k_dev, case.v_dev, case.bt_dev, case.lens_dev, bufs.tasks,
                   bufs.split_offsets, bufs.num_tasks, sm_scale, out, bufs.ws, fused=fused)
    return out


def run_rect(case, bufs, S, tile=32, sm_scale=1.0, poison_ws=True, row_ids=None, out=None):
    if poison_ws:
        bufs.partial_region().fill_(0xFF)
    if out is None:
        out = torch.full((case.B, case.hq, case.d), float("nan"), dtype=torch.float16, device=DEV)
    pkv.pkv_decode_rect(case.q_dev, case.k_dev, case.v_dev, case.bt_dev, case.lens_dev, S, tile, sm_scale,
                        out, bufs.ws, row_ids=row_ids)
    return out


def assert_close(out, ref, label=""):
    """The parity bar: max abs error <= 2e-3, normwise relative error <= 1e-2 and mean
    abs error < 3e-4."""
    o = out.float().cpu().numpy().astype(np.float64) if isinstance(out, torch.Tensor) else out
    assert np.all(np.isfinite(o)), f"{label}: non-finite output"
    err = np.abs(o - ref)
    amax = float(err.max()) if err.size else 0.0
    mean = float(err.mean()) if err.size else 0.0
    scale = float(np.abs(ref).max()) if ref.size else 0.0
    rel = amax / scale if scale > 0 else amax
    assert amax <= ABS_TOL, f"{label}: max abs err {amax:.3e}"
    assert rel <= REL_TOL, f"{label}: normwise rel err {rel:.3e}"
    assert mean < MEAN_TOL, f"{label}: mean abs err {mean:.3e}"
    return amax, rel


def error_stats(out, ref):
    """max |e|, mean |e| and the fraction within one fp16 ulp of fp16(ref)."""
    o = out.float().cpu().numpy().astype(np.float64)
    err = np.abs(o - ref)
    return float(err.max()), float(err.mean()), ulp_fraction(out, ref)


def ulp_fraction(out, ref):
    """Fraction of outputs within one fp16 ulp of fp16(ref)."""
    o = out.float().cpu().numpy().astype(np.float64)
    r16 = ref.astype(np.float16)
    spacing = np.spacing(np.abs(r16)).astype(np.float64)
    return float(np.mean(np.abs(o - r16.astype(np.float64)) <= spacing))
