"""Seeded synthetic inputs for paged GQA decode: lengths, block tables, Q/K/V values.

This module holds no attention or planning arithmetic. It is the one piece shared by
the fp64 oracle's tests and the HIP path's tests and benchmark: both sides receive
the same arrays from here.

Workload shapes follow the paper's setup (Sec. 3.6-3.8, Sec. 4.1): Hq=32, Hkv=8,
d=128, fp16, page size 16, and the page-table construction of Sec. 3.7.
"""
from .traces import (  # noqa: F401
    WORKLOADS,
    Workload,
    bimodal_lengths,
    make_workload,
    page_table,
    uniform_lengths,
    zipf_lengths,
)
from .values import (  # noqa: F401
    host_normal_f16,
    poison_unassigned_pages,
    q_values,
)
