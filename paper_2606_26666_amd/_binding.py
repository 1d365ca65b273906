"""ctypes binding of libpkv.so (include/pkv.h), with the same entry-point names.

Argument marshalling only: tensors are checked for device, dtype and contiguity and
passed as raw pointers with torch's current HIP stream. Every step of the decode path
runs in the library's kernels; there is no fallback when the library is missing.
"""
from __future__ import annotations

import ctypes
import os
import re

import torch

HERE = os.path.dirname(os.path.abspath(__file__))
# PKV_LIBRARY selects another build of the same sources (an A/B build for measurement)
LIB_PATH = os.environ.get("PKV_LIBRARY") or os.path.join(HERE, "libpkv.so")
HEADER = os.path.join(os.path.dirname(HERE), "include", "pkv.h")

PKV_OK = 0
PKV_ERR_INVALID_ARG = 1
PKV_ERR_UNSUPPORTED = 2
PKV_ERR_WORKSPACE = 3
PKV_ERR_HIP = 4
PKV_ERR_DEVICE = 5
PKV_DEVERR_SEQ_LEN = 1
PKV_DEVERR_PAGE_ID = 2
PKV_DEVERR_TASK = 4
PKV_FUSED_MERGE = 1
PKV_SPLIT_BATCH = 0
PKV_SPLIT_QUOTA = 1
TASK_FIELDS = 5  # row, kvh, split, t_begin, t_end


class PkvError(RuntimeError):
    def __init__(self, fn: str, status: int, msg: str):
        super().__init__(f"{fn}: {msg} (status {status})")
        self.status = status


class PlanParams(ctypes.Structure):
    _fields_ = [("page_size", ctypes.c_int32), ("tile_tokens", ctypes.c_int32),
                ("num_kv_heads", ctypes.c_int32), ("split_min", ctypes.c_int32),
                ("split_max", ctypes.c_int32), ("target_tasks", ctypes.c_int32), ("policy", ctypes.c_int32)]


_lib = None
_P, _I32, _F32, _SZ = ctypes.c_void_p, ctypes.c_int32, ctypes.c_float, ctypes.c_size_t
_SIGS = {
    "pkv_max_tasks": (_I32, [_I32, _I32, _I32]),
    "pkv_workspace_size": (_SZ, [_I32, _I32, _I32, _I32, _I32]),
    "pkv_workspace_init": (ctypes.c_int, [_P, _SZ, _I32, _I32, _P]),
    "pkv_plan": (ctypes.c_int, [_P, _P, _I32, _I32, _I32, ctypes.POINTER(PlanParams), _P, _I32, _P, _P,
                                _P, _SZ, _P]),
    "pkv_plan_host": (ctypes.c_int, [_P, _I32, _I32, ctypes.POINTER(PlanParams), _P, _I32, _P, _P]),
    "pkv_decode": (ctypes.c_int, [_P, _P, _P, _I32, _P, _I32, _P, _I32, _I32, _I32, _I32, _P, _P, _P, _I32,
                                  _F32, _I32, _P, _P, _SZ, _P]),
    "pkv_plan_decode": (ctypes.c_int, [_P, _P, _P, _I32, _P, _I32, _P, _I32, _I32, _I32, _I32,
                                       ctypes.POINTER(PlanParams), _P, _I32, _P, _P, _F32, _P, _P, _SZ, _P]),
    "pkv_plan_decode_noalloc": (ctypes.c_int, [_P, _P, _P, _I32, _P, _I32, _P, _I32, _I32, _I32, _I32,
                                               ctypes.POINTER(PlanParams), _P, _I32, _P, _P, _F32, _P, _P, _P]),
    "pkv_decode_timed": (ctypes.c_int, [_P, _P, _P, _I32, _P, _I32, _P, _I32, _I32, _I32, _I32, _P, _P, _P,
                                        _I32, _F32, _I32, _P, _P, _SZ, _P, _P, _P]),
    "pkv_plan_decode_timed": (ctypes.c_int, [_P, _P, _P, _I32, _P, _I32, _P, _I32, _I32, _I32, _I32,
                                             ctypes.POINTER(PlanParams), _P, _I32, _P, _P, _F32, _P, _P, _SZ,
                                             _P, _P, _P]),
    "pkv_decode_rect": (ctypes.c_int, [_P, _P, _P, _I32, _P, _I32, _P, _I32, _I32, _I32, _I32, _P, _I32, _I32,
                                       _I32, _F32, _P, _P, _SZ, _P]),
    "pkv_decode_buckets": (ctypes.c_int, [_P, _P, _P, _I32, _P, _I32, _P, _P, _I32, _I32, _I32, _I32, _I32,
                                          ctypes.POINTER(PlanParams), _F32, _P, _P, _SZ, _P,
                                          ctypes.POINTER(ctypes.c_int32)]),
    "pkv_check_device_status": (ctypes.c_int, [_P, _P, ctypes.POINTER(ctypes.c_uint32)]),
    "pkv_status_string": (ctypes.c_char_p, [ctypes.c_int]),
    "pkv_stream_copy": (ctypes.c_int, [_P, _P, _SZ, _P]),
    "pkv_stream_read": (ctypes.c_int, [_P, _SZ, _P, _P]),
    "pkv_stream_read_timed": (ctypes.c_int, [_P, _SZ, _P, _P, _P, _P]),
    "pkv_stream_read_nt_timed": (ctypes.c_int, [_P, _SZ, _P, _P, _P, _P]),
    "pkv_stream_read_pages": (ctypes.c_int, [_P, _P, _I32, _P, _I32, _I32, _I32, _I32, _P, _P, _I32, _I32, _P,
                                             _P, _P, _P]),
}


def lib() -> ctypes.CDLL:
    """Load libpkv.so built in-tree (paper_2606_26666_amd.build). Raises if absent."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with paper_2606_26666_amd.build.build()")
        L = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGS.items():
            fn = getattr(L, name)
            fn.restype = res
            fn.argtypes = args
        _lib = L
    return _lib


def header_functions() -> list[str]:
    """Names of the functions declared in include/pkv.h."""
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^\s*(?:[\w\s\*]+?)\b(pkv_\w+)\s*\(", text, flags=re.M)))


def _check(fn: str, st: int):
    if st != PKV_OK:
        raise PkvError(fn, st, lib().pkv_status_string(st).decode())


def _stream(stream) -> int:
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)


def _dev(t: torch.Tensor, dtype: torch.dtype, name: str) -> int:
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError(f"{name} must be a device tensor")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return t.data_ptr()


def pkv_max_tasks(B: int, Hkv: int, split_max: int) -> int:
    return int(lib().pkv_max_tasks(B, Hkv, split_max))


def pkv_workspace_size(B: int, Hq: int, Hkv: int, d: int, max_tasks: int) -> int:
    return int(lib().pkv_workspace_size(B, Hq, Hkv, d, max_tasks))


def pkv_workspace_init(ws: torch.Tensor, B: int, Hkv: int, stream=None):
    _check("pkv_workspace_init", lib().pkv_workspace_init(_dev(ws, torch.uint8, "ws"), ws.numel(), B, Hkv,
                                                          _stream(stream)))


def make_params(num_kv_heads: int, split_min: int, split_max: int, target_tasks: int,
                tile_tokens: int = 32, page_size: int = 16, policy: int = 0) -> PlanParams:
    return PlanParams(page_size, tile_tokens, num_kv_heads, split_min, split_max, target_tasks, policy)


def pkv_plan(seq_lens: torch.Tensor, block_table, num_pages: int, params: PlanParams, tasks: torch.Tensor,
             split_offsets: torch.Tensor, num_tasks: torch.Tensor, ws: torch.Tensor, *,
             max_pages_per_row: int | None = None, stream=None):
    """tasks: int32 [max_tasks, 5]; block_table may be None (no plan-time page check)."""
    B = seq_lens.numel()
    if max_pages_per_row is None:
        max_pages_per_row = block_table.shape[1]
    bt = 0 if block_table is None else _dev(block_table, torch.int32, "block_table")
    _check("pkv_plan", lib().pkv_plan(_dev(seq_lens, torch.int32, "seq_lens"), bt, B, max_pages_per_row,
                                      num_pages, ctypes.byref(params), _dev(tasks, torch.int32, "tasks"),
                                      tasks.numel() // TASK_FIELDS,
                                      _dev(split_offsets, torch.int32, "split_offsets"),
                                      _dev(num_tasks, torch.int32, "num_tasks"), _dev(ws, torch.uint8, "ws"),
                                      ws.numel(), _stream(stream)))


def pkv_plan_host(seq_lens, params: PlanParams, max_pages_per_row: int, with_tasks: bool = True):
    """Host planner: (tasks int32 [n, 5] or None, split_offsets int32 [B+1], n) from host
    lengths, identical to the device plan."""
    import numpy as np
    lens = np.ascontiguousarray(np.asarray(seq_lens, dtype=np.int32).reshape(-1))
    B = lens.size
    offs = np.zeros(B + 1, dtype=np.int32)
    n = ctypes.c_int32(0)
    _check("pkv_plan_host", lib().pkv_plan_host(lens.ctypes.data, B, int(max_pages_per_row), ctypes.byref(params),
                                                None, 0, offs.ctypes.data, ctypes.byref(n)))
    if not with_tasks:
        return None, offs, n.value
    tasks = np.zeros((max(1, n.value), TASK_FIELDS), dtype=np.int32)
    _check("pkv_plan_host", lib().pkv_plan_host(lens.ctypes.data, B, int(max_pages_per_row), ctypes.byref(params),
                                                tasks.ctypes.data, tasks.shape[0], offs.ctypes.data,
                                                ctypes.byref(n)))
    return tasks[:n.value], offs, n.value


def _events(events) -> tuple:
    """(start, stop) torch timing events -> raw handles. torch creates an event's handle
    on its first record, so each is recorded once here before its handle is taken."""
    if events is None:
        return None
    out = []
    for ev in events:
        ev.record()
        out.append(ev.cuda_event)
    return tuple(out)


def pkv_decode(q: torch.Tensor, k_cache: torch.Tensor, v_cache: torch.Tensor, block_table: torch.Tensor,
               seq_lens: torch.Tensor, tasks: torch.Tensor, split_offsets: torch.Tensor, num_tasks: torch.Tensor,
               sm_scale: float, out: torch.Tensor, ws: torch.Tensor, *, fused: bool = True, stream=None,
               events=None):
    """events: optional (start, stop) timing events stamped with the kernels' execution
    interval (pkv_decode_timed)."""
    B, Hq, d = q.shape
    num_pages, _, Hkv, _ = k_cache.shape
    ev = _events(events)
    args = (_dev(q, torch.float16, "q"), _dev(k_cache, torch.float16, "k_cache"),
            _dev(v_cache, torch.float16, "v_cache"), num_pages, _dev(block_table, torch.int32, "block_table"),
            block_table.shape[1], _dev(seq_lens, torch.int32, "seq_lens"), B, Hq, Hkv, d,
            _dev(tasks, torch.int32, "tasks"), _dev(split_offsets, torch.int32, "split_offsets"),
            _dev(num_tasks, torch.int32, "num_tasks"), tasks.numel() // TASK_FIELDS, float(sm_scale),
            PKV_FUSED_MERGE if fused else 0, _dev(out, torch.float16, "out"), _dev(ws, torch.uint8, "ws"),
            ws.numel(), _stream(stream))
    if ev is None:
        _check("pkv_decode", lib().pkv_decode(*args))
    else:
        _check("pkv_decode_timed", lib().pkv_decode_timed(*args, *ev))


def pkv_plan_decode(q: torch.Tensor, k_cache: torch.Tensor, v_cache: torch.Tensor, block_table: torch.Tensor,
                    seq_lens: torch.Tensor, params: PlanParams, tasks: torch.Tensor, split_offsets: torch.Tensor,
                    num_tasks: torch.Tensor, sm_scale: float, out: torch.Tensor, ws: torch.Tensor, *, stream=None,
                    events=None):
    """Plan, attend and merge in one launch (see include/pkv.h). `tasks` is written with the
    plan; its previous contents are only a scheduling hint (any contents are allowed).
    events: optional (start, stop) timing events (pkv_plan_decode_timed)."""
    B, Hq, d = q.shape
    num_pages, _, Hkv, _ = k_cache.shape
    ev = _events(events)
    args = (_dev(q, torch.float16, "q"), _dev(k_cache, torch.float16, "k_cache"),
            _dev(v_cache, torch.float16, "v_cache"), num_pages, _dev(block_table, torch.int32, "block_table"),
            block_table.shape[1], _dev(seq_lens, torch.int32, "seq_lens"), B, Hq, Hkv, d, ctypes.byref(params),
            _dev(tasks, torch.int32, "tasks"), tasks.numel() // TASK_FIELDS,
            _dev(split_offsets, torch.int32, "split_offsets"), _dev(num_tasks, torch.int32, "num_tasks"),
            float(sm_scale), _dev(out, torch.float16, "out"), _dev(ws, torch.uint8, "ws"), ws.numel(),
            _stream(stream))
    if ev is None:
        _check("pkv_plan_decode", lib().pkv_plan_decode(*args))
    else:
        _check("pkv_plan_decode_timed", lib().pkv_plan_decode_timed(*args, *ev))


def pkv_plan_decode_noalloc(q: torch.Tensor, k_cache: torch.Tensor, v_cache: torch.Tensor,
                            block_table: torch.Tensor, seq_lens: torch.Tensor, params: PlanParams,
                            tasks: torch.Tensor, split_offsets: torch.Tensor, num_tasks: torch.Tensor,
                            sm_scale: float, out: torch.Tensor, error_bits: torch.Tensor, *, stream=None):
    """pkv_plan_decode without a caller workspace: counters and partial states live in the
    library's per-device scratch (see include/pkv.h). error_bits: int32 [1] device tensor
    that device error bits are OR-ed into (the caller zeroes it)."""
    B, Hq, d = q.shape
    num_pages, _, Hkv, _ = k_cache.shape
    _check("pkv_plan_decode_noalloc", lib().pkv_plan_decode_noalloc(
        _dev(q, torch.float16, "q"), _dev(k_cache, torch.float16, "k_cache"),
        _dev(v_cache, torch.float16, "v_cache"), num_pages, _dev(block_table, torch.int32, "block_table"),
        block_table.shape[1], _dev(seq_lens, torch.int32, "seq_lens"), B, Hq, Hkv, d, ctypes.byref(params),
        _dev(tasks, torch.int32, "tasks"), tasks.numel() // TASK_FIELDS,
        _dev(split_offsets, torch.int32, "split_offsets"), _dev(num_tasks, torch.int32, "num_tasks"),
        float(sm_scale), _dev(out, torch.float16, "out"), _dev(error_bits, torch.int32, "error_bits"),
        _stream(stream)))


def _host_i32(x) -> tuple:
    import numpy as np
    arr = np.ascontiguousarray(np.asarray(x, dtype=np.int32))
    return arr, arr.ctypes.data_as(ctypes.c_void_p)


def pkv_decode_rect(q: torch.Tensor, k_cache: torch.Tensor, v_cache: torch.Tensor, block_table: torch.Tensor,
                    seq_lens: torch.Tensor, S: int, tile_tokens: int, sm_scale: float, out: torch.Tensor,
                    ws: torch.Tensor, *, row_ids=None, stream=None):
    """row_ids: optional host sequence of at most 64 rows (indexed Q/O)."""
    B, Hq, d = q.shape
    num_pages, _, Hkv, _ = k_cache.shape
    ids, ids_ptr, n = None, None, 0
    if row_ids is not None:
        ids, ids_ptr = _host_i32(row_ids)
        n = ids.size
    _check("pkv_decode_rect", lib().pkv_decode_rect(
        _dev(q, torch.float16, "q"), _dev(k_cache, torch.float16, "k_cache"),
        _dev(v_cache, torch.float16, "v_cache"), num_pages, _dev(block_table, torch.int32, "block_table"),
        block_table.shape[1], _dev(seq_lens, torch.int32, "seq_lens"), B, Hq, Hkv, d, ids_ptr, n, S, tile_tokens,
        float(sm_scale), _dev(out, torch.float16, "out"), _dev(ws, torch.uint8, "ws"), ws.numel(),
        _stream(stream)))


def pkv_decode_buckets(q: torch.Tensor, k_cache: torch.Tensor, v_cache: torch.Tensor, block_table: torch.Tensor,
                       seq_lens: torch.Tensor, host_seq_lens, bucket_tokens: int, params: PlanParams,
                       sm_scale: float, out: torch.Tensor, ws: torch.Tensor, *, stream=None) -> int:
    """Length-bucket route; returns the number of kernel launches issued."""
    B, Hq, d = q.shape
    num_pages, _, Hkv, _ = k_cache.shape
    lens, lens_ptr = _host_i32(host_seq_lens)
    launches = ctypes.c_int32(0)
    _check("pkv_decode_buckets", lib().pkv_decode_buckets(
        _dev(q, torch.float16, "q"), _dev(k_cache, torch.float16, "k_cache"),
        _dev(v_cache, torch.float16, "v_cache"), num_pages, _dev(block_table, torch.int32, "block_table"),
        block_table.shape[1], _dev(seq_lens, torch.int32, "seq_lens"), lens_ptr, B, Hq, Hkv, d,
        int(bucket_tokens), ctypes.byref(params), float(sm_scale), _dev(out, torch.float16, "out"),
        _dev(ws, torch.uint8, "ws"), ws.numel(), _stream(stream), ctypes.byref(launches)))
    return int(launches.value)


def pkv_check_device_status(ws: torch.Tensor, stream=None) -> int:
    """Synchronizes; returns the device error bits (0 when clean) and clears them."""
    bits = ctypes.c_uint32(0)
    st = lib().pkv_check_device_status(_dev(ws, torch.uint8, "ws"), _stream(stream), ctypes.byref(bits))
    if st not in (PKV_OK, PKV_ERR_DEVICE):
        _check("pkv_check_device_status", st)
    return int(bits.value)


def pkv_stream_copy(src: torch.Tensor, dst: torch.Tensor, stream=None):
    if not (src.is_cuda and dst.is_cuda and src.is_contiguous() and dst.is_contiguous()):
        raise TypeError("pkv_stream_copy needs contiguous device tensors")
    n = min(src.numel() * src.element_size(), dst.numel() * dst.element_size())
    _check("pkv_stream_copy", lib().pkv_stream_copy(src.data_ptr(), dst.data_ptr(), n - n % 16, _stream(stream)))


def pkv_stream_read(src: torch.Tensor, sink: torch.Tensor, stream=None, events=None):
    """Streaming read of `src`; events: optional (start, stop) stamped with the kernel's
    execution interval (pkv_stream_read_timed)."""
    if not (src.is_cuda and src.is_contiguous()):
        raise TypeError("pkv_stream_read needs a contiguous device tensor")
    n = src.numel() * src.element_size()
    args = (src.data_ptr(), n - n % 16, _dev(sink, torch.int32, "sink"), _stream(stream))
    if events is None:
        _check("pkv_stream_read", lib().pkv_stream_read(*args))
    else:
        _check("pkv_stream_read_timed", lib().pkv_stream_read_timed(*args, *_events(events)))


def pkv_stream_read_nt_timed(src: torch.Tensor, sink: torch.Tensor, stream=None, events=None):
    """Streaming read of `src` with non-temporal loads (the decode's K/V load policy);
    events: optional (start, stop) stamped with the kernel's execution interval."""
    if not (src.is_cuda and src.is_contiguous()):
        raise TypeError("pkv_stream_read_nt_timed needs a contiguous device tensor")
    n = src.numel() * src.element_size()
    args = (src.data_ptr(), n - n % 16, _dev(sink, torch.int32, "sink"), _stream(stream))
    ev = _events(events) if events is not None else (None, None)
    _check("pkv_stream_read_nt_timed", lib().pkv_stream_read_nt_timed(*args, *ev))


def pkv_stream_read_pages(k_cache: torch.Tensor, v_cache: torch.Tensor, block_table: torch.Tensor,
                          tasks: torch.Tensor, num_tasks: torch.Tensor, heads_per_workgroup: int,
                          sink: torch.Tensor, stream=None, events=None):
    """Read-only probe of the decode kernel's page pattern over a plan's task list
    (k_cache, v_cache [num_pages, 16, Hkv, d] fp16; tasks [max_tasks, 5] int32);
    events: optional (start, stop) stamped with the kernel's execution interval."""
    num_pages, _, hkv, d = k_cache.shape
    B, maxp = block_table.shape
    ev = _events(events) or (None, None)
    _check("pkv_stream_read_pages", lib().pkv_stream_read_pages(
        _dev(k_cache, torch.float16, "k_cache"), _dev(v_cache, torch.float16, "v_cache"), num_pages,
        _dev(block_table, torch.int32, "block_table"), maxp, B, hkv, d, _dev(tasks, torch.int32, "tasks"),
        _dev(num_tasks, torch.int32, "num_tasks"), tasks.shape[0], heads_per_workgroup,
        _dev(sink, torch.int32, "sink"), _stream(stream), *ev))


class DecodeBuffers:
    """Device buffers one decode stream needs: task list, split offsets, task count and
    workspace, sized for batches of up to B rows and split counts up to split_max (and
    rectangular grids up to rect_splits columns)."""

    def __init__(self, B: int, Hq: int, Hkv: int, d: int, split_max: int, device, rect_splits: int = 0):
        self.B, self.Hq, self.Hkv, self.d = B, Hq, Hkv, d
        self.max_tasks = pkv_max_tasks(B, Hkv, max(split_max, rect_splits))
        if self.max_tasks < 1:
            raise ValueError("bad sizes")
        self.tasks = torch.zeros((self.max_tasks, TASK_FIELDS), dtype=torch.int32, device=device)
        self.split_offsets = torch.zeros(B + 1, dtype=torch.int32, device=device)
        self.num_tasks = torch.zeros(1, dtype=torch.int32, device=device)
        self.ws_bytes = pkv_workspace_size(B, Hq, Hkv, d, self.max_tasks)
        self.ws = torch.zeros(self.ws_bytes, dtype=torch.uint8, device=device)
        pkv_workspace_init(self.ws, B, Hkv)

    def partial_region(self) -> torch.Tensor:
        """The partial-state slots as a byte view (tests fill it with NaN)."""
        off = 256 + ((self.B * self.Hkv * 4 + 255) // 256) * 256
        return self.ws[off:]
