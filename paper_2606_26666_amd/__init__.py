"""pkv: paged grouped-query decode attention for MI355X (gfx950).

The decode path (planner, split attention, merge) lives in libpkv.so (HIP kernels
behind the C ABI of include/pkv.h); this package is its Python binding.
"""
from ._binding import (  # noqa: F401
    PKV_DEVERR_PAGE_ID,
    PKV_DEVERR_SEQ_LEN,
    PKV_DEVERR_TASK,
    PKV_ERR_DEVICE,
    PKV_ERR_HIP,
    PKV_ERR_INVALID_ARG,
    PKV_ERR_UNSUPPORTED,
    PKV_ERR_WORKSPACE,
    PKV_FUSED_MERGE,
    PKV_OK,
    PKV_SPLIT_BATCH,
    PKV_SPLIT_QUOTA,
    DecodeBuffers,
    PkvError,
    PlanParams,
    header_functions,
    lib,
    make_params,
    pkv_check_device_status,
    pkv_decode,
    pkv_decode_buckets,
    pkv_decode_rect,
    pkv_max_tasks,
    pkv_plan,
    pkv_plan_host,
    pkv_plan_decode,
    pkv_plan_decode_noalloc,
    pkv_stream_copy,
    pkv_stream_read,
    pkv_stream_read_pages,
    pkv_workspace_init,
    pkv_workspace_size,
)
