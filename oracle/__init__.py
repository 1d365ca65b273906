"""fp64 CPU oracle for paged grouped-query decode attention and its workqueue planner.

TEST INFRASTRUCTURE. Only the tests, the smoke check and the benchmark's CPU-baseline
leg may import or run anything in this package. The HIP path never calls it, and it
shares no code, tables or constants with the HIP path: it is written from the paper's
definitions (Eq. 1 and Sec. 3.1-3.4) with numpy only.

  ref_decode        exact attention, Eq. (1), over a native block table (Sec. 3.2)
  ref_decode_split  split partial states and their merge (Sec. 3.3)
  ref_decode_rect   the rectangular (B, Hkv, S) split grid with neutral states (Sec. 3.3-3.4)
  ref_plan          the compact workqueue task list and split_offsets (Sec. 3.4)
"""
from .attention import (  # noqa: F401
    gather_row,
    ref_decode,
    ref_decode_rect,
    ref_decode_split,
    ref_merge,
    ref_split_state,
)
from .plan import (  # noqa: F401
    PlanParams,
    choose_split_count,
    ref_plan,
    row_split_bounds,
    row_split_counts,
    tile_quota,
)
