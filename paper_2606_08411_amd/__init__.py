"""AsyncLane decode-step hot path on MI355X (gfx950).

Three calls, backed by hand-written HIP kernels in libasynclane.so:

* ``lane_attn_forward``  shared-prefix lane-batched bidirectional attention
  over a lane tree, with compact-refresh prefix rows (paper Sections 3.2, 3.4)
* ``lmhead_confidence``  fused LM-head GEMM + online softmax: per masked
  position the max probability and its token, logits never stored
  (``lmhead_confidence_noalloc``: the same without a workspace, for callers
  that cannot allocate; ``lmhead_pack_weight`` + ``lmhead_confidence_packed``:
  the same from a one-time repacked copy of W that streams like a linear
  read)
* ``select_unmask``      per-lane threshold / top-k transfer, lookahead
  drafts, write-back and lane boundary statistics (eq. split_point,
  eq. fork_condition, ValidBoundary)
* ``al_refresh_window``  the compact cache refresh window length (Section
  3.4); the refresh forward itself is a refresh-only ``lane_attn_forward``
* ``AlSched``            the host active-lane scheduler (Section 3.3) that
  drives the three calls: plan, blocks, commit, collect

The functions are thin ctypes wrappers (see ``_lib``); they raise when the
library has not been built (``python -m paper_2606_08411_amd.build``).
"""
from ._lib import (  # noqa: F401
    AlSched,
    AsyncLaneError,
    al_refresh_window,
    LANE_STATS,
    MODE_THRESHOLD,
    MODE_TOPK,
    ROLE_GEN,
    ROLE_REF,
    lane_attn_forward,
    lane_attn_workspace_size,
    library,
    lmhead_confidence,
    lmhead_confidence_noalloc,
    lmhead_confidence_packed,
    lmhead_pack_weight,
    lmhead_packed_weight_size,
    lmhead_confidence_workspace_size,
    select_unmask,
)
