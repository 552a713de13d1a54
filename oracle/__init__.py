"""Plain, slow, fp64 CPU oracle for the AsyncLane decode-step hot path.

TEST INFRASTRUCTURE ONLY.  Nothing on the product path may import, call or
execute this package: only the tests, the smoke check and the benchmark's CPU
baseline leg use it.  It shares no code with the HIP library; its only input
is the seeded generator in ``synth``, which holds none of the method's
arithmetic.

Modules
-------
attention   lane-batched bidirectional attention over a shared prefix cache,
            in two independent forms, plus the compact-refresh row rewrite
            and refresh-row attention (paper Section 3.2 "Lane-local
            denoising", Section 3.4 "Shared-prefix lane batching" and
            "Compact cache refresh and reuse").
lmhead      hidden->vocab logits, max-probability confidence and argmax, in a
            full-softmax form and a chunked online form (Section 3.2, the
            confidence-based transfer rule; refine-lane EOS suppression).
refresh     the compact refresh window length (Section 3.4 "Compact cache
            refresh and reuse").
scheduler   the active-lane scheduler (Algorithm "AsyncLane active-lane
            decoding": fork, spawn, stop, output reconstruction, NFE).
select      per-lane confidence-threshold / top-k transfer and the lane
            boundary statistics: split point (eq. split_point), fill ratio
            and step condition (eq. fork_condition), valid prefix length
            (Section 3.2 "Advancement control").
"""
from . import attention, lmhead, refresh, scheduler, select  # noqa: F401
