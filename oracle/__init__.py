"""Float64 CPU oracle for the FLARE++ mixer forward (test infrastructure only).

Only the tests, ``__graft_entry__.smoke()`` and the benchmark's CPU-baseline
leg use this package; the HIP product path never imports it.
"""

from .flarepp_oracle import (  # noqa: F401
    flare_forward,
    materialised_operator,
    merge_heads,
    mixer_forward,
    partial_encode,
    project,
    sdpa,
    split_merge,
)
