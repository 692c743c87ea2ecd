"""fp64 CPU oracle for BDLM attention (test infrastructure only).

Only ``tests/``, ``__graft_entry__.smoke()`` and ``bench.py``'s
``cpu_baseline`` leg may import this package; the HIP library never does.
"""
from .bdlm_oracle import (  # noqa: F401
    CLEAN, CORRUPTED, CLEAN_INTRA_CAUSAL, CLEAN_INTRA_BLOCK,
    rows_of, joint_ranges, visible, attention_fwd_head, attention_bwd_head,
    fwd, bwd, lse_merge, joint_fwd, joint_bwd, count_visible_pairs,
)
