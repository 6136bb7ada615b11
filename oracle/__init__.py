"""fp64 CPU oracle for the LoGo attention layer forward (test infrastructure).

Only the tests, ``__graft_entry__.smoke()`` and the benchmark's CPU-baseline
leg use this package.  The HIP library never loads it and shares no code
with it.  The arithmetic lives in ``logo_oracle.c`` (plain C, fp64, OpenMP);
this module only builds that file with gcc and marshals numpy arrays.
"""
from .oracle import (  # noqa: F401
    LP,
    SEL_RATIO,
    SO,
    SEL_THRESHOLD,
    attn_bwd,
    attn_rows,
    branch_transform,
    budget_update,
    build,
    contextnorm,
    decode,
    fuse,
    fusion_bwd,
    gate_proj,
    library_path,
    logo_bwd,
    logo_bwd_sample,
    logo_fwd,
    logo_rows,
    num_threads,
    pmask_initial_threshold,
    realized_ratio,
    select,
    set_num_threads,
    thresholds,
)
