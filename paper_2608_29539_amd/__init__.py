"""MI355X-native forward pass of one LoGo attention layer.

A thin ctypes binding over ``liblogo.so`` (HIP kernels for gfx950, C ABI in
``include/logo.h``).  Every function here only checks tensors and marshals
pointers and the current torch stream into the C call of the same name; all
computation happens in the HIP kernels.  Importing the package does not load
the library; the first call does, and raises if it is missing (build it with
``paper_2608_29539_amd.build.build_library()``).
"""
from .binding import (  # noqa: F401
    LOGO_ENTRY_BWD,
    LOGO_ENTRY_COMBINE,
    LOGO_ENTRY_DECODE,
    LOGO_ENTRY_DENSE,
    LOGO_ENTRY_DENSE_BWD,
    LOGO_ENTRY_FWD,
    LOGO_ENTRY_FWD_QPHI,
    LOGO_ENTRY_FWD_TRAIN,
    LOGO_ENTRY_GLOBAL,
    LOGO_ENTRY_GLOBAL_BWD,
    LOGO_ENTRY_LOCAL,
    LOGO_ENTRY_SELECT,
    LOGO_PHI_LP,
    LOGO_PHI_SO,
    LOGO_SEL_RATIO,
    LOGO_SEL_THRESHOLD,
    LOGO_SEL_THRESHOLD_DEVICE,
    LogoError,
    Problem,
    exported_symbols,
    library,
    library_path,
    logo_attn_bwd,
    logo_attn_fwd,
    logo_attn_fwd_qphi,
    logo_attn_fwd_train,
    logo_branch_transform,
    logo_budget_update,
    logo_combine,
    logo_decode,
    logo_decode_noalloc,
    logo_dense_causal_attn,
    logo_dense_causal_attn_bwd,
    logo_dense_causal_attn_fwd_train,
    logo_gate_proj,
    logo_global_attn_sparse_q,
    logo_global_attn_sparse_q_bwd,
    logo_global_attn_sparse_q_fwd_train,
    logo_local_attn,
    logo_pmask_initial_threshold,
    logo_attn_fwd_launches,
    logo_ratio_capacity,
    logo_select,
    logo_status_str,
    logo_version,
    logo_workspace_bytes,
)
