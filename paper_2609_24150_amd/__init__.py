"""Acceptance-aware draft-training losses (EAL, WTV) and the simulated
acceptance-length GRPO reward on AMD Instinct MI355X (gfx950).

The computation runs in hand-written HIP kernels inside libaal.so (C ABI in
include/aal.h); this package only marshals torch tensors to it.
"""
from .api import (  # noqa: F401
    AAL_BF16,
    AAL_F32,
    AAL_FLAG_COOPERATIVE,
    AAL_FLAG_STREAMING,
    AAL_LAYOUT_SEQUENCES,
    AAL_LAYOUT_WINDOWS,
    AAL_VP_EAL,
    AAL_VP_WTV,
    aal_eal_fwd_bwd,
    aal_grpo_fwd_bwd,
    aal_grpo_workspace_bytes,
    aal_loss_fwd_bwd,
    aal_loss_workspace_bytes,
    aal_sim_accept_grpo,
    aal_stream_probe,
    aal_vp_accept_partials,
    aal_vp_grad,
    aal_vp_merge_rows,
    aal_vp_row_partials,
    aal_vp_sequence_scan,
    aal_vp_window_scan,
    aal_workspace_bytes,
    aal_wtv_fwd_bwd,
    workspace,
)
from ._lib import AalError, LIB_PATH  # noqa: F401
