"""ACE token-adaptive MoE layer for AMD Instinct MI355X (gfx950).

The layer (RMSNorm, router, top-k, the ACE skip mask of Alg. 4, dispatch,
grouped SwiGLU expert GEMMs and the gate-weighted combine) runs in hand-written
HIP kernels in libace.so behind the C ABI of include/ace.h.  This package is the
thin Python binding: `moe_forward` takes torch device tensors and enqueues the
layer on the current HIP stream (`prepare_forward` checks and marshals the
arguments once, for loops that call the same layer again); `tau_map` turns the
contribution scores of a score pass into the thresholds of requested skip
ratios (App. C.1); and `build_tables` computes the offline GSP / RCR tables
(Alg. 2, Alg. 3).
"""
from ._lib import (  # noqa: F401
    ACE_BF16, ACE_ERR_HIP, ACE_ERR_INVALID_ARG, ACE_ERR_UNSUPPORTED, ACE_ERR_WORKSPACE, ACE_F32,
    ACE_OK, ACE_SKIP_DISABLE, ACE_WRITE_SCORES, PROFILE_STAGES, AceError, Desc, LIB_PATH, Outputs,
    TAU_MAX_Q, Weights, abi_version, forward_raw, lib, profile_begin, profile_end, status_string,
    build_tables_raw, tables_workspace_size, tau_map_raw, tau_workspace_size, workspace_size,
)
from .layer import (  # noqa: F401
    PreparedForward, build_tables, make_desc, moe_forward, prepare_forward, tau_map, workspace,
)
