"""INT4 HQ-MM / LSS-MM linear operator for AMD MI355X (gfx950).

Python side of libhqlss: a thin ctypes binding with the same names as the C ABI in
include/hqlss.h.  It only marshals arguments (torch tensors -> device pointers, the
current HIP stream); every step of the operator runs in the library's HIP kernels.
Importing this package fails loudly when the library has not been built.
"""
from ._binding import (  # noqa: F401
    BUDGET_KEEP_NONZERO,
    DTYPE_CODES,
    HQLSSError,
    LSQ,
    Plan,
    Saved,
    debug_copy,
    debug_gemm_acc,
    debug_set_gemm_splits,
    hq_choose_hadamard_size,
    hq_linear_fwd,
    hq_linear_fwd_lsq,
    kernel_name,
    lib,
    lss_grad_plan,
    lss_linear_bwd,
    lss_linear_bwd_dw,
    lss_linear_bwd_dx,
    lss_linear_bwd_from_plan,
    lss_linear_bwd_lsq,
    lss_philox_offset_advance,
    status_string,
    timing_enable,
    timing_read,
    workspace,
    workspace_bytes,
    WS_FWD,
    WS_BWD_DX,
    WS_BWD_DW,
    WS_BWD,
    WS_FROM_PLAN,
    WS_PLAN,
    WS_HSIZE,
    WS_FWD_LSQ,
    WS_BWD_LSQ,
)
