"""libloglinear: log-linear attention (forward, backward and decoding) (Guo et al., "Log-Linear
Attention") on MI355X.

The computation lives in the HIP library libloglinear.so (C ABI: include/libloglinear.h);
this package is its Python binding.
"""

from ._lib import (  # noqa: F401
    LL_BF16, LL_F32, LL_GDN, LL_LAMBDA_DIAG, LL_LAMBDA_FULL, LL_MAMBA2, LL_MAMBA2_BWD, LLError, lib, ll_debug_level_map, ll_decode_state_bytes,
    ll_gdn_decode_init, ll_gdn_decode_step, ll_gdn_fwd, ll_gdn_fwd_staged, ll_mamba2_bwd, ll_mamba2_bwd_after_fwd,
    ll_mamba2_bwd_staged, ll_mamba2_bwd_workspace, ll_mamba2_decode_init, ll_mamba2_decode_step, ll_mamba2_fwd,
    ll_mamba2_fwd_grouped, ll_mamba2_fwd_matrix_lambda, ll_mamba2_fwd_noalloc, LL_NOALLOC_SCRATCH_BYTES, ll_mamba2_fwd_matrix_lambda_staged,
    ll_mamba2_fwd_staged, ll_mamba2_matrix_lambda_workspace, ll_num_levels, ll_status_string, ll_supported, ll_workspace_size,
    log_linear_mamba2,
)
