"""Learner-time on-policy-distillation loss for AMD Instinct MI355X (gfx950).

The computation lives in ``libopd.so`` (hand-written HIP kernels behind the C
ABI of ``include/opd.h``); this package is its thin Python binding.  PyTorch
provides device memory and streams only.
"""
from ._binding import (DENSE, DIAG_OUTPUTS, ESTIMATORS, EXPORTS, FLAG_FORCE_ROWWISE,
                       FLAG_FORCE_SPLITV, FLAG_SKIP_MASKED, K_MAX, LIB_PATH, TOPK, OpdCache,
                       OpdError, OpdMcDiag, OpdOpts, PreparedCall, lib, loss_fwd_bwd,
                       mc_diagnostics, prepare_loss_fwd_bwd, sample_actions, score_actions,
                       status_string, topk_support, validate_cache, version, workspace_bytes)

__all__ = ["DENSE", "DIAG_OUTPUTS", "ESTIMATORS", "EXPORTS", "FLAG_FORCE_ROWWISE",
           "FLAG_FORCE_SPLITV", "FLAG_SKIP_MASKED", "K_MAX", "LIB_PATH", "TOPK", "OpdCache",
           "OpdError", "OpdMcDiag", "OpdOpts", "PreparedCall", "lib", "loss_fwd_bwd",
           "mc_diagnostics", "prepare_loss_fwd_bwd", "sample_actions", "score_actions",
           "status_string", "topk_support", "validate_cache", "version", "workspace_bytes"]
