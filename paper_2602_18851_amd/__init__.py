"""MI355X-native per-head spectral norms of attention interaction matrices
(implicit power iteration, implicit GQA) and the per-layer FP8 E4M3 scale
of arXiv 2602.18851, behind a C ABI (include/spectral.h)."""

from .spectral import (  # noqa: F401
    EXPORTED,
    LIB_PATH,
    SN_BF16,
    SN_F32,
    SN_FLAG_GRAM,
    SN_FLAG_LAYER,
    SN_FLAG_VALU_K_SWEEP,
    Spectral,
    SpectralError,
    load_library,
    sn_params,
    sn_shape,
    spectral_alpha_select,
    spectral_auto_alpha,
    spectral_destroy,
    spectral_overflow_terms,
    spectral_slack_ratio,
    spectral_init,
    spectral_last_error,
    spectral_logits_fp8,
    spectral_logits_workspace_bytes,
    spectral_profile,
    spectral_profile_read,
    spectral_set_stream,
    spectral_step,
    spectral_step_layer,
    spectral_workspace_bytes,
)
