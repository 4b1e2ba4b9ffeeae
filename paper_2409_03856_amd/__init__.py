"""Sirius hot path on MI355X (gfx950): contextual-sparse SwiGLU FFN decode and the
full model's correction check, as hand-written HIP kernels behind a C ABI
(include/sirius.h, libsirius.so). This package is the thin Python binding.

Importing the package does not load the library; the first call does, and it
raises if libsirius.so has not been built (there is no CPU fallback).
"""

from ._lib import (  # noqa: F401
    SiriusError,
    lib,
    workspace,
    sirius_ffn_dense,
    sirius_ffn_cats,
    sirius_ffn_cats_noalloc,
    sirius_ffn_topk,
    sirius_cats_calibrate,
    sirius_griffin_select,
    sirius_ffn_condensed,
    sirius_verify_accept,
    sirius_tree_build_step,
    sirius_tree_verify,
    sirius_attn_kv,
    sirius_kv_rollback,
    sirius_rmsnorm,
    Model,
    sirius_model_workspace_size,
    sirius_model_forward,
    sirius_generate,
    sirius_fill_normal_bf16,
    sirius_workspace_size,
    sirius_profile_enable,
    sirius_profile_reset,
    sirius_profile_query,
    sirius_version,
    LIB_PATH,
    OP_FFN_DENSE,
    OP_FFN_CATS,
    OP_GRIFFIN_SELECT,
    OP_FFN_CONDENSED,
    OP_VERIFY,
    OP_CATS_CALIBRATE,
    OP_TREE_BUILD,
    OP_TREE_VERIFY,
    OP_FFN_TOPK,
    OP_ATTN_KV,
)
