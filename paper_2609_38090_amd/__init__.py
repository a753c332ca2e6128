"""MI355X-native Mira MoE expert step: Python binding of libmira.so.

The functions here carry the names of the C ABI (include/mira.h) and only
marshal arguments: every step runs in the HIP kernels of the library.  Tensor
arguments are torch tensors (or raw integer addresses); streams are torch
streams, raw hipStream_t integers, or None for the current stream.

Importing the package loads nothing; call load() (or any mira_* function).
If libmira.so has not been built, load() raises: there is no fallback.
"""
from ._binding import (  # noqa: F401
    MIRA_BF16,
    MIRA_DECODE_MAX_TOKENS,
    MIRA_F32,
    MIRA_FLAG_FORCE_DECODE,
    MIRA_FLAG_FORCE_PREFILL,
    MIRA_FLAG_INT4,
    MIRA_FLAG_SOFTMAX_ALL,
    MIRA_MAX_EXPERTS,
    MIRA_MAX_TOPK,
    MIRA_NOALLOC_SCRATCH_BYTES,
    MiraError,
    MixtureShape,
    MixtureWeights,
    MoEArgs,
    MoEShape,
    PredShape,
    lib_path,
    load,
    mira_last_error,
    mira_moe_experts,
    mira_moe_forward,
    mira_moe_forward_noalloc,
    mira_moe_route,
    mira_pack_experts,
    mira_packed_expert_bytes,
    mira_packed_expert_bytes_int4,
    mira_mixture_workspace_bytes,
    mira_predict,
    mira_predict_mixture,
    mira_predict_workspace_bytes,
    mira_profile_enable,
    mira_profile_read,
    mira_profile_select,
    mira_set_slot,
    mira_stage_expert,
    mira_version,
    mira_workspace_bytes,
)

EXPORTED_SYMBOLS = (
    "mira_packed_expert_bytes",
    "mira_packed_expert_bytes_int4",
    "mira_workspace_bytes",
    "mira_pack_experts",
    "mira_moe_forward",
    "mira_moe_forward_noalloc",
    "mira_moe_route",
    "mira_moe_experts",
    "mira_predict_workspace_bytes",
    "mira_predict",
    "mira_mixture_workspace_bytes",
    "mira_predict_mixture",
    "mira_stage_expert",
    "mira_set_slot",
    "mira_last_error",
    "mira_version",
    "mira_profile_enable",
    "mira_profile_read",
    "mira_profile_select",
)
