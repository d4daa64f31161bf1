"""MI355X-native Hydra-PPO hot path: LoRA-switchable linear, PPO scoring epilogue and advantage step.

The compute runs in libhydra.so (hand-written HIP kernels for gfx950 behind the
C ABI of include/hydra.h); this package only marshals PyTorch tensors into it.
"""
from ._binding import (  # noqa: F401
    EXPORTED,
    HYDRA_ERR_ALIGN,
    HYDRA_ERR_HIP,
    HYDRA_ERR_NULL,
    HYDRA_ERR_SHAPE,
    HYDRA_ERR_UNSUPPORTED,
    HYDRA_ERR_WORKSPACE,
    HYDRA_MAX_ADAPTERS,
    HYDRA_MAX_GROUP,
    HYDRA_MAX_RANK,
    HYDRA_SCORE_NOALLOC_MAX_BYTES,
    HYDRA_OK,
    HydraError,
    HydraLibraryMissing,
    LIB_PATH,
    hydra_lora_linear,
    hydra_lora_linear_backward,
    hydra_lora_linear_backward_workspace_bytes,
    hydra_lora_linear_group,
    hydra_lora_linear_workspace_bytes,
    hydra_lora_linear_ws,
    hydra_lora_linear_multi,
    hydra_ppo_advantages,
    hydra_ppo_loss,
    hydra_score,
    hydra_score_noalloc,
    hydra_score_logits,
    hydra_score_workspace_bytes,
    hydra_transpose_bf16,
    hydra_value_head,
    lib,
    status_string,
)
