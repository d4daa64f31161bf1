"""CPU float64 oracle for the Hydra-PPO hot path (test infrastructure only; see hydra_oracle)."""
from .hydra_oracle import (  # noqa: F401
    bf16_to_f64,
    lora_linear_ref,
    lora_linear_backward_ref,
    lora_linear_multi_ref,
    log_softmax_gather_ref,
    score_logits_ref,
    reward_ref,
    score_head_ref,
    score_head_two_input_ref,
)
from .ppo_oracle import (  # noqa: F401
    gae_ref,
    ppo_loss_ref,
    ppo_rewards_ref,
    value_head_ref,
)
