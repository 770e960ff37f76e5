"""MI355X-native fused policy loss for agentic RL (AgentRL, arXiv 2510.04206).

The computation lives in libagrl.so (HIP kernels for gfx950, C ABI in
include/agrl.h).  This package only marshals torch device tensors into that
ABI (``_binding``) and offers a small convenience layer (``api``) that
allocates outputs and the workspace with torch.
"""
from ._binding import (AGRL_BF16, AGRL_F32, AgrlError, agrl_get_device_error,
                       agrl_options, agrl_policy_loss_bwd, agrl_policy_loss_fwd,
                       agrl_policy_loss_vocab_chunk, agrl_policy_loss_workspace_size,
                       agrl_sequence_mean_weights, agrl_task_adv_norm, agrl_token_logprob,
                       agrl_token_logprob_workspace_size, lib)
from .api import PolicyLoss, TokenLogprob, sequence_mean_weights, task_adv_norm

__all__ = ["AGRL_BF16", "AGRL_F32", "AgrlError", "agrl_options", "agrl_task_adv_norm",
           "agrl_policy_loss_workspace_size", "agrl_policy_loss_vocab_chunk",
           "agrl_policy_loss_fwd", "agrl_policy_loss_bwd",
           "agrl_token_logprob", "agrl_token_logprob_workspace_size",
           "agrl_sequence_mean_weights", "agrl_get_device_error", "lib", "PolicyLoss",
           "TokenLogprob", "sequence_mean_weights", "task_adv_norm"]
