"""Convenience layer over the C ABI: allocates outputs/workspace with torch, then calls it."""
from __future__ import annotations

from typing import Optional

import torch

from . import _binding as B


def task_adv_norm(traj_id: torch.Tensor, action_mask: torch.Tensor, traj_task: torch.Tensor,
                  traj_group: Optional[torch.Tensor], reward: torch.Tensor, n_task: int,
                  n_group: int = 0, opt=None, with_tokens: bool = True, stream=None,
                  member_ranges: bool = True) -> dict:
    """agrl_task_adv_norm on device tensors; returns the outputs as a dict.

    member_ranges: pass a scratch array as agrl_options.adv_ranges (unless the
    options already name one), so that each group's and task's wave scans only
    its members' index span; the results are bit-identical without it."""
    dev = traj_id.device
    T_g, n_traj = traj_id.numel(), traj_task.numel()
    if member_ranges:
        o = B.agrl_options(**opt) if isinstance(opt, dict) else (opt or B.agrl_options())
        if not o.adv_ranges:
            n_seg = (n_group if traj_group is not None else 0) + n_task
            scratch = torch.empty(max(2 * n_seg, 1), dtype=torch.int32, device=dev)
            o.adv_ranges = scratch.data_ptr()
        opt = o
    out = dict(act_count=torch.empty(n_traj, dtype=torch.int32, device=dev),
               task_count=torch.empty(n_task, dtype=torch.int64, device=dev),
               task_mean=torch.empty(n_task, dtype=torch.float32, device=dev),
               task_std=torch.empty(n_task, dtype=torch.float32, device=dev),
               adv_traj=torch.empty(n_traj, dtype=torch.float32, device=dev),
               adv_tok=torch.empty(T_g, dtype=torch.float32, device=dev) if with_tokens else None)
    if member_ranges and "scratch" in locals():
        out["member_ranges"] = scratch     # kept alive with the outputs
    B.agrl_task_adv_norm(T_g, n_traj, n_task, n_group, traj_id, action_mask, traj_task,
                         traj_group, reward, opt, out["act_count"], out["task_count"],
                         out["task_mean"], out["task_std"], out["adv_traj"], out["adv_tok"],
                         stream)
    return out


def sequence_mean_weights(traj_id: torch.Tensor, action_mask: torch.Tensor, n_traj: int,
                          stream=None):
    """agrl_sequence_mean_weights: (seq_count [n_traj] int32, token_weight [T] fp32), the
    per-token weights of the sequence-level aggregation (pass token_weight's pointer as
    agrl_options.token_weight)."""
    dev = traj_id.device
    seq_count = torch.empty(n_traj, dtype=torch.int32, device=dev)
    token_weight = torch.empty(traj_id.numel(), dtype=torch.float32, device=dev)
    B.agrl_sequence_mean_weights(traj_id.numel(), n_traj, traj_id, action_mask, seq_count,
                                 token_weight, stream)
    return seq_count, token_weight


class PolicyLoss:
    """Forward/backward of the fused policy loss for one micro-batch shape.

    Holds the workspace (sized for T tokens with at most max_act action
    tokens) and the output buffers, so repeated steps allocate nothing.
    """

    def __init__(self, T: int, d: int, V: int, dtype: torch.dtype, max_act: int = 0,
                 eps_low: float = 0.2, eps_high: float = 0.2, n_norm: int = 0, opt=None,
                 device="cuda"):
        self.T, self.d, self.V, self.max_act = int(T), int(d), int(V), int(max_act)
        self.code = B.AGRL_BF16 if dtype == torch.bfloat16 else B.AGRL_F32
        self.eps_low, self.eps_high, self.n_norm = float(eps_low), float(eps_high), int(n_norm)
        self.opt = B.agrl_options(**opt) if isinstance(opt, dict) else opt
        self.ws_bytes = B.agrl_policy_loss_workspace_size(self.T, self.max_act, self.d, self.V,
                                                          self.code, self.opt)
        # vocabulary columns per backward chunk (the last chunk holds the rest)
        self.vocab_chunk = B.agrl_policy_loss_vocab_chunk(self.T, self.max_act, self.d, self.V,
                                                          self.code, self.opt)
        dev = torch.device(device)
        self.workspace = torch.empty(max(self.ws_bytes, 1), dtype=torch.uint8, device=dev)
        self.loss = torch.empty(1, dtype=torch.float32, device=dev)
        self.logp = torch.empty(self.T, dtype=torch.float32, device=dev)
        self.lse = torch.empty(self.T, dtype=torch.float32, device=dev)
        self.n_clip = torch.empty(2, dtype=torch.int64, device=dev)
        self.dH = torch.empty((self.T, self.d), dtype=torch.float32, device=dev)
        self.dW = torch.empty((self.V, self.d), dtype=torch.float32, device=dev)

    def forward(self, H, W, token_id, action_mask, adv_tok, old_logp, stream=None):
        B.agrl_policy_loss_fwd(self.T, self.max_act, self.d, self.V, self.code, H, W, token_id,
                               action_mask, adv_tok, old_logp, self.eps_low, self.eps_high,
                               self.n_norm, self.opt, self.workspace, self.ws_bytes, self.loss,
                               self.logp, self.lse, self.n_clip, stream)
        return self.loss, self.logp, self.lse, self.n_clip

    def backward(self, H, W, token_id, action_mask, adv_tok, old_logp, grad_loss: float = 1.0,
                 stream=None):
        B.agrl_policy_loss_bwd(self.T, self.max_act, self.d, self.V, self.code, H, W, token_id,
                               action_mask, adv_tok, old_logp, self.eps_low, self.eps_high,
                               self.n_norm, self.opt, self.lse, self.logp, float(grad_loss),
                               self.workspace, self.ws_bytes, self.dH, self.dW, stream)
        return self.dH, self.dW


class TokenLogprob:
    """Forward-only token log-probabilities for one packed-batch shape.

    Holds its workspace and outputs; ``__call__`` returns (logp, lse), fp32 [T],
    zero on observation tokens.
    """

    def __init__(self, T: int, d: int, V: int, dtype: torch.dtype, max_act: int = 0, opt=None,
                 device="cuda"):
        self.T, self.d, self.V, self.max_act = int(T), int(d), int(V), int(max_act)
        self.code = B.AGRL_BF16 if dtype == torch.bfloat16 else B.AGRL_F32
        self.opt = B.agrl_options(**opt) if isinstance(opt, dict) else opt
        self.ws_bytes = B.agrl_token_logprob_workspace_size(self.T, self.max_act, self.d, self.V,
                                                            self.code, self.opt)
        dev = torch.device(device)
        self.workspace = torch.empty(max(self.ws_bytes, 1), dtype=torch.uint8, device=dev)
        self.logp = torch.empty(self.T, dtype=torch.float32, device=dev)
        self.lse = torch.empty(self.T, dtype=torch.float32, device=dev)

    def __call__(self, H, W, token_id, action_mask, stream=None):
        B.agrl_token_logprob(self.T, self.max_act, self.d, self.V, self.code, H, W, token_id,
                             action_mask, self.opt, self.workspace, self.ws_bytes, self.logp,
                             self.lse, stream)
        return self.logp, self.lse
