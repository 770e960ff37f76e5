"""Full-vocabulary fp64 forward with a library matmul -- test infrastructure.

Part of the oracle: only the tests, the smoke check and the benchmark's CPU
baseline may use it.  It shares no code with the HIP library and never
imports it.

It computes the same definition as the forward of ``agrl_oracle.c``, the
token log-probability of App. B.1: for every action token n,
    z_n = (h_n W^T) / temperature            (all V logits, fp64)
    lse_n = M + log sum_v exp(z_{n,v} - M),  M = max_v z_{n,v}
    logp_n = z_{n, y_n} - lse_n
from the exact fp64 upcast of the bf16 / fp32 inputs.  The only difference
from the C loops is that z comes from a library fp64 matmul (torch on the
CPU), which makes the whole batch affordable at the full workload sizes.
Tokens are taken a block of rows at a time; each row's logits are formed
whole before its reduction.
"""
from __future__ import annotations

import numpy as np


def _as_f64(x):
    """fp64 CPU torch tensor of a torch tensor (any device) or a numpy array
    (uint16 = bf16 bits, else floating point).  The upcast is exact."""
    import torch
    if isinstance(x, torch.Tensor):
        return x.detach().to("cpu").to(torch.float64)
    a = np.ascontiguousarray(x)
    if a.dtype == np.uint16:
        a = (a.astype(np.uint32) << 16).view(np.float32)
    return torch.from_numpy(np.asarray(a, np.float64))


def token_logprob_fp64(H, W, token_id, mask, temperature=1.0, rows_per_block=256):
    """(logp, lse): fp64 arrays [T], the values above on action tokens, 0 elsewhere."""
    import torch
    m = np.asarray(mask).astype(bool)
    T = m.shape[0]
    y = np.asarray(token_id, np.int64)
    act = np.nonzero(m)[0]
    V = W.shape[0]
    if act.size and (y[act].min() < 0 or y[act].max() >= V):
        raise ValueError("token_logprob_fp64: token id out of range")
    Hd = _as_f64(H)
    Wt = _as_f64(W).t()
    inv_temp = 1.0 / float(temperature)
    logp = np.zeros(T)
    lse = np.zeros(T)
    for s in range(0, act.size, rows_per_block):
        rows = torch.from_numpy(act[s:s + rows_per_block])
        z = (Hd.index_select(0, rows) @ Wt) * inv_temp
        M = z.max(dim=1).values
        l = M + torch.log(torch.exp(z - M[:, None]).sum(dim=1))
        zy = z.gather(1, torch.from_numpy(y[act[s:s + rows_per_block]])[:, None])[:, 0]
        lse[act[s:s + rows_per_block]] = l.numpy()
        logp[act[s:s + rows_per_block]] = (zy - l).numpy()
        del z
    return logp, lse
