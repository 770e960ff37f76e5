"""Shared test helpers: run the HIP path on a workload, compare with the oracle."""
from __future__ import annotations

import math
import sys

import numpy as np
import torch

import oracle


def log(msg: str) -> None:
    """Name the case before a GPU step (flushed, so a crash still shows it)."""
    print(msg, file=sys.stderr, flush=True)


def rel_fro(a, b) -> float:
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    nb = np.linalg.norm(b)
    if nb == 0.0:
        return float(np.linalg.norm(a))
    return float(np.linalg.norm(a - b) / nb)


def to_dev(w, dev="cuda"):
    """Device copies of a workload's micro-batch inputs (H, W may already be there)."""
    return dict(
        H=w.H.to(dev), W=w.W.to(dev),
        token_id=torch.from_numpy(np.ascontiguousarray(w.token_id)).to(dev),
        mask=torch.from_numpy(np.ascontiguousarray(w.mask)).to(dev),
        old_logp=torch.from_numpy(np.ascontiguousarray(w.old_logp)).to(dev),
    )


def adv_inputs(w, dev="cuda", groups=True):
    return dict(
        traj_id=torch.from_numpy(w.g_traj_id).to(dev),
        mask=torch.from_numpy(w.g_mask).to(dev),
        traj_task=torch.from_numpy(w.traj_task).to(dev),
        traj_group=torch.from_numpy(w.traj_group).to(dev) if groups else None,
        reward=torch.from_numpy(w.reward).to(dev),
    )


def near_clip(logp, old, adv, mask, eps_lo, eps_hi, tol=1e-4):
    """Action tokens whose (oracle) ratio sits within tol of an active clip bound."""
    rho = np.exp(np.asarray(logp, np.float64) - np.asarray(old, np.float64))
    m = np.asarray(mask).astype(bool)
    a = np.asarray(adv)
    hi = (a > 0) & (np.abs(rho - (1 + eps_hi)) <= tol * (1 + eps_hi))
    lo = (a < 0) & (np.abs(rho - (1 - eps_lo)) <= tol)
    return m & (hi | lo)


# lse / logp, absolute: about 5x the largest error measured over every parity case
# (full-size workloads included: 1.8e-6 for lse, 8.5e-6 for logp at d = 5120),
# which follows from fp32 accumulation of bf16 products over d terms (~sqrt(d)
# roundings of 2^-24 relative on logits of magnitude ~1)
LSE_ATOL = 2e-5
LOGP_ATOL = 5e-5


def compare_loss(gpu, ref, w_mask, adv, old, eps_lo, eps_hi, *, loss_rel=1e-3, lp_atol=LOGP_ATOL,
                 lse_atol=LSE_ATOL, grad_rel=2e-2, check_grads=True):
    """Element-by-element comparison of one fwd(+bwd) against the oracle's whole batch."""
    m = np.asarray(w_mask).astype(bool)
    logp = gpu["logp"]
    lse = gpu["lse"]
    # masked positions are exactly 0
    assert np.all(logp[~m] == 0) and np.all(lse[~m] == 0)
    L, R = gpu["loss"], ref["loss"]
    if m.any():
        e_lse = float(np.abs(lse[m] - ref["lse"][m]).max())
        e_lp = float(np.abs(logp[m] - ref["logp"][m]).max())
        log(f"  max |d lse| {e_lse:.3e} (atol {lse_atol:.0e})  max |d logp| {e_lp:.3e} "
            f"(atol {lp_atol:.0e}); loss rel err {abs(L - R) / max(abs(R), 1e-30):.3e}")
    np.testing.assert_allclose(lse[m], ref["lse"][m], rtol=0, atol=lse_atol)
    np.testing.assert_allclose(logp[m], ref["logp"][m], rtol=0, atol=lp_atol)
    assert abs(L - R) <= loss_rel * abs(R) + 1e-7, (L, R)
    flips = near_clip(ref["logp"], old, adv, m, eps_lo, eps_hi)
    assert np.abs(np.asarray(gpu["n_clip"]) - ref["n_clip"]).sum() <= flips.sum()
    if check_grads:
        dH, dW = gpu["dH"], gpu["dW"]
        assert np.all(dH[~m] == 0) and not np.signbit(dH[~m]).any()
        eh, ew = rel_fro(dH, ref["dH"]), rel_fro(dW, ref["dW"])
        assert eh <= grad_rel, ("dH", eh)
        assert ew <= grad_rel, ("dW", ew)
        return eh, ew
    return None


def run_gpu(pl, d_in, adv_tok_dev, backward=True):
    """One forward (+backward) through the C ABI; results copied to the host."""
    loss, logp, lse, n_clip = pl.forward(d_in["H"], d_in["W"], d_in["token_id"], d_in["mask"],
                                         adv_tok_dev, d_in["old_logp"])
    out = {}
    if backward:
        dH, dW = pl.backward(d_in["H"], d_in["W"], d_in["token_id"], d_in["mask"], adv_tok_dev,
                             d_in["old_logp"])
    torch.cuda.synchronize()
    out["loss"] = float(loss.item())
    out["logp"] = logp.cpu().numpy().astype(np.float64)
    out["lse"] = lse.cpu().numpy().astype(np.float64)
    out["n_clip"] = n_clip.cpu().numpy()
    if backward:
        out["dH"] = dH.cpu().numpy()
        out["dW"] = dW.cpu().numpy()
    return out
