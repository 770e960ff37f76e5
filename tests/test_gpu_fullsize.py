"""Parity at the full workload sizes, in the launch configuration bench.py times.

The oracle cannot afford the whole batch at these sizes (about 1e14 fp64
flops), so the checks are:
  * sampled action tokens: lse, logp and the dH row against the oracle's
    per-token computation (same inputs, fp64);
  * properties that hold at any size: masked rows of dH are +0; the loss and
    the clip counts follow from the emitted log-probs; dH^T H == W^T dW (the
    loss depends on H and W only through H W^T, so its gradients satisfy this
    identity for any G, here up to fp32 accumulation); sampled rows of dW
    equal G^T H recomputed in fp64 from the forward's own lse and logp.
"""
import numpy as np
import pytest
import torch

import oracle
from workloads import gen

from helpers import log, rel_fro

pytestmark = pytest.mark.gpu


def _run(k, n_sample=12, n_dw_rows=6):
    import paper_2510_04206_amd as P
    dev = torch.device("cuda")
    w = gen.config(k, device=dev)
    eps_lo, eps_hi = w.spec.eps_lo, w.spec.eps_hi
    log(f"full-size workload {k}: {w.spec.name} T={w.T} N_act={w.n_act} T_g={w.T_g}")
    a = oracle.task_adv_norm(w.g_traj_id, w.g_mask, w.traj_task, w.traj_group, w.reward,
                             w.n_task, w.n_group)
    adv = a["adv_tok"][: w.T].copy()
    t = lambda x: torch.from_numpy(np.ascontiguousarray(x)).to(dev)
    ids, mask, old, adv_d = t(w.token_id), t(w.mask), t(w.old_logp), t(adv)
    pl = P.PolicyLoss(w.T, w.d, w.V, w.H.dtype, max_act=w.n_act, eps_low=eps_lo,
                      eps_high=eps_hi, device=dev)
    loss, logp, lse, n_clip = pl.forward(w.H, w.W, ids, mask, adv_d, old)
    dH, dW = pl.backward(w.H, w.W, ids, mask, adv_d, old)
    torch.cuda.synchronize()
    assert P.agrl_get_device_error() == 0
    m = w.mask.astype(bool)
    act = np.nonzero(m)[0]
    logp_h = logp.cpu().numpy().astype(np.float64)
    lse_h = lse.cpu().numpy().astype(np.float64)
    assert np.all(logp_h[~m] == 0) and np.all(lse_h[~m] == 0)

    # --- sampled tokens against the oracle
    rng = np.random.default_rng(1000 + k)
    toks = np.unique(np.concatenate([rng.choice(act, n_sample - 2, replace=False),
                                     [act[0], act[-1]]]))
    log(f"  oracle on {len(toks)} sampled tokens")
    r = oracle.token_sample(w.H, w.W, w.token_id, w.mask, adv, w.old_logp, toks,
                            eps_lo=eps_lo, eps_hi=eps_hi)
    np.testing.assert_allclose(lse_h[toks], r["lse"], rtol=1e-5, atol=2e-3)
    np.testing.assert_allclose(logp_h[toks], r["logp"], rtol=1e-5, atol=2e-3)
    rho = np.exp(r["logp"] - w.old_logp[toks].astype(np.float64))
    # rows whose clip decision sits within 1e-4 of a bound may legitimately differ
    near = ((adv[toks] > 0) & (np.abs(rho - (1 + eps_hi)) < 1e-4)) | \
           ((adv[toks] < 0) & (np.abs(rho - (1 - eps_lo)) < 1e-4))
    keep = ~near
    dH_s = dH[torch.from_numpy(toks).to(dev)].cpu().numpy()
    e = rel_fro(dH_s[keep], r["dH"][keep])
    log(f"  sampled dH rows rel fro {e:.2e}")
    assert e <= 2e-2

    # --- properties at full size
    off = torch.from_numpy(~m).to(dev)
    dH_off = dH[off]
    assert bool((dH_off == 0).all()) and not bool(torch.signbit(dH_off).any())
    A = adv[m].astype(np.float64)
    rho_all = np.exp(logp_h[m] - w.old_logp[m].astype(np.float64))
    s = np.minimum(rho_all * A, np.clip(rho_all, 1 - eps_lo, 1 + eps_hi) * A)
    L_ref = -s.sum() / m.sum()
    L = float(loss.item())
    assert abs(L - L_ref) <= 1e-4 * abs(L_ref) + 1e-7, (L, L_ref)
    hi = (A > 0) & (rho_all > 1 + eps_hi)
    lo = (A < 0) & (rho_all < 1 - eps_lo)
    border = ((A > 0) & (np.abs(rho_all - (1 + eps_hi)) < 1e-6)) | \
             ((A < 0) & (np.abs(rho_all - (1 - eps_lo)) < 1e-6))
    nc = n_clip.cpu().numpy()
    assert abs(int(nc[0]) - int(hi.sum())) + abs(int(nc[1]) - int(lo.sum())) <= int(border.sum())

    Hf, Wf = w.H.float(), w.W.float()
    lhs = dH.t() @ Hf
    rhs = Wf.t() @ dW
    ident = float(torch.linalg.norm(lhs - rhs) / torch.linalg.norm(rhs))
    log(f"  identity dH^T H vs W^T dW rel fro {ident:.2e}")
    assert ident <= 1e-3

    # sampled rows of dW from the forward's own lse / logp (fp64, test side)
    rows = np.unique(np.concatenate([rng.choice(w.V, n_dw_rows - 2, replace=False),
                                     w.token_id[act[:2]]]))
    idx = torch.from_numpy(act).to(dev)
    Ha = Hf[idx].double()
    lse_a = lse[idx].double()
    old_a = old[idx].double()
    A_a = adv_d[idx].double()
    rho_a = torch.exp(logp[idx].double() - old_a)
    cut = ((A_a > 0) & (rho_a > 1 + eps_hi)) | ((A_a < 0) & (rho_a < 1 - eps_lo))
    g = torch.where(cut, torch.zeros_like(rho_a), -A_a * rho_a / float(m.sum()))
    y_a = ids[idx].long()
    for v in rows.tolist():
        z = Ha @ Wf[v].double()
        Gv = g * ((y_a == v).double() - torch.exp(z - lse_a))
        ref_row = (Gv[:, None] * Ha).sum(0)
        ev = float(torch.linalg.norm(dW[v].double() - ref_row) / torch.linalg.norm(ref_row))
        assert ev <= 2e-2, (v, ev)
    log(f"  loss {L:.6g}; {len(rows)} dW rows consistent")


@pytest.mark.parametrize("k", [2, 3, 4, 5])
def test_full_size_workload(k):
    _run(k)
