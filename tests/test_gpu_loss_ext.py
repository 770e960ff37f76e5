"""GPU parity of the KL penalty and per-token loss weights against the oracle.

The KL term (App. A objectives, -beta D_KL; k3 and k1 estimators) and the
per-token weights (sequence-level aggregation of App. B.2's GRPO form, a
token mean per trajectory then a mean over trajectories) change only the
per-token loss and dL/dlogp; the same tolerances as the plain loss apply:
loss 1e-3 relative, logp 2e-3 absolute, dH/dW 2e-2 relative Frobenius.
"""
import numpy as np
import pytest
import torch

import oracle
from workloads import gen

from helpers import compare_loss, log, run_gpu, to_dev

pytestmark = pytest.mark.gpu


def _adv(w):
    a = oracle.task_adv_norm(w.g_traj_id, w.g_mask, w.traj_task, w.traj_group, w.reward,
                             w.n_task, w.n_group)
    return a["adv_tok"][: w.T].copy()


def seq_mean_weights(w):
    """w_t = 1 / (n_seq * n_tau(t)) over the micro-batch's action tokens: each
    trajectory's token mean, then the mean over its trajectories."""
    tid = w.g_traj_id[: w.T]
    m = w.mask.astype(bool)
    trajs, counts = np.unique(tid[m], return_counts=True)
    n_tau = dict(zip(trajs.tolist(), counts.tolist()))
    out = np.zeros(w.T, np.float32)
    for t in np.nonzero(m)[0]:
        out[t] = 1.0 / (len(trajs) * n_tau[int(tid[t])])
    return out


def _run(w, *, kl_beta=0.0, kl_est=0, ref=None, weight=None, eps=(0.2, 0.2)):
    import paper_2510_04206_amd as P
    adv = _adv(w)
    d_in = to_dev(w)
    opt = {}
    keep = []
    if kl_beta:
        ref_d = torch.from_numpy(ref).cuda()
        keep.append(ref_d)
        opt.update(kl_beta=kl_beta, kl_estimator=kl_est, ref_logp=ref_d.data_ptr())
    if weight is not None:
        w_d = torch.from_numpy(weight).cuda()
        keep.append(w_d)
        opt.update(token_weight=w_d.data_ptr())
    log(f"loss-ext case {w.spec.name} T={w.T} n_act={w.n_act} kl_beta={kl_beta} est={kl_est} "
        f"weights={weight is not None}")
    pl = P.PolicyLoss(w.T, w.d, w.V, w.H.dtype, max_act=w.n_act, eps_low=eps[0], eps_high=eps[1],
                      opt=opt)
    g = run_gpu(pl, d_in, torch.from_numpy(adv).cuda())
    assert P.agrl_get_device_error() == 0
    r = oracle.policy_loss(w.H, w.W, w.token_id, w.mask, adv, w.old_logp, eps_lo=eps[0],
                           eps_hi=eps[1], kl_beta=kl_beta, kl_estimator=kl_est, ref_logp=ref,
                           token_weight=weight)
    errs = compare_loss(g, r, w.mask, adv, w.old_logp, eps[0], eps[1])
    log(f"  loss gpu {g['loss']:.7g} oracle {r['loss']:.7g}; dH/dW rel fro {errs}")
    return g, r


def _ref(w, scale=0.3, seed=1):
    rng = np.random.default_rng(seed)
    return (w.old_logp + scale * rng.standard_normal(w.T)).astype(np.float32)


@pytest.mark.parametrize("est", [0, 1])
def test_kl_penalty(est):
    w = gen.make(gen.small_spec(V=3000, d=256, dtype="bf16", noise_std=0.2, name="kl"), seed=17)
    _run(w, kl_beta=0.1, kl_est=est, ref=_ref(w))


def test_kl_penalty_fp32_workload1():
    w = gen.config(1)
    _run(w, kl_beta=0.05, kl_est=0, ref=_ref(w, 0.1))


def test_sequence_mean_weights():
    w = gen.make(gen.small_spec(V=2000, d=192, dtype="bf16", name="seqmean"), seed=19)
    _run(w, weight=seq_mean_weights(w))


def test_weights_and_kl_decoupled_clip():
    w = gen.make(gen.small_spec(V=1500, d=128, dtype="bf16", noise_std=0.3, name="both"), seed=23)
    _run(w, kl_beta=0.2, kl_est=0, ref=_ref(w, 0.2, 3), weight=seq_mean_weights(w),
         eps=(0.2, 0.28))


def test_zero_beta_ignores_ref():
    """kl_beta = 0 never reads ref_logp (NULL is accepted) and matches the plain loss."""
    import paper_2510_04206_amd as P
    w = gen.make(gen.small_spec(V=700, d=64, dtype="bf16", name="beta0"), seed=29)
    adv = torch.from_numpy(_adv(w)).cuda()
    d_in = to_dev(w)
    log("kl_beta = 0 with a NULL ref_logp")
    a = run_gpu(P.PolicyLoss(w.T, w.d, w.V, w.H.dtype, max_act=w.n_act,
                             opt={"kl_beta": 0.0, "kl_estimator": 1}), d_in, adv)
    b = run_gpu(P.PolicyLoss(w.T, w.d, w.V, w.H.dtype, max_act=w.n_act), d_in, adv)
    assert a["loss"] == b["loss"]
    np.testing.assert_array_equal(a["dW"], b["dW"])
