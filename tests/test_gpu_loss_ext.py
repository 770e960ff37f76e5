"""GPU parity of the KL penalty and per-token loss weights against the oracle.

The KL term (App. A objectives, -beta D_KL; k3 and k1 estimators) and the
per-token weights (sequence-level aggregation of App. B.2's GRPO form, a
token mean per trajectory then a mean over trajectories) change only the
per-token loss and dL/dlogp; the same tolerances as the plain loss apply:
loss 1e-3 relative, lse 2e-5 and logp 5e-5 absolute, dH/dW 2e-2 relative Frobenius.
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


@pytest.mark.parametrize("k", [1, 2, 3])
def test_sequence_mean_weights_bit_exact(k):
    """agrl_sequence_mean_weights against the oracle on the workload's micro-batch
    (the global stream's first T tokens): counts and fp32 weights bit-exact."""
    import paper_2510_04206_amd as P
    w = gen.config(k, tensors=False)
    tid, mask = w.g_traj_id[: w.T], w.g_mask[: w.T]
    log(f"seq-mean weights case workload {k}: T={w.T} n_traj={w.n_traj}")
    c_ref, w_ref = oracle.sequence_mean_weights(tid, mask, w.n_traj)
    cnt, wt = P.sequence_mean_weights(torch.from_numpy(np.ascontiguousarray(tid)).cuda(),
                                      torch.from_numpy(np.ascontiguousarray(mask)).cuda(),
                                      w.n_traj)
    assert P.agrl_get_device_error() == 0
    np.testing.assert_array_equal(cnt.cpu().numpy(), c_ref)
    np.testing.assert_array_equal(wt.cpu().numpy(), w_ref)


def test_sequence_mean_weights_edges():
    import paper_2510_04206_amd as P
    dev = torch.device("cuda")
    log("seq-mean weights edges: padding only, empty, id out of range")
    # only padding and observations: no trajectory present, every weight 0
    tid = torch.tensor([-1, 0, 1, -1], dtype=torch.int32, device=dev)
    mask = torch.tensor([1, 0, 0, 1], dtype=torch.uint8, device=dev)
    cnt, wt = P.sequence_mean_weights(tid, mask, 2)
    assert cnt.tolist() == [0, 0] and wt.tolist() == [0.0] * 4
    # T = 0 still zeroes the counts
    cnt, wt = P.sequence_mean_weights(torch.empty(0, dtype=torch.int32, device=dev),
                                      torch.empty(0, dtype=torch.uint8, device=dev), 3)
    assert cnt.tolist() == [0, 0, 0] and wt.numel() == 0
    assert P.agrl_get_device_error() == 0
    # an id >= n_traj is flagged and skipped
    tid = torch.tensor([0, 5, 0, 1], dtype=torch.int32, device=dev)
    mask = torch.ones(4, dtype=torch.uint8, device=dev)
    cnt, wt = P.sequence_mean_weights(tid, mask, 2)
    assert P.agrl_get_device_error() == 2
    assert cnt.tolist() == [2, 1]
    np.testing.assert_array_equal(wt.cpu().numpy(), np.float32([0.25, 0, 0.25, 0.5]))


def test_library_weights_in_the_loss():
    """The loss under the library's weights: identical weights to the host-built
    ones, so identical GPU outputs."""
    import paper_2510_04206_amd as P
    w = gen.make(gen.small_spec(V=1800, d=128, dtype="bf16", name="seqlib"), seed=31)
    tid = np.ascontiguousarray(w.g_traj_id[: w.T])
    _, wt = P.sequence_mean_weights(torch.from_numpy(tid).cuda(),
                                    torch.from_numpy(np.ascontiguousarray(w.mask)).cuda(),
                                    w.n_traj)
    host = seq_mean_weights(w)
    np.testing.assert_array_equal(wt.cpu().numpy(), host)
    _run(w, weight=host)
