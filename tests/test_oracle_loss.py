"""Pins for the oracle's policy loss, forward and backward (CPU only).

The oracle is tied to: a hand-worked example with closed forms; full-logit
brute force through library routines (BLAS matmul + scipy logsumexp);
central finite differences of its own loss; the cross-entropy special case
checked against torch's autograd; and invariants of the gradient (rows of G
sum to zero, dH^T H == W^T dW, masked tokens inert, ratio == 1 when the
behaviour and current policies agree).
"""
import math

import numpy as np
import pytest
import torch
from scipy.special import logsumexp

import oracle
from workloads import gen


def _random_case(T, V, d, seed, noise=0.3, frac_act=0.6, adv_scale=1.0):
    rng = np.random.default_rng(seed)
    H = rng.standard_normal((T, d)).astype(np.float32)
    W = (0.5 * rng.standard_normal((V, d))).astype(np.float32)
    y = rng.integers(0, V, T).astype(np.int32)
    mask = (rng.random(T) < frac_act).astype(np.uint8)
    adv = (adv_scale * rng.standard_normal(T)).astype(np.float32)
    z = H.astype(np.float64) @ W.astype(np.float64).T
    lp = z[np.arange(T), y] - logsumexp(z, axis=1)
    old = (lp + noise * rng.standard_normal(T)).astype(np.float32)
    return H, W, y, mask, adv, old


def _brute(H, W, y, mask, adv, old, eps_lo, eps_hi, temp=1.0, n_norm=0):
    z = (H.astype(np.float64) @ W.astype(np.float64).T) / temp
    lse = logsumexp(z, axis=1)
    logp = z[np.arange(len(y)), y] - lse
    rho = np.exp(logp - old.astype(np.float64))
    A = adv.astype(np.float64)
    s = np.minimum(rho * A, np.clip(rho, 1 - eps_lo, 1 + eps_hi) * A)
    m = mask.astype(bool)
    N = n_norm if n_norm > 0 else m.sum()
    loss = -(s[m].sum() / N) if N > 0 else 0.0
    hi = int(np.sum(m & (A > 0) & (rho > 1 + eps_hi)))
    lo = int(np.sum(m & (A < 0) & (rho < 1 - eps_lo)))
    return dict(lse=np.where(m, lse, 0), logp=np.where(m, logp, 0), loss=loss, n_clip=[hi, lo])


def test_hand_worked_two_word_vocabulary():
    """V = 2, d = 1: h = 1, w = (1, -1), y = 0, so z = (1, -1).

    lse = 1 + log(1 + e^-2), logp = -log(1 + e^-2), p = (sigmoid(2), sigmoid(-2)).
    With old = logp - 0.5 the ratio is e^0.5 > 1.2:
      A = +1: clipped branch, loss = -1.2, gradient 0.
      A = -1: unclipped branch, loss = e^0.5, g = dL/dlogp = e^0.5 and
              dH = g (w_y - sum_v p_v w_v) = e^0.5 (1 - tanh(1)),
              dW_v = g (1[v=y] - p_v) h = e^0.5 (1 - sigmoid(2), -sigmoid(-2)).
    """
    H = np.array([[1.0]], np.float32)
    W = np.array([[1.0], [-1.0]], np.float32)
    y = np.array([0], np.int32)
    m = np.array([1], np.uint8)
    logp = -math.log1p(math.exp(-2.0))
    old = np.array([logp - 0.5], np.float32)
    dold = float(old[0]) - logp + 0.5          # fp32 rounding of old, carried exactly
    rho = math.exp(0.5 - dold)
    sig2 = 1.0 / (1.0 + math.exp(-2.0))

    r = oracle.policy_loss(H, W, y, m, np.array([1.0], np.float32), old)
    assert r["lse"][0] == pytest.approx(1.0 + math.log1p(math.exp(-2.0)), rel=1e-14)
    assert r["logp"][0] == pytest.approx(logp, rel=1e-14)
    assert r["loss"] == pytest.approx(-1.2, rel=1e-14)
    assert list(r["n_clip"]) == [1, 0]
    assert np.all(r["dH"] == 0) and np.all(r["dW"] == 0)

    r = oracle.policy_loss(H, W, y, m, np.array([-1.0], np.float32), old)
    assert r["loss"] == pytest.approx(rho, rel=1e-12)
    assert list(r["n_clip"]) == [0, 0]
    assert r["dH"][0, 0] == pytest.approx(rho * (1.0 - math.tanh(1.0)), rel=1e-12)
    assert r["dW"][0, 0] == pytest.approx(rho * (1.0 - sig2), rel=1e-12)
    assert r["dW"][1, 0] == pytest.approx(-rho * (1.0 - sig2), rel=1e-12)


@pytest.mark.parametrize("T,V,d", [(16, 7, 3), (40, 64, 16), (64, 1000, 64)])
@pytest.mark.parametrize("eps", [(0.2, 0.2), (0.2, 0.28)])
@pytest.mark.parametrize("temp", [1.0, 0.8])
def test_forward_against_full_logits(T, V, d, eps, temp):
    H, W, y, mask, adv, old = _random_case(T, V, d, seed=T * 7 + V)
    r = oracle.policy_loss(H, W, y, mask, adv, old, eps_lo=eps[0], eps_hi=eps[1],
                           temperature=temp, backward=False)
    b = _brute(H, W, y, mask, adv, old, eps[0], eps[1], temp)
    np.testing.assert_allclose(r["lse"], b["lse"], rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(r["logp"], b["logp"], rtol=1e-12, atol=1e-12)
    assert r["loss"] == pytest.approx(b["loss"], rel=1e-11, abs=1e-14)
    assert list(r["n_clip"]) == b["n_clip"]


def test_forward_against_full_logits_bf16_inputs():
    H, W, y, mask, adv, old = _random_case(48, 300, 32, seed=3)
    Hb = torch.from_numpy(H).to(torch.bfloat16)
    Wb = torch.from_numpy(W).to(torch.bfloat16)
    r = oracle.policy_loss(Hb, Wb, y, mask, adv, old, backward=False)
    b = _brute(Hb.float().numpy(), Wb.float().numpy(), y, mask, adv, old, 0.2, 0.2)
    np.testing.assert_allclose(r["logp"], b["logp"], rtol=1e-12, atol=1e-12)
    assert r["loss"] == pytest.approx(b["loss"], rel=1e-11)


def test_n_norm_override_scales_loss_and_gradient():
    H, W, y, mask, adv, old = _random_case(20, 30, 8, seed=5)
    a = oracle.policy_loss(H, W, y, mask, adv, old)
    b = oracle.policy_loss(H, W, y, mask, adv, old, n_norm=1000)
    n = int(mask.sum())
    assert b["loss"] == pytest.approx(a["loss"] * n / 1000, rel=1e-12)
    np.testing.assert_allclose(b["dW"], a["dW"] * n / 1000, rtol=1e-12, atol=1e-18)


def _fd_loss(H, W, y, mask, adv, old, eps, temp):
    return oracle.policy_loss(H, W, y, mask, adv, old, eps_lo=eps[0], eps_hi=eps[1],
                              temperature=temp, backward=False)


@pytest.mark.parametrize("temp", [1.0, 0.8])
def test_gradients_by_finite_differences(temp):
    """Central differences of the oracle's loss against its dH and dW.

    Inputs are fp32, so the step is taken on fp32 values and the exact
    perturbed difference is used.  Tokens whose log-ratio sits within 2e-3 of a
    clip boundary are masked out so the loss is smooth at every probe.
    """
    eps = (0.2, 0.25)
    T, V, d = 24, 17, 6
    H, W, y, mask, adv, old = _random_case(T, V, d, seed=11, noise=0.25)
    base = _fd_loss(H, W, y, mask, adv, old, eps, temp)
    delta = base["logp"] - old
    near = (np.abs(delta - math.log(1 + eps[1])) < 2e-3) | (np.abs(delta - math.log(1 - eps[0])) < 2e-3)
    mask = (mask.astype(bool) & ~near).astype(np.uint8)
    full = oracle.policy_loss(H, W, y, mask, adv, old, eps_lo=eps[0], eps_hi=eps[1], temperature=temp)
    assert full["n_clip"].sum() > 0           # clipped tokens are exercised too
    rng = np.random.default_rng(0)
    h = 1e-3
    for _ in range(12):
        n, k = int(rng.integers(T)), int(rng.integers(d))
        Hp, Hm = H.copy(), H.copy()
        Hp[n, k] += h
        Hm[n, k] -= h
        step = float(Hp[n, k]) - float(Hm[n, k])
        fd = (_fd_loss(Hp, W, y, mask, adv, old, eps, temp)["loss"]
              - _fd_loss(Hm, W, y, mask, adv, old, eps, temp)["loss"]) / step
        assert fd == pytest.approx(full["dH"][n, k], rel=2e-5, abs=1e-9)
    for _ in range(12):
        v, k = int(rng.integers(V)), int(rng.integers(d))
        Wp, Wm = W.copy(), W.copy()
        Wp[v, k] += h
        Wm[v, k] -= h
        step = float(Wp[v, k]) - float(Wm[v, k])
        fd = (_fd_loss(H, Wp, y, mask, adv, old, eps, temp)["loss"]
              - _fd_loss(H, Wm, y, mask, adv, old, eps, temp)["loss"]) / step
        assert fd == pytest.approx(full["dW"][v, k], rel=2e-5, abs=1e-9)


def test_cross_entropy_special_case_against_torch():
    """A == 1, old == logp and no clipping: ratio 1, loss -1, gradients of mean CE."""
    T, V, d = 32, 50, 12
    H, W, y, mask, _, _ = _random_case(T, V, d, seed=2)
    b = _brute(H, W, y, mask, np.ones(T, np.float32), np.zeros(T, np.float32), 0.2, 0.2)
    # old = logp exactly is not representable in fp32; the residual is carried through rho
    old = b["logp"].astype(np.float32)
    adv = np.ones(T, np.float32)
    r = oracle.policy_loss(H, W, y, mask, adv, old, eps_lo=1e30, eps_hi=1e30)
    m = mask.astype(bool)
    rho = np.exp(b["logp"] - old.astype(np.float64))
    assert r["loss"] == pytest.approx(-rho[m].mean(), rel=1e-12)
    assert r["loss"] == pytest.approx(-1.0, rel=1e-6)

    Ht = torch.tensor(H, dtype=torch.float64, requires_grad=True)
    Wt = torch.tensor(W, dtype=torch.float64, requires_grad=True)
    idx = torch.from_numpy(np.nonzero(m)[0])
    logits = Ht[idx] @ Wt.t()
    ce = torch.nn.functional.cross_entropy(logits, torch.from_numpy(y[m].astype(np.int64)),
                                           reduction="none")
    # the oracle's gradient carries rho_n = 1 + O(1e-7): weight CE by it
    (torch.from_numpy(rho[m]) * ce).mean().backward()
    np.testing.assert_allclose(r["dH"], Ht.grad.numpy(), rtol=1e-10, atol=1e-14)
    np.testing.assert_allclose(r["dW"], Wt.grad.numpy(), rtol=1e-10, atol=1e-14)


def test_ratio_one_gives_unclipped_gradient():
    """old == logp: rho == 1, never clipped, g_n = -A_n / N and L = -mean(A)."""
    T, V, d = 30, 40, 8
    H, W, y, mask, adv, _ = _random_case(T, V, d, seed=9)
    b = _brute(H, W, y, mask, adv, np.zeros(T, np.float32), 0.2, 0.2)
    old = b["logp"].astype(np.float32)
    r = oracle.policy_loss(H, W, y, mask, adv, old)
    m = mask.astype(bool)
    rho = np.exp(b["logp"] - old.astype(np.float64))
    np.testing.assert_allclose(r["g"][m], -adv[m] * rho[m] / m.sum(), rtol=1e-12)
    assert np.all(r["g"][~m] == 0)
    assert r["loss"] == pytest.approx(-(adv[m] * rho[m]).mean(), rel=1e-12)
    assert list(r["n_clip"]) == [0, 0]


def test_gradient_invariants():
    T, V, d = 40, 33, 10
    H, W, y, mask, adv, old = _random_case(T, V, d, seed=21)
    r = oracle.policy_loss(H, W, y, mask, adv, old)
    # rows of G sum to zero over the vocabulary, so the columns of dW sum to zero
    np.testing.assert_allclose(r["dW"].sum(axis=0), 0.0, atol=1e-14)
    # L depends on H and W only through H W^T: dH^T H == W^T dW
    lhs = r["dH"].T @ H.astype(np.float64)
    rhs = W.astype(np.float64).T @ r["dW"]
    np.testing.assert_allclose(lhs, rhs, rtol=1e-10, atol=1e-14)
    assert np.all(r["dH"][mask == 0] == 0)


def test_masked_tokens_are_inert():
    """Poisoned masked tokens (NaN hidden state, bad id, NaN adv/old) change nothing."""
    T, V, d = 36, 20, 8
    H, W, y, mask, adv, old = _random_case(T, V, d, seed=4)
    a = oracle.policy_loss(H, W, y, mask, adv, old)
    Hp, yp, ap, op = H.copy(), y.copy(), adv.copy(), old.copy()
    off = mask == 0
    Hp[off] = np.nan
    yp[off] = V + 5
    ap[off] = np.nan
    op[off] = np.nan
    b = oracle.policy_loss(Hp, W, yp, mask, ap, op)
    assert a["loss"] == b["loss"]
    for key in ("logp", "lse", "dW"):
        np.testing.assert_array_equal(a[key], b[key])
    np.testing.assert_array_equal(a["dH"], b["dH"])
    assert np.all(b["dH"][off] == 0) and not np.signbit(b["dH"][off]).any()


def test_no_action_tokens():
    T, V, d = 8, 5, 4
    H, W, y, _, adv, old = _random_case(T, V, d, seed=1)
    r = oracle.policy_loss(H, W, y, np.zeros(T, np.uint8), adv, old)
    assert r["loss"] == 0.0
    assert np.all(r["dH"] == 0) and np.all(r["dW"] == 0)


def test_token_sample_matches_whole_batch():
    w = gen.make(gen.small_spec(V=300, d=64, dtype="bf16"), seed=5)
    adv = np.random.default_rng(0).standard_normal(w.T).astype(np.float32)
    full = oracle.policy_loss(w.H, w.W, w.token_id, w.mask, adv, w.old_logp)
    toks = np.array([0, 3, int(np.nonzero(w.mask)[0][0]), w.T - 1])
    s = oracle.token_sample(w.H, w.W, w.token_id, w.mask, adv, w.old_logp, toks)
    np.testing.assert_array_equal(s["lse"], full["lse"][toks])
    np.testing.assert_array_equal(s["logp"], full["logp"][toks])
    np.testing.assert_array_equal(s["g"], full["g"][toks])
    np.testing.assert_array_equal(s["dH"], full["dH"][toks])


def test_config1_end_to_end_consistency():
    """Workload 1 through both oracle stages; cross-checked with full logits."""
    w = gen.config(1)
    a = oracle.task_adv_norm(w.g_traj_id, w.g_mask, w.traj_task, w.traj_group, w.reward,
                             w.n_task, w.n_group)
    adv = a["adv_tok"][: w.T]
    r = oracle.policy_loss(w.H, w.W, w.token_id, w.mask, adv, w.old_logp)
    b = _brute(w.H.numpy(), w.W.numpy(), w.token_id, w.mask, adv, w.old_logp, 0.2, 0.2)
    assert r["loss"] == pytest.approx(b["loss"], rel=1e-10)
    np.testing.assert_allclose(r["dW"].sum(axis=0), 0.0, atol=1e-12)


@pytest.mark.parametrize("eps", [(0.2, 0.28), (0.3, 0.2)])
def test_decoupled_clip_bounds_hand_placed_ratios(eps):
    """App. A (DAPO): clip(rho, 1 - eps_low, 1 + eps_high), bounds set independently.

    Ratios are placed on both sides of every bound for A = +1 and A = -1; the
    surrogate min(rho A, clip(rho) A) and which tokens stop the gradient follow
    by hand: A > 0 is cut off only above 1 + eps_high, A < 0 only below 1 - eps_low.
    """
    lo, hi = eps
    ratios = [1 - lo - 0.03, 1 - lo + 0.02, 0.95, 1.05, 1 + min(lo, hi) + 0.02,
              1 + hi - 0.02, 1 + hi + 0.03, 1 + max(lo, hi) + 0.05]
    rs = np.array(ratios * 2)
    A = np.array([1.0] * len(ratios) + [-1.0] * len(ratios), np.float32)
    T, V, d = len(rs), 9, 4
    rng = np.random.default_rng(8)
    H = rng.standard_normal((T, d)).astype(np.float32)
    W = rng.standard_normal((V, d)).astype(np.float32)
    y = rng.integers(0, V, T).astype(np.int32)
    mask = np.ones(T, np.uint8)
    lp = _brute(H, W, y, mask, A, np.zeros(T, np.float32), lo, hi)["logp"]
    old = (lp - np.log(rs)).astype(np.float32)
    rho = np.exp(lp - old.astype(np.float64))       # the fp32 rounding of old is carried
    r = oracle.policy_loss(H, W, y, mask, A, old, eps_lo=lo, eps_hi=hi)
    cut = ((A > 0) & (rho > 1 + hi)) | ((A < 0) & (rho < 1 - lo))
    s = np.where(A > 0, np.minimum(rho, 1 + hi), -np.maximum(rho, 1 - lo))
    assert r["loss"] == pytest.approx(-s.mean(), rel=1e-12)
    assert list(r["n_clip"]) == [int(((A > 0) & (rho > 1 + hi)).sum()),
                                 int(((A < 0) & (rho < 1 - lo)).sum())]
    np.testing.assert_allclose(r["g"], np.where(cut, 0.0, -A * rho / T), rtol=1e-12, atol=0)


@pytest.mark.parametrize("temp", [1.0, 0.7])
def test_token_logprob_against_full_log_softmax(temp):
    """The forward-only log-prob pass is log_softmax(H W^T / temperature) gathered at
    the sampled ids on action tokens (torch's log_softmax, fp64), 0 elsewhere."""
    H, W, y, mask, _, _ = _random_case(50, 333, 24, seed=21)
    r = oracle.token_logprob(H, W, y, mask, temperature=temp)
    z = torch.from_numpy(H).double() @ torch.from_numpy(W).double().T / temp
    ls = torch.log_softmax(z, dim=1)
    ref = ls[torch.arange(len(y)), torch.from_numpy(y).long()].numpy()
    m = mask.astype(bool)
    np.testing.assert_allclose(r["logp"][m], ref[m], rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(r["lse"][m], torch.logsumexp(z, 1).numpy()[m], rtol=1e-12)
    assert np.all(r["logp"][~m] == 0) and np.all(r["lse"][~m] == 0)


# ---------------------------------------------------------------------------
# KL penalty and per-token weights (App. A objectives: -beta * D_KL; sequence-
# level aggregation as per-token weights)

def _brute_ext(H, W, y, mask, adv, old, eps_lo, eps_hi, beta, est, ref, weight=None):
    """Full-logit brute force of L = -sum_n w_n (s_n - beta KL_n), w_n = 1/N by default."""
    z = H.astype(np.float64) @ W.astype(np.float64).T
    logp = z[np.arange(len(y)), y] - logsumexp(z, axis=1)
    rho = np.exp(logp - old.astype(np.float64))
    A = adv.astype(np.float64)
    s = np.minimum(rho * A, np.clip(rho, 1 - eps_lo, 1 + eps_hi) * A)
    r = ref.astype(np.float64)
    kl = (np.exp(r - logp) - (r - logp) - 1.0) if est == 0 else (logp - r)
    m = mask.astype(bool)
    w = np.full(len(y), 1.0 / m.sum()) if weight is None else weight.astype(np.float64)
    return -np.sum((w * (s - beta * kl))[m])


@pytest.mark.parametrize("est", [0, 1])
@pytest.mark.parametrize("beta", [0.05, 0.5])
def test_kl_loss_against_full_logits(est, beta):
    H, W, y, mask, adv, old = _random_case(40, 64, 16, seed=31)
    ref = (old + 0.3 * np.random.default_rng(2).standard_normal(40)).astype(np.float32)
    r = oracle.policy_loss(H, W, y, mask, adv, old, kl_beta=beta, kl_estimator=est, ref_logp=ref,
                           backward=False)
    assert r["loss"] == pytest.approx(_brute_ext(H, W, y, mask, adv, old, 0.2, 0.2, beta, est, ref),
                                      rel=1e-11)


def test_token_weights_against_full_logits():
    H, W, y, mask, adv, old = _random_case(40, 64, 16, seed=33)
    w = np.random.default_rng(4).random(40).astype(np.float32)
    ref = old.copy()
    r = oracle.policy_loss(H, W, y, mask, adv, old, token_weight=w, kl_beta=0.2, ref_logp=ref,
                           backward=False)
    assert r["loss"] == pytest.approx(_brute_ext(H, W, y, mask, adv, old, 0.2, 0.2, 0.2, 0, ref, w),
                                      rel=1e-11)


def test_kl_k3_vanishes_at_the_reference():
    """ref_logp == logp: k3 KL and its derivative are 0, so everything equals beta = 0."""
    H, W, y, mask, adv, old = _random_case(30, 50, 12, seed=35)
    r0 = oracle.policy_loss(H, W, y, mask, adv, old)
    r1 = oracle.policy_loss(H, W, y, mask, adv, old, kl_beta=0.7, kl_estimator=0,
                            ref_logp=r0["logp"].astype(np.float32))
    # ref is logp rounded to fp32: KL ~ (1e-8)^2, gradient ~ 1e-8
    assert r1["loss"] == pytest.approx(r0["loss"], rel=1e-9, abs=1e-12)
    np.testing.assert_allclose(r1["g"], r0["g"], rtol=0, atol=1e-8)
    np.testing.assert_allclose(r1["dH"], r0["dH"], rtol=0, atol=1e-8)


def test_kl_k1_adds_a_constant_logp_gradient():
    """k1: dKL/dlogp = 1, so g gains beta / N on every action token, clipped or not."""
    H, W, y, mask, adv, old = _random_case(30, 50, 12, seed=37, noise=0.4)
    ref = np.zeros(30, np.float32)
    r0 = oracle.policy_loss(H, W, y, mask, adv, old, backward=False)
    r1 = oracle.policy_loss(H, W, y, mask, adv, old, kl_beta=0.3, kl_estimator=1, ref_logp=ref,
                            backward=False)
    m = mask.astype(bool)
    assert r0["n_clip"].sum() > 0
    np.testing.assert_allclose(r1["g"][m] - r0["g"][m], 0.3 / m.sum(), rtol=1e-12)
    assert np.all(r1["g"][~m] == 0)


def test_uniform_token_weights_equal_the_token_mean():
    H, W, y, mask, adv, old = _random_case(30, 50, 12, seed=39)
    r0 = oracle.policy_loss(H, W, y, mask, adv, old)
    w = np.full(30, 1.0 / mask.sum(), np.float32)
    r1 = oracle.policy_loss(H, W, y, mask, adv, old, token_weight=w)
    # w is 1/N rounded to fp32
    assert r1["loss"] == pytest.approx(r0["loss"], rel=1e-7)
    np.testing.assert_allclose(r1["dW"], r0["dW"], rtol=1e-7, atol=1e-14)


@pytest.mark.parametrize("est", [0, 1])
def test_kl_and_weight_gradients_by_finite_differences(est):
    T, V, d = 20, 13, 5
    H, W, y, mask, adv, old = _random_case(T, V, d, seed=41, noise=0.2)
    rng = np.random.default_rng(5)
    ref = (old + 0.2 * rng.standard_normal(T)).astype(np.float32)
    w = (0.5 + rng.random(T)).astype(np.float32) / T
    kw = dict(kl_beta=0.4, kl_estimator=est, ref_logp=ref, token_weight=w, eps_lo=0.2, eps_hi=0.25)
    base = oracle.policy_loss(H, W, y, mask, adv, old, backward=False, **kw)
    delta = base["logp"] - old
    near = (np.abs(delta - math.log(1.25)) < 2e-3) | (np.abs(delta - math.log(0.8)) < 2e-3)
    mask = (mask.astype(bool) & ~near).astype(np.uint8)
    full = oracle.policy_loss(H, W, y, mask, adv, old, **kw)
    L = lambda H_, W_: oracle.policy_loss(H_, W_, y, mask, adv, old, backward=False, **kw)["loss"]
    h = 1e-3
    for _ in range(8):
        n, k = int(rng.integers(T)), int(rng.integers(d))
        Hp, Hm = H.copy(), H.copy()
        Hp[n, k] += h
        Hm[n, k] -= h
        fd = (L(Hp, W) - L(Hm, W)) / (float(Hp[n, k]) - float(Hm[n, k]))
        assert fd == pytest.approx(full["dH"][n, k], rel=2e-5, abs=1e-9)
    for _ in range(8):
        v, k = int(rng.integers(V)), int(rng.integers(d))
        Wp, Wm = W.copy(), W.copy()
        Wp[v, k] += h
        Wm[v, k] -= h
        fd = (L(H, Wp) - L(H, Wm)) / (float(Wp[v, k]) - float(Wm[v, k]))
        assert fd == pytest.approx(full["dW"][v, k], rel=2e-5, abs=1e-9)
