"""Pins for the oracle's sequence-level aggregation weights (CPU only).

App. B.2 writes GRPO's objective as (1/G) sum_i (1/|o_i|) sum_t (...): a token
mean within each response, then a mean over the responses.  The oracle turns
this into per-token weights w_t = 1/(n_seq * n_tau(t)) of a packed micro-batch.
The checks below tie it to that definition by other routes: a hand-worked
case, the sums the definition fixes, the equal-length special case (where it
is the token mean of App. A, DAPO), and the loss computed trajectory by
trajectory from the per-token surrogate.
"""
import numpy as np
import pytest

import oracle
from workloads import gen


def test_hand_worked_case():
    # trajectory 0: tokens 0,1 (actions); 1: tokens 2,5 (4 is an observation);
    # token 3 is padding; trajectory 2 has no action token in this micro-batch
    tid = np.array([0, 0, 1, -1, 1, 1, 2])
    mask = np.array([1, 1, 1, 1, 0, 1, 0])
    count, w = oracle.sequence_mean_weights(tid, mask, 3)
    np.testing.assert_array_equal(count, [2, 2, 0])
    np.testing.assert_array_equal(w, np.float32([0.25, 0.25, 0.25, 0, 0, 0.25, 0]))


def test_sums_fixed_by_the_definition():
    rng = np.random.default_rng(3)
    T, n_traj = 5000, 37
    tid = rng.integers(-1, n_traj, T)
    mask = (rng.random(T) < 0.6).astype(np.uint8)
    count, w = oracle.sequence_mean_weights(tid, mask, n_traj)
    sel = (tid >= 0) & (mask == 1)
    np.testing.assert_array_equal(count, np.bincount(tid[sel], minlength=n_traj))
    n_seq = int((count > 0).sum())
    assert np.all(w[~sel] == 0)
    # each present trajectory carries 1/n_seq in total, the micro-batch 1
    for j in range(n_traj):
        tot = w[(tid == j) & sel].astype(np.float64).sum()
        if count[j]:
            assert abs(tot - 1.0 / n_seq) <= 1e-7 / n_seq
        else:
            assert tot == 0
    assert abs(w.astype(np.float64).sum() - 1.0) <= 1e-6


def test_equal_lengths_reduce_to_the_token_mean():
    L, n = 12, 9
    tid = np.repeat(np.arange(n), L + 3)
    mask = np.tile(np.r_[np.zeros(3, np.uint8), np.ones(L, np.uint8)], n)
    _, w = oracle.sequence_mean_weights(tid, mask, n)
    N = int(mask.sum())
    np.testing.assert_array_equal(w[mask == 1], np.float32(1.0 / N))


def test_weighted_loss_is_the_mean_over_trajectories_of_token_means():
    """The oracle loss under these weights against App. B.2's form evaluated
    trajectory by trajectory from the per-token surrogate."""
    rng = np.random.default_rng(11)
    T, d, V, n_traj = 90, 16, 48, 6
    H = rng.standard_normal((T, d)).astype(np.float32)
    W = (0.3 * rng.standard_normal((V, d))).astype(np.float32)
    y = rng.integers(0, V, T).astype(np.int32)
    tid = np.sort(rng.integers(0, n_traj, T)).astype(np.int32)
    mask = (rng.random(T) < 0.7).astype(np.uint8)
    adv = rng.standard_normal(T).astype(np.float32)
    old = (rng.standard_normal(T) * 0.3 - 3.0).astype(np.float32)
    eps = 0.2
    _, w = oracle.sequence_mean_weights(tid, mask, n_traj)
    r = oracle.policy_loss(H, W, y, mask, adv, old, eps_lo=eps, eps_hi=eps, token_weight=w,
                           backward=False)
    # per-token surrogate from the log-softmax in fp64
    z = H.astype(np.float64) @ W.astype(np.float64).T
    logp = z[np.arange(T), y] - (np.log(np.exp(z - z.max(1, keepdims=True)).sum(1))
                                 + z.max(1))
    rho = np.exp(logp - old)
    s = np.minimum(rho * adv, np.clip(rho, 1 - eps, 1 + eps) * adv)
    means = [s[(tid == j) & (mask == 1)].mean() for j in range(n_traj)
             if ((tid == j) & (mask == 1)).any()]
    want = -np.mean(means)
    assert abs(r["loss"] - want) <= 1e-6 * max(1.0, abs(want))


def test_workload_micro_batch_against_a_python_loop():
    w = gen.config(1, tensors=False)
    tid, mask = w.g_traj_id[: w.T], w.mask
    count, wt = oracle.sequence_mean_weights(tid, mask, w.n_traj)
    cnt = {}
    for t in range(w.T):
        if tid[t] >= 0 and mask[t]:
            cnt[int(tid[t])] = cnt.get(int(tid[t]), 0) + 1
    n_seq = len(cnt)
    for t in range(w.T):
        want = np.float32(1.0 / (n_seq * cnt[int(tid[t])])) if (tid[t] >= 0 and mask[t]) else 0
        assert wt[t] == want


def test_out_of_range_id_rejected():
    with pytest.raises(ValueError):
        oracle.sequence_mean_weights(np.array([0, 3]), np.array([1, 1]), 2)
