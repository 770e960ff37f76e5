"""Pins for the oracle's advantage normalisation (CPU only).

Each check ties the oracle to something other than itself: hand-derived
closed forms (tests/golden/adv_norm_cases.json), integer brute force for the
counts, an independent fp64 formulation, and the invariants the paper states
for the normalised set (zero mean, unit variance; Sec. 3.2).
"""
import json
import os

import numpy as np
import pytest

import oracle
from workloads import gen

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "adv_norm_cases.json")


def _cases():
    with open(GOLDEN) as f:
        return json.load(f)["cases"]


@pytest.mark.parametrize("case", _cases(), ids=lambda c: c["name"])
def test_golden_closed_forms(case):
    tg = case["traj_group"]
    out = oracle.task_adv_norm(np.array(case["traj_id"]), np.array(case["mask"]),
                               np.array(case["traj_task"]),
                               None if tg is None else np.array(tg),
                               np.array(case["reward"], np.float32), case["n_task"],
                               case["n_group"], ddof=case["ddof"],
                               drop_uniform=case.get("drop_uniform", False))
    exp = case["expect"]
    exact = set(exp.get("exact", []))
    for key in ("act_count", "task_count"):
        np.testing.assert_array_equal(out[key], np.array(exp[key]))
    for key in ("adv_traj", "task_mean", "task_std"):
        if key not in exp:
            continue
        want = np.array(exp[key], np.float64)
        got = out[key].astype(np.float64)
        if key in exact:
            np.testing.assert_array_equal(got, want.astype(np.float32).astype(np.float64))
        else:
            np.testing.assert_allclose(got, want, rtol=exp["rel"], atol=exp.get("atol", 1e-12))


def _brute_counts(traj_id, mask, n_traj, traj_task, n_task):
    cnt = [0] * n_traj
    for t, m in zip(traj_id.tolist(), mask.tolist()):
        if t >= 0 and m:
            cnt[t] += 1
    task = [0] * n_task
    for j in range(n_traj):
        task[traj_task[j]] += cnt[j]
    return np.array(cnt), np.array(task)


@pytest.mark.parametrize("k", [1, 2, 3, 4, 5])
def test_counts_brute_force(k):
    w = gen.config(k, tensors=False)
    out = oracle.task_adv_norm(w.g_traj_id, w.g_mask, w.traj_task, w.traj_group, w.reward,
                               w.n_task, w.n_group)
    # counts by an independent route: numpy bincount over the action tokens
    sel = (w.g_mask == 1) & (w.g_traj_id >= 0)
    cnt = np.bincount(w.g_traj_id[sel], minlength=w.n_traj)
    np.testing.assert_array_equal(out["act_count"], cnt)
    np.testing.assert_array_equal(out["task_count"],
                                  np.bincount(w.traj_task, weights=cnt, minlength=w.n_task))
    if k == 1:   # plain-Python loop as well, on the small one
        c2, t2 = _brute_counts(w.g_traj_id, w.g_mask, w.n_traj, w.traj_task, w.n_task)
        np.testing.assert_array_equal(out["act_count"], c2)
        np.testing.assert_array_equal(out["task_count"], t2)
    # broadcast: adv_tok is the trajectory's value on action tokens, 0 elsewhere
    want = np.where(sel, out["adv_traj"][np.maximum(w.g_traj_id, 0)], 0.0).astype(np.float32)
    np.testing.assert_array_equal(out["adv_tok"], want)


def _fp64_reference(w, ddof=0, eps=1e-6, groups=True, drop_uniform=False, reward=None):
    """The two normalisation stages written with numpy fp64 reductions."""
    R = (w.reward if reward is None else reward).astype(np.float64)
    keep = np.ones(len(R), bool)
    if groups:
        A = np.zeros_like(R)
        for g in range(w.n_group):
            s = w.traj_group == g
            K = s.sum()
            if drop_uniform and K > 0 and np.all(R[s] == R[s][0]):
                keep[s] = False
                continue
            if K - ddof <= 0:
                continue
            mu = R[s].mean()
            sd = np.sqrt(((R[s] - mu) ** 2).sum() / (K - ddof))
            A[s] = (R[s] - mu) / (sd + eps)
    else:
        A = R.copy()
    sel = (w.g_mask == 1) & (w.g_traj_id >= 0)
    n = np.bincount(w.g_traj_id[sel], minlength=w.n_traj).astype(np.float64)
    out = np.zeros_like(R)
    for i in range(w.n_task):
        s = (w.traj_task == i) & keep
        N = n[s].sum()
        if N == 0:
            continue
        # expand to the token-level set explicitly
        tok = np.repeat(A[s], n[s].astype(np.int64))
        mu = tok.mean()
        sd = np.sqrt(((tok - mu) ** 2).sum() / (N - ddof)) if N - ddof > 0 else 0.0
        out[s] = (A[s] - mu) / (sd + eps)
    return out


@pytest.mark.parametrize("k", [1, 2, 3, 4, 5])
@pytest.mark.parametrize("groups", [True, False])
def test_fp32_against_fp64(k, groups):
    w = gen.config(k, tensors=False)
    out = oracle.task_adv_norm(w.g_traj_id, w.g_mask, w.traj_task,
                               w.traj_group if groups else None, w.reward, w.n_task, w.n_group)
    ref = _fp64_reference(w, groups=groups)
    # fp32 rounding of O(1) quantities, amplified at most by 1/sigma of the task
    np.testing.assert_allclose(out["adv_traj"], ref, rtol=2e-5, atol=2e-5)


@pytest.mark.parametrize("k", [1, 2, 3, 5])
def test_drop_uniform_groups_against_fp64(k):
    """DAPO dynamic sampling: planted all-equal groups are dropped (advantage 0,
    left out of the task statistics); the rest matches the fp64 formulation."""
    w = gen.config(k, tensors=False)
    R = w.reward.copy()
    rng = np.random.default_rng(k)
    for g in rng.choice(w.n_group, size=max(1, w.n_group // 4), replace=False):
        R[w.traj_group == g] = R[w.traj_group == g][0]
    out = oracle.task_adv_norm(w.g_traj_id, w.g_mask, w.traj_task, w.traj_group, R, w.n_task,
                               w.n_group, drop_uniform=True)
    ref = _fp64_reference(w, drop_uniform=True, reward=R)
    np.testing.assert_allclose(out["adv_traj"], ref, rtol=2e-5, atol=2e-5)
    dropped = np.zeros(w.n_traj, bool)
    for g in range(w.n_group):
        s = w.traj_group == g
        dropped[s] = np.all(R[s] == R[s][0])
    assert dropped.any() and np.all(out["adv_traj"][dropped] == 0)
    n = np.bincount(w.g_traj_id[(w.g_mask == 1) & (w.g_traj_id >= 0)], minlength=w.n_traj)
    for i in range(w.n_task):
        assert out["task_count"][i] == n[(w.traj_task == i) & ~dropped].sum()


@pytest.mark.parametrize("k", [1, 2, 3, 4, 5])
def test_normalised_set_zero_mean_unit_variance(k):
    """Sec. 3.2: per task, the token-level advantages have mean 0 and variance 1."""
    w = gen.config(k, tensors=False)
    out = oracle.task_adv_norm(w.g_traj_id, w.g_mask, w.traj_task, w.traj_group, w.reward,
                               w.n_task, w.n_group)
    n = out["act_count"].astype(np.float64)
    A = out["adv_traj"].astype(np.float64)
    for i in range(w.n_task):
        s = w.traj_task == i
        N = n[s].sum()
        assert N == out["task_count"][i]
        mean = (n[s] * A[s]).sum() / N
        assert abs(mean) <= 1e-5
        if out["task_std"][i] > 1e-3:
            var = (n[s] * A[s] ** 2).sum() / N
            assert abs(var - 1.0) <= 1e-4
        else:                         # all-equal rewards: every advantage is exactly 0
            assert np.all(A[s] == 0.0)


def test_zero_std_tasks_in_large_vocab_workload():
    """Workload 5 plants tasks whose rewards are all 0 or all 1."""
    w = gen.config(5, tensors=False)
    out = oracle.task_adv_norm(w.g_traj_id, w.g_mask, w.traj_task, w.traj_group, w.reward,
                               w.n_task, w.n_group)
    for i in (0, 1):
        s = w.traj_task == i
        assert np.all(out["adv_traj"][s] == 0.0)
        assert out["task_std"][i] == 0.0


def test_out_of_range_ids_rejected():
    with pytest.raises(ValueError):
        oracle.task_adv_norm(np.array([0, 5]), np.array([1, 1]), np.array([0]), None,
                             np.array([1.0], np.float32), 1)
    with pytest.raises(ValueError):
        oracle.task_adv_norm(np.array([0]), np.array([1]), np.array([3]), None,
                             np.array([1.0], np.float32), 1)
