"""GPU parity of agrl_task_adv_norm against the oracle: bit-exact (MI355X)."""
import json
import os

import numpy as np
import pytest
import torch

import oracle
from workloads import gen

from helpers import adv_inputs, log

pytestmark = pytest.mark.gpu

KEYS = ("act_count", "task_count", "task_mean", "task_std", "adv_traj", "adv_tok")


def _gpu(traj_id, mask, traj_task, traj_group, reward, n_task, n_group, ddof=0, drop=False,
         ranges=True):
    import paper_2510_04206_amd as P
    dev = "cuda"
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
    out = P.task_adv_norm(t(traj_id), t(mask), t(traj_task),
                          None if traj_group is None else t(traj_group), t(reward), n_task,
                          n_group, opt={"std_ddof": ddof, "drop_uniform_groups": int(drop)},
                          member_ranges=ranges)
    assert P.agrl_get_device_error() == 0
    return {k: v.cpu().numpy() for k, v in out.items()}


def _assert_bitwise(g, r):
    for k in KEYS:
        a, b = np.asarray(g[k]), np.asarray(r[k])
        if a.dtype == np.float32:
            np.testing.assert_array_equal(a.view(np.uint32), b.view(np.uint32), err_msg=k)
        else:
            np.testing.assert_array_equal(a, b, err_msg=k)


@pytest.mark.parametrize("k", [1, 2, 3, 4, 5])
@pytest.mark.parametrize("groups", [True, False])
@pytest.mark.parametrize("ddof", [0, 1])
def test_adv_norm_bit_exact(k, groups, ddof):
    w = gen.config(k, tensors=False)
    log(f"adv_norm workload {k} groups={groups} ddof={ddof} T_g={w.T_g}")
    tg = w.traj_group if groups else None
    r = oracle.task_adv_norm(w.g_traj_id, w.g_mask, w.traj_task, tg, w.reward, w.n_task,
                             w.n_group, ddof=ddof)
    g = _gpu(w.g_traj_id, w.g_mask, w.traj_task, tg, w.reward, w.n_task, w.n_group, ddof)
    _assert_bitwise(g, r)


GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "adv_norm_cases.json")


@pytest.mark.parametrize("case", json.load(open(GOLDEN))["cases"], ids=lambda c: c["name"])
def test_adv_norm_golden_cases(case):
    log(f"adv_norm golden {case['name']}")
    tg = None if case["traj_group"] is None else np.array(case["traj_group"], np.int32)
    args = (np.array(case["traj_id"], np.int32), np.array(case["mask"], np.uint8),
            np.array(case["traj_task"], np.int32), tg, np.array(case["reward"], np.float32),
            case["n_task"], case["n_group"])
    drop = case.get("drop_uniform", False)
    r = oracle.task_adv_norm(*args, ddof=case["ddof"], drop_uniform=drop)
    g = _gpu(*args, ddof=case["ddof"], drop=drop)
    _assert_bitwise(g, r)


@pytest.mark.parametrize("k", [1, 2, 3, 5])
@pytest.mark.parametrize("ddof", [0, 1])
def test_adv_norm_drop_uniform_groups_bit_exact(k, ddof):
    """DAPO dynamic sampling with planted all-equal groups (workload 5 also has
    whole tasks of equal rewards)."""
    w = gen.config(k, tensors=False)
    R = w.reward.copy()
    rng = np.random.default_rng(100 + k)
    for g in rng.choice(w.n_group, size=max(1, w.n_group // 4), replace=False):
        R[w.traj_group == g] = R[w.traj_group == g][0]
    log(f"adv_norm drop_uniform workload {k} ddof={ddof}")
    args = (w.g_traj_id, w.g_mask, w.traj_task, w.traj_group, R, w.n_task, w.n_group)
    r = oracle.task_adv_norm(*args, ddof=ddof, drop_uniform=True)
    g = _gpu(*args, ddof=ddof, drop=True)
    _assert_bitwise(g, r)


def test_adv_norm_edge_cases():
    """Empty trajectories, a task with no action tokens, padding tokens, many tasks."""
    rng = np.random.default_rng(3)
    n_traj, n_task, n_group = 300, 7, 75
    traj_task = rng.integers(0, n_task - 1, n_traj).astype(np.int32)   # task n_task-1 empty
    traj_group = (np.arange(n_traj) // 4).astype(np.int32)
    reward = rng.standard_normal(n_traj).astype(np.float32)
    T_g = 20011
    traj_id = rng.integers(-1, n_traj, T_g).astype(np.int32)
    traj_id[traj_id == 17] = 18                                      # trajectory 17 has no tokens
    mask = (rng.random(T_g) < 0.4).astype(np.uint8)
    log("adv_norm edge cases")
    for tg in (traj_group, None):
        args = (traj_id, mask, traj_task, tg, reward, n_task, n_group)
        _assert_bitwise(_gpu(*args), oracle.task_adv_norm(*args))


def test_adv_norm_out_of_range_ids_flagged():
    import paper_2510_04206_amd as P
    log("adv_norm out-of-range ids")
    traj_id = np.array([0, 1, 5], np.int32)
    mask = np.ones(3, np.uint8)
    t = lambda a: torch.from_numpy(a).cuda()
    P.task_adv_norm(t(traj_id), t(mask), t(np.array([0, 0], np.int32)), None,
                    t(np.array([1.0, 0.0], np.float32)), 1)
    assert P.agrl_get_device_error() & 2
    P.task_adv_norm(t(traj_id[:2]), t(mask[:2]), t(np.array([0, 3], np.int32)), None,
                    t(np.array([1.0, 0.0], np.float32)), 1)
    assert P.agrl_get_device_error() & 4
    assert P.agrl_get_device_error() == 0


def _shuffled(w, seed):
    """The same batch with the trajectories renumbered by a random permutation,
    so that no group or task occupies a contiguous index range."""
    rng = np.random.default_rng(seed)
    perm = rng.permutation(w.n_traj).astype(np.int32)      # old index -> new index
    inv = np.empty_like(perm)
    inv[perm] = np.arange(w.n_traj, dtype=np.int32)
    tid = w.g_traj_id.copy()
    tid[tid >= 0] = perm[tid[tid >= 0]]
    return (tid, w.g_mask, w.traj_task[inv], w.traj_group[inv], w.reward[inv], w.n_task,
            w.n_group)


@pytest.mark.parametrize("k", [1, 2, 3, 4, 5])
def test_adv_norm_member_ranges_bit_exact(k):
    """The member-range scans (agrl_options.adv_ranges) and the full scans give
    the oracle's bits, for trajectories stored segment by segment and for a
    random renumbering of them, with the group stage and DAPO's drop."""
    w = gen.config(k, tensors=False)
    R = w.reward.copy()
    rng = np.random.default_rng(200 + k)
    for g in rng.choice(w.n_group, size=max(1, w.n_group // 5), replace=False):
        R[w.traj_group == g] = R[w.traj_group == g][0]
    base = (w.g_traj_id, w.g_mask, w.traj_task, w.traj_group, R, w.n_task, w.n_group)
    for name, args in (("stored by segment", base), ("renumbered", _shuffled(w, 300 + k))):
        for drop in (False, True):
            log(f"adv_norm member ranges workload {k} {name} drop={drop}")
            r = oracle.task_adv_norm(*args, drop_uniform=drop)
            for ranges in (True, False):
                _assert_bitwise(_gpu(*args, drop=drop, ranges=ranges), r)
            tg_none = args[:3] + (None,) + args[4:]
            if not drop:
                r0 = oracle.task_adv_norm(*tg_none)
                _assert_bitwise(_gpu(*tg_none, ranges=True), r0)


def test_adv_norm_many_groups():
    """10^4 groups of 4 over 4 * 10^4 trajectories (a global batch far larger than
    the workloads'), bit-exact with and without member ranges; both timed."""
    import paper_2510_04206_amd as P
    rng = np.random.default_rng(7)
    n_group, K, n_task = 10000, 4, 50
    n_traj = n_group * K
    traj_group = np.repeat(np.arange(n_group, dtype=np.int32), K)
    traj_task = (traj_group * n_task // n_group).astype(np.int32)
    reward = rng.random(n_traj, dtype=np.float32)
    lens = rng.integers(20, 60, n_traj)
    traj_id = np.repeat(np.arange(n_traj, dtype=np.int32), lens)
    mask = (rng.random(traj_id.size) < 0.5).astype(np.uint8)
    args = (traj_id, mask, traj_task, traj_group, reward, n_task, n_group)
    r = oracle.task_adv_norm(*args)
    dev = "cuda"
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
    e = lambda n, dt: torch.empty(n, dtype=dt, device=dev)
    T_g = traj_id.size
    ins = (t(traj_id), t(mask), t(traj_task), t(traj_group), t(reward))
    outs = (e(n_traj, torch.int32), e(n_task, torch.int64), e(n_task, torch.float32),
            e(n_task, torch.float32), e(n_traj, torch.float32), e(T_g, torch.float32))
    scratch = e(2 * (n_group + n_task), torch.int32)
    for ranges in (True, False):
        _assert_bitwise(_gpu(*args, ranges=ranges), r)
        opt = P.agrl_options(adv_ranges=scratch.data_ptr() if ranges else None)
        call = lambda: P.agrl_task_adv_norm(T_g, n_traj, n_task, n_group, *ins, opt, *outs)
        call()                                                    # warm-up
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(5):
            call()
        e1.record()
        torch.cuda.synchronize()
        log(f"adv_norm {n_group} groups, {n_traj} trajectories, T_g={T_g}, "
            f"member ranges {ranges}: {e0.elapsed_time(e1) / 5 * 1e3:.1f} us per call")
