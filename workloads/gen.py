"""Seeded synthetic workloads for the fused policy-loss path.

This module builds inputs only.  It holds none of the method's arithmetic:
no advantage statistics, no log-softmax of the trained policy, no surrogate,
no gradients.  Both the CPU oracle (``oracle/``) and the HIP library are fed
from the same arrays produced here.

What is generated (paper, App. B.1 "Problem Definition"; Sec. 3.2):

* A global batch of trajectories organised as task -> sample (group) ->
  trajectory.  Each trajectory is a sequence of turns; a turn is an
  environment observation (masked out, ``mask == 0``) followed by the model's
  action tokens (``mask == 1``).  One scalar reward per trajectory.
* The global token stream is the trajectories concatenated in a seeded
  permutation.  The packed micro-batch the loss runs on is the first
  ``T_pack`` tokens of that stream (the last trajectory is truncated), so the
  micro-batch's per-token advantages are a prefix of the global ones.
* Hidden states ``H ~ N(0, 1)`` and LM head ``W ~ N(0, 0.02^2)``, rounded to
  bf16 (round-to-nearest-even) except for the fp32 workload.
* Rollout data: the sampled token ``y`` and the behaviour policy's log-prob
  ``old_logp``.  These are what an inference engine hands the trainer; the
  stand-in engine here samples ``y`` from the softmax of ``H W^T`` by inverse
  CDF with pre-drawn uniforms and reports its fp32 log-prob plus Gaussian
  noise (so ratios sit near 1 and some reach the clip bounds).  This is the
  only place a logit is formed in this module; it plays the rollout engine,
  not the trainer, and it runs in torch fp32 (on the GPU when one is given),
  never through the library under test.

Random streams: numpy PCG64 ``default_rng([seed, stream])`` for structure,
rewards, sampling uniforms and noise; torch generators seeded from ``seed``
for the large ``H`` and ``W`` (on the target device, so a GPU run draws them
there instead of copying gigabytes from the host).
"""
from __future__ import annotations

import dataclasses
from typing import Callable, List, Optional, Sequence, Tuple

import numpy as np
import torch

# numpy stream numbers
_S_STRUCT, _S_REWARD, _S_UNIF, _S_NOISE, _S_PERM = 0, 1, 2, 3, 4
BASE_SEED = 20251004


@dataclasses.dataclass
class TaskSpec:
    n_groups: int
    group_size: int
    # reward sampler: (rng, n) -> float32[n]
    reward: Callable[[np.random.Generator, int], np.ndarray]


@dataclasses.dataclass
class WorkloadSpec:
    name: str
    V: int
    d: int
    dtype: str                      # "f32" or "bf16"
    tasks: List[TaskSpec]
    turns: Tuple[int, int]          # inclusive range of turns per trajectory
    obs: Tuple[int, int]            # inclusive range of observation tokens per turn
    act: Tuple[int, int]            # inclusive range of action tokens per turn
    noise_std: float                # old_logp = rollout logp + N(0, noise_std^2)
    T_pack: Optional[int]           # micro-batch length; None = the whole stream
    eps_lo: float = 0.2
    eps_hi: float = 0.2
    h_std: float = 1.0
    w_std: float = 0.02


@dataclasses.dataclass
class Workload:
    spec: WorkloadSpec
    seed: int
    # global batch (advantage normalisation runs here)
    n_traj: int
    n_task: int
    n_group: int
    traj_task: np.ndarray           # int32[n_traj]
    traj_group: np.ndarray          # int32[n_traj]
    reward: np.ndarray              # float32[n_traj]
    g_traj_id: np.ndarray           # int32[T_g]
    g_mask: np.ndarray              # uint8[T_g]
    # packed micro-batch = the first T tokens of the global stream
    T: int
    H: Optional[torch.Tensor] = None        # [T, d] bf16/f32
    W: Optional[torch.Tensor] = None        # [V, d] bf16/f32
    token_id: Optional[np.ndarray] = None   # int32[T]
    old_logp: Optional[np.ndarray] = None   # float32[T] (0 on observation tokens)

    @property
    def T_g(self) -> int:
        return int(self.g_traj_id.shape[0])

    @property
    def traj_id(self) -> np.ndarray:
        return self.g_traj_id[: self.T]

    @property
    def mask(self) -> np.ndarray:
        return self.g_mask[: self.T]

    @property
    def n_act(self) -> int:
        return int(self.mask.sum())

    @property
    def V(self) -> int:
        return self.spec.V

    @property
    def d(self) -> int:
        return self.spec.d


# ----------------------------------------------------------------------------
# reward distributions
def bernoulli(p: float):
    return lambda rng, n: (rng.random(n) < p).astype(np.float32)


def uniform01():
    return lambda rng, n: rng.random(n).astype(np.float32)


def normal(mu: float, sd: float):
    return lambda rng, n: rng.normal(mu, sd, n).astype(np.float32)


def constant(c: float):
    return lambda rng, n: np.full(n, c, dtype=np.float32)


# ----------------------------------------------------------------------------
# the five workloads
def config_spec(k: int) -> WorkloadSpec:
    """Workload k in 1..5 (tiny fp32; 7B-, 32B-shaped; long-horizon; 256k vocab)."""
    rng = np.random.default_rng([BASE_SEED + k, 99])   # task-level parameters
    if k == 1:
        tasks = [TaskSpec(4, 4, bernoulli(0.5)) for _ in range(2)]
        return WorkloadSpec("tiny-fp32 V4096 d256", 4096, 256, "f32", tasks,
                            (3, 3), (24, 24), (8, 24), 0.05, None)
    if k == 2:
        ps = rng.uniform(0.1, 0.9, 5)
        tasks = [TaskSpec(16, 8, bernoulli(float(p))) for p in ps]
        return WorkloadSpec("7B-shaped V152064 d3584 T32768", 152064, 3584, "bf16", tasks,
                            (4, 12), (64, 512), (32, 256), 0.1, 32768)
    if k == 3:
        tasks = [TaskSpec(n, 8, uniform01()) for n in (40, 20, 10, 5, 5)]
        return WorkloadSpec("32B-shaped V152064 d5120 T65536", 152064, 5120, "bf16", tasks,
                            (4, 12), (64, 512), (32, 256), 0.2, 65536)
    if k == 4:
        tasks = [TaskSpec(n, 8, bernoulli(0.3)) for n in (7, 7, 6, 6, 6)]
        return WorkloadSpec("long-horizon V152064 d5120 T131072", 152064, 5120, "bf16", tasks,
                            (30, 50), (128, 1024), (16, 128), 0.1, 131072)
    if k == 5:
        tasks = []
        ps = rng.uniform(0.0, 1.0, 10)
        ps[0], ps[1] = 0.0, 1.0             # two tasks whose rewards are all equal
        for p in ps:
            tasks.append(TaskSpec(32, 4, bernoulli(float(p))))
        mus = rng.normal(0.0, np.sqrt(2.0), 10)
        for mu in mus:
            tasks.append(TaskSpec(32, 4, normal(float(mu), 1.0)))
        return WorkloadSpec("large-vocab V256000 d4096 T65536 20 tasks", 256000, 4096, "bf16",
                            tasks, (4, 12), (64, 512), (32, 256), 0.1, 65536)
    raise ValueError(f"no workload {k}")


def config_seed(k: int) -> int:
    return BASE_SEED + k


# ----------------------------------------------------------------------------
def build_structure(spec: WorkloadSpec, seed: int) -> Workload:
    """Trajectory layout, rewards and the global/micro-batch token streams."""
    rs = np.random.default_rng([seed, _S_STRUCT])
    rr = np.random.default_rng([seed, _S_REWARD])
    traj_task, traj_group, rewards, lengths = [], [], [], []
    pieces = []          # per trajectory: mask array
    g = 0
    for ti, task in enumerate(spec.tasks):
        for _ in range(task.n_groups):
            r = task.reward(rr, task.group_size)
            for j in range(task.group_size):
                n_turns = int(rs.integers(spec.turns[0], spec.turns[1] + 1))
                obs = rs.integers(spec.obs[0], spec.obs[1] + 1, n_turns)
                act = rs.integers(spec.act[0], spec.act[1] + 1, n_turns)
                m = np.concatenate([np.concatenate([np.zeros(o, np.uint8), np.ones(a, np.uint8)])
                                    for o, a in zip(obs, act)])
                pieces.append(m)
                traj_task.append(ti)
                traj_group.append(g)
                rewards.append(r[j])
            g += 1
    n_traj = len(pieces)
    perm = np.random.default_rng([seed, _S_PERM]).permutation(n_traj)
    g_mask = np.concatenate([pieces[p] for p in perm]).astype(np.uint8)
    g_traj = np.concatenate([np.full(pieces[p].shape[0], p, np.int32) for p in perm])
    T = g_mask.shape[0] if spec.T_pack is None else min(spec.T_pack, g_mask.shape[0])
    return Workload(spec=spec, seed=seed, n_traj=n_traj, n_task=len(spec.tasks), n_group=g,
                    traj_task=np.asarray(traj_task, np.int32),
                    traj_group=np.asarray(traj_group, np.int32),
                    reward=np.asarray(rewards, np.float32),
                    g_traj_id=g_traj, g_mask=g_mask, T=int(T))


def _randn(shape, std, seed, device, dtype):
    gen = torch.Generator(device=device).manual_seed(int(seed))
    x = torch.randn(shape, generator=gen, device=device, dtype=torch.float32)
    if std != 1.0:
        x.mul_(std)
    if dtype == "bf16":
        x = x.to(torch.bfloat16)          # round-to-nearest-even
    return x


def rollout_standin(H: torch.Tensor, W: torch.Tensor, mask: np.ndarray, unif: np.ndarray,
                    noise: np.ndarray, chunk: int = 2048) -> Tuple[np.ndarray, np.ndarray]:
    """The inference engine's side of the data: sampled ids and their log-probs.

    Samples y_t ~ softmax(h_t W^T) by inverse CDF on action tokens (fp32 on
    the tensors' device) and reports old_logp = logp_rollout + noise.
    Observation tokens get a uniform id and old_logp 0; they are never read.
    """
    T = H.shape[0]
    V = W.shape[0]
    dev = H.device
    y = np.floor(unif * V).astype(np.int64).clip(0, V - 1).astype(np.int32)
    old = np.zeros(T, np.float32)
    act = np.nonzero(mask)[0]
    Wf = W.float()
    u_all = torch.from_numpy(unif.astype(np.float64)).to(dev)
    for s in range(0, act.shape[0], chunk):
        rows = torch.from_numpy(act[s:s + chunk]).to(dev)
        z = H.index_select(0, rows).float() @ Wf.t()
        lp = torch.log_softmax(z, dim=1)
        cdf = torch.cumsum(lp.exp().double(), dim=1)
        u = u_all.index_select(0, rows) * cdf[:, -1]
        idx = torch.searchsorted(cdf, u.unsqueeze(1)).clamp_(max=V - 1)
        lp_y = lp.gather(1, idx).squeeze(1)
        y[act[s:s + chunk]] = idx.squeeze(1).to(torch.int32).cpu().numpy()
        old[act[s:s + chunk]] = lp_y.cpu().numpy()
        del z, lp, cdf
    old[act] = (old[act].astype(np.float64) + noise[act]).astype(np.float32)
    return y, old


def build_tensors(w: Workload, device="cpu") -> Workload:
    """Draw H, W on ``device`` and the rollout data (ids, old_logp)."""
    spec = w.spec
    dev = torch.device(device)
    w.H = _randn((w.T, spec.d), spec.h_std, w.seed * 2 + 1, dev, spec.dtype)
    w.W = _randn((spec.V, spec.d), spec.w_std, w.seed * 2 + 2, dev, spec.dtype)
    unif = np.random.default_rng([w.seed, _S_UNIF]).random(w.T)
    noise = np.random.default_rng([w.seed, _S_NOISE]).normal(0.0, spec.noise_std, w.T)
    w.token_id, w.old_logp = rollout_standin(w.H, w.W, w.mask, unif, noise)
    return w


def make(spec: WorkloadSpec, seed: int, device="cpu", tensors: bool = True) -> Workload:
    w = build_structure(spec, seed)
    if tensors:
        build_tensors(w, device)
    return w


def config(k: int, device="cpu", tensors: bool = True) -> Workload:
    return make(config_spec(k), config_seed(k), device, tensors)


def small_spec(V: int, d: int, dtype: str = "bf16", n_tasks: int = 3, n_groups: int = 2,
               group_size: int = 4, turns=(2, 4), obs=(5, 40), act=(3, 30),
               noise_std: float = 0.2, T_pack: Optional[int] = None,
               rewards: Optional[Sequence] = None, name: str = "small") -> WorkloadSpec:
    """A reduced workload of the same structure, for parity at oracle-friendly sizes."""
    if rewards is None:
        rewards = [uniform01() if i % 2 else bernoulli(0.5) for i in range(n_tasks)]
    tasks = [TaskSpec(n_groups, group_size, rewards[i % len(rewards)]) for i in range(n_tasks)]
    return WorkloadSpec(name, V, d, dtype, tasks, turns, obs, act, noise_std, T_pack)
