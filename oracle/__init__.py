"""CPU reference ("oracle") for the fused policy-loss path -- test infrastructure.

Only the tests, the smoke check and the benchmark's CPU-baseline leg may use
this package.  It shares no code with the HIP library and never imports it.
The arithmetic lives in ``agrl_oracle.c`` (plain C: fp32 advantage
normalisation in a fixed summation order, fp64 loss and gradients); this file
only compiles it with gcc and marshals numpy arrays through ctypes.  The one
exception is ``blas.py``: the same fp64 forward with the logits from a library
matmul, for whole batches at the full workload sizes.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_DIR = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_DIR, "agrl_oracle.c")
_LIB = os.path.join(_DIR, "liboracle.so")
_lib = None


def build(force: bool = True) -> str:
    """Compile the oracle (gcc, strict IEEE: no FMA contraction, no fast-math)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-std=c11", "-ffp-contract=off", "-fno-fast-math",
                               "-fPIC", "-shared", "-pthread", _SRC, "-o", tmp, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        build(force=False)
        _lib = ctypes.CDLL(_LIB)
    return _lib


def _p(a):
    return a.ctypes.data_as(ctypes.c_void_p) if a is not None else None


def _threads(n):
    if n:
        return int(n)
    return max(1, min(16, len(os.sched_getaffinity(0))))


def _as_input(x):
    """numpy view of a torch/numpy matrix: (array, is_bf16)."""
    try:
        import torch
        if isinstance(x, torch.Tensor):
            x = x.detach().cpu().contiguous()
            if x.dtype == torch.bfloat16:
                return x.view(torch.int16).numpy().view(np.uint16), 1
            return x.float().numpy(), 0
    except ImportError:  # pragma: no cover
        pass
    x = np.ascontiguousarray(x)
    if x.dtype == np.uint16:
        return x, 1
    return np.ascontiguousarray(x, np.float32), 0


def task_adv_norm(traj_id, mask, traj_task, traj_group, reward, n_task, n_group=0, ddof=0,
                  eps=1e-6, drop_uniform=False):
    """Group stage (GRPO, App. B.2) then task stage (Sec. 3.2) in fp32 with the
    fixed summation order; drop_uniform drops GRPO groups whose rewards are all
    equal (DAPO dynamic sampling, App. A)."""
    lib = _load()
    traj_id = np.ascontiguousarray(traj_id, np.int32)
    mask = np.ascontiguousarray(mask, np.uint8)
    traj_task = np.ascontiguousarray(traj_task, np.int32)
    reward = np.ascontiguousarray(reward, np.float32)
    if traj_group is not None:
        traj_group = np.ascontiguousarray(traj_group, np.int32)
    T_g, n_traj = traj_id.shape[0], traj_task.shape[0]
    out = dict(act_count=np.zeros(n_traj, np.int32), task_count=np.zeros(n_task, np.int64),
               task_mean=np.zeros(n_task, np.float32), task_std=np.zeros(n_task, np.float32),
               adv_traj=np.zeros(n_traj, np.float32), adv_tok=np.zeros(T_g, np.float32))
    f = lib.oracle_task_adv_norm_ext
    f.restype = ctypes.c_int
    rc = f(ctypes.c_int64(T_g), ctypes.c_int32(n_traj), ctypes.c_int32(n_task),
           ctypes.c_int32(n_group), _p(traj_id), _p(mask), _p(traj_task), _p(traj_group),
           _p(reward), ctypes.c_int32(ddof), ctypes.c_float(eps), ctypes.c_int32(int(drop_uniform)),
           _p(out["act_count"]), _p(out["task_count"]), _p(out["task_mean"]), _p(out["task_std"]),
           _p(out["adv_traj"]), _p(out["adv_tok"]))
    if rc == -2:
        raise ValueError("oracle_task_adv_norm: drop_uniform needs groups")
    if rc != 0:
        raise ValueError("oracle_task_adv_norm: id out of range")
    return out


def sequence_mean_weights(traj_id, mask, n_traj):
    """Per-token weights of the sequence-level aggregation (App. B.2, GRPO's mean
    over responses of per-response token means) for one micro-batch: returns
    (count [n_traj] int32, weights [T] fp32)."""
    lib = _load()
    traj_id = np.ascontiguousarray(traj_id, np.int32)
    mask = np.ascontiguousarray(mask, np.uint8)
    T = traj_id.shape[0]
    count = np.zeros(n_traj, np.int32)
    w = np.zeros(T, np.float32)
    f = lib.oracle_sequence_mean_weights
    f.restype = ctypes.c_int
    rc = f(ctypes.c_int64(T), ctypes.c_int32(n_traj), _p(traj_id), _p(mask), _p(count), _p(w))
    if rc != 0:
        raise ValueError("oracle_sequence_mean_weights: trajectory id out of range")
    return count, w


def policy_loss(H, W, token_id, mask, adv, old_logp, eps_lo=0.2, eps_hi=0.2, n_norm=0,
                temperature=1.0, grad_loss=1.0, backward=True, nthreads=None, kl_beta=0.0,
                kl_estimator=0, ref_logp=None, token_weight=None):
    """Whole-batch forward (+ backward): logp, lse, loss, n_clip, g, dH, dW (fp64).

    kl_beta / kl_estimator / ref_logp subtract beta * KL(pi || pi_ref) per token
    (App. A objectives; estimator 0 = k3, 1 = k1); token_weight replaces the
    1 / N token mean by per-token weights."""
    lib = _load()
    Hn, hb = _as_input(H)
    Wn, wb = _as_input(W)
    assert hb == wb
    T, d = Hn.shape
    V = Wn.shape[0]
    y = np.ascontiguousarray(token_id, np.int32)
    m = np.ascontiguousarray(mask, np.uint8)
    a = np.ascontiguousarray(adv, np.float32)
    o = np.ascontiguousarray(old_logp, np.float32)
    logp, lse, g = np.zeros(T), np.zeros(T), np.zeros(T)
    loss = np.zeros(1)
    n_clip = np.zeros(2, np.int64)
    dH = np.zeros((T, d)) if backward else None
    dW = np.zeros((V, d)) if backward else None
    ref = None if ref_logp is None else np.ascontiguousarray(ref_logp, np.float32)
    tw = None if token_weight is None else np.ascontiguousarray(token_weight, np.float32)
    f = lib.oracle_policy_loss_ext
    f.restype = ctypes.c_int
    rc = f(ctypes.c_int64(T), ctypes.c_int32(d), ctypes.c_int32(V), ctypes.c_int32(hb),
           _p(Hn), _p(Wn), _p(y), _p(m), _p(a), _p(o), ctypes.c_double(eps_lo),
           ctypes.c_double(eps_hi), ctypes.c_int64(n_norm), ctypes.c_double(temperature),
           ctypes.c_double(grad_loss), ctypes.c_double(kl_beta), ctypes.c_int(kl_estimator),
           _p(ref), _p(tw), ctypes.c_int(_threads(nthreads)), _p(logp), _p(lse),
           _p(loss), _p(n_clip), _p(g), _p(dH), _p(dW))
    if rc == -2:
        raise ValueError("oracle_policy_loss: kl_beta != 0 needs ref_logp")
    if rc != 0:
        raise ValueError("oracle_policy_loss: token id out of range")
    return dict(logp=logp, lse=lse, loss=float(loss[0]), n_clip=n_clip, g=g, dH=dH, dW=dW)


def token_logprob(H, W, token_id, mask, temperature=1.0, nthreads=None):
    """log pi(y_t | s_t) and the log-sum-exp of the logits of every action token
    (App. B.1 token log-probability), 0 elsewhere: the policy-loss forward's
    logp and lse, which do not depend on advantages or old log-probs."""
    T = np.asarray(mask).shape[0]
    r = policy_loss(H, W, token_id, mask, np.zeros(T, np.float32), np.zeros(T, np.float32),
                    temperature=temperature, backward=False, nthreads=nthreads)
    return dict(logp=r["logp"], lse=r["lse"])


def token_sample(H, W, token_id, mask, adv, old_logp, tokens, eps_lo=0.2, eps_hi=0.2, n_norm=0,
                 temperature=1.0, grad_loss=1.0, dH=True, nthreads=None):
    """lse, logp, g and (optionally) the dH row for the listed token positions only."""
    lib = _load()
    Hn, hb = _as_input(H)
    Wn, wb = _as_input(W)
    assert hb == wb
    T, d = Hn.shape
    V = Wn.shape[0]
    tok = np.ascontiguousarray(tokens, np.int64)
    k = tok.shape[0]
    lse, logp, g = np.zeros(k), np.zeros(k), np.zeros(k)
    out_dH = np.zeros((k, d)) if dH else None
    f = lib.oracle_token_sample
    f.restype = ctypes.c_int
    rc = f(ctypes.c_int64(T), ctypes.c_int32(d), ctypes.c_int32(V), ctypes.c_int32(hb),
           _p(Hn), _p(Wn), _p(np.ascontiguousarray(token_id, np.int32)),
           _p(np.ascontiguousarray(mask, np.uint8)), _p(np.ascontiguousarray(adv, np.float32)),
           _p(np.ascontiguousarray(old_logp, np.float32)), ctypes.c_double(eps_lo),
           ctypes.c_double(eps_hi), ctypes.c_int64(n_norm), ctypes.c_double(temperature),
           ctypes.c_double(grad_loss), ctypes.c_int(_threads(nthreads)), _p(tok), ctypes.c_int64(k),
           _p(lse), _p(logp), _p(g), _p(out_dH))
    if rc != 0:
        raise ValueError("oracle_token_sample: bad token index or id")
    return dict(lse=lse, logp=logp, g=g, dH=out_dH)


def token_logprob_full(H, W, token_id, mask, temperature=1.0):
    """fp64 logp and lse of every action token at any size (library matmul for
    the logits; same definition as policy_loss's forward, App. B.1)."""
    from .blas import token_logprob_fp64
    logp, lse = token_logprob_fp64(H, W, token_id, mask, temperature=temperature)
    return dict(logp=logp, lse=lse)


def surrogate_terms(mask, adv, old_logp, logp, eps_lo=0.2, eps_hi=0.2, n_norm=0, grad_loss=1.0):
    """Loss, clip counts and g = dL/dlogp of a micro-batch from fp64 log-probs of
    its action tokens (App. B.2 PPO surrogate, App. A token-level mean)."""
    lib = _load()
    m = np.ascontiguousarray(mask, np.uint8)
    T = m.shape[0]
    loss = np.zeros(1)
    n_clip = np.zeros(2, np.int64)
    g = np.zeros(T)
    f = lib.oracle_surrogate_terms
    f.restype = ctypes.c_int
    f(ctypes.c_int64(T), _p(m), _p(np.ascontiguousarray(adv, np.float32)),
      _p(np.ascontiguousarray(old_logp, np.float32)), _p(np.ascontiguousarray(logp, np.float64)),
      ctypes.c_double(eps_lo), ctypes.c_double(eps_hi), ctypes.c_int64(n_norm),
      ctypes.c_double(grad_loss), _p(loss), _p(n_clip), _p(g))
    return dict(loss=float(loss[0]), n_clip=n_clip, g=g)


def dw_rows(H, W, token_id, mask, lse, g, rows, temperature=1.0, nthreads=None):
    """Rows of dW = G^T H for the listed vocabulary entries, from every action
    token's lse and dL/dlogp: fp64 [len(rows), d]."""
    lib = _load()
    Hn, hb = _as_input(H)
    Wn, wb = _as_input(W)
    assert hb == wb
    T, d = Hn.shape
    V = Wn.shape[0]
    r = np.ascontiguousarray(rows, np.int64)
    out = np.zeros((r.shape[0], d))
    f = lib.oracle_dw_rows
    f.restype = ctypes.c_int
    rc = f(ctypes.c_int64(T), ctypes.c_int32(d), ctypes.c_int32(V), ctypes.c_int32(hb), _p(Hn),
           _p(Wn), _p(np.ascontiguousarray(token_id, np.int32)),
           _p(np.ascontiguousarray(mask, np.uint8)), ctypes.c_double(temperature),
           _p(np.ascontiguousarray(lse, np.float64)), _p(np.ascontiguousarray(g, np.float64)),
           _p(r), ctypes.c_int64(r.shape[0]), ctypes.c_int(_threads(nthreads)), _p(out))
    if rc != 0:
        raise ValueError("oracle_dw_rows: row or token id out of range")
    return out
