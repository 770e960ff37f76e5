"""ctypes binding of libagrl.so: the C ABI of include/agrl.h, same names.

Argument marshalling only.  Tensors must already be on the GPU with the
documented dtypes and layouts; every computation runs in the library's HIP
kernels.  There is no fallback: if the library is missing or a call fails,
an exception is raised.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libagrl.so")

AGRL_BF16 = 0
AGRL_F32 = 1
AGRL_NOALLOC_SCRATCH_BYTES = 64 << 20     # include/agrl.h
ERROR_BITS = {1: "token id out of range", 2: "trajectory id out of range",
              4: "task id out of range", 8: "group id out of range",
              16: "more action tokens than max_act"}

_c_i64, _c_i32, _c_f32, _c_p, _c_sz = (ctypes.c_int64, ctypes.c_int32, ctypes.c_float,
                                       ctypes.c_void_p, ctypes.c_size_t)


class agrl_options(ctypes.Structure):
    _fields_ = [("std_ddof", ctypes.c_int32), ("std_eps", ctypes.c_float),
                ("temperature", ctypes.c_float), ("dw_accumulate", ctypes.c_int32),
                ("g_chunk_bytes", ctypes.c_int64), ("phase_events", ctypes.c_void_p),
                ("kl_beta", ctypes.c_float), ("kl_estimator", ctypes.c_int32),
                ("ref_logp", ctypes.c_void_p), ("token_weight", ctypes.c_void_p),
                ("drop_uniform_groups", ctypes.c_int32), ("adv_ranges", ctypes.c_void_p)]


class AgrlError(RuntimeError):
    def __init__(self, fn: str, status: int, msg: str):
        super().__init__(f"{fn} failed with status {status}: {msg}")
        self.status = status


_lib = None

_SIGS = {
    "agrl_task_adv_norm": (_c_i32, [_c_i64, _c_i32, _c_i32, _c_i32, _c_p, _c_p, _c_p, _c_p, _c_p,
                                    _c_p, _c_p, _c_p, _c_p, _c_p, _c_p, _c_p, _c_p]),
    "agrl_policy_loss_workspace_size": (_c_sz, [_c_i64, _c_i64, _c_i32, _c_i32, _c_i32, _c_p]),
    "agrl_policy_loss_vocab_chunk": (_c_i64, [_c_i64, _c_i64, _c_i32, _c_i32, _c_i32, _c_p]),
    "agrl_policy_loss_fwd": (_c_i32, [_c_i64, _c_i64, _c_i32, _c_i32, _c_i32, _c_p, _c_p, _c_p,
                                      _c_p, _c_p, _c_p, _c_f32, _c_f32, _c_i64, _c_p, _c_p, _c_sz,
                                      _c_p, _c_p, _c_p, _c_p, _c_p]),
    "agrl_policy_loss_bwd": (_c_i32, [_c_i64, _c_i64, _c_i32, _c_i32, _c_i32, _c_p, _c_p, _c_p,
                                      _c_p, _c_p, _c_p, _c_f32, _c_f32, _c_i64, _c_p, _c_p, _c_p,
                                      _c_f32, _c_p, _c_sz, _c_p, _c_p, _c_p]),
    "agrl_token_logprob_workspace_size": (_c_sz, [_c_i64, _c_i64, _c_i32, _c_i32, _c_i32, _c_p]),
    "agrl_token_logprob": (_c_i32, [_c_i64, _c_i64, _c_i32, _c_i32, _c_i32, _c_p, _c_p, _c_p, _c_p,
                                    _c_p, _c_p, _c_sz, _c_p, _c_p, _c_p]),
    "agrl_token_logprob_noalloc": (_c_i32, [_c_i64, _c_i64, _c_i32, _c_i32, _c_i32, _c_p, _c_p,
                                            _c_p, _c_p, _c_p, _c_p, _c_p, _c_p]),
    "agrl_sequence_mean_weights": (_c_i32, [_c_i64, _c_i32, _c_p, _c_p, _c_p, _c_p, _c_p]),
    "agrl_status_string": (ctypes.c_char_p, [_c_i32]),
    "agrl_last_error": (ctypes.c_char_p, []),
    "agrl_get_device_error": (_c_i32, [_c_p, _c_p]),
}


def lib():
    """Load libagrl.so (built by paper_2510_04206_amd.build); raise if it is missing."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is not built; run paper_2510_04206_amd.build.build()")
        L = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGS.items():
            f = getattr(L, name)
            f.restype = res
            f.argtypes = args
        _lib = L
    return _lib


def exported_symbols():
    return list(_SIGS)


def _ptr(t: Optional[torch.Tensor]):
    """Device address of a contiguous GPU tensor (the ABI takes plain pointers)."""
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError("agrl: arrays must be GPU tensors (the ABI takes device pointers)")
    if not t.is_contiguous():
        raise ValueError("agrl: arrays must be contiguous (the ABI takes plain pointers)")
    return ctypes.c_void_p(t.data_ptr())


def _stream(stream) -> ctypes.c_void_p:
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def _check(fn: str, rc: int) -> None:
    if rc != 0:
        L = lib()
        raise AgrlError(fn, rc, (L.agrl_last_error() or b"").decode() or
                        L.agrl_status_string(rc).decode())


def _opts(opt) -> Optional[ctypes.POINTER(agrl_options)]:
    if opt is None:
        return None
    if isinstance(opt, dict):
        opt = agrl_options(**opt)
    return ctypes.byref(opt)


def dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.bfloat16:
        return AGRL_BF16
    if t.dtype == torch.float32:
        return AGRL_F32
    raise TypeError(f"unsupported dtype {t.dtype}")


def agrl_task_adv_norm(T_g, n_traj, n_task, n_group, traj_id, action_mask, traj_task, traj_group,
                       reward, opt, act_count, task_count, task_mean, task_std, adv_traj,
                       adv_tok, stream=None) -> None:
    _check("agrl_task_adv_norm", lib().agrl_task_adv_norm(
        T_g, n_traj, n_task, n_group, _ptr(traj_id), _ptr(action_mask), _ptr(traj_task),
        _ptr(traj_group), _ptr(reward), _opts(opt), _ptr(act_count), _ptr(task_count),
        _ptr(task_mean), _ptr(task_std), _ptr(adv_traj), _ptr(adv_tok), _stream(stream)))


def agrl_policy_loss_workspace_size(T, max_act, d, V, dtype, opt=None) -> int:
    return int(lib().agrl_policy_loss_workspace_size(T, max_act, d, V, dtype, _opts(opt)))


def agrl_policy_loss_vocab_chunk(T, max_act, d, V, dtype, opt=None) -> int:
    return int(lib().agrl_policy_loss_vocab_chunk(T, max_act, d, V, dtype, _opts(opt)))


def agrl_policy_loss_fwd(T, max_act, d, V, dtype, H, W, token_id, action_mask, adv_tok, old_logp,
                         clip_eps_low, clip_eps_high, n_norm, opt, workspace, ws_bytes, loss,
                         logp, lse, n_clip, stream=None) -> None:
    _check("agrl_policy_loss_fwd", lib().agrl_policy_loss_fwd(
        T, max_act, d, V, dtype, _ptr(H), _ptr(W), _ptr(token_id), _ptr(action_mask),
        _ptr(adv_tok), _ptr(old_logp), clip_eps_low, clip_eps_high, n_norm, _opts(opt),
        _ptr(workspace), ws_bytes, _ptr(loss), _ptr(logp), _ptr(lse), _ptr(n_clip),
        _stream(stream)))


def agrl_policy_loss_bwd(T, max_act, d, V, dtype, H, W, token_id, action_mask, adv_tok, old_logp,
                         clip_eps_low, clip_eps_high, n_norm, opt, lse, logp, grad_loss,
                         workspace, ws_bytes, dH, dW, stream=None) -> None:
    _check("agrl_policy_loss_bwd", lib().agrl_policy_loss_bwd(
        T, max_act, d, V, dtype, _ptr(H), _ptr(W), _ptr(token_id), _ptr(action_mask),
        _ptr(adv_tok), _ptr(old_logp), clip_eps_low, clip_eps_high, n_norm, _opts(opt),
        _ptr(lse), _ptr(logp), grad_loss, _ptr(workspace), ws_bytes, _ptr(dH), _ptr(dW),
        _stream(stream)))


def agrl_token_logprob_workspace_size(T, max_act, d, V, dtype, opt=None) -> int:
    return int(lib().agrl_token_logprob_workspace_size(T, max_act, d, V, dtype, _opts(opt)))


def agrl_token_logprob(T, max_act, d, V, dtype, H, W, token_id, action_mask, opt, workspace,
                       ws_bytes, logp, lse, stream=None) -> None:
    _check("agrl_token_logprob", lib().agrl_token_logprob(
        T, max_act, d, V, dtype, _ptr(H), _ptr(W), _ptr(token_id), _ptr(action_mask), _opts(opt),
        _ptr(workspace), ws_bytes, _ptr(logp), _ptr(lse), _stream(stream)))


def agrl_token_logprob_noalloc(T, max_act, d, V, dtype, H, W, token_id, action_mask, opt, logp,
                               lse, stream=None) -> None:
    _check("agrl_token_logprob_noalloc", lib().agrl_token_logprob_noalloc(
        T, max_act, d, V, dtype, _ptr(H), _ptr(W), _ptr(token_id), _ptr(action_mask), _opts(opt),
        _ptr(logp), _ptr(lse), _stream(stream)))


def agrl_sequence_mean_weights(T, n_traj, traj_id, action_mask, seq_count, token_weight,
                               stream=None) -> None:
    _check("agrl_sequence_mean_weights", lib().agrl_sequence_mean_weights(
        T, n_traj, _ptr(traj_id), _ptr(action_mask), _ptr(seq_count), _ptr(token_weight),
        _stream(stream)))


def agrl_get_device_error(stream=None) -> int:
    code = ctypes.c_int32(0)
    _check("agrl_get_device_error", lib().agrl_get_device_error(_stream(stream),
                                                                ctypes.byref(code)))
    return int(code.value)
