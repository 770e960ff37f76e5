"""The C ABI library on the CPU: it loads, exports every declared symbol, and
rejects bad arguments synchronously (before any HIP call, so no GPU is needed)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "agrl.h")

E_NULL, E_SHAPE, E_DTYPE, E_FLAGS, E_WS, E_HIP, E_UNSUP = -1, -2, -3, -4, -5, -6, -7


def _declared():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(agrl_\w+)\s*\(", src)))


@pytest.fixture(scope="module")
def L():
    from paper_2510_04206_amd import _binding
    return _binding.lib()


def test_exports_every_declared_symbol(L):
    names = _declared()
    assert {"agrl_task_adv_norm", "agrl_policy_loss_fwd", "agrl_policy_loss_bwd",
            "agrl_policy_loss_workspace_size"} <= set(names)
    for n in names:
        assert hasattr(L, n), n
    from paper_2510_04206_amd import _binding
    assert set(_binding.exported_symbols()) == set(names)


def test_status_strings(L):
    for code in (0, E_NULL, E_SHAPE, E_DTYPE, E_FLAGS, E_WS, E_HIP, E_UNSUP):
        assert L.agrl_status_string(code)
    assert L.agrl_status_string(12345) == b"unknown status"


def _fwd(L, **kw):
    a = dict(T=100, max_act=0, d=64, V=50, dt=0, H=1 << 12, W=1 << 12, ids=1 << 12, m=1 << 12,
             adv=1 << 12, old=1 << 12, lo=0.2, hi=0.2, n_norm=0, opt=None, ws=None, wsb=0,
             loss=1 << 12, logp=1 << 12, lse=1 << 12, ncl=None)
    a.update(kw)
    return L.agrl_policy_loss_fwd(a["T"], a["max_act"], a["d"], a["V"], a["dt"], a["H"], a["W"],
                                  a["ids"], a["m"], a["adv"], a["old"], a["lo"], a["hi"],
                                  a["n_norm"], a["opt"], a["ws"], a["wsb"], a["loss"], a["logp"],
                                  a["lse"], a["ncl"], None)


def test_forward_argument_errors(L):
    from paper_2510_04206_amd._binding import agrl_options
    assert _fwd(L, dt=7) == E_DTYPE
    assert _fwd(L, T=-1) == E_SHAPE
    assert _fwd(L, d=0) == E_SHAPE
    assert _fwd(L, V=0) == E_SHAPE
    assert _fwd(L, d=100) == E_UNSUP
    assert _fwd(L, lo=1.0) == E_FLAGS
    assert _fwd(L, lo=-0.1) == E_FLAGS
    assert _fwd(L, hi=float("inf")) == E_FLAGS
    assert _fwd(L, hi=float("nan")) == E_FLAGS
    assert _fwd(L, n_norm=-3) == E_SHAPE
    assert _fwd(L, H=None) == E_NULL
    assert _fwd(L, W=None) == E_NULL
    assert _fwd(L, ws=None) == E_WS
    assert b"workspace" in L.agrl_last_error()
    o = agrl_options(temperature=-1.0)
    assert _fwd(L, opt=ctypes.byref(o)) == E_FLAGS
    o = agrl_options(dw_accumulate=2)
    assert _fwd(L, opt=ctypes.byref(o)) == E_FLAGS
    o = agrl_options(kl_beta=0.1)                       # KL without a reference
    assert _fwd(L, opt=ctypes.byref(o)) == E_NULL
    o = agrl_options(kl_beta=float("inf"), ref_logp=1 << 12)
    assert _fwd(L, opt=ctypes.byref(o)) == E_FLAGS
    o = agrl_options(kl_beta=0.1, kl_estimator=2, ref_logp=1 << 12)
    assert _fwd(L, opt=ctypes.byref(o)) == E_FLAGS
    # a workspace that is one byte short
    need = L.agrl_policy_loss_workspace_size(100, 0, 64, 50, 0, None)
    assert _fwd(L, ws=1 << 12, wsb=need - 1) == E_WS


def test_backward_argument_errors(L):
    def bwd(**kw):
        a = dict(lse=1 << 12, logp=1 << 12, g=1.0, dH=1 << 12, dW=1 << 12, d=64)
        a.update(kw)
        return L.agrl_policy_loss_bwd(10, 0, a["d"], 50, 0, 1 << 12, 1 << 12, 1 << 12, 1 << 12,
                                      1 << 12, 1 << 12, 0.2, 0.2, 0, None, a["lse"], a["logp"],
                                      a["g"], None, 0, a["dH"], a["dW"], None)
    assert bwd(d=65) == E_UNSUP
    assert bwd() == E_WS
    need = L.agrl_policy_loss_workspace_size(10, 0, 64, 50, 0, None)
    assert L.agrl_policy_loss_bwd(10, 0, 64, 50, 0, 1 << 12, 1 << 12, 1 << 12, 1 << 12, 1 << 12,
                                  1 << 12, 0.2, 0.2, 0, None, None, 1 << 12, 1.0, 1 << 12, need,
                                  1 << 12, 1 << 12, None) == E_NULL
    assert L.agrl_policy_loss_bwd(10, 0, 64, 50, 0, 1 << 12, 1 << 12, 1 << 12, 1 << 12, 1 << 12,
                                  1 << 12, 0.2, 0.2, 0, None, 1 << 12, 1 << 12, float("inf"),
                                  1 << 12, need, 1 << 12, 1 << 12, None) == E_FLAGS
    for dh, dw in ((4100, 1 << 12), (1 << 12, 4104)):      # rows are written 16 B per lane
        assert L.agrl_policy_loss_bwd(10, 0, 64, 50, 0, 1 << 12, 1 << 12, 1 << 12, 1 << 12,
                                      1 << 12, 1 << 12, 0.2, 0.2, 0, None, 1 << 12, 1 << 12, 1.0,
                                      1 << 12, need, dh, dw, None) == E_UNSUP


def test_token_logprob_argument_errors(L):
    from paper_2510_04206_amd._binding import agrl_options
    p = 1 << 12
    f = L.agrl_token_logprob
    need = L.agrl_token_logprob_workspace_size(100, 0, 64, 50, 0, None)
    assert 0 < need < L.agrl_policy_loss_workspace_size(100, 0, 64, 50, 0, None)
    assert f(100, 0, 64, 50, 7, p, p, p, p, None, p, need, p, p, None) == E_DTYPE
    assert f(100, 0, 65, 50, 0, p, p, p, p, None, p, need, p, p, None) == E_UNSUP
    assert f(100, 0, 64, 50, 0, None, p, p, p, None, p, need, p, p, None) == E_NULL
    assert f(100, 0, 64, 50, 0, p, p, p, p, None, p, need, None, p, None) == E_NULL
    assert f(100, 0, 64, 50, 0, p, p, p, p, None, p, need - 1, p, p, None) == E_WS
    o = agrl_options(temperature=float("nan"))
    assert f(100, 0, 64, 50, 0, p, p, p, p, ctypes.byref(o), p, need, p, p, None) == E_FLAGS
    assert f(0, 0, 64, 50, 0, None, p, None, None, None, None, 0, None, None, None) == 0


def test_adv_norm_argument_errors(L):
    p = 1 << 12
    f = L.agrl_task_adv_norm
    assert f(-1, 1, 1, 0, p, p, p, None, p, None, p, p, p, p, p, None, None) == E_SHAPE
    assert f(10, 1, 1, 0, None, p, p, None, p, None, p, p, p, p, p, None, None) == E_NULL
    assert f(10, 1, 1, 0, p, p, p, p, p, None, p, p, p, p, p, None, None) == E_SHAPE  # n_group 0
    assert f(10, 1, 1, 0, p, p, None, None, p, None, p, p, p, p, p, None, None) == E_NULL
    assert f(10, 1, 1, 0, p, p, p, None, p, None, p, None, p, p, p, None, None) == E_NULL
    from paper_2510_04206_amd._binding import agrl_options
    o = agrl_options(std_ddof=2)
    assert f(10, 1, 1, 0, p, p, p, None, p, ctypes.byref(o), p, p, p, p, p, None, None) == E_FLAGS
    o = agrl_options(std_eps=-1.0)
    assert f(10, 1, 1, 0, p, p, p, None, p, ctypes.byref(o), p, p, p, p, p, None, None) == E_FLAGS
    o = agrl_options(drop_uniform_groups=1)            # dynamic sampling needs groups
    assert f(10, 1, 1, 0, p, p, p, None, p, ctypes.byref(o), p, p, p, p, p, None, None) == E_FLAGS
    o = agrl_options(drop_uniform_groups=2)
    assert f(10, 1, 1, 1, p, p, p, p, p, ctypes.byref(o), p, p, p, p, p, None, None) == E_FLAGS


def test_sequence_mean_weights_argument_errors(L):
    p = 1 << 12
    f = L.agrl_sequence_mean_weights
    assert f(-1, 1, p, p, p, p, None) == E_SHAPE
    assert f(10, -1, p, p, p, p, None) == E_SHAPE
    assert f(10, 1, None, p, p, p, None) == E_NULL
    assert f(10, 1, p, None, p, p, None) == E_NULL
    assert f(10, 1, p, p, p, None, None) == E_NULL
    assert f(10, 1, p, p, None, p, None) == E_NULL     # seq_count needed when n_traj > 0


def test_workspace_size(L):
    f = L.agrl_policy_loss_workspace_size
    assert f(0, 0, 64, 50, 0, None) == 0
    assert f(10, 0, 64, 50, 9, None) == 0
    small = f(65536, 1000, 5120, 152064, 0, None)
    big = f(65536, 20000, 5120, 152064, 0, None)
    assert 0 < small < big
    assert f(65536, 0, 5120, 152064, 0, None) >= big            # max_act <= 0 means T
    assert f(4096, 0, 256, 4096, 1, None) > f(4096, 0, 256, 4096, 0, None)   # fp32 is larger
    # the G budget bounds the chunked buffers
    from paper_2510_04206_amd._binding import agrl_options
    o = agrl_options(g_chunk_bytes=1 << 26)
    assert f(65536, 20000, 5120, 152064, 0, ctypes.byref(o)) < big
    # default bound: one chunk's G (bf16; dW reads it transposed) stays within
    # 4 GiB, so the whole T x V gradient is never held when it does not fit
    # (64k action rows x 152064 columns x 2 B = 18.6 GiB)
    full = 65536 * 152064 * 2
    assert f(65536, 65536, 5120, 152064, 0, None) < full
    assert f(65536, 65536, 5120, 152064, 0, None) < (4 << 30) + (3 << 30)   # + H_act, H^T, W^T
    # the 32B-shaped micro-batch (22793 action tokens, padded to 23040) walks
    # the vocabulary in two chunks of 76032 columns: G of 23040 x 93184 would
    # be the widest that fits, 152064 needs two chunks, evened out
    vc = L.agrl_policy_loss_vocab_chunk
    assert vc(65536, 22793, 5120, 152064, 0, None) == 76032
    # fp32 keeps G and G^T: half the columns per chunk for the same bound
    o = agrl_options(g_chunk_bytes=2 * 1024 * 4 * 512)
    assert vc(4096, 1000, 256, 4096, 1, ctypes.byref(o)) == 512
    assert vc(4096, 1000, 256, 4096, 0, ctypes.byref(o)) == 2048


def test_missing_library_fails_loudly(monkeypatch):
    from paper_2510_04206_amd import _binding
    monkeypatch.setattr(_binding, "_lib", None)
    monkeypatch.setattr(_binding, "LIB_PATH", "/nonexistent/libagrl.so")
    with pytest.raises(ImportError):
        _binding.lib()


def test_product_never_touches_the_oracle():
    pkg = os.path.join(ROOT, "paper_2510_04206_amd")
    for dirpath, _, files in os.walk(pkg):
        for fn in files:
            if fn.endswith((".py", ".hip", ".hpp", ".cpp", ".h")):
                src = open(os.path.join(dirpath, fn)).read()
                assert "oracle" not in src.lower(), fn


def test_binding_rejects_host_tensors():
    # the ABI takes device pointers: a host tensor is refused before any call
    import torch
    from paper_2510_04206_amd import _binding
    with pytest.raises(ValueError):
        _binding._ptr(torch.zeros(4))
    assert _binding._ptr(None) is None


def test_options_struct_layout_matches_header(tmp_path):
    """The binding's ctypes agrl_options has the C struct's size and field offsets
    (a C program built from include/agrl.h with gcc prints them)."""
    import shutil
    import subprocess
    from paper_2510_04206_amd._binding import agrl_options
    gcc = shutil.which("gcc")
    if gcc is None:
        pytest.skip("gcc not found")
    names = [f[0] for f in agrl_options._fields_]
    body = "".join(f'  printf("%s %zu\\n", "{n}", offsetof(agrl_options, {n}));\n' for n in names)
    src = tmp_path / "layout.c"
    src.write_text('#include <stddef.h>\n#include <stdio.h>\n#include "agrl.h"\nint main(void) {\n'
                   '  printf("size %zu\\n", sizeof(agrl_options));\n' + body + "  return 0;\n}\n")
    exe = tmp_path / "layout"
    subprocess.run([gcc, "-I", os.path.join(ROOT, "include"), str(src), "-o", str(exe)], check=True)
    got = dict(l.split() for l in subprocess.run([str(exe)], capture_output=True, text=True,
                                                  check=True).stdout.splitlines())
    assert int(got["size"]) == ctypes.sizeof(agrl_options)
    for n in names:
        assert int(got[n]) == getattr(agrl_options, n).offset, n
