"""The allocation-free log-prob entry point against the one that takes a workspace.

agrl_token_logprob_noalloc runs agrl_token_logprob's kernels on a fixed
per-device scratch array instead of a caller workspace.  Its outputs must be
bit-identical to agrl_token_logprob's on the same inputs, on two calls in a row
(the second smaller, so it runs on scratch the first one left behind), and
sizes beyond the array are refused before anything is launched.
"""
import ctypes

import numpy as np
import pytest
import torch

from workloads import gen

from helpers import log

pytestmark = pytest.mark.gpu


def _pair(w):
    """(logp, lse) from agrl_token_logprob with a torch workspace, and from the
    allocation-free entry point, on the same device inputs."""
    from paper_2510_04206_amd import _binding as B
    dev = torch.device("cuda")
    t = lambda x: torch.from_numpy(np.ascontiguousarray(x)).to(dev)
    H, W = w.H.to(dev), w.W.to(dev)
    ids, mask = t(w.token_id), t(w.mask)
    code = B.dtype_code(H)
    ws_bytes = B.agrl_token_logprob_workspace_size(w.T, w.n_act, w.d, w.V, code)
    assert 0 < ws_bytes <= B.AGRL_NOALLOC_SCRATCH_BYTES
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device=dev)
    ref = [torch.full((w.T,), 7.0, device=dev) for _ in range(2)]
    out = [torch.full((w.T,), 7.0, device=dev) for _ in range(2)]
    B.agrl_token_logprob(w.T, w.n_act, w.d, w.V, code, H, W, ids, mask, None, ws, ws_bytes,
                         ref[0], ref[1])
    B.agrl_token_logprob_noalloc(w.T, w.n_act, w.d, w.V, code, H, W, ids, mask, None, out[0],
                                 out[1])
    torch.cuda.synchronize()
    assert B.agrl_get_device_error() == 0
    return [x.cpu().numpy() for x in ref], [x.cpu().numpy() for x in out]


def test_noalloc_matches_workspace_entry_point_twice():
    cases = [gen.make(gen.small_spec(V=5000, d=512, dtype="bf16", n_tasks=4, n_groups=3,
                                     name="noalloc large"), seed=41),
             gen.make(gen.small_spec(V=700, d=128, dtype="bf16", name="noalloc small"), seed=42)]
    assert cases[1].n_act < cases[0].n_act and cases[1].T < cases[0].T
    for w in cases:
        log(f"noalloc logprob {w.spec.name} T={w.T} n_act={w.n_act} V={w.V} d={w.d}")
        ref, out = _pair(w)
        for r, o in zip(ref, out):
            np.testing.assert_array_equal(o.view(np.uint32), r.view(np.uint32))
        m = w.mask.astype(bool)
        assert np.all(out[0][~m] == 0) and np.isfinite(out[0][m]).all()


def test_noalloc_refuses_sizes_beyond_the_scratch():
    from paper_2510_04206_amd import _binding as B
    log("noalloc: oversized problem refused")
    dev = torch.device("cuda")
    T, d, V = 8192, 4096, 152064
    assert B.agrl_token_logprob_workspace_size(T, T, d, V, B.AGRL_BF16) > B.AGRL_NOALLOC_SCRATCH_BYTES
    H = torch.zeros((T, d), dtype=torch.bfloat16, device=dev)
    W = torch.zeros((V, d), dtype=torch.bfloat16, device=dev)
    ids = torch.zeros(T, dtype=torch.int32, device=dev)
    mask = torch.ones(T, dtype=torch.uint8, device=dev)
    logp = torch.full((T,), 7.0, device=dev)
    lse = torch.full((T,), 7.0, device=dev)
    with pytest.raises(B.AgrlError) as e:
        B.agrl_token_logprob_noalloc(T, T, d, V, B.AGRL_BF16, H, W, ids, mask, None, logp, lse)
    assert e.value.status == -5 and "scratch" in str(e.value)
    torch.cuda.synchronize()
    assert bool((logp == 7.0).all()) and bool((lse == 7.0).all())
