"""GPU parity of the forward-only token log-prob pass (agrl_token_logprob).

Against the oracle (log-softmax of the logits at the sampled ids, fp64) on
small workloads with ragged tiles, and bit-for-bit against the policy-loss
forward on the same inputs (same tiles, partials and merge), also at the
32B-shaped size.  Tolerances as for the forward's lse and logp (helpers.LSE_ATOL,
LOGP_ATOL): z is an fp32 sum of exact bf16 products over d terms.
"""
import numpy as np
import pytest
import torch

import oracle
from workloads import gen

from helpers import LOGP_ATOL, LSE_ATOL, log, to_dev

pytestmark = pytest.mark.gpu


def _logprob(w, d_in, max_act=None, opt=None):
    import paper_2510_04206_amd as P
    lp = P.TokenLogprob(w.T, w.d, w.V, w.H.dtype, max_act=w.n_act if max_act is None else max_act,
                        opt=opt)
    logp, lse = lp(d_in["H"], d_in["W"], d_in["token_id"], d_in["mask"])
    torch.cuda.synchronize()
    assert P.agrl_get_device_error() == 0
    return logp.cpu().numpy(), lse.cpu().numpy()


CASES = [
    ("fp32 workload 1", None),
    ("bf16 V1000 d128", dict(V=1000, d=128, dtype="bf16")),
    ("bf16 V5000 d512", dict(V=5000, d=512, dtype="bf16", n_tasks=4, n_groups=3)),
    ("fp32 V777 d64", dict(V=777, d=64, dtype="f32")),
]


@pytest.mark.parametrize("name,kw", CASES, ids=[c[0] for c in CASES])
def test_logprob_against_oracle(name, kw):
    w = gen.config(1) if kw is None else gen.make(gen.small_spec(name=name, **kw), seed=13)
    log(f"logprob case {name}: T={w.T} n_act={w.n_act} V={w.V} d={w.d}")
    d_in = to_dev(w)
    logp, lse = _logprob(w, d_in)
    r = oracle.token_logprob(w.H, w.W, w.token_id, w.mask)
    m = w.mask.astype(bool)
    assert np.all(logp[~m] == 0) and np.all(lse[~m] == 0)
    np.testing.assert_allclose(lse[m], r["lse"][m], rtol=0, atol=LSE_ATOL)
    np.testing.assert_allclose(logp[m], r["logp"][m], rtol=0, atol=LOGP_ATOL)


def test_logprob_temperature():
    w = gen.make(gen.small_spec(V=1300, d=192, dtype="bf16", name="lp temp"), seed=5)
    log("logprob temperature 0.8")
    logp, lse = _logprob(w, to_dev(w), opt={"temperature": 0.8})
    r = oracle.token_logprob(w.H, w.W, w.token_id, w.mask, temperature=0.8)
    m = w.mask.astype(bool)
    np.testing.assert_allclose(logp[m], r["logp"][m], rtol=0, atol=LOGP_ATOL)


def test_logprob_no_action_tokens_and_empty():
    import paper_2510_04206_amd as P
    w = gen.make(gen.small_spec(V=500, d=64, dtype="bf16", name="lp none"), seed=3)
    d_in = to_dev(w)
    d_in["mask"].zero_()
    log("logprob with no action tokens")
    logp, lse = _logprob(w, d_in, max_act=w.T)
    assert np.all(logp == 0) and np.all(lse == 0)
    # T == 0 enqueues nothing and succeeds
    P.agrl_token_logprob(0, 0, 64, 500, P.AGRL_BF16, d_in["H"], d_in["W"], None, None, None,
                         None, 0, None, None)


@pytest.mark.parametrize("k", [1, 3])
def test_logprob_bit_identical_to_policy_loss_forward(k):
    import paper_2510_04206_amd as P
    w = gen.config(k, device=torch.device("cuda"))
    log(f"logprob vs policy-loss forward, workload {k}: T={w.T} n_act={w.n_act}")
    d_in = to_dev(w)
    logp, lse = _logprob(w, d_in)
    adv = torch.zeros(w.T, dtype=torch.float32, device="cuda")
    pl = P.PolicyLoss(w.T, w.d, w.V, w.H.dtype, max_act=w.n_act)
    _, logp2, lse2, _ = pl.forward(d_in["H"], d_in["W"], d_in["token_id"], d_in["mask"], adv,
                                   d_in["old_logp"])
    torch.cuda.synchronize()
    np.testing.assert_array_equal(logp, logp2.cpu().numpy())
    np.testing.assert_array_equal(lse, lse2.cpu().numpy())
