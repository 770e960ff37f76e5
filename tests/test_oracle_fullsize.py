"""Pins for the oracle pieces the full-size parity tests use (CPU only).

token_logprob_full forms the logits with a library fp64 matmul; it is tied to
the C oracle's plain loops (which the other pins tie to the paper) on fp32
and bf16 inputs, several row blocks and a temperature, and to the hand-worked
two-word vocabulary.  surrogate_terms and dw_rows finish the forward and a
row of the backward from given log-probs; they are tied to the whole-batch
oracle's loss, clip counts, g and dW, and the loss to closed forms.
"""
import math

import numpy as np
import pytest
import torch

import oracle
from oracle import blas


def _case(T, V, d, seed, bf16):
    rng = np.random.default_rng(seed)
    H = torch.from_numpy(rng.standard_normal((T, d)).astype(np.float32))
    W = torch.from_numpy((0.3 * rng.standard_normal((V, d))).astype(np.float32))
    if bf16:
        H, W = H.to(torch.bfloat16), W.to(torch.bfloat16)
    y = rng.integers(0, V, T).astype(np.int32)
    mask = (rng.random(T) < 0.7).astype(np.uint8)
    adv = rng.standard_normal(T).astype(np.float32)
    old = (-np.log(V) + 0.4 * rng.standard_normal(T)).astype(np.float32)
    return H, W, y, mask, adv, old


@pytest.mark.parametrize("bf16,temp", [(False, 1.0), (True, 1.0), (True, 0.8)])
def test_full_logprob_matches_plain_loops(bf16, temp):
    H, W, y, mask, adv, old = _case(700, 333, 96, 3, bf16)
    r = oracle.policy_loss(H, W, y, mask, adv, old, temperature=temp, backward=False)
    # several row blocks, the last one partial
    logp, lse = blas.token_logprob_fp64(H, W, y, mask, temperature=temp, rows_per_block=128)
    m = mask.astype(bool)
    assert np.all(logp[~m] == 0) and np.all(lse[~m] == 0)
    np.testing.assert_allclose(lse, r["lse"], rtol=0, atol=1e-12)
    np.testing.assert_allclose(logp, r["logp"], rtol=0, atol=1e-12)
    f = oracle.token_logprob_full(H, W, y, mask, temperature=temp)
    np.testing.assert_allclose(f["logp"], r["logp"], rtol=0, atol=1e-12)


def test_full_logprob_two_word_vocabulary():
    """h = 1, w = (1, -1), y = 0: lse = 1 + log(1 + e^-2), logp = -log(1 + e^-2)."""
    f = oracle.token_logprob_full(np.array([[1.0]], np.float32), np.array([[1.0], [-1.0]], np.float32),
                                  np.array([0], np.int32), np.array([1], np.uint8))
    assert f["lse"][0] == pytest.approx(1.0 + math.log1p(math.exp(-2.0)), rel=1e-15)
    assert f["logp"][0] == pytest.approx(-math.log1p(math.exp(-2.0)), rel=1e-15)


def test_full_logprob_rejects_bad_ids():
    with pytest.raises(ValueError):
        oracle.token_logprob_full(np.ones((2, 4), np.float32), np.ones((3, 4), np.float32),
                                  np.array([0, 3], np.int32), np.array([1, 1], np.uint8))


def test_surrogate_terms_closed_form():
    """logp - old = 0.5: rho = e^0.5 > 1.2.  A = +1 clips (loss -1.2, g 0);
    A = -1 does not (loss e^0.5, g = e^0.5).  Two tokens: the mean."""
    m = np.array([1, 1, 0], np.uint8)
    logp = np.array([-1.0, -1.0, 0.0])
    old = np.array([-1.5, -1.5, 7.0], np.float32)
    r = oracle.surrogate_terms(m, np.array([1.0, -1.0, 3.0], np.float32), old, logp)
    assert r["loss"] == pytest.approx((-1.2 + math.exp(0.5)) / 2, rel=1e-14)
    assert list(r["n_clip"]) == [1, 0]
    assert r["g"][0] == 0.0 and r["g"][2] == 0.0
    assert r["g"][1] == pytest.approx(math.exp(0.5) / 2, rel=1e-14)


@pytest.mark.parametrize("eps", [(0.2, 0.2), (0.1, 0.28)])
def test_surrogate_terms_and_dw_rows_match_whole_batch(eps):
    H, W, y, mask, adv, old = _case(300, 257, 64, 5, True)
    r = oracle.policy_loss(H, W, y, mask, adv, old, eps_lo=eps[0], eps_hi=eps[1])
    s = oracle.surrogate_terms(mask, adv, old, r["logp"], eps_lo=eps[0], eps_hi=eps[1])
    assert s["loss"] == pytest.approx(r["loss"], rel=1e-14, abs=1e-16)
    np.testing.assert_array_equal(s["n_clip"], r["n_clip"])
    np.testing.assert_allclose(s["g"], r["g"], rtol=1e-14, atol=1e-18)
    rows = np.array([0, 17, 128, 256])
    dw = oracle.dw_rows(H, W, y, mask, r["lse"], s["g"], rows)
    np.testing.assert_allclose(dw, r["dW"][rows], rtol=1e-12, atol=1e-15)
    # the whole chain from the library-matmul forward
    f = oracle.token_logprob_full(H, W, y, mask)
    s2 = oracle.surrogate_terms(mask, adv, old, f["logp"], eps_lo=eps[0], eps_hi=eps[1])
    assert s2["loss"] == pytest.approx(r["loss"], rel=1e-11)
    dw2 = oracle.dw_rows(H, W, y, mask, f["lse"], s2["g"], rows)
    np.testing.assert_allclose(dw2, r["dW"][rows], rtol=1e-9, atol=1e-14)
