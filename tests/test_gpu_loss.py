"""GPU parity of the fused policy loss (forward + backward) against the oracle.

Small and medium workloads are compared element by element with the oracle's
whole-batch fp64 result: several 256-wide tiles in every GEMM dimension and
ragged tails (T, N_act, V not multiples of the tile).  Tolerances: loss 1e-3
relative, lse 2e-5 and logp 5e-5 absolute (fp32 accumulation of bf16 products over d),
dH and dW 2e-2 relative Frobenius (G rounded to bf16).
"""
import numpy as np
import pytest
import torch

import oracle
from workloads import gen

from helpers import compare_loss, log, rel_fro, run_gpu, to_dev

pytestmark = pytest.mark.gpu


def _adv(w):
    a = oracle.task_adv_norm(w.g_traj_id, w.g_mask, w.traj_task, w.traj_group, w.reward,
                             w.n_task, w.n_group)
    return a["adv_tok"][: w.T].copy()


def _run_case(w, *, eps=(0.2, 0.2), n_norm=0, temperature=1.0, opt=None, max_act=None,
              adv=None, grad_rel=2e-2):
    import paper_2510_04206_amd as P
    adv = _adv(w) if adv is None else adv
    o = dict(opt or {})
    if temperature != 1.0:
        o["temperature"] = temperature
    log(f"loss case {w.spec.name} T={w.T} n_act={w.n_act} V={w.V} d={w.d} eps={eps} "
        f"n_norm={n_norm} temp={temperature} opt={o}")
    d_in = to_dev(w)
    pl = P.PolicyLoss(w.T, w.d, w.V, w.H.dtype, max_act=w.n_act if max_act is None else max_act,
                      eps_low=eps[0], eps_high=eps[1], n_norm=n_norm, opt=o or None)
    g = run_gpu(pl, d_in, torch.from_numpy(adv).cuda())
    assert P.agrl_get_device_error() == 0
    r = oracle.policy_loss(w.H, w.W, w.token_id, w.mask, adv, w.old_logp, eps_lo=eps[0],
                           eps_hi=eps[1], n_norm=n_norm, temperature=temperature)
    errs = compare_loss(g, r, w.mask, adv, w.old_logp, eps[0], eps[1], grad_rel=grad_rel)
    log(f"  loss gpu {g['loss']:.7g} oracle {r['loss']:.7g}; dH/dW rel fro {errs}")
    return g, r


def test_workload1_fp32():
    _run_case(gen.config(1))


SMALL = [
    ("bf16 V1000 d128", dict(V=1000, d=128, dtype="bf16")),
    ("bf16 V5000 d512", dict(V=5000, d=512, dtype="bf16", n_tasks=4, n_groups=3)),
    ("fp32 V777 d64", dict(V=777, d=64, dtype="f32")),
    ("bf16 V300 d64 tiny", dict(V=300, d=64, dtype="bf16", n_tasks=1, n_groups=1, group_size=2,
                                 turns=(1, 2), obs=(1, 5), act=(1, 9))),
    # d not a multiple of 256 (a partial last column tile in dH and dW)
    ("bf16 V2048 d192", dict(V=2048, d=192, dtype="bf16")),
    ("bf16 V1408 d320", dict(V=1408, d=320, dtype="bf16", n_tasks=3)),
]


@pytest.mark.parametrize("name,kw", SMALL, ids=[s[0] for s in SMALL])
def test_small_workloads(name, kw):
    _run_case(gen.make(gen.small_spec(name=name, **kw), seed=11))


def test_options_temperature_decoupled_clip_n_norm():
    w = gen.make(gen.small_spec(V=1300, d=192, dtype="bf16", noise_std=0.3, name="opts"), seed=5)
    _run_case(w, eps=(0.2, 0.28), n_norm=3000, temperature=0.8)


def test_vocabulary_chunks_match_single_chunk():
    """A small G budget forces several vocabulary chunks (the last one ragged)."""
    w = gen.make(gen.small_spec(V=2000, d=128, dtype="bf16", name="chunks"), seed=7)
    g1, _ = _run_case(w)
    A_pad = (w.n_act + 255) // 256 * 256
    g3, _ = _run_case(w, opt={"g_chunk_bytes": 2 * A_pad * 2 * 768})     # chunks of <= 768 columns
    assert g1["loss"] == g3["loss"]
    np.testing.assert_array_equal(g1["dW"], g3["dW"])                    # dW rows do not mix chunks
    assert rel_fro(g3["dH"], g1["dH"]) < 1e-5


def test_vocabulary_chunks_short_last_chunk():
    """Four chunks, the last one 128 columns wide: the same result as one chunk,
    and parity with the oracle."""
    w = gen.make(gen.small_spec(V=1664, d=256, dtype="bf16", name="chunks wtr"), seed=8)
    g1, _ = _run_case(w)
    A_pad = (w.n_act + 255) // 256 * 256
    g4, _ = _run_case(w, opt={"g_chunk_bytes": A_pad * 2 * 512})       # chunks of 512 columns
    assert g1["loss"] == g4["loss"]
    np.testing.assert_array_equal(g1["dW"], g4["dW"])
    assert rel_fro(g4["dH"], g1["dH"]) < 1e-5


def _launch_tiles(n_act, V, d, vc):
    """Tiles of each matrix-core launch: forward (vocabulary x tokens), recompute
    per chunk (tokens x chunk columns), dH + dW per chunk (tokens x d, chunk x d)."""
    t = lambda x: -(-x // 256)
    chunks = [min(vc, V - v0) for v0 in range(0, V, vc)]
    return (t(V) * t(n_act), [t(n_act) * t(c) for c in chunks],
            [t(n_act) * t(d) + t(c) * t(d) for c in chunks])


@pytest.mark.timeout(600)
def test_whole_batch_multi_round_three_chunks():
    """A whole batch large enough for the persistent schedule to run several
    rounds of 256 tiles per launch (every workgroup takes several tiles, the
    queues' full-round and final partial-round branches both run), with three
    vocabulary chunks, the last one ragged: every output element against the
    oracle's whole batch."""
    import paper_2510_04206_amd as P
    w = gen.make(gen.small_spec(V=131000, d=384, dtype="bf16", n_tasks=3, n_groups=2,
                                group_size=7, name="whole batch V131000 d384"),
                 seed=32, device="cuda")
    A_pad = -(-w.n_act // 256) * 256
    opt = {"g_chunk_bytes": 49152 * A_pad * 2}
    vc = P.PolicyLoss(w.T, w.d, w.V, w.H.dtype, max_act=w.n_act, opt=opt).vocab_chunk
    fwd, rec, bwd = _launch_tiles(w.n_act, w.V, w.d, vc)
    log(f"  vocab chunk {vc}; tiles: forward {fwd}, recompute {rec}, dH + dW {bwd}")
    # ragged in every dimension: tokens, vocabulary, the last chunk and d
    assert len(rec) == 3 and w.V % 256 and (w.V - 2 * vc) % 256 and w.n_act % 256 and w.d % 256
    assert fwd >= 1024 and min(rec) >= 1024 and min(bwd) > 256
    _run_case(w, opt=opt)


def test_dw_accumulate():
    import paper_2510_04206_amd as P
    w = gen.make(gen.small_spec(V=600, d=128, dtype="bf16", name="acc"), seed=9)
    adv = _adv(w)
    d_in = to_dev(w)
    log("dw_accumulate")
    pl = P.PolicyLoss(w.T, w.d, w.V, w.H.dtype, max_act=w.n_act, opt={"dw_accumulate": 1})
    pl.dW.fill_(1.5)
    g = run_gpu(pl, d_in, torch.from_numpy(adv).cuda())
    ref = P.PolicyLoss(w.T, w.d, w.V, w.H.dtype, max_act=w.n_act)
    g0 = run_gpu(ref, d_in, torch.from_numpy(adv).cuda())
    np.testing.assert_array_equal(g["dW"], (g0["dW"] + np.float32(1.5)).astype(np.float32))


def test_deterministic():
    import paper_2510_04206_amd as P
    w = gen.make(gen.small_spec(V=3000, d=256, dtype="bf16", name="det"), seed=13)
    adv = torch.from_numpy(_adv(w)).cuda()
    d_in = to_dev(w)
    log("determinism")
    pl = P.PolicyLoss(w.T, w.d, w.V, w.H.dtype, max_act=w.n_act)
    a = run_gpu(pl, d_in, adv)
    b = run_gpu(pl, d_in, adv)
    assert a["loss"] == b["loss"]
    for k in ("logp", "lse", "dH", "dW", "n_clip"):
        np.testing.assert_array_equal(a[k], b[k])


def test_masked_tokens_inert_and_zero():
    """NaN hidden states, bad ids and NaN adv/old on masked tokens change nothing."""
    import paper_2510_04206_amd as P
    w = gen.make(gen.small_spec(V=700, d=128, dtype="bf16", name="poison"), seed=17)
    adv = _adv(w)
    d_in = to_dev(w)
    log("masked poison")
    pl = P.PolicyLoss(w.T, w.d, w.V, w.H.dtype, max_act=w.n_act)
    a = run_gpu(pl, d_in, torch.from_numpy(adv).cuda())
    off = torch.from_numpy(w.mask == 0).cuda()
    p_in = dict(d_in)
    p_in["H"] = d_in["H"].clone()
    p_in["H"][off] = float("nan")
    p_in["token_id"] = torch.where(off, torch.full_like(d_in["token_id"], w.V + 7), d_in["token_id"])
    p_in["old_logp"] = torch.where(off, torch.full_like(d_in["old_logp"], float("nan")),
                                   d_in["old_logp"])
    adv_p = torch.from_numpy(adv).cuda()
    adv_p = torch.where(off, torch.full_like(adv_p, float("nan")), adv_p)
    b = run_gpu(pl, p_in, adv_p)
    assert P.agrl_get_device_error() == 0
    assert a["loss"] == b["loss"]
    for k in ("logp", "lse", "dH", "dW", "n_clip"):
        np.testing.assert_array_equal(a[k], b[k])


def test_no_action_tokens_and_all_action_tokens():
    import paper_2510_04206_amd as P
    w = gen.make(gen.small_spec(V=512, d=64, dtype="bf16", name="edge"), seed=19)
    adv = _adv(w)
    d_in = to_dev(w)
    log("no action tokens")
    d0 = dict(d_in)
    d0["mask"] = torch.zeros_like(d_in["mask"])
    pl = P.PolicyLoss(w.T, w.d, w.V, w.H.dtype, max_act=w.n_act)
    g = run_gpu(pl, d0, torch.from_numpy(adv).cuda())
    assert g["loss"] == 0.0
    assert np.all(g["dH"] == 0) and np.all(g["dW"] == 0) and np.all(g["logp"] == 0)
    # every token an action token, ids at the top of the vocabulary
    w.g_mask[: w.T] = 1
    w.token_id[:] = np.where(np.arange(w.T) % 3 == 0, w.V - 1, w.token_id)
    adv = np.random.default_rng(0).standard_normal(w.T).astype(np.float32)
    _run_case(w, adv=adv)


def test_max_act_overflow_flagged():
    import paper_2510_04206_amd as P
    w = gen.make(gen.small_spec(V=400, d=64, dtype="bf16", name="flags"), seed=23)
    adv = torch.from_numpy(_adv(w)).cuda()
    d_in = to_dev(w)
    log("max_act overflow")
    pl = P.PolicyLoss(w.T, w.d, w.V, w.H.dtype, max_act=w.n_act - 1)
    loss, *_ = pl.forward(d_in["H"], d_in["W"], d_in["token_id"], d_in["mask"], adv,
                          d_in["old_logp"])
    assert np.isnan(loss.item())
    assert P.agrl_get_device_error() & 16
    assert P.agrl_get_device_error() == 0


# V = 400 is not a multiple of the 256-row tile: V pads the last vocabulary tile,
# V_pad + 5 lies beyond it, -3 is negative
@pytest.mark.parametrize("bad_id", [400, 517, -3])
def test_bad_token_id_poisons_outputs(bad_id):
    """An out-of-range id on an action token sets the error bit and turns that
    token's logp / lse, the loss, its dH row and dW into NaN; every other token's
    logp / lse is unchanged."""
    import paper_2510_04206_amd as P
    w = gen.make(gen.small_spec(V=400, d=64, dtype="bf16", name="bad ids"), seed=23)
    adv = torch.from_numpy(_adv(w)).cuda()
    d_in = to_dev(w)
    log(f"bad token id {bad_id}")
    pl = P.PolicyLoss(w.T, w.d, w.V, w.H.dtype, max_act=w.n_act)
    good = run_gpu(pl, d_in, adv)
    assert P.agrl_get_device_error() == 0
    act = np.nonzero(w.mask)[0]
    t_bad = int(act[len(act) // 2])
    p_in = dict(d_in)
    p_in["token_id"] = d_in["token_id"].clone()
    p_in["token_id"][t_bad] = bad_id
    g = run_gpu(pl, p_in, adv)
    assert P.agrl_get_device_error() & 1
    assert P.agrl_get_device_error() == 0
    assert np.isnan(g["loss"])
    assert np.isnan(g["logp"][t_bad]) and np.isnan(g["lse"][t_bad])
    others = np.ones(w.T, bool)
    others[t_bad] = False
    np.testing.assert_array_equal(g["logp"][others], good["logp"][others])
    np.testing.assert_array_equal(g["lse"][others], good["lse"][others])
    assert np.isnan(g["dH"][t_bad]).all()
    assert np.isnan(g["dW"]).all()
    # masked rows of dH stay +0
    off = w.mask == 0
    assert np.all(g["dH"][off] == 0)
    # the forward-only log-prob pass poisons the same token
    lp = P.TokenLogprob(w.T, w.d, w.V, w.H.dtype, max_act=w.n_act)
    logp, lse = lp(p_in["H"], p_in["W"], p_in["token_id"], p_in["mask"])
    torch.cuda.synchronize()
    assert P.agrl_get_device_error() & 1
    logp, lse = logp.cpu().numpy(), lse.cpu().numpy()
    assert np.isnan(logp[t_bad]) and np.isnan(lse[t_bad])
    np.testing.assert_array_equal(logp[others], good["logp"][others].astype(np.float32))


def test_argument_errors_on_gpu():
    import paper_2510_04206_amd as P
    log("argument errors")
    H = torch.zeros(64, 100, dtype=torch.bfloat16, device="cuda")
    W = torch.zeros(50, 100, dtype=torch.bfloat16, device="cuda")
    z = torch.zeros(64, device="cuda")
    ids = torch.zeros(64, dtype=torch.int32, device="cuda")
    m = torch.ones(64, dtype=torch.uint8, device="cuda")
    pl = P.PolicyLoss(64, 100, 50, torch.bfloat16)
    with pytest.raises(P.AgrlError) as e:          # d not a multiple of 64
        pl.forward(H, W, ids, m, z, z)
    assert e.value.status == -7
    pl = P.PolicyLoss(64, 64, 50, torch.bfloat16, eps_low=1.5)
    with pytest.raises(P.AgrlError) as e:          # clip bound out of range
        pl.forward(H[:, :64].contiguous(), W[:, :64].contiguous(), ids, m, z, z)
    assert e.value.status == -4


@pytest.mark.gpu
def test_binding_rejects_strided_tensors():
    from paper_2510_04206_amd import _binding
    log("binding: non-contiguous tensor refused")
    x = torch.zeros(8, 16, device="cuda").t()
    with pytest.raises(ValueError):
        _binding._ptr(x)
    assert _binding._ptr(x.contiguous()) is not None
