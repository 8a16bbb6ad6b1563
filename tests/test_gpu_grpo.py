"""GPU parity: group advantages and the GRPO token loss against the oracle."""
import numpy as np
import pytest
import torch

import oracle
from paper_2510_17158_amd import api, synth
from paper_2510_17158_amd.workloads import get

from gpu_util import require_gpu, say

pytestmark = pytest.mark.gpu

RTOL, ATOL = 1e-5, 1e-7


def _adv(r, P, G, eps):
    t = torch.from_numpy(np.asarray(r, np.float32)).cuda()
    out = torch.empty_like(t)
    api.advantages(t, P, G, eps, out)
    torch.cuda.synchronize()
    return out.cpu().numpy()


@pytest.mark.parametrize("P,G", [(8, 8), (1, 2), (3, 12), (257, 5)])
def test_advantages_match_oracle(P, G):
    require_gpu()
    say("advantages", P, G)
    rng = np.random.default_rng(P * 100 + G)
    r = np.where(rng.random(P * G) < 0.3, 0.0, rng.lognormal(0, 0.5, P * G)).astype(np.float32)
    r[:G] = 1.5 if P > 1 else r[:G]            # a degenerate group
    got = _adv(r, P, G, 1e-6)
    ref = oracle.advantages(r, P, G, 1e-6)
    np.testing.assert_allclose(got, ref, rtol=RTOL, atol=ATOL)
    if P > 1:
        assert np.all(got[:G] == 0.0)


def test_advantages_workload_rewards():
    require_gpu()
    w = get("7b")
    r = synth.make_rewards(w)
    np.testing.assert_allclose(_adv(r, w.n_prompts, w.group, w.adv_eps),
                               oracle.advantages(r, w.n_prompts, w.group, w.adv_eps),
                               rtol=RTOL, atol=ATOL)


def _loss(inp, eps, beta, agg):
    dev = {k: torch.from_numpy(np.ascontiguousarray(v)).cuda() for k, v in inp.items()}
    N, Tr = inp["logp"].shape
    loss = torch.empty(1, device="cuda")
    tl = torch.empty(N, Tr, device="cuda")
    dl = torch.empty(N, Tr, device="cuda")
    st = torch.empty(4, device="cuda")
    ws = api.alloc_workspace(None, api.OP_LOSS, N, Tr)
    api.token_loss(dev["logp"], dev["logp_old"], dev["logp_ref"], dev["mask"], dev["adv"], eps,
                   beta, agg, loss, tl, dl, st, ws=ws)
    torch.cuda.synchronize()
    return loss.item(), tl.cpu().numpy(), dl.cpu().numpy(), st.cpu().numpy()


@pytest.mark.parametrize("N,Tr,agg", [(64, 2048, 0), (64, 2048, 1), (3, 5, 0), (1, 1, 1),
                                      (33, 257, 0)])
def test_token_loss_matches_oracle(N, Tr, agg):
    require_gpu()
    say("token_loss", N, Tr, agg)
    inp = synth.make_loss_inputs(N, Tr, seed=N * 7 + Tr, drift=0.3)
    if N > 2:
        inp["mask"][1] = 0                      # a sequence with no trained token
        inp["logp"][2, np.flatnonzero(inp["mask"][2] == 0)[:1]] = np.nan  # masked-out NaN
    loss, tl, dl, st = _loss(inp, 0.2, 0.04, agg)
    ref = oracle.token_loss(inp["logp"], inp["logp_old"], inp["logp_ref"], inp["mask"],
                            inp["adv"], 0.2, 0.04, agg)
    assert loss == pytest.approx(ref["loss"], rel=RTOL, abs=ATOL)
    np.testing.assert_allclose(tl, ref["tok_loss"], rtol=RTOL, atol=ATOL)
    np.testing.assert_allclose(dl, ref["grad"], rtol=RTOL, atol=ATOL)
    np.testing.assert_allclose(st, [ref["kl_mean"], ref["clip_frac"], ref["ratio_mean"],
                                    ref["nonfinite"]], rtol=RTOL, atol=ATOL)


def test_token_loss_ratio_one_and_nonfinite():
    require_gpu()
    N, Tr = 4, 16
    lp = np.full((N, Tr), -1.25, np.float32)
    inp = dict(logp=lp, logp_old=lp.copy(), logp_ref=lp.copy(), mask=np.ones((N, Tr), np.uint8),
               adv=np.array([1.0, -0.5, 0.0, 2.0], np.float32))
    loss, tl, dl, st = _loss(inp, 0.2, 0.04, 0)
    # ratio 1, no KL: l = -A per token, gradient -A / (N * Tr)
    np.testing.assert_allclose(tl, -inp["adv"][:, None] * np.ones((N, Tr)), rtol=1e-7)
    np.testing.assert_allclose(dl, -inp["adv"][:, None] / (N * Tr) * np.ones((N, Tr)), rtol=1e-6)
    assert st[0] == 0.0 and st[1] == 0.0 and st[2] == pytest.approx(1.0)
    inp["logp"] = lp.copy()
    inp["logp"][1, 3] = np.inf
    loss, tl, dl, st = _loss(inp, 0.2, 0.04, 0)
    assert st[3] == 1.0 and not np.isfinite(loss)


@pytest.mark.parametrize("agg", [0, 1])
def test_sft_loss_matches_oracle(agg):
    """Distillation cross-entropy (Sec. VI-B) over target tokens: loss within 1e-5
    relative, gradient within fp32 rounding of the oracle's."""
    require_gpu()
    rng = np.random.default_rng(11 + agg)
    N, Tr = 33, 1500
    lp = (-rng.random((N, Tr)) * 6).astype(np.float32)
    m = (rng.random((N, Tr)) < 0.6).astype(np.uint8)
    m[3] = 0
    d_lp, d_m = torch.from_numpy(lp).cuda(), torch.from_numpy(m).cuda()
    loss = torch.empty(1, device="cuda")
    g = torch.full((N, Tr), float("nan"), device="cuda")
    ws = api.alloc_workspace(None, api.OP_LOSS, N, Tr)
    api.sft_loss(d_lp, d_m, agg, loss, g, ws=ws)
    torch.cuda.synchronize()
    ref = oracle.sft_loss(lp, m, agg)
    assert abs(loss.item() - ref["loss"]) <= 1e-5 * abs(ref["loss"]) + 1e-7
    np.testing.assert_allclose(g.cpu().numpy(), ref["grad"], rtol=2.0 ** -23, atol=0)


def test_exact_kl_matches_oracle():
    """Full-vocabulary KL of two logit rows (fp64 inside, fp32 out): within fp32
    rounding of the oracle plus 1e-10 (fp64 sums over 32000 terms), at two
    temperatures, equal logits giving 0."""
    require_gpu()
    rng = np.random.default_rng(5)
    R, V = 40, 32000
    z = (rng.standard_normal((R, V)) * 1.3).astype(np.float32)
    zr = (z + rng.standard_normal((R, V)) * rng.choice([1e-3, 0.05, 0.5], (R, 1))).astype(
        np.float32)
    zr[0] = z[0]
    dz, dzr = torch.from_numpy(z).cuda(), torch.from_numpy(zr).cuda()
    for T in (1.0, 0.8):
        kl = torch.empty(R, device="cuda")
        api.exact_kl(dz, dzr, T, kl)
        torch.cuda.synchronize()
        ref = oracle.exact_kl(z.astype(np.float64), zr.astype(np.float64), T)
        got = kl.cpu().numpy()
        np.testing.assert_allclose(got, ref, rtol=2.0 ** -23, atol=1e-10)
        assert abs(got[0]) <= 1e-10
