"""Pins of the oracle GRPO advantages and token loss: closed forms, the Eq. 1
reduction at ratio 1, the clip branches, torch autograd and finite differences."""
import numpy as np
import pytest
import torch

from oracle import advantages, token_loss


def test_advantages_mean0_std1():
    rng = np.random.default_rng(0)
    r = rng.lognormal(0, 0.5, 8 * 12)
    a = advantages(r, 8, 12, eps=0.0).reshape(8, 12)
    np.testing.assert_allclose(a.mean(axis=1), 0, atol=1e-14)
    np.testing.assert_allclose(a.std(axis=1, ddof=1), 1, rtol=1e-13)


def test_advantages_closed_forms():
    a = advantages([0.0, 1.0], 1, 2, eps=0.0)
    np.testing.assert_allclose(a, [-2 ** -0.5, 2 ** -0.5], rtol=1e-15)
    a = advantages([3.0, 3.0, 3.0, 3.0, 1.0, 2.0, 3.0, 4.0], 2, 4, eps=0.0)
    assert np.all(a[:4] == 0.0)
    s = np.std([1, 2, 3, 4], ddof=1)
    np.testing.assert_allclose(a[4:], (np.array([1, 2, 3, 4]) - 2.5) / s, rtol=1e-15)
    # eps enters the denominator
    np.testing.assert_allclose(advantages([0.0, 1.0], 1, 2, eps=0.5),
                               np.array([-0.5, 0.5]) / (2 ** -0.5 + 0.5), rtol=1e-15)
    with pytest.raises(ValueError):
        advantages([1.0], 1, 1)


def _one(lp, lo, lr, A, eps=0.2, beta=0.0):
    o = token_loss(np.array([[lp]]), np.array([[lo]]), np.array([[lr]]), np.ones((1, 1), np.uint8),
                   np.array([A]), eps, beta)
    return o


def test_ratio_one_reduces_to_policy_gradient():
    # rho = 1 and logp_ref = logp: loss = -A, d/dlogp = -A, kl = 0  (Eq. 1 at the current policy)
    for A in (-1.3, 0.0, 0.7):
        o = _one(-2.0, -2.0, -2.0, A, beta=0.04)
        assert o["loss"] == pytest.approx(-A, abs=1e-15)
        assert o["grad"][0, 0] == pytest.approx(-A, abs=1e-15)
        assert o["kl_mean"] == 0.0


@pytest.mark.parametrize("A,rho,s,g", [(1.0, 1.5, 1.2, 0.0), (-1.0, 0.5, -0.8, 0.0),
                                       (1.0, 0.5, 0.5, 0.5), (-1.0, 1.5, -1.5, -1.5),
                                       (1.0, 1.1, 1.1, 1.1)])
def test_clip_branches(A, rho, s, g):
    o = _one(np.log(rho), 0.0, np.log(rho), A)
    assert o["loss"] == pytest.approx(-s, rel=1e-13)
    assert o["grad"][0, 0] == pytest.approx(-g, rel=1e-13, abs=1e-15)
    assert o["clip_frac"] == (1.0 if g == 0.0 else 0.0)
    assert o["ratio_mean"] == pytest.approx(rho, rel=1e-13)


def test_kl_estimator_small_delta_and_sign():
    for d in (1e-3, -1e-3, 0.3, -2.0):
        o = _one(-1.0, -1.0, -1.0 + d, 0.0, beta=1.0)
        assert o["kl_mean"] >= 0
        if abs(d) < 1e-2:
            assert o["kl_mean"] == pytest.approx(d * d / 2 + d ** 3 / 6, rel=1e-6)
        assert o["loss"] == pytest.approx(np.exp(d) - d - 1, rel=1e-12)


def _inputs(seed, n=5, t=9):
    rng = np.random.default_rng(seed)
    lo = -rng.exponential(1.0, (n, t))
    lp = lo + 0.4 * rng.standard_normal((n, t))
    lr = lp + 0.3 * rng.standard_normal((n, t))
    m = (rng.random((n, t)) < 0.7).astype(np.uint8)
    m[0] = 0                                   # a fully masked sequence
    A = rng.standard_normal(n)
    return lp, lo, lr, m, A


@pytest.mark.parametrize("agg", [0, 1])
def test_gradient_matches_autograd_and_finite_differences(agg):
    lp, lo, lr, m, A = _inputs(agg)
    eps, beta = 0.2, 0.04
    o = token_loss(lp, lo, lr, m, A, eps, beta, agg)
    # independent: torch autograd through a direct transcription of the objective
    t = torch.tensor(lp, requires_grad=True)
    rho = torch.exp(t - torch.tensor(lo))
    At = torch.tensor(A)[:, None]
    s = torch.minimum(rho * At, torch.clamp(rho, 1 - eps, 1 + eps) * At)
    d = torch.tensor(lr) - t
    ell = -s + beta * (torch.exp(d) - d - 1)
    mt = torch.tensor(m, dtype=torch.float64)
    if agg == 0:
        L = ((ell * mt).sum(1) / mt.sum(1).clamp(min=1)).mean()
    else:
        L = (ell * mt).sum() / mt.sum().clamp(min=1)
    L.backward()
    assert o["loss"] == pytest.approx(L.item(), rel=1e-13)
    np.testing.assert_allclose(o["grad"], t.grad.numpy(), rtol=1e-12, atol=1e-15)
    # central finite differences of the oracle's own loss
    h = 1e-6
    for (i, j) in [(1, 0), (2, 3), (4, 8), (3, 5)]:
        e = np.zeros_like(lp)
        e[i, j] = h
        fd = (token_loss(lp + e, lo, lr, m, A, eps, beta, agg)["loss"]
              - token_loss(lp - e, lo, lr, m, A, eps, beta, agg)["loss"]) / (2 * h)
        assert fd == pytest.approx(o["grad"][i, j], rel=1e-5, abs=1e-9)


def test_masked_tokens_ignored_and_nonfinite_counted():
    lp, lo, lr, m, A = _inputs(3)
    lp2 = lp.copy()
    lp2[m == 0] = np.nan
    a = token_loss(lp, lo, lr, m, A, 0.2, 0.04)
    b = token_loss(lp2, lo, lr, m, A, 0.2, 0.04)
    assert a["loss"] == b["loss"] and b["nonfinite"] == 0
    lp3 = lp.copy()
    i, j = np.argwhere(m == 1)[0]
    lp3[i, j] = np.inf
    c = token_loss(lp3, lo, lr, m, A, 0.2, 0.04)
    assert c["nonfinite"] == 1 and not np.isfinite(c["loss"])
