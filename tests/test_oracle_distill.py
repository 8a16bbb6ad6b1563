"""Pins of the reward (Eq. 2-4), the distillation loss and the exact KL."""
import numpy as np

import oracle


def test_reward_case_table():
    """Each branch of r_perf and the tool term, values worked out by hand from
    Eq. 2-4: incorrect -2, correct but slower -1, t = t_base 0, twice as fast 1,
    capped at 10; tools: 3 of 6 available used -> 0.25, all -> 0.5, none -> 0."""
    rows = [  # correct, t_base, t, used, avail, expected
        (False, 1.0, 0.5, 0, 4, -2.0),
        (False, 1.0, 2.0, 6, 6, -1.5),
        (True, 1.0, 1.5, 0, 5, -1.0),
        (True, 1.0, 1.0, 0, 5, 0.0),
        (True, 2.0, 1.0, 3, 6, 1.25),
        (True, 0.881, 0.75, 1, 4, 0.881 / 0.75 - 1 + 0.125),
        (True, 30.0, 1.0, 4, 4, 10.5),
        (True, 11.0, 1.0, 2, 4, 10.25),
    ]
    c, tb, t, u, a, want = map(np.array, zip(*rows))
    got = oracle.reward(c, tb, t, u, a)
    np.testing.assert_allclose(got, want, rtol=0, atol=1e-12)
    # range of the paper's reward: [-2, 10.5]
    rng = np.random.default_rng(0)
    n = 10000
    r = oracle.reward(rng.random(n) < 0.7, rng.lognormal(0, 1, n), rng.lognormal(0, 1, n),
                      rng.integers(0, 7, n), rng.integers(4, 7, n))
    assert r.min() >= -2.0 and r.max() <= 10.5


def test_sft_loss_closed_form_and_gradient():
    rng = np.random.default_rng(1)
    lp = -rng.random((5, 9)) * 4
    m = rng.random((5, 9)) < 0.7
    m[2] = False
    for agg in (0, 1):
        r = oracle.sft_loss(lp, m, agg)
        if agg == 1:
            assert np.isclose(r["loss"], -lp[m].mean())
        else:
            per = [-lp[n][m[n]].mean() if m[n].any() else 0.0 for n in range(5)]
            assert np.isclose(r["loss"], np.mean(per))
        # gradient by central differences
        h = 1e-6
        g = np.zeros_like(lp)
        for i in range(lp.size):
            d = np.zeros(lp.size)
            d[i] = h
            d = d.reshape(lp.shape)
            g.flat[i] = (oracle.sft_loss(lp + d, m, agg)["loss"] -
                         oracle.sft_loss(lp - d, m, agg)["loss"]) / (2 * h)
        np.testing.assert_allclose(r["grad"], g, rtol=0, atol=1e-8)


def test_exact_kl_is_the_expectation_of_the_token_estimator():
    """sum_v p(v) (exp(d_v) - d_v - 1), d_v = log p_ref(v) - log p(v), equals
    KL(p || p_ref) exactly (sum_v p_ref(v) = 1); KL >= 0, 0 for equal or shifted
    logits; the temperature divides both logits."""
    rng = np.random.default_rng(2)
    z = rng.standard_normal((6, 300)) * 2
    zr = z + rng.standard_normal((6, 300)) * 0.3
    for T in (1.0, 0.7):
        kl = oracle.exact_kl(z, zr, T)
        lp = oracle.log_softmax(z / T)
        lq = oracle.log_softmax(zr / T)
        d = lq - lp
        k3 = np.sum(np.exp(lp) * (np.exp(d) - d - 1.0), axis=-1)
        np.testing.assert_allclose(kl, k3, rtol=1e-10, atol=1e-14)
        assert np.all(kl > 0)
    np.testing.assert_allclose(oracle.exact_kl(z, z + 3.0), 0.0, atol=1e-12)
    # two-point distribution: closed form
    p, q = 0.3, 0.6
    zz = np.log([[p, 1 - p]])
    qq = np.log([[q, 1 - q]])
    want = p * np.log(p / q) + (1 - p) * np.log((1 - p) / (1 - q))
    assert np.isclose(oracle.exact_kl(zz, qq)[0], want, rtol=1e-12)
