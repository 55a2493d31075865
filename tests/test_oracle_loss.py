"""Pins of the oracle's log-prob, clipped policy-ratio loss and gradients
(Eq. loss, App. E).

Library log-softmax, hand-computed scalar values of the clipped objective,
closed forms (ratio 1, zero advantage, zero projection) and central finite
differences of the summed loss with respect to the hidden states and the
vocabulary projection; for the KL penalty, the estimator's expectation under
pi_theta against the exact divergence of two small distributions, its zero
and second-order behaviour, and finite differences with the penalty on.
"""
import math

import numpy as np
import pytest
import scipy.special

from oracle import loss as OLS


def _problem(seed=0, r=6, H=5, V=11):
    rng = np.random.default_rng(seed)
    h = rng.standard_normal((r, H))
    w = 0.5 * rng.standard_normal((V, H))
    tgt = rng.integers(0, V, size=r)
    return rng, h, w, tgt


def test_logprob_matches_log_softmax():
    _, h, w, tgt = _problem()
    logp, lse, z = OLS.logprob(h, w, tgt, logit_scale=1.3)
    ref = scipy.special.log_softmax(1.3 * (h @ w.T), axis=1)
    assert np.allclose(logp, ref[np.arange(len(tgt)), tgt], atol=1e-13)


def test_zero_projection_gives_uniform():
    _, h, w, tgt = _problem()
    logp, _, _ = OLS.logprob(h, np.zeros_like(w), tgt)
    assert np.allclose(logp, -math.log(w.shape[0]), atol=1e-14)


@pytest.mark.parametrize("adv,rho,eps_l,eps_h,c,obj,clipped", [
    # A > 0: min(rho A, clip(rho) A)
    (2.0, 1.5, 0.2, 0.2, 0.0, 2.4, True),       # upper clip: 1.2 * 2
    (2.0, 0.5, 0.2, 0.2, 0.0, 1.0, False),      # below 1-eps: unclipped 0.5 * 2
    (2.0, 1.1, 0.2, 0.28, 0.0, 2.2, False),
    (1.0, 1.3, 0.2, 0.28, 0.0, 1.28, True),     # asymmetric upper bound 1.28
    # A < 0: = A * max(rho, clip(rho))
    (-2.0, 0.5, 0.2, 0.2, 0.0, -1.6, True),     # lower clip: 0.8 * -2
    (-2.0, 1.5, 0.2, 0.2, 0.0, -3.0, False),    # above 1+eps: unclipped
    (-1.0, 5.0, 0.2, 0.28, 3.0, -3.0, True),    # dual clip caps at c * A
    (-1.0, 2.0, 0.2, 0.28, 3.0, -2.0, False),
    (0.0, 1.7, 0.2, 0.2, 0.0, 0.0, False),
])
def test_clipped_objective_hand_values(adv, rho, eps_l, eps_h, c, obj, clipped):
    o, l, r, cl = OLS.clipped_objective(np.array([math.log(rho)]), np.array([0.0]),
                                        np.array([adv]), eps_l, eps_h, c)
    assert abs(o[0] - obj) < 1e-12 and abs(l[0] + obj) < 1e-12
    assert bool(cl[0]) == clipped


def test_ratio_one_closed_form():
    """old = current: rho = 1, loss = -A per row, g = -loss_scale * A."""
    _, h, w, tgt = _problem(2)
    logp, _, _ = OLS.logprob(h, w, tgt)
    adv = np.array([0.5, -1.0, 2.0, 0.0, 1.5, -0.3])
    out = OLS.loss_and_grads(h, w, tgt, logp, adv, 0.2, 0.2, loss_scale=0.25)
    assert np.allclose(out["loss_tok"], -adv, atol=1e-13)
    assert np.allclose(out["g"], -0.25 * adv, atol=1e-13)
    assert abs(out["loss_sum"] - 0.25 * (-adv).sum()) < 1e-13


def test_zero_advantage_zero_gradient():
    rng, h, w, tgt = _problem(3)
    old = rng.standard_normal(len(tgt))
    out = OLS.loss_and_grads(h, w, tgt, old, np.zeros(len(tgt)), 0.2, 0.2)
    assert not out["dh"].any() and not out["dw"].any()


@pytest.mark.parametrize("dual", [0.0, 3.0])
def test_gradients_finite_differences(dual):
    rng, h, w, tgt = _problem(4, r=8, H=6, V=13)
    logp, _, _ = OLS.logprob(h, w, tgt, 0.9)
    # ratios spread over both clip regions, kept away from the kinks
    shift = np.array([0.5, -0.5, 0.05, -0.05, 0.6, -0.7, 1.3, 0.0])
    old = logp - shift
    adv = np.array([1.0, -1.0, 0.7, -0.4, -1.2, 0.8, -0.9, 1.1])
    kw = dict(eps_low=0.2, eps_high=0.28, loss_scale=0.37, logit_scale=0.9, dual_clip_c=dual)
    out = OLS.loss_and_grads(h, w, tgt, old, adv, **kw)

    def total(h_, w_):
        return OLS.loss_and_grads(h_, w_, tgt, old, adv, want_grad=False, **kw)["loss_sum"]

    eps = 1e-6
    for which, grad in ((0, out["dh"]), (1, out["dw"])):
        d = rng.standard_normal(h.shape if which == 0 else w.shape)
        if which == 0:
            fd = (total(h + eps * d, w) - total(h - eps * d, w)) / (2 * eps)
        else:
            fd = (total(h, w + eps * d) - total(h, w - eps * d)) / (2 * eps)
        an = float((grad * d).sum())
        assert abs(fd - an) < 1e-6 * max(1.0, abs(an)), (which, fd, an)
    assert out["clipped"].any() and (~out["clipped"]).any()


# ---- KL penalty (lambda * D_KL(pi_theta || pi_ref) in Eq. loss)

def test_kl_estimate_expectation_is_exact_kl():
    """Averaged over tokens drawn from pi_theta (weights pi_theta over the
    whole vocabulary), the per-token estimate is the exact KL divergence
    sum pi_theta log(pi_theta / pi_ref), which fixes its sign convention."""
    rng = np.random.default_rng(7)
    V = 17
    z_t = rng.standard_normal(V) * 1.5
    z_r = z_t + 0.4 * rng.standard_normal(V)
    lp_t = z_t - scipy.special.logsumexp(z_t)
    lp_r = z_r - scipy.special.logsumexp(z_r)
    p_t = np.exp(lp_t)
    exact = float((p_t * (lp_t - lp_r)).sum())
    expected = float((p_t * OLS.kl_estimate(lp_t, lp_r)).sum())
    assert exact > 0
    assert abs(expected - exact) < 1e-12 * max(1.0, exact)


def test_kl_estimate_zero_and_positive():
    rng = np.random.default_rng(8)
    a = rng.standard_normal(50)
    assert np.array_equal(OLS.kl_estimate(a, a), np.zeros(50))
    b = a + rng.standard_normal(50)
    assert (OLS.kl_estimate(a, b) > 0).all()
    # second-order behaviour: (x^2)/2 for small x = ref - logp
    x = 1e-4
    assert abs(OLS.kl_estimate(np.array([0.0]), np.array([x]))[0] - x * x / 2) < 1e-12


def test_kl_zero_coefficient_is_the_plain_objective():
    rng, h, w, tgt = _problem(9)
    old = rng.standard_normal(len(tgt))
    adv = rng.standard_normal(len(tgt))
    ref = rng.standard_normal(len(tgt))
    a = OLS.loss_and_grads(h, w, tgt, old, adv, 0.2, 0.28)
    b = OLS.loss_and_grads(h, w, tgt, old, adv, 0.2, 0.28, ref_logp=ref, kl_coef=0.0)
    for k in ("loss_tok", "dh", "dw"):
        assert np.array_equal(a[k], b[k]), k
    assert a["loss_sum"] == b["loss_sum"]


def test_kl_gradients_finite_differences():
    """With a large KL coefficient, central differences of the summed loss
    match the analytic dh, dw (clipped rows still carry the KL gradient)."""
    rng, h, w, tgt = _problem(10, r=8, H=6, V=13)
    logp, _, _ = OLS.logprob(h, w, tgt, 0.9)
    shift = np.array([0.5, -0.5, 0.05, -0.05, 0.6, -0.7, 1.3, 0.0])
    old = logp - shift
    ref = logp + np.array([0.3, -0.2, 0.0, 0.8, -1.1, 0.25, 0.05, -0.4])
    adv = np.array([1.0, -1.0, 0.7, -0.4, -1.2, 0.8, -0.9, 1.1])
    kw = dict(eps_low=0.2, eps_high=0.28, loss_scale=0.37, logit_scale=0.9, ref_logp=ref,
              kl_coef=0.6)
    out = OLS.loss_and_grads(h, w, tgt, old, adv, **kw)
    assert out["clipped"].any()

    def total(h_, w_):
        return OLS.loss_and_grads(h_, w_, tgt, old, adv, want_grad=False, **kw)["loss_sum"]

    eps = 1e-6
    for which, grad in ((0, out["dh"]), (1, out["dw"])):
        d = rng.standard_normal(h.shape if which == 0 else w.shape)
        if which == 0:
            fd = (total(h + eps * d, w) - total(h - eps * d, w)) / (2 * eps)
        else:
            fd = (total(h, w + eps * d) - total(h, w - eps * d)) / (2 * eps)
        an = float((grad * d).sum())
        assert abs(fd - an) < 1e-6 * max(1.0, abs(an)), (which, fd, an)
