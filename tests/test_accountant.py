"""The privacy accountant against facts it does not compute the same way:
the Gaussian mechanism's closed form (q = 1), its exact (epsilon, delta)
curve, the Renyi divergence of the subsampled mixture integrated
numerically, and monotonicity and calibration properties."""
import math

import numpy as np
import pytest
from scipy import integrate
from scipy.optimize import brentq
from scipy.stats import norm

from paper_2609_40335_amd import accountant as acc


@pytest.mark.parametrize("sigma", [0.5, 1.1, 3.0])
@pytest.mark.parametrize("alpha", [2, 7, 64])
def test_full_batch_is_the_gaussian_mechanism(sigma, alpha):
    # q = 1: the Gaussian mechanism of sensitivity 1, RDP alpha / (2 sigma^2)
    assert acc.rdp_sampled_gaussian(1.0, sigma, alpha) == pytest.approx(alpha / (2 * sigma ** 2))
    # the binomial series at q -> 1 approaches the same value
    assert acc.rdp_sampled_gaussian(1 - 1e-12, sigma, alpha) == pytest.approx(
        alpha / (2 * sigma ** 2), rel=1e-6)


def _rdp_by_integration(q, sigma, alpha):
    """log E_{x ~ N(0, s^2)} [((1 - q) + q p1(x)/p0(x))^alpha] / (alpha - 1), with
    p1 = N(1, s^2): the Renyi divergence of the subsampled mixture from N(0, s^2).
    The integrand is evaluated in log space; its mass lies within 30 s of [0, alpha]."""
    def f(x):
        log_ratio = (2 * x - 1) / (2 * sigma ** 2)
        log_mix = np.logaddexp(math.log1p(-q), math.log(q) + log_ratio)
        return math.exp(-x * x / (2 * sigma ** 2) - math.log(sigma * math.sqrt(2 * math.pi))
                        + alpha * log_mix)
    val, _ = integrate.quad(f, -30 * sigma, alpha + 30 * sigma, epsabs=0, epsrel=1e-12,
                            limit=400, points=[0.0, float(alpha)])
    return math.log(val) / (alpha - 1)


@pytest.mark.parametrize("q,sigma,alpha", [(0.01, 0.8, 2), (0.01, 0.8, 3), (0.3, 2.0, 2),
                                           (0.3, 2.0, 5), (0.05, 1.2, 8)])
def test_series_matches_numerical_integration(q, sigma, alpha):
    assert acc.rdp_sampled_gaussian(q, sigma, alpha) == pytest.approx(
        _rdp_by_integration(q, sigma, alpha), rel=1e-8)


def test_monotonicity_and_limits():
    assert acc.rdp_sampled_gaussian(0.0, 1.0, 8) == 0.0
    r = [acc.rdp_sampled_gaussian(0.02, s, 16) for s in (0.6, 0.9, 1.5, 4.0)]
    assert all(a > b for a, b in zip(r, r[1:]))           # more noise, less privacy loss
    r = [acc.rdp_sampled_gaussian(q, 1.0, 16) for q in (0.001, 0.01, 0.1)]
    assert all(a < b for a, b in zip(r, r[1:]))           # larger batches, more loss
    e = [acc.epsilon(0.01, 1.0, T, 1e-5) for T in (100, 1000, 10000)]
    assert all(a < b for a, b in zip(e, e[1:]))           # composition


def test_conversion_uses_the_best_order():
    rdp = [1.0, 0.5, 0.8]
    orders = [2, 8, 32]
    eps, a = acc.epsilon_from_rdp(rdp, orders, 1e-5)
    by_hand = [r + math.log((o - 1) / o) - (math.log(1e-5) + math.log(o)) / (o - 1)
               for r, o in zip(rdp, orders)]
    assert eps == pytest.approx(min(by_hand)) and a == orders[int(np.argmin(by_hand))]


@pytest.mark.parametrize("target", [1.0, 3.0, 5.0])
def test_calibration_meets_the_budget_tightly(target):
    # the paper's SST-2 setting: N = 67349, batch 24 (q = 24 / N), 10 epochs, delta = N^-1.1
    n = 67349
    q = 24 / n
    steps = int(math.ceil(10 / q))
    delta = acc.paper_delta(n)
    s = acc.calibrate_sigma(target, delta, q, steps)
    assert acc.epsilon(q, s, steps, delta) <= target
    assert acc.epsilon(q, s * (1 - 1e-3), steps, delta) > target
    assert 0.3 < s < 10


def test_invalid_arguments():
    with pytest.raises(ValueError):
        acc.rdp_sampled_gaussian(1.5, 1.0, 4)
    with pytest.raises(ValueError):
        acc.rdp_sampled_gaussian(0.1, 0.0, 4)
    with pytest.raises(ValueError):
        acc.rdp_sampled_gaussian(0.1, 1.0, 1)
    with pytest.raises(ValueError):
        acc.epsilon_from_rdp([1.0], [2], 0.0)


# ---------------------------------------------------------------------------
# The conversion to (epsilon, delta), pinned by the exact privacy curve of the
# Gaussian mechanism (Balle & Wang, "Improving the Gaussian Mechanism for
# Differential Privacy", 2018, Thm. 8): with sensitivity 1 and noise std s,
#   delta(eps) = Phi(1/(2s) - eps s) - e^eps Phi(-1/(2s) - eps s).
# Any valid RDP conversion gives an epsilon at or above the exact one.
# ---------------------------------------------------------------------------
def _exact_gaussian_epsilon(delta, s):
    def d(e):
        return norm.cdf(1 / (2 * s) - e * s) - math.exp(e) * norm.cdf(-1 / (2 * s) - e * s)
    if d(0.0) <= delta:
        return 0.0
    return brentq(lambda e: d(e) - delta, 0.0, 500.0, xtol=1e-12)


GAUSS_CASES = [(s, d) for s in (0.5, 0.8, 1.0, 2.0, 5.0, 20.0) for d in (1e-5, 1e-8)]


def check_conversion_against_exact_gaussian(a):
    """One full-batch step (q = 1) is the Gaussian mechanism: the accountant's
    epsilon lies at or above the exact epsilon at the same delta (a lower
    value would overstate the privacy), and within 12 % + 0.01 of it (the
    looseness of the RDP route with integer orders, 5-11 % over these cases;
    the classic conversion eps_RDP + log(1/delta)/(alpha-1) is 16-50 % above)."""
    for s, d in GAUSS_CASES:
        exact = _exact_gaussian_epsilon(d, s)
        got = a.epsilon(1.0, s, 1, d)
        assert got >= exact * (1 - 1e-9), (s, d, got, exact)
        assert got <= 1.12 * exact + 0.01, (s, d, got, exact)


def test_conversion_against_exact_gaussian():
    check_conversion_against_exact_gaussian(acc)


@pytest.mark.parametrize("k", [2, 10, 1000])
def test_full_batch_steps_compose_like_one_step(k):
    # k Gaussian mechanisms of noise s compose to one of noise s / sqrt(k)
    # (the privacy loss random variables add); the exact epsilon of the
    # composition is that one step's, and the accountant matches both facts
    for s, d in [(1.0, 1e-5), (4.0, 1e-6), (30.0, 1e-8)]:
        if s / math.sqrt(k) < 0.5:
            continue        # epsilon beyond ~20: outside the curve's useful range
        many = acc.epsilon(1.0, s, k, d)
        one = acc.epsilon(1.0, s / math.sqrt(k), 1, d)
        assert many == pytest.approx(one, rel=1e-12)
        assert many >= _exact_gaussian_epsilon(d, s / math.sqrt(k)) * (1 - 1e-9)


def _classic_conversion(rdp, orders, delta):
    best = min((r + math.log(1 / delta) / (a - 1), a) for r, a in zip(rdp, orders))
    return max(best[0], 0.0), best[1]


def _sign_slip_conversion(rdp, orders, delta):
    best = min((r - math.log((a - 1) / a) - (math.log(delta) + math.log(a)) / (a - 1), a)
               for r, a in zip(rdp, orders))
    return max(best[0], 0.0), best[1]


@pytest.mark.parametrize("bad", [_classic_conversion, _sign_slip_conversion],
                         ids=["classic", "sign-slip"])
def test_pins_catch_a_wrong_conversion(monkeypatch, bad):
    monkeypatch.setattr(acc, "epsilon_from_rdp", bad)
    with pytest.raises(AssertionError):
        check_conversion_against_exact_gaussian(acc)


def test_classic_conversion_changes_the_paper_sigma(monkeypatch):
    # the paper's SST-2 setting (N = 67349, batch 24, 10 epochs, delta = N^-1.1,
    # epsilon = 3): the conversion in use is visible in the calibrated sigma
    n = 67349
    q = 24 / n
    steps = int(math.ceil(10 / q))
    delta = acc.paper_delta(n)
    s = acc.calibrate_sigma(3.0, delta, q, steps)
    monkeypatch.setattr(acc, "epsilon_from_rdp", _classic_conversion)
    s_classic = acc.calibrate_sigma(3.0, delta, q, steps)
    assert s_classic > s * 1.01
