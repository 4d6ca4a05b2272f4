"""The privacy accountant against facts it does not compute the same way:
the Gaussian mechanism's closed form (q = 1), the Renyi divergence of the
subsampled mixture integrated numerically, and monotonicity and calibration
properties."""
import math

import numpy as np
import pytest
from scipy import integrate

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
