"""Privacy accounting for the DP-SGD step: the noise multiplier sigma that a
privacy budget (epsilon, delta) allows, on the host.

The paper trains with a target epsilon (3, and 1 or 5 in its ablations) and
delta = N^-1.1 for a training set of N examples (Sec. "Training
Configurations"); sigma is then whatever the accountant of the training
library returns. This module is that accountant, written from the published
analyses:

  * one DP-SGD step on a Poisson-subsampled batch (each example kept with
    probability q) with Gaussian noise of standard deviation sigma * C on a
    sum of per-example gradients clipped to norm C is the sampled Gaussian
    mechanism; its Renyi differential privacy at integer order alpha >= 2 is
        eps_RDP(alpha) = log(A_alpha) / (alpha - 1),
        A_alpha = sum_{k=0}^{alpha} binom(alpha, k) (1-q)^(alpha-k) q^k
                  exp((k^2 - k) / (2 sigma^2))
    (Mironov, Talwar, Zhang, "Renyi Differential Privacy of the Sampled
    Gaussian Mechanism", 2019, Sec. 3.3), evaluated in log space;
  * RDP composes additively over steps;
  * an RDP guarantee converts to (epsilon, delta) by
        epsilon = eps_RDP + log((alpha-1)/alpha) - (log delta + log alpha)/(alpha-1)
    minimised over alpha (Balle, Barthe, Gaboardi, Hsu, Sato, "Hypothesis
    Testing Interpretations and Renyi Differential Privacy", 2020, Thm. 21).

Integer orders only; fractional orders would tighten epsilon slightly.
"""
from __future__ import annotations

import math
from typing import Iterable, Optional, Sequence

__all__ = ["DEFAULT_ORDERS", "rdp_sampled_gaussian", "epsilon_from_rdp", "epsilon",
           "calibrate_sigma", "paper_delta"]

DEFAULT_ORDERS = tuple(range(2, 65)) + (80, 96, 128, 160, 192, 256, 384, 512, 1024)


def _logsumexp(xs: Sequence[float]) -> float:
    m = max(xs)
    if m == -math.inf:
        return -math.inf
    return m + math.log(sum(math.exp(x - m) for x in xs))


def rdp_sampled_gaussian(q: float, sigma: float, alpha: int) -> float:
    """RDP of one step of the sampled Gaussian mechanism at integer order alpha."""
    if not (0.0 <= q <= 1.0):
        raise ValueError("q must lie in [0, 1]")
    if not sigma > 0:
        raise ValueError("sigma must be positive")
    if int(alpha) != alpha or alpha < 2:
        raise ValueError("alpha must be an integer >= 2")
    alpha = int(alpha)
    if q == 0.0:
        return 0.0
    if q == 1.0:
        return alpha / (2.0 * sigma * sigma)
    lq, l1q = math.log(q), math.log1p(-q)
    terms = []
    for k in range(alpha + 1):
        lbin = math.lgamma(alpha + 1) - math.lgamma(k + 1) - math.lgamma(alpha - k + 1)
        terms.append(lbin + (alpha - k) * l1q + k * lq + (k * k - k) / (2.0 * sigma * sigma))
    return _logsumexp(terms) / (alpha - 1)


def epsilon_from_rdp(rdp: Sequence[float], orders: Sequence[int], delta: float):
    """(epsilon, best order) from per-order RDP values of the whole run."""
    if not (0.0 < delta < 1.0):
        raise ValueError("delta must lie in (0, 1)")
    best, best_a = math.inf, None
    for r, a in zip(rdp, orders):
        e = r + math.log((a - 1) / a) - (math.log(delta) + math.log(a)) / (a - 1)
        if e < best:
            best, best_a = e, a
    return max(best, 0.0), best_a


def epsilon(q: float, sigma: float, steps: int, delta: float,
            orders: Iterable[int] = DEFAULT_ORDERS) -> float:
    """Epsilon after `steps` DP-SGD steps at sampling rate q and noise multiplier sigma."""
    orders = tuple(orders)
    rdp = [steps * rdp_sampled_gaussian(q, sigma, a) for a in orders]
    return epsilon_from_rdp(rdp, orders, delta)[0]


def calibrate_sigma(target_epsilon: float, delta: float, q: float, steps: int,
                    orders: Iterable[int] = DEFAULT_ORDERS, rel_tol: float = 1e-4,
                    sigma_max: float = 1e4) -> float:
    """Smallest noise multiplier (to rel_tol) whose run stays within target_epsilon."""
    if not target_epsilon > 0:
        raise ValueError("target_epsilon must be positive")
    orders = tuple(orders)
    lo, hi = 1e-3, 1.0
    while epsilon(q, hi, steps, delta, orders) > target_epsilon:
        lo, hi = hi, hi * 2.0
        if hi > sigma_max:
            raise ValueError("no noise multiplier below sigma_max meets the budget")
    while hi - lo > rel_tol * hi:
        mid = 0.5 * (lo + hi)
        if epsilon(q, mid, steps, delta, orders) > target_epsilon:
            lo = mid
        else:
            hi = mid
    return hi


def paper_delta(n_train: int) -> float:
    """delta = N^-1.1, the paper's choice for a training set of N examples."""
    return float(n_train) ** -1.1


def _main(argv: Optional[Sequence[str]] = None) -> int:
    import argparse
    ap = argparse.ArgumentParser(description="noise multiplier for a DP-SGD privacy budget")
    ap.add_argument("--epsilon", type=float, required=True)
    ap.add_argument("--n-train", type=int, required=True, help="training-set size N")
    ap.add_argument("--batch", type=int, required=True, help="expected batch size (q = batch / N)")
    ap.add_argument("--epochs", type=float, required=True)
    ap.add_argument("--delta", type=float, default=None, help="default: N^-1.1")
    a = ap.parse_args(argv)
    q = a.batch / a.n_train
    steps = int(math.ceil(a.epochs / q))
    delta = a.delta if a.delta is not None else paper_delta(a.n_train)
    s = calibrate_sigma(a.epsilon, delta, q, steps)
    print(f"q={q:.6g} steps={steps} delta={delta:.3g} sigma={s:.4f} "
          f"epsilon={epsilon(q, s, steps, delta):.4f}")
    return 0


if __name__ == "__main__":
    raise SystemExit(_main())
