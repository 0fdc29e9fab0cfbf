"""Beta-posterior effectiveness predictor and the SARA decision rule (oracle).

Paper references:
* Beta prior / conjugate posterior Beta(a0+s, b0+n-s): section 3.2.
* Closed-form predictor p_eff(n, s): Proposition 1, Eq. peff; proof in the
  appendix (Beta-function identity E[g^u (1-g)^v] = B(a+u, b+v) / B(a, b)).
* Two-threshold rule decide(n, s): Eq. decide, with the commit floor of the
  implementation-details appendix (commit_min, default k).

Readings where the paper is silent or ambiguous:
* n = 0: both the all-fail and the all-pass branch of Eq. peff apply; the
  predictor subtracts both saturation probabilities, giving
  1 - B(a0, b0+k)/B(a0, b0) - B(a0+k, b0)/B(a0, b0) (7/9 at k = 8, uniform prior).
* Abandon uses the strict comparison p_eff < tau, and a complete unmixed
  group (n = k) is abandoned (p_eff = 0), which makes tau -> 0 lossless.
* A mixed group below the commit floor continues with commit_min - n more
  rollouts at once; an unmixed group continues with one more rollout.

Pinned by tests: exact rationals, Polya-urn brute force, Monte Carlo, the
paper's uniform-prior simplification (k - n)/(k + 1), monotonicity.
"""
import math

COMMIT, ABANDON, CONTINUE = 1, 2, 3


def log_beta(a: float, b: float) -> float:
    return math.lgamma(a) + math.lgamma(b) - math.lgamma(a + b)


def posterior(n: int, s: int, alpha0: float = 1.0, beta0: float = 1.0):
    """Conjugate update: Beta(alpha0 + s, beta0 + n - s)."""
    return alpha0 + s, beta0 + (n - s)


def is_mixed(n: int, s: int) -> bool:
    return s >= 1 and (n - s) >= 1


def p_eff(n: int, s: int, k: int, alpha0: float = 1.0, beta0: float = 1.0) -> float:
    """P(the completed group of size k is mixed | n observed, s successes)."""
    if is_mixed(n, s):
        return 1.0
    r = k - n
    if r <= 0:
        return 0.0
    a, b = posterior(n, s, alpha0, beta0)
    lb = log_beta(a, b)
    p_sat = 0.0
    if s == 0:      # remaining r rollouts all fail
        p_sat += math.exp(log_beta(a, b + r) - lb)
    if s == n:      # remaining r rollouts all pass
        p_sat += math.exp(log_beta(a + r, b) - lb)
    return 1.0 - p_sat


def decide(n: int, s: int, k: int, commit_min: int, tau: float,
           alpha0: float = 1.0, beta0: float = 1.0):
    """Returns (decision, p_eff, n_more) for a quiescent prompt."""
    pe = p_eff(n, s, k, alpha0, beta0)
    mixed = is_mixed(n, s)
    if mixed and n >= commit_min:
        return COMMIT, pe, 0
    if n >= k:
        return ABANDON, pe, 0
    if (not mixed) and pe < tau:
        return ABANDON, pe, 0
    return CONTINUE, pe, (commit_min - n) if mixed else 1


def priority_key(pe: float, bits: int = 20) -> int:
    """Quantised yield index used to order pending rollouts (larger first)."""
    return int(math.floor(pe * float(1 << bits) + 0.5))
