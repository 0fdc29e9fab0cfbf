"""Pins of the oracle's predictor and decision rule against what the paper
and the mathematics fix (Prop. 1 / Eq. peff, Prop. 2, Eq. decide, Thm. 1-2)."""
import itertools
import math
import random
from fractions import Fraction

import mpmath
import numpy as np
import pytest
from scipy import stats

from oracle import predictor as P


def urn_p_mixed(n, s, k, a0: Fraction, b0: Fraction) -> Fraction:
    """Brute force: enumerate all 2^(k-n) completions with Polya-urn
    (sequential posterior-predictive) probabilities, exact rationals."""
    r = k - n
    total = Fraction(0)
    for seq in itertools.product((0, 1), repeat=r):
        pr = Fraction(1)
        nn, ss = n, s
        for x in seq:
            p1 = (a0 + ss) / (a0 + b0 + nn)
            pr *= p1 if x else (1 - p1)
            nn += 1
            ss += x
        if 1 <= ss <= k - 1:
            total += pr
    return total


def test_uniform_prior_simplification():
    # section 3.2: p_eff(n, 0) = (k - n) / (k + 1) with a uniform prior, n >= 1
    k = 8
    for n in range(1, k + 1):
        assert P.p_eff(n, 0, k) == pytest.approx((k - n) / (k + 1), abs=1e-14)
        assert P.p_eff(n, n, k) == pytest.approx((k - n) / (k + 1), abs=1e-14)
    # n = 0: both saturation branches apply -> 1 - 2/(k+1)
    assert P.p_eff(0, 0, k) == pytest.approx(7 / 9, abs=1e-14)


@pytest.mark.parametrize("k", [2, 3, 5, 8, 10])
def test_against_polya_urn_bruteforce(k):
    rng = random.Random(k)
    priors = [(Fraction(1), Fraction(1)), (Fraction(1, 2), Fraction(3, 2))] + [
        (Fraction(rng.randint(1, 40), 10), Fraction(rng.randint(1, 40), 10)) for _ in range(3)]
    for a0, b0 in priors:
        for n in range(0, k + 1):
            for s in range(0, n + 1):
                exact = urn_p_mixed(n, s, k, a0, b0)
                got = P.p_eff(n, s, k, float(a0), float(b0))
                assert abs(got - float(exact)) < 1e-13, (k, a0, b0, n, s)


def test_against_betabinomial_pmf_at_n0():
    # a fresh group's success count is Beta-Binomial(k, a0, b0)
    for (k, a0, b0) in [(8, 1.0, 1.0), (8, 0.3, 3.0), (6, 2.5, 0.7), (12, 1.7, 1.9)]:
        bb = stats.betabinom(k, a0, b0)
        assert P.p_eff(0, 0, k, a0, b0) == pytest.approx(1 - bb.pmf(0) - bb.pmf(k), abs=1e-13)


def test_against_mpmath_high_precision():
    mpmath.mp.dps = 40
    rng = random.Random(3)
    for _ in range(200):
        k = rng.randint(2, 16)
        n = rng.randint(0, k)
        s = rng.choice([0, n])
        a0, b0 = rng.uniform(0.1, 5), rng.uniform(0.1, 5)
        a, b, r = a0 + s, b0 + n - s, k - n
        ref = mpmath.mpf(1)
        if r == 0:
            ref = mpmath.mpf(1) if 1 <= s <= n - 1 else mpmath.mpf(0)
        else:
            lb = mpmath.log(mpmath.beta(a, b))
            if s == 0:
                ref -= mpmath.exp(mpmath.log(mpmath.beta(a, b + r)) - lb)
            if s == n:
                ref -= mpmath.exp(mpmath.log(mpmath.beta(a + r, b)) - lb)
        assert abs(P.p_eff(n, s, k, a0, b0) - float(ref)) < 1e-13


def test_monte_carlo():
    g = np.random.default_rng(11)
    for (n, s, k, a0, b0) in [(2, 0, 8, 1.0, 1.0), (3, 3, 8, 0.5, 0.5), (1, 0, 5, 2.0, 3.0)]:
        a, b = a0 + s, b0 + n - s
        M = 2_000_000
        gam = g.beta(a, b, size=M)
        x = g.binomial(k - n, gam)
        tot = x + s
        mixed = ((tot >= 1) & (tot <= k - 1)).mean()
        p = P.p_eff(n, s, k, a0, b0)
        assert abs(mixed - p) < 5 * math.sqrt(p * (1 - p) / M)


def test_conjugacy():
    # posterior density of gamma after (n, s) from Bayes' rule, numerically
    # normalised, equals the Beta(a0 + s, b0 + n - s) density
    mpmath.mp.dps = 30
    for (n, s, a0, b0) in [(4, 1, 1.0, 1.0), (6, 6, 0.3, 3.0), (3, 0, 2.0, 0.5)]:
        prior = lambda x: x ** (a0 - 1) * (1 - x) ** (b0 - 1)
        lik = lambda x: x ** s * (1 - x) ** (n - s)
        Z = mpmath.quad(lambda x: prior(x) * lik(x), [0, 0.5, 1])
        a, b = P.posterior(n, s, a0, b0)
        for x in (0.05, 0.3, 0.5, 0.77, 0.95):
            assert float(prior(x) * lik(x) / Z) == pytest.approx(stats.beta.pdf(x, a, b), rel=1e-9)
    # sequential updates commute: folding the outcomes in one at a time by
    # Bayes' rule on a grid (prior density times the likelihood of a single
    # outcome), in several orders, leaves a density proportional to the
    # Beta(a0 + s, b0 + n - s) density; the closed-form update applied one
    # observation at a time lands on the same parameters
    x = (np.arange(20000) + 0.5) / 20000
    rng = random.Random(11)
    for (a0, b0) in [(1.0, 1.0), (0.3, 3.0), (2.5, 0.7)]:
        outs = [1, 0, 0, 1, 1, 0, 1]
        want = stats.beta.pdf(x, *P.posterior(len(outs), sum(outs), a0, b0))
        perms = set()
        while len(perms) < 6:
            perm = outs[:]
            rng.shuffle(perm)
            perms.add(tuple(perm))
        for perm in perms:
            f = stats.beta.pdf(x, a0, b0)
            a, b = a0, b0
            for o in perm:
                f = f * (x if o else 1.0 - x)
                f = f / f.sum()
                a, b = P.posterior(1, o, a, b)
            assert (a, b) == P.posterior(len(outs), sum(outs), a0, b0)
            ratio = f[100:-100] / want[100:-100]
            assert ratio.max() / ratio.min() - 1.0 < 1e-9


def test_monotone_and_absorbing():
    rng = random.Random(5)
    for _ in range(100):
        k = rng.randint(2, 16)
        a0, b0 = rng.uniform(0.05, 8), rng.uniform(0.05, 8)
        fail = [P.p_eff(n, 0, k, a0, b0) for n in range(1, k + 1)]
        pas = [P.p_eff(n, n, k, a0, b0) for n in range(1, k + 1)]
        assert all(x > y for x, y in zip(fail, fail[1:]))
        assert all(x > y for x, y in zip(pas, pas[1:]))
        for n in range(2, k + 1):
            for s in range(1, n):
                assert P.p_eff(n, s, k, a0, b0) == 1.0


@pytest.mark.parametrize("tau,n_a", [(0.45, 4), (0.3, 6), (0.2, 7), (0.1, 8)])
def test_abandon_time(tau, n_a):
    k = 8
    # Thm. 2 proof: n_a = k - floor(tau (k + 1)) under the uniform prior
    assert n_a == k - math.floor(tau * (k + 1))
    for first in (0, 1):
        n = 2
        while True:
            s = n if first else 0
            d, pe, more = P.decide(n, s, k, k, tau)
            if d != P.CONTINUE:
                break
            assert more == 1
            n += 1
        assert d == P.ABANDON and n == n_a


def test_decide_truth_table_defaults():
    k, cm, tau = 8, 8, 0.45
    for n in range(2, k + 1):
        for s in range(0, n + 1):
            d, pe, more = P.decide(n, s, k, cm, tau)
            mixed = 1 <= s <= n - 1
            if mixed:
                assert (d, more) == ((P.COMMIT, 0) if n == k else (P.CONTINUE, k - n))
            else:
                assert d == (P.ABANDON if n >= 4 else P.CONTINUE)
    # early-commit floor
    assert P.decide(3, 1, 8, 4, 0.45)[0] == P.CONTINUE
    assert P.decide(3, 1, 8, 4, 0.45)[2] == 1
    assert P.decide(4, 1, 8, 4, 0.45)[0] == P.COMMIT
    # tau = 0: nothing is abandoned before n = k (lossless limit, Thm. 1)
    for n in range(1, 8):
        assert P.decide(n, 0, 8, 8, 0.0)[0] == P.CONTINUE
    assert P.decide(8, 0, 8, 8, 0.0)[0] == P.ABANDON
    # p_eff == tau continues (strict comparison, taken on the fp64 value)
    assert P.decide(4, 0, 8, 8, P.p_eff(4, 0, 8))[0] == P.CONTINUE
    assert P.decide(4, 0, 8, 8, math.nextafter(P.p_eff(4, 0, 8), 1.0))[0] == P.ABANDON


def test_reliability_calibration_under_prior():
    """Thm. 1: with gamma drawn from the prior, the fraction of abandoned
    groups that would have been mixed is exactly p_eff at abandonment (4/9)."""
    g = np.random.default_rng(2)
    M = 400_000
    gam = g.random(M)
    x = g.random((M, 8)) < gam[:, None]
    first4 = x[:, :4].sum(1)
    aband = (first4 == 0) | (first4 == 4)
    tot = x.sum(1)
    lost = aband & (tot >= 1) & (tot <= 7)
    frac = lost.sum() / aband.sum()
    assert abs(frac - P.p_eff(4, 0, 8)) < 5 * math.sqrt(0.25 / aband.sum())
    assert P.p_eff(4, 0, 8) < 0.45


def test_priority_key():
    assert P.priority_key(1.0) == 1 << 20
    assert P.priority_key(0.0) == 0
    assert P.priority_key(0.5) == 1 << 19
    # round half up, not floor: 2^20 * 2/3 = 699050.67, 2^20 * 4/9 = 466033.78,
    # 2^20 * 5/9 = 582542.22, and 1.5 / 2^20 sits on a half
    assert P.priority_key(2 / 3) == 699051
    assert P.priority_key(4 / 9) == 466034
    assert P.priority_key(5 / 9) == 582542
    assert P.priority_key(7 / 9) == 815559
    assert P.priority_key(1.5 / (1 << 20)) == 2
    assert P.priority_key(2 / 3, bits=4) == 11
