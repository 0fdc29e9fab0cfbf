"""Pins of the oracle's history warm start (implementation details,
"defaults and history warm-start"; reading in oracle/warm.py): the warm
prior against a closed form of Eq. peff, the abandonment times it implies
for saturated prompts revisited across steps, and the cold-start limit."""
import math

import numpy as np
import pytest

from oracle import controller as C
from oracle import predictor as P
from oracle import warm as WS


def alloc(**kw):
    a = dict(B=64, k=8, n0=2, commit_min=8, tau_low=0.45, alpha0=1.0, beta0=1.0,
             budget_N=10 ** 6, n_slots=4096, mode="sara", prio_quant_bits=20)
    a.update(kw)
    return a


def outcomes_of(p, step):
    """Bernoulli(p_set) outcomes keyed by (step, set prompt, j)."""
    def out(pairs, ids):
        res = []
        for (u, j) in pairs:
            g = np.random.default_rng([step, int(ids[u]), j])
            res.append((1, int(g.random() < p[ids[u]])))
        return res
    return out


def run_steps(a, p_set, pools, lam, warm=True):
    """Allocation steps over pools of set ids; returns per-step results and
    the final pseudo-counts."""
    D = len(p_set)
    ca, cb = [0.0] * D, [0.0] * D
    out = []
    for t, ids in enumerate(pools):
        pri = WS.priors(ids, ca, cb, a["alpha0"], a["beta0"]) if warm else None
        o = outcomes_of(p_set, t)
        res = C.simulate(a, len(ids), lambda pairs: o(pairs, ids), priors=pri)
        out.append(res)
        ca, cb = WS.update(ca, cb, list(ids), res["n_done"], res["successes"], res["drawn"], lam)
    return out, ca, cb


@pytest.mark.parametrize("b", [0.0, 1.5, 4.0, 7.0, 12.5])
def test_warm_prior_peff_closed_form(b):
    """Under a prior Beta(1, 1 + b) (b pseudo-failures carried over), an
    all-fail prefix of n gives p_eff = 1 - B(1, 1+b+k)/B(1, 1+b+n) =
    (k - n)/(1 + b + k) for n >= 1 (Eq. peff, s = 0 branch: the ratio of Beta
    functions with first argument 1 telescopes); at n = 0 both saturation
    terms apply, checked against the Beta-Binomial pmf."""
    k = 8
    for n in range(1, k + 1):
        assert P.p_eff(n, 0, k, 1.0, 1.0 + b) == pytest.approx((k - n) / (1 + b + k), abs=1e-13)
    # n = 0: 1 - P(all fail) - P(all pass) under Beta-Binomial(k, 1, 1+b)
    from scipy.stats import betabinom
    want = 1 - betabinom.pmf(0, k, 1.0, 1.0 + b) - betabinom.pmf(k, k, 1.0, 1.0 + b)
    assert P.p_eff(0, 0, k, 1.0, 1.0 + b) == pytest.approx(want, abs=1e-12)


def abandon_time(b, k=8, n0=2, tau=0.45):
    """First n >= n0 with (k - n)/(1 + b + k) < tau (all-fail prompt, prior Beta(1, 1+b))."""
    n = n0
    while n < k and not (k - n) / (1 + b + k) < tau:
        n += 1
    return n


@pytest.mark.parametrize("lam,expect", [(1.0, [4, 3, 2, 2, 2]), (0.5, [4, 4, 3, 3, 3]), (0.0, [4, 4, 4, 4, 4])])
def test_saturated_prompts_revisited(lam, expect):
    """A set of saturated prompts (p in {0, 1}) drawn in every step: with the
    counts carried as a <- lam (a + s), b <- lam (b + n - s), each prompt is
    abandoned at the first n >= n0 with (k - n)/(1 + c + k) < tau, c its
    carried count: 4, 3, 2, 2, .. rollouts at lam = 1 (c = 0, 4, 7, 9, ..),
    4, 4, 3, 3, .. at lam = 1/2 (c = 0, 2, 3, 3, ..) and always 4 cold."""
    D = 40
    p_set = np.random.default_rng(3).integers(0, 2, D).astype(float)
    pools = [np.arange(D, dtype=np.int32)] * 5
    a = alloc()
    res, ca, cb = run_steps(a, p_set, pools, lam)
    c = 0.0
    for t, r in enumerate(res):
        assert r["drawn"] == D and r["n_committed"] == 0
        assert abandon_time(c) == expect[t]
        for u in range(D):
            assert r["n_done"][u] == expect[t]
            assert r["status"][u] == C.ABANDONED
        c = lam * (c + expect[t])
    # all-fail prompts carry failures, all-pass prompts successes (the
    # symmetric prior gives the same abandonment times)
    for i in range(D):
        carried = (cb[i], ca[i]) if p_set[i] == 0 else (ca[i], cb[i])
        assert carried[1] == 0.0 and carried[0] == pytest.approx(c)


def test_cold_start_limit_and_undrawn_decay():
    """lam = 0 reproduces cold steps exactly; prompts a step does not draw
    only decay."""
    D, U = 300, 120
    g = np.random.default_rng(11)
    p_set = g.random(D)
    pools = [g.choice(D, U, replace=False).astype(np.int32) for _ in range(3)]
    a = alloc(B=16, budget_N=256, n_slots=64)
    warm, _, _ = run_steps(a, p_set, pools, 0.0)
    cold, _, _ = run_steps(a, p_set, pools, 0.0, warm=False)
    for w, c in zip(warm, cold):
        assert w["log_decisions"] == c["log_decisions"] and w["log_assign"] == c["log_assign"]
    # one step at lam = 1/2 by hand
    ca, cb = [1.0] * D, [2.0] * D
    r = C.simulate(a, U, lambda pairs: outcomes_of(p_set, 0)(pairs, pools[0]),
                   priors=WS.priors(pools[0], ca, cb, 1.0, 1.0))
    na, nb = WS.update(ca, cb, list(pools[0]), r["n_done"], r["successes"], r["drawn"], 0.5)
    drawn = {int(pools[0][u]): u for u in range(r["drawn"])}
    for i in range(D):
        if i in drawn:
            u = drawn[i]
            assert na[i] == 0.5 * (1.0 + r["successes"][u])
            assert nb[i] == 0.5 * (2.0 + r["n_done"][u] - r["successes"][u])
        else:
            assert (na[i], nb[i]) == (0.5, 1.0)


def test_warm_start_saves_rollouts_on_a_revisited_mixture():
    """On a revisited set drawn from the success-rate mixture, carried
    posteriors lower the rollouts per drawn prompt of later steps (saturated
    prompts are abandoned sooner) while the commit rate stays within noise."""
    from tests.test_oracle_controller import mixture_p
    D = 2000
    p_set = mixture_p(D, 17)
    pools = [np.arange(D, dtype=np.int32)] * 3
    a = alloc(B=10 ** 6)
    res_w, _, _ = run_steps(a, p_set, pools, 1.0)
    res_c, _, _ = run_steps(a, p_set, pools, 1.0, warm=False)
    rw = res_w[2]["rollouts"] / res_w[2]["drawn"]
    rc = res_c[2]["rollouts"] / res_c[2]["drawn"]
    assert rw < rc - 0.3
    cw = res_w[2]["n_committed"] / D
    cc = res_c[2]["n_committed"] / D
    assert abs(cw - cc) < 0.05
