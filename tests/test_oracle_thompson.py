"""Pins of the oracle's posterior-sampling priority (the index-policy
proposition's alternative to ordering by p_eff; reading in
oracle/thompson.py): the order-statistic draw has the Beta law, the index
averages to Eq. peff over the draw, and the priority never changes a verdict."""
import math

import numpy as np
import pytest
from scipy import stats

from oracle import controller as C
from oracle import predictor as P
from oracle import thompson as T

SEED = 0x1234_5678_9ABC_DEF0


@pytest.mark.parametrize("a,b", [(1, 1), (1, 5), (3, 2), (2, 7), (6, 1)])
def test_order_statistic_draw_is_beta(a, b):
    """The a-th smallest of a + b - 1 uniforms is Beta(a, b): KS test over
    4000 independent counters (uids)."""
    m = a + b - 1
    g = np.array([(T.order_statistic_word(SEED, 3, u, 0, a, m) + 0.5) * 2.0 ** -32 for u in range(4000)])
    res = stats.kstest(g, stats.beta(a, b).cdf)
    assert res.pvalue > 1e-3


@pytest.mark.parametrize("n,s,a0,b0", [(0, 0, 1.0, 1.0), (2, 0, 1.0, 1.0), (3, 3, 1.0, 1.0),
                                       (4, 0, 2.0, 3.0), (1, 1, 1.0, 4.0), (0, 0, 3.0, 1.0)])
def test_index_averages_to_peff(n, s, a0, b0):
    """E over the posterior draw of P(mixed group | g) is Eq. peff (the two
    orderings share their fixed points): Monte Carlo mean within 5 sigma."""
    k, N = 8, 6000
    x = np.array([T.index(SEED, 5, u, n, s, k, a0, b0) for u in range(N)])
    pe = P.p_eff(n, s, k, a0, b0)
    se = x.std(ddof=1) / math.sqrt(N)
    assert abs(x.mean() - pe) < 5 * se + 1e-12


def test_index_special_cases():
    k = 8
    assert T.index(SEED, 0, 7, 3, 1, k, 1.0, 1.0) == 1.0          # mixed
    assert T.index(SEED, 0, 7, 8, 0, k, 1.0, 1.0) == 0.0          # complete and unmixed
    # non-integer posterior parameters keep the p_eff index
    assert T.index(SEED, 0, 7, 2, 0, k, 1.5, 1.0) == P.p_eff(2, 0, k, 1.5, 1.0)
    # a draw is a pure function of (seed, step, uid, n): same inputs, same index
    assert T.index(SEED, 2, 9, 2, 0, k, 1.0, 1.0) == T.index(SEED, 2, 9, 2, 0, k, 1.0, 1.0)
    assert T.index(SEED, 2, 9, 2, 0, k, 1.0, 1.0) != T.index(SEED, 3, 9, 2, 0, k, 1.0, 1.0)
    # the a-th smallest: a = 1 is the minimum, a = m the maximum of the words
    from oracle.philox import philox4x32
    from oracle.sampler import key_of
    k0, k1 = key_of(SEED, 4)
    w = [int(v) for v in philox4x32(11, 0, 0, 2, k0, k1).reshape(-1)] + \
        [int(v) for v in philox4x32(11, 0, 1, 2, k0, k1).reshape(-1)]
    assert T.order_statistic_word(SEED, 4, 11, 0, 1, 7) == min(w[:7])
    assert T.order_statistic_word(SEED, 4, 11, 0, 7, 7) == max(w[:7])


def test_priority_never_changes_a_verdict():
    """With binding slots the two orderings assign rollouts differently, but
    every prompt's verdict depends only on its own outcome sequence."""
    from tests.test_oracle_controller import alloc, mixture_p, synthetic
    U = 400
    p = mixture_p(U, 23)
    Ls = np.random.default_rng(8).integers(1, 30, size=(U, 8))
    out = synthetic(p, lengths=lambda u, j: Ls[u, j])
    a = alloc(n_slots=24)
    ref = C.simulate(a, U, out)
    ts = C.simulate(dict(a, mode="sara_thompson"), U, out, draw_key=(SEED, 0))
    assert ts["log_assign"] != ref["log_assign"]
    for u in range(U):
        if ref["status"][u] and ts["status"][u]:
            assert (ts["status"][u], ts["n_done"][u], ts["successes"][u]) == (
                ref["status"][u], ref["n_done"][u], ref["successes"][u])
