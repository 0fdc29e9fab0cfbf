"""Pins of the oracle's allocation step (Algorithm 1 on the slot clock)
against closed forms of the rule, the paper's theorems and invariants."""
import math

import numpy as np
import pytest
from scipy.special import betaln

from oracle import controller as C
from oracle import predictor as P


def alloc(**kw):
    a = dict(B=64, k=8, n0=2, commit_min=8, tau_low=0.45, alpha0=1.0, beta0=1.0,
             budget_N=512, n_slots=512, mode="sara", prio_quant_bits=20)
    a.update(kw)
    return a


def synthetic(p, lengths=None, seed=0):
    """Bernoulli(p_uid) outcomes, schedule independent (keyed by uid, j)."""
    def outcomes(pairs):
        out = []
        for (u, j) in pairs:
            g = np.random.default_rng([seed, u, j])
            L = 1 if lengths is None else int(lengths(u, j))
            out.append((L, int(g.random() < p[u])))
        return out
    return outcomes


def mixture_p(U, seed, weights=(0.4, 0.3, 0.3)):
    g = np.random.default_rng(seed)
    c = g.choice(3, size=U, p=list(weights))
    return np.where(c == 0, g.beta(0.3, 3, U), np.where(c == 1, g.beta(3, 0.3, U), g.random(U)))


def moment(n, m):
    """E[g^n] and E[(1-g)^n] under the 0.4 Beta(.3,3) / 0.3 Beta(3,.3) / 0.3 U(0,1) mixture."""
    e1 = 0.4 * math.exp(betaln(0.3 + n, 3) - betaln(0.3, 3)) + 0.3 * math.exp(
        betaln(3 + n, 0.3) - betaln(3, 0.3)) + 0.3 / (n + 1)
    e0 = 0.4 * math.exp(betaln(0.3, 3 + n) - betaln(0.3, 3)) + 0.3 * math.exp(
        betaln(3, 0.3 + n) - betaln(3, 0.3)) + 0.3 / (n + 1)
    return e1 + e0


def check_invariants(a, res, U):
    k = a["k"]
    assert res["rollouts"] <= a["budget_N"]
    # k reserved per draw, k - n refunded at the verdict: what is left is N - spent
    assert res["budget_left"] == a["budget_N"] - res["rollouts"]
    if a["mode"] == "sara":
        assert res["n_committed"] <= a["B"]
    for u in range(res["drawn"]):
        n, s = res["n_done"][u], res["successes"][u]
        assert n == res["n_issued"][u]
        if res["status"][u] == C.COMMITTED:
            assert 1 <= s <= n - 1 and n >= a["commit_min"]
        else:
            assert res["status"][u] == C.ABANDONED
            assert s in (0, n) or n < a["commit_min"]
    # a slot never holds two rollouts at once
    busy = {}
    for (t0, slot, u, j) in res["log_assign"]:
        L = res["rollout"][(u, j)][0]
        for (a0, b0) in busy.get(slot, []):
            assert t0 > b0 or t0 + L - 1 < a0
        busy.setdefault(slot, []).append((t0, t0 + L - 1))


def round_synchronous(a, p_outcome, U):
    """Algorithm 1 written as synchronous rounds (equal lengths, ample slots)."""
    B, k, n0, cm, tau = a["B"], a["k"], a["n0"], a["commit_min"], a["tau_low"]
    budget, nxt, act, done_c = a["budget_N"], 0, {}, []
    stats = {}

    def draw():
        nonlocal budget, nxt
        while len(act) < B - len(done_c) and budget >= k and nxt < U:
            act[nxt] = n0
            stats[nxt] = [0, 0]
            budget -= k
            nxt += 1

    draw()
    while act:
        for u, cnt in list(act.items()):
            for _ in range(cnt):
                n, s = stats[u]
                stats[u] = [n + 1, s + p_outcome(u, n)]
        for u in sorted(act):
            n, s = stats[u]
            d, pe, more = P.decide(n, s, k, cm, tau)
            if d == P.CONTINUE:
                act[u] = more
            else:
                del act[u]
                budget += k - n
                if d == P.COMMIT:
                    done_c.append(u)
        draw()
    return sorted(done_c), stats, budget


def test_reduces_to_round_synchronous_algorithm():
    U = 400
    p = mixture_p(U, 1)
    a = alloc()
    out = synthetic(p)
    res = C.simulate(a, U, out)
    po = lambda u, j: out([(u, j)])[0][1]
    com, stats, budget = round_synchronous(a, po, U)
    assert res["committed"] == com
    assert res["budget_left"] == budget
    for u, (n, s) in stats.items():
        assert (res["n_done"][u], res["successes"][u]) == (n, s)
    check_invariants(a, res, U)


def test_closed_form_statistics_under_mixture():
    """P(commit | drawn) = 1 - E[g^4 + (1-g)^4]; rollouts per drawn prompt = 4 + 4 P(commit);
    lost fraction among abandoned = (E4 - E8) / E4 (decisions at n = 2, 3, 4)."""
    U = 20000
    p = mixture_p(U, 7)
    a = alloc(B=10 ** 6, budget_N=10 ** 7, n_slots=4096)
    res = C.simulate(a, U, synthetic(p, seed=3))
    drawn = res["drawn"]
    assert drawn == U
    pc = 1 - moment(4, 0)
    got_pc = res["n_committed"] / drawn
    assert abs(got_pc - pc) < 5 * math.sqrt(pc * (1 - pc) / drawn)
    assert abs(pc - 0.3438) < 1e-4
    got_roll = res["rollouts"] / drawn
    assert abs(got_roll - (4 + 4 * pc)) < 5 * 4 * math.sqrt(pc * (1 - pc) / drawn)
    # rollouts per effective group below fixed-k's k / Phi (Thm. 2)
    phi = 1 - moment(8, 0)
    assert abs(phi - 0.4707) < 1e-4
    assert (4 + 4 * pc) / pc < 8 / phi
    # counterfactual loss: abandoned prompts whose full group would have mixed
    g_lost, g_ab = 0, 0
    for u in range(drawn):
        if res["status"][u] == C.ABANDONED:
            g_ab += 1
            outs = synthetic(p, seed=3)([(u, j) for j in range(8)])
            s = sum(r for _, r in outs)
            g_lost += 1 <= s <= 7
    lost = (moment(4, 0) - moment(8, 0)) / moment(4, 0)
    assert abs(g_lost / g_ab - lost) < 5 * math.sqrt(lost * (1 - lost) / g_ab)
    assert g_lost / g_ab < 0.45   # Thm. 1 bound


def test_saturated_prompts_abandoned_after_probe():
    U = 300
    p = np.random.default_rng(4).integers(0, 2, U).astype(float)
    a = alloc()
    res = C.simulate(a, U, synthetic(p))
    assert res["n_committed"] == 0
    for u in range(res["drawn"]):
        assert res["status"][u] == C.ABANDONED and res["n_issued"][u] == 4
    assert res["rollouts"] == 4 * res["drawn"]
    check_invariants(a, res, U)


def test_fixed_budget_yield_dominance():
    """Thm. 3: at N = B k, SARA's expected effective groups >= Phi * B (uniform)."""
    B, k = 16, 8
    reps = 300
    phi = 1 - moment(8, 0)
    ys = []
    for r in range(reps):
        U = 200
        p = mixture_p(U, 100 + r)
        res = C.simulate(alloc(B=B, budget_N=B * k, n_slots=B * k), U, synthetic(p, seed=r))
        ys.append(res["n_committed"])
    m = np.mean(ys)
    se = np.std(ys) / math.sqrt(reps)
    assert m > phi * B + 2 * se
    assert abs(m - 8.19) < 5 * se


def test_ragged_lengths_and_binding_slots():
    U = 500
    p = mixture_p(U, 9)
    Ls = np.random.default_rng(5).integers(1, 40, size=(U, 8))
    for S in (1, 3, 17, 64, 512):
        a = alloc(n_slots=S)
        res = C.simulate(a, U, synthetic(p, lengths=lambda u, j: Ls[u, j]))
        check_invariants(a, res, U)
        # assignment within one refill uses ascending free slots and queue order
        by_t = {}
        for (t0, slot, u, j) in res["log_assign"]:
            by_t.setdefault(t0, []).append((slot, u, j))
        for t0, lst in by_t.items():
            slots = [x[0] for x in lst]
            assert slots == sorted(slots)
        # a prompt's verdict depends only on its own outcomes, not on the slots
        ref = C.simulate(alloc(n_slots=4096), U, synthetic(p, lengths=lambda u, j: Ls[u, j]))
        for u in range(U):
            if res["status"][u] and ref["status"][u]:
                assert (res["status"][u], res["n_done"][u], res["successes"][u]) == (
                    ref["status"][u], ref["n_done"][u], ref["successes"][u])
        tok = sum(Ls[u, j] for (u, j) in res["rollout"])
        assert res["tokens"] == tok


def test_pool_and_budget_exhaustion():
    p = mixture_p(10, 2)
    res = C.simulate(alloc(), 10, synthetic(p))       # pool binds
    assert res["drawn"] == 10 and res["n_committed"] < 64
    res = C.simulate(alloc(budget_N=20), 400, synthetic(p := mixture_p(400, 2)))  # budget binds
    assert res["rollouts"] <= 20
    res = C.simulate(alloc(budget_N=7), 400, synthetic(p))   # below one reservation
    assert res["drawn"] == 0 and res["decode_steps"] == 0


def test_fixed_k_mode_is_uniform_sampling():
    U = 192
    p = mixture_p(U, 12)
    a = alloc(mode="fixed_k", n0=8, tau_low=0.0, budget_N=3072)
    res = C.simulate(a, U, synthetic(p))
    assert res["drawn"] == U and res["rollouts"] == 8 * U
    # every prompt gets its full group; effective iff its 8 rewards are mixed
    for u in range(U):
        s = res["successes"][u]
        assert res["n_issued"][u] == 8
        assert (res["status"][u] == C.COMMITTED) == (1 <= s <= 7)
    # SARA's first n outcomes of a prompt are fixed-k's first n outcomes
    sara = C.simulate(alloc(B=64, budget_N=3072), U, synthetic(p))
    for (u, j), (L, r, _, _) in sara["rollout"].items():
        assert res["rollout"][(u, j)][1] == r


def expected_rollouts(g, m, n_a):
    """Eq. EN generalised to a commit floor m <= n_a: a prompt stops at
    N = min(max(T_mix, m), n_a), with Pr[T_mix > n] = g^n + (1-g)^n (n >= 1),
    so E[N] = m + sum_{n=m}^{n_a-1} (g^n + (1-g)^n); m = 2 is Eq. EN itself."""
    return m + sum(g ** n + (1 - g) ** n for n in range(m, n_a))


@pytest.mark.parametrize("g", [0.5, 0.2, 0.05])
def test_early_commit_expected_rollouts_eq_en(g):
    """Theorem 2 (Eq. EN): with the commit floor at the first mix (commit_min
    = 2) and a Bernoulli(g) reward stream, the mean rollouts per drawn prompt
    is 1 + sum_{n=1}^{n_a-1} (g^n + (1-g)^n), n_a = k - floor(tau (k+1)) = 4."""
    U = 20000
    p = np.full(U, g)
    a = alloc(commit_min=2, B=10 ** 6, budget_N=10 ** 7, n_slots=4096)
    res = C.simulate(a, U, synthetic(p, seed=11))
    assert res["drawn"] == U
    n_a = 8 - math.floor(0.45 * 9)
    assert n_a == 4
    en = 1 + sum(g ** n + (1 - g) ** n for n in range(1, n_a))
    assert en == pytest.approx(expected_rollouts(g, 2, n_a))
    # N takes values in {2, 3, 4}: variance <= 1, so 5 sigma <= 5 / sqrt(U)
    assert abs(res["rollouts"] / U - en) < 5 / math.sqrt(U)
    # a prompt commits iff it mixes by n_a, the moment it mixes
    pc = 1 - (g ** n_a + (1 - g) ** n_a)
    assert abs(res["n_committed"] / U - pc) < 5 * math.sqrt(pc * (1 - pc) / U)
    for u in range(U):
        n, s = res["n_done"][u], res["successes"][u]
        if res["status"][u] == C.COMMITTED:
            assert 1 <= s <= n - 1 and n <= n_a
            # the first n - 1 outcomes were all the same (committed at the first mix)
            outs = [r for _, r in synthetic(p, seed=11)([(u, j) for j in range(n)])]
            assert len(set(outs[:-1])) == 1 and outs[-1] != outs[0]
        else:
            assert n == n_a and s in (0, n)
    check_invariants(a, res, U)


@pytest.mark.parametrize("m", [2, 3, 4])
def test_commit_floor_mixture_rollouts(m):
    """Commit floor m under the workloads' success-rate mixture: E[N] =
    m + sum_{n=m}^{n_a-1} E[g^n + (1-g)^n]; commit probability 1 - E[g^4 + (1-g)^4]
    for every floor m <= n_a (mixing is absorbing, the abandonment point is unchanged)."""
    U = 20000
    p = mixture_p(U, 21)
    a = alloc(commit_min=m, B=10 ** 6, budget_N=10 ** 7, n_slots=4096)
    res = C.simulate(a, U, synthetic(p, seed=5))
    n_a = 4
    en = m + sum(moment(n, 0) for n in range(m, n_a))
    assert abs(res["rollouts"] / U - en) < 5 * 2 / math.sqrt(U)
    pc = 1 - moment(4, 0)
    assert abs(res["n_committed"] / U - pc) < 5 * math.sqrt(pc * (1 - pc) / U)
    # every committed group has between m and n_a members: variable group sizes
    sizes = [res["n_done"][u] for u in range(U) if res["status"][u] == C.COMMITTED]
    assert min(sizes) >= m and max(sizes) <= n_a
    if m < n_a:
        assert len(set(sizes)) > 1
    check_invariants(a, res, U)


@pytest.mark.parametrize("k,n0,tau", [(8, 2, 0.1), (8, 2, 0.3), (8, 2, 0.6), (8, 1, 0.45), (8, 4, 0.45),
                                      (4, 2, 0.45), (16, 2, 0.45), (8, 6, 0.45)])
def test_ablation_stopping_times_under_mixture(k, n0, tau):
    """tau, n0 and k ablations (commit floor k): an unmixed prompt stops at
    n_stop = max(n0, n_a), n_a = k - floor(tau (k+1)) (Theorem 2's proof under
    the uniform prior), a prompt mixed by then runs to k, so the rollouts per
    drawn prompt are n_stop + (k - n_stop)(1 - E[g^n_stop + (1-g)^n_stop])."""
    U = 12000
    p = mixture_p(U, 31)
    a = alloc(k=k, n0=n0, commit_min=k, tau_low=tau, B=10 ** 6, budget_N=10 ** 8, n_slots=4096)
    res = C.simulate(a, U, synthetic(p, seed=13))
    n_a = min(k, k - math.floor(tau * (k + 1)))
    n_stop = max(n0, n_a)
    pc = 1 - moment(n_stop, 0)
    assert abs(res["n_committed"] / U - pc) < 5 * math.sqrt(pc * (1 - pc) / U)
    want = n_stop + (k - n_stop) * pc
    assert abs(res["rollouts"] / U - want) < 5 * (k - n_stop) * math.sqrt(pc * (1 - pc) / U) + 1e-12
    for u in range(U):
        if res["status"][u] == C.ABANDONED:
            assert res["n_done"][u] == n_stop and res["successes"][u] in (0, n_stop)
        else:
            assert res["n_done"][u] == k
    check_invariants(a, res, U)
