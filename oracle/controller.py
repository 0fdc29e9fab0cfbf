"""One SARA allocation step as a slot-pool event simulation (oracle).

Follows Algorithm 1 (section 3.3): probe fresh prompts with n0 rollouts,
decide each prompt with Eq. decide once its outcomes are in, drop abandoned
prompts and hand their remaining budget to fresh prompts, give continuing
prompts more rollouts ordered by the yield index p_eff, and stop when B
effective groups are collected or the budget / prompt pool is exhausted.

The paper runs this in synchronous rounds on the host.  The reading used
here puts the same rule on the decode-step clock of a pool of S generation
slots (identical to the round-synchronous algorithm when all rollouts have
equal length and slots never bind):

state   per prompt uid: status, n_issued, n_done, s (successes), inflight,
        p_eff; scalars budget_left = N, next_uid, |A|, |C|; slots; queue Q.
decode  step t: every occupied slot emits one token; a rollout of length L
        assigned with start step t0 finishes at step t0 + L - 1, posts its
        reward and frees its slot.
decide  after step t, in ascending uid, every ACTIVE prompt with no rollout
        in flight is decided (predictor.decide): COMMIT (|C|+1, refund k-n),
        ABANDON (refund k-n), or CONTINUE (queue commit_min-n rollouts if
        mixed, else 1).
refill  draw uid = next_uid++ while |A| < B-|C| (ignored in fixed-k mode),
        budget_left >= k and next_uid < U; each draw reserves k rollouts of
        budget and queues n0 probes with the prior's p_eff.  Q is ordered by
        (quantised p_eff descending, uid, j) and its head is assigned to the
        free slots in ascending slot order; these rollouts start at step t+1.
end     when no prompt is active (then no slot is busy and Q is empty).

Budget reading: the paper's "budget left" and safety cap are unspecified;
k rollouts are reserved per drawn prompt and k - n refunded when it is
decided, so rollouts spent never exceed N.

History warm start (implementation details, "defaults and history
warm-start"): `priors` gives each pool prompt its own Beta(alpha0_u,
beta0_u) prior (see warm.py); its p_eff, decisions and the priority of its
probes then use that prior in place of Beta(alpha0, beta0).

mode "sara_thompson": pending rollouts are ordered by the posterior-sampling
index of thompson.py (drawn when they are queued, keyed by draw_key = (seed,
step index)) instead of p_eff; everything else is unchanged.
"""
from . import thompson
from .predictor import ABANDON, COMMIT, CONTINUE, decide, p_eff, priority_key

UNDRAWN, ACTIVE, COMMITTED, ABANDONED = 0, 1, 2, 3


def simulate(alloc: dict, U: int, outcomes, priors=None, draw_key=(0, 0)):
    """outcomes(list[(uid, j)]) -> list[(length, reward)] for newly started rollouts.
    priors: optional (alpha0_u, beta0_u) sequences of length U (warm start).
    draw_key: (seed, step index) of the posterior-sampling priority.

    Returns a dict with the decision / draw / assignment / finish logs and the
    per-prompt and per-rollout results."""
    B, k, n0, cm = alloc["B"], alloc["k"], alloc["n0"], alloc["commit_min"]
    tau, a0, b0 = alloc["tau_low"], alloc["alpha0"], alloc["beta0"]
    N, S, bits = alloc["budget_N"], alloc["n_slots"], alloc["prio_quant_bits"]
    fixed_k = alloc["mode"] == "fixed_k"
    ts = alloc["mode"] == "sara_thompson"

    status = [UNDRAWN] * U
    n_iss, n_done, succ, infl = [0] * U, [0] * U, [0] * U, [0] * U
    pe = [0.0] * U
    budget, next_uid, nA, nC = N, 0, 0, 0
    Q = []
    slots = [None] * S                  # (uid, j, finish step, reward, length)
    rollout = {}                        # (uid, j) -> (length, reward, start, slot)
    log_dec, log_draw, log_asg, log_fin = [], [], [], []
    if priors is None:
        pa, pb = [a0] * U, [b0] * U
    else:
        pa, pb = [float(x) for x in priors[0]], [float(x) for x in priors[1]]
        assert len(pa) == U and len(pb) == U
    prior = [p_eff(0, 0, k, pa[u], pb[u]) for u in range(U)]
    prio = [0.0] * U        # index of the prompt's pending rollouts

    def queue_index(u, n, s, pv):
        return thompson.index(draw_key[0], draw_key[1], u, n, s, k, pa[u], pb[u]) if ts else pv

    def refill(start):
        nonlocal budget, next_uid, nA
        while (fixed_k or nA < B - nC) and budget >= k and next_uid < U:
            u = next_uid
            next_uid += 1
            status[u] = ACTIVE
            budget -= k
            nA += 1
            pe[u] = prior[u]
            prio[u] = queue_index(u, 0, 0, prior[u])
            n_iss[u] = n0
            infl[u] = n0
            Q.extend((u, j) for j in range(n0))
            log_draw.append((start, u))
        Q.sort(key=lambda e: (-priority_key(prio[e[0]], bits), e[0], e[1]))
        free = [i for i in range(S) if slots[i] is None]
        m = min(len(free), len(Q))
        started = Q[:m]
        del Q[:m]
        res = outcomes(started) if m else []
        for i, ((u, j), (L, r)) in enumerate(zip(started, res)):
            assert L >= 1
            slots[free[i]] = (u, j, start + L - 1, int(r), int(L))
            rollout[(u, j)] = (int(L), int(r), start, free[i])
            log_asg.append((start, free[i], u, j))

    refill(0)
    t_last = -1
    while nA > 0:
        busy = [s for s in slots if s is not None]
        assert busy, "active prompts but no running rollout"
        t = min(s[2] for s in busy)
        for i in range(S):
            s = slots[i]
            if s is not None and s[2] == t:
                u, j, _, r, L = s
                n_done[u] += 1
                succ[u] += r
                infl[u] -= 1
                log_fin.append((t, i, u, j, L, r))
                slots[i] = None
        t_last = t
        for u in range(next_uid):
            if status[u] != ACTIVE or infl[u] != 0:
                continue
            n, s = n_done[u], succ[u]
            d, pv, more = decide(n, s, k, cm, tau, pa[u], pb[u])
            pe[u] = pv
            log_dec.append((t, u, d, n, s, pv))
            if d == COMMIT:
                status[u] = COMMITTED
                nC += 1
                nA -= 1
                budget += k - n
            elif d == ABANDON:
                status[u] = ABANDONED
                nA -= 1
                budget += k - n
            else:
                prio[u] = queue_index(u, n, s, pv)
                Q.extend((u, n_iss[u] + i) for i in range(more))
                n_iss[u] += more
                infl[u] += more
        refill(t + 1)

    committed = [u for u in range(U) if status[u] == COMMITTED]
    return dict(
        status=status, n_issued=n_iss, n_done=n_done, successes=succ, p_eff=pe,
        committed=committed, budget_left=budget, drawn=next_uid,
        n_committed=nC, n_abandoned=sum(1 for x in status if x == ABANDONED),
        decode_steps=t_last + 1, rollouts=sum(n_iss),
        tokens=sum(v[0] for v in rollout.values()), rollout=rollout,
        log_decisions=log_dec, log_draws=log_draw, log_assign=log_asg, log_finish=log_fin)
