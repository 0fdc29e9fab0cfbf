"""History warm start across allocation steps (oracle; test infrastructure).

The paper's implementation details ("defaults and history warm-start") let
each prompt carry its posterior into later steps with an exponential decay
lambda, so a prompt found saturated before starts skewed and is abandoned
after fewer probes; lambda and the exact carry are not specified.  Reading
taken here, for a finite prompt set revisited across steps:

* prompt p of the set keeps pseudo-counts (a_p, b_p) >= 0, initially 0;
* in a step whose pool prompt u is set prompt ids[u], u's prior is
  Beta(alpha0 + a_{ids[u]}, beta0 + b_{ids[u]}) (Eq. peff and Eq. decide
  then use it unchanged: the posterior after n outcomes with s successes is
  Beta(alpha0 + a + s, beta0 + b + n - s), Sec. 3.1's conjugate update);
* after the step, the end-of-step posterior's pseudo-counts decay by lambda
  for every prompt of the set: a_p <- lambda (a_p + s_p),
  b_p <- lambda (b_p + n_p - s_p), with (n_p, s_p) = (0, 0) for a prompt the
  step did not draw.  lambda = 0 is the cold start of a fresh Beta(alpha0,
  beta0) every step; lambda = 1 keeps every outcome ever seen.
"""


def priors(ids, a, b, alpha0: float, beta0: float):
    """Per pool prompt (alpha0_u, beta0_u) lists from the set's pseudo-counts."""
    pa = [alpha0 + float(a[i]) for i in ids]
    pb = [beta0 + float(b[i]) for i in ids]
    return pa, pb


def update(a, b, ids, n_done, succ, drawn: int, lam: float):
    """New (a, b) lists after a step: the drawn pool prompts u < drawn add
    their (s, n - s), then every entry is scaled by lambda."""
    a2, b2 = [float(x) for x in a], [float(x) for x in b]
    assert len(set(ids)) == len(ids), "pool prompts must be distinct set prompts"
    for u in range(drawn):
        p = ids[u]
        a2[p] = a2[p] + succ[u]
        b2[p] = b2[p] + (n_done[u] - succ[u])
    return [lam * x for x in a2], [lam * x for x in b2]
