"""Posterior-sampling (Thompson) priority for pending rollouts (oracle; test
infrastructure).

The paper's index-policy proposition names posterior sampling as an
alternative to ordering prompts by p_eff with the same fixed points.
Reading taken here: when a prompt's rollouts are queued (its draw, or a
CONTINUE decision after n outcomes with s successes) it gets the index

    p(g~) = P(its group of k ends mixed | g~, n, s),  g~ ~ Beta(a, b),
    a = alpha0 + s, b = beta0 + n - s   (the current posterior),

i.e. Eq. peff evaluated at one posterior draw instead of averaged over the
posterior: 1 - g~^k - (1-g~)^k before any outcome, 1 - (1-g~)^r after s = 0
of n (r = k - n), 1 - g~^r after s = n, 1 once mixed.  Its expectation over
the draw is p_eff.  Pending rollouts are then ordered by (quantised index
descending, uid, j) as with p_eff; decisions still use Eq. decide.

The draw: for integer a, b >= 1, Beta(a, b) is the law of the a-th smallest
of m = a + b - 1 independent uniforms (order statistics of the uniform).  The
uniforms are u_i = (w_i + 1/2) 2^-32 from the 32-bit words w_0, w_1, .. of
Philox4x32-10 under the sampler's key (seed, step index) at counters
(uid, n, c, 2), c = 0, 1, .. (4 words each; the last counter word 2 keeps
these draws apart from the token sampler's 0 and forced EOS's 1).  Prompts
whose posterior parameters are not integers, or with m > MAX_M, keep the
p_eff index.
"""
from .philox import philox4x32
from .predictor import is_mixed, p_eff
from .sampler import key_of

MAX_M = 4096


def order_statistic_word(seed: int, step: int, uid: int, n: int, a: int, m: int) -> int:
    """The a-th smallest of the m draw words of (uid, n)."""
    k0, k1 = key_of(seed, step)
    words = []
    c = 0
    while len(words) < m:
        words += [int(x) for x in philox4x32(uid, n, c, 2, k0, k1).reshape(-1)]
        c += 1
    return sorted(words[:m])[a - 1]


def power(x: float, e: int) -> float:
    """x^e by e successive fp64 multiplications (a fixed rounding sequence)."""
    p = 1.0
    for _ in range(e):
        p = p * x
    return p


def index(seed: int, step: int, uid: int, n: int, s: int, k: int, alpha0: float, beta0: float) -> float:
    if is_mixed(n, s):
        return 1.0
    r = k - n
    if r <= 0:
        return 0.0
    a, b = alpha0 + s, beta0 + (n - s)
    if a != int(a) or b != int(b) or a < 1 or b < 1 or a + b - 1 > MAX_M:
        return p_eff(n, s, k, alpha0, beta0)
    a, b = int(a), int(b)
    w = order_statistic_word(seed, step, uid, n, a, a + b - 1)
    g = (w + 0.5) * 2.0 ** -32
    if n == 0:
        return (1.0 - power(g, k)) - power(1.0 - g, k)
    if s == 0:
        return 1.0 - power(1.0 - g, r)
    return 1.0 - power(g, r)
