"""Token sampler (oracle): temperature, Gumbel-max, forced-EOS draw.

The paper samples rollouts at temperature 1.0 with an inference engine and
does not fix the sampler; the reading used here is Gumbel-max (argmax of
logit/T + Gumbel noise equals a draw from softmax(logit/T)) with every random
number taken from Philox4x32-10, so that a token is a pure function of
(seed, step, rollout id, generated index) and never of the slot schedule.

Key and counters (all 32-bit words):
* key      = (low word of seed, high word of seed XOR step index)
* Gumbel   : counter (rollout id, generated index, v // 4, 0), word v % 4
* forced EOS: counter (rollout id, generated index, 0, 1), word 0
Uniform from a word w: u = ((w >> 8) + 1/2) * 2^-24, exact and inside (0, 1).
Gumbel noise: g = -log(-log u) evaluated in fp64 and rounded to fp32.
Score: fp32(logit / T) + g in fp32; the token is the lowest id attaining the
maximum score.  Forced EOS fires when word 0 < forced_eos_u32.

Top-p (nucleus, Holtzman et al., ICLR'20) for top_p < 1: sort the vocabulary
by probability, largest first, and keep the shortest prefix whose mass reaches
top_p, together with every id tied with the last one kept; the Gumbel-max draw
then runs over that set only (a draw from the renormalised truncated
softmax).  Reading of "mass", fixed so that the cut is an integer decision:
z_v = fp32(logit_v / T) (+0 for a zero), weight q_v = floor(exp(z_v - z_max)
* 2^44) in fp64 then as an integer (the largest weight is 2^44), Q = sum of
q_v, target t = ceil(fp64(top_p) * fp64(Q)); the nucleus is {v : z_v >= z*}
with z* the largest z value whose set {z_v >= z*} holds weight >= t.
top_p = 1 keeps the whole vocabulary (no weight is dropped).

Pins (tests): Philox4x32-10 published known-answer vectors; uniformity and
Gumbel moments; chi-square of the Gumbel-max draw against softmax; the
nucleus against its prefix definition in 50-digit arithmetic, ties at the
cut, the greedy and top_p = 1 limits and minimality; chi-square of the top-p
draw against the renormalised truncated softmax; the forced-EOS frequency
and the rollout-length law it implies (truncated geometric).
"""
import math

import numpy as np

from .philox import philox4x32


def key_of(seed: int, step: int):
    return seed & 0xFFFFFFFF, ((seed >> 32) & 0xFFFFFFFF) ^ (step & 0xFFFFFFFF)


def uniforms(seed: int, step: int, rid: int, pos: int, V: int) -> np.ndarray:
    k0, k1 = key_of(seed, step)
    nb = (V + 3) // 4
    words = philox4x32(rid, pos, np.arange(nb, dtype=np.uint64), 0, k0, k1).reshape(-1)[:V]
    return ((words >> np.uint32(8)).astype(np.float64) + 0.5) * (2.0 ** -24)


def gumbel(seed: int, step: int, rid: int, pos: int, V: int) -> np.ndarray:
    u = uniforms(seed, step, rid, pos, V)
    return (-np.log(-np.log(u))).astype(np.float32)


def scores(logits32: np.ndarray, temperature: float, g: np.ndarray) -> np.ndarray:
    s = (np.asarray(logits32, dtype=np.float32) / np.float32(temperature)).astype(np.float32)
    return (s + g).astype(np.float32)


NUCLEUS_FRAC_BITS = 44


def nucleus_weights(logits32, temperature):
    """(z, integer weights q as uint64) of the top-p reading in the module
    header; q <= 2^44, so floor() of the fp64 product is exact."""
    z = (np.asarray(logits32, dtype=np.float32) / np.float32(temperature)).astype(np.float32)
    z = np.where(z == 0, np.float32(0.0), z).astype(np.float32)
    e = np.exp(z.astype(np.float64) - np.float64(z.max()))
    q = np.floor(e * 2.0 ** NUCLEUS_FRAC_BITS).astype(np.uint64)
    return z, q


def nucleus_target(top_p: float, Q: int) -> int:
    return int(math.ceil(float(np.float64(np.float32(top_p))) * float(Q)))


def nucleus(logits32, temperature, top_p):
    """Boolean mask of the top-p nucleus over the vocabulary: walk the z
    values from the largest down, one group of equal values at a time, and
    stop at the first group after which the kept weight reaches t."""
    V = len(logits32)
    if np.float32(top_p) >= 1:
        return np.ones(V, dtype=bool)
    z, q = nucleus_weights(logits32, temperature)
    t = nucleus_target(top_p, int(q.sum()))
    order = np.argsort(-z, kind="stable")
    zs = z[order]
    cum = np.cumsum(q[order])                      # exact: total < 2^63
    group_end = np.append(zs[1:] != zs[:-1], True)  # last position of each equal-z group
    first = int(np.nonzero(group_end & (cum >= np.uint64(t)))[0][0])
    return z >= zs[first]


def nucleus_margin(logits32, temperature, top_p) -> float:
    """Distance of the cut from the target, as a fraction of the total weight:
    how far the kept weight exceeds t, and how far the weight above the cut
    group falls short of it (the smaller of the two).  A cut decided by less
    than a few units of the last place of exp is reported near 0."""
    if np.float32(top_p) >= 1:
        return 1.0
    z, q = nucleus_weights(logits32, temperature)
    Q = int(q.sum())
    t = nucleus_target(top_p, Q)
    m = nucleus(logits32, temperature, top_p)
    kept = int(q[m].sum())
    above = int(q[z > np.min(z[m])].sum())
    return min(kept - t, t - 1 - above) / Q


def sample(logits32, temperature, seed, step, rid, pos, top_p=1.0):
    """Returns (token, score array) for one (rollout, position); ids outside
    the top-p nucleus get score -inf."""
    V = len(logits32)
    sc = scores(logits32, temperature, gumbel(seed, step, rid, pos, V))
    if np.float32(top_p) < 1:
        sc = np.where(nucleus(logits32, temperature, top_p), sc, np.float32(-np.inf)).astype(np.float32)
    return int(np.argmax(sc)), sc


def forced_eos_word(seed: int, step: int, rid: int, pos: int) -> int:
    k0, k1 = key_of(seed, step)
    return int(philox4x32(rid, pos, 0, 1, k0, k1)[0])


def forced_eos(seed, step, rid, pos, thresh_u32: int) -> bool:
    return thresh_u32 > 0 and forced_eos_word(seed, step, rid, pos) < thresh_u32


def near_tie(sc: np.ndarray, rel: float = 1e-5) -> bool:
    """True when the two best scores are within rel * max(1, |best|)."""
    top = np.partition(sc.astype(np.float64), -2)[-2:]
    if not np.isfinite(top[0]):
        return False
    return (top[1] - top[0]) <= rel * max(1.0, abs(top[1]))
