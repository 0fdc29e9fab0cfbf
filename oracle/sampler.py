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
"""
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


def sample(logits32, temperature, seed, step, rid, pos):
    """Returns (token, score array) for one (rollout, position)."""
    V = len(logits32)
    sc = scores(logits32, temperature, gumbel(seed, step, rid, pos, V))
    return int(np.argmax(sc)), sc


def forced_eos_word(seed: int, step: int, rid: int, pos: int) -> int:
    k0, k1 = key_of(seed, step)
    return int(philox4x32(rid, pos, 0, 1, k0, k1)[0])


def forced_eos(seed, step, rid, pos, thresh_u32: int) -> bool:
    return thresh_u32 > 0 and forced_eos_word(seed, step, rid, pos) < thresh_u32


def near_tie(sc: np.ndarray, rel: float = 1e-5) -> bool:
    """True when the two best scores are within rel * max(1, |best|)."""
    top = np.partition(sc.astype(np.float64), -2)[-2:]
    return (top[1] - top[0]) <= rel * max(1.0, abs(top[1]))
