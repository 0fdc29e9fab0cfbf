"""Synthetic verifiable reward (oracle).

The binary reward r(q, o) of section 2 is replaced by a Bernoulli(p_q) draw
made deterministic by hashing the generated token sequence: a chain of the
SplitMix64 output finalizer (Steele, Lea, Flood, OOPSLA'14),

    h0 = mix(seed_r XOR mix(step * 2^32 + uid)),  h <- mix(h XOR (t + 1)) per token,
    reward = [ (h >> 11) * 2^-53 < p_uid ]        (exact in fp64),

with seed_r = seed XOR 0xD1B54A32D192ED03.  The rollout index j is not hashed,
so identical responses to one prompt earn identical rewards.  The paper gives
no such function, so the chain is our own definition: the mixing function is
pinned by SplitMix64's published outputs and the reward frequency against p;
tests also check the two codings below against each other.
"""
import numpy as np

MASK = (1 << 64) - 1
SEED_R_XOR = 0xD1B54A32D192ED03


def mix64(z: int) -> int:
    z &= MASK
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & MASK
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & MASK
    return z ^ (z >> 31)


def hash_init(seed: int, step: int, uid: int) -> int:
    return mix64((seed ^ SEED_R_XOR) ^ mix64((step << 32) + uid))


def hash_tokens(seed: int, step: int, uid: int, tokens) -> int:
    h = hash_init(seed, step, uid)
    for t in tokens:
        h = mix64(h ^ (int(t) + 1))
    return h


def reward_of_hash(h: int, p: float) -> int:
    return int((h >> 11) * (2.0 ** -53) < p)


# second, independent coding (numpy uint64 wrap-around arithmetic) used by tests
def mix64_np(z: np.ndarray) -> np.ndarray:
    z = np.asarray(z, dtype=np.uint64)
    with np.errstate(over="ignore"):
        z = (z ^ (z >> np.uint64(30))) * np.uint64(0xBF58476D1CE4E5B9)
        z = (z ^ (z >> np.uint64(27))) * np.uint64(0x94D049BB133111EB)
    return z ^ (z >> np.uint64(31))
