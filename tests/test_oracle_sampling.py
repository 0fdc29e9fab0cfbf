"""Pins of the oracle's Philox generator, sampler, reward hash and GRPO
advantages against published values, distributions and closed forms."""
import math

import numpy as np
import pytest
from scipy import stats

from oracle import grpo, reward, sampler
from oracle.philox import philox4x32


def test_philox_known_answers():
    # published known-answer vectors of Philox4x32-10 (Random123 distribution)
    f = 0xFFFFFFFF
    cases = [((0, 0, 0, 0), (0, 0), (0x6627E8D5, 0xE169C58D, 0xBC57AC4C, 0x9B00DBD8)),
             ((f, f, f, f), (f, f), (0x408F276D, 0x41C83B0E, 0xA20BC7C6, 0x6D5451FD)),
             ((0x243F6A88, 0x85A308D3, 0x13198A2E, 0x03707344), (0xA4093822, 0x299F31D0),
              (0xD16CFE09, 0x94FDCCEB, 0x5001E420, 0x24126EA1))]
    for ctr, key, want in cases:
        got = tuple(int(x) for x in philox4x32(*ctr, *key))
        assert got == want


def test_uniforms_and_gumbel_moments():
    u = np.concatenate([sampler.uniforms(99, 3, rid, pos, 4096) for rid in range(8) for pos in range(8)])
    assert u.min() > 0 and u.max() < 1
    assert abs(u.mean() - 0.5) < 5 * math.sqrt(1 / 12 / len(u))
    assert stats.kstest(u, "uniform").pvalue > 1e-4
    g = np.concatenate([sampler.gumbel(5, 0, rid, 0, 4096) for rid in range(16)]).astype(np.float64)
    assert abs(g.mean() - np.euler_gamma) < 5 * (math.pi / math.sqrt(6)) / math.sqrt(len(g))


def test_gumbel_max_is_softmax_sampling():
    V = 16
    logits = np.linspace(-2, 1.5, V).astype(np.float32)
    for T in (1.0, 0.7):
        n = 20000
        toks = np.array([sampler.sample(logits, T, 123, 0, rid, 3)[0] for rid in range(n)])
        p = np.exp(logits.astype(np.float64) / T)
        p /= p.sum()
        obs = np.bincount(toks, minlength=V)
        chi = stats.chisquare(obs, p * n)
        assert chi.pvalue > 1e-4


def test_token_is_lowest_id_on_ties():
    sc = np.array([0.5, 2.0, 2.0, 1.0], dtype=np.float32)
    assert int(np.argmax(sc)) == 1
    assert sampler.near_tie(sc)


def test_forced_eos_frequency():
    thr = (1 << 32) // 800
    hits = sum(sampler.forced_eos(77, 0, rid, pos, thr) for rid in range(400) for pos in range(400))
    n = 160000
    assert abs(hits - n / 800) < 5 * math.sqrt(n / 800)
    assert not sampler.forced_eos(77, 0, 1, 1, 0)


def test_splitmix64_published_outputs():
    # SplitMix64 seeded with 0 (state += golden gamma, then the finalizer)
    gamma = 0x9E3779B97F4A7C15
    assert reward.mix64(gamma) == 0xE220A8397B1DCDAF
    assert reward.mix64(2 * gamma) == 0x6E789E6AA1B965F4


def test_reward_hash_two_codings_agree():
    g = np.random.default_rng(0)
    for _ in range(50):
        toks = g.integers(0, 151936, size=g.integers(1, 60))
        seed, step, uid = int(g.integers(0, 2**63)), int(g.integers(0, 300)), int(g.integers(0, 256))
        h = reward.hash_tokens(seed, step, uid, toks)
        z = reward.mix64_np(np.uint64((seed ^ reward.SEED_R_XOR) & reward.MASK) ^ reward.mix64_np(
            np.uint64((step << 32) + uid)))
        for t in toks:
            z = reward.mix64_np(z ^ np.uint64(int(t) + 1))
        assert int(z) == h


def test_reward_frequency_tracks_p():
    g = np.random.default_rng(1)
    for p in (0.0, 0.03, 0.5, 0.9, 1.0):
        n = 4000
        r = [reward.reward_of_hash(reward.hash_tokens(9, 0, u, g.integers(0, 512, 8)), p) for u in range(n)]
        if p in (0.0, 1.0):
            assert sum(r) == n * p
        else:
            assert abs(np.mean(r) - p) < 5 * math.sqrt(p * (1 - p) / n)


def test_grpo_binary_closed_form_and_saturation():
    eps = 1e-6
    offs = [0, 8, 16, 24, 28]
    r = [1, 0, 0, 0, 0, 0, 0, 0] + [1] * 8 + [0] * 8 + [1, 1, 0, 1]
    a = grpo.advantages(r, offs, eps)
    for g in range(4):
        lo, hi = offs[g], offs[g + 1]
        m, s = hi - lo, sum(r[lo:hi])
        if s in (0, m):
            assert np.all(a[lo:hi] == 0.0)   # saturated group: zero advantage
        else:
            sd = math.sqrt(s * (m - s) / (m * (m - 1)))
            for i in range(lo, hi):
                want = ((1 - s / m) if r[i] else (-s / m)) / (sd + eps)
                assert a[i] == pytest.approx(want, rel=1e-12)
            assert abs(a[lo:hi].sum()) < 1e-12
            assert a[lo:hi].std(ddof=1) == pytest.approx(sd / (sd + eps), rel=1e-9)


def test_grpo_matches_library_statistics():
    g = np.random.default_rng(3)
    r = g.random(50)
    offs = [0, 3, 10, 11, 30, 50]
    a = grpo.advantages(r, offs)
    for lo, hi in zip(offs, offs[1:]):
        x = r[lo:hi]
        if hi - lo >= 2:
            assert np.allclose(a[lo:hi], (x - x.mean()) / (x.std(ddof=1) + 1e-6))
        else:
            assert np.all(a[lo:hi] == 0)


# --- top-p nucleus -----------------------------------------------------------

def _nucleus_by_prefix(logits, T, top_p):
    """The nucleus by its plain definition, in 50-digit arithmetic: walk the
    ids by (probability desc, id asc) and stop at the first prefix whose mass
    reaches top_p, then add every id tied with the last one."""
    import mpmath
    mpmath.mp.dps = 50
    z = [mpmath.mpf(float(np.float32(np.float32(x) / np.float32(T)))) for x in logits]
    zmax = max(z)
    w = [mpmath.e ** (zi - zmax) for zi in z]
    tot = sum(w)
    order = sorted(range(len(z)), key=lambda v: (-w[v], v))
    cum = mpmath.mpf(0)
    target = mpmath.mpf(float(np.float32(top_p)))
    for n, v in enumerate(order):
        cum += w[v] / tot
        if cum >= target:
            cut = w[v]
            return np.array([wi >= cut for wi in w]), float(abs(cum - target))
    raise AssertionError


def test_nucleus_matches_the_prefix_definition():
    rng = np.random.default_rng(11)
    checked = 0
    for trial in range(60):
        V = int(rng.integers(2, 40))
        logits = (rng.standard_normal(V) * rng.choice([0.3, 1.0, 3.0])).astype(np.float32)
        if trial % 5 == 0:   # exact ties, also at the cut
            logits[rng.integers(0, V, size=V // 2)] = logits[0]
        T = float(rng.choice([1.0, 0.7, 1.3]))
        top_p = float(rng.choice([0.05, 0.3, 0.5, 0.9, 0.95, 0.999]))
        want, gap = _nucleus_by_prefix(logits, T, top_p)
        if gap < 1e-9:
            continue
        got = sampler.nucleus(logits, T, top_p)
        assert np.array_equal(got, want), (trial, logits, T, top_p)
        assert sampler.nucleus_margin(logits, T, top_p) > 0
        checked += 1
    assert checked >= 50


def test_nucleus_ties_at_the_cut_are_kept():
    # p = (0.4, 0.2, 0.2, 0.2): at top_p 0.5 the prefix stops inside the tie
    logits = np.log(np.array([2.0, 1.0, 1.0, 1.0])).astype(np.float32)
    m = sampler.nucleus(logits, 1.0, 0.5)
    assert m.tolist() == [True, True, True, True]
    assert sampler.nucleus(logits, 1.0, 0.3).tolist() == [True, False, False, False]


def test_nucleus_limits():
    rng = np.random.default_rng(3)
    logits = rng.standard_normal(300).astype(np.float32)
    # top_p = 1 keeps every id, also those whose weight is below 2^-44
    logits[7] = -200.0
    assert sampler.nucleus(logits, 1.0, 1.0).all()
    # a tiny top_p keeps only the most likely id (greedy)
    m = sampler.nucleus(logits, 1.0, 1e-7)
    assert m.sum() == 1 and m[int(np.argmax(logits))]
    # the nucleus is minimal: its mass reaches top_p, without its cut group it does not
    p = np.exp(logits.astype(np.float64) - logits.max())
    p /= p.sum()
    for top_p in (0.2, 0.6, 0.9):
        m = sampler.nucleus(logits, 1.0, top_p)
        zc = logits[m].min()
        assert p[m].sum() >= top_p - 1e-12
        assert p[logits > zc].sum() < top_p
        # the sample never leaves the nucleus
        for rid in range(50):
            tok, sc = sampler.sample(logits, 1.0, 5, 0, rid, 1, top_p)
            assert m[tok]
            assert np.isneginf(sc[~m]).all()


def test_top_p_sampling_is_truncated_softmax():
    V = 12
    logits = np.linspace(-1.5, 1.0, V).astype(np.float32)
    T, top_p = 0.9, 0.8
    m = sampler.nucleus(logits, T, top_p)
    assert 2 <= m.sum() < V
    p = np.where(m, np.exp(logits.astype(np.float64) / T), 0.0)
    p /= p.sum()
    n = 20000
    toks = np.array([sampler.sample(logits, T, 321, 2, rid, 0, top_p)[0] for rid in range(n)])
    obs = np.bincount(toks, minlength=V)
    assert obs[~m].sum() == 0
    assert stats.chisquare(obs[m], p[m] * n).pvalue > 1e-4
    # top_p = 1 is the plain sampler, token for token
    for rid in range(200):
        assert sampler.sample(logits, T, 9, 0, rid, 4, 1.0)[0] == sampler.sample(logits, T, 9, 0, rid, 4)[0]


# --- rollout length distributions --------------------------------------------

def test_forced_eos_lengths_match_the_truncated_geometric():
    """3B workload: a forced EOS with per-token probability thr / 2^32
    (thr = floor(2^32 / 800)) ends a rollout at its first firing, else at the
    2048-token cap.  Closed form: P(capped) = (1 - p)^2048 = 7.73%, mean
    length (1 - (1 - p)^2048) / p = 738.3."""
    import workloads as W
    from oracle.philox import philox4x32
    cfg = W.get_config("qwen3b_shape")
    thr, cap = cfg["alloc"]["forced_eos_u32"], cfg["alloc"]["max_new"]
    assert thr == (1 << 32) // 800 and cap == 2048
    seed, step = W.sampling_seed(cfg), 0
    k0, k1 = sampler.key_of(seed, step)
    R = 3000
    rid = np.arange(R, dtype=np.uint64)[:, None]
    pos = np.arange(cap, dtype=np.uint64)[None, :]
    words = philox4x32(rid, pos, 0, 1, k0, k1)[..., 0]
    for r, i in [(0, 0), (7, 11), (2999, 2047), (1234, 600)]:
        assert int(words[r, i]) == sampler.forced_eos_word(seed, step, r, i)
    fired = words < np.uint32(thr)
    L = np.where(fired.any(axis=1), fired.argmax(axis=1) + 1, cap).astype(np.float64)
    p = thr / 2.0 ** 32
    capped = (1 - p) ** cap
    mean = (1 - capped) / p
    assert abs(capped - 0.0773) < 5e-4 and abs(mean - 738.3) < 0.5
    var = sum((2 * i - 1) * (1 - p) ** (i - 1) for i in range(1, cap + 1)) - mean ** 2
    assert abs(L.mean() - mean) < 5 * math.sqrt(var / R)
    assert abs(np.mean(L == cap) - capped) < 5 * math.sqrt(capped * (1 - capped) / R)


def test_long_rollout_lengths_match_the_clamped_lognormal():
    """Long-rollout workload: lengths clamp(round(exp(ln 1200 + 0.6 z)), 1,
    4096).  Closed forms of the lognormal: E[min(X, c)] = e^(mu + s^2/2)
    Phi((ln c - mu - s^2) / s) + c P(X >= c) = 1415 and P(X >= 4096) = 2.0%."""
    import workloads as W
    cfg = W.get_config("long_ragged_1p5b")
    L = np.concatenate([W.make_pool(cfg, t)["forced_len"].reshape(-1) for t in range(4)]).astype(np.float64)
    mu, s, c = math.log(1200.0), 0.6, 4096.0
    z = (math.log(c) - mu) / s
    p_cap = stats.norm.sf(z)
    mean = math.exp(mu + s * s / 2) * stats.norm.cdf(z - s) + c * p_cap
    assert abs(mean - 1415) < 2 and abs(p_cap - 0.0204) < 5e-4
    sd = float(np.sqrt(np.mean((np.minimum(np.exp(mu + s * np.random.default_rng(0).standard_normal(200000)), c)
                                - mean) ** 2)))
    assert abs(L.mean() - mean) < 5 * sd / math.sqrt(len(L)) + 0.5   # + rounding to integers
    assert abs(np.mean(L >= c) - p_cap) < 5 * math.sqrt(p_cap * (1 - p_cap) / len(L))
    assert L.min() >= 1 and L.max() <= c
