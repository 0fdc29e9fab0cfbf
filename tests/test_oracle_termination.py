"""Pins of the oracle's rollout termination (oracle/run.py).

The verifiable reward of section 2 ("RLVR and GRPO") is a function of the
completed response, so where a rollout stops decides what is hashed.  These
tests drive the oracle's rollout generator with hand-made token tables (and
the tiny model for the sampler paths) and check each stopping rule by its
observable result: lengths, the last token, and which token is appended
versus recorded as sampled.
"""
import numpy as np
import pytest

import workloads as W
from oracle import run, sampler

EOS = 511


def _cfg(max_new=12, forced_eos_u32=0):
    cfg = W.get_config("tiny_f32")
    cfg["model"]["eos_id"] = EOS
    cfg["alloc"].update(max_new=max_new, forced_eos_u32=forced_eos_u32)
    return cfg


def _source(cfg, table, forced_len=None, model_free=True, weights=None):
    pool = W.make_pool(cfg, 0)
    if forced_len is not None:
        pool["forced_len"] = forced_len
    return run.RolloutSource(cfg, weights, pool, W.sampling_seed(cfg), forced_tokens=table,
                             model_free=model_free), pool


def test_eos_ends_the_rollout_and_counts_in_its_length():
    cfg = _cfg()
    k, mn = cfg["alloc"]["k"], cfg["alloc"]["max_new"]
    tab = np.full((cfg["alloc"]["pool_U"] * k, mn), 7, np.int32)
    tab[0, 5] = EOS          # rollout (0, 0): EOS at index 5 -> 6 tokens
    tab[1, 0] = EOS          # rollout (0, 1): EOS first -> 1 token
    tab[2, mn - 1] = EOS     # rollout (0, 2): EOS exactly at the cap
    tab[3, 6:] = EOS         # only the first EOS counts
    src, _ = _source(cfg, tab)
    out = src.outcomes([(0, 0), (0, 1), (0, 2), (0, 3)])
    assert [L for L, _ in out] == [6, 1, mn, 7]
    r = src.results
    assert list(r[(0, 0)]["tokens"]) == [7] * 5 + [EOS]
    assert list(r[(0, 1)]["tokens"]) == [EOS]
    assert r[(0, 2)]["tokens"][-1] == EOS and len(r[(0, 2)]["tokens"]) == mn
    assert list(r[(0, 3)]["tokens"]) == [7] * 6 + [EOS]


def test_max_new_caps_a_rollout_without_eos():
    for mn in (1, 2, 12):
        cfg = _cfg(max_new=mn)
        k = cfg["alloc"]["k"]
        tab = np.full((cfg["alloc"]["pool_U"] * k, mn), 3, np.int32)
        src, _ = _source(cfg, tab)
        (L, _), = src.outcomes([(5, 7)])
        assert L == mn
        assert np.all(src.results[(5, 7)]["tokens"] == 3)


def test_no_eos_token_when_eos_is_disabled():
    cfg = _cfg()
    cfg["model"]["eos_id"] = -1
    k, mn = cfg["alloc"]["k"], cfg["alloc"]["max_new"]
    tab = np.full((cfg["alloc"]["pool_U"] * k, mn), EOS, np.int32)   # id 511 is an ordinary token
    src, _ = _source(cfg, tab)
    (L, _), = src.outcomes([(0, 0)])
    assert L == mn


def test_forced_length_gives_exactly_that_many_tokens_ending_in_eos():
    cfg = _cfg()
    U, k, mn = cfg["alloc"]["pool_U"], cfg["alloc"]["k"], cfg["alloc"]["max_new"]
    tab = np.full((U * k, mn), 9, np.int32)
    fl = np.full((U, k), mn, np.int32)
    fl[0, :4] = [1, 2, 5, mn]
    tab[4, 2] = EOS          # (0, 4): a natural EOS before the forced length wins
    fl[0, 4] = 8
    src, _ = _source(cfg, tab, forced_len=fl)
    out = src.outcomes([(0, j) for j in range(5)])
    assert [L for L, _ in out] == [1, 2, 5, mn, 3]
    for j, Lf in enumerate([1, 2, 5, mn]):
        toks = src.results[(0, j)]["tokens"]
        assert len(toks) == Lf and toks[-1] == EOS and np.all(toks[:-1] == 9)
    # with EOS disabled the forced length still stops the rollout, without a replacement
    cfg2 = _cfg()
    cfg2["model"]["eos_id"] = -1
    src2, _ = _source(cfg2, tab, forced_len=fl)
    (L, _), = src2.outcomes([(0, 2)])
    assert L == 5 and np.all(src2.results[(0, 2)]["tokens"] == 9)


def test_reward_hashes_the_completed_response_including_eos():
    cfg = _cfg()
    U, k, mn = cfg["alloc"]["pool_U"], cfg["alloc"]["k"], cfg["alloc"]["max_new"]
    tab = np.full((U * k, mn), 4, np.int32)
    tab[0, 3] = EOS
    tab[1, 3] = 4            # same first three tokens, no EOS -> runs to the cap
    src, _ = _source(cfg, tab)
    src.outcomes([(0, 0), (0, 1)])
    a, b = src.results[(0, 0)], src.results[(0, 1)]
    assert len(a["tokens"]) == 4 and len(b["tokens"]) == mn
    assert a["hash"] != b["hash"]
    # identical responses of one prompt hash alike (the hash excludes j)
    tab[2, :] = tab[0, :]
    src.outcomes([(0, 2)])
    assert src.results[(0, 2)]["hash"] == a["hash"] and src.results[(0, 2)]["reward"] == a["reward"]


@pytest.fixture(scope="module")
def tiny_weights():
    return W.make_weights(W.get_config("tiny_f32"))


def test_forced_eos_draw_overrides_the_sampled_token(tiny_weights):
    # always-on forced EOS: every rollout is one EOS token long, sampled and appended
    cfg = _cfg(forced_eos_u32=(1 << 32) - 1)
    src, _ = _source(cfg, None, model_free=False, weights=tiny_weights)
    out = src.outcomes([(u, j) for u in range(3) for j in range(2)])
    assert all(L == 1 for L, _ in out)
    for d in src.results.values():
        assert list(d["tokens"]) == [EOS] and list(d["sampled"]) == [EOS]
    # at 1/4 per token: each rollout stops at its first forced draw (or a sampled EOS)
    p4 = (1 << 32) // 4
    cfg = _cfg(max_new=24, forced_eos_u32=p4)
    src, pool = _source(cfg, None, model_free=False, weights=tiny_weights)
    seed, step = W.sampling_seed(cfg), pool["step"]
    pairs = [(u, j) for u in range(4) for j in range(8)]
    src.outcomes(pairs)
    stopped_by_draw = 0
    for (u, j) in pairs:
        d = src.results[(u, j)]
        rid = u * 8 + j
        draws = [sampler.forced_eos(seed, step, rid, i, p4) for i in range(24)]
        L = len(d["tokens"])
        assert not any(draws[:L - 1])
        assert all(t != EOS for t in d["tokens"][:L - 1])
        if draws[L - 1]:
            stopped_by_draw += 1
            assert d["tokens"][-1] == EOS and d["sampled"][-1] == EOS
        elif L < 24:
            assert d["tokens"][-1] == EOS
    assert stopped_by_draw >= 16


def test_teacher_forcing_appends_the_forced_token_and_records_the_sample(tiny_weights):
    cfg = _cfg(max_new=10)
    U, k, mn = cfg["alloc"]["pool_U"], cfg["alloc"]["k"], cfg["alloc"]["max_new"]
    g = np.random.default_rng(3)
    tab = g.integers(0, EOS, (U * k, mn)).astype(np.int32)
    tab[1, 6] = EOS                      # the forced EOS ends rollout (0, 1) after 7 tokens
    pool = W.make_pool(cfg, 0)
    seed = W.sampling_seed(cfg)
    src = run.RolloutSource(cfg, tiny_weights, pool, seed, forced_tokens=tab,
                            keep_logits=lambda u, j, i: True)
    src.outcomes([(0, 0), (0, 1)])
    a, b = src.results[(0, 0)], src.results[(0, 1)]
    assert np.array_equal(a["tokens"], tab[0]) and len(b["tokens"]) == 7
    assert np.array_equal(b["tokens"], tab[1, :7])
    # the recorded choice is the sampler's on the logits of the forced context
    for (u, j), d in ((0, 0), a), ((0, 1), b):
        for i in range(len(d["tokens"])):
            tok, _ = sampler.sample(src.logits[(u, j, i)], 1.0, seed, pool["step"], u * k + j, i)
            assert d["sampled"][i] == tok
    # the sample differs from the forced token somewhere (the table is random)
    assert np.any(a["sampled"] != a["tokens"])
