"""Seeded synthetic inputs for the SARA rollout-allocation hot path.

This module only *produces inputs*: model weights, prompt pools, per-prompt
success rates and forced-length tables.  It holds none of the method's
arithmetic, so both the HIP path and the CPU oracle may read it.

Workloads (stand-ins for the paper's MATH/Countdown runs with
R1-Distill-Qwen-1.5B / Qwen2.5-3B, which are not available):

* ``tiny_f32``          2-layer fp32 decoder, B=16, k=8, n0=2, tau=0.45, N=128.
* ``qwen1p5b_shape``    Qwen2.5-1.5B-shaped bf16 decoder, B=64, N=512, 512 slots.
* ``qwen3b_shape``      Qwen2.5-3B-shaped bf16 decoder, B=64, N=512, forced EOS 1/800.
* ``long_ragged_1p5b``  1.5B shape, 256 slots, lognormal forced lengths,
                        300 allocation steps with a drifting success-rate mixture.
* ``pool_3b``           3B shape, candidate pool of 192 prompts, goal B=64, cap 6Bk,
                        plus the fixed-k baseline on the whole pool.

Paper defaults (B=64, k=8, n0=2, tau=0.45, commit floor k, Beta(1,1) prior,
safety cap 6Bk) come from the implementation-details appendix; the per-prompt
success-rate mixture imitates the mass at s=0 and s=k of the paper's
success-count histogram (section 2, "Effective and saturated groups").

Seeding: every array is drawn from ``numpy.random.SeedSequence`` entropy lists
``[master, stream, ...]`` so results do not depend on thread count or call order.
"""
from __future__ import annotations

import copy
import math
from concurrent.futures import ThreadPoolExecutor

import numpy as np

# ----------------------------------------------------------------------------
# model shapes
# ----------------------------------------------------------------------------
_TINY = dict(n_layers=2, d_model=256, n_heads=4, n_kv_heads=4, head_dim=64,
             d_ffn=1024, vocab=512, rope_theta=1.0e4, rms_eps=1e-6,
             dtype="f32", eos_id=-1)
_Q15 = dict(n_layers=28, d_model=1536, n_heads=12, n_kv_heads=2, head_dim=128,
            d_ffn=8960, vocab=151936, rope_theta=1.0e6, rms_eps=1e-6,
            dtype="bf16", eos_id=151935)
_Q3 = dict(n_layers=36, d_model=2048, n_heads=16, n_kv_heads=2, head_dim=128,
           d_ffn=11008, vocab=151936, rope_theta=1.0e6, rms_eps=1e-6,
           dtype="bf16", eos_id=151935)

FORCED_EOS_1_IN_800 = (1 << 32) // 800   # P(EOS) = x / 2^32 per generated token


def _alloc(**kw):
    base = dict(B=64, k=8, n0=2, commit_min=8, tau_low=0.45, alpha0=1.0, beta0=1.0,
                budget_N=512, pool_U=256, n_slots=512, kv_block=16, max_prompt=512,
                max_new=1024, mode="sara", temperature=1.0, top_p=1.0,
                forced_eos_u32=0, prio_quant_bits=20)
    base.update(kw)
    return base


CONFIGS = {
    "tiny_f32": dict(
        name="tiny_f32", index=0, model=dict(_TINY),
        alloc=_alloc(B=16, budget_N=128, pool_U=64, n_slots=128, max_prompt=32, max_new=64),
        prompt_len=(32, 32), mixture="standard", forced_len=None, steps=1),
    "qwen1p5b_shape": dict(
        name="qwen1p5b_shape", index=1, model=dict(_Q15),
        alloc=_alloc(),
        prompt_len=(128, 512), mixture="standard", forced_len=None, steps=1),
    "qwen3b_shape": dict(
        name="qwen3b_shape", index=2, model=dict(_Q3),
        alloc=_alloc(max_new=2048, forced_eos_u32=FORCED_EOS_1_IN_800),
        prompt_len=(128, 512), mixture="standard", forced_len=None, steps=1),
    "long_ragged_1p5b": dict(
        name="long_ragged_1p5b", index=3, model=dict(_Q15),
        alloc=_alloc(n_slots=256, max_new=4096),
        prompt_len=(128, 512), mixture="drift",
        forced_len=dict(mu=math.log(1200.0), sigma=0.6, cap=4096), steps=300),
    "pool_3b": dict(
        name="pool_3b", index=4, model=dict(_Q3),
        alloc=_alloc(pool_U=192, budget_N=6 * 64 * 8, max_prompt=1024, max_new=2048,
                     forced_eos_u32=FORCED_EOS_1_IN_800),
        prompt_len=(256, 1024), mixture="standard", forced_len=None, steps=1),
}
CONFIG_ORDER = ["tiny_f32", "qwen1p5b_shape", "qwen3b_shape", "long_ragged_1p5b", "pool_3b"]


def get_config(name: str) -> dict:
    return copy.deepcopy(CONFIGS[name])


def fixed_k_variant(cfg: dict) -> dict:
    """Uniform / dynamic-sampling baseline: every drawn prompt gets k rollouts,
    no early abandonment (n0 = k, tau = 0), and the goal B is ignored."""
    c = copy.deepcopy(cfg)
    a = c["alloc"]
    a.update(mode="fixed_k", n0=a["k"], tau_low=0.0)
    c["name"] = cfg["name"] + "+fixed_k"
    return c


def parity_slice(cfg: dict, *, B=4, N=None, slots=None, prompt_len=(16, 40), max_new=12,
                 forced_eos_u32=(1 << 32) // 16, pool_U=None) -> dict:
    """Reduced allocation sizes on the *full* model shape, small enough for the
    CPU oracle to generate every rollout token by token."""
    c = copy.deepcopy(cfg)
    a = c["alloc"]
    k = a["k"]
    N = N if N is not None else B * k
    a.update(B=B, budget_N=N, n_slots=slots if slots is not None else N,
             pool_U=pool_U if pool_U is not None else 4 * B, max_prompt=max(prompt_len[1], 2),
             max_new=max_new)
    if c["model"]["eos_id"] >= 0:
        a["forced_eos_u32"] = forced_eos_u32
    c["prompt_len"] = prompt_len
    if c["forced_len"] is not None:
        c["forced_len"] = dict(mu=math.log(max(2.0, max_new / 3.0)), sigma=0.6, cap=max_new)
    c["name"] = cfg["name"] + "@slice"
    c["steps"] = 1
    return c


# ----------------------------------------------------------------------------
# seeds
# ----------------------------------------------------------------------------
def master_seed(cfg: dict) -> int:
    return 1000 + int(cfg["index"])


def sampling_seed(cfg: dict) -> int:
    """64-bit key material for the counter-based sampler and the reward hash."""
    w = np.random.SeedSequence([master_seed(cfg), 3]).generate_state(2, np.uint32)
    return int(w[0]) | (int(w[1]) << 32)


# ----------------------------------------------------------------------------
# weights
# ----------------------------------------------------------------------------
def weight_specs(model: dict):
    """Fixed tensor order and shapes ([out, in] row-major, `in` contiguous)."""
    d, hd = model["d_model"], model["head_dim"]
    hq, hkv, f, V = model["n_heads"], model["n_kv_heads"], model["d_ffn"], model["vocab"]
    specs = [("embed", (V, d))]
    for l in range(model["n_layers"]):
        specs += [(f"l{l}.attn_norm", (d,)), (f"l{l}.wq", (hq * hd, d)),
                  (f"l{l}.wk", (hkv * hd, d)), (f"l{l}.wv", (hkv * hd, d)),
                  (f"l{l}.wo", (d, hq * hd)), (f"l{l}.ffn_norm", (d,)),
                  (f"l{l}.wg", (f, d)), (f"l{l}.wu", (f, d)), (f"l{l}.wd", (d, f))]
    specs += [("final_norm", (d,)), ("lm_head", (V, d))]
    return specs


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round-to-nearest-even fp32 -> bf16 bit patterns (uint16); finite inputs."""
    b = np.ascontiguousarray(x, dtype=np.float32).reshape(-1).view(np.uint32)
    out = np.empty(b.shape, dtype=np.uint16)

    def conv(c):
        s = b[c * _CHUNK:(c + 1) * _CHUNK]
        out[c * _CHUNK:(c + 1) * _CHUNK] = (s + np.uint32(0x7FFF) + ((s >> np.uint32(16)) & np.uint32(1))) \
            >> np.uint32(16)

    n_chunks = (b.size + _CHUNK - 1) // _CHUNK
    if n_chunks <= 1:
        conv(0)
    else:
        with ThreadPoolExecutor(max_workers=min(16, n_chunks)) as ex:
            list(ex.map(conv, range(n_chunks)))
    return out.reshape(np.shape(x))


_CHUNK = 1 << 22


def _normal_tensor(master: int, t_index: int, numel: int, std: float) -> np.ndarray:
    out = np.empty(numel, dtype=np.float32)
    n_chunks = (numel + _CHUNK - 1) // _CHUNK

    def fill(c):
        lo, hi = c * _CHUNK, min(numel, (c + 1) * _CHUNK)
        g = np.random.Generator(np.random.PCG64(np.random.SeedSequence([master, 0, t_index, c])))
        out[lo:hi] = g.standard_normal(hi - lo, dtype=np.float32) * np.float32(std)

    if n_chunks == 1:
        fill(0)
    else:
        with ThreadPoolExecutor(max_workers=min(16, n_chunks)) as ex:
            list(ex.map(fill, range(n_chunks)))
    return out


def make_weights(cfg: dict, std: float = 0.02) -> dict:
    """Random-init weights: N(0, std^2) matrices, unit norm weights.

    fp32 models get float32 arrays; bf16 models get uint16 bf16 bit patterns
    (round-to-nearest-even of the fp32 draw), identical for every consumer."""
    model = cfg["model"]
    master = master_seed(cfg)
    out = {}
    for ti, (name, shape) in enumerate(weight_specs(model)):
        numel = int(np.prod(shape))
        if len(shape) == 1:
            w = np.ones(numel, dtype=np.float32)
        else:
            w = _normal_tensor(master, ti, numel, std)
        w = w.reshape(shape)
        out[name] = f32_to_bf16_bits(w) if model["dtype"] == "bf16" else w
    return out


# ----------------------------------------------------------------------------
# prompt pools
# ----------------------------------------------------------------------------
def mixture_weights(cfg: dict, step: int):
    """(w_hard, w_easy, w_mid) for Beta(0.3,3), Beta(3,0.3), U(0,1)."""
    if cfg["mixture"] == "drift":
        T = max(1, cfg["steps"] - 1)
        f = min(step, T) / T
        return 0.40 - 0.20 * f, 0.30 + 0.20 * f, 0.30
    return 0.40, 0.30, 0.30


def make_pool(cfg: dict, step: int = 0) -> dict:
    """Prompt pool of one allocation step.

    Returns tokens (int32, concatenated), offsets (int32, U+1), p (float64, U),
    forced_len (int32 [U, k] or None)."""
    m, a = cfg["model"], cfg["alloc"]
    U, k = a["pool_U"], a["k"]
    master = master_seed(cfg)
    g = np.random.Generator(np.random.PCG64(np.random.SeedSequence([master, 1, step])))
    lo, hi = cfg["prompt_len"]
    lens = g.integers(lo, hi + 1, size=U).astype(np.int32)
    lens = np.minimum(lens, a["max_prompt"]).astype(np.int32)
    offsets = np.zeros(U + 1, dtype=np.int32)
    offsets[1:] = np.cumsum(lens)
    # uniform token ids in [0, V-1): the last id is reserved for EOS
    tokens = g.integers(0, m["vocab"] - 1, size=int(offsets[-1])).astype(np.int32)

    h = np.random.Generator(np.random.PCG64(np.random.SeedSequence([master, 2, step])))
    wh, we, wm = mixture_weights(cfg, step)
    comp = h.choice(3, size=U, p=[wh, we, wm])
    p = np.where(comp == 0, h.beta(0.3, 3.0, size=U),
                 np.where(comp == 1, h.beta(3.0, 0.3, size=U), h.random(size=U)))
    p = p.astype(np.float64)
    forced = None
    fl = cfg.get("forced_len")
    if fl is not None:
        z = h.standard_normal(size=(U, k))
        L = np.rint(np.exp(fl["mu"] + fl["sigma"] * z))
        forced = np.clip(L, 1, min(fl["cap"], a["max_new"])).astype(np.int32)
    return dict(tokens=tokens, offsets=offsets, p=p, forced_len=forced, step=step)


def pool_with_lengths(cfg: dict, lengths, step: int = 0) -> dict:
    """A pool like ``make_pool``'s whose prompt lengths are given (edge and
    long-context cases): tokens uniform in [0, V-1), success rates from the
    workload's mixture at that step, no forced lengths."""
    m = cfg["model"]
    lens = np.asarray(lengths, dtype=np.int32)
    assert lens.min() >= 1 and lens.max() <= cfg["alloc"]["max_prompt"] and len(lens) == cfg["alloc"]["pool_U"]
    master = master_seed(cfg)
    g = np.random.Generator(np.random.PCG64(np.random.SeedSequence([master, 5, step, len(lens)])))
    offsets = np.zeros(len(lens) + 1, dtype=np.int32)
    offsets[1:] = np.cumsum(lens)
    tokens = g.integers(0, m["vocab"] - 1, size=int(offsets[-1])).astype(np.int32)
    wh, we, wm = mixture_weights(cfg, step)
    comp = g.choice(3, size=len(lens), p=[wh, we, wm])
    p = np.where(comp == 0, g.beta(0.3, 3.0, size=len(lens)),
                 np.where(comp == 1, g.beta(3.0, 0.3, size=len(lens)), g.random(size=len(lens))))
    return dict(tokens=tokens, offsets=offsets, p=p.astype(np.float64), forced_len=None, step=step)


def prompt_set(cfg: dict, D: int) -> dict:
    """A finite set of D prompts revisited across allocation steps (history
    warm start): tokens (concatenated), offsets (D+1) and success rates p,
    drawn like a pool's (lengths U[prompt_len], tokens uniform in [0, V-1),
    p from the workload's step-0 mixture)."""
    m = cfg["model"]
    master = master_seed(cfg)
    g = np.random.Generator(np.random.PCG64(np.random.SeedSequence([master, 4, D])))
    lo, hi = cfg["prompt_len"]
    lens = np.minimum(g.integers(lo, hi + 1, size=D), cfg["alloc"]["max_prompt"]).astype(np.int32)
    offsets = np.zeros(D + 1, dtype=np.int32)
    offsets[1:] = np.cumsum(lens)
    tokens = g.integers(0, m["vocab"] - 1, size=int(offsets[-1])).astype(np.int32)
    wh, we, wm = mixture_weights(cfg, 0)
    comp = g.choice(3, size=D, p=[wh, we, wm])
    p = np.where(comp == 0, g.beta(0.3, 3.0, size=D),
                 np.where(comp == 1, g.beta(3.0, 0.3, size=D), g.random(size=D))).astype(np.float64)
    return dict(tokens=tokens, offsets=offsets, p=p)


def set_pool(cfg: dict, pset: dict, step: int) -> dict:
    """Pool of one allocation step over a prompt set: pool_U distinct set
    prompts chosen per step (seeded), in that order; `ids` maps pool index
    to set index.  Forced lengths (if the workload has them) as make_pool's."""
    a = cfg["alloc"]
    U, k = a["pool_U"], a["k"]
    D = len(pset["p"])
    master = master_seed(cfg)
    g = np.random.Generator(np.random.PCG64(np.random.SeedSequence([master, 5, step])))
    ids = g.choice(D, size=U, replace=False).astype(np.int32)
    offs = pset["offsets"]
    parts = [pset["tokens"][offs[i]:offs[i + 1]] for i in ids]
    lens = np.array([len(x) for x in parts], dtype=np.int32)
    offsets = np.zeros(U + 1, dtype=np.int32)
    offsets[1:] = np.cumsum(lens)
    forced = None
    fl = cfg.get("forced_len")
    if fl is not None:
        h = np.random.Generator(np.random.PCG64(np.random.SeedSequence([master, 2, step])))
        z = h.standard_normal(size=(U, k))
        L = np.rint(np.exp(fl["mu"] + fl["sigma"] * z))
        forced = np.clip(L, 1, min(fl["cap"], a["max_new"])).astype(np.int32)
    return dict(tokens=np.concatenate(parts).astype(np.int32), offsets=offsets,
                p=pset["p"][ids].astype(np.float64), forced_len=forced, step=step, ids=ids)


def saturated_pool(pool: dict, seed: int = 7) -> dict:
    """Same prompts with every success rate forced to 0 or 1."""
    q = dict(pool)
    g = np.random.Generator(np.random.PCG64(seed))
    q["p"] = g.integers(0, 2, size=pool["p"].shape[0]).astype(np.float64)
    return q
