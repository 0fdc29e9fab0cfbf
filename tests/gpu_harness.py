"""Helpers that run the HIP path through the C ABI and line its results up
with the oracle's (tests only)."""
import numpy as np

import workloads as W


_WEIGHTS = {}


_WEIGHT_CACHE_MODELS = 8


def cached_weights(cfg):
    """Weights of cfg's model (its shape and master seed), generated once per
    test session and shared by every test of that model: the four workloads'
    full models and their 2-layer truncations hold about 26 GB of host
    memory; beyond _WEIGHT_CACHE_MODELS models the least recently used goes."""
    key = (W.master_seed(cfg), tuple(sorted(cfg["model"].items())))
    if key in _WEIGHTS:
        _WEIGHTS[key] = _WEIGHTS.pop(key)          # most recently used last
    else:
        while len(_WEIGHTS) >= _WEIGHT_CACHE_MODELS:
            _WEIGHTS.pop(next(iter(_WEIGHTS)))
        _WEIGHTS[key] = W.make_weights(cfg)
    return _WEIGHTS[key]


def device_setup(cfg, weights=None):
    import torch

    import paper_2607_26253_amd as sara
    if weights is None:
        weights = W.make_weights(cfg)
    specs = W.weight_specs(cfg["model"])
    dw = sara.upload_weights(specs, weights)
    ctx = sara.Sara(cfg["model"], cfg["alloc"], W.sampling_seed(cfg), dw)
    del dw
    torch.cuda.synchronize()
    return ctx, weights


def upload_pool(pool):
    import torch
    d_tok = torch.from_numpy(pool["tokens"]).cuda()
    d_p = torch.from_numpy(pool["p"]).cuda()
    d_fl = torch.from_numpy(np.ascontiguousarray(pool["forced_len"].reshape(-1))).cuda() \
        if pool.get("forced_len") is not None else None
    return d_tok, d_p, d_fl


def forced_table(cfg, rollouts_detail, key="tokens"):
    a = cfg["alloc"]
    tab = np.zeros((a["pool_U"] * a["k"], a["max_new"]), np.int32)
    for (u, j), d in rollouts_detail.items():
        t = d[key]
        tab[u * a["k"] + j, :len(t)] = t
    return tab


def run_gpu_step(ctx, cfg, pool, forced=None, model_free=False, capture_logits=False,
                 use_graph=False, max_steps=1_000_000):
    """Drive one allocation step; returns stats, logs, rollouts and (optionally)
    the logits of every occupied slot at every decode step."""
    import torch
    d_tok, d_p, d_fl = upload_pool(pool)
    d_forced = torch.from_numpy(forced).cuda() if forced is not None else None
    ctx.sara_begin_step(d_tok, pool["offsets"], d_p, d_fl, pool["step"])
    logits = {}
    S, V = cfg["alloc"]["n_slots"], cfg["model"]["vocab"]
    if use_graph and not capture_logits and not model_free:
        ctx.sara_run(d_forced, graph_iters=8)
    else:
        buf = torch.zeros((S, V), dtype=torch.float32, device="cuda") if capture_logits else None
        for t in range(max_steps):
            q = ctx.sara_query()
            if q["done"]:
                break
            ctx.sara_decode_step(d_forced, buf, model_free)
            if capture_logits:
                logits[t] = buf.cpu().numpy().copy()
            ctx.sara_posterior_decide()
            ctx.sara_refill()
    ctx.sara_finish_step(1e-6)
    stats = ctx.sara_query()
    logs = ctx.read_logs()
    roll = ctx.read_rollouts()
    adv = ctx.read_advantages()
    torch.cuda.synchronize()
    return dict(stats=stats, logs=logs, roll=roll, adv=adv, logits=logits)


def oracle_logs(res):
    """Oracle logs in the ABI's row formats."""
    dec = np.array([(t, u, d, n, s, 0) for (t, u, d, n, s, _) in res["log_decisions"]], np.int64).reshape(-1, 6)
    pe = np.array([x[5] for x in res["log_decisions"]], np.float64)
    draws = np.array(res["log_draws"], np.int64).reshape(-1, 2)
    asg = np.array(res["log_assign"], np.int64).reshape(-1, 4)
    fin = np.array(res["log_finish"], np.int64).reshape(-1, 6)
    return dict(decisions=dec, p_eff=pe, draws=draws, assigns=asg, finishes=fin)


def compare_logs(gpu_logs, ora):
    o = oracle_logs(ora)
    g = gpu_logs
    assert np.array_equal(g["draws"], o["draws"]), "draw log differs"
    assert np.array_equal(g["assigns"], o["assigns"]), "assignment log differs"
    assert np.array_equal(g["finishes"], o["finishes"]), "finish log differs"
    assert np.array_equal(g["decisions"][:, :5], o["decisions"][:, :5]), "decision log differs"
    assert np.max(np.abs(g["p_eff"] - o["p_eff"]), initial=0.0) <= 1e-12


def slot_rows(gpu):
    """(t, slot) -> (uid, j, gen) from the assignment and finish logs."""
    L = {}
    for (t, s, u, j, Ln, r) in gpu["logs"]["finishes"]:
        L[(u, j)] = Ln
    m = {}
    for (t0, s, u, j) in gpu["logs"]["assigns"]:
        for g in range(L[(u, j)]):
            m[(t0 + g, s)] = (u, j, g)
    return m
