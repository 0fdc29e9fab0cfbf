"""GPU-vs-oracle parity through the C ABI (needs an MI355X)."""
import math

import numpy as np
import pytest

import workloads as W
from oracle import controller as OC
from oracle import grpo as OG
from oracle import predictor as OP
from oracle import run as ORUN
from oracle import sampler as OS
from tests.gpu_harness import compare_logs, device_setup, forced_table, run_gpu_step, slot_rows, upload_pool

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch_cuda():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    import paper_2607_26253_amd  # noqa: F401  (fails loudly when libsara.so is missing)
    return torch


def test_peff_batch_matches_oracle(torch_cuda):
    """Eq. peff through the C ABI with a prior per prompt: shared priors over
    every (n, s) of several k, then warm-start priors Beta(a0 + a, b0 + b)
    with fractional pseudo-counts (the history warm start's carried counts),
    each entry against the oracle within 1e-12; invalid entries give NaN."""
    import paper_2607_26253_amd as sara
    torch = torch_cuda

    def run(al, be, ns, ss, k):
        f64 = lambda v: torch.tensor(v, dtype=torch.float64, device="cuda")
        i32 = lambda v: torch.tensor(v, dtype=torch.int32, device="cuda")
        out = torch.empty(len(ns), dtype=torch.float64, device="cuda")
        sara.sara_peff_batch(f64(al), f64(be), i32(ns), i32(ss), k, out)
        return out.cpu().numpy()

    for (k, a0, b0) in [(8, 1.0, 1.0), (8, 0.3, 3.0), (16, 2.5, 0.7), (2, 1.0, 1.0), (31, 0.05, 7.5)]:
        ns, ss = [], []
        for n in range(0, k + 1):
            for s in range(0, n + 1):
                ns.append(n)
                ss.append(s)
        got = run([a0] * len(ns), [b0] * len(ns), ns, ss, k)
        want = np.array([OP.p_eff(n, s, k, a0, b0) for n, s in zip(ns, ss)])
        assert np.max(np.abs(got - want)) <= 1e-12
    g = np.random.default_rng(12)
    m, k = 4000, 8
    a = g.choice([0.0, 0.5, 1.75, 3.0, 6.25], m) * g.random(m)
    b = g.choice([0.0, 0.5, 1.75, 3.0, 6.25], m) * g.random(m)
    al, be = 1.0 + a, 1.0 + b
    ns = g.integers(0, k + 1, m)
    ss = np.array([g.integers(0, n + 1) for n in ns])
    got = run(al.tolist(), be.tolist(), ns.tolist(), ss.tolist(), k)
    want = np.array([OP.p_eff(int(n), int(s), k, x, y) for n, s, x, y in zip(ns, ss, al, be)])
    assert np.max(np.abs(got - want)) <= 1e-12
    bad = run([0.0, -1.0, float("inf"), 1.0, 1.0, 1.0], [1.0, 1.0, 1.0, float("nan"), 1.0, 1.0],
              [0, 0, 0, 0, 3, 9], [0, 0, 0, 0, 4, 0], k)
    assert np.all(np.isnan(bad))


def test_poll_reports_done_flag_asynchronously(torch_cuda):
    """sara_poll enqueues a write of (done, error word) into pinned host
    memory and returns at once; the values agree with sara_query mid-step and
    after the step has ended."""
    import time
    import paper_2607_26253_amd as sara
    torch = torch_cuda
    cfg, w, pool, seed = _tiny()
    ctx, _ = device_setup(cfg, w)
    d_tok, d_p, d_fl = upload_pool(pool)
    h = torch.full((2,), -7, dtype=torch.int32).pin_memory()
    ctx.sara_begin_step(d_tok, pool["offsets"], d_p, d_fl, pool["step"])

    def poll():
        h[0] = -1
        ctx.sara_poll(h)
        t0 = time.time()
        while int(h[0]) == -1:
            assert time.time() - t0 < 30.0, "poll flag never arrived"
        return int(h[0]), int(h[1])

    for _ in range(5):
        ctx.sara_decode_step(None, None, False)
        ctx.sara_posterior_decide()
        ctx.sara_refill()
    assert poll() == (0, 0)
    assert ctx.sara_query()["done"] == 0
    ctx.sara_run(None, graph_iters=8)
    assert poll() == (1, 0)
    assert ctx.sara_query()["done"] == 1
    ctx.close()


def test_grpo_matches_oracle(torch_cuda):
    import paper_2607_26253_amd as sara
    torch = torch_cuda
    g = np.random.default_rng(0)
    sizes = [8, 8, 1, 0, 5, 64, 130, 2, 8]
    off = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int32)
    r = np.where(g.random(off[-1]) < 0.4, 1.0, 0.0).astype(np.float32)
    r[8:16] = 1.0   # saturated group
    d_r, d_off = torch.from_numpy(r).cuda(), torch.from_numpy(off).cuda()
    d_a = torch.full((len(r),), 7.0, dtype=torch.float32, device="cuda")
    sara.grpo_group_advantages(d_r, d_off, 1e-6, d_a)
    got = d_a.cpu().numpy()
    want = OG.advantages(r, off, 1e-6)
    assert np.allclose(got, want, rtol=1e-6, atol=1e-6)
    assert np.all(got[8:16] == 0.0)


def test_gumbel_fast_noise_error_bound(torch_cuda):
    """The fused sampler is exact when its fp32 noise estimate stays within
    2e-5 of the exact noise; measured over all 2^24 inputs, with a 2x margin."""
    import paper_2607_26253_amd as sara
    err = sara.sara_gumbel_fast_max_error()
    print(f"max |fast - exact| Gumbel noise over 2^24 inputs: {err:.3e}", flush=True)
    assert 0.0 <= err <= 1e-5


@pytest.mark.parametrize("V", [512, 151936])
def test_sampler_on_oracle_logits(torch_cuda, V):
    import paper_2607_26253_amd as sara
    torch = torch_cuda
    g = np.random.default_rng(V)
    n = 48
    logits = (g.standard_normal((n, V)) * 0.8).astype(np.float32)
    rid = np.arange(n, dtype=np.int32) * 3 + 1
    pos = (np.arange(n, dtype=np.int32) * 7) % 1024
    seed, step = W.sampling_seed(W.get_config("qwen1p5b_shape")), 5
    for temp, eos, feos in [(1.0, -1, 0), (0.7, V - 1, (1 << 32) // 16)]:
        d_tok = torch.empty(n, dtype=torch.int32, device="cuda")
        sara.sara_sample_logits(torch.from_numpy(logits).cuda(), torch.from_numpy(rid).cuda(),
                                torch.from_numpy(pos).cuda(), seed, step, temp, eos, feos, d_tok)
        got = d_tok.cpu().numpy()
        ties = 0
        for i in range(n):
            tok, sc = OS.sample(logits[i], temp, seed, step, int(rid[i]), int(pos[i]))
            if eos >= 0 and OS.forced_eos(seed, step, int(rid[i]), int(pos[i]), feos):
                tok = eos
            if got[i] != tok:
                assert OS.near_tie(sc), (i, got[i], tok)
                ties += 1
        assert ties <= 1


@pytest.mark.parametrize("V", [509, 512, 151936])
def test_top_p_sampler_on_given_logits(torch_cuda, V):
    """Nucleus sampling through the stand-alone entry point against the
    oracle's nucleus and Gumbel-max draw: every token equal, except where the
    oracle's cut lies within 1e-8 of the total weight of its target (an exp
    rounding apart) or the two best scores nearly tie."""
    import paper_2607_26253_amd as sara
    torch = torch_cuda
    g = np.random.default_rng(V + 1)
    small = V < 1000        # 509: rows read one float at a time, else as float4
    n = 24 if small else 10
    scale = np.where(np.arange(n) % 2 == 0, 0.8, 6.0)[:, None]
    logits = (g.standard_normal((n, V)) * scale).astype(np.float32)
    logits[1, : V // 3] = logits[1, 0]          # a large tie group
    logits[3, g.integers(0, V, 64)] = logits[3].max()   # ties at the maximum
    rid = np.arange(n, dtype=np.int32) * 5 + 2
    pos = (np.arange(n, dtype=np.int32) * 11) % 1024
    seed, step = W.sampling_seed(W.get_config("qwen1p5b_shape")), 3
    cases = [(1.0, 0.9), (0.7, 0.5)] if small else [(1.0, 0.95), (1.0, 0.3)]
    if small:
        cases.append((1.3, 1e-6))
    for temp, top_p in cases:
        d_tok = torch.empty(n, dtype=torch.int32, device="cuda")
        sara.sara_sample_logits(torch.from_numpy(logits).cuda(), torch.from_numpy(rid).cuda(),
                                torch.from_numpy(pos).cuda(), seed, step, temp, -1, 0, d_tok, top_p=top_p)
        got = d_tok.cpu().numpy()
        skipped = 0
        for i in range(n):
            tok, sc = OS.sample(logits[i], temp, seed, step, int(rid[i]), int(pos[i]), top_p)
            assert OS.nucleus(logits[i], temp, top_p)[got[i]], (i, top_p)
            if got[i] != tok:
                assert OS.near_tie(sc) or OS.nucleus_margin(logits[i], temp, top_p) < 1e-8, (i, got[i], tok)
                skipped += 1
        print(f"[top-p] V={V} T={temp} top_p={top_p}: {n - skipped}/{n} rows equal", flush=True)
        assert skipped <= 1


def test_tiny_top_p_step_matches_oracle(torch_cuda):
    """A whole allocation step of the fp32 model sampling from the top-p 0.9
    nucleus: teacher-forced logits <= 1e-3, logs bit-exact, the sampler's own
    tokens equal the oracle's, then free running from the captured graph
    reproduces the oracle's rollouts token for token."""
    cfg, w, pool, seed = _tiny()
    cfg["alloc"].update(B=8, budget_N=64, pool_U=32, n_slots=64, max_new=32, top_p=0.9)
    ora = ORUN.run_step(cfg, w, pool, seed, keep_logits=lambda u, j, i: True)
    ctx, _ = device_setup(cfg, w)
    gpu = run_gpu_step(ctx, cfg, pool, forced=forced_table(cfg, ora["rollouts_detail"]), capture_logits=True)
    compare_logs(gpu["logs"], ora)
    worst = max(float(np.max(np.abs(gpu["logits"][t][s] - ora["logits"][(u, j, i)])))
                for (t, s), (u, j, i) in slot_rows(gpu).items())
    assert worst <= 1e-3, worst
    k = cfg["alloc"]["k"]
    diff = sum(int(np.sum(gpu["roll"]["sampled"][u * k + j][:d["length"]] != d["tokens"]))
               for (u, j), d in ora["rollouts_detail"].items())
    assert diff <= 2
    ctx.close()
    ctx, _ = device_setup(cfg, w)
    free = run_gpu_step(ctx, cfg, pool, use_graph=True)
    for (u, j), d in ora["rollouts_detail"].items():
        assert np.array_equal(free["roll"]["tokens"][u * k + j][:d["length"]], d["tokens"]), (u, j)
    compare_logs(free["logs"], ora)
    ctx.close()


def _tiny():
    cfg = W.get_config("tiny_f32")
    w = W.make_weights(cfg)
    pool = W.make_pool(cfg, 0)
    seed = W.sampling_seed(cfg)
    return cfg, w, pool, seed


@pytest.fixture(scope="module")
def tiny_oracle():
    cfg, w, pool, seed = _tiny()
    res = ORUN.run_step(cfg, w, pool, seed, keep_logits=lambda u, j, i: True)
    return cfg, w, pool, seed, res


def test_tiny_teacher_forced_logits_tokens_and_decisions(torch_cuda, tiny_oracle):
    cfg, w, pool, seed, ora = tiny_oracle
    ctx, _ = device_setup(cfg, w)
    forced = forced_table(cfg, ora["rollouts_detail"])
    gpu = run_gpu_step(ctx, cfg, pool, forced=forced, capture_logits=True)
    # decisions, draws, assignments, finishes: bit-exact
    compare_logs(gpu["logs"], ora)
    st = gpu["stats"]
    assert (st["committed"], st["rollouts"], st["tokens"], st["decode_steps"]) == (
        ora["n_committed"], ora["rollouts"], ora["tokens"], ora["decode_steps"])
    # logits of every occupied slot at every step: max |d| <= 1e-3 (fp32 model)
    rows = slot_rows(gpu)
    worst = 0.0
    for (t, s), (u, j, i) in rows.items():
        gl = gpu["logits"][t][s]
        ol = ora["logits"][(u, j, i)]
        worst = max(worst, float(np.max(np.abs(gl - ol))))
    assert worst <= 1e-3, worst
    # the sampler's own choice equals the oracle token except at near ties
    k = cfg["alloc"]["k"]
    ties = 0
    for (u, j), d in ora["rollouts_detail"].items():
        got = gpu["roll"]["sampled"][u * k + j][:d["length"]]
        diff = np.nonzero(got != d["tokens"])[0]
        ties += len(diff)
    assert ties <= 2
    # rewards and GRPO advantages
    for (u, j), d in ora["rollouts_detail"].items():
        assert gpu["roll"]["reward"][u * k + j] == d["reward"]
        assert gpu["roll"]["length"][u * k + j] == d["length"]
    off, r, a = gpu["adv"]
    assert np.array_equal(off, ora["grpo_offsets"])
    assert np.array_equal(r, ora["grpo_rewards"])
    assert np.allclose(a, ora["advantages"], rtol=1e-6, atol=1e-6)
    ctx.close()


def test_tiny_free_running_matches_oracle(torch_cuda, tiny_oracle):
    cfg, w, pool, seed, ora = tiny_oracle
    ctx, _ = device_setup(cfg, w)
    gpu = run_gpu_step(ctx, cfg, pool, use_graph=True)
    k = cfg["alloc"]["k"]
    diverged = False
    for (u, j), d in ora["rollouts_detail"].items():
        got = gpu["roll"]["tokens"][u * k + j][:d["length"]]
        if not np.array_equal(got, d["tokens"]):
            diverged = True
    if not diverged:
        compare_logs(gpu["logs"], ora)
    else:
        pytest.fail("free-running GPU tokens diverged from the oracle")
    ctx.close()


def _model_free_case(cfg, U_tokens_seed=3):
    a = cfg["alloc"]
    U, k, mn = a["pool_U"], a["k"], a["max_new"]
    g = np.random.default_rng(U_tokens_seed)
    V = cfg["model"]["vocab"]
    tab = g.integers(0, V, size=(U * k, mn)).astype(np.int32)
    return tab


@pytest.mark.parametrize("name,mode", [("qwen1p5b_shape", "sara"), ("long_ragged_1p5b", "sara"),
                                       ("pool_3b", "sara"), ("pool_3b", "fixed_k"),
                                       ("qwen3b_shape", "sara"),
                                       ("qwen1p5b_shape", "commit_min=2"), ("qwen1p5b_shape", "commit_min=4"),
                                       ("long_ragged_1p5b", "sara_thompson"),
                                       ("long_ragged_1p5b", "step=150"), ("long_ragged_1p5b", "step=299")])
def test_controller_full_size_model_free(torch_cuda, name, mode):
    """Full-size allocation parameters of each workload; tokens from a table
    (decoder skipped), so the controller, hash reward and termination are
    checked bit-exactly against the oracle's event simulation.  The
    commit_min cases are the early-commit variant (commit at the first mix,
    Theorem 2's proof, and the floor of 4 of the commit-floor ablation): groups
    of 2..8 rollouts, so the GRPO advantages run over variable group sizes.
    The sara_thompson case orders pending rollouts by the posterior-sampling
    index on the workload whose 256 slots bind, so its assignment log differs
    from the p_eff ordering's and must still match the oracle exactly.  The
    step= cases run later steps of the drifting long-rollout workload."""
    full = W.get_config(name)
    if mode == "fixed_k":
        full = W.fixed_k_variant(full)
    elif mode.startswith("commit_min="):
        full["alloc"]["commit_min"] = int(mode.split("=")[1])
    elif mode == "sara_thompson":
        full["alloc"]["mode"] = "sara_thompson"
    step = int(mode.split("=")[1]) if mode.startswith("step=") else 0
    cfg = W.get_config("tiny_f32")
    cfg["alloc"] = dict(full["alloc"])
    cfg["alloc"]["max_prompt"] = 32
    cfg["model"]["eos_id"] = 511
    cfg["forced_len"] = full["forced_len"]
    cfg["index"] = full["index"]
    cfg["steps"] = full["steps"]
    cfg["mixture"] = full["mixture"]
    cfg["prompt_len"] = (8, 32)
    a = cfg["alloc"]
    a["max_new"] = min(a["max_new"], 96)
    if cfg["forced_len"] is not None:
        cfg["forced_len"] = dict(cfg["forced_len"], cap=a["max_new"], mu=math.log(40.0))
    # later steps of the drifting workload: other success-rate weights, the
    # step index in the sampler key and the reward hash
    pool = W.make_pool(cfg, step)
    tab = _model_free_case(cfg)
    # EOS in the table ends rollouts early: sprinkle it with probability 1/40
    g = np.random.default_rng(9)
    tab[g.random(tab.shape) < 1 / 40] = 511
    w = W.make_weights(W.get_config("tiny_f32"))
    ctx, _ = device_setup(cfg, w)
    gpu = run_gpu_step(ctx, cfg, pool, forced=tab, model_free=True)
    seed = W.sampling_seed(cfg)
    ora = ORUN.run_step(cfg, None, pool, seed, forced_tokens=tab, model_free=True)
    compare_logs(gpu["logs"], ora)
    st = gpu["stats"]
    assert (st["committed"], st["rollouts"], st["tokens"], st["decode_steps"], st["budget_left"]) == (
        ora["n_committed"], ora["rollouts"], ora["tokens"], ora["decode_steps"], ora["budget_left"])
    off, r, adv = gpu["adv"]
    assert np.array_equal(off, ora["grpo_offsets"])
    assert np.allclose(adv, ora["advantages"], rtol=1e-6, atol=1e-6)
    if mode.startswith("commit_min="):
        sizes = np.diff(off)
        assert sizes.size == 0 or sizes.min() >= a["commit_min"]
    if mode == "sara_thompson":
        ref = ORUN.run_step(dict(cfg, alloc=dict(a, mode="sara")), None, pool, seed, forced_tokens=tab,
                            model_free=True)
        assert ref["log_assign"] != ora["log_assign"], "slots never bound: the priority made no difference"
    ctx.close()


def test_saturated_pool_abandoned_after_probe(torch_cuda):
    cfg = W.get_config("tiny_f32")
    cfg["alloc"].update(B=64, budget_N=512, n_slots=512, pool_U=256)
    pool = W.saturated_pool(W.make_pool(cfg, 0))
    tab = _model_free_case(cfg)
    w = W.make_weights(W.get_config("tiny_f32"))
    ctx, _ = device_setup(cfg, w)
    gpu = run_gpu_step(ctx, cfg, pool, forced=tab, model_free=True)
    ro = gpu["roll"]
    drawn = gpu["stats"]["drawn"]
    assert gpu["stats"]["committed"] == 0
    assert np.all(ro["status"][:drawn] == 3) and np.all(ro["n"][:drawn] == 4)
    assert gpu["stats"]["rollouts"] == 4 * drawn
    ctx.close()


@pytest.mark.parametrize("lam", [0.5, 1.0])
def test_warm_start_multi_step_model_free(torch_cuda, lam):
    """History warm start over a revisited prompt set: four allocation steps
    with the 1.5B workload's allocation (B=64, k=8, N=512, 512 slots), each
    pool 256 distinct prompts of a 512-prompt set, tokens from a table
    (decoder skipped).  Every step's decision / draw / assignment / finish
    logs are bit-exact against the oracle run under the oracle's carried
    priors, and after every step the device pseudo-counts equal the oracle's
    update exactly."""
    from oracle import warm as OW
    torch = torch_cuda
    full = W.get_config("qwen1p5b_shape")
    cfg = W.get_config("tiny_f32")
    cfg["alloc"] = dict(full["alloc"])
    cfg["alloc"]["max_prompt"] = 32
    cfg["alloc"]["max_new"] = 64
    cfg["model"]["eos_id"] = 511
    cfg["index"] = full["index"]
    cfg["prompt_len"] = (8, 32)
    a = cfg["alloc"]
    U = a["pool_U"]
    D = 2 * U
    pset = W.prompt_set(cfg, D)
    w = W.make_weights(W.get_config("tiny_f32"))
    ctx, _ = device_setup(cfg, w)
    seed = W.sampling_seed(cfg)
    ca, cb = [0.0] * D, [0.0] * D
    d_a = torch.zeros(D, dtype=torch.float64, device="cuda")
    d_b = torch.zeros(D, dtype=torch.float64, device="cuda")
    saved = []
    for step in range(4):
        pool = W.set_pool(cfg, pset, step)
        assert len(set(pool["ids"].tolist())) == U
        d_ids = torch.from_numpy(pool["ids"]).cuda()
        ctx.sara_set_warm_start(d_ids, d_a, d_b)
        tab = _model_free_case(cfg, 30 + step)
        g = np.random.default_rng(40 + step)
        tab[g.random(tab.shape) < 1 / 20] = 511
        print(f"[warm] lambda {lam} step {step}", flush=True)
        gpu = run_gpu_step(ctx, cfg, pool, forced=tab, model_free=True)
        ctx.sara_warm_start_update(lam)
        pri = OW.priors(pool["ids"], ca, cb, a["alpha0"], a["beta0"])
        ora = ORUN.run_step(cfg, None, pool, seed, forced_tokens=tab, model_free=True, priors=pri)
        compare_logs(gpu["logs"], ora)
        st = gpu["stats"]
        assert (st["committed"], st["rollouts"], st["tokens"], st["decode_steps"], st["budget_left"]) == (
            ora["n_committed"], ora["rollouts"], ora["tokens"], ora["decode_steps"], ora["budget_left"])
        assert st["error"] == 0
        ca, cb = OW.update(ca, cb, pool["ids"].tolist(), ora["n_done"], ora["successes"], ora["drawn"], lam)
        torch.cuda.synchronize()
        assert np.array_equal(d_a.cpu().numpy(), np.array(ca))
        assert np.array_equal(d_b.cpu().numpy(), np.array(cb))
        saved.append(ora["rollouts"] / max(ora["drawn"], 1))
        del d_ids
    ctx.sara_set_warm_start(None)
    print(f"[warm] rollouts per drawn prompt by step: {[round(x, 3) for x in saved]}", flush=True)
    ctx.close()


def _edge_pool(cfg, lengths):
    """The workload's pool with prompt lengths cycled from `lengths` (tokens
    regenerated, uniform in [0, V-1))."""
    pool = W.make_pool(cfg, 0)
    U = len(pool["p"])
    lens = np.array([lengths[u % len(lengths)] for u in range(U)], dtype=np.int32)
    offsets = np.zeros(U + 1, dtype=np.int32)
    offsets[1:] = np.cumsum(lens)
    g = np.random.default_rng(77)
    pool["tokens"] = g.integers(0, cfg["model"]["vocab"] - 1, size=int(offsets[-1])).astype(np.int32)
    pool["offsets"] = offsets
    return pool


@pytest.mark.parametrize("name", ["tiny_f32", "qwen1p5b_shape"])
def test_prompt_length_edges(torch_cuda, name):
    """Prompts of 1 token (no prompt KV: the first generated token attends to
    itself only), 2, 15-17 (one page and its neighbours), 31-33 and the
    maximum; teacher-forced logits against the oracle (fp32: <= 1e-3; bf16
    2-layer slice: <= 3e-2 rms) and every log bit-exact."""
    from tests.test_gpu_bf16_slices import row_errors
    if name == "tiny_f32":
        cfg = W.get_config("tiny_f32")
        cfg["alloc"].update(B=4, budget_N=32, n_slots=32, pool_U=16, max_new=12)
        lengths = [1, 16, 17, 32, 2, 15, 31, 1]
    else:
        full = W.get_config(name)
        cfg = W.parity_slice(full, B=3, N=32, prompt_len=(1, 48), max_new=10, pool_U=8)
        cfg["model"]["n_layers"] = 2
        lengths = [1, 17, 16, 48, 2, 15, 33, 1]
    w = W.make_weights(cfg)
    pool = _edge_pool(cfg, lengths)
    seed = W.sampling_seed(cfg)
    ora = ORUN.run_step(cfg, w, pool, seed, keep_logits=lambda u, j, i: True)
    drawn_lens = {int(pool["offsets"][u + 1] - pool["offsets"][u]) for (u, _j) in ora["rollouts_detail"]}
    assert 1 in drawn_lens and 16 in drawn_lens and 17 in drawn_lens
    ctx, _ = device_setup(cfg, w)
    gpu = run_gpu_step(ctx, cfg, pool, forced=forced_table(cfg, ora["rollouts_detail"]), capture_logits=True)
    compare_logs(gpu["logs"], ora)
    if name == "tiny_f32":
        worst = max(float(np.max(np.abs(gpu["logits"][t][s] - ora["logits"][(u, j, i)])))
                    for (t, s), (u, j, i) in slot_rows(gpu).items())
        assert worst <= 1e-3, worst
    else:
        worst = max(e["max"] for e in row_errors(gpu, ora["logits"]))
        assert worst <= 3e-2, worst
    print(f"[edges] {name}: prompt lengths {sorted(drawn_lens)}, worst {worst:.3g}", flush=True)
    ctx.close()


@pytest.mark.parametrize("over", [dict(budget_N=7), dict(n_slots=1, budget_N=24), dict(max_new=1),
                                  dict(n0=8, commit_min=8), dict(n0=1, commit_min=2, B=1),
                                  dict(pool_U=1, B=4)])
def test_tiny_allocation_edges(torch_cuda, over):
    """Degenerate allocations on the fp32 model: a budget below one
    reservation (nothing drawn, the step ends at once), a single slot, one
    generated token per rollout, all k probes at once, a goal of one group
    committed at the first mix, and a one-prompt pool; every log and count
    bit-exact against the oracle."""
    cfg = W.get_config("tiny_f32")
    cfg["alloc"].update(B=4, budget_N=32, n_slots=16, pool_U=12, max_new=6)
    cfg["alloc"].update(over)
    w = W.make_weights(cfg)
    pool = W.make_pool(cfg, 0)
    seed = W.sampling_seed(cfg)
    ora = ORUN.run_step(cfg, w, pool, seed, keep_logits=lambda u, j, i: True)
    ctx, _ = device_setup(cfg, w)
    gpu = run_gpu_step(ctx, cfg, pool, forced=forced_table(cfg, ora["rollouts_detail"]))
    compare_logs(gpu["logs"], ora)
    st = gpu["stats"]
    assert (st["committed"], st["rollouts"], st["tokens"], st["decode_steps"], st["budget_left"], st["drawn"]) == (
        ora["n_committed"], ora["rollouts"], ora["tokens"], ora["decode_steps"], ora["budget_left"], ora["drawn"])
    if over.get("budget_N") == 7:
        assert st["drawn"] == 0 and st["decode_steps"] == 0 and st["done"] == 1
    off, r, a = gpu["adv"]
    assert np.array_equal(off, ora["grpo_offsets"])
    assert np.allclose(a, ora["advantages"], rtol=1e-6, atol=1e-6)
    ctx.close()


def test_ablation_sweeps_with_exact_counterfactuals(torch_cuda):
    """The tau, n0 and k ablations on the device, with exact counterfactual
    labels (mechanism and ablation figures: sweeps, lost groups, decision
    quality, Fig. 3a and 3c analogs).  Model-free rollouts of equal length
    over a 2048-prompt pool of the success-rate mixture; for every k the
    fixed-k run on the same token table labels each drawn prompt with its
    full group (its first n rewards are SARA's, by the logical rollout keys).
    At every point: the GPU's decision, draw, assignment and finish logs equal
    the oracle's; the table rows computed from the GPU's results equal the
    oracle-written golden file tests/golden/ablation_sweeps.txt; each
    abandonment happens at n_stop = max(n0, k - floor(tau (k+1))) on an
    all-same prefix and each commit at n = k on a mixed one; and the rollouts
    per drawn prompt match sum_u [n_stop + (k - n_stop) q_u],
    q_u = 1 - p_u^n_stop - (1-p_u)^n_stop, within 5 sigma."""
    from tests.golden import make_ablation_table as AB
    w = W.make_weights(W.get_config("tiny_f32"))
    golden = AB.read_golden()
    labels, label_runs = {}, {}

    def gpu_run(cfg):
        pool = W.make_pool(cfg, 0)
        ctx, _ = device_setup(cfg, w)
        g = run_gpu_step(ctx, cfg, pool, forced=AB.token_table(cfg), model_free=True)
        ctx.close()
        ora, _ = AB.oracle_run(cfg)
        compare_logs(g["logs"], ora)
        st, rs = g["stats"], g["roll"]
        return g, dict(drawn=st["drawn"], rollouts=st["rollouts"], committed=st["committed"],
                       decode_steps=st["decode_steps"], status=rs["status"], n=rs["n"], reward=rs["reward"],
                       decisions=g["logs"]["decisions"][:, :5], assigns=g["logs"]["assigns"]), pool

    lines = []
    for (k, n0, tau) in AB.POINTS:
        if k not in labels:
            _, lab, _ = gpu_run(AB.label_config(k))
            labels[k], label_runs[k] = lab["reward"], lab
        cfg = AB.point_config(k, n0, tau)
        g, run, pool = gpu_run(cfg)
        p = pool["p"]
        st, rs = g["stats"], g["roll"]
        assert label_runs[k]["drawn"] >= st["drawn"]
        ns = AB.n_stop(k, n0, tau)
        want, var = 0.0, 0.0
        for u in range(st["drawn"]):
            n, s_ = int(rs["n"][u]), int(rs["s"][u])
            assert np.array_equal(rs["reward"][u * k:u * k + n], labels[k][u * k:u * k + n])
            if rs["status"][u] == 2:
                assert n == k and 1 <= s_ <= k - 1
            else:
                assert rs["status"][u] == 3 and n == ns and s_ in (0, n)
            q = 1 - p[u] ** ns - (1 - p[u]) ** ns
            want += ns + (k - ns) * q
            var += (k - ns) ** 2 * q * (1 - q)
        assert abs(st["rollouts"] - want) <= 5 * math.sqrt(var) + 1e-9
        lines += AB.summarize(k, n0, tau, run, labels[k])
        if (k, n0, tau) == AB.DEFAULT:
            lines.append(AB.fig3c("sara", k, run))
            lines.append(AB.fig3c("fixed_k", k, label_runs[k]))
    for l in lines:
        print("[sweep]", l, flush=True)
    assert lines == golden


@pytest.mark.parametrize("variant", ["warm_start", "thompson"])
def test_graph_replay_matches_eager_over_steps(torch_cuda, variant):
    """The captured decode / decide / refill graph and the eager calls give
    the same step, step after step, with warm-start priors carried between
    steps or with the posterior-sampling priority on binding slots (fp32
    model, three steps, free-running tokens): identical tokens, logs and
    counts, and (warm start) identical carried pseudo-counts."""
    from oracle import warm as OW  # noqa: F401  (the reading both paths implement)
    torch = torch_cuda
    cfg = W.get_config("tiny_f32")
    cfg["alloc"].update(B=8, budget_N=64, pool_U=24, n_slots=64 if variant == "warm_start" else 6, max_new=16)
    if variant == "thompson":
        cfg["alloc"]["mode"] = "sara_thompson"
    w = W.make_weights(cfg)
    D = 48
    pset = W.prompt_set(cfg, D)
    runs = []
    for use_graph in (False, True):
        ctx, _ = device_setup(cfg, w)
        d_a = torch.zeros(D, dtype=torch.float64, device="cuda")
        d_b = torch.zeros(D, dtype=torch.float64, device="cuda")
        out = []
        for step in range(3):
            pool = W.set_pool(cfg, pset, step)
            d_ids = torch.from_numpy(pool["ids"]).cuda()
            if variant == "warm_start":
                ctx.sara_set_warm_start(d_ids, d_a, d_b)
            g = run_gpu_step(ctx, cfg, pool, use_graph=use_graph)
            if variant == "warm_start":
                ctx.sara_warm_start_update(0.5)
            torch.cuda.synchronize()
            out.append((g, d_a.cpu().numpy().copy(), d_b.cpu().numpy().copy()))
        ctx.close()
        runs.append(out)
    for step, ((ge, ae, be), (gg, ag, bg)) in enumerate(zip(*runs)):
        for key in ("decisions", "draws", "assigns", "finishes"):
            assert np.array_equal(ge["logs"][key], gg["logs"][key]), (step, key)
        assert np.array_equal(ge["roll"]["tokens"], gg["roll"]["tokens"]), step
        for f in ("committed", "rollouts", "tokens", "decode_steps", "budget_left"):
            assert ge["stats"][f] == gg["stats"][f], (step, f)
        assert np.array_equal(ae, ag) and np.array_equal(be, bg)
    if variant == "warm_start":
        assert np.any(runs[0][-1][1] > 0) or np.any(runs[0][-1][2] > 0)
