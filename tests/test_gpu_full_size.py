"""Full-size parity in the launch configuration bench.py times (HIP-graph
replay, full slot pools and generation lengths): the Qwen2.5-1.5B-shaped
workload (512 slots, 1024 new tokens), the 3B-shaped one (36 layers, forced
EOS 1/800, up to 2048 new tokens) and the long-rollout one at the last step
of its drift (256 binding slots, lognormal forced lengths up to 4096).

The oracle cannot generate a full step, so it checks what it can compute
one by one or what holds at any size:
* controller: the oracle's event simulation fed the GPU's per-rollout
  (length, reward) reproduces every decision, draw, assignment and finish
  bit-exactly (p_eff within 1e-12);
* reward: the oracle's hash chain over each rollout's GPU tokens gives the
  GPU's reward;
* GRPO advantages of the committed groups;
* tokens: at sampled positions (within a rollout's first 384 tokens, which
  bounds the oracle's forward) of sampled rollouts, the oracle's own logits
  (one teacher-forced forward over the GPU's tokens) and sampler give the
  GPU's token (bf16 rounding noise flips a near tie now and then, so >= 90%
  agreement is required);
* logits: the step replayed eagerly for its first decode steps, teacher
  forced with the GPU's own tokens, in the same launch configuration (full
  slot pool, full depth): every row of three sampled rollouts within the
  full-depth bounds of the bf16 slices against the oracle's forward;
* invariants: budget, lengths, committed groups mixed, token count."""
import numpy as np
import pytest

import workloads as W
from oracle import controller as OC
from oracle import grpo as OG
from oracle import reward as OR
from oracle import sampler as OS
from oracle.model import Decoder
from tests.gpu_harness import cached_weights, compare_logs, device_setup, forced_table, run_gpu_step
from tests.test_gpu_bf16_slices import FULL_DEPTH_MAX_REL

pytestmark = pytest.mark.gpu


POSITION_CAP = 384
LOGIT_STEPS = 4


@pytest.mark.parametrize("name,step", [("qwen1p5b_shape", 0), ("qwen3b_shape", 0), ("long_ragged_1p5b", 299)])
def test_full_size_step(name, step):
    import torch
    assert torch.cuda.is_available()
    cfg = W.get_config(name)
    a, m = cfg["alloc"], cfg["model"]
    k, U = a["k"], a["pool_U"]
    pool = W.make_pool(cfg, step)
    print(f"[full] {name} step {step}: {m['n_layers']} layers, {a['n_slots']} slots, max_new {a['max_new']}",
          flush=True)
    seed = W.sampling_seed(cfg)
    ctx, w = device_setup(cfg, cached_weights(cfg))
    print("[full] running the GPU step (graph replay)", flush=True)
    gpu = run_gpu_step(ctx, cfg, pool, use_graph=True)
    # the same step again, eager and teacher forced with the GPU's own tokens,
    # for its first decode steps with the logits captured
    tf = forced_table(cfg, {(u, j): dict(tokens=gpu["roll"]["tokens"][u * k + j][:L])
                            for (t_, s_, u, j, L, r_) in gpu["logs"]["finishes"]})
    print(f"[full] teacher-forced eager replay of the first {LOGIT_STEPS} decode steps", flush=True)
    tfr = run_gpu_step(ctx, cfg, pool, forced=tf, capture_logits=True, max_steps=LOGIT_STEPS)
    ctx.close()
    st = gpu["stats"]
    print(f"[full] GPU: {st['rollouts']} rollouts, {st['tokens']} tokens, {st['committed']} committed, "
          f"{st['decode_steps']} decode steps", flush=True)
    fin = gpu["logs"]["finishes"]
    outcome = {(int(u), int(j)): (int(L), int(r)) for (t, s, u, j, L, r) in fin}

    # controller replay
    ora = OC.simulate(a, U, lambda pairs: [outcome[p] for p in pairs], draw_key=(seed, pool["step"]))
    compare_logs(gpu["logs"], ora)
    assert (st["committed"], st["rollouts"], st["tokens"], st["decode_steps"], st["budget_left"]) == (
        ora["n_committed"], ora["rollouts"], ora["tokens"], ora["decode_steps"], ora["budget_left"])

    # rewards from the GPU's tokens, lengths and invariants
    ro = gpu["roll"]
    for (u, j), (L, r) in outcome.items():
        toks = ro["tokens"][u * k + j][:L]
        assert L <= a["max_new"] and np.all(toks >= 0)
        h = OR.hash_tokens(seed, pool["step"], u, toks)
        assert OR.reward_of_hash(h, float(pool["p"][u])) == r == ro["reward"][u * k + j]
    assert st["rollouts"] <= a["budget_N"] and st["tokens"] == sum(L for L, _ in outcome.values())
    for u in ora["committed"]:
        assert 1 <= ora["successes"][u] <= ora["n_done"][u] - 1

    # GRPO advantages
    off, rw, adv = gpu["adv"]
    offs, rws = [0], []
    for u in ora["committed"]:
        rws += [outcome[(u, j)][1] for j in range(ora["n_issued"][u])]
        offs.append(len(rws))
    assert np.array_equal(off, np.array(offs))
    assert np.allclose(adv, OG.advantages(rws, offs), rtol=1e-6, atol=1e-6)

    # tokens at sampled positions, from the oracle's logits
    dec = Decoder(m, w)
    g = np.random.default_rng(0)
    keys = sorted(outcome)
    picks = [keys[i] for i in g.choice(len(keys), size=3, replace=False)]
    agree, total = 0, 0
    for (u, j) in picks:
        L = outcome[(u, j)][0]
        prompt = pool["tokens"][pool["offsets"][u]:pool["offsets"][u + 1]]
        P = len(prompt)
        gen = ro["tokens"][u * k + j][:L]
        Lc = min(L, POSITION_CAP)
        pos = sorted(set([0, Lc - 1] + list(g.choice(Lc, size=min(6, Lc), replace=False))))
        seq = np.concatenate([prompt, gen[:max(pos)]])
        cache = dec.new_cache(len(seq))
        logits = dec.forward(seq, np.arange(len(seq)), cache, logit_rows=[P - 1 + i for i in pos])
        for n, i in enumerate(pos):
            tok, sc = OS.sample(logits[n], a["temperature"], seed, pool["step"], u * k + j, i)
            if m["eos_id"] >= 0 and OS.forced_eos(seed, pool["step"], u * k + j, i, a["forced_eos_u32"]):
                tok = m["eos_id"]
            agree += int(tok == ro["sampled"][u * k + j][i])
            total += 1
        print(f"[full] rollout ({u},{j}) L={L}: checked positions {pos}", flush=True)
    print(f"[full] sampled-position agreement {agree}/{total}", flush=True)
    assert agree >= 0.9 * total

    # logits of the teacher-forced replay: rows (decode step t, slot) of
    # three rollouts started at the first decode step, against the oracle's
    # forward over the same tokens (the oracle's own fp32-vs-fp64 spread,
    # printed beside, on the first of them)
    assert np.array_equal(tfr["logs"]["assigns"][:len(tfr["logs"]["assigns"])],
                          gpu["logs"]["assigns"][:len(tfr["logs"]["assigns"])])
    first = [(int(s_), int(u), int(j)) for (t0, s_, u, j) in tfr["logs"]["assigns"] if t0 == 0]
    chosen = [first[i] for i in g.choice(len(first), size=3, replace=False)]
    dec64 = Decoder(m, w, gemm_acc="f64")
    worst, worst_rms, floor = 0.0, 0.0, 0.0
    for c, (slot, u, j) in enumerate(chosen):
        L = outcome[(u, j)][0]
        n = min(LOGIT_STEPS, L)
        prompt = pool["tokens"][pool["offsets"][u]:pool["offsets"][u + 1]]
        P = len(prompt)
        seq = np.concatenate([prompt, ro["tokens"][u * k + j][:n - 1]])
        rows = [P - 1 + i for i in range(n)]
        lo = dec.forward(seq, np.arange(len(seq)), dec.new_cache(len(seq)), logit_rows=rows)
        lo64 = dec64.forward(seq, np.arange(len(seq)), dec64.new_cache(len(seq)), logit_rows=rows) if c == 0 else None
        for i in range(n):
            gl = tfr["logits"][i][slot].astype(np.float64)
            o = lo[i].astype(np.float64)
            rms = np.sqrt(np.mean(o * o))
            worst = max(worst, float(np.max(np.abs(gl - o)) / rms))
            worst_rms = max(worst_rms, float(np.sqrt(np.mean((gl - o) ** 2)) / rms))
            if lo64 is not None:
                floor = max(floor, float(np.max(np.abs(lo64[i].astype(np.float64) - o)) / rms))
    print(f"[full] teacher-forced logits of rollouts {[(u, j) for (_, u, j) in chosen]}, steps 0-{LOGIT_STEPS - 1}: "
          f"max|d|/rms {worst:.4f}, relative rms {worst_rms:.4f}, oracle fp32-vs-fp64 {floor:.4f}", flush=True)
    assert worst_rms <= 3e-2
    assert worst <= FULL_DEPTH_MAX_REL[name]
