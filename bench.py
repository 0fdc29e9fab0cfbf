"""Benchmark of the SARA rollout-allocation hot path on one MI355X.

One bench step = one allocation step of the named workload: prefill of the
step's prompt pool, the decode / decide / refill loop until no prompt is
active (replayed from a HIP graph), and GRPO advantages of the committed
groups.  Inputs (weights, prompt pools) are resident in HBM before the timed
region.  Prints one JSON line.

value  = rollout tokens generated per second over the timed steps.  Whole
allocation steps are timed until --steps are done or --time-budget seconds
are spent (always at least one); `steps` and `warmup` report the counts
actually run.
roofline: one further allocation step replayed from the same graph, with one
eager iteration after every --profile-chunk loop iterations whose kernels are
timed from the dispatch's own start/end stamps (HIP events on the library's
stream); the dominant kernel is the class with the largest summed time, its
achieved rate is algorithmic bytes (or flops, when its intensity is past the
ridge point) per launch over its mean duration.
cpu_baseline: the CPU oracle generating rollouts of the same model shape on a
bounded sample (two prompts' prefill + a few rollouts x a few tokens).
"""
import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import workloads as W  # noqa: E402

HBM_PEAK_GBS = 8000.0
BF16_PEAK_TFLOPS = 2500.0
TRAFFIC_PROFILE = os.path.join(ROOT, "profiles", "hbm_traffic_decode_qwen1p5b_shape_32rows.md")
KERNEL_SOURCE = os.path.join(ROOT, "paper_2607_26253_amd", "csrc", "model_kernels.hip")


# the workload and options the committed counter summary was taken on
TRAFFIC_WORKLOAD = "qwen1p5b_shape"


def measured_traffic(kernel, cfg, mode="sara", top_p=1.0):
    """HBM-side bytes per launch of `kernel` from the committed rocprofv3
    FETCH_SIZE / WRITE_SIZE summary (calibrated on a copy of known size), with
    the algorithmic bytes of the same launches; None when the summary does not
    cover the kernel, was taken on another workload (the counters depend on
    the weight shapes) or the kernel source changed since it was taken."""
    if cfg["name"] != TRAFFIC_WORKLOAD or mode != "sara" or top_p != 1.0:
        return None
    import hashlib
    try:
        text = open(TRAFFIC_PROFILE).read()
        src = hashlib.sha256(open(KERNEL_SOURCE, "rb").read()).hexdigest()
    except OSError:
        return None
    if f"model_kernels.hip sha256 {src}" not in text:
        return None
    for line in text.splitlines():
        cells = [c.strip() for c in line.strip().strip("|").split("|")]
        if len(cells) == 7 and cells[0] == f"`{kernel}`" and cells[5] != "-":
            return {"traffic": float(cells[4]), "alg_bytes_per_launch": float(cells[5]), "ratio": float(cells[6]),
                    "regime": "16 eager decode iterations at 32 rows (start of allocation step 0, goal B = 16)",
                    "source": os.path.relpath(TRAFFIC_PROFILE, ROOT)}
    return None


def describe(cfg):
    m, a = cfg["model"], cfg["alloc"]
    return (f"{cfg['name']}: {m['n_layers']}L d{m['d_model']} {m['n_heads']}Q/{m['n_kv_heads']}KV x{m['head_dim']} "
            f"ffn{m['d_ffn']} V{m['vocab']} {m['dtype']}; B={a['B']} k={a['k']} n0={a['n0']} tau={a['tau_low']} "
            f"N={a['budget_N']} slots={a['n_slots']} pool={a['pool_U']} prompts U{list(cfg['prompt_len'])} "
            f"max_new={a['max_new']} mode={a['mode']}" + (f" top_p={a['top_p']}" if a.get("top_p", 1.0) != 1.0 else ""))


def cpu_baseline(cfg, weights):
    """Oracle rollout generation rate on a bounded sample, host cores (about
    10-15 s on a 16-thread host: prefill of two prompts, then 32 lockstep
    decode steps of 8 rollouts)."""
    from oracle import run as ORUN
    try:
        from threadpoolctl import threadpool_info
        threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [os.cpu_count()])
    except Exception:
        threads = os.cpu_count()
    c = W.get_config(cfg["name"])
    a = c["alloc"]
    pool = W.make_pool(c, 10_000)
    seed = W.sampling_seed(c)
    src = ORUN.RolloutSource(c, weights, pool, seed)
    t0 = time.time()
    for name, _ in W.weight_specs(c["model"]):   # weight conversion outside the timing
        src.dec.w(name)
    t_setup = time.time() - t0
    prompts, rollouts, new_tokens = 2, 4, 32
    a_max = a["max_new"]
    src.a = dict(a, max_new=new_tokens)
    t0 = time.time()
    pairs = [(u, j) for u in range(prompts) for j in range(rollouts)]
    src._generate(pairs)
    t_run = time.time() - t0
    n_tok = sum(src.results[pr]["length"] for pr in pairs)
    P = [int(pool["offsets"][u + 1] - pool["offsets"][u]) for u in range(prompts)]
    src.a = dict(a, max_new=a_max)
    return dict(value=n_tok / t_run, unit="tokens/s", cores=int(threads), kind="oracle",
                sample=(f"{cfg['name']} shape: prefill of {prompts} prompts ({P} tokens) + {rollouts} rollouts "
                        f"each x up to {new_tokens} tokens, lockstep ({n_tok} generated tokens / wall time incl. "
                        f"prefill; weight conversion {t_setup:.1f}s excluded)"),
                seconds=t_run)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=2)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--config", default="qwen1p5b_shape")
    ap.add_argument("--mode", default="sara", choices=["sara", "fixed_k", "sara_thompson"],
                    help="allocation rule: SARA (default), the fixed-k baseline on the whole pool "
                         "(every drawn prompt gets its k rollouts at once), or SARA with the "
                         "posterior-sampling queue priority")
    ap.add_argument("--top-p", type=float, default=1.0,
                    help="nucleus sampling mass (default 1: the full softmax, as every workload uses)")
    ap.add_argument("--first-step", type=int, default=0,
                    help="allocation-step index of the first pool (the long-rollout workload's success-rate "
                         "mixture drifts with it); warm-up, timed and profiled steps take consecutive indices")
    ap.add_argument("--graph-iters", type=int, default=16)
    ap.add_argument("--chunk-iters", type=int, default=2048)
    ap.add_argument("--time-budget", type=float, default=60.0,
                    help="wall-clock seconds of timed work: whole allocation steps run until --steps are "
                         "done or this is spent (at least one); the line reports the steps actually timed")
    ap.add_argument("--warmup-budget", type=float, default=10.0,
                    help="further warm-up steps start only within this many seconds (one always runs)")
    ap.add_argument("--profile-budget", type=float, default=45.0,
                    help="wall-clock seconds of the kernel-timed pass")
    ap.add_argument("--profile-chunk", type=int, default=48,
                    help="graph-replayed loop iterations between two kernel-timed eager iterations")
    ap.add_argument("--no-profile", action="store_true")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--counter-pass", type=int, default=0,
                    help="counter mode: run this many eager decode/decide/refill iterations of step 0 with "
                         "per-kernel event profiling and print each kernel class's algorithmic bytes per "
                         "launch (pair it with rocprofv3 --pmc over the same run), then exit")
    ap.add_argument("--counter-rows", type=int, default=0,
                    help="counter mode: goal B = rows / n0, so the first decode iterations run about this "
                         "many rows (default: the workload's B)")
    ap.add_argument("--decode-iters", type=int, default=0,
                    help="profiling mode: only replay this many decode/decide/refill iterations of "
                         "step 0 from the HIP graph (for kernel traces), then exit")
    args = ap.parse_args()
    if args.steps < 1 or args.warmup < 0:
        ap.error("--steps must be >= 1 and --warmup >= 0")
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for {args.gpus}): the allocation step would "
              f"shard by prompts (a model replica, slot pool and controller per GPU, no traffic "
              f"inside a step), which this benchmark does not launch.", file=sys.stderr)
        sys.exit(2)

    import torch

    import paper_2607_26253_amd as sara
    assert torch.cuda.is_available(), "bench.py needs a HIP device"
    torch.cuda.set_device(0)
    cfg = W.get_config(args.config)
    if args.mode == "fixed_k":
        cfg = W.fixed_k_variant(cfg)
    elif args.mode == "sara_thompson":
        cfg["alloc"]["mode"] = "sara_thompson"
    if args.top_p != 1.0:
        cfg["alloc"]["top_p"] = args.top_p
    if args.counter_pass and args.counter_rows:
        cfg["alloc"]["B"] = max(1, args.counter_rows // cfg["alloc"]["n0"])
    t0 = time.time()
    weights = W.make_weights(cfg)
    t_w = time.time() - t0
    print(f"[bench] {describe(cfg)}; weights generated in {t_w:.1f}s", file=sys.stderr, flush=True)
    dw = sara.upload_weights(W.weight_specs(cfg["model"]), weights)
    ctx = sara.Sara(cfg["model"], cfg["alloc"], W.sampling_seed(cfg), dw)
    del dw
    torch.cuda.synchronize()
    torch.cuda.empty_cache()

    if args.counter_pass:
        p = W.make_pool(cfg, 0)
        d_tok, d_p = torch.from_numpy(p["tokens"]).cuda(), torch.from_numpy(p["p"]).cuda()
        d_fl = torch.from_numpy(np.ascontiguousarray(p["forced_len"].reshape(-1))).cuda() \
            if p["forced_len"] is not None else None
        ctx.sara_begin_step(d_tok, p["offsets"], d_p, d_fl, p["step"])
        torch.cuda.synchronize()
        print("[bench] counter pass: prefill done", file=sys.stderr, flush=True)
        ctx.sara_reset_profile()
        ctx.sara_set_profiling(True)
        for it in range(args.counter_pass):
            ctx.sara_decode_step(None, None, False)
            ctx.sara_posterior_decide()
            ctx.sara_refill()
        ctx.sara_set_profiling(False)
        prof = ctx.sara_read_profile()
        q = ctx.sara_query()
        print(json.dumps({"mode": "counter_pass", "workload": describe(cfg), "iters": args.counter_pass,
                          "running_slots": q["running"],
                          "classes": {k["name"]: {"launches": k["launches"],
                                                  "alg_bytes_per_launch": k["bytes"] / k["launches"],
                                                  "alg_flops_per_launch": k["flops"] / k["launches"],
                                                  "event_us": 1e3 * k["ms"] / k["launches"]}
                                      for k in prof if k["launches"] > 0}}), flush=True)
        ctx.close()
        return

    if args.decode_iters:
        p = W.make_pool(cfg, 0)
        d_tok, d_p = torch.from_numpy(p["tokens"]).cuda(), torch.from_numpy(p["p"]).cuda()
        d_fl = torch.from_numpy(np.ascontiguousarray(p["forced_len"].reshape(-1))).cuda() \
            if p["forced_len"] is not None else None
        ctx.sara_begin_step(d_tok, p["offsets"], d_p, d_fl, p["step"])
        torch.cuda.synchronize()
        print("[bench] decode-iters: prefill done", file=sys.stderr, flush=True)
        ctx.sara_run(None, graph_iters=args.graph_iters, max_iters=args.graph_iters)
        torch.cuda.synchronize()
        print("[bench] decode-iters: graph captured and replayed once", file=sys.stderr, flush=True)
        t0 = time.perf_counter()
        n = ctx.sara_run(None, graph_iters=args.graph_iters, max_iters=args.decode_iters)
        dt = time.perf_counter() - t0
        q = ctx.sara_query()
        print(json.dumps({"mode": "decode_iters", "workload": describe(cfg), "iters": n,
                          "ms_per_iter": 1e3 * dt / n, "running_slots": q["running"], "tokens": q["tokens"]}))
        ctx.close()
        return

    # Whole allocation steps run until the requested count is reached or the
    # step's wall-clock budget is spent (one step of the 1.5B workload takes
    # tens of seconds); the line reports the counts actually run.
    n_pools = max(1, args.warmup) + max(1, args.steps) + 1
    pools = []
    for s in range(n_pools):
        p = W.make_pool(cfg, args.first_step + s)
        d_tok = torch.from_numpy(p["tokens"]).cuda()
        d_p = torch.from_numpy(p["p"]).cuda()
        d_fl = torch.from_numpy(np.ascontiguousarray(p["forced_len"].reshape(-1))).cuda() \
            if p["forced_len"] is not None else None
        pools.append((p, d_tok, d_p, d_fl))
    torch.cuda.synchronize()

    def one_step(i, tag):
        p, d_tok, d_p, d_fl = pools[i]
        ctx.sara_begin_step(d_tok, p["offsets"], d_p, d_fl, p["step"])
        iters = 0
        while True:
            # replay the decode/decide/refill graph in chunks; each chunk reports progress
            iters += ctx.sara_run(None, graph_iters=args.graph_iters, max_iters=args.chunk_iters)
            q = ctx.sara_query()
            print(f"[bench] {tag}: {iters} loop iterations, {q['tokens']} tokens, {q['committed']} committed",
                  file=sys.stderr, flush=True)
            if q["done"]:
                break
        ctx.sara_finish_step(1e-6)
        return ctx.sara_query()

    # warm-up: builds and instantiates the decode graph (one step is enough)
    n_warm, tw = 0, time.perf_counter()
    while n_warm < args.warmup and (n_warm == 0 or time.perf_counter() - tw < args.warmup_budget):
        st = one_step(n_warm, f"warmup {n_warm}")
        print(f"[bench] warmup step {n_warm}: {st['tokens']} tokens, {st['decode_steps']} decode steps",
              file=sys.stderr, flush=True)
        n_warm += 1

    torch.cuda.synchronize()
    stats = []
    t0 = time.perf_counter()
    while len(stats) < args.steps:
        i = len(stats)
        stats.append(one_step(n_warm + i, f"step {i}"))
        if time.perf_counter() - t0 >= args.time_budget:
            break
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    n_steps = len(stats)
    for i, st in enumerate(stats):
        print(f"[bench] step {i}: tokens {st['tokens']} rollouts {st['rollouts']} committed {st['committed']} "
              f"abandoned {st['abandoned']} drawn {st['drawn']} decode steps {st['decode_steps']}",
              file=sys.stderr, flush=True)
    tokens = sum(s["tokens"] for s in stats)
    committed = sum(s["committed"] for s in stats)
    rollouts = sum(s["rollouts"] for s in stats)
    decode_steps = sum(s["decode_steps"] for s in stats)

    out = {
        "metric": "rollout tokens/s + effective groups/s on 1 GPU; decode HBM GB/s % of peak",
        "value": tokens / dt, "unit": "tokens/s", "n_gpus": 1, "steps": n_steps,
        "warmup": n_warm, "ms_per_step": 1e3 * dt / n_steps, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": cfg["model"]["dtype"],
        "data": "synthetic (random-init weights, seeded prompt pools and success rates)",
        "config": {"workload": describe(cfg),
                   "allocation_steps": [args.first_step + n_warm + i for i in range(n_steps)]},
        "steps_requested": args.steps, "warmup_requested": args.warmup,
        "time_budget_s": args.time_budget, "timed_s": dt,
        "effective_groups_per_s": committed / dt,
        "rollouts_per_effective_group": (rollouts / committed) if committed else None,
        "tokens_per_effective_group": (tokens / committed) if committed else None,
        "decode_steps_per_s": decode_steps / dt,
        "per_step": [{k: s[k] for k in ("tokens", "rollouts", "committed", "abandoned", "drawn", "decode_steps")}
                     for s in stats],
    }

    if not args.no_profile:
        # One further allocation step on its own pool, replayed from the same
        # graph in chunks of --profile-chunk loop iterations, with one eager
        # iteration after each chunk timed kernel by kernel: the sample spans
        # the whole step (every occupancy it goes through) at graph speed.
        p, d_tok, d_p, d_fl = pools[n_warm + n_steps]
        ctx.sara_begin_step(d_tok, p["offsets"], d_p, d_fl, p["step"])
        ctx.sara_reset_profile()
        it, n_prof, done = 0, 0, False
        tprof = time.perf_counter()
        while not done and time.perf_counter() - tprof < args.profile_budget:
            ctx.sara_set_profiling(True)
            ctx.sara_decode_step(None, None, False)
            ctx.sara_set_profiling(False)
            ctx.sara_posterior_decide()
            ctx.sara_refill()
            it += 1
            n_prof += 1
            it += ctx.sara_run(None, graph_iters=args.graph_iters, max_iters=args.profile_chunk)
            done = bool(ctx.sara_query()["done"])
            if n_prof % 64 == 0:
                print(f"[bench] profiled pass: {it} loop iterations, {n_prof} profiled",
                      file=sys.stderr, flush=True)
        prof = ctx.sara_read_profile()
        tprof = time.perf_counter() - tprof
        allc = [k for k in prof if k["launches"] > 0]
        dec = [k for k in allc if not k["name"].startswith(".")]      # kernels (no sub-classes)
        tot_ms = sum(k["ms"] for k in dec)
        tot_by = sum(k["bytes"] for k in dec)
        dom = max(dec, key=lambda k: k["ms"])
        per_launch_ms = dom["ms"] / dom["launches"]
        per_launch_by = dom["bytes"] / dom["launches"]
        per_launch_fl = dom["flops"] / dom["launches"]
        ach_gbs = per_launch_by / (per_launch_ms * 1e-3) / 1e9
        ach_tfs = per_launch_fl / (per_launch_ms * 1e-3) / 1e12
        # roof from the kernel's arithmetic intensity against the ridge point
        # (peak flop/s over peak byte/s)
        ridge = BF16_PEAK_TFLOPS * 1e12 / (HBM_PEAK_GBS * 1e9)
        mfma = cfg["model"]["dtype"] == "bf16" and per_launch_by > 0 and per_launch_fl / per_launch_by > ridge
        tr = measured_traffic(dom["name"], cfg, args.mode, args.top_p)
        out["roofline"] = {
            "kernel": dom["name"], "bound": "mfma" if mfma else "hbm",
            "achieved": ach_tfs if mfma else ach_gbs,
            "peak": BF16_PEAK_TFLOPS if mfma else HBM_PEAK_GBS, "unit": "TFLOP/s" if mfma else "GB/s",
            "frac": (ach_tfs / BF16_PEAK_TFLOPS) if mfma else (ach_gbs / HBM_PEAK_GBS),
            "traffic": tr["traffic"] if tr else None,
            "traffic_measured_at": ({k: tr[k] for k in ("regime", "alg_bytes_per_launch", "ratio", "source")}
                                    if tr else None),
            "avg_launch_us": per_launch_ms * 1e3, "alg_bytes_per_launch": per_launch_by,
            "alg_flops_per_launch": per_launch_fl, "intensity_flop_per_byte": per_launch_fl / per_launch_by,
            "ridge_flop_per_byte": ridge, "launches_timed": dom["launches"],
            "hbm_gbs": ach_gbs, "tflops": ach_tfs,
        }
        out["decode_profile"] = {
            "profiled_iterations": n_prof, "loop_iterations": it, "step_done": done,
            "kernel_time_ms": tot_ms, "alg_bytes": tot_by,
            "decode_hbm_gbs": tot_by / (tot_ms * 1e-3) / 1e9,
            "decode_hbm_frac": tot_by / (tot_ms * 1e-3) / 1e9 / HBM_PEAK_GBS,
            "classes": {k["name"]: {"launches": k["launches"], "ms": round(k["ms"], 3),
                                    "avg_us": round(1e3 * k["ms"] / k["launches"], 2),
                                    "GBps": round(k["bytes"] / (k["ms"] * 1e-3) / 1e9, 1) if k["ms"] else None,
                                    "TFLOPs": round(k["flops"] / (k["ms"] * 1e-3) / 1e12, 1) if k["ms"] else None}
                        for k in allc},
            "wall_s": tprof,
        }
        print(f"[bench] profiled {n_prof} of {it} loop iterations; dominant {dom['name']}: {ach_gbs:.0f} GB/s; "
              f"decode kernels {out['decode_profile']['decode_hbm_gbs']:.0f} GB/s", file=sys.stderr, flush=True)

    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(cfg, weights)
    ctx.close()
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
