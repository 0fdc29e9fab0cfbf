"""The oracle's full allocation step on the tiny fp32 workload."""
import numpy as np

import workloads as W
from oracle import controller as C
from oracle import run


def test_tiny_step_end_to_end():
    cfg = W.get_config("tiny_f32")
    w, pool, seed = W.make_weights(cfg), W.make_pool(cfg, 0), W.sampling_seed(cfg)
    res = run.run_step(cfg, w, pool, seed)
    a = cfg["alloc"]
    assert res["rollouts"] <= a["budget_N"]
    assert res["tokens"] == 64 * res["rollouts"]          # no EOS in this workload
    assert res["decode_steps"] % 64 == 0
    assert len(res["grpo_offsets"]) == res["n_committed"] + 1
    # teacher forcing with the oracle's own tokens reproduces everything
    ft = {u * 8 + j: d["tokens"] for (u, j), d in res["rollouts_detail"].items()}
    res2 = run.run_step(cfg, w, pool, seed, forced_tokens=ft)
    assert res2["log_decisions"] == res["log_decisions"]
    assert res2["log_assign"] == res["log_assign"]
    for key, d in res["rollouts_detail"].items():
        assert np.array_equal(res2["rollouts_detail"][key]["sampled"], d["tokens"])
    # model-free mode with the same token table gives the same outcomes
    ftab = np.zeros((64 * 8, 64), dtype=np.int32)
    for rid, t in ft.items():
        ftab[rid] = t
    res3 = run.run_step(cfg, w, pool, seed, forced_tokens=ftab, model_free=True)
    assert res3["log_decisions"] == res["log_decisions"]
