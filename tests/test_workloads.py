import numpy as np

import workloads as W


def test_configs_match_stated_shapes():
    c = W.get_config("qwen1p5b_shape")["model"]
    assert (c["n_layers"], c["d_model"], c["n_heads"], c["n_kv_heads"], c["head_dim"], c["d_ffn"], c["vocab"]) == (
        28, 1536, 12, 2, 128, 8960, 151936)
    c = W.get_config("qwen3b_shape")["model"]
    assert (c["n_layers"], c["d_model"], c["n_heads"], c["n_kv_heads"], c["d_ffn"]) == (36, 2048, 16, 2, 11008)
    a = W.get_config("pool_3b")["alloc"]
    assert (a["pool_U"], a["B"], a["budget_N"], a["n_slots"]) == (192, 64, 3072, 512)
    assert W.get_config("long_ragged_1p5b")["alloc"]["n_slots"] == 256
    # weights streamed per decode step (everything but the gathered embedding) -> 3.087 GB bf16
    n = sum(int(np.prod(s)) for nm, s in W.weight_specs(W.get_config("qwen1p5b_shape")["model"])
            if nm != "embed")
    assert abs(2 * n / 1e9 - 3.087) < 0.01


def test_pool_is_deterministic_and_in_range():
    cfg = W.get_config("qwen1p5b_shape")
    a, b = W.make_pool(cfg, 0), W.make_pool(cfg, 0)
    assert np.array_equal(a["tokens"], b["tokens"]) and np.array_equal(a["p"], b["p"])
    L = np.diff(a["offsets"])
    assert L.min() >= 128 and L.max() <= 512 and len(L) == 256
    assert a["tokens"].max() < 151935 and a["tokens"].min() >= 0
    assert not np.array_equal(W.make_pool(cfg, 1)["p"], a["p"])


def test_drift_and_forced_lengths():
    cfg = W.get_config("long_ragged_1p5b")
    assert W.mixture_weights(cfg, 0) == (0.40, 0.30, 0.30)
    wh, we, wm = W.mixture_weights(cfg, 299)
    assert abs(wh - 0.20) < 1e-12 and abs(we - 0.50) < 1e-12
    pool = W.make_pool(cfg, 0)
    fl = pool["forced_len"]
    assert fl.shape == (256, 8) and fl.min() >= 1 and fl.max() <= 4096


def test_weights_deterministic_small():
    cfg = W.get_config("tiny_f32")
    w1, w2 = W.make_weights(cfg), W.make_weights(cfg)
    for k in w1:
        assert np.array_equal(w1[k], w2[k])
    assert abs(w1["lm_head"].std() - 0.02) < 1e-3
