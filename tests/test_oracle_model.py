"""Pins of the oracle decoder against an independent torch-CPU functional
forward (full causal sequence, library attention / norm / activation), the
decode-with-cache path against full recompute, and bf16 rounding against
torch's conversion.  The paper prints no logits: parity of the decoder
itself is unpinned by the paper and rests on these checks."""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

import workloads as W
from oracle.model import Decoder, bf16_round


def small_cfg(dtype):
    cfg = W.get_config("tiny_f32")
    cfg["model"].update(n_layers=2, d_model=128, n_heads=4, n_kv_heads=2, head_dim=32,
                        d_ffn=256, vocab=300, dtype=dtype, rope_theta=1.0e4)
    return cfg


def torch_reference(model, weights, tokens):
    """Full causal forward in torch fp64 (bf16 models: rounding at the same
    storage points, GEMMs on bf16 values accumulated in fp32)."""
    bf = model["dtype"] == "bf16"

    def wt(name):
        a = weights[name]
        if bf:
            a = (torch.from_numpy(a.astype(np.int32)) << 16).to(torch.int32).view(torch.float32)
            return a.to(torch.float64)
        return torch.from_numpy(np.asarray(a, dtype=np.float64))

    rnd = (lambda t: t.to(torch.float32).to(torch.bfloat16).to(torch.float64)) if bf else (lambda t: t)
    mm = (lambda x, w: (x.float() @ w.float().T).double()) if bf else (lambda x, w: x @ w.T)
    T = len(tokens)
    d, hq, hkv, hd = model["d_model"], model["n_heads"], model["n_kv_heads"], model["head_dim"]
    pos = torch.arange(T, dtype=torch.float64)
    inv = 1.0 / (model["rope_theta"] ** (torch.arange(0, hd, 2, dtype=torch.float64) / hd))
    rot = torch.polar(torch.ones(T, hd // 2, dtype=torch.float64), pos[:, None] * inv[None, :])

    def rope(x):  # x: (T, H, hd); pairs (i, i + hd/2) as complex numbers
        z = torch.complex(x[..., : hd // 2], x[..., hd // 2:]) * rot[:, None, :]
        return torch.cat([z.real, z.imag], dim=-1)

    h = wt("embed")[torch.as_tensor(tokens)]
    for l in range(model["n_layers"]):
        x = rnd(F.rms_norm(h, (d,), wt(f"l{l}.attn_norm"), model["rms_eps"]))
        q = rnd(rope(mm(x, wt(f"l{l}.wq")).view(T, hq, hd)))
        k = rnd(rope(mm(x, wt(f"l{l}.wk")).view(T, hkv, hd)))
        v = rnd(mm(x, wt(f"l{l}.wv")).view(T, hkv, hd))
        o = F.scaled_dot_product_attention(q.transpose(0, 1)[None], k.transpose(0, 1)[None],
                                           v.transpose(0, 1)[None], is_causal=True, enable_gqa=True)
        o = rnd(o[0].transpose(0, 1).reshape(T, hq * hd))
        h = h + mm(o, wt(f"l{l}.wo"))
        x = rnd(F.rms_norm(h, (d,), wt(f"l{l}.ffn_norm"), model["rms_eps"]))
        a = rnd(F.silu(mm(x, wt(f"l{l}.wg"))) * mm(x, wt(f"l{l}.wu")))
        h = h + mm(a, wt(f"l{l}.wd"))
    x = rnd(F.rms_norm(h, (d,), wt("final_norm"), model["rms_eps"]))
    return mm(x, wt("lm_head")).numpy()


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_decode_matches_torch_full_forward(dtype):
    cfg = small_cfg(dtype)
    w = W.make_weights(cfg)
    dec = Decoder(cfg["model"], w)
    g = np.random.default_rng(0)
    seq = g.integers(0, 299, size=40)
    P = 17
    ref = torch_reference(cfg["model"], w, seq)
    # oracle: prefill P-1 tokens, then one position at a time with the KV cache
    cache = dec.new_cache(len(seq))
    dec.forward(seq[:P - 1], np.arange(P - 1), cache, want_logits=False)
    rows = []
    for t in range(P - 1, len(seq)):
        rows.append(dec.forward_batch([seq[t]], [t], [cache])[0])
    got = np.stack(rows).astype(np.float64)
    want = ref[P - 1:]
    rms = np.sqrt((want ** 2).mean(axis=1))
    err = np.abs(got - want).max(axis=1)
    tol = 1e-6 if dtype == "f32" else 1e-2   # oracle logits are returned as fp32
    assert np.all(err <= tol * np.maximum(rms, 1e-30)), err / rms
    # full-sequence oracle forward equals its own cached decode
    cache2 = dec.new_cache(len(seq))
    full = dec.forward(seq, np.arange(len(seq)), cache2)
    assert np.abs(full[P - 1:] - got).max() <= (1e-6 if dtype == "f32" else 1e-2 * rms.max())


def test_batched_lockstep_equals_single_rows():
    cfg = small_cfg("f32")
    w = W.make_weights(cfg)
    dec = Decoder(cfg["model"], w)
    g = np.random.default_rng(1)
    seqs = [g.integers(0, 299, size=n) for n in (9, 14, 21)]
    caches = []
    for s in seqs:
        c = dec.new_cache(40)
        dec.forward(s[:-1], np.arange(len(s) - 1), c, want_logits=False)
        caches.append(c)
    batched = dec.forward_batch([s[-1] for s in seqs], [len(s) - 1 for s in seqs], caches)
    for s, b in zip(seqs, batched):
        c = dec.new_cache(40)
        single = dec.forward(s, np.arange(len(s)), c)[-1]
        assert np.abs(single - b).max() < 1e-5


def test_bf16_rounding_matches_torch():
    g = np.random.default_rng(2)
    x = np.concatenate([g.standard_normal(100000) * 10.0 ** g.integers(-8, 8, 100000),
                        [0.0, -0.0, 1.0, 1.00390625, 1.01171875, 3.0e38, -1.5e-39]])
    want = torch.from_numpy(x).to(torch.float32).to(torch.bfloat16).to(torch.float64).numpy()
    assert np.array_equal(bf16_round(x), want)
    bits = W.f32_to_bf16_bits(x.astype(np.float32))
    tb = torch.from_numpy(x.astype(np.float32)).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(bits, tb)
