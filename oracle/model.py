"""Pre-norm GQA decoder used to generate rollouts (oracle).

The paper generates rollouts with R1-Distill-Qwen-1.5B / Qwen2.5-3B in bf16;
those weights are unavailable, so random-init decoders of the same shapes
stand in.  Architecture (reading of "Qwen2.5-shaped"): token embedding;
per layer RMSNorm -> attention with grouped KV heads (query head h reads KV
head h // (Hq / Hkv)), rotate-half RoPE, scale 1/sqrt(hd), no biases ->
residual -> RMSNorm -> SwiGLU W_d(silu(W_g x) * W_u x) -> residual; final
RMSNorm and an untied LM head.

Precision.  fp32 models: every operation in fp64 here.  bf16 models: values
are rounded to bf16 (round-to-nearest-even of the fp32 value) at exactly the
points where a bf16 engine stores them - the inputs of every weight GEMM
(normed activations, attention output, SwiGLU product), the rotated query and
key and the value written to the KV cache; residual stream, norms, softmax
and accumulation stay wide.  GEMMs with bf16 operands accumulate in fp32
(numpy sgemm) as a bf16 engine does; all other arithmetic is fp64.

Clock: prefill computes K/V for prompt positions 0..P-2; generated token i
takes prompt[P-1] (i = 0) or token i-1 as input at position P-1+i.

The paper prints no logits to compare with; the decoder is pinned instead
by tests against an independent torch-CPU functional forward (library
attention and activations), against a full causal recompute of the decode
logits, and by the bf16 rounding against torch's conversion.
"""
import numpy as np


def bf16_round(x: np.ndarray) -> np.ndarray:
    """fp32 value of x rounded to bf16 (RNE), returned as float64."""
    f = np.ascontiguousarray(np.asarray(x, dtype=np.float32))
    b = f.view(np.uint32)
    r = ((b + np.uint32(0x7FFF) + ((b >> np.uint32(16)) & np.uint32(1))) & np.uint32(0xFFFF0000))
    return r.view(np.float32).astype(np.float64)


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


class Decoder:
    def __init__(self, model: dict, weights: dict, gemm_acc: str = "f32"):
        """gemm_acc: accumulation of bf16 GEMMs, "f32" (a bf16 engine's) or
        "f64" (used only to measure the model's sensitivity to rounding order)."""
        self.m = model
        self.bf16 = model["dtype"] == "bf16"
        self.gemm_acc = gemm_acc
        self.L = model["n_layers"]
        self.d = model["d_model"]
        self.hq, self.hkv, self.hd = model["n_heads"], model["n_kv_heads"], model["head_dim"]
        self.V = model["vocab"]
        self.eps = model["rms_eps"]
        self._raw = weights
        self._cache = {}
        half = self.hd // 2
        self.inv_freq = model["rope_theta"] ** (-(2.0 * np.arange(half, dtype=np.float64)) / self.hd)

    # -- weights ----------------------------------------------------------
    def w(self, name):
        if name not in self._cache:
            a = self._raw[name]
            if self.bf16 and a.dtype == np.uint16:
                a = bf16_bits_to_f32(a)
            # bf16 models: keep fp32 copies (exact) for sgemm; fp32 models: fp64
            self._cache[name] = np.ascontiguousarray(a, dtype=np.float32 if self.bf16 else np.float64)
        return self._cache[name]

    def rnd(self, x):
        return bf16_round(x) if self.bf16 else x

    def mm(self, x, name):
        """x @ W^T with W stored [out, in]."""
        W = self.w(name)
        if self.bf16 and self.gemm_acc == "f32":
            return (np.asarray(x, dtype=np.float32) @ W.T).astype(np.float64)
        if self.bf16:
            return np.asarray(x, dtype=np.float64) @ W.astype(np.float64).T
        return x @ W.T

    def rmsnorm(self, h, name):
        g = self.w(name).astype(np.float64)
        return h / np.sqrt(np.mean(h * h, axis=-1, keepdims=True) + self.eps) * g

    def rope(self, x, pos):
        """x: (T, H, hd); pos: (T,). Rotate-half convention."""
        ang = np.asarray(pos, dtype=np.float64)[:, None] * self.inv_freq[None, :]
        c, s = np.cos(ang)[:, None, :], np.sin(ang)[:, None, :]
        half = self.hd // 2
        x1, x2 = x[..., :half], x[..., half:]
        return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)

    @staticmethod
    def silu(x):
        return x / (1.0 + np.exp(-x))

    # -- attention over a cache ------------------------------------------
    def _attend(self, q, K, V, n_ctx):
        """q: (Hq, hd) one query; K, V: (Hkv, T, hd); attends to [0, n_ctx)."""
        grp = self.hq // self.hkv
        o = np.empty((self.hq, self.hd))
        scale = 1.0 / np.sqrt(self.hd)
        for h in range(self.hq):
            g = h // grp
            sc = (K[g, :n_ctx] @ q[h]) * scale
            sc = sc - sc.max()
            p = np.exp(sc)
            p /= p.sum()
            o[h] = p @ V[g, :n_ctx]
        return o

    def _attend_causal(self, q, K, V, positions):
        """Causal scaled dot-product attention of T consecutive queries:
        q: (T, Hq, hd) at `positions`; query t attends to cache positions
        [0, positions[t]], i.e. softmax(q K^T / sqrt(hd) + causal mask) V per
        head, with masked scores set to -inf (weight exactly 0)."""
        T = len(positions)
        grp = self.hq // self.hkv
        n = int(positions[-1]) + 1
        scale = 1.0 / np.sqrt(self.hd)
        masked = np.arange(n)[None, :] > np.asarray(positions)[:, None]
        o = np.empty((T, self.hq, self.hd))
        for h in range(self.hq):
            g = h // grp
            sc = (q[:, h, :] @ K[g, :n].T) * scale
            sc[masked] = -np.inf
            sc = sc - sc.max(axis=1, keepdims=True)
            p = np.exp(sc)
            p /= p.sum(axis=1, keepdims=True)
            o[:, h] = p @ V[g, :n]
        return o

    def new_cache(self, T_max):
        return [(np.zeros((self.hkv, T_max, self.hd)), np.zeros((self.hkv, T_max, self.hd)))
                for _ in range(self.L)]

    # -- forward over a set of new positions of ONE sequence --------------
    def forward(self, tokens, positions, cache, want_logits=True, logit_rows=None):
        """Append tokens at `positions` (consecutive, ascending) to `cache`, causal.
        logit_rows: optional indices of the rows whose logits are returned."""
        tokens = np.asarray(tokens, dtype=np.int64)
        positions = np.asarray(positions, dtype=np.int64)
        T = len(tokens)
        emb = self.w("embed")
        h = emb[tokens].astype(np.float64)
        for l in range(self.L):
            x = self.rnd(self.rmsnorm(h, f"l{l}.attn_norm"))
            q = self.mm(x, f"l{l}.wq").reshape(T, self.hq, self.hd)
            k = self.mm(x, f"l{l}.wk").reshape(T, self.hkv, self.hd)
            v = self.mm(x, f"l{l}.wv").reshape(T, self.hkv, self.hd)
            q = self.rnd(self.rope(q, positions))
            k = self.rnd(self.rope(k, positions))
            v = self.rnd(v)
            K, Vc = cache[l]
            K[:, positions, :] = k.transpose(1, 0, 2)
            Vc[:, positions, :] = v.transpose(1, 0, 2)
            o = self._attend_causal(q, K, Vc, positions)
            o = self.rnd(o.reshape(T, self.hq * self.hd))
            h = h + self.mm(o, f"l{l}.wo")
            x = self.rnd(self.rmsnorm(h, f"l{l}.ffn_norm"))
            a = self.rnd(self.silu(self.mm(x, f"l{l}.wg")) * self.mm(x, f"l{l}.wu"))
            h = h + self.mm(a, f"l{l}.wd")
        if not want_logits:
            return None
        if logit_rows is not None:
            h = h[np.asarray(logit_rows)]
        x = self.rnd(self.rmsnorm(h, "final_norm"))
        return self.mm(x, "lm_head").astype(np.float32)

    def forward_batch(self, tokens, positions, caches):
        """One decode position for several independent sequences (lockstep).

        Row r appends tokens[r] at positions[r] to caches[r]; returns fp32
        logits (R, V).  Same arithmetic as `forward`, batched for the GEMMs."""
        tokens = np.asarray(tokens, dtype=np.int64)
        positions = np.asarray(positions, dtype=np.int64)
        R = len(tokens)
        h = self.w("embed")[tokens].astype(np.float64)
        for l in range(self.L):
            x = self.rnd(self.rmsnorm(h, f"l{l}.attn_norm"))
            q = self.mm(x, f"l{l}.wq").reshape(R, self.hq, self.hd)
            k = self.mm(x, f"l{l}.wk").reshape(R, self.hkv, self.hd)
            v = self.mm(x, f"l{l}.wv").reshape(R, self.hkv, self.hd)
            q = self.rnd(self.rope(q, positions))
            k = self.rnd(self.rope(k, positions))
            v = self.rnd(v)
            o = np.empty((R, self.hq, self.hd))
            for r in range(R):
                K, Vc = caches[r][l]
                K[:, positions[r], :] = k[r]
                Vc[:, positions[r], :] = v[r]
                o[r] = self._attend(q[r], K, Vc, positions[r] + 1)
            o = self.rnd(o.reshape(R, self.hq * self.hd))
            h = h + self.mm(o, f"l{l}.wo")
            x = self.rnd(self.rmsnorm(h, f"l{l}.ffn_norm"))
            a = self.rnd(self.silu(self.mm(x, f"l{l}.wg")) * self.mm(x, f"l{l}.wu"))
            h = h + self.mm(a, f"l{l}.wd")
        x = self.rnd(self.rmsnorm(h, "final_norm"))
        return self.mm(x, "lm_head").astype(np.float32)
