"""A full allocation step on the CPU (oracle): controller + rollout generation.

A rollout (uid, j) is a pure function of the weights, the prompt, the seed,
the step index and its logical id uid * k + j, so the oracle generates each
rollout whole when the controller starts it and hands the controller only its
length and reward.  Rollouts started at the same refill are generated in
lockstep (batched GEMMs), each with its own KV cache seeded from its prompt's
prefill.

Termination of rollout (uid, j) at generated index i (length = i + 1):
token == eos_id (when eos_id >= 0), i + 1 == max_new, or i + 1 == the forced
length L[uid, j] when a forced-length table is given (then the token at that
index is replaced by eos_id when eos_id >= 0).  A forced-EOS draw (sampler)
replaces the sampled token by eos_id.  A teacher-forcing table replaces the
token actually appended (the sampler's own choice is still recorded).
"""
import numpy as np

from . import controller, grpo, reward, sampler
from .model import Decoder


class RolloutSource:
    def __init__(self, cfg, weights, pool, seed, step=None, forced_tokens=None,
                 keep_logits=None, model_free=False, gemm_acc="f32"):
        self.cfg = cfg
        self.m, self.a = cfg["model"], cfg["alloc"]
        self.pool = pool
        self.seed = seed
        self.step = pool["step"] if step is None else step
        self.forced_tokens = forced_tokens           # dict rid -> int array, or [U*k, max_new]
        self.keep_logits = keep_logits              # callable(uid, j, i) -> bool, or None
        self.model_free = model_free
        self.dec = None if model_free else Decoder(self.m, weights, gemm_acc=gemm_acc)
        self.prefix = {}
        self.results = {}
        self.logits = {}

    def prompt(self, u):
        o = self.pool["offsets"]
        return self.pool["tokens"][o[u]:o[u + 1]]

    def _forced(self, rid):
        ft = self.forced_tokens
        if ft is None:
            return None
        return ft[rid] if not isinstance(ft, dict) else ft.get(rid)

    def _prefill(self, u):
        if u not in self.prefix:
            P = len(self.prompt(u))
            cache = self.dec.new_cache(P - 1 + self.a["max_new"])
            if P > 1:
                self.dec.forward(self.prompt(u)[:P - 1], np.arange(P - 1), cache, want_logits=False)
            self.prefix[u] = (P, cache)
        return self.prefix[u]

    def outcomes(self, pairs):
        todo = [(u, j) for (u, j) in pairs if (u, j) not in self.results]
        if todo:
            self._generate(todo)
        return [(self.results[p]["length"], self.results[p]["reward"]) for p in pairs]

    def _generate(self, pairs):
        m, a = self.m, self.a
        k, eos, max_new = a["k"], m["eos_id"], a["max_new"]
        fl = self.pool.get("forced_len")
        rows = []
        for (u, j) in pairs:
            P = len(self.prompt(u))
            row = dict(u=u, j=j, rid=u * k + j, P=P, toks=[], sampled=[], ties=0,
                       done=False, Lf=int(fl[u, j]) if fl is not None else None)
            if not self.model_free:
                _, cache = self._prefill(u)
                row["cache"] = [(K.copy(), V.copy()) for (K, V) in cache]
            rows.append(row)
        for i in range(max_new):
            live = [r for r in rows if not r["done"]]
            if not live:
                break
            if not self.model_free:
                toks_in = [int(self.prompt(r["u"])[-1]) if i == 0 else r["toks"][-1] for r in live]
                pos = [r["P"] - 1 + i for r in live]
                logits = self.dec.forward_batch(toks_in, pos, [r["cache"] for r in live])
            for ri, r in enumerate(live):
                if self.model_free:
                    tok = int(self._forced(r["rid"])[i])
                    samp = tok
                else:
                    samp, sc = sampler.sample(logits[ri], a["temperature"], self.seed,
                                              self.step, r["rid"], i, a.get("top_p", 1.0))
                    if sampler.near_tie(sc):
                        r["ties"] += 1
                    if self.keep_logits is not None and self.keep_logits(r["u"], r["j"], i):
                        self.logits[(r["u"], r["j"], i)] = logits[ri].copy()
                    if eos >= 0 and sampler.forced_eos(self.seed, self.step, r["rid"], i,
                                                       a["forced_eos_u32"]):
                        samp = eos
                    ft = self._forced(r["rid"])
                    tok = int(ft[i]) if ft is not None else samp
                fin = False
                if r["Lf"] is not None and i + 1 == r["Lf"]:
                    if eos >= 0:
                        tok = eos
                    fin = True
                if eos >= 0 and tok == eos:
                    fin = True
                if i + 1 == max_new:
                    fin = True
                r["toks"].append(tok)
                r["sampled"].append(samp)
                if fin:
                    r["done"] = True
        for r in rows:
            h = reward.hash_tokens(self.seed, self.step, r["u"], r["toks"])
            self.results[(r["u"], r["j"])] = dict(
                tokens=np.array(r["toks"], dtype=np.int32), sampled=np.array(r["sampled"], dtype=np.int32),
                length=len(r["toks"]), hash=h,
                reward=reward.reward_of_hash(h, float(self.pool["p"][r["u"]])), near_ties=r["ties"])


def run_step(cfg, weights, pool, seed, forced_tokens=None, keep_logits=None, model_free=False,
             gemm_acc="f32", priors=None):
    """priors: optional per pool prompt (alpha0_u, beta0_u) (history warm start)."""
    src = RolloutSource(cfg, weights, pool, seed, forced_tokens=forced_tokens,
                        keep_logits=keep_logits, model_free=model_free, gemm_acc=gemm_acc)
    res = controller.simulate(cfg["alloc"], len(pool["p"]), src.outcomes, priors=priors,
                              draw_key=(seed, pool["step"]))
    k = cfg["alloc"]["k"]
    offs, rws = [0], []
    for u in res["committed"]:
        n = res["n_issued"][u]
        rws += [res["rollout"][(u, j)][1] for j in range(n)]
        offs.append(offs[-1] + n)
    res["grpo_offsets"] = np.array(offs, dtype=np.int32)
    res["grpo_rewards"] = np.array(rws, dtype=np.float32)
    res["advantages"] = grpo.advantages(res["grpo_rewards"], res["grpo_offsets"])
    res["rollouts_detail"] = src.results
    res["logits"] = src.logits
    res["k"] = k
    return res
