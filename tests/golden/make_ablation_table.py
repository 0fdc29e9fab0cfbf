"""Writes tests/golden/ablation_sweeps.txt from the oracle alone.

The mechanism and ablation figures of the paper (section 4.3, Fig. 3a and
3c; the appendix paragraphs on sensitivity to the threshold and probe size,
savings growing with group size, and decision quality) are reproduced here
on synthetic inputs: model-free rollouts of 4 tokens (a seeded token table)
over a 2048-prompt pool of the success-rate mixture, budget 2048, commit
floor k, the tiny workload's reward seed.  For every group size k a fixed-k
run (every drawn prompt gets all k rollouts, budget 4096) on the same table
labels each prompt with its full group: the logical rollout keys make a
prompt's first n rewards the same in both runs, so the labels are exact
counterfactuals.

Rows (all integers, compared exactly by the GPU test):
  point k n0 tau n_stop drawn rollouts committed abandoned lost decode_steps
      lost = abandoned prompts whose full group of k is mixed
  fig3a k n0 tau d_1 .. d_k
      d_n = drawn prompts whose label is settled after n observed rollouts
      (a committed prompt at its first mix in j order, an abandoned one at
      its abandonment)
  fig3c mode k c:r ...
      r = rollouts issued when the c-th effective group is committed
      (mode sara at the default point, fixed_k for the same k)

Run:  python tests/golden/make_ablation_table.py
"""
import os
import sys

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import workloads as W  # noqa: E402

OUT = os.path.join(HERE, "ablation_sweeps.txt")
POINTS = ([(8, 2, tau) for tau in (0.1, 0.3, 0.45, 0.6)] + [(8, n0, 0.45) for n0 in (1, 4)]
          + [(k, 2, 0.45) for k in (4, 16)])
DEFAULT = (8, 2, 0.45)
FIG3C_COUNTS = (8, 16, 32, 64, 96, 128)
TABLE_SEED = 5
COMMIT, ABANDON = 1, 2


def base_config():
    c = W.get_config("tiny_f32")
    c["alloc"].update(B=10 ** 6, budget_N=2048, pool_U=2048, n_slots=512, max_new=4)
    c["model"]["eos_id"] = -1
    return c


def point_config(k, n0, tau):
    c = base_config()
    c["alloc"].update(k=k, n0=n0, commit_min=k, tau_low=tau)
    return c


def label_config(k):
    fk = W.fixed_k_variant(point_config(k, 2, 0.45))
    fk["alloc"]["budget_N"] = 4096
    return fk


def token_table(cfg):
    a = cfg["alloc"]
    g = np.random.default_rng(TABLE_SEED)
    return g.integers(0, cfg["model"]["vocab"], size=(a["pool_U"] * a["k"], a["max_new"])).astype(np.int32)


def n_stop(k, n0, tau):
    return max(n0, min(k, k - int(np.floor(tau * (k + 1)))))


def summarize(k, n0, tau, run, labels=None):
    """run: dict with drawn, rollouts, committed, decode_steps, status[u]
    (2 committed, 3 abandoned), n[u], reward[u*k+j], decisions rows (t, u,
    code, n, s), assigns rows (t, slot, u, j).  labels: reward[u*k+j] of the
    fixed-k run for the same k.  Returns the golden lines of this point."""
    drawn = int(run["drawn"])
    status, n, rew = run["status"], run["n"], run["reward"]
    lines = []
    if labels is not None:
        committed = sum(1 for u in range(drawn) if status[u] == 2)
        abandoned = sum(1 for u in range(drawn) if status[u] == 3)
        lost = 0
        for u in range(drawn):
            s_full = int(sum(labels[u * k + j] for j in range(k)))
            if status[u] == 3 and 1 <= s_full <= k - 1:
                lost += 1
        lines.append(f"point {k} {n0} {tau:.2f} {n_stop(k, n0, tau)} {drawn} {int(run['rollouts'])} {committed} "
                     f"{abandoned} {lost} {int(run['decode_steps'])}")
        settled = []
        for u in range(drawn):
            if status[u] == 2:
                r = [int(rew[u * k + j]) for j in range(int(n[u]))]
                settled.append(next(i + 1 for i in range(1, len(r)) if r[i] != r[0]))
            else:
                settled.append(int(n[u]))
        d = [sum(1 for x in settled if x <= m) for m in range(1, k + 1)]
        lines.append(f"fig3a {k} {n0} {tau:.2f} " + " ".join(map(str, d)))
    return lines


def fig3c(mode, k, run):
    asg = np.asarray(run["assigns"]).reshape(-1, 4)
    dec = np.asarray(run["decisions"]).reshape(-1, 5)
    t_commit = [int(r[0]) for r in dec if int(r[2]) == COMMIT]
    starts = np.sort(asg[:, 0])
    pts = []
    for c in FIG3C_COUNTS:
        if c <= len(t_commit):
            pts.append(f"{c}:{int(np.searchsorted(starts, t_commit[c - 1], side='right'))}")
    return f"fig3c {mode} {k} " + " ".join(pts)


def oracle_run(cfg):
    from oracle import run as ORUN
    pool = W.make_pool(cfg, 0)
    res = ORUN.run_step(cfg, None, pool, W.sampling_seed(cfg), forced_tokens=token_table(cfg), model_free=True)
    k, U = cfg["alloc"]["k"], cfg["alloc"]["pool_U"]
    rew = np.zeros(U * k, np.int64)
    for (u, j), (L, r, _, _) in res["rollout"].items():
        rew[u * k + j] = r
    st = np.array(res["status"])
    return res, dict(drawn=res["drawn"], rollouts=res["rollouts"], committed=res["n_committed"],
                     decode_steps=res["decode_steps"], status=st, n=np.array(res["n_done"]), reward=rew,
                     decisions=[(t, u, d, n, s) for (t, u, d, n, s, _) in res["log_decisions"]],
                     assigns=res["log_assign"])


def oracle_lines():
    lines, labels, label_runs = [], {}, {}
    for k in sorted({p[0] for p in POINTS}):
        _, lab = oracle_run(label_config(k))
        labels[k] = lab["reward"]
        label_runs[k] = lab
    for (k, n0, tau) in POINTS:
        _, run = oracle_run(point_config(k, n0, tau))
        lines += summarize(k, n0, tau, run, labels[k])
        if (k, n0, tau) == DEFAULT:
            lines.append(fig3c("sara", k, run))
            lines.append(fig3c("fixed_k", k, label_runs[k]))
    return lines


def read_golden():
    with open(OUT) as f:
        return [l.strip() for l in f if l.strip() and not l.startswith("#")]


def main():
    lines = oracle_lines()
    with open(OUT, "w") as f:
        f.write("# written by tests/golden/make_ablation_table.py (oracle only); see its docstring\n")
        for l in lines:
            f.write(l + "\n")
    print("\n".join(lines))


if __name__ == "__main__":
    main()
