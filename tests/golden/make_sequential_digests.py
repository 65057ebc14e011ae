"""Stored oracle results for the within-block sequential competition (Supp. E,
"Within-block competition") at two full sizes:

* single_layer: 12 banks of one group, budget 4,680, banks filled by the
  empty-bank rule from block 0, then 4,680 candidates of block 1 (30%
  near-duplicates) offered one per step;
* long_rollout, layer 0: 12 banks of one group, budget 18,720, blocks 0-5 of
  4,680 candidates (block 0 fills the empty banks by the empty-bank rule, block
  1 takes about 4,600 steps into banks of 4,680 states, and from block 2 on no
  step is taken on this input: every candidate pushes some state of the group
  over its bound).

The oracle walks 4,680 steps of 12 banks in one to five minutes per block, too
long for a test that holds a GPU, so this script runs it once on the CPU and
stores the number of taken steps and, per bank, SHA-256 digests of the
candidate order, the scores, the released and admitted lists and the committed
bank (provenance, density, baseline, norms, keys, values).  Inputs are the
seeded draws of the input generator module; nothing here reads a GPU result.
Run from the repository root:

    python tests/golden/make_sequential_digests.py [single_layer] [long_rollout] [--ckpt DIR]
"""

import json
import os
import sys

import numpy as np

OUT = "sequential_single_layer.json"


def run(path: str):
    from golden.make_rollout_digests import digest
    from oracle import BankState, Params, update_layer
    from paper_2608_27922_amd import synth

    cfg = synth.WORKLOADS["single_layer"]
    H, M, N = cfg.heads, cfg.budget, cfg.n_cand
    case = synth.single_update_case(cfg)
    banks = [BankState.empty(M, cfg.d) for _ in range(H)]
    banks, _ = update_layer(banks, [case["init_K"][h].astype(np.float64) for h in range(H)],
                            [case["init_V"][h] for h in range(H)], 0, Params(sigma2_log2=cfg.sigma2_log2))
    init = [{"m": b.m, "rho": digest(b.rho, np.int64), "base": digest(b.base, np.int64),
             "prov": digest(b.prov, np.int64)} for b in banks]
    prm = Params(sigma2_log2=cfg.sigma2_log2, sequential=True)
    new, rec = update_layer(banks, [case["seg_K"][h].astype(np.float64) for h in range(H)],
                            [case["seg_V"][h] for h in range(H)], 1, prm)
    heads = []
    for h in range(H):
        hr, nb = rec.heads[h], new[h]
        heads.append({
            "m_after": nb.m, "n_evicted": int(hr.evicted.size), "n_admitted": int(hr.admitted.size),
            "order": digest(hr.pi, np.int32), "score_q": digest(hr.score_q, np.int64),
            "evicted": digest(hr.evicted, np.int32), "admitted": digest(hr.admitted, np.int32),
            "prov": digest(nb.prov, np.int64), "rho": digest(nb.rho, np.int64), "base": digest(nb.base, np.int64),
            "knorm": digest((nb.K * nb.K).sum(1), np.float32), "k": digest(nb.K, np.float32),
            "v": digest(nb.V, np.float32),
        })
    out = {"workload": "single_layer", "policy": "sequential", "steps_taken": int(rec.steps.sum()),
           "init": init, "heads": heads}
    with open(path, "w") as f:
        json.dump(out, f, indent=0)
    print(f"steps taken {out['steps_taken']} of {N}; occupancy {[b.m for b in new]}", flush=True)


ROLLOUT_OUT = "sequential_long_rollout_L0.json"
ROLLOUT_BLOCKS = 6


def seq_entry(hr, nb, m_before: int):
    from golden.make_rollout_digests import digest
    return {
        "m_before": m_before, "m_after": nb.m, "n_evicted": int(hr.evicted.size), "n_admitted": int(hr.admitted.size),
        "order": digest(hr.pi, np.int32),
        "score_q": digest(hr.score_q if hr.score_q is not None else np.zeros(hr.pi.size, np.int64), np.int64),
        "evicted": digest(hr.evicted, np.int32), "admitted": digest(hr.admitted, np.int32),
        "prov": digest(nb.prov, np.int64), "rho": digest(nb.rho, np.int64), "base": digest(nb.base, np.int64),
        "knorm": digest((nb.K * nb.K).sum(1), np.float32), "k": digest(nb.K, np.float32),
        "v": digest(nb.V, np.float32),
    }


def run_rollout(path: str, ckpt=None):
    """Layer 0 of the long rollout under the sequential policy, blocks 0..ROLLOUT_BLOCKS-1;
    with a checkpoint directory the run saves its state after every block and resumes."""
    from golden.make_rollout_digests import _load, _save
    from oracle import BankState, Params, update_layer
    from paper_2608_27922_amd import synth

    cfg = synth.WORKLOADS["long_rollout"]
    H = cfg.heads
    budgets = synth.budgets(cfg)[:H]
    streams = [synth.HeadStream(cfg, 0, h) for h in range(H)]
    banks = [BankState.empty(int(budgets[h]), cfg.d) for h in range(H)]
    prm = Params(sigma2_log2=cfg.sigma2_log2, sequential=True)
    steps = []
    cp = os.path.join(ckpt, "sequential_long_rollout_L0") if ckpt else None
    if cp:
        saved, saved_steps = _load(cp, H, BankState)
        if saved is not None:
            banks, steps = saved, saved_steps
    for t in range(len(steps), ROLLOUT_BLOCKS):
        K = [s.keys(t, cfg.n_cand).astype(np.float64) for s in streams]
        V = [s.values(t, cfg.n_cand) for s in streams]
        new, rec = update_layer(banks, K, V, t, prm)
        steps.append((int(rec.r_star), [seq_entry(rec.heads[h], new[h], banks[h].m) for h in range(H)]))
        banks = new
        if cp:
            _save(cp, banks, steps)
        print(f"long_rollout L0 block {t}: steps {rec.r_star} occupancy {[b.m for b in banks][:4]}", flush=True)
    out = {"workload": "long_rollout", "layer": 0, "policy": "sequential", "blocks": ROLLOUT_BLOCKS,
           "steps": [{"steps_taken": r, "heads": e} for r, e in steps]}
    with open(path, "w") as f:
        json.dump(out, f, indent=0)


if __name__ == "__main__":
    import argparse
    here = os.path.dirname(os.path.abspath(__file__))
    sys.path.insert(0, os.path.dirname(os.path.dirname(here)))
    sys.path.insert(0, os.path.dirname(here))
    ap = argparse.ArgumentParser()
    ap.add_argument("which", nargs="*", default=["single_layer", "long_rollout"])
    ap.add_argument("--ckpt", default=None)
    a = ap.parse_args()
    if "single_layer" in a.which:
        run(os.path.join(here, OUT))
    if "long_rollout" in a.which:
        run_rollout(os.path.join(here, ROLLOUT_OUT), a.ckpt)
