"""Stored oracle results for the within-block sequential competition at the
single_layer size: 12 banks of one group, budget 4,680, banks filled by the
empty-bank rule from block 0, then 4,680 candidates of block 1 (30%
near-duplicates) offered one per step (Supp. E, "Within-block competition").

The oracle walks the 4,680 steps of 12 banks in about a minute, too long for a
test that holds a GPU, so this script runs it once on the CPU and stores the
number of taken steps and, per bank, SHA-256 digests of the candidate order,
the scores, the released and admitted lists and the committed bank (provenance,
density, baseline, norms, keys, values).  Inputs are the seeded draws of the
input generator module (the same case the benchmark times); nothing here reads
a GPU result.  Run from the repository root:

    python tests/golden/make_sequential_digests.py
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


if __name__ == "__main__":
    here = os.path.dirname(os.path.abspath(__file__))
    sys.path.insert(0, os.path.dirname(os.path.dirname(here)))
    sys.path.insert(0, os.path.dirname(here))
    run(os.path.join(here, OUT))
