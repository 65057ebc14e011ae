"""Stored oracle results for an update sequence at the interface limits.

N = 8,191 candidates per block (DKV_MAX_CANDIDATES: the source index packs
into 13 bits of the sort key) and a budget of 32,767 states (DKV_MAX_CAPACITY:
the slot packs into 15 bits of the eviction key), two heads sharing the prefix
(group size 2), d = 128, bf16, tau = 16 (so that admissions continue on this
nearly flat synthetic geometry): blocks 0-3 fill the banks to 32,764 states
through the empty-bank rule and full admissions, and blocks 4-5 must release
about 8,190 states each by the densest fill, with slot indices up to 32,766.  The oracle needs minutes per
block at these sizes, so this script runs it once, on the CPU, and stores the
per-block scalars and SHA-256 digests that the GPU test compares against
(the same digests as the full-size rollout runs).

Inputs are the seeded HeadStream draws of the input generator module; nothing
here reads a GPU result.  Run from the repository root:

    python tests/golden/make_limit_digests.py
"""

import json
import os
import sys

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
if __name__ == "__main__":
    sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))
    sys.path.insert(0, HERE)

try:  # imported by the tests as golden.make_limit_digests
    from .make_rollout_digests import head_entry
except ImportError:  # run as a script
    from make_rollout_digests import head_entry  # noqa: E402

BLOCKS = 6
DUP_EVERY = 2  # near-duplicate blocks at t = 2, 4
TAU_NUM = 16   # tau = 16 / 2^0


def limits_config():
    from paper_2608_27922_amd import synth
    return synth.Config(seed_id=99, name="limits", layers=1, heads=2, d=128, dtype="bf16", n_cand=8191,
                        n_query=64, n_window=64, budget=32767, clusters=64, blocks=BLOCKS, group_size=2,
                        sigma2_log2=6, drift=0.05)


def block_inputs(cfg, streams, t, bank_keys):
    """Keys and values of block t (near-duplicates of the current bank keys on the
    near-duplicate blocks)."""
    K = np.stack([s.keys(t, cfg.n_cand) for s in streams])
    V = np.stack([s.values(t, cfg.n_cand) for s in streams])
    if t > 0 and t % DUP_EVERY == 0:
        for h, s in enumerate(streams):
            if len(bank_keys[h]):
                K[h] = s.near_duplicates(K[h], np.asarray(bank_keys[h], np.float32), t)
    return K, V


def run(path):
    from oracle import BankState, Params, update_layer
    from paper_2608_27922_amd import synth

    cfg = limits_config()
    prm = Params(sigma2_log2=cfg.sigma2_log2, tau_num=TAU_NUM)
    streams = [synth.HeadStream(cfg, 0, h) for h in range(cfg.heads)]
    banks = [BankState.empty(cfg.budget, cfg.d) for _ in range(cfg.heads)]
    out = {"config": "limits", "blocks": BLOCKS, "tau_num": TAU_NUM, "steps": []}
    for t in range(BLOCKS):
        K, V = block_inputs(cfg, streams, t, [b.K for b in banks])
        nb, rec = update_layer(banks, [K[h].astype(np.float64) for h in range(cfg.heads)],
                               [V[h] for h in range(cfg.heads)], t, prm)
        step = {"r_star": [rec.r_star], "heads": [head_entry(rec.heads[h], nb[h], banks[h].m, cfg.n_cand)
                                                   for h in range(cfg.heads)]}
        banks = nb
        out["steps"].append(step)
        print(f"limits block {t}: r* {rec.r_star} occupancy {[b.m for b in banks]} "
              f"evicted {[int(h.evicted.size) for h in rec.heads]}", flush=True)
    with open(path, "w") as f:
        json.dump(out, f, indent=0)


if __name__ == "__main__":
    run(os.path.join(HERE, "limits.json"))
