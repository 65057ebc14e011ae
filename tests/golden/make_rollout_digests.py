"""Stored oracle results for the full-size 30-layer x 12-head rollout workloads.

The oracle needs one to two minutes per block for a whole layer at budgets of
9,360 and 18,720 tokens, far too long for a test that holds a GPU.  This script
runs it once, on the CPU, over sampled layers of each workload at the stated
length (every block of the run) and stores, per block and per head, the scalars
of the update (r*, occupancy, evictions, admissions) and SHA-256 digests of
every array the GPU must reproduce bit for bit (candidate order, scores, first
crossings, projected densities, eviction and admission lists, and the committed
bank: provenance, density, baseline, norms, keys, values), plus the fp64
attention of sampled query rows after the last block.

Groups of heads that share no prefix (the head-wise workload runs every head as
its own group) are independent, so they run in parallel worker processes.

Inputs are the seeded HeadStream draws of the input generator module; nothing
here reads a GPU result.  Run from the repository root:

    python tests/golden/make_rollout_digests.py [--jobs J] [--threads T] [--ckpt DIR] [workload[:layer] ...]

Output: tests/golden/rollout_<workload>_L<layer>.json and
tests/golden/rollout_<workload>_L<layer>_attention.npy.
"""

import hashlib
from typing import Dict

import numpy as np

# name -> (blocks, sampled layers, heads whose attention rows are stored)
RUNS: Dict[str, tuple] = {
    "rollout": (20, (0, 29), (0, 5, 11)),
    "long_rollout": (80, (0,), (0, 5, 11)),
    "headwise_budgets": (160, (17,), (0, 1, 6, 7)),
}
ATT_ROWS = 32


def cases():
    """(workload, layer) pairs with stored digests."""
    return [(name, layer) for name, (_, layers, _) in RUNS.items() for layer in layers]


def digest(a, dtype) -> str:
    """First 32 hex digits of SHA-256 over the little-endian bytes of `a` as `dtype`."""
    b = np.ascontiguousarray(np.asarray(a), dtype=np.dtype(dtype).newbyteorder("<")).tobytes()
    return hashlib.sha256(b).hexdigest()[:32]


def attention_rows(n_query: int) -> np.ndarray:
    return np.linspace(0, n_query - 1, ATT_ROWS).round().astype(np.int64)


def layer_block(cfg, streams, t: int):
    """Keys and values of block t for every head of the sampled layer."""
    K = np.stack([s.keys(t, cfg.n_cand) for s in streams])
    V = np.stack([s.values(t, cfg.n_cand) for s in streams])
    return K, V


def head_entry(hr, nb, m_before: int, n: int):
    """Scalars and digests of one head's update (oracle HeadRecord + new BankState)."""
    sq = hr.score_q if hr.score_q is not None else np.zeros(n, np.int64)
    return {
        "m_before": m_before, "m_after": nb.m, "n_evicted": int(hr.evicted.size),
        "n_admitted": int(hr.admitted.size),
        "order": digest(hr.pi, np.int32), "score_q": digest(sq, np.int64),
        "first_cross": digest(hr.first_cross, np.int32), "rho_tilde": digest(hr.rho_tilde, np.int64),
        "evicted": digest(hr.evicted, np.int32), "admitted": digest(hr.admitted, np.int32),
        "prov": digest(nb.prov, np.int64), "rho": digest(nb.rho, np.int64), "base": digest(nb.base, np.int64),
        "knorm": digest((nb.K * nb.K).sum(1), np.float32), "k": digest(nb.K, np.float32),
        "v": digest(nb.V, np.float32),
    }


def _save(path, banks, steps):
    """Checkpoint of a group's run after a block: the oracle banks and the entries so far."""
    import json
    import os
    arrs = {}
    for j, b in enumerate(banks):
        arrs.update({f"{j}_K": b.K, f"{j}_V": b.V, f"{j}_rho": b.rho, f"{j}_base": b.base, f"{j}_prov": b.prov,
                     f"{j}_budget": np.array(b.budget)})
    np.savez(path + ".tmp.npz", **arrs)
    with open(path + ".tmp.json", "w") as f:
        json.dump(steps, f)
    os.replace(path + ".tmp.npz", path + ".npz")
    os.replace(path + ".tmp.json", path + ".json")


def _load(path, n, BankState):
    import json
    import os
    if not (os.path.exists(path + ".npz") and os.path.exists(path + ".json")):
        return None, []
    z = np.load(path + ".npz")
    banks = [BankState(int(z[f"{j}_budget"]), z[f"{j}_K"], z[f"{j}_V"], z[f"{j}_rho"], z[f"{j}_base"],
                       z[f"{j}_prov"]) for j in range(n)]
    with open(path + ".json") as f:
        return banks, [tuple(s) for s in json.load(f)]


def run_group(args):
    """The whole run of one group of heads of the sampled layer: per block the
    group's r* and head entries, then the fp64 attention rows of its heads that
    are in the stored set.  With a checkpoint directory the run saves its state
    after every block and resumes from the last saved block."""
    from oracle import BankState, Params, attention, update_layer
    from paper_2608_27922_amd import synth

    name, layer, heads, ckpt = args
    blocks, _, att_heads = RUNS[name]
    cfg = synth.WORKLOADS[name]
    H = cfg.heads
    budgets = synth.budgets(cfg)[layer * H:(layer + 1) * H]
    prm = Params(sigma2_log2=cfg.sigma2_log2)
    streams = [synth.HeadStream(cfg, layer, h) for h in heads]
    banks = [BankState.empty(int(budgets[h]), cfg.d) for h in heads]
    steps = []
    path = f"{ckpt}/{name}_L{layer}_h{heads[0]}-{heads[-1]}" if ckpt else None
    if path:
        saved, saved_steps = _load(path, len(heads), BankState)
        if saved is not None:
            banks, steps = saved, saved_steps
    for t in range(len(steps), blocks):
        K, V = layer_block(cfg, streams, t)
        nb, rec = update_layer(banks, [K[j].astype(np.float64) for j in range(len(heads))],
                               [V[j] for j in range(len(heads))], t, prm)
        steps.append((rec.r_star, [head_entry(rec.heads[j], nb[j], banks[j].m, cfg.n_cand)
                                   for j in range(len(heads))]))
        banks = nb
        if path:
            _save(path, banks, steps)
        print(f"{name} L{layer} heads {heads[0]}-{heads[-1]} block {t}: r* {rec.r_star} "
              f"occupancy {[b.m for b in banks][:4]}", flush=True)
    rows = attention_rows(cfg.n_query)
    att = {}
    for j, h in enumerate(heads):
        if h in att_heads:
            s = streams[j]
            att[h] = attention(s.queries(blocks)[rows], banks[j].K, banks[j].V, s.keys(blocks, cfg.n_window),
                               s.values(blocks, cfg.n_window), 1.0 / np.sqrt(cfg.d))
    return heads, steps, att


def run(name: str, layer: int, path_prefix: str, jobs: int = 1, ckpt=None):
    import json
    from concurrent.futures import ProcessPoolExecutor

    from paper_2608_27922_amd import synth

    blocks, _, att_heads = RUNS[name]
    cfg = synth.WORKLOADS[name]
    H, gs = cfg.heads, cfg.group_size
    budgets = synth.budgets(cfg)[layer * H:(layer + 1) * H]
    groups = [(name, layer, tuple(range(g0, g0 + gs)), ckpt) for g0 in range(0, H, gs)]
    if jobs > 1 and len(groups) > 1:
        with ProcessPoolExecutor(max_workers=min(jobs, len(groups))) as ex:
            results = list(ex.map(run_group, groups))
    else:
        results = [run_group(g) for g in groups]
    out = {"workload": name, "layer": layer, "blocks": blocks, "budgets": [int(b) for b in budgets],
           "group_size": gs, "steps": []}
    for t in range(blocks):
        step = {"r_star": [], "heads": []}
        for heads, steps, _ in results:
            r_star, entries = steps[t]
            step["r_star"].append(r_star)
            step["heads"].extend(entries)
        out["steps"].append(step)
    att = {}
    for _, _, a in results:
        att.update(a)
    out["attention_heads"] = list(att_heads)
    with open(f"{path_prefix}{name}_L{layer}.json", "w") as f:
        json.dump(out, f, indent=0)
    np.save(f"{path_prefix}{name}_L{layer}_attention.npy", np.stack([att[h] for h in att_heads]))


if __name__ == "__main__":
    import argparse
    import os
    import sys
    here = os.path.dirname(os.path.abspath(__file__))
    sys.path.insert(0, os.path.dirname(os.path.dirname(here)))
    ap = argparse.ArgumentParser()
    ap.add_argument("--jobs", type=int, default=1, help="worker processes for independent head groups")
    ap.add_argument("--threads", type=int, default=1, help="threads for the per-head steps of a layer update")
    ap.add_argument("--ckpt", default=None, help="directory for per-block checkpoints (resume after a stop)")
    ap.add_argument("which", nargs="*", help="workload or workload:layer (default: every stored case)")
    a = ap.parse_args()
    if a.threads > 1:
        from concurrent.futures import ThreadPoolExecutor

        import oracle.densitykv_ref as ref
        ref.HEAD_MAP = ThreadPoolExecutor(a.threads).map
    todo = []
    for w in a.which or [n for n in RUNS]:
        nm, _, ly = w.partition(":")
        todo += [(nm, int(ly))] if ly else [(nm, L) for L in RUNS[nm][1]]
    for nm, ly in todo:
        run(nm, ly, os.path.join(here, "rollout_"), a.jobs, a.ckpt)
