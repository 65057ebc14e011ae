"""Pins of the oracle's per-state and per-step records, and their sensitivity (CPU only).

The GPU parity tests compare the kernels' first crossings, per-step violator
counts and released-slot lists with the oracle's.  These records feed no later
decision of the oracle itself, so the decision pins alone would not catch a
mistake in them.  Here they are checked against the exact-rational brute force
(tests/exact_rational.py), which rebuilds every hypothetical bank from its
definition:

* first crossing of a historical state: the smallest tested prefix length r
  with g_i(r) >= tau (Eqs. 8-9), R + 1 when it never violates; and the counts
  satisfy c_r = #{first crossing <= r};
* within-block sequential competition (Supp. E): the violator count of every
  head at every step, rejected steps included, and the pre-block slots whose
  occupant was released during the block.

``test_planted_mistakes_fail`` then plants plausible mistakes in a copy of the
oracle's source (sentinel R instead of R + 1, a crossing one prefix late, a
released list that also counts states of the current block, per-step counts
taken only when the step is feasible) and checks that the matching pin fails.
"""

import importlib.util
import os
import sys
from fractions import Fraction as F

import numpy as np
import pytest

import exact_rational as xr
import oracle.densitykv_ref as ref_module

ORACLE_SRC = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "oracle",
                          "densitykv_ref.py")


def _exact_bank(mod, bank):
    return [{"key": tuple(F(float(v)) for v in bank.K[i]), "b": F(int(bank.base[i]), mod.Q23),
             "prov": int(bank.prov[i])} for i in range(bank.m)]


def first_cross_pin(mod):
    """Random three-head rollouts (shared prefix, empty start, evictions): every
    head's first crossings equal the brute force's first violating prefix length,
    and c_r = #{first crossing <= r}.  The rollouts must contain states that never
    violate (sentinel R + 1) and states that cross at some 0 < r <= R."""
    d, H, M = 2, 3, 7
    prm = mod.Params(sigma2_log2=0, p=2)
    never = crossing = 0
    for seed in range(5):
        rng = np.random.default_rng(500 + seed)
        heads = [mod.BankState.empty(M, d) for _ in range(H)]
        for blk in range(1, 7):
            N = int(rng.integers(2, 6))
            Ks = [np.rint(rng.standard_normal((N, d)) * 4) / 2 for _ in range(H)]
            new, rec = mod.update_layer(heads, Ks, [k.astype(np.float32) for k in Ks], blk, prm)
            for h in range(H):
                if heads[h].m == 0:
                    continue
                _, info = xr.update(_exact_bank(mod, heads[h]), [tuple(F(float(v)) for v in row) for row in Ks[h]],
                                    M, sigma2=1, p=2, block_id=blk, r_star=rec.r_star)
                fc = rec.heads[h].first_cross
                assert fc.tolist() == info["first_violation"], f"seed {seed} block {blk} head {h}: first crossing"
                assert [int(np.count_nonzero(fc <= r)) for r in range(rec.R + 1)] == rec.heads[h].c.tolist()
                never += int(np.count_nonzero(fc == rec.R + 1))
                crossing += int(np.count_nonzero((fc > 0) & (fc <= rec.R)))
            heads = new
    assert never > 0 and crossing > 0


def sequential_record_pin(mod):
    """Random three-head rollouts of the within-block sequential competition
    (tau = 3, so that steps both release violators and are rejected): per-step
    violator counts of every head that held states at the start of the block,
    and its released pre-block slots, equal the brute force's."""
    d, H, M = 2, 3, 6
    prm = mod.Params(sigma2_log2=0, p=2, tau_num=3, sequential=True)
    rejected = released = viol_steps = 0
    for seed in range(4):
        rng = np.random.default_rng(300 + seed)
        heads = [mod.BankState.empty(M, d) for _ in range(H)]
        for blk in range(1, 8):
            N = int(rng.integers(3, 7))
            Ks = [np.rint(rng.standard_normal((N, d)) * 4) / 2 for _ in range(H)]
            cands = [[tuple(F(float(v)) for v in row) for row in Ks[h]] for h in range(H)]
            _, info = xr.update_sequential([_exact_bank(mod, b) for b in heads], cands, [M] * H, sigma2=1, p=2,
                                           tau=F(3), block_id=blk)
            new, rec = mod.update_layer(heads, Ks, [k.astype(np.float32) for k in Ks], blk, prm)
            for h in range(H):
                if heads[h].m == 0:
                    continue
                hr = rec.heads[h]
                assert hr.c.tolist() == info["counts"][h], f"seed {seed} block {blk} head {h}: per-step counts"
                assert hr.evicted.tolist() == info["released"][h], f"seed {seed} block {blk} head {h}: released"
                released += len(info["released"][h])
                viol_steps += sum(1 for c in info["counts"][h] if c > 0)
            rejected += sum(1 for ok in info["steps"] if not ok) if any(b.m for b in heads) else 0
            heads = new
    assert rejected > 0 and released > 0 and viol_steps > 0


def test_first_cross_matches_exact_bruteforce():
    first_cross_pin(ref_module)


def test_sequential_counts_and_released_match_exact_bruteforce():
    sequential_record_pin(ref_module)


# (description, text in the oracle source, planted replacement, pin that must fail)
PLANTS = [
    ("first-crossing sentinel R instead of R + 1",
     "fc = np.full(m, R + 1, np.int64)", "fc = np.full(m, R, np.int64)", first_cross_pin),
    ("first crossing one prefix late",
     "fc[i] = hit[0]", "fc[i] = hit[0] + 1", first_cross_pin),
    ("released list also counts states admitted in the same block",
     "if (int(w[\"prov\"][ev]) >> 32) != int(block_id):", "if True:", sequential_record_pin),
    ("per-step counts only where the step is feasible",
     "nviol[h, j] = viol.size", "nviol[h, j] = viol.size if viol.size <= e else 0", sequential_record_pin),
]


def _planted(src_old: str, src_new: str):
    with open(ORACLE_SRC) as f:
        src = f.read()
    assert src.count(src_old) == 1, f"plant target not found once: {src_old!r}"
    name = "_planted_oracle"
    spec = importlib.util.spec_from_loader(name, loader=None)
    mod = importlib.util.module_from_spec(spec)
    sys.modules[name] = mod   # dataclasses resolve their module through sys.modules
    try:
        exec(compile(src.replace(src_old, src_new), ORACLE_SRC + " (planted)", "exec"), mod.__dict__)
    except BaseException:
        del sys.modules[name]
        raise
    return mod


@pytest.mark.parametrize("plant", PLANTS, ids=[p[0] for p in PLANTS])
def test_planted_mistakes_fail(plant):
    _, old, new, pin = plant
    mod = _planted(old, new)
    try:
        with pytest.raises(AssertionError):
            pin(mod)
    finally:
        sys.modules.pop("_planted_oracle", None)
