"""Pins of the CPU oracle against what the paper and mathematics fix (CPU only).

Each test checks the oracle against something other than itself: closed
forms of the Soft-Riesz weight (Eq. 2; Supp. B), an exact rational rounding
chain, coordinate-wise brute force distances, the energy insertion identity
(Supp. B), hand-worked updates (tests/golden/hand_examples.json), an exact
rational brute force of the whole update (tests/exact_rational.py), the
post-commit invariants (Supp. C), and a scale symmetry of the weight.
"""

import json
import os
from fractions import Fraction as F

import numpy as np
import pytest

import exact_rational as xr
from oracle import (Q23, BankState, Params, attention, candidate_scores, density_from_scratch,
                    pair_d2, pair_d2_bruteforce, soft_riesz_weight, update_layer, weight_q23)
from paper_2608_27922_amd import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "hand_examples.json")


# ---------------------------------------------------------------- helpers

def rn32(x: F) -> F:
    """Round a rational to the nearest binary32 value, ties to even (normal range)."""
    if x == 0:
        return F(0)
    sign = -1 if x < 0 else 1
    a = abs(x)
    e = a.numerator.bit_length() - a.denominator.bit_length()
    if F(2) ** e > a:
        e -= 1
    if F(2) ** (e + 1) <= a:
        e += 1
    scaled = a / F(2) ** (e - 23)          # in [2^23, 2^24)
    q, r = divmod(scaled.numerator, scaled.denominator)
    twice = 2 * r
    if twice > scaled.denominator or (twice == scaled.denominator and q % 2 == 1):
        q += 1
    return sign * F(q) * F(2) ** (e - 23)


def rne_int(x: F) -> int:
    q, r = divmod(x.numerator, x.denominator)
    twice = 2 * r
    if twice > x.denominator or (twice == x.denominator and q % 2 == 1):
        q += 1
    return q


def contract_weight_exact(d2: F, s: int, p: int) -> int:
    """C2/C3 evaluated with exact rationals and explicit binary32 roundings."""
    u = d2 / F(2) ** s
    t = rn32(1 + u)
    tp = t if p == 1 else rn32(t * t)
    if p == 4:
        tp = rn32(tp * tp)
    w = rn32(1 / tp)
    return rne_int(w * Q23)


def bank_from_keys(keys, budget, prm, block_id=1, d=1):
    """Bank produced by the empty-bank rule (Alg. 1, first branch)."""
    K = np.asarray(keys, np.float64).reshape(len(keys), d)
    empty = BankState.empty(budget, d)
    (bank,), _ = update_layer([empty], [K], [K.astype(np.float32)], block_id, prm)
    return bank


def frac(s):
    n, d = s.split("/") if "/" in s else (s, "1")
    return F(int(n), int(d))


# ---------------------------------------------------------------- weight pins

@pytest.mark.parametrize("p", [1, 2, 4])
@pytest.mark.parametrize("s", [5, 6])
def test_weight_closed_forms(p, s):
    """d2 = j * sigma^2 gives w = (1 + j)^-p exactly (Eq. 2, eps = 1); d2 = 0 gives
    eps^-p = 1 for coinciding keys (Supp. B)."""
    sigma2 = 2.0 ** s
    for j in [0, 1, 3, 7, 15]:
        w = soft_riesz_weight(np.array([j * sigma2]), Params(sigma2_log2=s, p=p))[0]
        assert w == np.float32(1.0 / (1 + j) ** p)
        W = weight_q23(np.array([j * sigma2]), Params(sigma2_log2=s, p=p))[0]
        assert W == Q23 // (1 + j) ** p
    # monotone non-increasing in distance, within [0, 1]; far weights of order below
    # 2^-24 vanish in the Q23 fixed point (p = 4, sigma^2 = 32 at the grid's edge)
    d2 = np.arange(0, 2017, 0.25)
    W = weight_q23(d2, Params(sigma2_log2=s, p=p))
    assert W[0] == Q23 and np.all(np.diff(W) <= 0) and np.all(W >= 0)


@pytest.mark.parametrize("s,p", [(6, 2), (5, 2), (6, 1), (6, 4), (4, 2), (8, 2)])
def test_weight_matches_exact_rounding_chain(s, p):
    """NumPy binary32 arithmetic reproduces C2/C3 computed with exact rationals and
    explicit round-to-nearest-even at every step."""
    rng = np.random.default_rng(1000 + s * 10 + p)
    n = rng.integers(0, 8_258_049, 300)           # d2 * 2^12 over the whole grid range
    n = np.concatenate([n, [0, 1, 2, 4095, 4096, 8_258_048]])
    d2 = n / 4096.0
    W = weight_q23(d2, Params(sigma2_log2=s, p=p))
    for ni, Wi in zip(n, W):
        assert Wi == contract_weight_exact(F(int(ni), 4096), s, p), ni


def test_pair_d2_equals_bruteforce():
    """Gram expansion (C1) equals the coordinate-wise squared distance on grid keys,
    including the extreme grid values."""
    rng = np.random.default_rng(7)
    for d in (1, 3, 64, 128):
        A = synth.random_grid_keys(rng, (17, d), scale=0.7)
        B = synth.random_grid_keys(rng, (9, d), scale=0.7)
        A[0] = 127 / 64.0
        B[0] = -127 / 64.0
        got = pair_d2(A, B)
        ref = pair_d2_bruteforce(A, B)
        assert np.array_equal(got, ref)
        # integer grid units: exactly an integer number of 2^-12
        assert np.array_equal(got * 4096, np.rint(got * 4096))


def test_density_energy_identity_and_duplicates():
    """Phi_A(x) = E(A + x) - E(A) with E = sum(Phi)/2 (Supp. B insertion identity), and
    every duplicate of a distinct entry contributes eps^-p = 1 (Supp. B)."""
    prm = Params()
    rng = np.random.default_rng(3)
    A = synth.random_grid_keys(rng, (40, 16))
    A[5] = A[9]                                   # indexed duplicates
    A[11] = A[9]
    x = synth.random_grid_keys(rng, (1, 16))
    phiA = density_from_scratch(A, prm)
    phiAx = density_from_scratch(np.vstack([A, x]), prm)
    assert phiA.sum() % 2 == 0
    E_A, E_Ax = phiA.sum() // 2, phiAx.sum() // 2
    assert E_Ax - E_A == weight_q23(pair_d2(x, A), prm).sum() == phiAx[-1]
    # duplicates: 9 sees 5 and 11 at weight exactly 1
    W = weight_q23(pair_d2(A, A), prm)
    assert W[9, 5] == W[9, 11] == Q23
    others = [j for j in range(40) if j not in (5, 9, 11)]
    assert phiA[9] == 2 * Q23 + W[9, others].sum()
    # a single-entry multiset has zero density
    assert density_from_scratch(A[:1], prm)[0] == 0


# ---------------------------------------------------------------- hand-worked updates

def _golden():
    with open(GOLDEN) as f:
        return json.load(f)


@pytest.mark.parametrize("case", _golden()["cases"], ids=lambda c: c["name"])
def test_hand_examples_exact_bruteforce(case):
    """The independent exact-rational brute force reproduces every hand-derived value."""
    keys = [(F(str(k)),) for k in case["bank_keys"]]
    bank = xr.build(keys, case["budget"]) if keys else []
    cands = [(F(str(k)),) for k in case["cands"]]
    new, info = xr.update(bank, cands, case["budget"], block_id=2)
    assert info["r_star"] == case["r_star"]
    assert info["evicted"] == case["evicted"] and info["admitted"] == case["admitted"]
    if "pi" in case:
        assert info["pi"] == case["pi"]
    if "c" in case:
        assert info["c"] == case["c"]
    if "first_cross" in case:
        assert info["first_violation"] == case["first_cross"]
    if "scores" in case:
        assert info["scores"] == [frac(s) for s in case["scores"]]
    assert [float(s["key"][0]) for s in new] == [float(k) for k in case["final_keys"]]
    assert [s["rho"] for s in new] == [frac(s) for s in case["final_rho"]]
    assert [s["b"] for s in new] == [frac(s) for s in case["final_base"]]


@pytest.mark.parametrize("case", _golden()["cases"], ids=lambda c: c["name"])
def test_hand_examples_oracle(case):
    """Oracle decisions equal the hand-worked ones; its Q23 densities round to them."""
    g = _golden()
    prm = Params(**g["params"])
    if case["bank_keys"]:
        bank = bank_from_keys(case["bank_keys"], case["budget"], prm, block_id=1)
    else:
        bank = BankState.empty(case["budget"], 1)
    K = np.asarray(case["cands"], np.float64).reshape(-1, 1)
    (new,), rec = update_layer([bank], [K], [K.astype(np.float32) + 1000.0], 2, prm)
    hr = rec.heads[0]
    assert rec.r_star == case["r_star"]
    assert list(hr.evicted) == case["evicted"]
    assert list(hr.admitted) == case["admitted"]
    if "pi" in case:
        assert list(hr.pi) == case["pi"]
    if "c" in case:
        assert list(hr.c) == case["c"]
    if "first_cross" in case:
        assert list(hr.first_cross) == case["first_cross"]
    assert list(new.K[:, 0]) == [float(k) for k in case["final_keys"]]
    # values moved unchanged with their keys
    assert np.array_equal(new.V[new.prov >> 32 == 2, 0] - 1000.0,
                          new.K[new.prov >> 32 == 2, 0].astype(np.float32))
    n_terms = new.m + len(case["cands"]) + 1
    tol = n_terms * 2.0 ** -22
    for q, ref in zip(new.rho, case["final_rho"]):
        assert abs(q / Q23 - float(frac(ref))) <= tol
    for q, ref in zip(new.base, case["final_base"]):
        assert abs(q / Q23 - float(frac(ref))) <= tol
    if "scores" in case and bank.m:
        S, E, s_real = candidate_scores(bank.K, bank.base, K, prm)
        for sr, ref in zip(s_real, case["scores"]):
            assert abs(sr - float(frac(ref))) <= 1e-5 * float(frac(ref))
    if "projected_tie" in case:
        tie = hr.rho_tilde[[0, 3]]
        assert tie[0] == tie[1]
        assert abs(tie[0] / Q23 - float(frac(case["projected_tie"]))) <= 8 * 2.0 ** -22


# ---------------------------------------------------------------- random tiny rollouts vs exact

def _to_exact_bank(bank: BankState):
    return [{"key": tuple(F(float(v)) for v in bank.K[i]), "b": F(int(bank.base[i]), Q23),
             "prov": int(bank.prov[i])} for i in range(bank.m)]


@pytest.mark.parametrize("seed", range(6))
def test_tiny_rollout_matches_exact_bruteforce(seed):
    """Oracle and the exact-rational brute force agree on every decision of a random
    multi-head rollout (shared prefix, empty start, evictions, ragged occupancy)."""
    rng = np.random.default_rng(seed)
    d, H, M = 2, 3, 7
    prm = Params(sigma2_log2=0, p=2)
    heads = [BankState.empty(M, d) for _ in range(H)]
    for blk in range(1, 7):
        N = int(rng.integers(2, 5))
        Ks = [np.rint(rng.standard_normal((N, d)) * 4) / 2 for _ in range(H)]
        new, rec = update_layer(heads, Ks, [k.astype(np.float32) for k in Ks], blk, prm)
        # exact brute force of the shared prefix: every head's c_r, then r*
        infos = []
        for h in range(H):
            _, info = xr.update(_to_exact_bank(heads[h]),
                                [tuple(F(float(v)) for v in row) for row in Ks[h]], M,
                                sigma2=1, p=2, block_id=blk)
            infos.append(info)
        R = rec.R
        feas = [r for r in range(R + 1)
                if all(infos[h]["c"][r] <= infos[h]["e"][r] for h in range(H))]
        assert rec.r_star == (max(feas) if feas else 0)
        for h in range(H):
            assert list(rec.heads[h].c) == infos[h]["c"]
            if heads[h].m:
                assert list(rec.heads[h].pi) == infos[h]["pi"]
        heads = new
        for h in range(H):
            exact = [xr.phi([tuple(F(float(v)) for v in row) for row in heads[h].K], i, 1, 2)
                     for i in range(heads[h].m)]
            for q, ref in zip(heads[h].rho, exact):
                assert abs(q / Q23 - float(ref)) <= heads[h].m * 2.0 ** -22


POLICIES = {
    "source_order": dict(source_order=True),
    "refresh_base": dict(refresh_base=True),
    "densest": dict(eviction="densest"),
    "mandatory_source": dict(eviction="mandatory_source"),
}


@pytest.mark.parametrize("policy", list(POLICIES))
def test_policy_rollouts_match_exact_bruteforce(policy):
    """The policy ablations of Table 1(b) (Supp. E): on random multi-head rollouts the
    oracle's order, violator counts, shared r*, eviction and admission sets, commit
    layout, densities and baselines equal the exact-rational brute force run with the
    same policy, and the policy changes at least one decision against the default."""
    kw = POLICIES[policy]
    d, H, M = 2, 3, 7
    prm = Params(sigma2_log2=0, p=2, **kw)
    differs = 0
    for seed in range(4):
        rng = np.random.default_rng(100 + seed)
        heads = [BankState.empty(M, d) for _ in range(H)]
        for blk in range(1, 8):
            N = int(rng.integers(2, 6))
            Ks = [np.rint(rng.standard_normal((N, d)) * 4) / 2 for _ in range(H)]
            new, rec = update_layer(heads, Ks, [k.astype(np.float32) for k in Ks], blk, prm)
            cands = [[tuple(F(float(v)) for v in row) for row in Ks[h]] for h in range(H)]
            infos = [xr.update(_to_exact_bank(heads[h]), cands[h], M, sigma2=1, p=2, block_id=blk, **kw)[1]
                     for h in range(H)]
            feas = [r for r in range(rec.R + 1) if all(infos[h]["c"][r] <= infos[h]["e"][r] for h in range(H))]
            assert rec.r_star == (max(feas) if feas else 0)
            for h in range(H):
                xb, info = xr.update(_to_exact_bank(heads[h]), cands[h], M, sigma2=1, p=2, block_id=blk,
                                     r_star=rec.r_star, **kw)
                _, dflt = xr.update(_to_exact_bank(heads[h]), cands[h], M, sigma2=1, p=2, block_id=blk,
                                    r_star=rec.r_star)
                hr, nb = rec.heads[h], new[h]
                assert list(hr.c) == info["c"]
                if heads[h].m:
                    assert list(hr.pi) == info["pi"]
                assert hr.evicted.tolist() == info["evicted"]
                assert hr.admitted.tolist() == info["admitted"]
                assert nb.prov.tolist() == [s["prov"] for s in xb]
                tol = max(nb.m, 1) * 2.0 ** -22
                for q, s in zip(nb.rho, xb):
                    assert abs(q / Q23 - float(s["rho"])) <= tol
                for q, s in zip(nb.base, xb):
                    assert abs(q / Q23 - float(s["b"])) <= tol
                if policy == "source_order":
                    differs += heads[h].m > 0 and info["pi"] != sorted(range(N), key=lambda x: (info["scores"][x], x))
                elif policy == "refresh_base":
                    old = {int(pv): int(bs) for pv, bs in zip(heads[h].prov, heads[h].base)}
                    differs += any(int(pv) in old and int(bs) != old[int(pv)] for pv, bs in zip(nb.prov, nb.base))
                else:
                    differs += info["evicted"] != dflt["evicted"]
            heads = new
    assert differs > 0, "the policy never changed a decision in these rollouts"


@pytest.mark.parametrize("kw", [dict(tau_num=3), dict(tau_num=2), dict(tau_num=3, source_order=True),
                                dict(tau_num=3, refresh_base=True)])
def test_sequential_rollouts_match_exact_bruteforce(kw):
    """Within-block sequential competition (Supp. E): on random multi-head rollouts
    the oracle's per-step decisions, commit layout, densities and baselines equal
    the exact-rational brute force, which recomputes every density from its
    definition at every step; the rollouts take steps with releases, release states
    admitted earlier in the same block, and decide differently from the default."""
    d, H, M = 2, 3, 6
    prm = Params(sigma2_log2=0, p=2, sequential=True, **kw)
    dflt = Params(sigma2_log2=0, p=2, **{k: v for k, v in kw.items() if k != "sequential"})
    taken = released_same_block = differs = 0
    for seed in range(4):
        rng = np.random.default_rng(300 + seed)
        heads = [BankState.empty(M, d) for _ in range(H)]
        for blk in range(1, 8):
            N = int(rng.integers(3, 7))
            Ks = [np.rint(rng.standard_normal((N, d)) * 4) / 2 for _ in range(H)]
            cands = [[tuple(F(float(v)) for v in row) for row in Ks[h]] for h in range(H)]
            xb, info = xr.update_sequential([_to_exact_bank(b) for b in heads], cands, [M] * H, sigma2=1, p=2,
                                            tau=F(kw["tau_num"]), block_id=blk,
                                            source_order=kw.get("source_order", False),
                                            refresh_base=kw.get("refresh_base", False))
            new, rec = update_layer(heads, Ks, [k.astype(np.float32) for k in Ks], blk, prm)
            ref, _ = update_layer(heads, Ks, [k.astype(np.float32) for k in Ks], blk, dflt)
            if any(b.m for b in heads):
                assert rec.steps.tolist() == info["steps"]
                taken += int(rec.steps.sum())
                released_same_block += sum(int(rec.steps.sum()) - len(rec.heads[h].admitted) for h in range(H))
            for h in range(H):
                nb = new[h]
                if heads[h].m:
                    assert rec.heads[h].pi.tolist() == info["orders"][h]
                assert nb.prov.tolist() == [s["prov"] for s in xb[h]]
                assert np.array_equal(nb.K, np.array([[float(v) for v in s["key"]] for s in xb[h]]).reshape(nb.K.shape))
                tol = max(nb.m, 1) * 2.0 ** -22
                for q, s in zip(nb.rho, xb[h]):
                    assert abs(q / Q23 - float(s["rho"])) <= tol
                for q, s in zip(nb.base, xb[h]):
                    assert abs(q / Q23 - float(s["b"])) <= tol
                differs += nb.prov.tolist() != ref[h].prov.tolist()
            heads = new
    assert taken > 0 and differs > 0
    if kw["tau_num"] == 3:
        assert released_same_block > 0, "no state admitted earlier in a block was released by a later one"


def test_sequential_release_tie_goes_to_earlier_admission():
    """An exact densest-release tie in the sequential variant: bank {-10, -1, 1, 10}
    (full, M = 4), candidate 0, tau = 4 so that no state violates; -1 and 1 have the
    same projected density, and the earlier-admitted -1 (smaller provenance) leaves."""
    prm = Params(sigma2_log2=0, p=1, tau_num=4, sequential=True)
    keys = np.array([[-10.0], [-1.0], [1.0], [10.0]])
    bank, _ = update_layer([BankState.empty(4, 1)], [keys], [keys.astype(np.float32)], 0, prm)
    assert bank[0].prov.tolist() == [0, 1, 2, 3]
    new, rec = update_layer(bank, [np.array([[0.0]])], [np.zeros((1, 1), np.float32)], 1, prm)
    assert rec.steps.tolist() == [True]
    assert new[0].prov.tolist() == [0, (1 << 32) | 0, 2, 3]
    xb, info = xr.update_sequential([_to_exact_bank(bank[0])], [[(F(0),)]], [4], sigma2=1, p=1, tau=F(4),
                                    block_id=1)
    assert info["steps"] == [True]
    assert [s["prov"] for s in xb[0]] == new[0].prov.tolist()


def _to_exact_bank_kv(bank: BankState):
    return [{"key": tuple(F(float(v)) for v in np.concatenate([bank.K[i], bank.V[i]])),
             "b": F(int(bank.base[i]), Q23), "prov": int(bank.prov[i])} for i in range(bank.m)]


def test_kv_descriptor_rollouts_match_exact_bruteforce():
    """The [K; V] retention geometry (Supp. E, "Retention geometry"): on random
    multi-head rollouts every decision, the commit layout and the densities equal the
    exact-rational brute force run on the concatenated key-value descriptors, the
    stored keys and values are the candidates' own rows, and the geometry changes at
    least one decision against the key-only default."""
    d, H, M = 2, 3, 7
    prm = Params(sigma2_log2=1, p=2, kv_descriptor=True)
    key_only = Params(sigma2_log2=1, p=2)
    differs = 0
    for seed in range(4):
        rng = np.random.default_rng(200 + seed)
        heads = [BankState.empty(M, d) for _ in range(H)]
        ref_heads = [BankState.empty(M, d) for _ in range(H)]
        for blk in range(1, 8):
            N = int(rng.integers(2, 6))
            Ks = [np.rint(rng.standard_normal((N, d)) * 4) / 2 for _ in range(H)]
            Vs = [(np.rint(rng.standard_normal((N, d)) * 4) / 2).astype(np.float32) for _ in range(H)]
            new, rec = update_layer(heads, Ks, Vs, blk, prm)
            _, rec_k = update_layer(heads, Ks, Vs, blk, key_only)
            cands = [[tuple(F(float(v)) for v in np.concatenate([Ks[h][i], Vs[h][i]])) for i in range(N)]
                     for h in range(H)]
            infos = [xr.update(_to_exact_bank_kv(heads[h]), cands[h], M, sigma2=2, p=2, block_id=blk)[1]
                     for h in range(H)]
            feas = [r for r in range(rec.R + 1) if all(infos[h]["c"][r] <= infos[h]["e"][r] for h in range(H))]
            assert rec.r_star == (max(feas) if feas else 0)
            for h in range(H):
                xb, info = xr.update(_to_exact_bank_kv(heads[h]), cands[h], M, sigma2=2, p=2, block_id=blk,
                                     r_star=rec.r_star)
                hr, nb = rec.heads[h], new[h]
                assert list(hr.c) == info["c"]
                if heads[h].m:
                    assert list(hr.pi) == info["pi"]
                assert hr.evicted.tolist() == info["evicted"] and hr.admitted.tolist() == info["admitted"]
                assert nb.prov.tolist() == [s["prov"] for s in xb]
                for i, s in enumerate(xb):
                    assert tuple(F(float(v)) for v in np.concatenate([nb.K[i], nb.V[i]])) == s["key"]
                tol = max(nb.m, 1) * 2.0 ** -22
                for q, s in zip(nb.rho, xb):
                    assert abs(q / Q23 - float(s["rho"])) <= tol
                for q, s in zip(nb.base, xb):
                    assert abs(q / Q23 - float(s["b"])) <= tol
                differs += (hr.evicted.tolist() != rec_k.heads[h].evicted.tolist() or
                            hr.pi.tolist() != rec_k.heads[h].pi.tolist())
            heads = new
    assert differs > 0, "the [K; V] descriptor never changed a decision in these rollouts"


def test_refresh_base_keeps_delta_floor():
    """Refreshed baselines (Table 1(b), Supp. E) still obey b >= delta (Eq. 5): isolated
    keys have rho = 0 after the update, so every refreshed baseline is delta."""
    prm = Params(sigma2_log2=0, p=2, refresh_base=True)
    keys = np.array([[0.0], [1000.0]])
    bank, _ = update_layer([BankState.empty(4, 1)], [keys], [keys.astype(np.float32)], 0, prm)
    new, rec = update_layer(bank, [np.array([[-1000.0]])], [np.zeros((1, 1), np.float32)], 1, prm)
    assert rec.r_star == 1 and new[0].m == 3
    assert new[0].rho.tolist() == [0, 0, 0]
    assert new[0].base.tolist() == [prm.delta_q] * 3
    xb, _ = xr.update(_to_exact_bank(bank[0]), [(F(-1000),)], 4, sigma2=1, p=2, refresh_base=True)
    assert [float(s["b"]) for s in xb] == [1e-6] * 3


# ---------------------------------------------------------------- invariants on cluster data

def _small_cfg(**kw):
    base = dict(seed_id=91, name="pin", layers=1, heads=4, d=16, dtype="f32", n_cand=24,
                n_query=8, n_window=8, budget=48, clusters=4, blocks=10, group_size=4,
                sigma2_log2=3, drift=0.05)
    base.update(kw)
    return synth.Config(**base)


def _check_invariants(prev, new, rec, cand_K, cand_V, block_id, prm, history_V):
    H = len(prev)
    T, k = prm.tau_num, prm.tau_log2_den
    assert len({b.m for b in new}) == 1 or len({b.budget for b in new}) > 1
    for h in range(H):
        b0, b1, hr = prev[h], new[h], rec.heads[h]
        assert b1.m <= b1.budget                                      # Eq. 4
        assert np.array_equal(b1.rho, density_from_scratch(b1.K, prm))  # exact maintenance
        assert np.all((b1.rho << k) < T * b1.base)                    # invariant after commit
        assert np.all(b1.base >= prm.delta_q)
        assert len(set(b1.prov.tolist())) == b1.m
        old = dict(zip(b0.prov.tolist(), b0.base.tolist()))
        for pv, bs in zip(b1.prov.tolist(), b1.base.tolist()):
            if pv in old:
                assert bs == old[pv]                                  # frozen baseline
            else:
                assert pv >> 32 == block_id                           # retained subset of history
        for s in range(b1.m):                                          # values move with keys
            blk, src = int(b1.prov[s]) >> 32, int(b1.prov[s]) & 0xFFFFFFFF
            assert np.array_equal(b1.V[s], history_V[(h, blk)][src])
        # eviction rule at r*
        e = max(0, b0.m + rec.r_star - b0.budget)
        assert hr.e == e
        if b0.m:
            viol = (hr.rho_tilde << k) >= T * b0.base
            assert set(np.nonzero(viol)[0]) <= set(hr.evicted.tolist())
            assert hr.evicted.size == max(e, int(viol.sum()))
            fill = [s for s in hr.evicted if not viol[s]]
            kept = [s for s in range(b0.m) if s not in set(hr.evicted.tolist()) and not viol[s]]
            if fill and kept:
                assert min(hr.rho_tilde[fill]) >= max(hr.rho_tilde[kept])
        if e == 0:
            assert hr.evicted.size == 0                               # no eviction under budget
    # r* is feasible and maximal, from densities recomputed over bank (+) prefix
    R = rec.R
    feas = []
    for r in range(R + 1):
        ok = True
        for h in range(H):
            b0 = prev[h]
            if b0.m == 0:
                continue
            pre = cand_K[h][rec.heads[h].pi[:r]]
            phi = density_from_scratch(np.vstack([b0.K, pre]), prm)[: b0.m]
            c = int(np.count_nonzero((phi << k) >= T * b0.base))
            ok &= c <= max(0, b0.m + r - b0.budget)
        feas.append(ok)
    assert feas[rec.r_star] and not any(feas[rec.r_star + 1:])


@pytest.mark.parametrize("cfg_kw", [dict(), dict(budget=30, n_cand=24), dict(group_size=1, heads=3)])
def test_rollout_invariants(cfg_kw):
    cfg = _small_cfg(**cfg_kw)
    prm = Params(sigma2_log2=cfg.sigma2_log2)
    streams = [synth.HeadStream(cfg, 0, h) for h in range(cfg.heads)]
    groups = [list(range(g, g + cfg.group_size)) for g in range(0, cfg.heads, cfg.group_size)]
    banks = [BankState.empty(cfg.budget, cfg.d) for _ in range(cfg.heads)]
    history_V = {}
    for t in range(cfg.blocks):
        Ks = [s.keys(t, cfg.n_cand).astype(np.float64) for s in streams]
        Vs = [s.values(t, cfg.n_cand) for s in streams]
        for h in range(cfg.heads):
            history_V[(h, t)] = Vs[h]
        for g in groups:
            prev = [banks[h] for h in g]
            new, rec = update_layer(prev, [Ks[h] for h in g], [Vs[h] for h in g], t, Params(sigma2_log2=cfg.sigma2_log2))
            _check_invariants(prev, new, rec, [Ks[h] for h in g], None, t, prm,
                              {(i, blk): history_V[(h, blk)] for i, h in enumerate(g)
                               for blk in range(t + 1)})
            for i, h in enumerate(g):
                banks[h] = new[i]


def test_corrupted_bank_no_feasible_prefix():
    """A bank that already violates the growth bound before the update (outside the
    paper's precondition) has no feasible prefix: r* = 0, every violator is evicted
    and the remaining states are compacted (C8, C10)."""
    prm = Params(sigma2_log2=0, p=1)
    bank = bank_from_keys([0, 3, 6, 9, 12], 8, prm)   # under budget: e_r = 0 for r <= 2
    bank.base[1] = bank.rho[1] // 4      # rho >= 2 b: a violator at r = 0
    bank.base[2] = bank.rho[2] // 4
    K = np.array([[20.0], [21.0]])
    (new,), rec = update_layer([bank], [K], [K.astype(np.float32)], 2, prm)
    assert rec.r_star == 0
    assert list(rec.heads[0].evicted) == [1, 2]
    # slots 1 and 2 are freed and the occupancy drops to 3: the survivors at slots
    # >= 3 (keys 9 and 12) move into holes 1 and 2, both in ascending order.
    assert list(new.K[:, 0]) == [0.0, 9.0, 12.0]
    assert np.array_equal(new.rho, density_from_scratch(new.K, prm))


# ---------------------------------------------------------------- symmetry and score

def test_scale_symmetry():
    """Halving every key and dividing sigma^2 by 4 leaves u = d2 / sigma^2, hence every
    weight, density and decision, unchanged (the scale separation of Supp. B)."""
    cfg = _small_cfg(heads=2, group_size=2, blocks=4)
    streams = [synth.HeadStream(cfg, 0, h) for h in range(2)]
    p1, p2 = Params(sigma2_log2=4), Params(sigma2_log2=2)
    a = [BankState.empty(cfg.budget, cfg.d) for _ in range(2)]
    b = [BankState.empty(cfg.budget, cfg.d) for _ in range(2)]
    for t in range(cfg.blocks):
        Ks = [s.keys(t, cfg.n_cand).astype(np.float64) for s in streams]
        Vs = [s.values(t, cfg.n_cand) for s in streams]
        a, ra = update_layer(a, Ks, Vs, t, p1)
        b, rb = update_layer(b, [k / 2 for k in Ks], Vs, t, p2)
        assert ra.r_star == rb.r_star
        for x, y in zip(a, b):
            assert np.array_equal(x.prov, y.prov) and np.array_equal(x.rho, y.rho)
            assert np.array_equal(x.base, y.base) and np.array_equal(x.K, 2 * y.K)


def test_score_proxy_orders_like_exact_score():
    """The fixed-point score S_x orders candidates like the exact s_h(x) of Eq. 6 and
    equals 2^(23-E) m s_h(x) within the per-term rounding bound."""
    rng = np.random.default_rng(11)
    prm = Params(sigma2_log2=1, p=2)
    K = np.rint(rng.standard_normal((6, 2)) * 4) / 2
    empty = BankState.empty(10, 2)
    (bank,), _ = update_layer([empty], [K], [K.astype(np.float32)], 1, prm)
    C = np.rint(rng.standard_normal((12, 2)) * 4) / 2
    S, E, s_real = candidate_scores(bank.K, bank.base, C, prm)
    exact = []
    for x in C:
        tot = sum(xr.weight(tuple(F(float(v)) for v in k), tuple(F(float(v)) for v in x), 2, 2)
                  / F(int(b), Q23) for k, b in zip(bank.K, bank.base))
        exact.append(tot / bank.m)
    for sr, ex in zip(s_real, exact):
        assert abs(sr - float(ex)) <= 1e-5 * float(ex)
    order_exact = sorted(range(len(C)), key=lambda i: (exact[i], i))
    assert list(np.argsort(S, kind="stable")) == order_exact


# ---------------------------------------------------------------- attention pins

def test_attention_special_cases():
    rng = np.random.default_rng(5)
    d = 8
    q = rng.standard_normal((4, d))
    v = rng.standard_normal((1, d))
    k = rng.standard_normal((1, d))
    out = attention(q, k, v, np.zeros((0, d)), np.zeros((0, d)), 0.3)
    assert np.allclose(out, np.repeat(v, 4, 0), rtol=0, atol=1e-15)     # one key: O = V
    K = np.repeat(rng.standard_normal((1, d)), 5, 0)
    V = rng.standard_normal((5, d))
    out = attention(q, K[:3], V[:3], K[3:], V[3:], 0.7)                  # identical keys
    assert np.allclose(out, np.repeat(V.mean(0, keepdims=True), 4, 0), atol=1e-14)


def test_attention_key_order_invariance():
    """Softmax attention does not depend on the order of the keys (with their values):
    the sink + window + bank context (Supp. D) is the bank call with the sink appended
    to the window, whatever the segment order."""
    rng = np.random.default_rng(8)
    d = 16
    q = rng.standard_normal((9, d))
    Kb, Vb = rng.standard_normal((30, d)), rng.standard_normal((30, d))
    Kw, Vw = rng.standard_normal((11, d)), rng.standard_normal((11, d))
    Ks, Vs = rng.standard_normal((7, d)), rng.standard_normal((7, d))
    a = attention(q, Kb, Vb, np.concatenate([Kw, Ks]), np.concatenate([Vw, Vs]), 0.25)
    perm = rng.permutation(48)
    K = np.concatenate([Kb, Kw, Ks])[perm]
    V = np.concatenate([Vb, Vw, Vs])[perm]
    b = attention(q, K[:20], V[:20], K[20:], V[20:], 0.25)
    assert np.allclose(a, b, rtol=0, atol=1e-12)
    # brute force: explicit softmax weights over the concatenated keys
    s = q @ np.concatenate([Kb, Kw, Ks]).T * 0.25
    w = np.exp(s) / np.exp(s).sum(1, keepdims=True)
    assert np.allclose(a, w @ np.concatenate([Vb, Vw, Vs]), rtol=0, atol=1e-12)


def test_attention_matches_torch_sdpa_fp64():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(9)
    d, nq, mb, w = 64, 33, 70, 21
    q = rng.standard_normal((nq, d))
    kb, vb = rng.standard_normal((mb, d)), rng.standard_normal((mb, d))
    kw, vw = rng.standard_normal((w, d)), rng.standard_normal((w, d))
    got = attention(q, kb, vb, kw, vw, 1.0 / np.sqrt(d))
    ref = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(q)[None], torch.from_numpy(np.vstack([kb, kw]))[None],
        torch.from_numpy(np.vstack([vb, vw]))[None]).numpy()[0]
    assert np.allclose(got, ref, rtol=1e-12, atol=1e-12)
    # zero query: uniform weights, output = mean of all values
    z = attention(np.zeros((1, d)), kb, vb, kw, vw, 0.125)
    assert np.allclose(z[0], np.vstack([vb, vw]).mean(0), atol=1e-13)
