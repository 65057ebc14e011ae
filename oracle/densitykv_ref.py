"""DensityKV oracle: the bank update for one layer and the bank attention, on the CPU.

TEST INFRASTRUCTURE ONLY (see the package docstring): a plain, slow, obviously
correct NumPy transcription of the paper's method, used to check the HIP path.

Arithmetic contract
-------------------
The paper states every decision (candidate order, violator counts, the shared
prefix, the eviction set) on real numbers and does not fix a summation order
or a rounding.  Sums of thousands of floating-point terms differ in their last
bits between reduction trees, and near-ties then flip.  The oracle therefore
fixes the following reading, under which every decision is a deterministic
function of the inputs and any correct implementation reproduces it bit for
bit:

C0  Keys lie on the grid n/64 with integer |n| <= 127 (exact in bf16 and fp32).
    Every key-key inner product is then an integer multiple of 2^-12 below
    2^21 in magnitude, so the Gram is exact in fp32 or fp64 in any order.
C1  Squared distance d2 = |k_i|^2 + |k_j|^2 - 2<k_i, k_j> (Sec. 3.2: squared
    Euclidean distance supports batched evaluation); exact by C0.
C2  Soft-Riesz weight (Sec. 3.3, Eq. 2) with eps = 1 and sigma^2 = 2^s, every
    step one IEEE binary32 operation rounded to nearest-even:
        u = d2 * 2^-s (exact), t = 1 + u, t_p = t | t*t | (t*t)*(t*t) for
        p = 1 | 2 | 4, w = 1 / t_p.
C3  Fixed point: W = RNE(w * 2^23) (an integer in [0, 2^23]).  Every density,
    prefix and score is an exact int64 sum of such terms, so tiling and
    summation order play no role (Supp. C, "Decision granularity versus
    computational tiling").  delta is stored as RNE(delta * 2^23).
C4  Density Phi_A(i) = sum over j != i (by index) of W_ij (Eq. 3); duplicate
    keys of distinct entries contribute 2^23 each (Supp. B, eps^-p = 1).
C5  Baseline b = max(Phi of the final bank, delta), frozen (Eq. 5).
C6  Candidate score (Eq. 6) as a fixed-point proxy of m * s_h(x):
        inv_i = fp32(fp64(2^23) / fp64(b_i))        (= 1/b_i in real units),
        E     = binary exponent of max_i inv_i       (max inv < 2^E),
        bs_i  = inv_i * 2^(23 - E)                   (exact, <= 2^23),
        A_ix  = RNE(w_ix * bs_i)                     (exact product, one rounding),
        S_x   = sum_i A_ix   (int64).
    S_x = 2^(23-E) * m * s_h(x) up to the per-term rounding; 1/m and 2^(23-E)
    are common to all candidates of the head, so they do not change the order.
    Ties of S_x are broken by source order (stable sort, Alg. 1).
C7  Violation test of Eqs. 8-9 without a division: state i violates at prefix
    r iff 2^k * (rho_i + P_i(r)) >= T * b_i with tau = T / 2^k.
C8  e_r = max(0, m + r - M) (Eq. 10); r* is the largest r in [0, min(N, M)]
    feasible for every head of the layer (Eq. 11), found by testing every r
    (feasibility is not monotone in r).  With a state that already violates
    before the update no r is feasible; r* is then 0.
C9  Eviction (Sec. 3.4 step 3): all violators at r*, then the non-violators
    of largest unnormalised projected density rho~(r*) until e_{r*} are
    released.  The paper leaves fill ties open; this reading evicts the
    earlier-admitted state first (smaller provenance, then lower slot).
C10 Commit layout (Eq. 12; the paper does not fix slot order): survivors keep
    their slots; admitted candidates, in ascending source index, fill the
    evicted slots in ascending order and are then appended.  Holes left when
    more states are evicted than admitted are closed by moving the survivors
    that sit at or beyond the new occupancy into them (both ascending).
    Provenance is (block_id << 32) | source index.
C11 Maintenance (Supp. C, "Exact density maintenance"): survivors
    rho <- rho + sum_admitted W - sum_evicted W; new states
    rho <- Phi over the final bank, b <- max(rho, delta).
C12 Empty bank: the first min(N, M) candidates in source order, rho = Phi of
    the resulting bank, b = max(rho, delta) (Alg. 1, first branch).

Policy ablations (Supp. E, "Candidate ordering", "Density baseline",
"Eviction rule"; Table 1(b)), each off by default:
V1  source_order: the tested prefixes follow the candidates' source order
    instead of the score order; the scores are still reported.
V2  refresh_base: after every update every retained state's baseline is
    recomputed from its current density, b <- max(rho, delta).
V3  eviction = "densest": no mandatory set; the e_{r*} states of largest
    rho~(r*) are released (ties as in C9).  The prefix rule (C7-C8) is
    unchanged, so a violator that is not among them stays in the bank.
V4  eviction = "mandatory_source": all violators, then the non-violators in
    source order, read as admission order (ascending provenance, then slot).
The independent per-head variant is a layer of one head (group size 1).
V5  kv_descriptor: the retention geometry uses the concatenated vector [k; v]
    (Supp. E, "Retention geometry"; the post-RoPE [K;V] rows of Table 1(b))
    for every density, score and crossing; attention and the stored rows are
    unchanged.  C0 then applies to the values too (the synthetic values of
    this mode are drawn on the key grid).
V6  sequential: within-block competition (Supp. E, "Within-block competition";
    Supp. C, "Insertion hysteresis"; Sec. 4.5): admission one candidate at a
    time, each tested against the bank that the earlier candidates of the same
    block have already changed.  Reading: the candidates keep the order of C6 (or V1), fixed
    at the start of the block, and are taken one at a time.  Step j tests the
    j-th candidate x of every head as a one-candidate prefix against that
    head's current bank, which already holds the candidates admitted at
    earlier steps with their exactly maintained densities and their baselines
    frozen when they entered: violators are the states with
    2^k (rho_i + W_ix) >= T b_i, e = max(0, m + 1 - M) (so e <= 1), and the
    j-th candidates enter iff every head of the layer has at most e violators
    (a rejected step drops them).  On entry each head releases its violator,
    or, with none and e = 1, its state of largest rho_i + W_ix (ties as C9);
    survivors rho_i += W_ix - W_i,released; the new state's rho is the sum of
    W_xi over the survivors, b = max(rho, delta); it takes the released slot,
    else the next free one.  A head whose bank is empty at the start of the
    block takes the empty-bank rule (C12) and stays out of the shared test.
    V2 is applied at the end of the block; V3-V5 are not combined with V6.
"""

from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Optional, Sequence

import numpy as np

Q23 = 1 << 23  # fixed-point scale: weight 1.0 == 2^23

# The per-head steps of one layer update share no data (only r* couples the
# heads), so they are applied with HEAD_MAP, the builtin map unless a caller
# that runs the oracle at full size sets a thread pool's map; the results do
# not depend on it.
HEAD_MAP = map


@dataclass(frozen=True)
class Params:
    """Method parameters (Sec. 4.1 defaults: eps = 1, p = 2, sigma = 8,
    delta = 1e-6, tau = 2).  sigma^2 = 2^sigma2_log2; tau = tau_num / 2^tau_log2_den."""

    sigma2_log2: int = 6
    p: int = 2
    tau_num: int = 2
    tau_log2_den: int = 0
    delta_q: int = 8  # RNE(1e-6 * 2^23)
    # policy ablations (V1-V4 above); the defaults are the paper's policy
    source_order: bool = False
    refresh_base: bool = False
    eviction: str = "default"  # "default" | "densest" | "mandatory_source"
    kv_descriptor: bool = False
    sequential: bool = False

    def __post_init__(self):
        if self.p not in (1, 2, 4):
            raise ValueError("p must be 1, 2 or 4")
        if self.tau_num <= 0 or self.tau_log2_den < 0:
            raise ValueError("tau must be a positive dyadic rational")
        if self.delta_q < 1:
            raise ValueError("delta must be at least one fixed-point unit")
        if self.eviction not in ("default", "densest", "mandatory_source"):
            raise ValueError("eviction must be 'default', 'densest' or 'mandatory_source'")
        if self.sequential and (self.eviction != "default" or self.kv_descriptor):
            raise ValueError("the sequential variant combines only with source_order and refresh_base")

    @property
    def tau(self) -> float:
        return self.tau_num / float(1 << self.tau_log2_den)


@dataclass
class BankState:
    """One (layer, head) bank (Eq. 4): exact keys/values, cached density rho,
    frozen baseline b, provenance, and the per-head budget M.  Row s is slot s."""

    budget: int
    K: np.ndarray      # (m, d) keys as float64 (exact copies of the stored keys)
    V: np.ndarray      # (m, d) values, moved unchanged with their keys
    rho: np.ndarray    # (m,) int64, Q23 current density
    base: np.ndarray   # (m,) int64, Q23 frozen insertion baseline
    prov: np.ndarray   # (m,) int64, (block_id << 32) | source index

    @property
    def m(self) -> int:
        return int(self.K.shape[0])

    @classmethod
    def empty(cls, budget: int, d: int, v_dtype=np.float32, dv: Optional[int] = None) -> "BankState":
        dv = d if dv is None else dv
        return cls(budget=int(budget), K=np.zeros((0, d), np.float64),
                   V=np.zeros((0, dv), v_dtype), rho=np.zeros(0, np.int64),
                   base=np.zeros(0, np.int64), prov=np.zeros(0, np.int64))

    def copy(self) -> "BankState":
        return BankState(self.budget, self.K.copy(), self.V.copy(), self.rho.copy(),
                         self.base.copy(), self.prov.copy())


@dataclass
class HeadRecord:
    """Per-head intermediates of one update (for parity checks and logging)."""

    pi: np.ndarray                 # candidate order (source indices), length N
    score_q: Optional[np.ndarray]  # S_x of C6 in source order, or None for an empty bank
    score_exp: int                 # E of C6 (0 for an empty bank)
    first_cross: np.ndarray        # per old slot: smallest r with a violation, R+1 if none
    c: np.ndarray                  # violator counts c_r, r = 0..R (sequential: per step)
    e: int                         # e_{r*}
    rho_tilde: np.ndarray          # per old slot: rho + P(r*)
    evicted: np.ndarray            # old slots, ascending
    admitted: np.ndarray           # source indices, ascending
    admitted_slot: np.ndarray      # new slot of each admitted candidate (same order)


@dataclass
class UpdateRecord:
    r_star: int
    R: int
    heads: List[HeadRecord] = field(default_factory=list)
    # sequential variant (V6): per step, whether the j-th candidates entered
    steps: Optional[np.ndarray] = None


# ----------------------------------------------------------------------------
# Geometry and Soft-Riesz weight (Sec. 3.2-3.3, Eqs. 2-3; Supp. B)
# ----------------------------------------------------------------------------

def pair_d2(A: np.ndarray, B: np.ndarray) -> np.ndarray:
    """Squared Euclidean distances |a_i - b_j|^2 via the Gram expansion (C1).

    Exact in float64 for keys on the 1/64 grid (C0): each partial sum is an
    integer multiple of 2^-12 far below 2^53, so the BLAS order is irrelevant."""
    A = np.asarray(A, np.float64)
    B = np.asarray(B, np.float64)
    na = np.einsum("ij,ij->i", A, A)
    nb = np.einsum("ij,ij->i", B, B)
    return na[:, None] + nb[None, :] - 2.0 * (A @ B.T)


def pair_d2_bruteforce(A: np.ndarray, B: np.ndarray) -> np.ndarray:
    """|a_i - b_j|^2 summed coordinate by coordinate (test pin for pair_d2)."""
    A = np.asarray(A, np.float64)
    B = np.asarray(B, np.float64)
    diff = A[:, None, :] - B[None, :, :]
    return (diff * diff).sum(axis=2)


def soft_riesz_weight(d2: np.ndarray, prm: Params) -> np.ndarray:
    """w = (eps + d2 / sigma^2)^-p with eps = 1 (Eq. 2), in binary32 per C2."""
    d2_32 = np.asarray(d2, np.float64).astype(np.float32)
    if not np.array_equal(d2_32.astype(np.float64), np.asarray(d2, np.float64)):
        raise ValueError("squared distance not exact in binary32: keys are off the contract grid")
    u = d2_32 * np.float32(2.0 ** (-prm.sigma2_log2))
    t = np.float32(1.0) + u
    if prm.p == 1:
        tp = t
    elif prm.p == 2:
        tp = t * t
    else:
        t2 = t * t
        tp = t2 * t2
    return (np.float32(1.0) / tp).astype(np.float32)


def weight_q23(d2: np.ndarray, prm: Params) -> np.ndarray:
    """W = RNE(w * 2^23) as int64 (C3)."""
    w = soft_riesz_weight(d2, prm)
    return np.rint(w.astype(np.float64) * Q23).astype(np.int64)


def density_from_scratch(K: np.ndarray, prm: Params) -> np.ndarray:
    """Phi_A(i) = sum_{j != i} W(k_i, k_j) over the indexed multiset A (Eq. 3)."""
    m = K.shape[0]
    if m == 0:
        return np.zeros(0, np.int64)
    W = weight_q23(pair_d2(K, K), prm)
    W[np.arange(m), np.arange(m)] = 0  # exclude j == i by index only
    return W.sum(axis=1)


def candidate_scores(bankK: np.ndarray, base: np.ndarray, Kc: np.ndarray, prm: Params):
    """Mean-normalised disturbance s_h(x) (Eq. 6) as the fixed-point proxy S_x of C6.

    Returns (S, E, s_real) with S int64 per candidate, E the common exponent and
    s_real = S * 2^(E - 23) / m (the score in real units, for reports)."""
    m = bankK.shape[0]
    w = soft_riesz_weight(pair_d2(bankK, Kc), prm)                    # (m, N) fp32
    inv = (float(Q23) / np.asarray(base, np.int64).astype(np.float64)).astype(np.float32)
    E = int(np.frexp(np.float64(inv.max()))[1])
    bs = np.ldexp(inv.astype(np.float64), 23 - E)                       # exact rescale
    A = np.rint(w.astype(np.float64) * bs[:, None])                    # exact product, one RNE
    S = A.astype(np.int64).sum(axis=0)
    s_real = S.astype(np.float64) * 2.0 ** (E - 23) / m
    return S, E, s_real


# ----------------------------------------------------------------------------
# Online bank update for one layer (Sec. 3.4; Supp. C, Algorithm 1)
# ----------------------------------------------------------------------------

def _violates(rho_tilde: np.ndarray, base: np.ndarray, prm: Params) -> np.ndarray:
    """g_i(r) = rho~_i(r) / b_i >= tau (Eqs. 8-9), as the exact product test of C7."""
    return (rho_tilde << prm.tau_log2_den) >= prm.tau_num * base


def update_layer(heads: Sequence[BankState], cand_K: Sequence[np.ndarray],
                 cand_V: Sequence[np.ndarray], block_id: int, prm: Params):
    """One DensityKV update of a layer whose heads share the admitted prefix length.

    ``heads`` holds the per-head banks of one layer (or a single head for the
    independent per-head variant); ``cand_K[h]``/``cand_V[h]`` are the N
    candidates of head h in source order.  Returns (new banks, UpdateRecord)."""
    H = len(heads)
    if H == 0:
        raise ValueError("need at least one head")
    N = int(cand_K[0].shape[0])
    if any(int(k.shape[0]) != N for k in cand_K):
        raise ValueError("every head receives the same number of candidates")
    if N >= (1 << 13):
        raise ValueError("at most 8191 candidates per block")
    if prm.sequential:
        return _update_layer_sequential(heads, cand_K, cand_V, block_id, prm)
    # Prefix lengths tested: 0 <= r <= min(N, M) (Eq. 11).
    R = min(N, min(h.budget for h in heads))
    Kc64 = [np.asarray(k, np.float64) for k in cand_K]

    def desc(K, V):
        """Retention descriptor: the key, or [key; value] (V5)."""
        K = np.asarray(K, np.float64)
        return np.hstack([K, np.asarray(V, np.float64)]) if prm.kv_descriptor else K

    Dc = [desc(Kc64[h], cand_V[h]) for h in range(H)]                  # candidate descriptors
    Db = [desc(heads[h].K, heads[h].V) for h in range(H)]              # bank descriptors

    # ---- Step 1: per-head candidate order (Eq. 6-7; Alg. 1) ----------------
    def order_of(h):
        bank = heads[h]
        if bank.m == 0:
            # Empty bank: source-ordered candidates (Alg. 1, first branch).
            return np.arange(N, dtype=np.int64), (None, 0)
        S, E, _ = candidate_scores(Db[h], bank.base, Dc[h], prm)
        if prm.source_order:
            return np.arange(N, dtype=np.int64), (S, E)                     # V1
        return np.argsort(S, kind="stable").astype(np.int64), (S, E)       # ties: source order

    step1 = list(HEAD_MAP(order_of, range(H)))
    orders = [o for o, _ in step1]
    scores = [sc for _, sc in step1]

    # ---- Step 2: violators c_r for every tested prefix, shared r* (Eqs. 8-11)
    def prefix_of(h):
        bank, pi = heads[h], orders[h]
        m = bank.m
        if m == 0:
            P = np.zeros((0, R + 1), np.int64)
        else:
            Wc = weight_q23(pair_d2(Db[h], Dc[h][pi[:R]]), prm)        # (m, R)
            # Column-wise cumulative sums give every prefix contribution at once
            # (Supp. C, "Decision granularity versus computational tiling").
            P = np.concatenate([np.zeros((m, 1), np.int64), np.cumsum(Wc, axis=1)], axis=1)
        c = np.zeros(R + 1, np.int64)
        for r in range(R + 1):                     # each tested prefix length
            c[r] = np.count_nonzero(_violates(bank.rho + P[:, r], bank.base, prm))
        fc = np.full(m, R + 1, np.int64)
        for i in range(m):                         # first r at which state i violates
            hit = np.nonzero(_violates(bank.rho[i] + P[i, :], bank.base[i], prm))[0]
            if hit.size:
                fc[i] = hit[0]
        return P, c, fc

    step2 = list(HEAD_MAP(prefix_of, range(H)))
    prefix = [P for P, _, _ in step2]
    counts = [c for _, c, _ in step2]
    first_cross = [fc for _, _, fc in step2]

    def e_of(h: int, r: int) -> int:               # required evictions (Eq. 10)
        return max(0, heads[h].m + r - heads[h].budget)

    r_star = 0
    for r in range(R + 1):
        if all(counts[h][r] <= e_of(h, r) for h in range(H)):
            r_star = r                              # largest r feasible for every head

    # ---- Step 3: evict, commit, maintain densities (Eq. 12; Supp. C) --------
    def commit_of(h):
        bank, pi = heads[h], orders[h]
        m = bank.m
        e = e_of(h, r_star)
        rho_t = bank.rho + prefix[h][:, r_star] if m else np.zeros(0, np.int64)
        viol = _violates(rho_t, bank.base, prm)
        if prm.eviction == "densest":
            viol = np.zeros(m, bool)                                    # V3: no mandatory set
        mandatory = np.nonzero(viol)[0]
        evict = list(mandatory)
        if len(evict) < e:
            rest = np.nonzero(~viol)[0]
            if prm.eviction == "mandatory_source":
                # V4: admission order (provenance), then slot
                key_order = np.lexsort((rest, bank.prov[rest]))
            else:
                # decreasing rho~(r*); ties: earlier admission (provenance), then slot
                key_order = np.lexsort((rest, bank.prov[rest], -rho_t[rest]))
            evict.extend(rest[key_order[: e - len(evict)]])
        evicted = np.array(sorted(int(s) for s in evict), np.int64)
        admitted = np.sort(pi[:r_star])

        ev_mask = np.zeros(m, bool)
        ev_mask[evicted] = True
        surv = np.nonzero(~ev_mask)[0]
        Kc, Vc = Kc64[h], np.asarray(cand_V[h])
        Dbh, Dch = Db[h], Dc[h]

        # Exact density maintenance for survivors.
        rho_surv = bank.rho[surv].copy()
        if surv.size and admitted.size:
            rho_surv += weight_q23(pair_d2(Dbh[surv], Dch[admitted]), prm).sum(axis=1)
        if surv.size and evicted.size:
            rho_surv -= weight_q23(pair_d2(Dbh[surv], Dbh[evicted]), prm).sum(axis=1)

        # New states: density over the final bank (co-admitted included), frozen.
        if admitted.size:
            rho_new = np.zeros(admitted.size, np.int64)
            if surv.size:
                rho_new += weight_q23(pair_d2(Dch[admitted], Dbh[surv]), prm).sum(axis=1)
            rho_new += density_from_scratch(Dch[admitted], prm)
            base_new = np.maximum(rho_new, prm.delta_q)
        else:
            rho_new = np.zeros(0, np.int64)
            base_new = np.zeros(0, np.int64)

        # Commit layout (C10).
        m_new = m - evicted.size + admitted.size
        d = bank.K.shape[1] if m else Kc.shape[1]
        size = max(m, m_new)
        K = np.zeros((size, d), np.float64)
        V = np.zeros((size,) + Vc.shape[1:], Vc.dtype)
        rho = np.zeros(size, np.int64)
        base = np.zeros(size, np.int64)
        prov = np.zeros(size, np.int64)
        occupied = np.zeros(size, bool)
        K[surv], V[surv] = bank.K[surv], bank.V[surv]
        rho[surv], base[surv], prov[surv] = rho_surv, bank.base[surv], bank.prov[surv]
        occupied[surv] = True
        holes = list(evicted)
        slots = []
        for k, x in enumerate(admitted):
            s = int(holes[k]) if k < len(holes) else m + (k - len(holes))
            slots.append(s)
            K[s], V[s] = Kc[x], Vc[x]
            rho[s], base[s] = rho_new[k], base_new[k]
            prov[s] = (int(block_id) << 32) | int(x)
            occupied[s] = True
        if len(holes) > admitted.size:
            low_holes = [s for s in range(m_new) if not occupied[s]]
            movers = [s for s in range(m_new, size) if occupied[s]]
            assert len(low_holes) == len(movers)
            for dst, src in zip(low_holes, movers):
                K[dst], V[dst] = K[src], V[src]
                rho[dst], base[dst], prov[dst] = rho[src], base[src], prov[src]
        if prm.refresh_base:
            base = np.maximum(rho, prm.delta_q)                         # V2
        nb = BankState(bank.budget, K[:m_new].copy(), V[:m_new].copy(), rho[:m_new].copy(),
                       base[:m_new].copy(), prov[:m_new].copy())
        S, E = scores[h]
        return nb, HeadRecord(pi=pi, score_q=S, score_exp=E, first_cross=first_cross[h],
                              c=counts[h], e=e, rho_tilde=rho_t, evicted=evicted,
                              admitted=admitted, admitted_slot=np.array(slots, np.int64))

    step3 = list(HEAD_MAP(commit_of, range(H)))
    record = UpdateRecord(r_star=r_star, R=R, heads=[hr for _, hr in step3])
    new_heads = [nb for nb, _ in step3]
    return new_heads, record


def _update_layer_sequential(heads: Sequence[BankState], cand_K: Sequence[np.ndarray],
                             cand_V: Sequence[np.ndarray], block_id: int, prm: Params):
    """Within-block sequential competition (V6), one candidate per step."""
    H, N = len(heads), int(cand_K[0].shape[0])
    Kc64 = [np.asarray(k, np.float64) for k in cand_K]
    empty = [heads[h].m == 0 for h in range(H)]
    # the empty-bank rule for the heads that start empty (C12, through the default path)
    start = {}
    for h in range(H):
        if empty[h]:
            nb, rec1 = update_layer([heads[h]], [cand_K[h]], [cand_V[h]], block_id,
                                    Params(prm.sigma2_log2, prm.p, prm.tau_num, prm.tau_log2_den, prm.delta_q,
                                           refresh_base=prm.refresh_base))
            start[h] = (nb[0], rec1.heads[0])
    # candidate order fixed at the start of the block (C6 / V1)
    orders, scores = [], []
    for h in range(H):
        if empty[h]:
            orders.append(np.arange(N, dtype=np.int64))
            scores.append((None, 0))
            continue
        S, E, _ = candidate_scores(heads[h].K, heads[h].base, Kc64[h], prm)
        orders.append(np.arange(N, dtype=np.int64) if prm.source_order
                      else np.argsort(S, kind="stable").astype(np.int64))
        scores.append((S, E))
    # working banks: slots [0, m), capacity M
    work = []
    for h in range(H):
        b = heads[h]
        cap = max(b.budget, b.m)
        d = b.K.shape[1] if b.m else Kc64[h].shape[1]
        Vc = np.asarray(cand_V[h])
        K = np.zeros((cap, d), np.float64)
        V = np.zeros((cap,) + Vc.shape[1:], Vc.dtype)
        K[:b.m], V[:b.m] = b.K, b.V
        rho, base, prov = (np.zeros(cap, np.int64) for _ in range(3))
        rho[:b.m], base[:b.m], prov[:b.m] = b.rho, b.base, b.prov
        work.append(dict(K=K, V=V, rho=rho, base=base, prov=prov, m=b.m, released=set(), entered=[]))
    live = [h for h in range(H) if not empty[h]]
    steps = np.zeros(N, bool)
    nviol = np.zeros((H, N), np.int64)   # violators of every head at every step (record only)
    for j in range(N):
        tests = {}
        ok = True
        for h in live:
            w, x = work[h], int(orders[h][j])
            m = w["m"]
            W = weight_q23(pair_d2(w["K"][:m], Kc64[h][x:x + 1]), prm)[:, 0]
            rt = w["rho"][:m] + W
            viol = np.nonzero(_violates(rt, w["base"][:m], prm))[0]
            e = max(0, m + 1 - heads[h].budget)
            tests[h] = (x, W, rt, viol, e)
            nviol[h, j] = viol.size
            ok = ok and viol.size <= e
        if not ok or not live:
            continue
        steps[j] = True
        for h in live:
            w = work[h]
            x, W, rt, viol, e = tests[h]
            m = w["m"]
            if viol.size:
                ev = int(viol[0])
            elif e == 1:
                slots = np.arange(m)
                ev = int(slots[np.lexsort((slots, w["prov"][:m], -rt))[0]])  # C9 ties
            else:
                ev = -1
            surv = np.array([s for s in range(m) if s != ev], np.int64)
            if ev >= 0 and surv.size:
                Wev = weight_q23(pair_d2(w["K"][surv], w["K"][ev:ev + 1]), prm)[:, 0]
            else:
                Wev = np.zeros(surv.size, np.int64)
            w["rho"][surv] = rt[surv] - Wev
            rho_x = int(W[surv].sum())
            t = ev if ev >= 0 else m
            if ev >= 0:
                if (int(w["prov"][ev]) >> 32) != int(block_id):
                    w["released"].add(ev)          # an old state left its slot
            else:
                w["m"] = m + 1
            w["K"][t], w["V"][t] = Kc64[h][x], np.asarray(cand_V[h])[x]
            w["rho"][t], w["base"][t] = rho_x, max(rho_x, prm.delta_q)
            w["prov"][t] = (int(block_id) << 32) | x
    record = UpdateRecord(r_star=int(steps.sum()), R=N, steps=steps)
    new_heads = []
    for h in range(H):
        if empty[h]:
            nb, hr = start[h]
            new_heads.append(nb)
            record.heads.append(hr)
            continue
        w, m = work[h], work[h]["m"]
        base = w["base"][:m].copy()
        if prm.refresh_base:
            base = np.maximum(w["rho"][:m], prm.delta_q)
        nb = BankState(heads[h].budget, w["K"][:m].copy(), w["V"][:m].copy(), w["rho"][:m].copy(), base,
                       w["prov"][:m].copy())
        new_heads.append(nb)
        fresh = (nb.prov >> 32) == int(block_id)
        admitted = np.sort((nb.prov[fresh] & 0xFFFFFFFF).astype(np.int64))
        S, E = scores[h]
        none = np.zeros(0, np.int64)
        record.heads.append(HeadRecord(pi=orders[h], score_q=S, score_exp=E, first_cross=none, c=nviol[h],
                                       e=0, rho_tilde=none, evicted=np.array(sorted(w["released"]), np.int64),
                                       admitted=admitted, admitted_slot=np.nonzero(fresh)[0].astype(np.int64)))
    return new_heads, record


# ----------------------------------------------------------------------------
# Native attention over the retained bank plus the local window
# ----------------------------------------------------------------------------

def attention(q: np.ndarray, k_bank: np.ndarray, v_bank: np.ndarray,
              k_win: np.ndarray, v_win: np.ndarray, scale: float) -> np.ndarray:
    """softmax(q K^T * scale) V over the concatenated [bank; window] keys, in float64.

    The logit is q^T k / sqrt(d_k) (Sec. 3.2); the backbone's native attention
    reads the bank together with the local window (Sec. 1, Fig. 1)."""
    K = np.concatenate([np.asarray(k_bank, np.float64), np.asarray(k_win, np.float64)], axis=0)
    V = np.concatenate([np.asarray(v_bank, np.float64), np.asarray(v_win, np.float64)], axis=0)
    s = (np.asarray(q, np.float64) @ K.T) * float(scale)
    s -= s.max(axis=1, keepdims=True)
    p = np.exp(s)
    p /= p.sum(axis=1, keepdims=True)
    return p @ V
