"""Exact rational brute force of the DensityKV update, for tiny banks (test pin only).

Independent of ``oracle/``: it works in ``fractions.Fraction`` and, for every
tested prefix length r, builds the hypothetical multiset bank (+) P_r and
recomputes each historical state's density from its definition (Eq. 3),
instead of using cached densities and cumulative sums.  After the commit every
density is recomputed from scratch over the final bank.  This is the paper's
update (Sec. 3.4, Eqs. 5-12; Supp. C, Algorithm 1) evaluated in real
arithmetic, so any oracle decision on a well-separated tiny case must agree
with it, and every oracle fixed-point density must round to it.

The policy ablations of Table 1(b) (Supp. E) are options of ``update``:
source-order candidates, refreshed baselines, densest-only eviction and
mandatory + source-order eviction (source order of a bank state = its
admission order, i.e. ascending provenance).  ``update_sequential`` is the
within-block competition variant, one candidate per step for a whole layer.
"""

from fractions import Fraction as F


def weight(a, b, sigma2, p):
    """(1 + |a - b|^2 / sigma^2)^-p with eps = 1 (Eq. 2)."""
    d2 = sum((F(x) - F(y)) ** 2 for x, y in zip(a, b))
    return F(1) / (F(1) + d2 / F(sigma2)) ** p


def phi(keys, i, sigma2, p):
    """Soft-Riesz density of entry i in the indexed multiset ``keys`` (Eq. 3)."""
    return sum((weight(keys[i], keys[j], sigma2, p) for j in range(len(keys)) if j != i), F(0))


def update(bank, cands, M, sigma2=1, p=1, tau=F(2), delta=F(1, 10 ** 6), block_id=1, r_star=None,
           source_order=False, refresh_base=False, eviction="default"):
    """bank: list of dicts {key, b, prov}; cands: list of key tuples (source order).

    ``r_star`` forces the admitted prefix length (a layer's shared r*); by default
    it is this bank's own largest feasible r.  Returns (new_bank, info) where
    new_bank lists dicts {key, rho, b, prov} in the commit layout
    survivors-in-place / admitted-into-holes-then-appended."""
    N, m = len(cands), len(bank)
    R = min(N, M)
    keys = [s["key"] for s in bank]
    if m == 0:
        pi = list(range(N))
        scores = None
    else:
        scores = [sum((weight(k, x, sigma2, p) / s["b"] for k, s in zip(keys, bank)), F(0)) / m
                  for x in cands]
        pi = list(range(N)) if source_order else sorted(range(N), key=lambda x: (scores[x], x))
    c, proj = [], []
    for r in range(R + 1):
        hyp = keys + [cands[pi[j]] for j in range(r)]
        pr = [phi(hyp, i, sigma2, p) for i in range(m)]
        proj.append(pr)
        c.append(sum(1 for i in range(m) if pr[i] / bank[i]["b"] >= tau))
    e = [max(0, m + r - M) for r in range(R + 1)]
    # first tested prefix length at which each state violates, R + 1 if none
    first = [next((r for r in range(R + 1) if proj[r][i] / bank[i]["b"] >= tau), R + 1) for i in range(m)]
    feas = [r for r in range(R + 1) if c[r] <= e[r]]
    if r_star is None:
        r_star = max(feas) if feas else 0
    pr = proj[r_star]
    viol = [i for i in range(m) if pr[i] / bank[i]["b"] >= tau]
    evict = [] if eviction == "densest" else list(viol)
    if eviction == "mandatory_source":
        fill_key = lambda i: (bank[i]["prov"], i)
    else:
        fill_key = lambda i: (-pr[i], bank[i]["prov"], i)
    rest = sorted((i for i in range(m) if i not in evict), key=fill_key)
    evict += rest[: max(0, e[r_star] - len(evict))]
    evict = sorted(evict)
    admitted = sorted(pi[:r_star])
    # commit layout
    slots = {i: dict(bank[i]) for i in range(m) if i not in evict}
    holes = list(evict)
    for k, x in enumerate(admitted):
        s = holes[k] if k < len(holes) else m + k - len(holes)
        slots[s] = {"key": cands[x], "b": None, "prov": (block_id << 32) | x}
    m_new = m - len(evict) + len(admitted)
    low = [s for s in range(m_new) if s not in slots]
    high = sorted(s for s in slots if s >= m_new)
    for dst, src in zip(low, high):
        slots[dst] = slots.pop(src)
    new_bank = [slots[s] for s in range(m_new)]
    fk = [s["key"] for s in new_bank]
    for i, s in enumerate(new_bank):
        s["rho"] = phi(fk, i, sigma2, p)
        if s["b"] is None or refresh_base:
            s["b"] = max(s["rho"], delta)
    info = dict(r_star=r_star, pi=pi, scores=scores, c=c, e=e, evicted=evict, admitted=admitted,
                violators=viol, projected=pr, first_violation=first)
    return new_bank, info


def build(cands, M, **kw):
    """A bank produced by the empty-bank rule from ``cands``."""
    bank, _ = update([], cands, M, **kw)
    return bank


def update_sequential(banks, cands, Ms, sigma2=1, p=1, tau=F(2), delta=F(1, 10 ** 6), block_id=1,
                      source_order=False, refresh_base=False):
    """Within-block sequential competition for a layer (Supp. E): step j offers the
    j-th candidate of every head (order fixed at the start of the block) to that
    head's current bank; every density is recomputed from its definition over the
    hypothetical bank.  The step is taken iff every head whose bank was not empty
    at the start has at most e = max(0, m + 1 - M) violators; then each such head
    releases its violator, or with none and e = 1 its densest state (ties: earlier
    provenance, then slot), and the candidate takes that slot (else the next one)
    with baseline max(Phi over the bank it enters, delta).  Heads that start empty
    take the empty-bank rule.  Returns (new banks, info)."""
    H, N = len(banks), len(cands[0])
    out, orders, live = [None] * H, [None] * H, []
    for h in range(H):
        if not banks[h]:
            out[h] = update([], cands[h], Ms[h], sigma2=sigma2, p=p, tau=tau, delta=delta, block_id=block_id,
                            refresh_base=refresh_base)[0]
            continue
        live.append(h)
        keys = [s["key"] for s in banks[h]]
        sc = [sum((weight(k, x, sigma2, p) / s["b"] for k, s in zip(keys, banks[h])), F(0)) / len(keys)
              for x in cands[h]]
        orders[h] = list(range(N)) if source_order else sorted(range(N), key=lambda x: (sc[x], x))
    work = {h: [{"key": s["key"], "b": s["b"], "prov": s["prov"]} for s in banks[h]] for h in live}
    steps = []
    counts = {h: [] for h in live}          # violators of every live head at every step
    released = {h: set() for h in live}     # slots whose pre-block occupant was released
    for j in range(N):
        tests, ok = {}, bool(live)
        for h in live:
            bank, x = work[h], orders[h][j]
            hyp = [s["key"] for s in bank] + [cands[h][x]]
            pr = [phi(hyp, i, sigma2, p) for i in range(len(bank))]
            viol = [i for i in range(len(bank)) if pr[i] / bank[i]["b"] >= tau]
            e = max(0, len(bank) + 1 - Ms[h])
            tests[h] = (x, pr, viol, e)
            counts[h].append(len(viol))
            ok = ok and len(viol) <= e
        steps.append(ok)
        if not ok:
            continue
        for h in live:
            x, pr, viol, e = tests[h]
            bank = work[h]
            if viol:
                t = viol[0]
            elif e == 1:
                t = min(range(len(bank)), key=lambda i: (-pr[i], bank[i]["prov"], i))
            else:
                t = len(bank)
                bank.append(None)
            if t < len(bank) and bank[t] is not None and bank[t]["prov"] >> 32 != block_id:
                released[h].add(t)
            bank[t] = {"key": cands[h][x], "b": None, "prov": (block_id << 32) | x}
            bank[t]["b"] = max(phi([s["key"] for s in bank], t, sigma2, p), delta)
    for h in live:
        keys = [s["key"] for s in work[h]]
        for i, s in enumerate(work[h]):
            s["rho"] = phi(keys, i, sigma2, p)
            if refresh_base:
                s["b"] = max(s["rho"], delta)
        out[h] = work[h]
    return out, dict(steps=steps, orders=orders, counts=counts,
                     released={h: sorted(released[h]) for h in live})
