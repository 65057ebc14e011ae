"""Full-size runs of the three 30-layer x 12-head rollout workloads: all 360 banks
updated by one launch per block, as the library is used.  Needs an MI355X.

Parity with the oracle: sampled layers of each run (layers 0 and 29 of the
rollout, one layer of the other two) are drawn from the seeded input generator,
and every block of the run at its stated length (20, 80 and 160 blocks) is
compared: after every block the device results for the sampled layer's 12 banks
(candidate order, scores, first crossings, projected densities, eviction and
admission lists, and the committed bank bytes) must hash to the digests the
oracle wrote for the same inputs (tests/golden/make_rollout_digests.py; the
oracle needs minutes per block at these budgets, so it is not rerun here).
After the last block, sampled query rows of the bank attention are compared
with the oracle's fp64 attention within the bf16 tolerance.

Properties checked on every one of the 360 banks after every block, at full
size: occupancy within budget; r* shared inside each layer; the eviction count
equals max(0, m + r* - M); the order sorts the score keys; the admitted set is
the first r* of the order; every violator at r* is evicted and every other
evicted state is at least as dense as every kept one; the violation flags agree
with the projected densities; the maintained density equals the density
recomputed from scratch; the growth bound rho < tau b; the baseline floor; and
every retained token carries the key and value it was admitted with (checked
through 64-bit fingerprints of every admitted row, so that the history of a
160-block run need not stay in memory).  The layers that are not compared with
the oracle draw their tokens on the device from a seeded torch generator.
"""

import json
import os

import numpy as np
import pytest

torch = pytest.importorskip("torch")

pytestmark = pytest.mark.gpu

from golden.make_rollout_digests import RUNS, attention_rows, cases, digest, layer_block  # noqa: E402
from gpu_util import attention_error, dev, host  # noqa: E402
from paper_2608_27922_amd import api, synth  # noqa: E402

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    api.lib()


def _bank_entry(bank, out, b, m_before, n):
    """Digests of one bank's update; the order, scores, first crossings and
    projected densities only when the update was asked for them (trace)."""
    m = int(bank.occupancy[b])
    ne, na = int(out.n_evicted[b]), int(out.n_admitted[b])
    i64 = lambda t: t.cpu().numpy().astype(np.int64)
    trace = {} if out.first_cross is None else {
        "order": digest(out.order[b, :n].cpu().numpy(), np.int32),
        "score_q": digest(i64(out.score_q[b, :n]), np.int64),
        "first_cross": digest(out.first_cross[b, :m_before].cpu().numpy(), np.int32),
        "rho_tilde": digest(i64(out.rho_tilde[b, :m_before]), np.int64),
    }
    return {
        "m_before": m_before, "m_after": m, "n_evicted": ne, "n_admitted": na, **trace,
        "evicted": digest(out.evicted[b, :ne].cpu().numpy(), np.int32),
        "admitted": digest(out.admitted[b, :na].cpu().numpy(), np.int32),
        "prov": digest(i64(bank.prov[b, :m]), np.int64), "rho": digest(i64(bank.rho[b, :m]), np.int64),
        "base": digest(i64(bank.base[b, :m]), np.int64),
        "knorm": digest(bank.knorm[b, :m].cpu().numpy(), np.float32),
        "k": digest(host(bank.k[b, :m]), np.float32), "v": digest(host(bank.v[b, :m]), np.float32),
    }


class RowPrints:
    """64-bit fingerprints of every candidate row of every block: a fixed random
    linear form over the row's 32-bit words, so that a retained row can be
    checked against the row it was admitted with without keeping the history."""

    def __init__(self, d, seed=5):
        g = torch.Generator(device="cuda")
        g.manual_seed(seed)
        self.w = torch.randint(1, 1 << 31, (d // 2,), generator=g, device="cuda", dtype=torch.int64)
        self.k, self.v = [], []

    def of(self, rows):
        """[..., d] bf16 -> [...] int64."""
        words = rows.contiguous().view(torch.int32).to(torch.int64)
        return (words * self.w).sum(-1)

    def add(self, K, V):
        self.k.append(self.of(K))
        self.v.append(self.of(V))

    def check(self, bank, occupied, ctx, chunk=40):
        B, Mcap = bank.B, bank.Mcap
        hk, hv = torch.stack(self.k), torch.stack(self.v)      # [T, B, N]
        for b0 in range(0, B, chunk):
            b1 = min(B, b0 + chunk)
            occ = occupied[b0:b1]
            blk = (bank.prov[b0:b1] >> 32)[occ]
            sidx = (bank.prov[b0:b1] & 0xFFFFFFFF)[occ]
            bidx = torch.arange(b0, b1, device="cuda")[:, None].expand(b1 - b0, Mcap)[occ]
            assert torch.equal(self.of(bank.k[b0:b1])[occ], hk[blk, bidx, sidx]), \
                f"{ctx}: a retained key differs from its admitted key"
            assert torch.equal(self.of(bank.v[b0:b1])[occ], hv[blk, bidx, sidx]), \
                f"{ctx}: a retained value differs from its admitted value"


def _properties(bank, out, prm, m_prev, base_prev, prints, gs, N, ctx):
    occ = bank.occupancy.long()
    budget = bank.budget.long()
    rs = out.r_star.long().repeat_interleave(gs)
    assert torch.all(occ <= budget), f"{ctx}: occupancy above budget"
    assert torch.equal(out.n_admitted.long(), rs), f"{ctx}: admitted count differs from the group's r*"
    e = torch.clamp(m_prev + rs - budget, min=0)
    assert torch.equal(out.n_evicted.long(), e), f"{ctx}: eviction count differs from max(0, m + r* - M)"
    assert torch.equal(occ, m_prev + rs - e), f"{ctx}: occupancy differs from m + r* - e"
    if out.first_cross is not None:
        _trace_properties(bank, out, prm, m_prev, base_prev, rs, N, ctx)
    _bank_properties(bank, prm, prints, N, ctx)


def _trace_properties(bank, out, prm, m_prev, base_prev, rs, N, ctx):
    """The order, the admitted prefix and the eviction rule, from the trace outputs."""
    B, Mcap = bank.B, bank.Mcap
    ar = torch.arange(Mcap, device="cuda")
    # order sorts the score keys (S << 13 | x) ascending; empty banks keep source order
    src = torch.arange(N, device="cuda")
    keys = (out.score_q[:, :N] << 13) | src
    sk = torch.gather(keys, 1, out.order[:, :N].long())
    assert bool(torch.all(sk[:, 1:] > sk[:, :-1])), f"{ctx}: order does not sort the score keys"
    assert torch.equal(torch.sort(out.order[:, :N], dim=1).values.long(), src.expand(B, N)), f"{ctx}: order not a permutation"
    # admitted set = first r* of the order
    first = torch.where(src[None, :] < rs[:, None], out.order[:, :N].long(), N)
    adm = torch.where(src[None, :] < rs[:, None], out.admitted[:, :N].long(), N)
    assert torch.equal(torch.sort(first, 1).values, adm), f"{ctx}: admitted set is not the order's prefix"

    # eviction rule on the old slots
    old = ar[None, :] < m_prev[:, None]
    viol_fc = (out.first_cross.long() <= rs[:, None]) & old
    ev_mask = torch.zeros(B, Mcap + 1, dtype=torch.bool, device="cuda")
    ev_idx = torch.where(ar[None, :] < out.n_evicted[:, None].long(), out.evicted.long(), Mcap)
    ev_mask.scatter_(1, ev_idx, True)
    ev_mask = ev_mask[:, :Mcap]
    assert bool(torch.all(ev_mask[viol_fc])), f"{ctx}: a violator at r* was not evicted"
    kept_nv = old & ~ev_mask & ~viol_fc
    fill = ev_mask & ~viol_fc
    neg = torch.iinfo(torch.int64).min
    kept_max = torch.where(kept_nv, out.rho_tilde, torch.full_like(out.rho_tilde, neg)).amax(1)
    fill_min = torch.where(fill, out.rho_tilde, torch.full_like(out.rho_tilde, torch.iinfo(torch.int64).max)).amin(1)
    assert bool(torch.all(fill_min >= kept_max)), f"{ctx}: a kept state is denser than an evicted one"
    # the first crossings (prefix-scan kernels) agree with the projected densities at r*
    # (fix-up kernel): violation at r* <=> 2^k rho~ >= T b
    viol_rt = ((out.rho_tilde << prm.tau_log2_den) >= prm.tau_num * base_prev) & old
    assert torch.equal(viol_rt, viol_fc), f"{ctx}: first crossings disagree with the projected densities"


def _bank_properties(bank, prm, prints, N, ctx):
    """Baselines, the growth bound, exact maintenance, provenance and retained rows."""
    B, Mcap = bank.B, bank.Mcap
    ar = torch.arange(Mcap, device="cuda")
    occ = bank.occupancy.long()
    occupied = ar[None, :] < occ[:, None]
    rho, base = bank.rho, bank.base
    assert bool(torch.all(base[occupied] >= prm.delta_q)), f"{ctx}: baseline below delta"
    assert bool(torch.all((rho[occupied] << prm.tau_log2_den) < prm.tau_num * base[occupied])), \
        f"{ctx}: growth bound rho < tau b violated"
    # exact maintenance: maintained rho == density recomputed from scratch
    z = torch.zeros(B, 1, bank.d, dtype=bank.dtype, device="cuda")
    _, _, dens = api.score(bank, z, z, prm, want_q=False, want_f32=False, want_density=True)
    assert torch.equal(dens[occupied], rho[occupied]), f"{ctx}: maintained density differs from recomputation"
    # provenance unique; each retained token holds the key/value it was admitted with
    prov = torch.where(occupied, bank.prov, torch.full_like(bank.prov, -1))
    sp = torch.sort(prov, 1).values
    dup = (sp[:, 1:] == sp[:, :-1]) & (sp[:, 1:] >= 0)
    assert not bool(torch.any(dup)), f"{ctx}: duplicate provenance inside a bank"
    blk = (bank.prov >> 32)[occupied]
    sidx = (bank.prov & 0xFFFFFFFF)[occupied]
    assert bool(torch.all((blk >= 0) & (blk < len(prints.k)) & (sidx < N))), f"{ctx}: provenance out of range"
    prints.check(bank, occupied, ctx)


def _golden(name, layer):
    """Oracle digests of (workload, sampled layer) over the workload's stated length."""
    stem = os.path.join(GOLDEN, f"rollout_{name}_L{layer}")
    if not os.path.exists(stem + ".json"):
        return None, None
    with open(stem + ".json") as f:
        return json.load(f), np.load(stem + "_attention.npy")


@pytest.mark.parametrize("name,layer", cases(), ids=[f"{n}-L{ly}" for n, ly in cases()])
def test_full_size_workload(name, layer):
    gold, ref_att = _golden(name, layer)
    if gold is None:
        pytest.skip(f"oracle digests for {name} layer {layer} not generated")
    cfg = synth.WORKLOADS[name]
    blocks, att_heads = gold["blocks"], gold["attention_heads"]
    assert gold["layer"] == layer and blocks == cfg.blocks, "digests of a shorter run"
    H, d, N, gs = cfg.heads, cfg.d, cfg.n_cand, cfg.group_size
    B = cfg.layers * H
    print(f"workload {name}: {B} banks, {blocks} blocks, sampled layer {layer}", flush=True)
    budgets = synth.budgets(cfg)
    assert [int(x) for x in budgets[layer * H:(layer + 1) * H]] == gold["budgets"]
    prm = api.Params(sigma2_log2=cfg.sigma2_log2)
    bank = api.Bank(B, int(budgets.max()), d, dtype=torch.bfloat16, group_size=gs,
                    budget=torch.from_numpy(budgets))
    ws = api.alloc_workspace(bank, N)
    streams = [synth.HeadStream(cfg, layer, h) for h in range(H)]
    prints = RowPrints(d)
    sl = slice(layer * H, (layer + 1) * H)
    for t in range(blocks):
        K = torch.empty(B, N, d, dtype=torch.bfloat16, device="cuda")
        V = torch.empty_like(K)
        for L in range(cfg.layers):
            if L != layer:
                K[L * H:(L + 1) * H], V[L * H:(L + 1) * H] = synth.torch_layer_block(cfg, L, t, N, "cuda")
        Kl, Vl = layer_block(cfg, streams, t)
        K[sl], V[sl] = dev(Kl, "bf16"), dev(Vl, "bf16")
        prints.add(K, V)
        m_prev = bank.occupancy.long().clone()
        base_prev = bank.base.clone()
        # odd blocks without the trace outputs: the update may then end its
        # crossing search after the first 1,024 ordered candidates
        out = api.UpdateOut(bank, N, trace=t % 2 == 0)
        api.update_bank(bank, K, V, t, prm, workspace=ws, out=out)
        torch.cuda.synchronize()
        ctx = f"{name} L{layer} block {t}" + ("" if t % 2 == 0 else " (no trace)")
        step = gold["steps"][t]
        for g, rs in enumerate(step["r_star"]):
            assert int(out.r_star[layer * H // gs + g]) == rs, f"{ctx}: r* of group {g}"
        for h in range(H):
            got = _bank_entry(bank, out, layer * H + h, int(m_prev[layer * H + h]), N)
            want = step["heads"][h]
            bad = [k for k in got if got[k] != want[k]]
            assert not bad, f"{ctx} head {h}: differs from the oracle in {bad}"
        _properties(bank, out, prm, m_prev, base_prev, prints, gs, N, ctx)
        del K, V, out
        print(f"  block {t}: r* {step['r_star'][:3]} occupancy {step['heads'][0]['m_after']} "
              f"evicted {sum(hh['n_evicted'] for hh in step['heads'])} ok", flush=True)
    q = torch.empty(B, cfg.n_query, d, dtype=torch.bfloat16, device="cuda")
    for L in range(cfg.layers):
        if L != layer:
            q[L * H:(L + 1) * H], _ = synth.torch_layer_block(cfg, L, blocks, cfg.n_query, "cuda")
    wk_all, wv_all = [], []
    for L in range(cfg.layers):
        k_, v_ = synth.torch_layer_block(cfg, L, blocks + 1, cfg.n_window, "cuda")
        wk_all.append(k_)
        wv_all.append(v_)
    wk, wv = torch.cat(wk_all).contiguous(), torch.cat(wv_all).contiguous()
    q[sl] = dev(np.stack([s.queries(blocks) for s in streams]), "bf16")
    wk[sl] = dev(np.stack([s.keys(blocks, cfg.n_window) for s in streams]), "bf16")
    wv[sl] = dev(np.stack([s.values(blocks, cfg.n_window) for s in streams]), "bf16")
    o = api.bank_attention(bank, q, wk, wv)
    rows = torch.from_numpy(attention_rows(cfg.n_query)).cuda()
    worst = 0.0
    for i, h in enumerate(att_heads):
        got = host(o[layer * H + h].index_select(0, rows))
        worst = max(worst, attention_error(got, ref_att[i]))
    assert torch.isfinite(o.float()).all(), "non-finite attention output"
    print(f"  attention: max row-normalised error {worst:.3e} over {len(att_heads)} heads x {rows.numel()} rows",
          flush=True)
    assert worst <= 2e-2


def test_interface_limits():
    """N = 8,191 candidates and a budget of 32,767 states (the interface maxima: the
    13-bit source index of the sort key and the 15-bit slot of the eviction key), two
    heads sharing the prefix: fills, partial admissions, mandatory and fill evictions,
    every block against the stored oracle digests plus the full-bank properties."""
    from golden.make_limit_digests import BLOCKS, TAU_NUM, block_inputs, limits_config
    path = os.path.join(GOLDEN, "limits.json")
    if not os.path.exists(path):
        pytest.skip("oracle digests for the interface limits not generated")
    with open(path) as f:
        gold = json.load(f)
    cfg = limits_config()
    H, d, N = cfg.heads, cfg.d, cfg.n_cand
    print(f"limits: {H} banks, N {N}, budget {cfg.budget}, {BLOCKS} blocks", flush=True)
    prm = api.Params(sigma2_log2=cfg.sigma2_log2, tau_num=TAU_NUM)
    bank = api.Bank(H, cfg.budget, d, dtype=torch.bfloat16, group_size=cfg.group_size)
    ws = api.alloc_workspace(bank, N)
    streams = [synth.HeadStream(cfg, 0, h) for h in range(H)]
    prints = RowPrints(d)
    for t in range(BLOCKS):
        bank_keys = [host(bank.k[h, :int(bank.occupancy[h])]) for h in range(H)]
        Kn, Vn = block_inputs(cfg, streams, t, bank_keys)
        K, V = dev(Kn, "bf16"), dev(Vn, "bf16")
        prints.add(K, V)
        m_prev = bank.occupancy.long().clone()
        base_prev = bank.base.clone()
        out = api.UpdateOut(bank, N, trace=True)
        api.update_bank(bank, K, V, t, prm, workspace=ws, out=out)
        torch.cuda.synchronize()
        ctx = f"limits block {t}"
        step = gold["steps"][t]
        assert int(out.r_star[0]) == step["r_star"][0], f"{ctx}: r*"
        for h in range(H):
            got = _bank_entry(bank, out, h, int(m_prev[h]), N)
            want = step["heads"][h]
            bad = [k for k in want if got[k] != want[k]]
            assert not bad, f"{ctx} head {h}: differs from the oracle in {bad}"
        _properties(bank, out, prm, m_prev, base_prev, prints, cfg.group_size, N, ctx)
        print(f"  block {t}: r* {step['r_star'][0]} occupancy {[int(x) for x in bank.occupancy.cpu()]} ok", flush=True)


def test_single_layer_sequential_full_size():
    """The within-block sequential competition at the size the benchmark times
    (12 banks in one group, budget 4,680, banks filled by the empty-bank rule,
    then 4,680 candidates with 30% near-duplicates offered one per step), as one
    update call: the number of taken steps and, per bank, the order, scores,
    released and admitted lists and the committed bank bytes must hash to the
    digests the oracle wrote for the same inputs
    (tests/golden/make_sequential_digests.py)."""
    path = os.path.join(GOLDEN, "sequential_single_layer.json")
    if not os.path.exists(path):
        pytest.skip("oracle digests for the sequential single_layer run not generated")
    with open(path) as f:
        ref = json.load(f)
    cfg = synth.WORKLOADS["single_layer"]
    H, M, N, d = cfg.heads, cfg.budget, cfg.n_cand, cfg.d
    print("sequential single_layer: build the case", flush=True)
    case = synth.single_update_case(cfg)
    bank = api.Bank(H, M, d, dtype=torch.bfloat16, group_size=cfg.group_size)
    api.update_bank(bank, dev(case["init_K"], "bf16"), dev(case["init_V"], "bf16"), 0,
                    api.Params(sigma2_log2=cfg.sigma2_log2))
    torch.cuda.synchronize()
    i64 = lambda t: t.cpu().numpy().astype(np.int64)
    for b in range(H):
        m = int(bank.occupancy[b])
        got = {"m": m, "rho": digest(i64(bank.rho[b, :m]), np.int64), "base": digest(i64(bank.base[b, :m]), np.int64),
               "prov": digest(i64(bank.prov[b, :m]), np.int64)}
        assert got == ref["init"][b], f"initial bank {b}"
    print("sequential single_layer: update", flush=True)
    prm = api.Params(sigma2_log2=cfg.sigma2_log2, flags=api.POLICY_SEQUENTIAL)
    out = api.UpdateOut(bank, N, trace=True)
    api.update_bank(bank, dev(case["seg_K"], "bf16"), dev(case["seg_V"], "bf16"), 1, prm, out=out)
    torch.cuda.synchronize()
    assert int(out.r_star[0].item()) == ref["steps_taken"]
    for b in range(H):
        m = int(bank.occupancy[b])
        ne, na = int(out.n_evicted[b]), int(out.n_admitted[b])
        got = {
            "m_after": m, "n_evicted": ne, "n_admitted": na,
            "order": digest(out.order[b, :N].cpu().numpy(), np.int32),
            "score_q": digest(i64(out.score_q[b, :N]), np.int64),
            "evicted": digest(out.evicted[b, :ne].cpu().numpy(), np.int32),
            "admitted": digest(out.admitted[b, :na].cpu().numpy(), np.int32),
            "prov": digest(i64(bank.prov[b, :m]), np.int64), "rho": digest(i64(bank.rho[b, :m]), np.int64),
            "base": digest(i64(bank.base[b, :m]), np.int64),
            "knorm": digest(bank.knorm[b, :m].cpu().numpy(), np.float32),
            "k": digest(host(bank.k[b, :m]), np.float32), "v": digest(host(bank.v[b, :m]), np.float32),
        }
        bad = [k for k in got if got[k] != ref["heads"][b][k]]
        assert not bad, f"bank {b}: {bad}"


def test_long_rollout_sequential_full_size():
    """The within-block sequential competition on layer 0 of the long rollout
    (12 banks in one group, budget 18,720, 4,680 candidates per block): blocks
    0-5 (block 0 fills the empty banks by the empty-bank rule, block 1 takes
    about 4,600 steps into banks of 4,680 states, later blocks take none on this
    input, every step tested against banks of 9,280 states).  The pairwise
    weights of the group (12 x 23,400^2 x 4 bytes) take the default workspace,
    one group per batch.  Per block, the number of taken
    steps and, per bank, the order, scores, released and admitted lists and the
    committed bank bytes must hash to the oracle's digests
    (tests/golden/make_sequential_digests.py)."""
    path = os.path.join(GOLDEN, "sequential_long_rollout_L0.json")
    if not os.path.exists(path):
        pytest.skip("oracle digests for the sequential long-rollout run not generated")
    with open(path) as f:
        ref = json.load(f)
    cfg = synth.WORKLOADS["long_rollout"]
    H, N, d = cfg.heads, cfg.n_cand, cfg.d
    budgets = synth.budgets(cfg)[:H]
    bank = api.Bank(H, int(budgets.max()), d, dtype=torch.bfloat16, group_size=cfg.group_size,
                    budget=torch.from_numpy(budgets))
    prm = api.Params(sigma2_log2=cfg.sigma2_log2, flags=api.POLICY_SEQUENTIAL)
    ws = api.alloc_workspace(bank, N, prm.flags)
    streams = [synth.HeadStream(cfg, 0, h) for h in range(H)]
    assert ref["blocks"] == len(ref["steps"])
    for t, step in enumerate(ref["steps"]):
        print(f"sequential long rollout: block {t}", flush=True)
        K, V = layer_block(cfg, streams, t)
        m_prev = [int(x) for x in bank.occupancy.cpu()]
        out = api.UpdateOut(bank, N, trace=True)
        api.update_bank(bank, dev(K, "bf16"), dev(V, "bf16"), t, prm, workspace=ws, out=out)
        torch.cuda.synchronize()
        assert int(out.r_star[0].item()) == step["steps_taken"], f"block {t}: steps taken"
        for b in range(H):
            got = _bank_entry(bank, out, b, m_prev[b], N)
            bad = [k for k in step["heads"][b] if got[k] != step["heads"][b][k]]
            assert not bad, f"block {t} bank {b}: differs from the oracle in {bad}"
        print(f"  block {t}: steps {step['steps_taken']} occupancy {[int(x) for x in bank.occupancy.cpu()][:4]} ok",
              flush=True)
