"""Keys off the 1/64 grid (needs an MI355X).

Real bf16 post-RoPE keys need not lie on the grid that makes every Gram exact;
the library accepts them, and its decisions then carry the fp32 rounding of the
Gram, so they are not compared with the oracle bit for bit.  What must still
hold is checked here on near-duplicate off-grid keys (where fp32 cancellation
can round a squared distance below zero):

* the per-pair weight never exceeds eps^-p = 1, i.e. W <= 2^23, also for
  squared distances the rounding pushed below zero;
* after every update: occupancy within budget, one r* per group, eviction count
  max(0, m + r* - M), unique provenance, every retained key and value equal to
  the row it was admitted with, baselines at least delta, densities in
  [0, 2^23 (m - 1)], and every candidate score within [0, 2^23 m].
"""

import numpy as np
import pytest

torch = pytest.importorskip("torch")

pytestmark = pytest.mark.gpu

from paper_2608_27922_amd import api  # noqa: E402


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    api.lib()


def test_weight_of_negative_squared_distance_is_capped():
    d2 = torch.tensor([-3.0, -0.5, -1e-3, 0.0, 1e-3, 64.0], device="cuda")
    for p in (1, 2, 4):
        w = api.pair_weight_q23(d2, api.Params(sigma2_log2=6, p=p)).cpu().numpy()
        assert w.max() <= 1 << 23
        assert (w[:4] == 1 << 23).all(), w


@pytest.mark.parametrize("d,gs", [(128, 4), (64, 1)])
def test_offgrid_near_duplicates_keep_invariants(d, gs):
    rng = np.random.default_rng(40 + d)
    B, M, N = 8, 1500, 700
    bank = api.Bank(B, M, d, dtype=torch.bfloat16, group_size=gs)
    prm = api.Params(sigma2_log2=6 if d == 128 else 5)
    ws = api.alloc_workspace(bank, max(M, N))
    centres = rng.standard_normal((B, 16, d)) * 0.3
    hist_k, hist_v = [], []
    for t in range(5):
        n = M if t == 0 else N
        z = rng.integers(0, 16, (B, n))
        x = centres[np.arange(B)[:, None], z] + 0.3 * rng.standard_normal((B, n, d))
        if t > 0:   # a third of the block: near-duplicates (1e-3 perturbations) of bank keys
            k = n // 3
            src = bank.k[:, :k].float().cpu().numpy()
            x[:, :k] = src + 1e-3 * rng.standard_normal((B, k, d))
        K = torch.from_numpy(x.astype(np.float32)).to(torch.bfloat16).cuda().contiguous()
        V = torch.from_numpy(rng.standard_normal((B, n, d)).astype(np.float32)).to(torch.bfloat16).cuda()
        hist_k.append(K)
        hist_v.append(V)
        m_prev = bank.occupancy.long().clone()
        out = api.UpdateOut(bank, n, trace=True)
        api.update_bank(bank, K, V, t, prm, workspace=ws, out=out)
        torch.cuda.synchronize()
        occ = bank.occupancy.long()
        budget = bank.budget.long()
        rs = out.r_star.long().repeat_interleave(gs)
        assert torch.all(occ <= budget), f"block {t}: occupancy above budget"
        e = torch.clamp(m_prev + rs - budget, min=0)
        assert torch.equal(out.n_evicted.long(), e), f"block {t}: eviction count"
        assert torch.equal(occ, m_prev + rs - e), f"block {t}: occupancy"
        sq = out.score_q[:, :n]
        assert bool(torch.all(sq >= 0)) and bool(torch.all(sq <= (1 << 23) * m_prev[:, None].clamp(min=1))), \
            f"block {t}: a score term exceeds 2^23"
        ar = torch.arange(M, device="cuda")
        live = ar[None, :] < occ[:, None]
        rho, base = bank.rho[live], bank.base[live]
        mm = occ[:, None].expand(B, M)[live]
        assert bool(torch.all(rho >= 0)) and bool(torch.all(rho <= (1 << 23) * (mm - 1))), f"block {t}: density range"
        assert bool(torch.all(base >= prm.delta_q)), f"block {t}: baseline below delta"
        prov = torch.where(live, bank.prov, torch.full_like(bank.prov, -1))
        sp = torch.sort(prov, 1).values
        assert not bool(torch.any((sp[:, 1:] == sp[:, :-1]) & (sp[:, 1:] >= 0))), f"block {t}: duplicate provenance"
        blk, sidx = (bank.prov >> 32)[live], (bank.prov & 0xFFFFFFFF)[live]
        bidx = torch.arange(B, device="cuda")[:, None].expand(B, M)[live]
        for s in range(t + 1):
            sel = blk == s
            assert torch.equal(bank.k[live][sel], hist_k[s][bidx[sel], sidx[sel]]), f"block {t}: retained key"
            assert torch.equal(bank.v[live][sel], hist_v[s][bidx[sel], sidx[sel]]), f"block {t}: retained value"
        assert bool(torch.all((blk >= 0) & (blk <= t))), f"block {t}: provenance outside the history"
    assert int(occ.min()) > 0
