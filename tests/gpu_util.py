"""Helpers shared by the GPU parity tests: move seeded inputs to the device, mirror
the device banks into oracle BankStates, and compare the two bit for bit."""

import numpy as np
import torch

from oracle import BankState, Params as OParams, update_layer
from paper_2608_27922_amd import api

TORCH_DT = {"bf16": torch.bfloat16, "f32": torch.float32}


def dev(a: np.ndarray, dtype: str) -> torch.Tensor:
    """float32 array holding exact dtype values -> contiguous device tensor."""
    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(TORCH_DT[dtype])
    return t.cuda().contiguous()


def host(t: torch.Tensor) -> np.ndarray:
    return t.detach().float().cpu().numpy()


def oracle_params(p: api.Params) -> OParams:
    f = p.flags
    eviction = ("densest" if f & api.POLICY_DENSEST_ONLY else
                "mandatory_source" if f & api.POLICY_SOURCE_FILL else "default")
    return OParams(sigma2_log2=p.sigma2_log2, p=p.p, tau_num=p.tau_num, tau_log2_den=p.tau_log2_den,
                   delta_q=p.delta_q, source_order=bool(f & api.POLICY_SOURCE_ORDER),
                   refresh_base=bool(f & api.POLICY_REFRESH_BASE), eviction=eviction,
                   kv_descriptor=bool(f & api.POLICY_KV_DESCRIPTOR),
                   sequential=bool(f & api.POLICY_SEQUENTIAL))


def mirror(bank: api.Bank, b: int) -> BankState:
    """The device state of bank b as an oracle BankState."""
    m = int(bank.occupancy[b].item())
    return BankState(budget=min(int(bank.budget[b].item()), bank.Mcap),
                     K=host(bank.k[b, :m]).astype(np.float64), V=host(bank.v[b, :m]),
                     rho=bank.rho[b, :m].cpu().numpy().astype(np.int64),
                     base=bank.base[b, :m].cpu().numpy().astype(np.int64),
                     prov=bank.prov[b, :m].cpu().numpy().astype(np.int64))


def oracle_step(obanks, K, V, block_id, prm: OParams, gs: int):
    """Oracle update of every group; K, V: [B, N, d] float32 arrays."""
    new, recs = [None] * len(obanks), []
    for g0 in range(0, len(obanks), gs):
        idx = list(range(g0, g0 + gs))
        nb, rec = update_layer([obanks[i] for i in idx], [K[i].astype(np.float64) for i in idx],
                               [V[i] for i in idx], block_id, prm)
        for j, i in enumerate(idx):
            new[i] = nb[j]
        recs.append(rec)
    return new, recs


def assert_bank_equal(bank: api.Bank, b: int, ob: BankState, ctx="", kv=False):
    m = int(bank.occupancy[b].item())
    assert m == ob.m, f"{ctx} bank {b}: occupancy {m} != {ob.m}"
    prov = bank.prov[b, :m].cpu().numpy()
    assert np.array_equal(prov, ob.prov), f"{ctx} bank {b}: provenance differs"
    assert np.array_equal(host(bank.k[b, :m]).astype(np.float64), ob.K), f"{ctx} bank {b}: keys differ"
    assert np.array_equal(host(bank.v[b, :m]), np.asarray(ob.V, np.float32)), f"{ctx} bank {b}: values differ"
    assert np.array_equal(bank.rho[b, :m].cpu().numpy(), ob.rho), f"{ctx} bank {b}: rho differs"
    assert np.array_equal(bank.base[b, :m].cpu().numpy(), ob.base), f"{ctx} bank {b}: base differs"
    kn = bank.knorm[b, :m].cpu().numpy().astype(np.float64)
    ref = (ob.K * ob.K).sum(1)
    if kv:  # [K; V] geometry: the descriptor norm
        ref = ref + (np.asarray(ob.V, np.float64) ** 2).sum(1)
    assert np.array_equal(kn, ref), f"{ctx} bank {b}: knorm differs"


def assert_trace_equal(out: api.UpdateOut, recs, gs: int, prev_obanks, N: int, ctx="", sequential=False):
    """Every output of one update against the oracle records (the sequential
    competition writes no first crossings or projected densities)."""
    r_star = out.r_star.cpu().numpy()
    for g, rec in enumerate(recs):
        assert r_star[g] == rec.r_star, f"{ctx} group {g}: r* {r_star[g]} != {rec.r_star}"
        for j, hr in enumerate(rec.heads):
            b = g * gs + j
            m = prev_obanks[b].m
            if N > 0:
                assert np.array_equal(out.order[b, :N].cpu().numpy(), hr.pi), f"{ctx} bank {b}: order differs"
                sq = out.score_q[b, :N].cpu().numpy()
                ref = hr.score_q if hr.score_q is not None else np.zeros(N, np.int64)
                assert np.array_equal(sq, ref), f"{ctx} bank {b}: scores differ"
            if m and not sequential:
                assert np.array_equal(out.first_cross[b, :m].cpu().numpy(), hr.first_cross), \
                    f"{ctx} bank {b}: first crossing differs"
                assert np.array_equal(out.rho_tilde[b, :m].cpu().numpy(), hr.rho_tilde), \
                    f"{ctx} bank {b}: projected density differs"
            ne = int(out.n_evicted[b].item())
            assert ne == hr.evicted.size, f"{ctx} bank {b}: n_evicted {ne} != {hr.evicted.size}"
            assert np.array_equal(out.evicted[b, :ne].cpu().numpy(), hr.evicted), f"{ctx} bank {b}: evicted differ"
            na = int(out.n_admitted[b].item())
            assert na == hr.admitted.size
            assert np.array_equal(out.admitted[b, :na].cpu().numpy(), hr.admitted), f"{ctx} bank {b}: admitted differ"


def attention_error(got: np.ndarray, ref: np.ndarray) -> float:
    """max over rows of |o - o_ref|_inf / |o_ref|_inf."""
    num = np.abs(got - ref).max(axis=-1)
    den = np.maximum(np.abs(ref).max(axis=-1), 1e-30)
    return float((num / den).max())
