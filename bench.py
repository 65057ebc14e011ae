#!/usr/bin/env python3
"""Benchmark of the DensityKV hot path on one MI355X.

A step is one pass of the whole hot path over one block: the density-guided
update of every (layer, head) bank from the block's candidates, then the
attention of the next block's queries over the retained bank plus that
block's tokens as the local window.

Default workload: the long rollout, 30 layers x 12 heads (360 banks, one
launch per call), d = 128, bf16, per-head budget 18,720, 80 blocks of 4,680
candidates, 4,680 queries per block over bank + 4,680-token window, 256
clusters with 16 active per block and a recurring active set every 10 blocks.
Every input block of the run is drawn on the device before anything is timed
(about 104 GB of the 288 GB of HBM).  The rollout starts from empty banks and
runs its blocks in order: the first `--warmup` blocks are untimed warm-up, the
next `--steps` blocks are the timed region (bracketed by device
synchronisations), the remaining blocks complete the rollout; when warm-up +
steps exceed the rollout's length it starts again from empty banks.  HIP events
on the stream time the update and the attention of every block of the first
full pass: the record reports block 0 (the empty-bank update) separately and
the median and total over the others.

value = candidate tokens per second per layer-head over the timed steps (every
bank processes N candidates per step, concurrently).  Beside it: the update
and attention times, the attention's roofline (the dominant kernel: one
k_attn_mfma launch per attention call), the update's algorithmic Gram work
against the bf16 MFMA peak, and the CPU oracle timed on a bounded sample of
the same workload.  `--workload single_layer` (or `tiny`) times one update
into full banks plus one attention instead, with the pre-update bank restored
before every step.
"""

import argparse
import hashlib
import gc
import json
import os
import re
import sys
import time

import numpy as np

PEAK_BF16_TFLOPS = 2500.0
PEAK_HBM_GBS = 8000.0
ROOT = os.path.dirname(os.path.abspath(__file__))
ATTN_SOURCE = os.path.join(ROOT, "paper_2608_27922_amd", "csrc", "dkv_attention.hip")
METRIC = "bank-update tokens/s per layer-head + bank-attention TFLOP/s (roofline %)"
ROLLOUTS = ("rollout", "long_rollout", "headwise_budgets")
# dkv_params.flags of each policy ablation (Table 1(b); independent per-head = group size 1)
# (kv_descriptor: the [K; V] retention geometry; the workload's values are not on the key grid, so
# this mode is a timing run only, its decisions carry the fp32 rounding of the descriptor Gram;
# sequential: the within-block competition of Supp. E, one candidate per step)
POLICIES = {"default": 0, "source_order": 0x1, "refresh_base": 0x2, "densest_only": 0x4, "source_fill": 0x8,
            "kv_descriptor": 0x10, "sequential": 0x20}


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="long_rollout",
                    help="long_rollout (default), rollout, headwise_budgets, single_layer or tiny")
    ap.add_argument("--blocks", type=int, default=0,
                    help="rollout workloads: blocks per pass (default: the workload's full length)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--policy", default="default", choices=sorted(POLICIES),
                    help="policy ablation of Table 1(b) run by the update (default: the paper's policy)")
    ap.add_argument("--seq-groups", type=int, default=0,
                    help="sequential policy: groups whose pairwise weights the workspace holds at once "
                         "(default: as many as fit in 32 GiB)")
    ap.add_argument("--cpu-heads", type=int, default=0,
                    help="heads in the oracle sample (default: 8 for the rollouts, 12 for single_layer)")
    ap.add_argument("--no-sink-attention", action="store_true",
                    help="single_layer: skip the sink + window + bank attention at the deployment shape")
    ap.add_argument("--copy-probe-mb", type=int, default=0,
                    help="also run a plain elementwise copy (negation) of this many MiB: the known-size "
                         "reference that scales the HBM byte counters")
    return ap.parse_args()


def measured_traffic(workload):
    """HBM bytes per launch of the attention kernel on this workload from the committed
    counter summary (FETCH_SIZE + WRITE_SIZE, each scaled by the copy-kernel
    calibration), or None when the summary is absent or the kernel source changed
    after the counters were taken."""
    try:
        text = open(os.path.join(ROOT, "profiles", f"k_attn_mfma_{workload}_traffic.md")).read()
    except OSError:
        return None
    want = re.search(r"source_sha256:\s*([0-9a-f]{64})", text)
    val = re.search(r"traffic_bytes_per_launch:\s*([0-9]+)", text)
    if not want or not val:
        return None
    have = hashlib.sha256(open(ATTN_SOURCE, "rb").read()).hexdigest()
    return int(val.group(1)) if have == want.group(1) else None


def host_info():
    """What the oracle baseline ran on: CPU model, usable cores, BLAS library and threads."""
    info = {"cpu_model": None, "affinity_cores": len(os.sched_getaffinity(0)), "numpy": np.__version__}
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                info["cpu_model"] = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    try:
        blas = np.show_config(mode="dicts")["Build Dependencies"]["blas"]
        info["blas"] = f"{blas.get('name')} {blas.get('version')}"
    except Exception:  # noqa: BLE001 - report what is available
        info["blas"] = None
    try:
        import threadpoolctl
        pools = threadpoolctl.threadpool_info()
        info["blas_threads"] = max((p["num_threads"] for p in pools if p.get("user_api") == "blas"), default=None)
        info["openmp_threads"] = max((p["num_threads"] for p in pools if p.get("user_api") == "openmp"),
                                     default=None)
    except Exception:  # noqa: BLE001
        info["blas_threads"] = info["openmp_threads"] = None
    return info


def blas_threads(n):
    """Set the BLAS thread count explicitly for the oracle sample."""
    try:
        import threadpoolctl
        return threadpoolctl.threadpool_limits(limits=n, user_api="blas")
    except Exception:  # noqa: BLE001
        return None


def gram_pairs(m, N, R, r, e):
    """Key-key weights per bank that the method needs (Supp. C cost paragraph): the
    candidate scores (Eq. 6) m N; the prefix densities in score order (Eq. 8) m R;
    exact maintenance, each symmetric pair once: every survivor against the admitted
    and the evicted states (m - e)(r + e) (the admitted candidates' densities over
    the survivors are the same pairs), and the distinct pairs among the admitted
    r (r - 1) / 2."""
    surv = m - e
    return m * N + m * R + surv * (r + e) + r * (r - 1) // 2


# ----------------------------------------------------------------------------
# Rollout workloads (the default)
# ----------------------------------------------------------------------------

class _Out:
    """dkv_update_out with only r_star and n_evicted written, into history rows."""

    def __init__(self, api, r_star, n_evicted):
        self.api, self.r_star, self.n_evicted = api, r_star, n_evicted

    def c(self):
        return self.api.DkvUpdateOut(self.r_star.data_ptr(), None, self.n_evicted.data_ptr(),
                                     None, None, None, None, None, None)


def rollout_cpu_baseline(cfg, n_heads):
    """The oracle, as it stands, on a bounded sample of the rollout: the first two
    updates (the empty-bank block, then one block into the half-filled banks) of
    layer 0, `n_heads` heads as one group, and the attention of the next block's
    queries for those heads (NumPy draws of the same recipe)."""
    from oracle import BankState, Params, attention, update_layer
    from paper_2608_27922_amd import synth
    threads = len(os.sched_getaffinity(0))
    lim = blas_threads(threads)
    prm = Params(sigma2_log2=cfg.sigma2_log2)
    budgets = synth.budgets(cfg)[:n_heads]
    streams = [synth.HeadStream(cfg, 0, h) for h in range(n_heads)]
    banks = [BankState.empty(int(budgets[h]), cfg.d) for h in range(n_heads)]
    gs = min(cfg.group_size, n_heads)
    t0 = time.perf_counter()
    for t in range(2):
        K = [s.keys(t, cfg.n_cand).astype(np.float64) for s in streams]
        V = [s.values(t, cfg.n_cand) for s in streams]
        new = []
        for g0 in range(0, n_heads, gs):
            nb, _ = update_layer(banks[g0:g0 + gs], K[g0:g0 + gs], V[g0:g0 + gs], t, prm)
            new += nb
        banks = new
    t1 = time.perf_counter()
    for h, s in enumerate(streams):
        attention(s.queries(2), banks[h].K, banks[h].V, s.keys(2, cfg.n_window), s.values(2, cfg.n_window),
                  1.0 / np.sqrt(cfg.d))
    t2 = time.perf_counter()
    info = host_info()
    del lim
    per_head = (t2 - t0) / n_heads
    return {"value": 2 * cfg.n_cand / per_head, "unit": "tokens/s per layer-head", "cores": threads,
            "kind": "oracle",
            "sample": f"{cfg.name}, layer 0, heads 0-{n_heads - 1} as one group: blocks 0 and 1 "
                      f"({cfg.n_cand} candidates each; the empty-bank rule, then an update into banks of "
                      f"{banks[0].m} states) plus one attention of {cfg.n_query} queries over bank + "
                      f"{cfg.n_window} window per head; updates {t1 - t0:.2f} s, attention {t2 - t1:.2f} s; "
                      "NumPy draws of the same recipe",
            "host": info}


def run_rollout(args, api, synth, torch):
    cfg = synth.WORKLOADS[args.workload]
    L, H, d, N, W, nq = cfg.layers, cfg.heads, cfg.d, cfg.n_cand, cfg.n_window, cfg.n_query
    B, gs = L * H, cfg.group_size
    G = B // gs
    T = args.blocks or cfg.blocks
    budgets = synth.budgets(cfg)
    Mcap = int(budgets.max())
    dev = torch.device("cuda:0")
    bank = api.Bank(B, Mcap, d, dtype=torch.bfloat16, group_size=gs, budget=torch.from_numpy(budgets))
    prm = api.Params(sigma2_log2=cfg.sigma2_log2, flags=POLICIES[args.policy])
    ws = api.alloc_workspace(bank, N, prm.flags, seq_groups=args.seq_groups or None)
    # every input of the pass, resident in HBM before anything is timed:
    # block t's K/V are the candidates of update t and the window of attention t - 1
    gen = synth.TorchRollout(cfg, dev)
    kv = [(gen.keys(t, N), gen.values(t, N)) for t in range(T + 1)]
    qs = [gen.queries(t) for t in range(1, T + 1)]
    del gen
    out = torch.empty(B, nq, d, dtype=torch.bfloat16, device=dev)
    rs_hist = torch.zeros(T, G, dtype=torch.int32, device=dev)
    ne_hist = torch.zeros(T, B, dtype=torch.int32, device=dev)
    stream = torch.cuda.current_stream()

    # one small update + attention first, so the first rollout block pays no one-off start-up cost
    wb = api.Bank(gs, 64, d, dtype=torch.bfloat16, group_size=gs)
    api.update_bank(wb, kv[0][0][:gs, :64].contiguous(), kv[0][1][:gs, :64].contiguous(), 0, prm)
    api.bank_attention(wb, qs[0][:gs, :64].contiguous(), None, None)
    torch.cuda.synchronize()
    del wb

    def block(t, ev=None):
        if ev is not None:
            ev[0].record(stream)
        api.update_bank(bank, kv[t][0], kv[t][1], t, prm, workspace=ws,
                        out=_Out(api, rs_hist[t], ne_hist[t]))
        if ev is not None:
            ev[1].record(stream)
        api.bank_attention(bank, qs[t], kv[t + 1][0], kv[t + 1][1], out=out)
        if ev is not None:
            ev[2].record(stream)

    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(T)]
    t_start, t_end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    # (pass, block) in execution order: warm-up, then the timed steps, and at least one whole pass
    total = args.warmup + args.steps
    schedule = [(i // T, i % T) for i in range(max(total, T))]
    for i, (p, t) in enumerate(schedule):
        if t == 0:
            bank.occupancy.zero_()          # a pass starts from empty banks
        if i == args.warmup:
            torch.cuda.synchronize()
            t_start.record(stream)
        block(t, evs[t] if p == 0 else None)
        if i == total - 1:
            t_end.record(stream)
    torch.cuda.synchronize()
    seq = bool(prm.flags & api.POLICY_SEQUENTIAL)
    if seq and bool((rs_hist < 0).any()):
        raise SystemExit("a group's sequential walk gave up waiting for its records (r_star = -1)")
    timed = [t for _, t in schedule[args.warmup:total]]
    total_ms = t_start.elapsed_time(t_end)
    ms_step = total_ms / args.steps
    upd = np.array([e[0].elapsed_time(e[1]) for e in evs])
    att = np.array([e[1].elapsed_time(e[2]) for e in evs])

    # occupancy before every block, r* and evictions of every block of the first pass
    rs = np.repeat(rs_hist.cpu().numpy().astype(np.int64), gs, axis=1)      # [T, B]
    ne = ne_hist.cpu().numpy().astype(np.int64)
    Mb = np.minimum(budgets.astype(np.int64), Mcap)
    m = np.zeros((T + 1, B), np.int64)
    for t in range(T):
        m[t + 1] = m[t] + rs[t] - ne[t]
    R = np.minimum(N, np.minimum.reduceat(Mb, np.arange(0, B, gs))).repeat(gs)
    pairs = np.stack([gram_pairs(m[t], N, R, rs[t], ne[t]) for t in range(T)])     # [T, B]
    # each pair's Gram entry is a dot product of descriptors: the key, or [k; v] in the [K; V] geometry
    dd = 2 * d if prm.flags & api.POLICY_KV_DESCRIPTOR else d
    gram_flops = 2.0 * dd * pairs.sum(1)
    att_flops = 4.0 * nq * d * (m[1:] + W).sum(1)                                     # [T]
    att_tf = att_flops / (att * 1e-3) / 1e12
    gram_tf = gram_flops / (upd * 1e-3) / 1e12
    tb = np.array(timed)
    att_tf_timed = float(att_flops[tb].sum() / (att[tb].sum() * 1e-3) / 1e12)
    rest = np.arange(1, T)
    commit_bytes = (rs * (4 * d + 28)).sum(1) * 2    # admitted K/V rows + metadata, read + written
    result = {
        "metric": METRIC,
        "value": round(N / (ms_step * 1e-3), 1),
        "unit": "tokens/s per layer-head",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": cfg.dtype, "data": "synthetic",
        "config": {"workload": f"{cfg.name}: {L} layers x {H} heads ({B} banks, one launch per call), d={d}, "
                               f"{cfg.dtype}, budget {cfg.budget if not cfg.ragged else list(cfg.ragged)}, "
                               f"{T} blocks of {N} candidates, {nq} queries per block over bank + {W}-token "
                               f"window, {cfg.clusters} clusters"
                               + (f", {cfg.active} active, recurring every {cfg.revisit} blocks" if cfg.active else "")
                               + (f", centre drift {cfg.drift}" if cfg.drift else ""),
                   "banks": B, "group_size": gs, "candidates": N, "budget": int(Mcap), "blocks": T,
                   "queries": nq, "window": W, "head_dim": d, "policy": args.policy,
                   "timed_blocks": [int(tb.min()), int(tb.max())]},
        "update_ms": round(float(upd[tb].mean()), 4),
        "attention_ms": round(float(att[tb].mean()), 4),
        "attention_tflops": round(att_tf_timed, 2),
        "roofline": {"bound": "mfma", "kernel": "k_attn_mfma (bank attention)", "achieved": round(att_tf_timed, 2),
                     "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s", "frac": round(att_tf_timed / PEAK_BF16_TFLOPS, 4),
                     "traffic": measured_traffic(cfg.name)},
        "rollout": {
            "blocks": T,
            "block0": {"update_ms": round(float(upd[0]), 4), "attention_ms": round(float(att[0]), 4)},
            "median_ms": round(float(np.median(upd[rest] + att[rest])), 4) if T > 1 else None,
            "median_update_ms": round(float(np.median(upd[rest])), 4) if T > 1 else None,
            "median_attention_ms": round(float(np.median(att[rest])), 4) if T > 1 else None,
            "total_ms": round(float((upd + att).sum()), 3),
            "total_update_ms": round(float(upd.sum()), 3),
            "total_attention_ms": round(float(att.sum()), 3),
            "update_tokens_per_s_per_layer_head": round(T * N / (upd.sum() * 1e-3), 1),
            "attention_tflops": round(float(att_flops.sum() / (att.sum() * 1e-3) / 1e12), 2),
            "update_gram_tflop": round(float(gram_flops.sum() / 1e12), 3),
            "update_gram_tflops": round(float(gram_flops.sum() / (upd.sum() * 1e-3) / 1e12), 2),
            "update_gram_frac_of_bf16_peak": round(float(gram_flops.sum() / (upd.sum() * 1e-3) / 1e12)
                                                   / PEAK_BF16_TFLOPS, 4),
            "median_update_gram_frac_of_bf16_peak": round(float(np.median(gram_tf[rest])) / PEAK_BF16_TFLOPS, 4)
            if T > 1 else None,
            "update_gram_note": "work-equivalent: the method's Gram pairs (m R prefix pairs of Eq. 8 included) over "
                                "the update time; where the first 256 ordered candidates decide r*, the crossing "
                                "search evaluates m x 256 of the m R prefix pairs",
            "median_attention_frac_of_bf16_peak": round(float(np.median(att_tf[rest])) / PEAK_BF16_TFLOPS, 4)
            if T > 1 else None,
            "r_star_mean_per_block": [round(float(x), 1) for x in rs_hist.float().mean(1).cpu().numpy()],
            "occupancy_mean_after": round(float(m[T].mean()), 1),
            "commit_bytes_total": int(commit_bytes.sum()),
        },
    }
    if seq:   # the Gram accounting is the default update's; the sequential walk has its own
        for k in ("update_gram_tflop", "update_gram_tflops", "update_gram_frac_of_bf16_peak",
                  "median_update_gram_frac_of_bf16_peak", "update_gram_note"):
            result["rollout"][k] = None
    del kv, qs, out, bank, ws
    torch.cuda.empty_cache()
    return result


# ----------------------------------------------------------------------------
# Single-update workloads (tiny, single_layer)
# ----------------------------------------------------------------------------

def sink_attention(api, synth, torch, steps=10):
    """densitykv_bank_attention_sink at the paper's deployment context (Supp. D): 12 heads,
    d = 128, bf16, a 1,560-token sink, a 7,800-token window and full banks of 9,360
    retained states, 4,680 queries (one block).  Timed with HIP events on the stream."""
    cfg = synth.Config(seed_id=41, name="deploy", layers=1, heads=12, d=128, dtype="bf16", n_cand=4680,
                       n_query=4680, n_window=7800, budget=9360, clusters=64, blocks=1, group_size=12,
                       sigma2_log2=6, drift=0.0)
    B, d, M, ns, nw, nq = cfg.heads, cfg.d, cfg.budget, 1560, cfg.n_window, cfg.n_query
    bank = api.Bank(B, M, d, dtype=torch.bfloat16, group_size=B)
    kb, vb = synth.torch_layer_block(cfg, 0, 0, M, "cuda", seed=1)
    bank.k.copy_(kb)
    bank.v.copy_(vb)
    bank.occupancy.fill_(M)
    sk, sv = synth.torch_layer_block(cfg, 0, 1, ns, "cuda", seed=1)
    wk, wv = synth.torch_layer_block(cfg, 0, 2, nw, "cuda", seed=1)
    q, _ = synth.torch_layer_block(cfg, 0, 3, nq, "cuda", seed=1)
    out = torch.empty_like(q)
    stream = torch.cuda.current_stream()
    for _ in range(3):
        api.bank_attention_sink(bank, q, sk, sv, wk, wv, out=out)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record(stream)
    for _ in range(steps):
        api.bank_attention_sink(bank, q, sk, sv, wk, wv, out=out)
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / steps
    flops = 4.0 * B * nq * (M + nw + ns) * d
    tf = flops / (ms * 1e-3) / 1e12
    return {"context": f"sink {ns} + window {nw} + bank {M} keys, {nq} queries, {B} heads, d={d}, bf16",
            "ms": round(ms, 4), "tflops": round(tf, 2), "frac_of_bf16_peak": round(tf / PEAK_BF16_TFLOPS, 4)}


def single_cpu_baseline(case, cfg, n_heads):
    """The oracle, as it stands, on a bounded sample: one update + one attention for
    `n_heads` heads treated as one group (rank 0 only)."""
    from oracle import BankState, Params, attention, update_layer
    threads = len(os.sched_getaffinity(0))
    lim = blas_threads(threads)
    prm = Params(sigma2_log2=cfg.sigma2_log2)
    hs = range(n_heads)
    banks = [BankState.empty(cfg.budget, cfg.d) for _ in hs]
    banks, _ = update_layer(banks, [case["init_K"][h].astype(np.float64) for h in hs],
                            [case["init_V"][h] for h in hs], 0, prm)
    t0 = time.perf_counter()
    banks, _ = update_layer(banks, [case["seg_K"][h].astype(np.float64) for h in hs],
                            [case["seg_V"][h] for h in hs], 1, prm)
    t1 = time.perf_counter()
    for h in hs:
        attention(case["q"][h], banks[h].K, banks[h].V, case["win_K"][h], case["win_V"][h], 1.0 / np.sqrt(cfg.d))
    t2 = time.perf_counter()
    info = host_info()
    del lim
    step_s = (t2 - t0) / n_heads  # per layer-head
    return {"value": cfg.n_cand / step_s, "unit": "tokens/s per layer-head", "cores": threads,
            "kind": "oracle",
            "sample": f"{n_heads} head(s) of the same workload: one update (N={cfg.n_cand} into a full bank of "
                      f"{cfg.budget}) + one attention ({cfg.n_query} queries over bank + {cfg.n_window} window), "
                      f"update {t1 - t0:.2f} s, attention {t2 - t1:.2f} s",
            "host": info}


def run_single(args, api, synth, torch):
    cfg = synth.WORKLOADS[args.workload]
    dt = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32
    case = synth.single_update_case(cfg)
    to = lambda a: torch.from_numpy(np.ascontiguousarray(a, np.float32)).to(dt).cuda().contiguous()
    prm = api.Params(sigma2_log2=cfg.sigma2_log2)
    run_prm = api.Params(sigma2_log2=cfg.sigma2_log2, flags=POLICIES[args.policy])
    B, N, d = cfg.heads, cfg.n_cand, cfg.d
    bank = api.Bank(B, cfg.budget, d, dtype=dt, group_size=cfg.group_size)
    init_k, init_v = to(case["init_K"]), to(case["init_V"])
    seg_k, seg_v = to(case["seg_K"]), to(case["seg_V"])
    q, wk, wv = to(case["q"]), to(case["win_K"]), to(case["win_V"])
    ws = api.alloc_workspace(bank, max(N, cfg.budget), run_prm.flags)
    api.update_bank(bank, init_k, init_v, 0, prm, workspace=ws)   # starts full (empty-bank rule)
    torch.cuda.synchronize()
    snap = bank.snapshot()
    m0 = bank.occupancy.cpu().numpy().astype(np.int64)
    out = torch.empty_like(q)
    stream = torch.cuda.current_stream()
    G = B // cfg.group_size
    rs_hist = torch.zeros(args.steps + 1, G, dtype=torch.int32, device="cuda")
    ne_hist = torch.zeros(args.steps + 1, B, dtype=torch.int32, device="cuda")

    def step(k=None, ev=None):
        bank.restore(snap)
        if ev is not None:
            ev[0].record(stream)
        o = _Out(api, rs_hist[k], ne_hist[k]) if k is not None else None
        api.update_bank(bank, seg_k, seg_v, 1, run_prm, workspace=ws, out=o)
        if ev is not None:
            ev[1].record(stream)
        api.bank_attention(bank, q, wk, wv, out=out)
        if ev is not None:
            ev[2].record(stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(args.steps)]
    t_start = torch.cuda.Event(enable_timing=True)
    t_end = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t_start.record(stream)
    for k in range(args.steps):
        step(k, evs[k])
    t_end.record(stream)
    torch.cuda.synchronize()
    if args.policy == "sequential" and bool((rs_hist < 0).any()):
        raise SystemExit("a group's sequential walk gave up waiting for its records (r_star = -1)")
    total_ms = t_start.elapsed_time(t_end)
    ms_step = total_ms / args.steps
    upd_ms = float(np.mean([e[0].elapsed_time(e[1]) for e in evs]))
    att_ms = float(np.mean([e[1].elapsed_time(e[2]) for e in evs]))
    m_after = bank.occupancy.cpu().numpy()
    att_flops = float(sum(4.0 * cfg.n_query * (int(m) + cfg.n_window) * d for m in m_after))
    att_tflops = att_flops / (att_ms * 1e-3) / 1e12
    r = np.repeat(rs_hist[0].cpu().numpy().astype(np.int64), cfg.group_size)
    e = ne_hist[0].cpu().numpy().astype(np.int64)
    R = np.minimum(N, bank.budget.cpu().numpy().astype(np.int64))
    pairs = gram_pairs(m0, N, R, r, e)
    dd = 2 * d if run_prm.flags & api.POLICY_KV_DESCRIPTOR else d   # descriptor width of the Gram
    gram_tf = 2.0 * dd * float(pairs.sum()) / (upd_ms * 1e-3) / 1e12

    result = {
        "metric": METRIC,
        "value": round(N / (ms_step * 1e-3), 1),
        "unit": "tokens/s per layer-head",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": cfg.dtype, "data": "synthetic",
        "config": {"workload": f"{cfg.name}: {cfg.layers} layer x {cfg.heads} heads, d={d}, "
                               f"{cfg.dtype}, budget {cfg.budget} (starts full), segment {N}"
                               + (f" ({int(cfg.dup_frac * 100)}% near-duplicates)" if cfg.dup_frac else "")
                               + f", {cfg.n_query} queries over bank + {cfg.n_window}-token window",
                   "banks": B, "group_size": cfg.group_size, "candidates": N, "budget": cfg.budget,
                   "queries": cfg.n_query, "window": cfg.n_window, "head_dim": d, "policy": args.policy},
        "update_ms": round(upd_ms, 4),
        "update_tokens_per_s_per_layer_head": round(N / (upd_ms * 1e-3), 1),
        "attention_ms": round(att_ms, 4),
        "attention_tflops": round(att_tflops, 2),
        "roofline": {"bound": "mfma", "kernel": "k_attn_mfma (bank attention)", "achieved": round(att_tflops, 2),
                     "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s", "frac": round(att_tflops / PEAK_BF16_TFLOPS, 4),
                     "traffic": measured_traffic(cfg.name)},
    }
    if args.policy != "sequential":
        result["update_gram"] = {"pairs": int(pairs.sum()), "tflop": round(2.0 * dd * float(pairs.sum()) / 1e12, 4),
                                 "tflops": round(gram_tf, 2), "frac_of_bf16_peak": round(gram_tf / PEAK_BF16_TFLOPS, 4),
                                 "r_star": int(r.max()), "evicted_per_bank": int(e.max())}
    else:
        # the walk offers the N candidates one per step: latency per step, not a roofline, bounds it
        result["sequential"] = {"steps_per_update": N, "update_us_per_step": round(upd_ms * 1e3 / N, 3)}
    if not args.no_sink_attention and cfg.name == "single_layer":
        result["sink_attention"] = sink_attention(api, synth, torch)
    del bank, ws, snap
    if not args.no_cpu_baseline and args.policy == "default":
        result["cpu_baseline"] = single_cpu_baseline(case, cfg, min(args.cpu_heads or 12, cfg.heads))
    return result


def main():
    args = parse()
    if args.gpus != 1:
        print(json.dumps({"error": "this build runs on one GPU only; --gpus must be 1 "
                                   "(the banks of different layers would shard across GPUs with no communication)"}))
        sys.exit(2)
    import torch
    from paper_2608_27922_amd import api, synth

    torch.cuda.set_device(0)
    api.lib()
    if args.workload in ROLLOUTS:
        result = run_rollout(args, api, synth, torch)
        if not args.no_cpu_baseline and args.policy == "default":
            result["cpu_baseline"] = rollout_cpu_baseline(synth.WORKLOADS[args.workload], args.cpu_heads or 8)
    elif args.workload in ("tiny", "single_layer"):
        result = run_single(args, api, synth, torch)
    else:
        raise SystemExit(f"unknown workload {args.workload}")
    if args.copy_probe_mb:
        nbytes = args.copy_probe_mb << 20
        src = torch.ones(nbytes // 4, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            torch.neg(src, out=dst)      # reads and writes nbytes each
        torch.cuda.synchronize()
        result["copy_probe_bytes"] = nbytes
        del src, dst
    print(json.dumps(result), flush=True)
    # Return every device allocation while the runtime (and any profiler attached
    # to it) is fully up, rather than leaving it to the process's exit handlers.
    torch.cuda.synchronize()
    gc.collect()
    torch.cuda.empty_cache()
    torch.cuda.synchronize()


if __name__ == "__main__":
    main()
