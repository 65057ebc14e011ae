#!/usr/bin/env python3
"""Benchmark of the DensityKV hot path on one MI355X.

A step is one pass of the whole hot path over one block: the density-guided
update of every (layer, head) bank from the block's candidates, then the
attention of the next block's queries over the retained bank plus the local
window.  Workload (default): one layer x 12 heads, d = 128, bf16, per-head
budget 4,680, banks start full (built by the empty-bank rule), one incoming
segment of 4,680 candidates with 30% near-duplicates, 4,680 queries over
bank + a 4,680-token window.  Every step restores the pre-update bank with one
device-to-device copy of the packed bank state (inside the timed region) so
that all steps do the same work.

Prints one JSON line.  value = candidate tokens per second per layer-head for
the whole step (update + attention); the update-only rate and the attention
TFLOP/s are reported beside it, with the roofline of the dominant kernel and
the CPU oracle timed on a bounded sample.  update_gram gives the update's
algorithmic Gram work (pairs of the score, prefix, partial-tile and maintenance
stages at 2 d flops each) and its rate against the bf16 MFMA peak over the
whole update time.  Two extra fields time the sink +
window + bank attention at the paper's deployment shape and one block of the
rollout configuration at full scale (360 banks in one launch).
"""

import argparse
import hashlib
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
TRAFFIC_SUMMARY = os.path.join(ROOT, "profiles", "k_attn_mfma_single_layer_traffic.md")
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
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="single_layer", help="tiny or single_layer")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--policy", default="default", choices=sorted(POLICIES),
                    help="policy ablation of Table 1(b) run by the update (default: the paper's policy)")
    ap.add_argument("--cpu-heads", type=int, default=12,
                    help="heads in the oracle sample (12 = the whole single_layer step, about 10 s on 16 host threads)")
    ap.add_argument("--no-sink-attention", action="store_true",
                    help="skip the extra measurement of the sink + window + bank attention at the deployment shape")
    ap.add_argument("--no-rollout-block", action="store_true",
                    help="skip the extra measurement of one rollout block at full scale (360 banks)")
    ap.add_argument("--rollout-block-only", action="store_true",
                    help="run only the full-scale rollout block and print its figures (for profiling)")
    ap.add_argument("--copy-probe-mb", type=int, default=0,
                    help="also run a plain elementwise copy (negation) of this many MiB: the known-size "
                         "reference that scales the HBM byte counters")
    return ap.parse_args()


def measured_traffic():
    """HBM bytes per launch of the attention kernel from the committed counter summary
    (FETCH_SIZE + WRITE_SIZE, each scaled by the copy-kernel calibration), or None when
    the summary is absent or the kernel source changed after the counters were taken."""
    try:
        text = open(TRAFFIC_SUMMARY).read()
    except OSError:
        return None
    want = re.search(r"source_sha256:\s*([0-9a-f]{64})", text)
    val = re.search(r"traffic_bytes_per_launch:\s*([0-9]+)", text)
    if not want or not val:
        return None
    have = hashlib.sha256(open(ATTN_SOURCE, "rb").read()).hexdigest()
    return int(val.group(1)) if have == want.group(1) else None


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


def update_gram_work(api, torch, bank, snap, seg_k, seg_v, prm, ws, N, d, upd_ms):
    """Algorithmic Gram work of the timed update and its rate against the bf16 MFMA
    peak: per bank m*N pairs for the candidate scores (Eq. 6), m*R for the prefix
    densities (Eq. 8, R = min(N, M)), m*64 for the partial tile at r*, and
    (m + r*)*e + r*^2 for the density maintenance (Supp. C), at 2 d flops per pair;
    m, r* and e are those of the timed update (rerun once with its outputs)."""
    bank.restore(snap)
    m0 = bank.occupancy.cpu().numpy().astype(np.int64)
    M = bank.budget.cpu().numpy().astype(np.int64)
    out = api.UpdateOut(bank, N)
    api.update_bank(bank, seg_k, seg_v, 1, prm, workspace=ws, out=out)
    torch.cuda.synchronize()
    r = np.repeat(out.r_star.cpu().numpy().astype(np.int64), bank.gs)
    e = out.n_evicted.cpu().numpy().astype(np.int64)
    R = np.minimum(N, M)
    pairs = m0 * N + m0 * R + m0 * np.minimum(64, R) + (m0 + r) * e + r * r
    flops = 2.0 * d * float(pairs.sum())
    tf = flops / (upd_ms * 1e-3) / 1e12
    return {"pairs": int(pairs.sum()), "tflop": round(flops / 1e12, 4), "tflops": round(tf, 2),
            "frac_of_bf16_peak": round(tf / PEAK_BF16_TFLOPS, 4), "r_star": int(out.r_star.max().item()),
            "evicted_per_bank": int(e.max())}


def rollout_block(api, synth, torch, steps=3):
    """One block of the rollout configuration at full scale: 30 layers x 12 heads
    (360 banks, one launch), d = 128, bf16, budget 9,360, 4,680 candidates per
    bank, 4,680 queries over bank + 4,680-token window.  Three blocks fill the
    banks first (device-drawn, as the non-compared layers of the full-size
    tests); each timed step restores that state, updates with block 3 and runs
    the attention.  Timed with HIP events on the stream."""
    cfg = synth.WORKLOADS["rollout"]
    L, H, d, N, M, nq = cfg.layers, cfg.heads, cfg.d, cfg.n_cand, cfg.budget, cfg.n_query
    B = L * H

    def block(t, n, seed=0):
        ks, vs = zip(*(synth.torch_layer_block(cfg, layer, t, n, "cuda", seed=seed) for layer in range(L)))
        return torch.cat(ks).contiguous(), torch.cat(vs).contiguous()

    bank = api.Bank(B, M, d, dtype=torch.bfloat16, group_size=cfg.group_size)
    ws = api.alloc_workspace(bank, N)
    prm = api.Params(sigma2_log2=cfg.sigma2_log2)
    for t in range(3):
        k, v = block(t, N)
        api.update_bank(bank, k, v, t, prm, workspace=ws)
    seg_k, seg_v = block(3, N)
    q, _ = block(3, nq, seed=1)
    del k, v
    out = torch.empty_like(q)
    upd = api.UpdateOut(bank, N)
    torch.cuda.synchronize()
    snap = bank.snapshot()
    stream = torch.cuda.current_stream()
    times = []
    for it in range(steps + 1):
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
        ev[0].record(stream)
        bank.restore(snap)
        ev[1].record(stream)
        api.update_bank(bank, seg_k, seg_v, 3, prm, workspace=ws, out=upd)
        ev[2].record(stream)
        api.bank_attention(bank, q, seg_k, seg_v, out=out)
        ev[3].record(stream)
        torch.cuda.synchronize()
        if it > 0:   # the first pass is a warm-up
            times.append([ev[0].elapsed_time(ev[3]), ev[1].elapsed_time(ev[2]), ev[2].elapsed_time(ev[3])])
    step_ms, upd_ms, att_ms = (float(np.mean(c)) for c in zip(*times))
    m_after = bank.occupancy.cpu().numpy()
    # algorithmic Gram work of the timed update (the same per-bank pair counts as update_gram)
    r = np.repeat(upd.r_star.cpu().numpy().astype(np.int64), cfg.group_size)
    e = upd.n_evicted.cpu().numpy().astype(np.int64)
    bank.restore(snap)
    m0 = bank.occupancy.cpu().numpy().astype(np.int64)
    R = min(N, M)
    gram_flops = 2.0 * d * float((m0 * N + m0 * R + m0 * min(64, R) + (m0 + r) * e + r * r).sum())
    gram_tf = gram_flops / (upd_ms * 1e-3) / 1e12
    flops = float(sum(4.0 * nq * (int(m) + N) * d for m in m_after))
    tf = flops / (att_ms * 1e-3) / 1e12
    res = {"context": f"rollout: {L} layers x {H} heads ({B} banks, one launch), d={d}, bf16, budget {M}, "
                      f"block 3 ({N} candidates) into full banks, {nq} queries over bank + {N}-token window",
           "ms_per_step": round(step_ms, 3), "update_ms": round(upd_ms, 3), "attention_ms": round(att_ms, 3),
           "tokens_per_s_per_layer_head": round(N / (step_ms * 1e-3), 1),
           "update_tokens_per_s_per_layer_head": round(N / (upd_ms * 1e-3), 1),
           "attention_tflops": round(tf, 2), "attention_frac_of_bf16_peak": round(tf / PEAK_BF16_TFLOPS, 4),
           "update_gram_tflop": round(gram_flops / 1e12, 3), "update_gram_tflops": round(gram_tf, 2),
           "update_gram_frac_of_bf16_peak": round(gram_tf / PEAK_BF16_TFLOPS, 4),
           "mean_r_star": round(float(upd.r_star.float().mean().item()), 1),
           "mean_occupancy": round(float(m_after.mean()), 1)}
    del bank, ws, snap, seg_k, seg_v, q, out
    torch.cuda.empty_cache()
    return res


def cpu_baseline(case, cfg, n_heads):
    """The oracle, as it stands, on a bounded sample: one update + one attention for
    `n_heads` heads treated as one group (rank 0 only)."""
    from oracle import BankState, Params, attention, update_layer
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
    threads = int(os.environ.get("OMP_NUM_THREADS", "0")) or len(os.sched_getaffinity(0))
    step_s = (t2 - t0) / n_heads  # per layer-head
    return {"value": cfg.n_cand / step_s, "unit": "tokens/s per layer-head", "cores": threads,
            "kind": "oracle",
            "sample": f"{n_heads} head(s) of the same workload: one update (N={cfg.n_cand} into a full bank of "
                      f"{cfg.budget}) + one attention ({cfg.n_query} queries over bank + {cfg.n_window} window), "
                      f"update {t1 - t0:.2f} s, attention {t2 - t1:.2f} s"}


def main():
    args = parse()
    if args.gpus != 1:
        print(json.dumps({"error": "this build runs on one GPU only; --gpus must be 1 "
                                   "(banks shard by layer without communication; see the design notes)"}))
        sys.exit(2)
    import torch
    from paper_2608_27922_amd import api, synth

    if args.rollout_block_only:
        torch.cuda.set_device(0)
        print(json.dumps({"rollout_block": rollout_block(api, synth, torch, steps=args.steps)}), flush=True)
        return
    cfg = synth.WORKLOADS[args.workload]
    if not cfg.starts_full:
        raise SystemExit("bench workload must be a single-update workload (tiny or single_layer)")
    torch.cuda.set_device(0)
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
    out = torch.empty_like(q)
    stream = torch.cuda.current_stream()

    def step(ev=None):
        bank.restore(snap)
        if ev is not None:
            ev[0].record(stream)
        api.update_bank(bank, seg_k, seg_v, 1, run_prm, workspace=ws)
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
        step(evs[k])
    t_end.record(stream)
    torch.cuda.synchronize()
    total_ms = t_start.elapsed_time(t_end)
    ms_step = total_ms / args.steps
    upd_ms = float(np.mean([e[0].elapsed_time(e[1]) for e in evs]))
    att_ms = float(np.mean([e[1].elapsed_time(e[2]) for e in evs]))
    m_after = bank.occupancy.cpu().numpy()
    att_flops = float(sum(4.0 * cfg.n_query * (int(m) + cfg.n_window) * d for m in m_after))
    att_tflops = att_flops / (att_ms * 1e-3) / 1e12
    value = N / (ms_step * 1e-3)   # every bank processes N candidates per step, concurrently

    result = {
        "metric": "bank-update tokens/s per layer-head + bank-attention TFLOP/s (roofline %)",
        "value": round(value, 1),
        "unit": "tokens/s per layer-head",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": cfg.dtype, "data": "synthetic",
        "config": {"workload": f"{cfg.name}: {cfg.layers} layer x {cfg.heads} heads, d={d}, "
                               f"{cfg.dtype}, budget {cfg.budget} (starts full), segment {N} (30% near-duplicates), "
                               f"{cfg.n_query} queries over bank + {cfg.n_window}-token window",
                   "banks": B, "group_size": cfg.group_size, "candidates": N, "budget": cfg.budget,
                   "queries": cfg.n_query, "window": cfg.n_window, "head_dim": d, "policy": args.policy},
        "update_ms": round(upd_ms, 4),
        "update_tokens_per_s_per_layer_head": round(N / (upd_ms * 1e-3), 1),
        "attention_ms": round(att_ms, 4),
        "attention_tflops": round(att_tflops, 2),
        "roofline": {"bound": "mfma", "kernel": "bank attention", "achieved": round(att_tflops, 2),
                     "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s", "frac": round(att_tflops / PEAK_BF16_TFLOPS, 4),
                     "traffic": measured_traffic()},
    }
    if args.policy != "sequential":
        result["update_gram"] = update_gram_work(api, torch, bank, snap, seg_k, seg_v, run_prm, ws, N, d, upd_ms)
    else:
        # the walk offers the N candidates one per step: latency per step, not a roofline, bounds it
        result["sequential"] = {"steps_per_update": N, "update_us_per_step": round(upd_ms * 1e3 / N, 3)}
    if not args.no_sink_attention:
        result["sink_attention"] = sink_attention(api, synth, torch)
    if not args.no_rollout_block:
        result["rollout_block"] = rollout_block(api, synth, torch)
    if args.copy_probe_mb:
        nbytes = args.copy_probe_mb << 20
        src = torch.ones(nbytes // 4, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            torch.neg(src, out=dst)      # reads and writes nbytes each
        torch.cuda.synchronize()
        result["copy_probe_bytes"] = nbytes
    if not args.no_cpu_baseline and args.policy == "default":
        result["cpu_baseline"] = cpu_baseline(case, cfg, min(args.cpu_heads, cfg.heads))
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
