#!/usr/bin/env python3
"""Throughput of the TGV-KV eviction pass and of decode over the pruned cache, on one MI355X.

One step is the whole hot path over one batch of synthetic prefills (inputs
already resident in HBM): text statistics and text scores, TVB budgets,
text-weighted vision scores (only for layers whose budget reaches past the
text), TPR selection, gather-compaction, then the workload's decode steps over
the compacted cache.  Every stage is one library call; HIP events on the stream
the kernels run on bracket each call.

Prints one JSON line.  `value` is prefill tokens evicted per second
(batch * N / eviction time); decode attention time per step, per-kernel
roofline fractions and the fp64 oracle's CPU time on a bounded sample are
reported alongside.
"""

from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "prefill tokens/s evicted (score+select+compact); decode attn μs/step; % roofline"
HBM_PEAK_GBS = 8000.0          # MI355X HBM3E
BF16_PEAK_TFLOPS = 2500.0      # MI355X dense bf16 MFMA
COUNTERS = os.path.join(ROOT, "profiles", "hbm_counters.json")


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default="llavanext")
    ap.add_argument("--rho", type=float, default=None, help="retention ratio (default: the workload's first)")
    ap.add_argument("--decode-steps", type=int, default=None)
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=10.0, help="target length of the oracle sample")
    ap.add_argument("--score-all-layers", action="store_true",
                    help="compute vision scores for every layer (by default layers whose budget only "
                         "covers text skip them)")
    return ap.parse_args()


def source_hash(files):
    h = hashlib.sha256()
    for f in files:
        with open(os.path.join(ROOT, "paper_2606_03075_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


KERNEL_SOURCES = {
    "score_stats": ["score.hip", "tgvkv_device.h"],
    "score_vision": ["score.hip", "tgvkv_device.h"],
    "compact": ["compact.hip", "tgvkv_device.h"],
    "decode": ["decode.hip", "tgvkv_device.h"],
}


def traffic_for(kernel, workload, launches_bytes_unit=None):
    """HBM bytes per launch from committed rocprofv3 counters, if they match the current source."""
    try:
        with open(COUNTERS) as f:
            data = json.load(f)
    except (OSError, ValueError):
        return None
    rec = data.get(workload, {}).get(kernel)
    if not rec or rec.get("source_hash") != source_hash(KERNEL_SOURCES[kernel]):
        return None
    return rec.get("bytes_per_launch")


def cpu_baseline(cfg, t, dec, tot, budget_s):
    """The fp64 oracle, as it stands, on whole sequences of the same inputs until ~budget_s seconds."""
    import numpy as np
    import oracle.tgvkv_oracle as O
    from workloads import bf16_bits_to_f32
    try:
        import threadpoolctl
        blas = max((i.get("num_threads", 1) for i in threadpoolctl.threadpool_info()), default=1)
    except Exception:  # pragma: no cover
        blas = 1
    nseq = 0
    idx0 = None
    t0 = time.perf_counter()
    for b in range(cfg.batch):
        q = bf16_bits_to_f32(t["q_text"][b])
        k = bf16_bits_to_f32(t["k"][b])
        _, budgets, idx = O.evict_sequence(q, k, cfg.n_sys, cfg.n_vis, cfg.n_qst, tot)
        for l in range(cfg.layers):
            O.compact_slice(t["k"][b, l], t["v"][b, l], idx[l], 0)
        if idx0 is None:
            idx0 = idx
        nseq += 1
        if time.perf_counter() - t0 >= budget_s:
            break
    t_evict = time.perf_counter() - t0
    # one decode step of sequence 0 over its pruned cache, every layer, scaled to the batch
    tau = O.default_scale(cfg.head_dim)
    t1 = time.perf_counter()
    for l in range(cfg.layers):
        sel = idx0[l][0]
        Kc = [bf16_bits_to_f32(t["k"][0, l, h][sel]) for h in range(cfg.heads_kv)]
        Vc = [bf16_bits_to_f32(t["v"][0, l, h][sel]) for h in range(cfg.heads_kv)]
        O.decode_reference(bf16_bits_to_f32(dec["q"][:1, 0, l]), bf16_bits_to_f32(dec["k_new"][:1, 0, l]),
                           bf16_bits_to_f32(dec["v_new"][:1, 0, l]), Kc, Vc, tau)
    dsec = (time.perf_counter() - t1) * cfg.batch
    return {
        "value": nseq * cfg.n_tokens / t_evict,
        "unit": "tokens/s",
        "cores": int(blas),
        "kind": "oracle",
        "sample": f"{nseq} of {cfg.batch} sequences x {cfg.layers} layers (score, budget, select, compact), "
                  f"{t_evict:.1f} s; decode: one step of one sequence, scaled to the batch",
        "decode_ms_per_step": dsec * 1e3,
        "affinity_cores": len(os.sched_getaffinity(0)),
    }


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py runs on one GPU only: the eviction pass shards by sequence with no communication, "
              "so the single-GPU number is the per-GPU throughput (use --gpus 1).", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2606_03075_amd import binding as bd
    from workloads import CONFIGS, make_decode_tensors, make_prefill_tensors, total_budget

    bd.load_library()
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    cfg = CONFIGS[args.workload]
    rho = args.rho if args.rho is not None else cfg.rhos[0]
    T = cfg.decode_steps if args.decode_steps is None else args.decode_steps
    B, L, N = cfg.batch, cfg.layers, cfg.n_tokens
    tot = total_budget(rho, N, L)

    t0 = time.perf_counter()
    t = make_prefill_tensors(cfg, seed=args.seed)
    dec = make_decode_tensors(cfg, seed=args.seed, steps=max(T, 1))
    log(f"[bench] generated {cfg.name} inputs in {time.perf_counter() - t0:.1f} s")

    def dev(x):
        return torch.from_numpy(np.ascontiguousarray(x).view(np.int16)).view(torch.bfloat16).cuda()

    q_d, k_d, v_d = dev(t["q_text"]), dev(t["k"]), dev(t["v"])
    dq, dk, dv = dev(dec["q"]), dev(dec["k_new"]), dev(dec["v_new"])
    p = bd.problem_from(cfg)
    buf = bd.EvictionBuffers(p, None, tot, max(T, 1))
    skip = not args.score_all_layers
    stream = torch.cuda.current_stream()
    STAGES = ["score_stats", "score_text", "budget", "score_vision", "select", "compact"]

    def one_step(events=None):
        rec = (lambda i: events[i].record(stream)) if events is not None else (lambda i: None)
        rec(0)
        buf.score(q_d, k_d, bd.SCORE_STATS)
        rec(1)
        buf.score(q_d, k_d, bd.SCORE_TEXT)
        rec(2)
        buf.budget()
        rec(3)
        buf.score(q_d, k_d, bd.SCORE_VISION, budgets=buf.budgets if skip else None)
        rec(4)
        buf.select()
        rec(5)
        buf.compact(k_d, v_d)
        rec(6)
        for s in range(T):
            buf.decode(s, dq[s], dk[s], dv[s])
            rec(7 + s)

    for _ in range(args.warmup):
        one_step()
    torch.cuda.synchronize()
    nev = 7 + T
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(nev)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    w0 = time.perf_counter()
    for k in range(args.steps):
        one_step(evs[k])
    torch.cuda.synchronize()
    wall = time.perf_counter() - w0

    stage_ms = {s: 0.0 for s in STAGES}
    dec_ms = 0.0
    step_ms = 0.0
    for k in range(args.steps):
        e = evs[k]
        for i, s in enumerate(STAGES):
            stage_ms[s] += e[i].elapsed_time(e[i + 1]) / args.steps
        if T:
            dec_ms += e[6].elapsed_time(e[6 + T]) / args.steps / T
        step_ms += e[0].elapsed_time(e[nev - 1]) / args.steps
    evict_ms = sum(stage_ms.values())
    tokens_per_s = B * N / (evict_ms * 1e-3)

    # algorithmic bytes per launch (K/V, queries and outputs read or written once)
    H, Hkv, D, Nq, Nv = cfg.heads_q, cfg.heads_kv, cfg.head_dim, cfg.n_qst, cfg.n_vis
    budgets = buf.budgets.cpu().numpy()
    vis_layers = int((budgets > cfg.n_text).sum()) if skip else B * L
    qq = B * L * H * Nq * D * 2
    alg = {
        "score_stats": B * L * Hkv * N * D * 2 + qq + B * L * H * Nq * 8,
        "score_vision": vis_layers * (Hkv * Nv * D * 2 + H * Nq * D * 2 + 2 * Hkv * Nv * 4 + Nv * 4),
        "compact": 4 * B * tot * Hkv * D * 2,
        "decode": (B * tot + B * L * (T + 1) / 2.0) * Hkv * D * 4 + B * L * (H * D * 2 + 2 * Hkv * D * 2 + H * D * 4),
    }
    per_launch_ms = {"score_stats": stage_ms["score_stats"], "score_vision": stage_ms["score_vision"],
                     "compact": stage_ms["compact"], "decode": dec_ms}
    launches = {"score_stats": 1, "score_vision": 1, "compact": 1, "decode": T}
    roofs = {}
    for kname, ms in per_launch_ms.items():
        if ms <= 0:
            continue
        gbs = alg[kname] / (ms * 1e-3) / 1e9
        tr = traffic_for(kname, cfg.name)
        roofs[kname] = {"bound": "hbm", "achieved": round(gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                        "frac": round(gbs / HBM_PEAK_GBS, 4), "traffic": tr, "kernel": kname,
                        "alg_bytes_per_launch": int(alg[kname]), "avg_launch_ms": round(ms, 4),
                        "ms_per_step": round(ms * launches[kname], 4)}
    dominant = max(roofs, key=lambda k: roofs[k]["ms_per_step"])
    flops = 2.0 * B * L * H * D * (Nq * (cfg.n_sys + Nv) + Nq * (Nq + 1) / 2)
    mfma_pct = flops / (stage_ms["score_stats"] * 1e-3) / (BF16_PEAK_TFLOPS * 1e12)

    line = {
        "metric": METRIC,
        "value": round(tokens_per_s, 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(step_ms, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": f"{cfg.name}: batch {B}, {L} layers, {H} heads ({Hkv} KV), head_dim {D}, "
                               f"{cfg.n_sys}+{Nv}+{Nq} tokens, retention {rho:g}, {T} decode steps",
                   "batch": B, "layers": L, "heads_q": H, "heads_kv": Hkv, "head_dim": D,
                   "n_sys": cfg.n_sys, "n_vis": Nv, "n_qst": Nq, "retention": rho, "total_budget_per_seq": tot,
                   "decode_steps": T, "vision_scored_layers": vis_layers},
        "evict_ms": round(evict_ms, 4),
        "decode_us_per_step": round(dec_ms * 1e3, 2),
        "stage_ms": {k: round(v, 4) for k, v in stage_ms.items()},
        "score_stats_mfma_frac_of_peak": round(mfma_pct, 4),
        "roofline": roofs[dominant],
        "roofline_kernels": roofs,
        "wall_ms_per_step": round(wall / args.steps * 1e3, 3),
    }
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(cfg, t, dec, tot, args.cpu_seconds)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
