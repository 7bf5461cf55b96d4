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
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="llavanext")
    ap.add_argument("--rho", type=float, default=None, help="retention ratio (default: the workload's first)")
    ap.add_argument("--lse-from-prefill", action="store_true",
                    help="the text rows' normalisers come from the prefill (computed before the timed region "
                         "by the library's own statistics sweep, standing in for a prefill attention kernel's "
                         "row log-sum-exp): scoring reads K once")
    ap.add_argument("--budget-rule", default="tv", choices=("tv", "uniform", "tt"),
                    help="layer budgets by text->vision mass (TVB), equally, or by text->text mass")
    ap.add_argument("--vision-rank", default="twr", choices=("twr", "attention_sum"),
                    help="vision importance: text-weighted ranking or the plain text-row attention sum")
    ap.add_argument("--no-tpr", action="store_true", help="rank text and vision tokens together (no TPR)")
    ap.add_argument("--vision-only", action="store_true",
                    help="vision-only eviction (every layer keeps all text; rho is the retained share of the "
                         "vision tokens) instead of eviction among all tokens")
    ap.add_argument("--cache", default="contiguous", choices=("contiguous", "paged"),
                    help="compacted cache layout: one segment per (sequence, layer), or pages of a pool "
                         "assigned by the page-table kernel (decode then takes a per-sequence step)")
    ap.add_argument("--page-size", type=int, default=16, help="rows per page of the paged cache")
    ap.add_argument("--decode-steps", type=int, default=None)
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--tv-gap", type=float, default=None,
                    help="draw the question-row queries with the per-layer depth profile of this strength "
                         "(default: the workload's i.i.d. text queries)")
    ap.add_argument("--no-depth-profile", action="store_true",
                    help="skip the extra run of the same workload with the depth profile (tv_gap 6)")
    ap.add_argument("--no-flush-mall", dest="flush_mall", action="store_false",
                    help="do not flush the MALL before timed passes (by default every timed pass starts after a "
                         "512 MB read of an unrelated buffer, so the MALL holds none of its inputs and no dirty "
                         "lines; passes after a 512 MB write, and back-to-back passes, are timed separately)")
    ap.add_argument("--no-ceilings", action="store_true",
                    help="skip the in-run read / copy / matrix-core ceiling measurements")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=10.0, help="target length of the oracle sample")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="instead of the benchmark, copy a 1 GiB buffer 5 times (a plain copy kernel of known "
                         "size, to scale rocprofv3 FETCH_SIZE / WRITE_SIZE counters to bytes)")
    ap.add_argument("--ingest-counters", nargs=4, metavar=("FETCH_CSV", "WRITE_CSV", "COPY_FETCH_CSV",
                                                            "COPY_WRITE_CSV"),
                    help="turn rocprofv3 --pmc counter files of a bench run and of a --calibrate-copy run into "
                         "profiles/hbm_counters.json (HBM bytes per launch of each kernel)")
    ap.add_argument("--ingest-mfma-counters", metavar="PMC_CSV",
                    help="turn a rocprofv3 --pmc run of this bench with SQ_INSTS_MFMA SQ_VALU_MFMA_BUSY_CYCLES "
                         "GRBM_GUI_ACTIVE SQ_INSTS_VALU SQ_INSTS_VALU_TRANS_F32 into profiles/mfma_counters.json "
                         "(matrix-core work per launch of each scoring kernel)")
    ap.add_argument("--schedule", default="auto", choices=("auto", "two_step", "phases", "lse_in"),
                    help="scoring schedule: vision scores after the budgets only for layers that need them "
                         "(auto, two_step), or one launch per phase for every layer (phases)")
    return ap.parse_args()


def source_hash(files):
    """Hash of a kernel's sources and of the device compile flags of its main (first)
    source (either changes the code)."""
    from paper_2606_03075_amd import build as _build
    h = hashlib.sha256(" ".join(_build.device_flags(files[0])).encode())
    for f in files:
        with open(os.path.join(ROOT, "paper_2606_03075_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


KERNEL_SOURCES = {
    "score_text": ["score.hip", "score_core.h", "tgvkv_device.h"],
    "score_stats": ["score.hip", "score_core.h", "tgvkv_device.h"],
    "score_vision": ["score.hip", "score_core.h", "tgvkv_device.h"],
    "compact": ["compact.hip", "tgvkv_rows.h", "tgvkv_device.h"],
    "decode": ["decode.hip", "tgvkv_rows.h", "tgvkv_device.h"],
}


def counter_key(workload, vision_only=False, cache="contiguous", rho=None, lse_in=False):
    """Key of a workload's counters in profiles/hbm_counters.json (the eviction mode, the scoring
    schedule, the cache layout and a retention other than the workload's first change the bytes)."""
    from workloads import CONFIGS
    rho_tag = "" if rho is None or rho == CONFIGS[workload].rhos[0] else f"@rho{rho:g}"
    return (workload + rho_tag + (":vision_only" if vision_only else "") + (":lse_in" if lse_in else "")
            + (":paged" if cache == "paged" else ""))


def traffic_for(kernel, workload, decode_steps=None):
    """HBM bytes per launch from committed rocprofv3 counters, if they match the current source."""
    try:
        with open(COUNTERS) as f:
            data = json.load(f)
    except (OSError, ValueError):
        return None
    rec = data.get(workload, {}).get(kernel)
    if not rec or rec.get("source_hash") != source_hash(KERNEL_SOURCES[kernel]):
        return None
    if kernel == "decode" and rec.get("decode_steps") != decode_steps:
        return None  # per-launch decode bytes depend on how many steps were averaged
    return rec.get("bytes_per_launch")


def decode_in_graph(buf, dq, dk, dv, T, reps):
    """Decode time per step with the T steps captured in one HIP graph and replayed (after
    the timed region; a replay rewrites each step's cache slot with the same row).  The
    launch gaps between steps are gone; each kernel is unchanged.  None if capture fails."""
    import torch
    if T <= 0:
        return None
    try:
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            for s_ in range(T):
                buf.decode(s_, dq[s_], dk[s_], dv[s_])
        g.replay()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(max(reps, 1)):
            g.replay()
        e1.record()
        torch.cuda.synchronize()
        return round(e0.elapsed_time(e1) * 1e3 / (max(reps, 1) * T), 2)
    except RuntimeError as exc:
        log(f"[bench] decode graph capture failed: {exc}")
        return None


def cpu_baseline(cfg, t, dec, tot, budget_s, vision_only=False, opts=None):
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
        _, budgets, idx = O.evict_sequence(q, k, cfg.n_sys, cfg.n_vis, cfg.n_qst, tot, vision_only=vision_only,
                                           budget_rule=opts.budget_rule if opts else 0,
                                           vision_rank=opts.vision_rank if opts else 0,
                                           joint_rank=bool(opts.joint_rank) if opts else False)
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


COPY_BYTES = 1 << 30
# bench stage -> the kernel whose counters stand for it ("score_text" is sweep 1 with the
# text pass, the kernel the two-step schedule runs for that stage)
KERNEL_NAMES = {"score_text": "score_stats_text_kernel", "score_stats": "score_stats_kernel",
                "score_vision": "score_vision_kernel", "compact": "compact_kernel", "decode": "decode_kernel"}
# rocprofv3 names of the kernels behind each bench stage (decode runs on the vector or the matrix cores)
KERNEL_MATCH = {"decode": ("decode_kernel<", "decode_mfma_kernel<")}


def calibrate_copy():
    import torch
    a = torch.empty(COPY_BYTES, dtype=torch.uint8, device="cuda")
    b = torch.empty_like(a)
    for _ in range(5):
        b.copy_(a)
    torch.cuda.synchronize()
    print(json.dumps({"calibration": "copy", "bytes_read": COPY_BYTES, "bytes_written": COPY_BYTES, "launches": 5}))


def _counter_rows(path):
    import csv
    with open(path) as f:
        return list(csv.DictReader(f))


def _per_kernel_kib(rows, counter):
    """Mean counter value per dispatch, grouped by kernel-name substring."""
    acc = {}
    for r in rows:
        if r.get("Counter_Name") != counter:
            continue
        name = r.get("Kernel_Name", "")
        acc.setdefault(name, []).append(float(r["Counter_Value"]))
    return {k: sum(v) / len(v) for k, v in acc.items()}


def ingest_counters(fetch_csv, write_csv, copy_fetch_csv, copy_write_csv, workload, decode_steps):
    fetch = _per_kernel_kib(_counter_rows(fetch_csv), "FETCH_SIZE")
    write = _per_kernel_kib(_counter_rows(write_csv), "WRITE_SIZE")
    cf = _per_kernel_kib(_counter_rows(copy_fetch_csv), "FETCH_SIZE")
    cw = _per_kernel_kib(_counter_rows(copy_write_csv), "WRITE_SIZE")
    copy_f = max(cf.values())       # the 1 GiB copy dominates the calibration run
    copy_w = max(cw.values())
    scale_f = COPY_BYTES / copy_f   # bytes per counter unit, from the copy of known size
    scale_w = COPY_BYTES / copy_w
    out = {"_calibration": {"copy_bytes": COPY_BYTES, "fetch_size_per_copy": copy_f, "write_size_per_copy": copy_w,
                            "fetch_scale": scale_f, "write_scale": scale_w}}
    rec = {}
    for key, kname in KERNEL_NAMES.items():
        pats = KERNEL_MATCH.get(key, (kname,))
        fk = [v for n, v in fetch.items() if any(p in n for p in pats)]
        wk = [v for n, v in write.items() if any(p in n for p in pats)]
        if not fk or not wk:
            continue
        fb, wb = max(fk) * scale_f, max(wk) * scale_w
        rec[key] = {"fetch_bytes": fb, "write_bytes": wb, "bytes_per_launch": fb + wb,
                    "source_hash": source_hash(KERNEL_SOURCES[key])}
        if key == "decode":
            rec[key]["decode_steps"] = decode_steps  # the counter run's mean over its steps
    try:
        with open(COUNTERS) as f:
            data = json.load(f)
    except (OSError, ValueError):
        data = {}
    data[workload] = rec
    data["_calibration"] = out["_calibration"]
    with open(COUNTERS, "w") as f:
        json.dump(data, f, indent=1)
    print(json.dumps(data[workload]))


MFMA_COUNTERS = os.path.join(ROOT, "profiles", "mfma_counters.json")
MFMA_FLOPS = 2 * 16 * 16 * 32   # v_mfma_f32_16x16x32_bf16, the only matrix instruction the scoring kernels issue
SIMDS = 256 * 4                 # MI355X: 256 compute units x 4 SIMDs, each with its own matrix core
XCDS = 8                        # GRBM_GUI_ACTIVE is counted per XCD and summed over the 8
SCORE_KERNELS = ("score_text", "score_stats", "score_vision")
MFMA_PMC = ("SQ_INSTS_MFMA", "SQ_VALU_MFMA_BUSY_CYCLES", "GRBM_GUI_ACTIVE", "SQ_INSTS_VALU", "SQ_INSTS_VALU_TRANS_F32")


def ingest_mfma_counters(csv_path, workload):
    """Per-launch means of the matrix-core counters of each scoring kernel (wave-level instruction
    counts summed over the chip; busy cycles summed over the SIMDs; GPU-active cycles of the dispatch)."""
    rows = _counter_rows(csv_path)
    per = {c: _per_kernel_kib(rows, c) for c in MFMA_PMC}
    rec = {}
    for key in SCORE_KERNELS:
        kname = KERNEL_NAMES[key]
        names = [n for n in per["SQ_INSTS_MFMA"] if kname + "<" in n or n.endswith(kname)]
        if not names:
            continue
        n = max(names, key=lambda x: per["SQ_INSTS_MFMA"][x])  # the launch shape the bench times
        durs = [(int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) for r in rows
                if r.get("Kernel_Name") == n and r.get("Counter_Name") == "SQ_INSTS_MFMA"]
        rec[key] = {"pmc_run_launch_ns": sum(durs) / max(len(durs), 1),"mfma_instrs": per["SQ_INSTS_MFMA"][n], "mfma_busy_cycles": per["SQ_VALU_MFMA_BUSY_CYCLES"][n],
                    "gpu_active_cycles": per["GRBM_GUI_ACTIVE"][n], "valu_instrs": per["SQ_INSTS_VALU"][n],
                    "trans_instrs": per["SQ_INSTS_VALU_TRANS_F32"][n],
                    "source_hash": source_hash(KERNEL_SOURCES[key])}
    try:
        with open(MFMA_COUNTERS) as f:
            data = json.load(f)
    except (OSError, ValueError):
        data = {}
    data[workload] = rec
    with open(MFMA_COUNTERS, "w") as f:
        json.dump(data, f, indent=1)
    print(json.dumps(rec))


def mfma_summary(c, launch_ms):
    """What one scoring kernel's matrix-core counters say at a measured launch time: the
    issued MFMA rate against the dense bf16 peak and the busy fraction (busy cycles are
    summed over the SIMDs, GPU-active cycles over the XCDs)."""
    issued = c["mfma_instrs"] * MFMA_FLOPS / (launch_ms * 1e-3) / 1e12
    return {
        "mfma_instrs_per_launch": int(c["mfma_instrs"]),
        "issued_tflops": round(issued, 1),
        "issued_frac_of_peak": round(issued / BF16_PEAK_TFLOPS, 4),
        "mfma_busy_frac": round(c["mfma_busy_cycles"] / (SIMDS / XCDS * c["gpu_active_cycles"]), 4),
        "valu_instrs_per_mfma": round(c["valu_instrs"] / max(c["mfma_instrs"], 1), 2),
        "trans_instrs_per_launch": int(c["trans_instrs"]),
    }


def mfma_for(kernel, workload):
    """Committed matrix-core counters of a scoring kernel, if they match the current source."""
    try:
        with open(MFMA_COUNTERS) as f:
            rec = json.load(f).get(workload, {}).get(kernel)
    except (OSError, ValueError):
        return None
    if not rec or rec.get("source_hash") != source_hash(KERNEL_SOURCES[kernel]):
        return None
    return rec


FLUSH_BYTES = 512 << 20       # read (or written) before a timed pass so the 256 MB MALL holds none of its inputs
CEILING_BYTES = 1 << 30       # read / copy ceiling stream
CEILING_MFMA_WG = 512         # 2 waves per SIMD on all 1024 SIMDs
CEILING_MFMA_ITERS = 20000


def measure_ceilings(bd, reps=5):
    """The chip's achievable rates, measured in this process (HIP events on the launch stream):
    a 1 GiB non-temporal read stream and a 1 GiB copy (the access pattern of the key sweeps,
    compaction and decode), and back-to-back dense bf16 MFMAs on every SIMD."""
    import torch
    stream = torch.cuda.current_stream()
    src = torch.empty(CEILING_BYTES, dtype=torch.uint8, device="cuda")
    src.fill_(1)
    dst = torch.empty_like(src)
    sink = torch.zeros(1, dtype=torch.int32, device="cuda")
    out = torch.empty(CEILING_MFMA_WG * 256, dtype=torch.float32, device="cuda")

    def timed(fn):
        fn()  # warm-up launch
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        best = None
        for _ in range(reps):
            e0.record(stream)
            fn()
            e1.record(stream)
            torch.cuda.synchronize()
            ms = e0.elapsed_time(e1)
            best = ms if best is None else min(best, ms)
        return best

    read_ms = timed(lambda: bd.tgvkv_ceiling_read(src, sink))
    copy_ms = timed(lambda: bd.tgvkv_ceiling_copy(src, dst))
    flops = [0]

    def mfma():
        flops[0] = bd.tgvkv_ceiling_mfma(CEILING_MFMA_WG, CEILING_MFMA_ITERS, out)

    mfma_ms = timed(mfma)
    del src, dst
    return {
        "read_gbs": round(CEILING_BYTES / (read_ms * 1e-3) / 1e9, 1),
        "copy_gbs": round(2 * CEILING_BYTES / (copy_ms * 1e-3) / 1e9, 1),
        "mfma_bf16_tflops": round(flops[0] / (mfma_ms * 1e-3) / 1e12, 1),
        "how": f"best of {reps}: 1 GiB read and 1 GiB copy with 16-byte non-temporal loads (copy counts read "
               f"+ write bytes); {CEILING_MFMA_WG} workgroups x 4 waves x {CEILING_MFMA_ITERS} rounds of 8 "
               f"independent v_mfma_f32_16x16x32_bf16",
    }


def main():
    args = parse()
    if args.ingest_mfma_counters:
        ingest_mfma_counters(args.ingest_mfma_counters,
                             counter_key(args.workload, args.vision_only, args.cache, args.rho,
                                         args.lse_from_prefill))
        return
    if args.ingest_counters:
        from workloads import CONFIGS
        T = CONFIGS[args.workload].decode_steps if args.decode_steps is None else args.decode_steps
        ingest_counters(*args.ingest_counters,
                        workload=counter_key(args.workload, args.vision_only, args.cache, args.rho, args.lse_from_prefill),
                        decode_steps=T)
        return
    if args.calibrate_copy:
        calibrate_copy()
        return
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py runs on one GPU only: the eviction pass shards by sequence with no communication, "
              "so the single-GPU number is the per-GPU throughput (use --gpus 1).", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2606_03075_amd import binding as bd
    from workloads import CONFIGS, DEPTH_PROFILE_TV_GAP, depth_profile, make_decode_tensors, make_prefill_tensors, \
        total_budget
    from workloads.gen import gen_qtext_slice, f32_to_bf16_bits

    bd.load_library()
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    cfg = CONFIGS[args.workload]
    if args.tv_gap is not None:
        cfg = depth_profile(cfg, args.tv_gap)
    rho = args.rho if args.rho is not None else cfg.rhos[0]
    T = cfg.decode_steps if args.decode_steps is None else args.decode_steps
    B, L, N = cfg.batch, cfg.layers, cfg.n_tokens
    # vision-only: the budget counts vision tokens (no forced positions are used here)
    tot = total_budget(rho, cfg.n_vis if args.vision_only else N, L)

    t0 = time.perf_counter()
    t = make_prefill_tensors(cfg, seed=args.seed)
    dec = make_decode_tensors(cfg, seed=args.seed, steps=max(T, 1))
    log(f"[bench] generated {cfg.name} inputs (tv_gap {cfg.tv_gap:g}) in {time.perf_counter() - t0:.1f} s")

    def dev(x):
        return torch.from_numpy(np.ascontiguousarray(x).view(np.int16)).view(torch.bfloat16).cuda()

    q_d, k_d, v_d = dev(t["q_text"]), dev(t["k"]), dev(t["v"])
    dq, dk, dv = dev(dec["q"]), dev(dec["k_new"]), dev(dec["v_new"])
    p = bd.problem_from(cfg)
    opts = bd.make_opts(vision_only=args.vision_only,
                        budget_rule={"tv": bd.BUDGET_TV, "uniform": bd.BUDGET_UNIFORM, "tt": bd.BUDGET_TT}[
                            args.budget_rule],
                        vision_rank={"twr": bd.RANK_TWR, "attention_sum": bd.RANK_ATTENTION_SUM}[args.vision_rank],
                        joint_rank=args.no_tpr)
    buf = bd.EvictionBuffers(p, opts, tot, max(T, 1))
    stream = torch.cuda.current_stream()
    schedule = args.schedule
    if args.lse_from_prefill:
        schedule = "lse_in"

    def prefill_normalisers():
        # what a prefill attention kernel returns for the text rows (their row log-sum-exp),
        # produced here, outside the timed region, by the library's own statistics sweep
        buf.score(q_d, k_d, bd.SCORE_STATS | bd.SCORE_TEXT)
        torch.cuda.synchronize()

    if args.lse_from_prefill:
        prefill_normalisers()

    paged = args.cache == "paged"
    if paged:
        # the pool, its free list and the per-step step vectors are set up outside the timed region
        width, n_pages = bd.page_plan(p, opts, tot, max(T, 1), args.page_size)
        pool = bd.PagedPool(cfg.heads_kv, cfg.head_dim, args.page_size, n_pages)
        free_ids = torch.arange(n_pages, dtype=torch.int32, device="cuda")
        table = torch.empty((B * L, width), dtype=torch.int32, device="cuda")
        used = torch.zeros((1,), dtype=torch.int64, device="cuda")
        steps_d = torch.arange(max(T, 1), dtype=torch.int32, device="cuda")[:, None].repeat(1, B).contiguous()
        log(f"[bench] paged cache: {n_pages} pages of {args.page_size} rows, table width {width}")
    flush_buf = None
    if args.flush_mall:
        flush_buf = torch.ones(FLUSH_BYTES // 4, dtype=torch.float32, device="cuda")
        flush_sum = torch.empty((), dtype=torch.float32, device="cuda")
    flush = "read" if args.flush_mall else None

    def do_flush():
        if flush == "read":
            torch.sum(flush_buf, dim=0, out=flush_sum)  # 512 MB of clean lines replace whatever the MALL held
        elif flush == "write":
            flush_buf.zero_()  # 512 MB of dirty lines, as a prefill that just wrote the cache leaves it

    sched_now = [schedule]  # the schedule one_step runs (the one-sweep variant below switches it)

    def one_step(events=None, decode=True):
        names = []

        def mark(name):
            names.append(name)
            if events is not None:
                ev = torch.cuda.Event(enable_timing=True)
                ev.record(stream)
                events.append((name, ev))

        do_flush()  # outside the timed intervals
        mark("start")
        sched = buf.evict(q_d, k_d, v_d, schedule=sched_now[0], marks=mark, compact=not paged)
        if paged:
            bd.tgvkv_page_table(p, opts, buf.budgets, tot, max(T, 1), args.page_size, free_ids, table, used)
            mark("pages")
            bd.tgvkv_compact_paged(p, opts, k_d, v_d, buf.idx, buf.budgets, buf.idx_offsets, tot, table,
                                   args.page_size, pool.k_pool, pool.v_pool, unit_order=buf.unit_order)
            mark("compact")
        for s_ in range(T if decode else 0):
            mark("decode_gap")  # launch gap before the step: in the step time, not in the kernel's
            if paged:
                pool.decode(p, opts, table, buf.budgets, max(T, 1), steps_d[s_], dq[s_], dk[s_], dv[s_], buf.out,
                            buf.ws_decode, unit_order=buf.unit_order)
            else:
                buf.decode(s_, dq[s_], dk[s_], dv[s_])
            mark("decode")
        return sched

    def run(n_warm, n_timed, decode=True):
        """n_warm untimed steps, then n_timed steps with events; returns per-stage mean times."""
        for _ in range(n_warm):
            one_step(decode=decode)
        torch.cuda.synchronize()
        timed = [[] for _ in range(n_timed)]
        w0 = time.perf_counter()
        sched = None
        for k in range(n_timed):
            sched = one_step(timed[k], decode=decode)
        torch.cuda.synchronize()
        wall = time.perf_counter() - w0
        stage_ms, dec_ms, dec_gap_ms, step_ms = {}, 0.0, 0.0, 0.0
        evict_per_step, decode_launch_us = [], []
        for evs in timed:
            ev_step = 0.0
            for (n0, e0), (n1, e1) in zip(evs[:-1], evs[1:]):
                raw = e0.elapsed_time(e1)
                ms = raw / n_timed
                if n1 == "decode":
                    dec_ms += ms / max(T, 1)
                    decode_launch_us.append(raw * 1e3)
                elif n1 == "decode_gap":
                    dec_gap_ms += ms / max(T, 1)
                else:
                    stage_ms[n1] = stage_ms.get(n1, 0.0) + ms
                    ev_step += raw
            evict_per_step.append(ev_step)
            step_ms += evs[0][1].elapsed_time(evs[-1][1]) / n_timed
        return {"sched": sched, "stage_ms": stage_ms, "evict_ms": sum(stage_ms.values()), "dec_ms": dec_ms,
                "dec_gap_ms": dec_gap_ms, "step_ms": step_ms, "wall": wall, "evict_per_step": evict_per_step,
                "decode_launch_us": decode_launch_us}

    def spread(xs, nd):
        if not xs:
            return None
        q = np.percentile(np.asarray(xs, np.float64), [10, 50, 90])
        return {"p10": round(float(q[0]), nd), "median": round(float(q[1]), nd), "p90": round(float(q[2]), nd)}

    thr = buf.forced_or_text()

    def vision_layers(sched):
        budgets = buf.budgets.cpu().numpy()
        return int((budgets > thr).sum()) if sched == "two_step" else B * L

    # ---- the timed steps: each pass starts after a 512 MB read of an unrelated buffer (cold: the
    # MALL holds none of its inputs and nothing dirty), and is followed by every decode step
    main_run = run(args.warmup, args.steps)
    sched = main_run["sched"]
    stage_ms, dec_ms, evict_ms = main_run["stage_ms"], main_run["dec_ms"], main_run["evict_ms"]
    vis_layers = vision_layers(sched)
    decode_graph_us = None if paged else decode_in_graph(buf, dq, dk, dv, T, args.steps)
    # ---- the eviction pass after a 512 MB write (the MALL full of dirty lines, whose write-back
    # then competes with the pass's reads), and back to back with no flush and no decode in
    # between (warm: what the previous pass left in the MALL and L2, its compaction's writes
    # included)
    after_write_ms = warm_ms = None
    if args.flush_mall:
        flush = "write"
        after_write_ms = run(args.warmup, args.steps, decode=False)["evict_ms"]
        flush = None
        warm_ms = run(args.warmup, args.steps, decode=False)["evict_ms"]
        flush = "read"
    ceilings = None if args.no_ceilings else measure_ceilings(bd)
    tokens_per_s = B * N / (evict_ms * 1e-3)

    # algorithmic bytes per launch: what the method must move, each once (K and the text
    # queries for scoring, the retained K/V read and written for compaction, the pruned
    # cache plus new tokens for a decode step); score_vision's key bytes are the second
    # sweep over K, traffic of this implementation rather than of the method
    H, Hkv, D, Nq, Nv = cfg.heads_q, cfg.heads_kv, cfg.head_dim, cfg.n_qst, cfg.n_vis
    kept = buf.kept  # tokens each sequence keeps
    k_bytes = B * L * Hkv * N * D * 2
    q_bytes = B * L * H * cfg.n_text * D * 2
    compact_bytes = 4 * B * kept * Hkv * D * 2
    alg = {
        "score": k_bytes + q_bytes,
        "score_text": k_bytes + q_bytes,
        "score_stats": k_bytes + B * L * H * Nq * D * 2,
        "score_vision": vis_layers * (Hkv * Nv * D * 2 + H * Nq * D * 2),
        "compact": compact_bytes,
        "decode": (B * kept + B * L * (T + 1) / 2.0) * Hkv * D * 4 + B * L * (H * D * 2 + 2 * Hkv * D * 2 + H * D * 4),
    }
    kinds = {k: "algorithmic" for k in alg}
    kinds["score_vision"] = "implementation: the second sweep over the vision keys (re-read)"

    def achieved_peak(kname):
        if ceilings is None:
            return None
        return ceilings["copy_gbs"] if kname == "compact" else ceilings["read_gbs"]

    roofs = {}
    for kname in ("score", "score_text", "score_stats", "score_vision", "compact", "decode"):
        ms = dec_ms if kname == "decode" else stage_ms.get(kname, 0.0)
        if ms <= 0:
            continue
        gbs = alg[kname] / (ms * 1e-3) / 1e9
        ap = achieved_peak(kname)
        roofs[kname] = {"bound": "hbm", "achieved": round(gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                        "frac": round(gbs / HBM_PEAK_GBS, 4),
                        "traffic": traffic_for(kname, counter_key(cfg.name, args.vision_only, args.cache, rho,
                                                                   args.lse_from_prefill), T),
                        "kernel": kname, "alg_bytes_per_launch": int(alg[kname]), "bytes_kind": kinds[kname],
                        "avg_launch_ms": round(ms, 4),
                        "ms_per_step": round(ms * (T if kname == "decode" else 1), 4),
                        "achieved_peak": ap, "frac_of_achieved": round(gbs / ap, 4) if ap else None}
    dominant = max(roofs, key=lambda k: roofs[k]["ms_per_step"])
    # the whole eviction pass against what the method must move once: K and the text queries,
    # and the retained K/V read and written by compaction
    pass_bytes = k_bytes + q_bytes + compact_bytes

    def pass_roof(ms):
        gbs = pass_bytes / (ms * 1e-3) / 1e9
        ap = ceilings["read_gbs"] if ceilings else None
        return {"bound": "hbm", "achieved": round(gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(gbs / HBM_PEAK_GBS, 4), "alg_bytes": int(pass_bytes),
                "alg_bytes_are": "K + text-row queries once, plus the retained K/V read and written",
                "evict_ms": round(ms, 4), "roof_ms": round(pass_bytes / (HBM_PEAK_GBS * 1e9) * 1e3, 4),
                "roof_tokens_per_s": round(B * N / (pass_bytes / (HBM_PEAK_GBS * 1e9)), 1),
                "achieved_peak": ap, "frac_of_achieved": round(gbs / ap, 4) if ap else None}

    # scoring's algorithmic matrix work: one QK^T over the logits every text row can see
    # (system row i sees i + 1 keys, question row i sees the system and vision keys and i + 1
    # question keys), 2 * head_dim flops each; the implementation's second sweep is not counted
    Ns = cfg.n_sys
    logits = Ns * (Ns + 1) / 2 + Nq * (Ns + Nv) + Nq * (Nq + 1) / 2
    score_flops = 2.0 * B * L * H * D * logits
    score_ms = sum(v for k, v in stage_ms.items() if k in ("score",) + SCORE_KERNELS)
    ckey = counter_key(cfg.name, args.vision_only, args.cache, rho, args.lse_from_prefill)
    per_kernel = {}
    for kname in SCORE_KERNELS + ("score",):
        ms = stage_ms.get(kname, 0.0)
        if ms <= 0:
            continue
        c = mfma_for(kname, ckey) if kname != "score" else None
        ent = {"avg_launch_ms": round(ms, 4), "counters": None}
        if c is not None:
            ent["counters"] = mfma_summary(c, ms)
        per_kernel[kname] = ent
    scoring_mfma = None
    if score_ms > 0:
        tf = score_flops / (score_ms * 1e-3) / 1e12
        mp = ceilings["mfma_bf16_tflops"] if ceilings else None
        scoring_mfma = {"alg_flops": int(score_flops), "score_ms": round(score_ms, 4), "alg_tflops": round(tf, 1),
                        "peak_tflops": BF16_PEAK_TFLOPS, "alg_frac_of_peak": round(tf / BF16_PEAK_TFLOPS, 4),
                        "achieved_peak_tflops": mp, "alg_frac_of_achieved": round(tf / mp, 4) if mp else None,
                        "kernels": per_kernel}

    recipe = (f"text queries and keys i.i.d. N(0,1)" if cfg.tv_gap == 0 else
              f"depth profile: question-row vision logits shifted per layer (tv_gap {cfg.tv_gap:g})")
    line = {
        "metric": METRIC,
        "value": round(tokens_per_s, 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(main_run["step_ms"], 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": f"{cfg.name}: batch {B}, {L} layers, {H} heads ({Hkv} KV), head_dim {D}, "
                               f"{cfg.n_sys}+{Nv}+{Nq} tokens, retention {rho:g}"
                               f"{' of vision tokens (all text kept)' if args.vision_only else ''}"
                               f"{', text-row normalisers from the prefill' if args.lse_from_prefill else ''}"
                               f", {T} decode steps"
                               f"{f', paged cache ({args.page_size}-row pages)' if paged else ''}; {recipe}; "
                               f"vision noise {cfg.vis_sigma:g}{', sink on token 0' if cfg.sink else ''}"
                               f"{f', {cfg.frames} frames' if cfg.frames else ''}",
                   "batch": B, "layers": L, "heads_q": H, "heads_kv": Hkv, "head_dim": D,
                   "n_sys": cfg.n_sys, "n_vis": Nv, "n_qst": Nq, "retention": rho, "total_budget_per_seq": tot,
                   "tv_gap": cfg.tv_gap, "vision_noise": cfg.vis_sigma,
                   "vision_only": bool(args.vision_only),
                   "normalisers_from_prefill": bool(args.lse_from_prefill),
                   "budget_rule": args.budget_rule, "vision_rank": args.vision_rank, "tpr": not args.no_tpr,
                   "decode_steps": T, "vision_scored_layers": vis_layers, "schedule": sched,
                   "cache": args.cache, "page_size": args.page_size if paged else None,
                   "mall_before_each_pass": "512 MB read of an unrelated buffer" if args.flush_mall else
                   "what the previous step's decode left"},
        "evict_ms": round(evict_ms, 4),
        "evict_ms_spread": spread(main_run["evict_per_step"], 4),
        "evict_ms_after_write": round(after_write_ms, 4) if after_write_ms is not None else None,
        "evict_ms_warm": round(warm_ms, 4) if warm_ms is not None else None,
        "evict_roofline": pass_roof(evict_ms),
        "decode_launch_us_spread": spread(main_run["decode_launch_us"], 2),
        "decode_us_per_step": round(dec_ms * 1e3, 2),
        "decode_us_per_step_with_launch_gaps": round((dec_ms + main_run["dec_gap_ms"]) * 1e3, 2),
        "decode_us_per_step_graph": decode_graph_us,
        "stage_ms": {k: round(v, 4) for k, v in stage_ms.items()},
        "schedule": sched,
        "scoring_mfma": scoring_mfma,
        "roofline": roofs[dominant],
        "roofline_kernels": roofs,
        "ceilings": ceilings,
        "wall_ms_per_step": round(main_run["wall"] / args.steps * 1e3, 3),
    }

    # ---- the same inputs with every text row's normaliser taken from the prefill (one K sweep:
    # text and vision scores and the TV mass in one pass, then the budgets), as a labelled variant
    if sched == "two_step" and not args.no_depth_profile:
        prefill_normalisers()
        sched_now[0] = "lse_in"
        lp = run(args.warmup, args.steps, decode=False)
        sched_now[0] = schedule
        line["normalisers_from_prefill"] = {
            "value": round(B * N / (lp["evict_ms"] * 1e-3), 1), "unit": "tokens/s",
            "evict_ms": round(lp["evict_ms"], 4), "evict_ms_spread": spread(lp["evict_per_step"], 4),
            "evict_roofline": pass_roof(lp["evict_ms"]),
            "stage_ms": {k: round(v, 4) for k, v in lp["stage_ms"].items()},
            "note": "the text rows' log-sum-exp is given (as a prefill attention kernel returns it), "
                    "produced outside the timed region by the library's own statistics sweep",
        }

    # ---- the same workload with the depth profile of the text-to-vision attention (only the
    # question-row queries change), as a labelled variant beside the i.i.d. headline
    if not args.no_depth_profile and cfg.tv_gap == 0 and not args.vision_only and not args.no_tpr \
            and args.budget_rule == "tv":
        dcfg = depth_profile(cfg)
        t1 = time.perf_counter()
        qd = np.stack([np.stack([f32_to_bf16_bits(gen_qtext_slice(dcfg, args.seed, b, l)) for l in range(L)])
                       for b in range(B)])
        q_d.copy_(dev(qd))
        del qd
        if args.lse_from_prefill:
            prefill_normalisers()
        log(f"[bench] depth-profile queries in {time.perf_counter() - t1:.1f} s")
        dp = run(args.warmup, args.steps)
        dvl = vision_layers(dp["sched"])
        line["depth_profile"] = {
            "tv_gap": DEPTH_PROFILE_TV_GAP,
            "value": round(B * N / (dp["evict_ms"] * 1e-3), 1), "unit": "tokens/s",
            "evict_ms": round(dp["evict_ms"], 4), "evict_ms_spread": spread(dp["evict_per_step"], 4),
            "evict_roofline": pass_roof(dp["evict_ms"]),
            "decode_us_per_step": round(dp["dec_ms"] * 1e3, 2),
            "stage_ms": {k: round(v, 4) for k, v in dp["stage_ms"].items()},
            "vision_scored_layers": dvl,
            "budgets_seq0": buf.budgets[0].tolist(),
        }
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(cfg, t, dec, tot, args.cpu_seconds, args.vision_only, opts)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
