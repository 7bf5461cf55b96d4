"""End-to-end GPU parity: eviction pass (score, budget, vision score, select, compact) then decode steps.

Inputs are the seeded workloads; the oracle runs on the same bf16 values.
"""

import numpy as np
import pytest

import oracle.tgvkv_oracle as O
from paper_2606_03075_amd import binding as bd
from tests.gpu_util import (DECODE_ATOL, assert_close_rel, bf16_host_bits, budget_allowed, dev_bf16, host,
                            idx_allowed, log)
from workloads import bf16_bits_to_f32, make_decode_tensors, make_prefill_tensors, total_budget
from workloads.configs import CONFIGS, custom_config

pytestmark = pytest.mark.gpu


class _Tiled:
    """Host view of a batch whose sequence b holds generated sequence src[b] (index axis `axis`)."""

    def __init__(self, arr, src, axis):
        self.arr, self.src, self.axis = arr, src, axis

    def __getitem__(self, key):
        key = list(key) if isinstance(key, tuple) else [key]
        key[self.axis] = self.src[key[self.axis]]
        return self.arr[tuple(key)]


def _inputs(cfg, seed, steps, gen_seqs):
    """Host inputs (indexable by sequence) and their device copies for the whole batch.

    With gen_seqs, only those sequences are generated; sequence b of the batch then
    holds generated sequence gen_seqs[b % len(gen_seqs)] (each listed sequence holds its own
    data), so the device runs the full-size batch while the oracle checks real sequences.
    """
    if gen_seqs is None:
        t = make_prefill_tensors(cfg, seed=seed)
        dec = make_decode_tensors(cfg, seed=seed, steps=steps)
        dev_t = {n: dev_bf16(a) for n, a in t.items()}
        dev_dec = [{n: dev_bf16(dec[n][st]) for n in dec} for st in range(steps)]
        return t, dec, dev_t, dev_dec
    import torch
    gen_seqs = list(gen_seqs)
    src = [b % len(gen_seqs) for b in range(cfg.batch)]
    assert all(src[b] == i for i, b in enumerate(gen_seqs)), "each generated sequence must map to itself"
    tg = make_prefill_tensors(cfg, seed=seed, seqs=gen_seqs)
    dg = make_decode_tensors(cfg, seed=seed, steps=steps, seqs=gen_seqs)
    dev_t = {}
    for n, a in tg.items():
        part = dev_bf16(a)
        dev_t[n] = torch.stack([part[src[b]] for b in range(cfg.batch)])
        del part
    dev_dec = []
    for st in range(steps):
        d = {}
        for n, a in dg.items():
            part = dev_bf16(a[st])
            d[n] = torch.stack([part[src[b]] for b in range(cfg.batch)])
        dev_dec.append(d)
    t = {n: _Tiled(a, src, 0) for n, a in tg.items()}
    dec = {n: _Tiled(a, src, 1) for n, a in dg.items()}
    return t, dec, dev_t, dev_dec


def run_and_check(cfg, rho, head_mode=0, forced=(0, 0), steps=2, seed=0, skip_text_only=True, check_seqs=None,
                  decode_seqs=None, schedule="auto", vision_only=False, gen_seqs=None, budget_rule=0, vision_rank=0,
                  joint_rank=False):
    import torch
    log(f"e2e {cfg.name} rho={rho} mode={head_mode} forced={forced} steps={steps} vision_only={vision_only} "
        f"budget_rule={budget_rule} vision_rank={vision_rank} joint_rank={joint_rank}")
    t, dec, dev_t, dev_dec = _inputs(cfg, seed, steps, gen_seqs)
    B, L, N = cfg.batch, cfg.layers, cfg.n_tokens
    p = bd.problem_from(cfg)
    o = bd.make_opts(head_mode=head_mode, n_sink=forced[0], n_recent=forced[1], vision_only=vision_only,
                     budget_rule=budget_rule, vision_rank=vision_rank, joint_rank=joint_rank)
    # vision-only eviction (App. B.3): text and forced positions are all kept, rho is the retained
    # share of the other vision tokens
    nfv = O.forced_vision_count(cfg.n_sys, cfg.n_vis, cfg.n_qst, *forced)
    tot = total_budget(rho, cfg.n_vis - nfv if vision_only else N, L)
    kept = bd.kept_per_sequence(p, o, tot)
    assert kept == tot + (L * (cfg.n_text + nfv) if vision_only else 0)
    buf = bd.EvictionBuffers(p, o, tot, max(steps, 1))
    q_d, k_d, v_d = dev_t["q_text"], dev_t["k"], dev_t["v"]
    check_seqs = range(B) if check_seqs is None else check_seqs
    orc = {}

    def oracle_seq(b):
        if b not in orc:
            orc[b] = O.evict_sequence(bf16_bits_to_f32(t["q_text"][b]), bf16_bits_to_f32(t["k"][b]), cfg.n_sys,
                                      cfg.n_vis, cfg.n_qst, tot, None, head_mode, *forced, vision_only=vision_only,
                                      budget_rule=budget_rule, vision_rank=vision_rank, joint_rank=joint_rank)
        return orc[b]

    if schedule == "lse_in":
        # the rows' normalisers a prefill kernel would return: here the fp64 oracle's, rounded to fp32
        # (computed once per generated sequence when the batch repeats generated sequences)
        src = t["q_text"].src if gen_seqs is not None else list(range(B))
        first = {}
        for b in range(B):
            first.setdefault(src[b], b)
        lse = np.stack([np.stack([sc["lse"] for sc in oracle_seq(first[src[b]])[0]]) for b in range(B)])
        lse = lse.astype(np.float32)
        buf.lse.copy_(torch.from_numpy(lse))
    sched = buf.evict(q_d, k_d, v_d, schedule=schedule if skip_text_only else "phases")
    log(f"  schedule {sched}")
    outs = []
    for st in range(steps):
        buf.decode(st, dev_dec[st]["q"], dev_dec[st]["k_new"], dev_dec[st]["v_new"])
        outs.append(host(buf.out).copy())
    torch.cuda.synchronize()

    g = 1 if head_mode == 0 else cfg.heads_kv
    budgets = host(buf.budgets)
    io, so = host(buf.idx_offsets), host(buf.seg_offsets)
    idx = host(buf.idx)
    kc, vc = bf16_host_bits(buf.kc), bf16_host_bits(buf.vc)
    tv = host(buf.tv_mass)
    nf = len(O.forced_positions(N, *forced))
    swaps = flips = 0
    tau = 1.0 / np.sqrt(cfg.head_dim)
    D, Hkv = cfg.head_dim, cfg.heads_kv
    assert np.all(budgets.sum(axis=1) == kept)
    decode_seqs = set(range(B) if decode_seqs is None else decode_seqs)
    for b in check_seqs:
        scores, ob, oidx = oracle_seq(b)
        assert budgets[b].sum() == kept
        masses = O.budget_masses([s["tv_mass"] for s in scores], budget_rule, cfg.n_text)
        if vision_only:
            base = cfg.n_text + nfv
            assert np.all(budgets[b] >= base)
            ok_b = budget_allowed(budgets[b] - base, ob - base, masses, tot, cfg.n_vis - nfv, 0)
        else:
            ok_b = budget_allowed(budgets[b], ob, masses, tot, N, nf)
        assert ok_b, (b, budgets[b], ob)
        flips += int(np.abs(budgets[b] - ob).sum()) // 2
        for l in range(L):
            sc = scores[l]
            assert_close_rel("tv_mass", tv[b, l], sc["tv_mass"])
            assert_close_rel("s_txt", host(buf.s_txt[b, l]), sc["s_txt"])
            assert_close_rel("w_txt", host(buf.w_txt[b, l]), sc["w_txt"])
            needs_vis = budgets[b, l] > buf.forced_or_text()
            if needs_vis or sched in ("phases", "lse_in"):
                assert_close_rel("s_vis", host(buf.s_vis[b, l]), sc["s_vis"])
            if budgets[b, l] != ob[l]:
                continue  # a rounding-cut trade: this layer's set is legitimately different
            bl = b * L + l
            bsz = int(budgets[b, l])
            agree = True
            for gg in range(g):
                gidx = idx[io[bl] + gg * bsz: io[bl] + (gg + 1) * bsz]
                vscale = (cfg.n_text if vision_rank == 0 else 1.0) if joint_rank else None
                s_ = idx_allowed(gidx, oidx[l][gg], sc["s_vis"][gg], sc["s_txt"][gg], bsz, cfg, *forced,
                                 vis_scale=vscale)
                swaps += s_
                agree = agree and s_ == 0
            if not agree:
                continue
            # compacted cache is bit-exact for the agreed sets; then decode against the oracle
            cap = bsz + max(steps, 1)
            Kc, Vc = [], []
            for h in range(Hkv):
                sel = oidx[l][0 if head_mode == 0 else h]
                base = (int(so[bl]) * Hkv + h * cap) * D
                got_k = kc[base: base + bsz * D].reshape(bsz, D)
                got_v = vc[base: base + bsz * D].reshape(bsz, D)
                assert np.array_equal(got_k, t["k"][b, l, h][sel]) and np.array_equal(got_v, t["v"][b, l, h][sel])
                Kc.append(bf16_bits_to_f32(t["k"][b, l, h][sel]))
                Vc.append(bf16_bits_to_f32(t["v"][b, l, h][sel]))
            if steps and b in decode_seqs:
                ref = O.decode_reference(bf16_bits_to_f32(dec["q"][:, b, l]), bf16_bits_to_f32(dec["k_new"][:, b, l]),
                                         bf16_bits_to_f32(dec["v_new"][:, b, l]), Kc, Vc, tau)
                for st in range(steps):
                    err = np.abs(outs[st][b, l] - ref[st]).max()
                    assert err <= DECODE_ATOL, (b, l, st, err)
    log(f"  budgets flips={flips} boundary swaps={swaps}")
    return buf


@pytest.mark.parametrize("schedule", ["auto", "phases"])
@pytest.mark.parametrize("head_mode", [0, 1])
@pytest.mark.parametrize("forced", [(0, 0), (4, 1)])
def test_small_ragged(lib, head_mode, forced, schedule):
    cfg = custom_config(batch=2, layers=4, heads_q=8, heads_kv=4, head_dim=128, n_sys=6, n_vis=230, n_qst=21)
    for rho in (0.05, 0.2, 0.6, 1.0):
        run_and_check(cfg, rho, head_mode, forced, steps=3, seed=1, schedule=schedule)


def test_gqa_video_small(lib):
    cfg = custom_config(name="vid", batch=2, layers=3, heads_q=28, heads_kv=4, head_dim=128, n_sys=16, n_vis=512,
                        n_qst=48, frames=4)
    for rho in (0.05, 0.1):
        run_and_check(cfg, rho, 0, steps=3, seed=2)


@pytest.mark.parametrize("rho", CONFIGS["tiny"].rhos)
def test_tiny_config(lib, rho):
    run_and_check(CONFIGS["tiny"], rho, steps=1, seed=0)


@pytest.mark.parametrize("rho", CONFIGS["llava15"].rhos)
def test_llava15_config(lib, rho):
    run_and_check(CONFIGS["llava15"], rho, steps=8, seed=0)


def test_llava15_all_layers_scored(lib):
    run_and_check(CONFIGS["llava15"], 0.05, steps=0, seed=4, skip_text_only=False)


def test_edge_shapes(lib):
    # no question text (no text->vision mass: uniform budgets, position ties), no vision, no system text
    run_and_check(custom_config(name="noq", batch=1, layers=3, heads_q=4, heads_kv=2, n_sys=9, n_vis=70, n_qst=0),
                  0.3, steps=2)
    run_and_check(custom_config(name="nov", batch=1, layers=3, heads_q=4, heads_kv=2, n_sys=9, n_vis=0, n_qst=12),
                  0.5, steps=2)
    run_and_check(custom_config(name="nos", batch=1, layers=3, heads_q=4, heads_kv=4, head_dim=64, n_sys=0, n_vis=90,
                                n_qst=17), 0.25, steps=2)
    # budget 0 everywhere, then decode over the appended tokens only
    run_and_check(custom_config(name="zero", batch=1, layers=2, heads_q=4, heads_kv=4, n_sys=3, n_vis=40, n_qst=5),
                  0.0, steps=3)


# ----------------------------------------------------------------------------- vision-only eviction
@pytest.mark.parametrize("head_mode", [0, 1])
@pytest.mark.parametrize("forced", [(0, 0), (4, 1)])
def test_vision_only_small(lib, head_mode, forced):
    cfg = custom_config(batch=2, layers=4, heads_q=8, heads_kv=4, head_dim=128, n_sys=6, n_vis=230, n_qst=21)
    for rho in (0.0, 0.05, 0.3, 1.0):
        run_and_check(cfg, rho, head_mode, forced, steps=3, seed=5, vision_only=True)
    # no system text: the forced sink is a vision token, kept beside the vision budget like the text
    cfg = custom_config(name="nos", batch=1, layers=3, heads_q=4, heads_kv=4, head_dim=64, n_sys=0, n_vis=90,
                        n_qst=17)
    run_and_check(cfg, 0.1, head_mode, forced, steps=2, seed=6, vision_only=True)


@pytest.mark.parametrize("rho", [0.05, 0.1, 0.2])
def test_vision_only_llava15(lib, rho):
    run_and_check(CONFIGS["llava15"], rho, steps=4, seed=0, vision_only=True)


def test_vision_only_gqa_video(lib):
    cfg = custom_config(name="vid", batch=2, layers=3, heads_q=28, heads_kv=4, head_dim=128, n_sys=16, n_vis=512,
                        n_qst=48, frames=4)
    run_and_check(cfg, 0.1, 0, steps=3, seed=2, vision_only=True)


# ----------------------------------------------------------------------------- normalisers from the prefill
@pytest.mark.parametrize("head_mode", [0, 1])
@pytest.mark.parametrize("forced", [(0, 0), (4, 1)])
def test_lse_in_small(lib, head_mode, forced):
    cfg = custom_config(batch=2, layers=4, heads_q=8, heads_kv=4, head_dim=128, n_sys=6, n_vis=230, n_qst=21)
    for rho in (0.05, 0.3, 1.0):
        run_and_check(cfg, rho, head_mode, forced, steps=2, seed=7, schedule="lse_in")
    run_and_check(cfg, 0.1, head_mode, forced, steps=2, seed=8, schedule="lse_in", vision_only=True)


def test_lse_in_shapes(lib):
    # GQA video, d64 tiny, no question text, no vision, no system text
    run_and_check(custom_config(name="vid", batch=2, layers=3, heads_q=28, heads_kv=4, head_dim=128, n_sys=16,
                                n_vis=512, n_qst=48, frames=4), 0.1, steps=2, seed=2, schedule="lse_in")
    run_and_check(CONFIGS["tiny"], 0.5, steps=1, seed=0, schedule="lse_in")
    run_and_check(custom_config(name="noq", batch=1, layers=3, heads_q=4, heads_kv=2, n_sys=9, n_vis=70, n_qst=0),
                  0.3, steps=2, schedule="lse_in")
    run_and_check(custom_config(name="nov", batch=1, layers=3, heads_q=4, heads_kv=2, n_sys=9, n_vis=0, n_qst=12),
                  0.5, steps=2, schedule="lse_in")
    run_and_check(custom_config(name="nos", batch=1, layers=3, heads_q=4, heads_kv=4, head_dim=64, n_sys=0,
                                n_vis=90, n_qst=17), 0.25, steps=2, schedule="lse_in")


def test_lse_in_long_text(lib):
    # text keys staged in two chunks (they do not fit beside the normalisers in 64 KB of LDS):
    # GQA with 320 text tokens, and one head per KV head with the 13B shape's 291
    run_and_check(custom_config(name="lt2", batch=1, layers=2, heads_q=4, heads_kv=2, head_dim=128, n_sys=40,
                                n_vis=300, n_qst=280), 0.3, steps=2, seed=9, schedule="lse_in")
    run_and_check(custom_config(name="lt1", batch=1, layers=2, heads_q=2, heads_kv=2, head_dim=128, n_sys=35,
                                n_vis=200, n_qst=256), 0.2, steps=2, seed=10, schedule="lse_in")


def test_lse_in_llava15(lib):
    run_and_check(CONFIGS["llava15"], 0.1, steps=4, seed=0, schedule="lse_in")


# ----------------------------------------------------------------------------- the paper's variants
@pytest.mark.parametrize("budget_rule", [0, 1, 2])
@pytest.mark.parametrize("vision_rank", [0, 1])
@pytest.mark.parametrize("joint_rank", [False, True])
def test_variants_small(lib, budget_rule, vision_rank, joint_rank):
    """Layer budgets by TV mass / equally / by TT mass; TWR or the plain attention sum; with or without TPR."""
    cfg = custom_config(batch=2, layers=4, heads_q=8, heads_kv=4, head_dim=128, n_sys=6, n_vis=230, n_qst=21)
    for rho in (0.05, 0.3):
        for forced in [(0, 0), (4, 1)]:
            run_and_check(cfg, rho, 0, forced, steps=2, seed=9, budget_rule=budget_rule, vision_rank=vision_rank,
                          joint_rank=joint_rank)
    run_and_check(cfg, 0.1, 1, (0, 0), steps=2, seed=10, budget_rule=budget_rule, vision_rank=vision_rank,
                  joint_rank=joint_rank, schedule="lse_in")


def test_variants_llava15(lib):
    cfg = CONFIGS["llava15"]
    run_and_check(cfg, 0.05, steps=2, seed=0, budget_rule=2, vision_rank=1, joint_rank=True)
    run_and_check(cfg, 0.2, steps=2, seed=0, budget_rule=1, vision_rank=0, joint_rank=True)
    run_and_check(cfg, 0.1, steps=2, seed=0, budget_rule=1, vision_rank=1, vision_only=True)
