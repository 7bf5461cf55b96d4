"""Stage-by-stage GPU parity: each kernel gets inputs that the test draws itself, identical for both sides.

No GPU output ever feeds the oracle: budgets are checked on seeded mass vectors,
selection on seeded score vectors (with ties), compaction on seeded index sets,
decode on a seeded cache; scoring on seeded workloads.
"""

import numpy as np
import pytest

import oracle.tgvkv_oracle as O
from paper_2606_03075_amd import binding as bd
from tests.gpu_util import (DECODE_ATOL, assert_close_rel, bf16_host_bits, dev_bf16, host, log,
                            oracle_scores)
from workloads import bf16_bits_to_f32, f32_to_bf16_bits, make_prefill_tensors
from workloads.configs import CONFIGS, custom_config

pytestmark = pytest.mark.gpu


def _torch():
    import torch
    return torch


# ----------------------------------------------------------------------------- budgets
def _mass_cases(rng, L):
    yield rng.random(L).astype(np.float32)
    yield np.full(L, 0.37, np.float32)
    yield np.zeros(L, np.float32)
    m = rng.random(L).astype(np.float32) * 1e-3
    m[0] = 50.0
    yield m
    m = rng.random(L).astype(np.float32)
    m[::3] = 0.0
    yield m
    m = rng.random(L).astype(np.float32)
    m[1 % L] = np.nan
    m[2 % L] = -1.0
    m[3 % L] = np.inf
    yield m
    yield (rng.integers(1, 4, L) / 4).astype(np.float32)   # many equal fractions


def _longest_first(budgets):
    """Decode dispatch order: rank-major over sequences, each sequence's layers by (budget desc, layer asc)."""
    B, L = budgets.shape
    out = np.empty(B * L, np.int32)
    for b in range(B):
        ranks = sorted(range(L), key=lambda l: (-int(budgets[b, l]), l))
        for r, l in enumerate(ranks):
            out[r * B + b] = b * L + l
    return out


@pytest.mark.parametrize("budget_rule", [0, 1, 2])
@pytest.mark.parametrize("L,N,n_sink,n_recent", [(32, 2979, 0, 0), (28, 8256, 4, 1), (5, 13, 0, 0),
                                                 (1, 168, 0, 0), (40, 3171, 4, 1), (7, 3, 1, 1),
                                                 (257, 97, 2, 1), (512, 40, 0, 0)])
def test_budget_kernel_exact(lib, L, N, n_sink, n_recent, budget_rule):
    torch = _torch()
    rng = np.random.default_rng(L * 1000 + N)
    cases = list(_mass_cases(rng, L))
    B = len(cases)
    masses = np.stack(cases)
    p = bd.make_problem(B, L, 4, 4, 128, 1, N - 2, 1)
    o = bd.make_opts(n_sink=n_sink, n_recent=n_recent, budget_rule=budget_rule)
    nt = 2
    nf = len(O.forced_positions(N, n_sink, n_recent))
    for total in sorted({0, 1, L, (L * N) // 20, (L * N) // 3, L * N - 1, L * N}):
        for reserve in (0, 7):
            tv = torch.from_numpy(masses).cuda()
            budgets = torch.empty((B, L), dtype=torch.int32, device="cuda")
            io = torch.empty(B * L + 1, dtype=torch.int64, device="cuda")
            so = torch.empty(B * L + 1, dtype=torch.int64, device="cuda")
            order = torch.full((B * L,), -1, dtype=torch.int32, device="cuda")
            bd.tgvkv_budget(p, o, tv, total, reserve, budgets, io, so, unit_order=order)
            torch.cuda.synchronize()
            gb = host(budgets)
            for b in range(B):
                ob = O.layer_budgets(O.budget_masses(masses[b].astype(np.float64), budget_rule, nt), total, N, nf)
                assert np.array_equal(gb[b], ob), (b, total, gb[b], ob)
            assert np.array_equal(host(io), O.flat_offsets(gb.reshape(-1)))
            assert np.array_equal(host(so), O.flat_offsets(gb.reshape(-1) + reserve))
            assert np.array_equal(host(order), _longest_first(gb))


@pytest.mark.parametrize("L,ns,nv,nq,n_sink,n_recent", [(32, 35, 2880, 64, 0, 0), (28, 16, 8192, 48, 4, 1),
                                                          (5, 0, 13, 3, 4, 1), (7, 2, 3, 1, 1, 1),
                                                          (3, 9, 0, 12, 0, 0)])
def test_budget_kernel_vision_only_exact(lib, L, ns, nv, nq, n_sink, n_recent):
    """Vision-only eviction (App. B.3): the vision budget is shared out, every layer adds its text."""
    torch = _torch()
    rng = np.random.default_rng(L * 100 + nv)
    cases = list(_mass_cases(rng, L))
    B = len(cases)
    masses = np.stack(cases)
    nt = ns + nq
    p = bd.make_problem(B, L, 4, 4, 128, ns, nv, nq)
    o = bd.make_opts(n_sink=n_sink, n_recent=n_recent, vision_only=True)
    nfv = O.forced_vision_count(ns, nv, nq, n_sink, n_recent)
    cap = L * (nv - nfv)
    for total in sorted({v for v in (0, 1, L, cap // 20, cap // 3, cap - 1, cap) if 0 <= v <= cap}):
        for reserve in (0, 5):
            tv = torch.from_numpy(masses).cuda()
            budgets = torch.empty((B, L), dtype=torch.int32, device="cuda")
            io = torch.empty(B * L + 1, dtype=torch.int64, device="cuda")
            so = torch.empty(B * L + 1, dtype=torch.int64, device="cuda")
            order = torch.full((B * L,), -1, dtype=torch.int32, device="cuda")
            bd.tgvkv_budget(p, o, tv, total, reserve, budgets, io, so, unit_order=order)
            torch.cuda.synchronize()
            gb = host(budgets)
            assert np.array_equal(host(order), _longest_first(gb))
            for b in range(B):
                ob = O.vision_only_budgets(masses[b].astype(np.float64), total, nt, nv, nfv)
                assert np.array_equal(gb[b], ob), (b, total, gb[b], ob)
            assert np.array_equal(host(io), O.flat_offsets(gb.reshape(-1)))
            assert np.array_equal(host(so), O.flat_offsets(gb.reshape(-1) + reserve))


# ----------------------------------------------------------------------------- selection
@pytest.mark.parametrize("rank", ["tpr", "joint_twr", "joint_sum"])
@pytest.mark.parametrize("head_mode", [0, 1])
# the last shape is longer than the kernel's LDS key buffer (12288 keys): keys are re-read from memory
@pytest.mark.parametrize("shape", [(3, 40, 5), (0, 30, 4), (8, 144, 16), (35, 576, 40), (2, 0, 9), (16, 1300, 48),
                                   (16, 13000, 48)])
@pytest.mark.parametrize("forced", [(0, 0), (4, 1)])
def test_select_kernel_exact(lib, head_mode, shape, forced, rank):
    torch = _torch()
    ns, nv, nq = shape
    N, nt = ns + nv + nq, ns + nq
    B, L, Hkv = 2, 6, 2
    g = 1 if head_mode == 0 else Hkv
    rng = np.random.default_rng(N * 7 + head_mode)
    # scores on a coarse grid (many exact ties), including -0.0 and +0.0
    sv = (rng.integers(0, 6, (B, L, g, nv)) / 8).astype(np.float32)
    st = (rng.integers(0, 6, (B, L, g, nt)) / 8).astype(np.float32)
    sv[sv == 0] = np.where(rng.random(int((sv == 0).sum())) < 0.5, -0.0, 0.0)
    # budgets covering every regime: forced only, text top-k, all text + vision top-k, everything
    bud = np.zeros((B, L), np.int64)
    choices = [0, 1, min(3, N), max(0, nt - 1), nt, min(N, nt + 1), min(N, nt + nv // 3), N]
    for b in range(B):
        for l in range(L):
            bud[b, l] = choices[(b * L + l) % len(choices)]
    io = O.flat_offsets((bud * g).reshape(-1))
    p = bd.make_problem(B, L, 4, Hkv, 128, ns, nv, nq)
    joint = rank != "tpr"
    vrank = 1 if rank == "joint_sum" else 0
    o = bd.make_opts(head_mode=head_mode, n_sink=forced[0], n_recent=forced[1], vision_rank=vrank, joint_rank=joint)
    vscale = float(nt) if vrank == 0 else 1.0   # scores on a grid of 1/8: the scaled values are exact in fp32
    d_sv = torch.from_numpy(sv).cuda() if nv else torch.zeros(1, device="cuda")
    d_st = torch.from_numpy(st).cuda() if nt else torch.zeros(1, device="cuda")
    d_b = torch.from_numpy(bud.astype(np.int32)).cuda()
    d_io = torch.from_numpy(io).cuda()
    d_idx = torch.full((max(1, int(io[-1])),), -1, dtype=torch.int32, device="cuda")
    bd.tgvkv_select(p, o, d_sv, d_st, d_b, d_io, d_idx)
    torch.cuda.synchronize()
    gi = host(d_idx)
    for b in range(B):
        for l in range(L):
            bl = b * L + l
            for gg in range(g):
                if joint:
                    want = O.joint_select(sv[b, l, gg].astype(np.float64), st[b, l, gg].astype(np.float64),
                                          int(bud[b, l]), ns, nv, nq, *forced, vis_scale=vscale)
                else:
                    want = O.tpr_select(sv[b, l, gg].astype(np.float64), st[b, l, gg].astype(np.float64),
                                        int(bud[b, l]), ns, nv, nq, *forced)
                got = gi[io[bl] + gg * bud[b, l]: io[bl] + (gg + 1) * bud[b, l]]
                assert np.array_equal(got, want), (b, l, gg, bud[b, l], got[:12], want[:12])


# ----------------------------------------------------------------------------- compaction
@pytest.mark.parametrize("head_mode,D", [(0, 128), (1, 128), (0, 64)])
def test_compact_bit_exact(lib, head_mode, D):
    torch = _torch()
    B, L, Hkv, ns, nv, nq, reserve = 2, 3, 4, 5, 200, 11, 3
    N = ns + nv + nq
    g = 1 if head_mode == 0 else Hkv
    rng = np.random.default_rng(D + head_mode)
    k = rng.integers(0, 65536, (B, L, Hkv, N, D), dtype=np.uint16)
    v = rng.integers(0, 65536, (B, L, Hkv, N, D), dtype=np.uint16)
    total = 170
    bud = np.stack([O.layer_budgets(rng.random(L), total, N) for _ in range(B)])
    bud[0, 0] = 0
    bud[0, 1] += total - bud[0].sum()
    io = O.flat_offsets((bud * g).reshape(-1))
    so = O.flat_offsets((bud + reserve).reshape(-1))
    idx = np.zeros(int(io[-1]), np.int32)
    sets = {}
    for b in range(B):
        for l in range(L):
            for gg in range(g):
                s = np.sort(rng.choice(N, int(bud[b, l]), replace=False)).astype(np.int32)
                sets[(b, l, gg)] = s
                idx[io[b * L + l] + gg * bud[b, l]: io[b * L + l] + (gg + 1) * bud[b, l]] = s
    p = bd.make_problem(B, L, Hkv, Hkv, D, ns, nv, nq)
    o = bd.make_opts(head_mode=head_mode)
    slots = int(so[-1])
    kc = torch.zeros(slots * Hkv * D, dtype=torch.bfloat16, device="cuda")
    vc = torch.zeros_like(kc)
    bd.tgvkv_compact(p, o, dev_bf16(k), dev_bf16(v), torch.from_numpy(idx).cuda(),
                     torch.from_numpy(bud.astype(np.int32)).cuda(), torch.from_numpy(io).cuda(),
                     torch.from_numpy(so).cuda(), total, reserve, kc, vc)
    torch.cuda.synchronize()
    hk, hv = bf16_host_bits(kc), bf16_host_bits(vc)
    for b in range(B):
        for l in range(L):
            bl = b * L + l
            cap = int(bud[b, l]) + reserve
            for h in range(Hkv):
                s = sets[(b, l, 0 if head_mode == 0 else h)]
                base = (int(so[bl]) * Hkv + h * cap) * D
                got_k = hk[base: base + len(s) * D].reshape(len(s), D)
                got_v = hv[base: base + len(s) * D].reshape(len(s), D)
                ck, cv = O.compact_slice(k[b, l], v[b, l], [s] if head_mode == 0 else
                                         [sets[(b, l, x)] for x in range(Hkv)], head_mode)
                assert np.array_equal(got_k, ck[h]) and np.array_equal(got_v, cv[h])
                # reserved decode slots untouched
                assert not hk[base + len(s) * D: base + cap * D].any()
    # the same compaction dispatched in a shuffled unit order writes the same cache
    kc2, vc2 = torch.zeros_like(kc), torch.zeros_like(vc)
    perm = torch.from_numpy(rng.permutation(B * L).astype(np.int32)).cuda()
    bd.tgvkv_compact(p, o, dev_bf16(k), dev_bf16(v), torch.from_numpy(idx).cuda(),
                     torch.from_numpy(bud.astype(np.int32)).cuda(), torch.from_numpy(io).cuda(),
                     torch.from_numpy(so).cuda(), total, reserve, kc2, vc2, unit_order=perm)
    torch.cuda.synchronize()
    # compare bit patterns: the random 16-bit rows include NaN encodings
    assert np.array_equal(bf16_host_bits(kc2), hk) and np.array_equal(bf16_host_bits(vc2), hv)


# ----------------------------------------------------------------------------- decode
@pytest.mark.parametrize("H,Hkv,D,B,L", [(4, 4, 128, 2, 3), (28, 4, 128, 1, 2), (8, 2, 64, 1, 4),
                                         (32, 32, 128, 4, 32), (16, 1, 128, 1, 1), (12, 4, 128, 1, 2),
                                         (10, 2, 64, 2, 2)])
def test_decode_kernel(lib, H, Hkv, D, B, L):
    torch = _torch()
    rng = np.random.default_rng(H * 100 + D)
    reserve, T = 6, 4
    N = 700
    bud = rng.integers(0, 300, (B, L))
    bud[0, 0] = 0
    so = O.flat_offsets((bud + reserve).reshape(-1))
    slots = int(so[-1])
    cache_k = f32_to_bf16_bits(rng.standard_normal((slots * Hkv * D,)).astype(np.float32))
    cache_v = f32_to_bf16_bits(rng.standard_normal((slots * Hkv * D,)).astype(np.float32))
    q = f32_to_bf16_bits(rng.standard_normal((T, B, L, H, D)).astype(np.float32) * 1.5)
    kn = f32_to_bf16_bits(rng.standard_normal((T, B, L, Hkv, D)).astype(np.float32))
    vn = f32_to_bf16_bits(rng.standard_normal((T, B, L, Hkv, D)).astype(np.float32))
    p = bd.make_problem(B, L, H, Hkv, D, 1, N - 2, 1)
    o = bd.make_opts()
    kc, vc = dev_bf16(cache_k), dev_bf16(cache_v)
    out = torch.empty((B, L, H, D), dtype=torch.float32, device="cuda")
    ws = torch.empty(max(1, bd.workspace_size(p, o, bd.CALL_DECODE)), dtype=torch.uint8, device="cuda")
    d_b = torch.from_numpy(bud.astype(np.int32)).cuda()
    d_so = torch.from_numpy(so).cuda()
    tau = 1.0 / np.sqrt(D)
    worst = 0.0
    # a second copy of the cache decoded in a shuffled unit order must give the same bits
    kc2, vc2 = kc.clone(), vc.clone()
    out2 = torch.empty_like(out)
    perm = torch.from_numpy(rng.permutation(B * L).astype(np.int32)).cuda()
    for t in range(T):
        bd.tgvkv_decode_attn(p, o, kc, vc, d_b, d_so, reserve, t, dev_bf16(q[t]), dev_bf16(kn[t]),
                             dev_bf16(vn[t]), out, ws)
        bd.tgvkv_decode_attn(p, o, kc2, vc2, d_b, d_so, reserve, t, dev_bf16(q[t]), dev_bf16(kn[t]),
                             dev_bf16(vn[t]), out2, ws, unit_order=perm)
        torch.cuda.synchronize()
        assert torch.equal(out, out2), "decode output depends on the dispatch order"
        got = host(out)
        for b in range(B):
            for l in range(L):
                bl = b * L + l
                n, cap = int(bud[b, l]), int(bud[b, l]) + reserve
                Kc, Vc = [], []
                for h in range(Hkv):
                    base = (int(so[bl]) * Hkv + h * cap) * D
                    kk = bf16_bits_to_f32(cache_k[base: base + n * D].reshape(n, D))
                    vv = bf16_bits_to_f32(cache_v[base: base + n * D].reshape(n, D))
                    kk = np.concatenate([kk, bf16_bits_to_f32(kn[:t + 1, b, l, h])])
                    vv = np.concatenate([vv, bf16_bits_to_f32(vn[:t + 1, b, l, h])])
                    Kc.append(kk)
                    Vc.append(vv)
                ref = O.decode_attention(bf16_bits_to_f32(q[t, b, l]), Kc, Vc, tau)
                err = np.abs(got[b, l] - ref).max()
                worst = max(worst, float(err))
                assert err <= DECODE_ATOL, (t, b, l, err)
    # the kernel appended every step's token into the cache
    hk = bf16_host_bits(kc)
    for b in range(B):
        for l in range(L):
            bl = b * L + l
            n, cap = int(bud[b, l]), int(bud[b, l]) + reserve
            for h in range(Hkv):
                base = (int(so[bl]) * Hkv + h * cap + n) * D
                assert np.array_equal(hk[base: base + T * D].reshape(T, D), kn[:, b, l, h])
    assert torch.equal(kc, kc2) and torch.equal(vc, vc2)
    log(f"decode H={H} Hkv={Hkv} D={D}: max abs err {worst:.2e}")


# ----------------------------------------------------------------------------- scoring
SCORE_SHAPES = {
    "mha_d128_ragged": custom_config(batch=2, layers=2, heads_q=4, heads_kv=4, head_dim=128, n_sys=5, n_vis=150,
                                     n_qst=19),
    "gqa7_d128": custom_config(batch=1, layers=2, heads_q=14, heads_kv=2, head_dim=128, n_sys=16, n_vis=300,
                               n_qst=48),
    "mha_d64_tiny": CONFIGS["tiny"],
    "nsys0": custom_config(batch=1, layers=2, heads_q=4, heads_kv=2, head_dim=64, n_sys=0, n_vis=77, n_qst=33),
    "nqst0": custom_config(batch=1, layers=2, heads_q=4, heads_kv=2, head_dim=128, n_sys=9, n_vis=70, n_qst=0),
    "nvis0": custom_config(batch=1, layers=1, heads_q=4, heads_kv=4, head_dim=128, n_sys=7, n_vis=0, n_qst=21),
    "many_rows": custom_config(batch=1, layers=1, heads_q=16, heads_kv=1, head_dim=128, n_sys=12, n_vis=130,
                               n_qst=40),
    "long_text": custom_config(batch=1, layers=1, heads_q=2, heads_kv=2, head_dim=128, n_sys=35, n_vis=200,
                               n_qst=300),
    # four 16-row blocks per KV head (the vision sweep's own launch shape)
    "four_blocks": custom_config(batch=2, layers=2, heads_q=4, heads_kv=4, head_dim=128, n_sys=7, n_vis=333,
                                 n_qst=61),
    "four_blocks_gqa_d64": custom_config(batch=1, layers=2, heads_q=8, heads_kv=4, head_dim=64, n_sys=3, n_vis=201,
                                         n_qst=29),
    # three 16-row blocks per KV head (two slots over two key parts)
    "three_blocks": custom_config(batch=1, layers=2, heads_q=4, heads_kv=4, head_dim=128, n_sys=11, n_vis=180,
                                  n_qst=40),
    # twelve 16-row blocks per KV head (four slots per wave)
    "twelve_blocks_gqa4": custom_config(batch=1, layers=2, heads_q=8, heads_kv=2, head_dim=128, n_sys=6, n_vis=260,
                                        n_qst=45),
    "twelve_blocks_gqa4_d64": custom_config(batch=1, layers=2, heads_q=8, heads_kv=2, head_dim=64, n_sys=2,
                                            n_vis=190, n_qst=37),
    # sixteen 16-row blocks of one head (the 13B stress shape's row plan, text pass fed from the
    # sweep's registers): causal question-key blocks skipped, full and diagonal
    "sixteen_blocks_long_question": custom_config(batch=1, layers=2, heads_q=2, heads_kv=2, head_dim=128, n_sys=35,
                                                  n_vis=150, n_qst=250),
    # seven system-key blocks staged for that text pass; and one past its limit of 128 system keys
    "ten_blocks_long_system": custom_config(batch=1, layers=2, heads_q=3, heads_kv=3, head_dim=128, n_sys=100,
                                            n_vis=90, n_qst=150),
    "ten_blocks_system_past_limit": custom_config(batch=1, layers=1, heads_q=2, heads_kv=2, head_dim=128,
                                                  n_sys=140, n_vis=50, n_qst=150),
}


@pytest.mark.parametrize("name", sorted(SCORE_SHAPES))
@pytest.mark.parametrize("head_mode", [0, 1])
def test_score_matches_oracle(lib, name, head_mode):
    torch = _torch()
    cfg = SCORE_SHAPES[name]
    log(f"score {name} mode={head_mode}")
    phases = bd.SCORE_ALL
    t = make_prefill_tensors(cfg, seed=3, names=("q_text", "k"))
    p = bd.problem_from(cfg)
    o = bd.make_opts(head_mode=head_mode)
    buf = bd.EvictionBuffers(p, o, 0, 1)
    q_d, k_d = dev_bf16(t["q_text"]), dev_bf16(t["k"])
    buf.score(q_d, k_d, phases)
    torch.cuda.synchronize()
    worst = {}
    for b in range(cfg.batch):
        for l in range(cfg.layers):
            r = oracle_scores(t["q_text"][b, l], t["k"][b, l], cfg, head_mode)
            worst["lse"] = assert_close_rel("lse", host(buf.lse[b, l]), r["lse"], atol=1e-4)
            worst["s_txt"] = assert_close_rel("s_txt", host(buf.s_txt[b, l]), r["s_txt"])
            worst["w_txt"] = assert_close_rel("w_txt", host(buf.w_txt[b, l]), r["w_txt"])
            worst["tv_mass"] = assert_close_rel("tv_mass", host(buf.tv_mass[b, l]), r["tv_mass"])
            worst["s_vis"] = assert_close_rel("s_vis", host(buf.s_vis[b, l]), r["s_vis"])
    log(f"  max rel err: {worst}")
    # determinism: a second run gives identical bits
    s1 = host(buf.s_vis).copy(), host(buf.s_txt).copy(), host(buf.tv_mass).copy()
    buf.score(q_d, k_d, phases)
    torch.cuda.synchronize()
    assert np.array_equal(s1[0], host(buf.s_vis)) and np.array_equal(s1[1], host(buf.s_txt))
    assert np.array_equal(s1[2], host(buf.tv_mass))


def _ramp_inputs(cfg, direction, seed=11):
    """Text queries all close to one direction u and keys whose component along u ramps over the
    sequence, so every text row's logits climb (or fall) along the keys by about 30 in base-2 units:
    the statistics sweep's running reference max moves many times and its sums hold terms far above 1
    between moves."""
    rng = np.random.default_rng(seed)
    B, L, H, Hkv, D, N = cfg.batch, cfg.layers, cfg.heads_q, cfg.heads_kv, cfg.head_dim, cfg.n_tokens
    u = rng.standard_normal(D).astype(np.float32)
    u /= np.linalg.norm(u)
    q = 12.0 * u + 0.2 * rng.standard_normal((B, L, H, cfg.n_text, D)).astype(np.float32)
    a = np.linspace(-4.0, 16.0, N, dtype=np.float32)
    if direction == "falling":
        a = a[::-1].copy()
    elif direction == "zigzag":
        a = np.where(np.arange(N) % 97 < 48, a, -a)
    k = a[:, None] * u + 0.3 * rng.standard_normal((B, L, Hkv, N, D)).astype(np.float32)
    return f32_to_bf16_bits(q.astype(np.float32)), f32_to_bf16_bits(k.astype(np.float32))


@pytest.mark.parametrize("direction", ["rising", "falling", "zigzag"])
@pytest.mark.parametrize("shape", ["gqa7_d128", "twelve_blocks_gqa4", "four_blocks", "sixteen_blocks_long_question"])
def test_score_moving_max(lib, shape, direction):
    """Logits that climb along the keys: the reference max of every row moves again and again, with
    up to 2^8-sized terms summed between moves; the scores still match the oracle."""
    torch = _torch()
    cfg = SCORE_SHAPES[shape]
    log(f"score moving max {shape} {direction}")
    qb, kb = _ramp_inputs(cfg, direction)
    p = bd.problem_from(cfg)
    buf = bd.EvictionBuffers(p, bd.make_opts(), 0, 1)
    buf.score(dev_bf16(qb), dev_bf16(kb), bd.SCORE_ALL)
    torch.cuda.synchronize()
    for b in range(cfg.batch):
        for l in range(cfg.layers):
            r = oracle_scores(qb[b, l], kb[b, l], cfg, 0)
            assert_close_rel("lse", host(buf.lse[b, l]), r["lse"], atol=1e-4)
            assert_close_rel("s_txt", host(buf.s_txt[b, l]), r["s_txt"])
            assert_close_rel("w_txt", host(buf.w_txt[b, l]), r["w_txt"])
            assert_close_rel("tv_mass", host(buf.tv_mass[b, l]), r["tv_mass"])
            assert_close_rel("s_vis", host(buf.s_vis[b, l]), r["s_vis"])
