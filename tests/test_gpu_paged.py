"""Paged cache and continuous batching on the GPU.

* page assignment: the table and the page count equal a host prefix-sum construction;
* paged compaction: the rows gathered back through the table are bit-identical to the
  contiguous cache, and no pool row outside the batch's pages is written;
* paged decode at a uniform step: outputs and appended rows bit-identical to the
  contiguous decode (the same arithmetic over other addresses);
* continuous batching: two prefill batches of different lengths share one pool and
  decode as one batch, each sequence at its own step, with sequences joining late and
  retiring early; every active output against the fp64 oracle, idle ones untouched.
"""

import numpy as np
import pytest

import oracle.tgvkv_oracle as O
from paper_2606_03075_amd import binding as bd
from tests.gpu_util import DECODE_ATOL, bf16_host_bits, dev_bf16, host, idx_allowed, log
from workloads import bf16_bits_to_f32, make_prefill_tensors, total_budget
from workloads.configs import CONFIGS, custom_config

pytestmark = pytest.mark.gpu

SENTINEL = 0x7FC1  # a bf16 NaN pattern no copy produces from the finite workloads


def _fill_pool(pool):
    import torch
    pool.k_pool.view(torch.int16).fill_(SENTINEL)
    pool.v_pool.view(torch.int16).fill_(SENTINEL)


def _gather(pool_bits, table_row, rows, page):
    """Rows [0, rows) of one (sequence, layer) from a pool [n_pages][Hkv][P][D] -> [Hkv][rows][D]."""
    out = []
    for n0 in range(0, rows, page):
        pg = int(table_row[n0 // page])
        assert pg >= 0, "row without a page"
        out.append(pool_bits[pg][:, : min(page, rows - n0)])
    Hkv, D = pool_bits.shape[1], pool_bits.shape[3]
    return np.concatenate(out, axis=1) if out else np.zeros((Hkv, 0, D), pool_bits.dtype)


def _contig(cache_bits, so, bl, Hkv, D, cap, rows):
    base = int(so[bl]) * Hkv * D
    seg = cache_bits[base: base + Hkv * cap * D].reshape(Hkv, cap, D)
    return seg[:, :rows]


# ----------------------------------------------------------------------------- page assignment
@pytest.mark.parametrize("B,L", [(3, 500), (2, 37), (1, 1)])
@pytest.mark.parametrize("page,reserve", [(1, 0), (16, 5), (64, 3)])
def test_page_table_kernel(lib, page, reserve, B, L):
    """Segments split over many workgroups (1500 segments: 167 groups of 9; 74: 9 groups, the last
    one short; 1: one group); budgets summing to the total per sequence."""
    import torch
    N, total = 700, 600
    prob = bd.make_problem(B, L, 4, 2, 128, 10, 600, 90)
    rng = np.random.default_rng(11 + page)
    budgets = np.stack([rng.multinomial(total, rng.dirichlet(np.ones(L) * 0.3)) for _ in range(B)]).astype(np.int32)
    budgets[0, :] = 0
    budgets[0, -1] = total  # one layer takes the whole budget
    width, pool_bound = bd.page_plan(prob, None, total, reserve, page)
    n_free = pool_bound + 7
    free = rng.permutation(n_free + 100)[:n_free].astype(np.int32)
    d_budgets = torch.from_numpy(budgets).cuda()
    d_free = torch.from_numpy(free).cuda()
    table = torch.full((B * L, width), -7, dtype=torch.int32, device="cuda")
    used = torch.zeros((1,), dtype=torch.int64, device="cuda")
    log(f"page table B={B} L={L} page={page} reserve={reserve} width={width} bound={pool_bound}")
    bd.tgvkv_page_table(prob, None, d_budgets, total, reserve, page, d_free, table, used)
    torch.cuda.synchronize()
    need = -(-(budgets.reshape(-1).astype(np.int64) + reserve) // page)
    start = np.concatenate([[0], np.cumsum(need)])
    expect = np.full((B * L, width), -1, np.int32)
    for i in range(B * L):
        expect[i, : need[i]] = free[start[i]: start[i] + need[i]]
    assert int(used.item()) == int(need.sum()) <= pool_bound
    assert np.array_equal(host(table), expect)


# ----------------------------------------------------------------------------- paged vs contiguous
def _evict(cfg, rho, reserve, seed, head_mode=0, forced=(0, 0), vision_only=False):
    t = make_prefill_tensors(cfg, seed=seed)
    dev = {n: dev_bf16(a) for n, a in t.items()}
    p = bd.problem_from(cfg)
    o = bd.make_opts(head_mode=head_mode, n_sink=forced[0], n_recent=forced[1], vision_only=vision_only)
    nfv = O.forced_vision_count(cfg.n_sys, cfg.n_vis, cfg.n_qst, *forced)
    tot = total_budget(rho, cfg.n_vis - nfv if vision_only else cfg.n_tokens, cfg.layers)
    buf = bd.EvictionBuffers(p, o, tot, reserve)
    buf.evict(dev["q_text"], dev["k"], dev["v"])
    return t, dev, buf


def _decode_inputs(rng, B, L, H, Hkv, D):
    def bits(shape):
        x = rng.standard_normal(shape).astype(np.float32)
        return (x.view(np.uint32) >> 16).astype(np.uint16)
    return bits((B, L, H, D)), bits((B, L, Hkv, D)), bits((B, L, Hkv, D))


def _paged_matches_contiguous(cfg, rho, page, steps, seed, shuffle=True, **kw):
    import torch
    t, dev, buf = _evict(cfg, rho, steps, seed, **kw)
    p, o = buf.problem, buf.opts
    B, L, H, Hkv, D = cfg.batch, cfg.layers, cfg.heads_q, cfg.heads_kv, cfg.head_dim
    width, bound = bd.page_plan(p, o, buf.total_budget, steps, page)
    n_pages = bound + 5
    pool = bd.PagedPool(Hkv, D, page, n_pages)
    _fill_pool(pool)
    if shuffle:
        pool.free = list(np.random.default_rng(seed).permutation(n_pages))
    log(f"paged {cfg.name} rho={rho} page={page} steps={steps} width={width} pages<={bound} {kw}")
    table = pool.admit(buf, dev["k"], dev["v"])
    torch.cuda.synchronize()
    budgets, so, tab = host(buf.budgets), host(buf.seg_offsets), host(table)
    used = set(int(x) for x in tab.reshape(-1) if x >= 0)
    assert len(used) == n_pages - len(pool.free), "pages used twice or counted wrong"
    kc, vc = bf16_host_bits(buf.kc), bf16_host_bits(buf.vc)
    kp, vp = bf16_host_bits(pool.k_pool), bf16_host_bits(pool.v_pool)
    for bl in range(B * L):
        bsz = int(budgets.reshape(-1)[bl])
        assert np.count_nonzero(tab[bl] >= 0) == -(-(bsz + steps) // page)
        assert np.array_equal(_gather(kp, tab[bl], bsz, page), _contig(kc, so, bl, Hkv, D, bsz + steps, bsz))
        assert np.array_equal(_gather(vp, tab[bl], bsz, page), _contig(vc, so, bl, Hkv, D, bsz + steps, bsz))
    untouched = [i for i in range(n_pages) if i not in used]
    assert np.all(kp[untouched] == SENTINEL) and np.all(vp[untouched] == SENTINEL)

    # decode: every sequence at the same step, against the contiguous decode, bit for bit
    rng = np.random.default_rng(seed + 100)
    out_p = torch.empty_like(buf.out)
    steps_d = torch.zeros((B,), dtype=torch.int32, device="cuda")
    for st in range(steps):
        q, kn, vn = (dev_bf16(x) for x in _decode_inputs(rng, B, L, H, Hkv, D))
        buf.decode(st, q, kn, vn)
        steps_d.fill_(st)
        pool.decode(p, o, table, buf.budgets, steps, steps_d, q, kn, vn, out_p, buf.ws_decode,
                    unit_order=buf.unit_order if st % 2 else None)
        torch.cuda.synchronize()
        assert torch.equal(out_p, buf.out), f"step {st}: paged decode differs from contiguous"
    kc, vc = bf16_host_bits(buf.kc), bf16_host_bits(buf.vc)
    kp, vp = bf16_host_bits(pool.k_pool), bf16_host_bits(pool.v_pool)
    for bl in range(B * L):
        rows = int(budgets.reshape(-1)[bl]) + steps
        assert np.array_equal(_gather(kp, tab[bl], rows, page), _contig(kc, so, bl, Hkv, D, rows, rows))
        assert np.array_equal(_gather(vp, tab[bl], rows, page), _contig(vc, so, bl, Hkv, D, rows, rows))
    assert np.all(kp[untouched] == SENTINEL) and np.all(vp[untouched] == SENTINEL)
    return pool, table


@pytest.mark.parametrize("page", [1, 16, 64])
@pytest.mark.parametrize("rho", [0.0, 0.05, 0.3, 1.0])
def test_paged_matches_contiguous_small(lib, page, rho):
    cfg = custom_config(batch=2, layers=4, heads_q=8, heads_kv=4, head_dim=128, n_sys=6, n_vis=230, n_qst=21)
    _paged_matches_contiguous(cfg, rho, page, steps=3, seed=1)


def test_paged_head_mode_gqa_d64(lib):
    cfg = custom_config(name="g", batch=2, layers=3, heads_q=16, heads_kv=2, head_dim=64, n_sys=4, n_vis=300,
                        n_qst=19)
    _paged_matches_contiguous(cfg, 0.1, 32, steps=5, seed=3, head_mode=1, forced=(4, 1))
    _paged_matches_contiguous(cfg, 0.1, 8, steps=2, seed=4, vision_only=True, shuffle=False)


def test_paged_llava15(lib):
    cfg = CONFIGS["llava15"]
    _paged_matches_contiguous(cfg, 0.05, 16, steps=8, seed=0)


def test_paged_table_width_limit(lib):
    """A segment of 4096 one-row pages, the widest table the library takes (its page ids are
    staged in LDS): every token kept (N = 4094) plus 2 decode steps."""
    import torch
    cfg = custom_config(name="wide", batch=1, layers=1, heads_q=2, heads_kv=1, head_dim=64, n_sys=10, n_vis=4070,
                        n_qst=14)
    width, _ = bd.page_plan(bd.problem_from(cfg), None, cfg.n_tokens, 2, 1)
    assert width == 4096
    _paged_matches_contiguous(cfg, 1.0, 1, steps=2, seed=6)


# ----------------------------------------------------------------------------- continuous batching
def _oracle_cache(t, cfg, tot, b, gpu_idx, io, budgets, L):
    """Per layer: oracle retained rows (K, V per KV head) where the GPU's set matches the oracle's."""
    scores, ob, oidx = O.evict_sequence(bf16_bits_to_f32(t["q_text"][b]), bf16_bits_to_f32(t["k"][b]), cfg.n_sys,
                                        cfg.n_vis, cfg.n_qst, tot)
    caches = {}
    for l in range(L):
        bl = b * L + l
        if budgets[b, l] != ob[l]:
            continue
        gidx = gpu_idx[io[bl]: io[bl] + budgets[b, l]]
        if idx_allowed(gidx, oidx[l][0], scores[l]["s_vis"][0], scores[l]["s_txt"][0], int(ob[l]), cfg) != 0:
            continue
        sel = oidx[l][0]
        caches[l] = ([bf16_bits_to_f32(t["k"][b, l, h][sel]) for h in range(cfg.heads_kv)],
                     [bf16_bits_to_f32(t["v"][b, l, h][sel]) for h in range(cfg.heads_kv)])
    return caches


def test_continuous_batching(lib):
    """Batch A (2 sequences) starts decoding; batch B (2 sequences of another length) is admitted
    two steps later into the same pool; A's second sequence retires after three steps.  One paged
    decode launch per iteration serves all four slots, each at its own step."""
    import torch
    R, page = 6, 16
    L, H, Hkv, D = 3, 8, 2, 128
    cfg_a = custom_config(name="a", batch=2, layers=L, heads_q=H, heads_kv=Hkv, head_dim=D, n_sys=5, n_vis=150,
                          n_qst=12)
    cfg_b = custom_config(name="b", batch=2, layers=L, heads_q=H, heads_kv=Hkv, head_dim=D, n_sys=9, n_vis=90,
                          n_qst=30)
    ta, deva, bufa = _evict(cfg_a, 0.2, R, seed=21)
    tb, devb, bufb = _evict(cfg_b, 0.3, R, seed=22)
    wa, pa = bd.page_plan(bufa.problem, None, bufa.total_budget, R, page)
    wb, pb = bd.page_plan(bufb.problem, None, bufb.total_budget, R, page)
    pool = bd.PagedPool(Hkv, D, page, pa + pb + 3)
    _fill_pool(pool)
    pool.free = list(np.random.default_rng(5).permutation(pool.n_pages))
    tab_a = pool.admit(bufa, deva["k"], deva["v"])
    tab_b = pool.admit(bufb, devb["k"], devb["v"])
    width = max(wa, wb)
    pad = lambda t: torch.nn.functional.pad(t, (0, width - t.shape[1]), value=-1)
    table = torch.cat([pad(tab_a), pad(tab_b)]).contiguous()
    budgets = torch.cat([bufa.budgets, bufb.budgets]).contiguous()
    prob = bd.make_problem(4, L, H, Hkv, D, 1, 0, 0)
    ws = torch.empty((max(1, bd.workspace_size(prob, None, bd.CALL_DECODE)),), dtype=torch.uint8, device="cuda")
    schedule = [[0, 0, -1, -1], [1, 1, -1, -1], [2, 2, 0, 0], [3, R, 1, 1], [4, -1, 2, 2], [5, -1, 3, 3]]
    rng = np.random.default_rng(9)
    out = torch.empty((4, L, H, D), dtype=torch.float32, device="cuda")
    outs, inputs = [], []
    for it, steps in enumerate(schedule):
        q, kn, vn = _decode_inputs(rng, 4, L, H, Hkv, D)
        inputs.append((q, kn, vn))
        out.fill_(float("nan"))
        steps_d = torch.tensor(steps, dtype=torch.int32, device="cuda")
        log(f"continuous batching iteration {it} steps {steps}")
        pool.decode(prob, None, table, budgets, R, steps_d, dev_bf16(q), dev_bf16(kn), dev_bf16(vn), out, ws)
        outs.append(host(out).copy())
    torch.cuda.synchronize()

    tau = 1.0 / np.sqrt(D)
    checked = 0
    for slot, (t, cfg, buf, b) in enumerate([(ta, cfg_a, bufa, 0), (ta, cfg_a, bufa, 1), (tb, cfg_b, bufb, 0),
                                            (tb, cfg_b, bufb, 1)]):
        caches = _oracle_cache(t, cfg, buf.total_budget, b, host(buf.idx), host(buf.idx_offsets), host(buf.budgets),
                               L)
        its = [i for i, s in enumerate(schedule) if 0 <= s[slot] < R]
        assert [schedule[i][slot] for i in its] == list(range(len(its)))
        for i, s in enumerate(schedule):
            if not 0 <= s[slot] < R:
                assert np.all(np.isnan(outs[i][slot])), f"idle slot {slot} written at iteration {i}"
        for l, (Kc, Vc) in caches.items():
            ref = O.decode_reference(np.stack([bf16_bits_to_f32(inputs[i][0][slot, l]) for i in its]),
                                     np.stack([bf16_bits_to_f32(inputs[i][1][slot, l]) for i in its]),
                                     np.stack([bf16_bits_to_f32(inputs[i][2][slot, l]) for i in its]), Kc, Vc, tau)
            for j, i in enumerate(its):
                err = np.abs(outs[i][slot, l] - ref[j]).max()
                assert err <= DECODE_ATOL, (slot, l, i, err)
                checked += 1
    log(f"  continuous batching: {checked} (slot, layer, step) outputs checked against the oracle")
    assert checked >= 30
    # a retired sequence's pages go back to the pool
    n_free = len(pool.free)
    pool.release(tab_a[L:2 * L])
    assert len(pool.free) == n_free + int((host(tab_a[L:2 * L]) >= 0).sum())
