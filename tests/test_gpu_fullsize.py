"""Parity at the full workload sizes, in the launch configuration the benchmark times.

The whole batch runs on the GPU exactly as bench.py runs it (text statistics,
budgets, vision scores only for layers whose budget reaches past the text,
selection, compaction, every decode step); the oracle checks whole sequences
(every layer, so the budgets are checked too) where it finishes in seconds, and
properties that hold at any size everywhere.
"""

import numpy as np
import pytest

from tests.gpu_util import log
from tests.test_gpu_e2e import run_and_check
from workloads.configs import CONFIGS, depth_profile

pytestmark = pytest.mark.gpu


def _properties(buf, cfg):
    budgets = buf.budgets.cpu().numpy()
    io = buf.idx_offsets.cpu().numpy()
    idx = buf.idx.cpu().numpy()
    L = cfg.layers
    for b in range(cfg.batch):
        for l in range(L):
            bl = b * L + l
            sel = idx[io[bl]: io[bl + 1]]
            assert len(sel) == budgets[b, l]
            assert np.all(np.diff(sel) > 0) and (len(sel) == 0 or (sel[0] >= 0 and sel[-1] < cfg.n_tokens))
            text = np.concatenate([np.arange(cfg.n_sys), cfg.n_sys + cfg.n_vis + np.arange(cfg.n_qst)])
            if budgets[b, l] > cfg.n_text:
                assert np.isin(text, sel).all()
            else:
                assert np.isin(sel, text).all()


@pytest.mark.parametrize("recipe", ["iid", "depth"])
def test_llavanext_full(lib, recipe):
    """batch 4 x 32 layers x 32 heads, 35 + 2880 + 64 tokens, 5 % retention, 128 decode steps; i.i.d.
    text queries (every layer's budget passes N_t) and the depth profile (budgets spread over an
    order of magnitude, a third of the layers keep text only), both as the benchmark runs them."""
    cfg = CONFIGS["llavanext"] if recipe == "iid" else depth_profile(CONFIGS["llavanext"])
    buf = run_and_check(cfg, cfg.rhos[0], steps=cfg.decode_steps, seed=0, check_seqs=range(cfg.batch),
                        decode_seqs=[0])
    _properties(buf, cfg)
    log(f"  llavanext budgets seq0: {buf.budgets[0].tolist()}")


@pytest.mark.parametrize("rho", CONFIGS["qwen2vl_video"].rhos)
def test_qwen2vl_video_full(lib, rho):
    """batch 8 x 28 layers x 28 heads over 4 KV heads, 16 + 8192 + 48 tokens, 128 decode steps."""
    cfg = CONFIGS["qwen2vl_video"]
    buf = run_and_check(cfg, rho, steps=cfg.decode_steps, seed=0, check_seqs=[0, 7], decode_seqs=[0])
    _properties(buf, cfg)


def test_qwen2vl_video_full_lse_in(lib):
    """The one-sweep schedule (every text row's normaliser given, as a prefill kernel returns it)
    at the full Qwen2-VL batch: the mass-collecting vision sweep runs split over two shares of the
    vision keys there (896 units), and the TV masses, scores, budgets, sets and cache must still
    match.  Sequences 0 and 7 are generated and checked; the batch repeats them."""
    cfg = CONFIGS["qwen2vl_video"]
    buf = run_and_check(cfg, cfg.rhos[0], steps=8, seed=0, check_seqs=[0, 7], decode_seqs=[0], gen_seqs=[0, 7],
                        schedule="lse_in")
    _properties(buf, cfg)


def test_llavanext_full_lse_in(lib):
    """The one-sweep schedule at the benchmark's LLaVA-NeXT batch (4096 units, one row slot per
    wave in the mass-collecting vision sweep, the unit's text keys staged in LDS for the text
    pass): TV masses, scores, budgets, sets and cache against the oracle.  Sequences 0 and 3 are
    generated and checked; the batch repeats them."""
    cfg = CONFIGS["llavanext"]
    buf = run_and_check(cfg, cfg.rhos[0], steps=8, seed=0, check_seqs=[0, 3], decode_seqs=[0], gen_seqs=[0, 3],
                        schedule="lse_in")
    _properties(buf, cfg)


def test_llavanext_full_vision_only(lib):
    """Vision-only eviction (App. B.3) at the benchmark's LLaVA-NeXT batch: every layer keeps all
    its text and a TVB share of 5 % of the vision tokens, so compaction and decode carry more rows.
    Sequences 0 and 3 are generated and checked; the batch repeats them."""
    cfg = CONFIGS["llavanext"]
    buf = run_and_check(cfg, cfg.rhos[0], steps=8, seed=0, check_seqs=[0, 3], decode_seqs=[0], gen_seqs=[0, 3],
                        vision_only=True)
    budgets = buf.budgets.cpu().numpy()
    assert np.all(budgets >= cfg.n_text)  # all text kept in every layer


def test_llavanext_full_no_tpr(lib):
    """Text and vision ranked together (TPR off, an ablation of Table 5) at the benchmark's
    LLaVA-NeXT batch: every layer needs its vision scores, and the joint top-k runs over all
    2979 positions.  Sequences 0 and 3 are generated and checked; the batch repeats them."""
    cfg = CONFIGS["llavanext"]
    run_and_check(cfg, cfg.rhos[0], steps=4, seed=0, check_seqs=[0, 3], decode_seqs=[0], gen_seqs=[0, 3],
                  joint_rank=True)


@pytest.mark.parametrize("recipe", ["iid", "depth"])
def test_stress13b_full(lib, recipe):
    """batch 16 x 40 layers x 40 heads, 35 + 2880 + 256 tokens, 5 % retention, 256 decode steps.

    With i.i.d. text queries every layer's budget (158 or 159) is below N_t = 291, so every layer
    takes the text-top-k case of Eq. (10); with the depth profile the shallowest layers keep all
    text plus vision tokens.

    Sequences 0 and 15 are generated and checked against the oracle (every layer); the other
    sequences of the batch repeat them (even ones sequence 0, odd ones sequence 15), so the
    device runs the full-size batch, and sequences holding the same data must agree exactly.
    """
    cfg = CONFIGS["stress13b"] if recipe == "iid" else depth_profile(CONFIGS["stress13b"])
    buf = run_and_check(cfg, cfg.rhos[0], steps=cfg.decode_steps, seed=0, check_seqs=[0, 15], decode_seqs=[0],
                        gen_seqs=[0, 15])
    _properties(buf, cfg)
    budgets = buf.budgets.cpu().numpy()
    io = buf.idx_offsets.cpu().numpy()
    idx = buf.idx.cpu().numpy()
    L = cfg.layers
    for b in range(2, cfg.batch):
        ref = 0 if b % 2 == 0 else 15
        assert np.array_equal(budgets[b], budgets[ref]), b
        for l in range(L):
            got = idx[io[b * L + l]: io[b * L + l + 1]]
            want = idx[io[ref * L + l]: io[ref * L + l + 1]]
            assert np.array_equal(got, want), (b, l)
    log(f"  stress13b budgets seq0: {buf.budgets[0].tolist()}")


@pytest.mark.parametrize("name", ["llavanext", "qwen2vl_video"])
def test_paged_full(lib, name):
    """The bench's paged launch configuration at full size (16-row pages, longest-first order):
    the pool gathered through the table equals the contiguous cache bit for bit, and 16 decode
    steps with a per-sequence step vector equal the contiguous decode bit for bit (one query
    head per KV head at LLaVA-NeXT, the matrix-core decode at Qwen2-VL's seven)."""
    import torch
    from paper_2606_03075_amd import binding as bd
    from tests.test_gpu_e2e import _inputs
    from workloads import total_budget

    cfg = CONFIGS[name]
    T, page = 16, 16
    t, dec, dev_t, dev_dec = _inputs(cfg, 0, T, [0, 1])
    p = bd.problem_from(cfg)
    tot = total_budget(cfg.rhos[0], cfg.n_tokens, cfg.layers)
    buf = bd.EvictionBuffers(p, None, tot, T)
    buf.evict(dev_t["q_text"], dev_t["k"], dev_t["v"])
    width, n_pages = bd.page_plan(p, None, tot, T, page)
    pool = bd.PagedPool(cfg.heads_kv, cfg.head_dim, page, n_pages)
    pool.free = list(np.random.default_rng(0).permutation(n_pages))
    table = pool.admit(buf, dev_t["k"], dev_t["v"])
    del dev_t
    out_p = torch.empty_like(buf.out)
    for st in range(T):
        buf.decode(st, dev_dec[st]["q"], dev_dec[st]["k_new"], dev_dec[st]["v_new"])
        steps = torch.full((cfg.batch,), st, dtype=torch.int32, device="cuda")
        pool.decode(p, None, table, buf.budgets, T, steps, dev_dec[st]["q"], dev_dec[st]["k_new"],
                    dev_dec[st]["v_new"], out_p, buf.ws_decode, unit_order=buf.unit_order)
        torch.cuda.synchronize()
        assert torch.equal(out_p, buf.out), f"step {st}"
    # every row of every (sequence, layer): the pool through the table against the contiguous segments
    Hkv, D, L = cfg.heads_kv, cfg.head_dim, cfg.layers
    budgets = buf.budgets.cpu().numpy().reshape(-1)
    so = buf.seg_offsets.cpu().numpy()
    tab = table.cpu().numpy()
    kc = buf.kc.view(torch.int16)
    vc = buf.vc.view(torch.int16)
    kp = pool.k_pool.view(torch.int16)
    vp = pool.v_pool.view(torch.int16)
    for bl in range(cfg.batch * L):
        rows = int(budgets[bl]) + T
        n_pg = -(-rows // page)
        pages = torch.from_numpy(tab[bl, :n_pg].astype(np.int64)).cuda()
        base = int(so[bl]) * Hkv * D
        for src, pool_t in ((kc, kp), (vc, vp)):
            seg = src[base: base + Hkv * rows * D].view(Hkv, rows, D)
            got = pool_t[pages].permute(1, 0, 2, 3).reshape(Hkv, n_pg * page, D)[:, :rows]
            assert torch.equal(got, seg), bl
    log(f"  {name} paged: {cfg.batch * L} segments, {n_pages} pages, table width {width}")
