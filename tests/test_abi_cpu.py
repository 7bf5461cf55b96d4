"""The C-ABI library loads, exports what include/tgvkv.h declares, and rejects bad calls on the host.

No compute call is made here: every call below must fail validation (or have
nothing to do) before the library touches the HIP runtime.  Fake non-null
pointers are used only when no GPU is present, so a validation bug can never
reach a kernel launch on real hardware.
"""

import ctypes
import os
import re

import pytest

from paper_2606_03075_amd import binding as bd

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _gpu():
    try:
        import torch
        return torch.cuda.is_available()
    except Exception:
        return False


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(bd.LIB_PATH):
        from paper_2606_03075_amd import build
        build.build()
    return bd.load_library()


def declared_functions(header="tgvkv.h"):
    with open(os.path.join(ROOT, "include", header)) as f:
        text = f.read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(tgvkv_[a-z0-9_]+)\s*\(", text)))


def test_exports_every_declared_symbol(lib):
    headers = sorted(f for f in os.listdir(os.path.join(ROOT, "include")) if f.endswith(".h"))
    assert headers == ["tgvkv.h", "tgvkv_ceiling.h"], headers
    names = declared_functions()
    assert set(bd.EXPORTS) <= set(names) and len(names) == len(bd.EXPORTS), names
    ceiling = declared_functions("tgvkv_ceiling.h")
    assert sorted(ceiling) == sorted(bd.CEILING_EXPORTS), ceiling
    for n in names + ceiling:
        assert hasattr(lib, n), n
    assert lib.tgvkv_abi_version() == bd.ABI_VERSION == 8
    for st in (0, -1, -2, -3, -4, -5):
        assert lib.tgvkv_status_string(st)
    assert lib.tgvkv_status_string(7) == b"unknown status"


def P(**kw):
    base = dict(batch=1, layers=2, heads_q=4, heads_kv=2, head_dim=128, n_sys=3, n_vis=40, n_qst=5)
    base.update(kw)
    return bd.make_problem(**base)


def test_workspace_size(lib):
    assert bd.workspace_size(P(), None, bd.CALL_SCORE) > 0
    assert bd.workspace_size(P(head_dim=96), None, bd.CALL_SCORE) == 0
    assert bd.workspace_size(P(heads_q=3), None, bd.CALL_SCORE) == 0
    assert bd.workspace_size(P(), None, 9) == 0
    # decode needs a split workspace only for small (b, l, kv-head) counts
    assert bd.workspace_size(P(), None, bd.CALL_DECODE) > 0
    assert bd.workspace_size(P(batch=64, layers=32, heads_q=32, heads_kv=32), None, bd.CALL_DECODE) == 0


@pytest.mark.skipif(_gpu(), reason="fake pointers are used only where no GPU exists")
def test_validation_before_any_launch(lib):
    fake = ctypes.c_void_p(0x10000)
    odd = ctypes.c_void_p(0x10008)
    big = ctypes.c_size_t(1 << 40)
    s = ctypes.c_void_p(0)
    ok = ctypes.byref(P())
    opts = bd.make_opts()
    # invalid problems
    for bad, code in [(P(batch=-1), -1), (P(layers=0), -1), (P(heads_q=3), -1), (P(n_sys=0, n_vis=0, n_qst=0), -1),
                      (P(head_dim=96), -2), (P(layers=600), -2), (P(heads_q=64, heads_kv=2), -2)]:
        r = lib.tgvkv_score(ctypes.byref(bad), None, 7, fake, fake, fake, fake, fake, fake, fake, None, fake, big, s)
        assert r == code, (bad.head_dim, r)
    assert lib.tgvkv_score(None, None, 7, fake, fake, fake, fake, fake, fake, fake, None, fake, big, s) == -1
    # bad options
    for o in (bd.make_opts(head_mode=2), bd.make_opts(n_sink=-1), bd.make_opts(sm_scale=float("nan")),
              bd.TgvkvOpts(0.0, 0, 0, 0, 2), bd.make_opts(budget_rule=3), bd.make_opts(vision_rank=2),
              bd.TgvkvOpts(0.0, 0, 0, 0, 0, 0, 0, 2), bd.make_opts(vision_only=True, joint_rank=True)):
        assert lib.tgvkv_score(ok, ctypes.byref(o), 7, fake, fake, fake, fake, fake, fake, fake, None, fake, big,
                               s) == -1
    # phases, null and misaligned pointers, workspace
    assert lib.tgvkv_score(ok, None, 0, fake, fake, fake, fake, fake, fake, fake, None, fake, big, s) == -1
    assert lib.tgvkv_score(ok, None, 8, fake, fake, fake, fake, fake, fake, fake, None, fake, big, s) == -1
    # bit 8 is not a phase (it was the removed persistent schedule's flag): with any phases, refused
    assert lib.tgvkv_score(ok, None, 8 | 4, fake, fake, fake, fake, fake, fake, fake, None, fake, big, s) == -1
    assert lib.tgvkv_score(ok, None, 8 | 1, fake, fake, fake, fake, fake, fake, fake, None, fake, big, s) == -1
    assert lib.tgvkv_score(ok, None, 8 | 7, fake, fake, fake, fake, fake, fake, fake, fake, fake, big, s) == -1
    # normalisers from the caller: only with exactly TEXT|VISION, no budgets
    assert lib.tgvkv_score(ok, None, 16, fake, fake, fake, fake, fake, fake, fake, None, fake, big, s) == -1
    assert lib.tgvkv_score(ok, None, 16 | 7, fake, fake, fake, fake, fake, fake, fake, None, fake, big, s) == -1
    assert lib.tgvkv_score(ok, None, 16 | 2, fake, fake, fake, fake, fake, fake, fake, None, fake, big, s) == -1
    assert lib.tgvkv_score(ok, None, 16 | 6, fake, fake, fake, fake, fake, fake, fake, fake, fake, big, s) == -1
    assert lib.tgvkv_score(ok, None, 16 | 8 | 6, fake, fake, fake, fake, fake, fake, fake, None, fake, big, s) == -1
    assert lib.tgvkv_score(ok, None, 32, fake, fake, fake, fake, fake, fake, fake, None, fake, big, s) == -1
    assert lib.tgvkv_score(ok, None, 7, None, fake, fake, fake, fake, fake, fake, None, fake, big, s) == -1
    assert lib.tgvkv_score(ok, None, 7, odd, fake, fake, fake, fake, fake, fake, None, fake, big, s) == -1
    assert lib.tgvkv_score(ok, None, 2, fake, fake, fake, None, fake, fake, fake, None, fake, big, s) == -1
    assert lib.tgvkv_score(ok, None, 4, fake, fake, fake, fake, fake, fake, None, None, fake, big, s) == -1
    assert lib.tgvkv_score(ok, None, 7, fake, fake, fake, fake, fake, fake, fake, None, None, big, s) == -3
    assert lib.tgvkv_score(ok, None, 7, fake, fake, fake, fake, fake, fake, fake, None, fake, 16, s) == -3
    # budgets: capacity and arguments
    L, N = 2, 48
    assert lib.tgvkv_budget(ok, None, fake, L * N + 1, 0, fake, fake, fake, None, s) == -4
    assert lib.tgvkv_budget(ok, None, fake, -1, 0, fake, fake, fake, None, s) == -1
    assert lib.tgvkv_budget(ok, None, fake, 10, -1, fake, fake, fake, None, s) == -1
    assert lib.tgvkv_budget(ok, None, None, 10, 0, fake, fake, fake, None, s) == -1
    # vision-only eviction: the budget counts vision tokens, at most L * n_vis
    vo = ctypes.byref(bd.make_opts(vision_only=True))
    Nv = 40
    assert lib.tgvkv_budget(ok, vo, fake, L * Nv + 1, 0, fake, fake, fake, None, s) == -4
    assert lib.tgvkv_compact(ok, vo, fake, fake, fake, fake, fake, fake, L * Nv + 1, 0, fake, fake, None, s) == -4
    # select / compact / decode arguments
    assert lib.tgvkv_select(ok, None, fake, fake, None, fake, fake, s) == -1
    assert lib.tgvkv_select(ok, None, None, fake, fake, fake, fake, s) == -1
    assert lib.tgvkv_compact(ok, None, fake, fake, fake, fake, fake, fake, L * N + 1, 0, fake, fake, None, s) == -4
    assert lib.tgvkv_compact(ok, None, fake, fake, fake, fake, fake, fake, 10, 0, fake, None, None, s) == -1
    assert lib.tgvkv_compact(ok, None, fake, odd, fake, fake, fake, fake, 10, 0, fake, fake, None, s) == -1
    dec = lambda step, kn, out, ws, n: lib.tgvkv_decode_attn(ok, None, fake, fake, fake, fake, 4, step, fake, kn, fake,
                                                             out, ws, n, None, s)
    assert dec(4, fake, fake, fake, big) == -4
    assert dec(-1, fake, fake, fake, big) == -4
    assert dec(0, fake, None, fake, big) == -1
    assert dec(0, fake, fake, None, 0) == -3
    # the scratch-free variant validates the same way, before looking up its buffer
    na = lambda prob, step, kn, out: lib.tgvkv_decode_attn_noalloc(prob, None, fake, fake, fake, fake, 4, step, fake,
                                                                   kn, fake, out, None, s)
    assert na(ok, 4, fake, fake) == -4
    assert na(ok, -1, fake, fake) == -4
    assert na(ok, 0, None, fake) == -1
    assert na(ok, 0, fake, None) == -1
    assert na(ok, 0, odd, fake) == -1
    assert na(ctypes.byref(P(heads_q=3)), 0, fake, fake) == -1
    assert na(ctypes.byref(P(head_dim=96)), 0, fake, fake) == -2


def _plan(problem, opts, total, reserve, page):
    return bd.page_plan(problem, opts, total, reserve, page)


def _splits(total, layers, cap):
    """Every way of writing total as layers parts in [0, cap] (tiny cases only)."""
    if layers == 1:
        if 0 <= total <= cap:
            yield (total,)
        return
    for b in range(0, min(cap, total) + 1):
        for rest in _splits(total - b, layers - 1, cap):
            yield (b,) + rest


@pytest.mark.parametrize("total,reserve,page", [(0, 0, 1), (10, 4, 8), (37, 3, 4), (96, 0, 16), (50, 9, 2),
                                                (96, 5, 64)])
def test_page_plan_bounds_every_budget_split(lib, total, reserve, page):
    """The plan's width is the largest segment's page count over every budget split the
    budget call can produce, and the pool bound covers the worst split's total."""
    prob = P(layers=2, n_sys=3, n_vis=40, n_qst=5)  # N = 48
    width, pool = _plan(prob, None, total, reserve, page)
    need = lambda b: -(-(b + reserve) // page)
    splits = list(_splits(total, 2, 48))
    assert width == max(1, max(max(need(b) for b in sp) for sp in splits))
    assert pool >= max(sum(need(b) for b in sp) for sp in splits)
    assert pool <= (total + 2 * (reserve + page - 1)) // page


def test_page_plan_vision_only(lib):
    """Vision-only eviction keeps N_t text tokens per layer beside the vision budget."""
    prob = P(layers=2, n_sys=3, n_vis=40, n_qst=5)
    vo = bd.make_opts(vision_only=True)
    width, pool = _plan(prob, vo, 10, 4, 8)
    assert width == -(-(8 + 10 + 4) // 8)            # b_max = N_t + min(n_vis, V_tot)
    assert pool == (2 * 8 + 10 + 2 * (4 + 7)) // 8   # K = L*N_t + V_tot


def test_page_plan_rejects_bad_arguments(lib):
    out_w, out_p = ctypes.c_int32(), ctypes.c_int64()
    ok = ctypes.byref(P())
    for page in (0, 3, 6, 8192, -4):
        assert lib.tgvkv_page_plan(ok, None, 10, 4, page, ctypes.byref(out_w), ctypes.byref(out_p)) == -1
    assert lib.tgvkv_page_plan(ok, None, 2 * 48 + 1, 4, 8, ctypes.byref(out_w), ctypes.byref(out_p)) == -4
    assert lib.tgvkv_page_plan(ok, None, 10, -1, 8, ctypes.byref(out_w), ctypes.byref(out_p)) == -1
    assert lib.tgvkv_page_plan(ok, None, 10, 4, 8, None, ctypes.byref(out_p)) == -1
    # a segment wider than 4096 pages is beyond the LDS copy of its page ids
    assert lib.tgvkv_page_plan(ok, None, 48, 5000, 1, ctypes.byref(out_w), ctypes.byref(out_p)) == -2


@pytest.mark.skipif(_gpu(), reason="fake pointers are used only where no GPU exists")
def test_paged_validation_before_any_launch(lib):
    fake = ctypes.c_void_p(0x10000)
    odd = ctypes.c_void_p(0x10008)
    big = ctypes.c_size_t(1 << 40)
    s = ctypes.c_void_p(0)
    ok = ctypes.byref(P())
    width, pool = _plan(P(), None, 10, 4, 8)
    # page table: width and pool bound, page size, pointers
    assert lib.tgvkv_page_table(ok, None, fake, 10, 4, 8, fake, pool, fake, width - 1, fake, s) == -4
    assert lib.tgvkv_page_table(ok, None, fake, 10, 4, 8, fake, pool - 1, fake, width, fake, s) == -4
    assert lib.tgvkv_page_table(ok, None, fake, 10, 4, 6, fake, pool, fake, width, fake, s) == -1
    assert lib.tgvkv_page_table(ok, None, fake, 10, 4, 8, fake, pool, fake, 5000, fake, s) == -2
    assert lib.tgvkv_page_table(ok, None, None, 10, 4, 8, fake, pool, fake, width, fake, s) == -1
    assert lib.tgvkv_page_table(ok, None, fake, 10, 4, 8, fake, pool, fake, width, None, s) == -1
    assert lib.tgvkv_page_table(ok, None, fake, 2 * 48 + 1, 4, 8, fake, 999, fake, 64, fake, s) == -4
    # paged compaction: the table must hold b_max rows
    cp = lambda table, width, page, vpool, n_pages: lib.tgvkv_compact_paged(
        ok, None, fake, fake, fake, fake, fake, 10, table, width, page, fake, vpool, n_pages, None, s)
    assert cp(fake, 1, 8, fake, 64) == -4
    assert cp(fake, 2, 8, fake, 0) == -1
    assert cp(fake, 2, 8, odd, 64) == -1
    assert cp(None, 2, 8, fake, 64) == -1
    assert cp(fake, 2, 5, fake, 64) == -1
    assert cp(fake, 2, 8, fake, 1 << 31) == -2
    # paged decode: steps are required, workspace as for contiguous decode
    assert lib.tgvkv_decode_attn_paged(ok, None, fake, fake, 64, 8, fake, 2, fake, 4, None, fake, fake, fake, fake,
                                       fake, big, None, s) == -1
    assert lib.tgvkv_decode_attn_paged(ok, None, fake, fake, 64, 8, fake, 2, fake, 4, fake, fake, fake, fake, fake,
                                       None, 0, None, s) == -3
    assert lib.tgvkv_decode_attn_paged(ok, None, fake, fake, 64, 12, fake, 2, fake, 4, fake, fake, fake, fake, fake,
                                       fake, big, None, s) == -1
    assert lib.tgvkv_decode_attn_paged(ok, None, odd, fake, 64, 8, fake, 2, fake, 4, fake, fake, fake, fake, fake,
                                       fake, big, None, s) == -1
    assert lib.tgvkv_decode_attn_paged(ok, None, fake, fake, 64, 8, fake, 0, fake, 4, fake, fake, fake, fake, fake,
                                       fake, big, None, s) == -1


@pytest.mark.parametrize("shape", [(3, 40, 5), (0, 30, 4), (6, 0, 9), (2, 7, 0)])
@pytest.mark.parametrize("forced", [(0, 0), (4, 1), (50, 50)])
def test_sizes_follow_the_oracle(lib, shape, forced):
    """K and the vision threshold from tgvkv_sizes against the oracle's budgets and forced positions."""
    import numpy as np
    import oracle.tgvkv_oracle as O
    ns, nv, nq = shape
    L, N, nt = 3, ns + nv + nq, ns + nq
    prob = P(layers=L, n_sys=ns, n_vis=nv, n_qst=nq)
    n_forced = len(O.forced_positions(N, *forced))
    nfv = O.forced_vision_count(ns, nv, nq, *forced)
    masses = np.array([0.2, 0.5, 0.3])
    for total in sorted({0, 1, L * N // 4, L * N}):
        o = bd.make_opts(n_sink=forced[0], n_recent=forced[1])
        assert bd.tgvkv_sizes(prob, o, total) == (total, nt + nfv)
        o = bd.make_opts(n_sink=forced[0], n_recent=forced[1], joint_rank=True)
        assert bd.tgvkv_sizes(prob, o, total) == (total, n_forced)
    vo = bd.make_opts(n_sink=forced[0], n_recent=forced[1], vision_only=True)
    cap = L * (nv - nfv)
    for vtot in sorted({v for v in (0, 1, cap) if v <= cap}):
        kept = int(O.vision_only_budgets(masses, vtot, nt, nv, nfv).sum())
        assert bd.tgvkv_sizes(prob, vo, vtot) == (kept, nt + nfv)
    with pytest.raises(bd.TgvkvError):
        bd.tgvkv_sizes(prob, vo, cap + 1)


def test_sizes_reject_bad_arguments(lib):
    kept, thr = ctypes.c_int64(-7), ctypes.c_int32(-7)
    ok = ctypes.byref(P())  # L = 2, N = 48
    assert lib.tgvkv_sizes(ok, None, -1, ctypes.byref(kept), ctypes.byref(thr)) == -1
    assert lib.tgvkv_sizes(ok, None, 2 * 48 + 1, ctypes.byref(kept), ctypes.byref(thr)) == -4
    assert lib.tgvkv_sizes(ctypes.byref(P(heads_q=3)), None, 0, ctypes.byref(kept), ctypes.byref(thr)) == -1
    assert lib.tgvkv_sizes(None, None, 0, ctypes.byref(kept), ctypes.byref(thr)) == -1
    assert (kept.value, thr.value) == (-7, -7)
    assert lib.tgvkv_sizes(ok, None, 10, None, None) == 0
    assert lib.tgvkv_sizes(ok, None, 10, ctypes.byref(kept), None) == 0 and kept.value == 10
    with pytest.raises(bd.TgvkvError):
        bd.tgvkv_sizes(P(), None, -1)


def test_empty_batch_is_a_no_op(lib):
    z = ctypes.byref(P(batch=0))
    s = ctypes.c_void_p(0)
    assert lib.tgvkv_score(z, None, 7, None, ctypes.c_void_p(0x10000), None, None, None, None, None, None, None,
                           0, s) == 0
    assert lib.tgvkv_budget(z, None, None, 5, 0, None, ctypes.c_void_p(0x10000), ctypes.c_void_p(0x10000), None, s) == 0
    assert lib.tgvkv_select(z, None, None, None, None, None, None, s) == 0
    assert lib.tgvkv_compact(z, None, None, None, None, None, None, None, 5, 0, None, None, None, s) == 0
    assert lib.tgvkv_decode_attn(z, None, None, None, None, None, 2, 0, None, None, None, None, None, 0, None, s) == 0
    used = ctypes.c_void_p(0x10000)
    assert lib.tgvkv_page_table(z, None, None, 5, 2, 4, None, 0, None, 8, used, s) == 0
    assert lib.tgvkv_compact_paged(z, None, None, None, None, None, None, 5, None, 8, 4, None, None, 1, None, s) == 0
    assert lib.tgvkv_decode_attn_paged(z, None, None, None, 1, 4, None, 8, None, 2, None, None, None, None, None,
                                       None, 0, None, s) == 0


def test_binding_fails_loudly_without_library(tmp_path):
    with pytest.raises(RuntimeError):
        bd.load_library(str(tmp_path / "missing.so"))


@pytest.mark.skipif(_gpu(), reason="fake pointers are used only where no GPU exists")
def test_ceiling_validation_before_any_launch(lib):
    fake = ctypes.c_void_p(0x10000)
    odd = ctypes.c_void_p(0x10008)
    s = ctypes.c_void_p(0)
    assert lib.tgvkv_ceiling_read(None, 16, fake, s) == -1
    assert lib.tgvkv_ceiling_read(fake, 0, fake, s) == -1
    assert lib.tgvkv_ceiling_read(fake, 24, fake, s) == -1       # not a multiple of 16
    assert lib.tgvkv_ceiling_read(odd, 16, fake, s) == -1        # not 16-byte aligned
    assert lib.tgvkv_ceiling_read(fake, 16, None, s) == -1
    assert lib.tgvkv_ceiling_copy(fake, None, 16, s) == -1
    assert lib.tgvkv_ceiling_copy(fake, odd, 16, s) == -1
    assert lib.tgvkv_ceiling_copy(fake, fake, -16, s) == -1
    assert lib.tgvkv_ceiling_mfma(0, 10, fake, s) == -1
    assert lib.tgvkv_ceiling_mfma(4, 0, fake, s) == -1
    assert lib.tgvkv_ceiling_mfma(4, 10, None, s) == -1
    # 4 waves per workgroup, 8 MFMAs of 16 x 16 x 32 (2 flops each) per round
    assert lib.tgvkv_ceiling_mfma_flops(3, 5) == 3 * 4 * 5 * 8 * 2 * 16 * 16 * 32
    assert lib.tgvkv_ceiling_mfma_flops(0, 5) == 0
