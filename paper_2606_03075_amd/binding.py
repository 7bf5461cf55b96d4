"""Python binding of libtgvkv: the C ABI of include/tgvkv.h through ctypes.

Argument marshalling only.  Each function takes torch tensors that already live
in device memory, checks that they are contiguous, on the GPU and of the
expected element type, passes their addresses and torch's current HIP stream to
the C entry point of the same name, and raises TgvkvError on a negative status.
Every step of the computation runs in the library's HIP kernels; there is no
fallback path.
"""

from __future__ import annotations

import ctypes
import os
from typing import Optional

_HERE = os.path.dirname(os.path.abspath(__file__))
# TGVKV_LIBRARY names another build of the same ABI (e.g. the host-sanitized one of build.py)
LIB_PATH = os.environ.get("TGVKV_LIBRARY") or os.path.join(_HERE, "libtgvkv.so")

TGVKV_OK, TGVKV_E_INVAL, TGVKV_E_UNSUPPORTED, TGVKV_E_WORKSPACE, TGVKV_E_CAPACITY, TGVKV_E_HIP = 0, -1, -2, -3, -4, -5
SCORE_STATS, SCORE_TEXT, SCORE_VISION, SCORE_ALL = 1, 2, 4, 7
SCORE_LSE_IN = 16  # lse holds the text rows' normalisers from the caller's prefill: K is read once
CALL_SCORE, CALL_DECODE = 0, 1

ABI_VERSION = 8  # TGVKV_ABI_VERSION of the library this binding marshals for
EXPORTS = ("tgvkv_score", "tgvkv_budget", "tgvkv_select", "tgvkv_compact", "tgvkv_decode_attn",
           "tgvkv_decode_attn_noalloc",
           "tgvkv_page_plan", "tgvkv_page_table", "tgvkv_compact_paged", "tgvkv_decode_attn_paged",
           "tgvkv_sizes", "tgvkv_workspace_size", "tgvkv_status_string", "tgvkv_abi_version")
# measurement kernels (include/tgvkv_ceiling.h): the chip's achievable stream and matrix-core rates
CEILING_EXPORTS = ("tgvkv_ceiling_read", "tgvkv_ceiling_copy", "tgvkv_ceiling_mfma", "tgvkv_ceiling_mfma_flops")


class TgvkvProblem(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("layers", ctypes.c_int32), ("heads_q", ctypes.c_int32),
                ("heads_kv", ctypes.c_int32), ("head_dim", ctypes.c_int32), ("n_sys", ctypes.c_int32),
                ("n_vis", ctypes.c_int32), ("n_qst", ctypes.c_int32)]


class TgvkvOpts(ctypes.Structure):
    _fields_ = [("sm_scale", ctypes.c_float), ("head_mode", ctypes.c_int32), ("n_sink", ctypes.c_int32),
                ("n_recent", ctypes.c_int32), ("vision_only", ctypes.c_int32), ("budget_rule", ctypes.c_int32),
                ("vision_rank", ctypes.c_int32), ("joint_rank", ctypes.c_int32)]


class TgvkvError(RuntimeError):
    def __init__(self, fn: str, status: int, text: str):
        super().__init__(f"{fn} failed: status {status} ({text})")
        self.status = status


_lib: Optional[ctypes.CDLL] = None


def load_library(path: Optional[str] = None) -> ctypes.CDLL:
    """Load libtgvkv.so (built in-tree by __graft_entry__.build()); raises if it is missing."""
    global _lib
    if _lib is not None and path is None:
        return _lib
    p = path or LIB_PATH
    if not os.path.exists(p):
        raise RuntimeError(f"{p} is not built; run __graft_entry__.build() (hipcc for gfx950)")
    lib = ctypes.CDLL(p)
    P = ctypes.POINTER(TgvkvProblem)
    O = ctypes.POINTER(TgvkvOpts)
    vp, i32, i64, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
    lib.tgvkv_score.argtypes = [P, O, i32, vp, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]
    lib.tgvkv_budget.argtypes = [P, O, vp, i64, i32, vp, vp, vp, vp, vp]
    lib.tgvkv_select.argtypes = [P, O, vp, vp, vp, vp, vp, vp]
    lib.tgvkv_compact.argtypes = [P, O, vp, vp, vp, vp, vp, vp, i64, i32, vp, vp, vp, vp]
    lib.tgvkv_decode_attn.argtypes = [P, O, vp, vp, vp, vp, i32, i32, vp, vp, vp, vp, vp, sz, vp, vp]
    lib.tgvkv_decode_attn_noalloc.argtypes = [P, O, vp, vp, vp, vp, i32, i32, vp, vp, vp, vp, vp, vp]
    lib.tgvkv_page_plan.argtypes = [P, O, i64, i32, i32, vp, vp]
    lib.tgvkv_page_table.argtypes = [P, O, vp, i64, i32, i32, vp, i64, vp, i32, vp, vp]
    lib.tgvkv_compact_paged.argtypes = [P, O, vp, vp, vp, vp, vp, i64, vp, i32, i32, vp, vp, i64, vp, vp]
    lib.tgvkv_decode_attn_paged.argtypes = [P, O, vp, vp, i64, i32, vp, i32, vp, i32, vp, vp, vp, vp, vp, vp, sz,
                                            vp, vp]
    lib.tgvkv_sizes.argtypes = [P, O, i64, vp, vp]
    lib.tgvkv_workspace_size.argtypes = [P, O, i32]
    lib.tgvkv_workspace_size.restype = sz
    lib.tgvkv_status_string.argtypes = [ctypes.c_int]
    lib.tgvkv_status_string.restype = ctypes.c_char_p
    lib.tgvkv_abi_version.argtypes = []
    lib.tgvkv_ceiling_read.argtypes = [vp, i64, vp, vp]
    lib.tgvkv_ceiling_copy.argtypes = [vp, vp, i64, vp]
    lib.tgvkv_ceiling_mfma.argtypes = [i32, i32, vp, vp]
    lib.tgvkv_ceiling_mfma_flops.argtypes = [i32, i32]
    lib.tgvkv_ceiling_mfma_flops.restype = ctypes.c_longlong
    for name in ("tgvkv_score", "tgvkv_budget", "tgvkv_select", "tgvkv_compact", "tgvkv_decode_attn",
                 "tgvkv_decode_attn_noalloc", "tgvkv_page_plan", "tgvkv_page_table", "tgvkv_compact_paged", "tgvkv_decode_attn_paged",
                 "tgvkv_sizes", "tgvkv_abi_version", "tgvkv_ceiling_read", "tgvkv_ceiling_copy",
                 "tgvkv_ceiling_mfma"):
        getattr(lib, name).restype = ctypes.c_int32
    if lib.tgvkv_abi_version() != ABI_VERSION:
        raise RuntimeError(f"{p} has ABI {lib.tgvkv_abi_version()}, this binding needs {ABI_VERSION}; "
                           "rebuild it with __graft_entry__.build()")
    if path is None:
        _lib = lib
    return lib


def make_problem(batch, layers, heads_q, heads_kv, head_dim, n_sys, n_vis, n_qst) -> TgvkvProblem:
    return TgvkvProblem(batch, layers, heads_q, heads_kv, head_dim, n_sys, n_vis, n_qst)


def problem_from(cfg) -> TgvkvProblem:
    """Problem of a workload config (anything with the eight shape attributes)."""
    return make_problem(cfg.batch, cfg.layers, cfg.heads_q, cfg.heads_kv, cfg.head_dim, cfg.n_sys, cfg.n_vis,
                        cfg.n_qst)


BUDGET_TV, BUDGET_UNIFORM, BUDGET_TT = 0, 1, 2        # layer budgets by TV mass, equally, by TT mass
RANK_TWR, RANK_ATTENTION_SUM = 0, 1                     # vision importance


def make_opts(sm_scale: float = 0.0, head_mode: int = 0, n_sink: int = 0, n_recent: int = 0,
              vision_only: bool = False, budget_rule: int = BUDGET_TV, vision_rank: int = RANK_TWR,
              joint_rank: bool = False) -> TgvkvOpts:
    """Options; the defaults are the paper's TGV-KV (TVB, TWR, TPR over all tokens)."""
    return TgvkvOpts(sm_scale, head_mode, n_sink, n_recent, int(bool(vision_only)), int(budget_rule),
                     int(vision_rank), int(bool(joint_rank)))


def tgvkv_sizes(problem, opts, total_budget: int = 0):
    """(K, vision threshold) from tgvkv_sizes: the tokens one sequence keeps for a total_budget
    given to tgvkv_budget, and the budget a layer must exceed to need vision scores."""
    kept, thr = ctypes.c_int64(0), ctypes.c_int32(0)
    _check("tgvkv_sizes", load_library().tgvkv_sizes(ctypes.byref(problem), _opts_ref(opts), int(total_budget),
                                                     ctypes.byref(kept), ctypes.byref(thr)))
    return kept.value, thr.value


def kept_per_sequence(problem, opts, total_budget: int) -> int:
    """Tokens one sequence keeps for a total_budget given to tgvkv_budget (its idx / cache sizing)."""
    return tgvkv_sizes(problem, opts, total_budget)[0]


def status_string(status: int) -> str:
    return load_library().tgvkv_status_string(status).decode()


def _check(fn: str, status: int):
    if status != TGVKV_OK:
        raise TgvkvError(fn, status, status_string(status))


def _ptr(t, dtypes=None, name="tensor"):
    if t is None:
        return None
    import torch
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if not t.is_cuda:
        raise ValueError(f"{name} must be in GPU memory")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtypes is not None and t.dtype not in dtypes:
        raise TypeError(f"{name} has dtype {t.dtype}, expected one of {dtypes}")
    return ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    import torch
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def _bf16():
    import torch
    return (torch.bfloat16, torch.int16)


def _f32():
    import torch
    return (torch.float32,)


def workspace_size(problem: TgvkvProblem, opts: Optional[TgvkvOpts], which: int) -> int:
    return int(load_library().tgvkv_workspace_size(ctypes.byref(problem), _opts_ref(opts), which))


def _opts_ref(opts):
    return ctypes.byref(opts) if opts is not None else None


def tgvkv_score(problem, opts, phases, q_text, k, lse, s_txt, w_txt, tv_mass, s_vis, budgets=None,
                workspace=None, stream=None):
    import torch
    lib = load_library()
    ws_bytes = workspace.numel() * workspace.element_size() if workspace is not None else 0
    st = lib.tgvkv_score(ctypes.byref(problem), _opts_ref(opts), int(phases),
                         _ptr(q_text, _bf16(), "q_text"), _ptr(k, _bf16(), "k"), _ptr(lse, _f32(), "lse"),
                         _ptr(s_txt, _f32(), "s_txt"), _ptr(w_txt, _f32(), "w_txt"),
                         _ptr(tv_mass, _f32(), "tv_mass"), _ptr(s_vis, _f32(), "s_vis"),
                         _ptr(budgets, (torch.int32,), "budgets"), _ptr(workspace, None, "workspace"),
                         ws_bytes, _stream(stream))
    _check("tgvkv_score", st)


def tgvkv_budget(problem, opts, tv_mass, total_budget, decode_reserve, budgets, idx_offsets, seg_offsets,
                 stream=None, unit_order=None):
    import torch
    st = load_library().tgvkv_budget(ctypes.byref(problem), _opts_ref(opts), _ptr(tv_mass, _f32(), "tv_mass"),
                                     int(total_budget), int(decode_reserve),
                                     _ptr(budgets, (torch.int32,), "budgets"),
                                     _ptr(idx_offsets, (torch.int64,), "idx_offsets"),
                                     _ptr(seg_offsets, (torch.int64,), "seg_offsets"),
                                     _ptr(unit_order, (torch.int32,), "unit_order"), _stream(stream))
    _check("tgvkv_budget", st)


def tgvkv_select(problem, opts, s_vis, s_txt, budgets, idx_offsets, idx, stream=None):
    import torch
    st = load_library().tgvkv_select(ctypes.byref(problem), _opts_ref(opts), _ptr(s_vis, _f32(), "s_vis"),
                                     _ptr(s_txt, _f32(), "s_txt"), _ptr(budgets, (torch.int32,), "budgets"),
                                     _ptr(idx_offsets, (torch.int64,), "idx_offsets"),
                                     _ptr(idx, (torch.int32,), "idx"), _stream(stream))
    _check("tgvkv_select", st)


def tgvkv_compact(problem, opts, k, v, idx, budgets, idx_offsets, seg_offsets, total_budget, decode_reserve,
                  kc, vc, stream=None, unit_order=None):
    import torch
    st = load_library().tgvkv_compact(ctypes.byref(problem), _opts_ref(opts), _ptr(k, _bf16(), "k"),
                                      _ptr(v, _bf16(), "v"), _ptr(idx, (torch.int32,), "idx"),
                                      _ptr(budgets, (torch.int32,), "budgets"),
                                      _ptr(idx_offsets, (torch.int64,), "idx_offsets"),
                                      _ptr(seg_offsets, (torch.int64,), "seg_offsets"), int(total_budget),
                                      int(decode_reserve), _ptr(kc, _bf16(), "kc"), _ptr(vc, _bf16(), "vc"),
                                      _ptr(unit_order, (torch.int32,), "unit_order"), _stream(stream))
    _check("tgvkv_compact", st)


def tgvkv_decode_attn(problem, opts, kc, vc, budgets, seg_offsets, decode_reserve, step, q, k_new, v_new, out,
                      workspace=None, stream=None, unit_order=None):
    import torch
    ws_bytes = workspace.numel() * workspace.element_size() if workspace is not None else 0
    st = load_library().tgvkv_decode_attn(ctypes.byref(problem), _opts_ref(opts), _ptr(kc, _bf16(), "kc"),
                                          _ptr(vc, _bf16(), "vc"), _ptr(budgets, (torch.int32,), "budgets"),
                                          _ptr(seg_offsets, (torch.int64,), "seg_offsets"), int(decode_reserve),
                                          int(step), _ptr(q, _bf16(), "q"), _ptr(k_new, _bf16(), "k_new"),
                                          _ptr(v_new, _bf16(), "v_new"), _ptr(out, _f32(), "out"),
                                          _ptr(workspace, None, "workspace"), ws_bytes,
                                          _ptr(unit_order, (torch.int32,), "unit_order"), _stream(stream))
    _check("tgvkv_decode_attn", st)


def tgvkv_decode_attn_noalloc(problem, opts, kc, vc, budgets, seg_offsets, decode_reserve, step, q, k_new, v_new,
                              out, stream=None, unit_order=None):
    """tgvkv_decode_attn without a workspace: split partials in the library's per-GPU static buffer."""
    import torch
    st = load_library().tgvkv_decode_attn_noalloc(ctypes.byref(problem), _opts_ref(opts), _ptr(kc, _bf16(), "kc"),
                                                  _ptr(vc, _bf16(), "vc"), _ptr(budgets, (torch.int32,), "budgets"),
                                                  _ptr(seg_offsets, (torch.int64,), "seg_offsets"),
                                                  int(decode_reserve), int(step), _ptr(q, _bf16(), "q"),
                                                  _ptr(k_new, _bf16(), "k_new"), _ptr(v_new, _bf16(), "v_new"),
                                                  _ptr(out, _f32(), "out"),
                                                  _ptr(unit_order, (torch.int32,), "unit_order"), _stream(stream))
    _check("tgvkv_decode_attn_noalloc", st)


# --------------------------------------------------------------------------- measurement kernels
def _ceiling_check(fn: str, status: int):
    if status != 0:
        raise RuntimeError(f"{fn} failed: status {status}")


def tgvkv_ceiling_read(src, sink, stream=None):
    """One non-temporal 16-byte read stream over the bytes of src (a contiguous device tensor)."""
    import torch
    _ceiling_check("tgvkv_ceiling_read", load_library().tgvkv_ceiling_read(
        _ptr(src, None, "src"), src.numel() * src.element_size(), _ptr(sink, (torch.int32,), "sink"),
        _stream(stream)))


def tgvkv_ceiling_copy(src, dst, stream=None):
    """Copy src to dst (same byte size) with the read stream's loads and non-temporal stores."""
    nbytes = src.numel() * src.element_size()
    if dst.numel() * dst.element_size() != nbytes:
        raise ValueError("src and dst must have the same byte size")
    _ceiling_check("tgvkv_ceiling_copy", load_library().tgvkv_ceiling_copy(
        _ptr(src, None, "src"), _ptr(dst, None, "dst"), nbytes, _stream(stream)))


def tgvkv_ceiling_mfma(workgroups, iters, out, stream=None):
    """Back-to-back dense bf16 MFMAs; returns the launch's flops (out: float32 [workgroups * 256])."""
    if out.numel() < workgroups * 256:
        raise ValueError("out must hold workgroups * 256 floats")
    lib = load_library()
    _ceiling_check("tgvkv_ceiling_mfma", lib.tgvkv_ceiling_mfma(int(workgroups), int(iters),
                                                                _ptr(out, _f32(), "out"), _stream(stream)))
    return int(lib.tgvkv_ceiling_mfma_flops(int(workgroups), int(iters)))


# --------------------------------------------------------------------------- paged cache
def page_plan(problem, opts, total_budget, decode_reserve, page_size):
    """(max_pages, pool_pages): table width and pool-page bound of a batch (host only)."""
    mp, pool = ctypes.c_int32(0), ctypes.c_int64(0)
    st = load_library().tgvkv_page_plan(ctypes.byref(problem), _opts_ref(opts), int(total_budget),
                                        int(decode_reserve), int(page_size), ctypes.byref(mp), ctypes.byref(pool))
    _check("tgvkv_page_plan", st)
    return int(mp.value), int(pool.value)


def _table_width(block_table, problem) -> int:
    if block_table is None or block_table.dim() != 2 or block_table.shape[0] != problem.batch * problem.layers:
        raise ValueError("block_table must be a [batch * layers, max_pages] tensor")
    return int(block_table.shape[1])


def _pool_pages(k_pool, v_pool, problem, page_size) -> int:
    """n_pages of a pool, after checking both pools are [n_pages, heads_kv, page_size, head_dim]."""
    if k_pool is None or v_pool is None or k_pool.shape != v_pool.shape or k_pool.dim() != 4 or \
            tuple(k_pool.shape[1:]) != (problem.heads_kv, int(page_size), problem.head_dim):
        raise ValueError("k_pool and v_pool must both be [n_pages, heads_kv, page_size, head_dim]")
    return int(k_pool.shape[0])


def tgvkv_page_table(problem, opts, budgets, total_budget, decode_reserve, page_size, free_pages, block_table,
                     pages_used, stream=None):
    import torch
    st = load_library().tgvkv_page_table(ctypes.byref(problem), _opts_ref(opts),
                                         _ptr(budgets, (torch.int32,), "budgets"), int(total_budget),
                                         int(decode_reserve), int(page_size),
                                         _ptr(free_pages, (torch.int32,), "free_pages"), int(free_pages.numel()),
                                         _ptr(block_table, (torch.int32,), "block_table"),
                                         _table_width(block_table, problem),
                                         _ptr(pages_used, (torch.int64,), "pages_used"),
                                         _stream(stream))
    _check("tgvkv_page_table", st)


def tgvkv_compact_paged(problem, opts, k, v, idx, budgets, idx_offsets, total_budget, block_table, page_size,
                        k_pool, v_pool, stream=None, unit_order=None):
    import torch
    n_pages = _pool_pages(k_pool, v_pool, problem, page_size)
    st = load_library().tgvkv_compact_paged(ctypes.byref(problem), _opts_ref(opts), _ptr(k, _bf16(), "k"),
                                            _ptr(v, _bf16(), "v"), _ptr(idx, (torch.int32,), "idx"),
                                            _ptr(budgets, (torch.int32,), "budgets"),
                                            _ptr(idx_offsets, (torch.int64,), "idx_offsets"), int(total_budget),
                                            _ptr(block_table, (torch.int32,), "block_table"),
                                            _table_width(block_table, problem), int(page_size),
                                            _ptr(k_pool, _bf16(), "k_pool"), _ptr(v_pool, _bf16(), "v_pool"),
                                            n_pages, _ptr(unit_order, (torch.int32,), "unit_order"),
                                            _stream(stream))
    _check("tgvkv_compact_paged", st)


def tgvkv_decode_attn_paged(problem, opts, k_pool, v_pool, page_size, block_table, budgets, decode_reserve, steps,
                            q, k_new, v_new, out, workspace=None, stream=None, unit_order=None):
    import torch
    n_pages = _pool_pages(k_pool, v_pool, problem, page_size)
    ws_bytes = workspace.numel() * workspace.element_size() if workspace is not None else 0
    st = load_library().tgvkv_decode_attn_paged(ctypes.byref(problem), _opts_ref(opts),
                                                _ptr(k_pool, _bf16(), "k_pool"), _ptr(v_pool, _bf16(), "v_pool"),
                                                n_pages, int(page_size),
                                                _ptr(block_table, (torch.int32,), "block_table"),
                                                _table_width(block_table, problem),
                                                _ptr(budgets, (torch.int32,), "budgets"),
                                                int(decode_reserve), _ptr(steps, (torch.int32,), "steps"),
                                                _ptr(q, _bf16(), "q"), _ptr(k_new, _bf16(), "k_new"),
                                                _ptr(v_new, _bf16(), "v_new"), _ptr(out, _f32(), "out"),
                                                _ptr(workspace, None, "workspace"), ws_bytes,
                                                _ptr(unit_order, (torch.int32,), "unit_order"), _stream(stream))
    _check("tgvkv_decode_attn_paged", st)


# --------------------------------------------------------------------------- whole-pass helpers
class EvictionBuffers:
    """Device buffers of one eviction pass plus decode, allocated once for a problem.

    torch is used only to own device memory; every computation is a library call.
    """

    def __init__(self, problem: TgvkvProblem, opts: Optional[TgvkvOpts], total_budget: int,
                 decode_reserve: int, device="cuda"):
        import torch
        p = problem
        self.problem, self.opts = p, opts
        self.total_budget, self.decode_reserve = int(total_budget), int(decode_reserve)
        B, L, H, Hkv, D = p.batch, p.layers, p.heads_q, p.heads_kv, p.head_dim
        Nt, Nv = p.n_sys + p.n_qst, p.n_vis
        g = 1 if opts is None or opts.head_mode == 0 else Hkv
        f32 = dict(dtype=torch.float32, device=device)
        self.lse = torch.empty((B, L, H, Nt), **f32)
        self.s_txt = torch.empty((B, L, g, Nt), **f32)
        self.w_txt = torch.empty((B, L, g, Nt), **f32)
        self.tv_mass = torch.empty((B, L), **f32)
        self.s_vis = torch.zeros((B, L, g, Nv), **f32)
        self.budgets = torch.empty((B, L), dtype=torch.int32, device=device)
        self.unit_order = torch.empty((max(1, B * L),), dtype=torch.int32, device=device)  # decode dispatch
        self.idx_offsets = torch.empty((B * L + 1,), dtype=torch.int64, device=device)
        self.seg_offsets = torch.empty((B * L + 1,), dtype=torch.int64, device=device)
        self.kept = kept_per_sequence(p, opts, self.total_budget)
        self.idx = torch.empty((max(1, B * self.kept * g),), dtype=torch.int32, device=device)
        slots = B * (self.kept + L * self.decode_reserve)
        self.kc = torch.empty((max(1, slots * Hkv * D),), dtype=torch.bfloat16, device=device)
        self.vc = torch.empty_like(self.kc)
        self.out = torch.empty((B, L, H, D), **f32)
        self.ws_score = torch.empty((max(1, workspace_size(p, opts, CALL_SCORE)),), dtype=torch.uint8,
                                    device=device)
        self.ws_decode = torch.empty((max(1, workspace_size(p, opts, CALL_DECODE)),), dtype=torch.uint8,
                                     device=device)

    def score(self, q_text, k, phases=SCORE_ALL, budgets=None, stream=None):
        tgvkv_score(self.problem, self.opts, phases, q_text, k, self.lse, self.s_txt, self.w_txt, self.tv_mass,
                    self.s_vis, budgets, self.ws_score, stream)

    def budget(self, stream=None):
        tgvkv_budget(self.problem, self.opts, self.tv_mass, self.total_budget, self.decode_reserve, self.budgets,
                     self.idx_offsets, self.seg_offsets, stream, self.unit_order)

    def select(self, stream=None):
        tgvkv_select(self.problem, self.opts, self.s_vis, self.s_txt, self.budgets, self.idx_offsets, self.idx,
                     stream)

    def compact(self, k, v, stream=None):
        tgvkv_compact(self.problem, self.opts, k, v, self.idx, self.budgets, self.idx_offsets, self.seg_offsets,
                      self.total_budget, self.decode_reserve, self.kc, self.vc, stream, self.unit_order)

    def forced_or_text(self) -> int:
        """A layer needs vision scores only when its budget exceeds this: |forced U T| with TPR,
        |forced| when text and vision are ranked jointly."""
        return tgvkv_sizes(self.problem, self.opts, self.total_budget)[1]

    def schedule(self) -> str:
        """'two_step': text statistics and text scores, budgets, then vision scores only for the
        layers whose budget reaches past the text (never more work than scoring every layer)."""
        return "two_step"

    def evict(self, q_text, k, v, schedule="auto", stream=None, marks=None, compact=True):
        """Score, budget, select and (unless compact=False, e.g. for a paged cache) compact.

        schedule: 'auto' (= 'two_step'), 'two_step', 'phases' (every scoring phase as its own
        launch, vision scores for every layer) or 'lse_in' (self.lse
        already holds every text row's normaliser from the caller's prefill: text and vision
        scores and the TV mass in one K pass, then the budgets).  marks(name) is called after
        each stage (for event timing).
        """
        mark = marks if marks is not None else (lambda name: None)
        sched = self.schedule() if schedule == "auto" else schedule
        if sched == "two_step":
            self.score(q_text, k, SCORE_STATS | SCORE_TEXT, stream=stream)
            mark("score_text")
            self.budget(stream)
            mark("budget")
            self.score(q_text, k, SCORE_VISION, budgets=self.budgets, stream=stream)
            mark("score_vision")
        elif sched == "lse_in":
            self.score(q_text, k, SCORE_TEXT | SCORE_VISION | SCORE_LSE_IN, stream=stream)
            mark("score")
            self.budget(stream)
            mark("budget")
        elif sched == "phases":
            self.score(q_text, k, SCORE_STATS, stream=stream)
            mark("score_stats")
            self.score(q_text, k, SCORE_TEXT, stream=stream)
            mark("score_text")
            self.budget(stream)
            mark("budget")
            self.score(q_text, k, SCORE_VISION, stream=stream)
            mark("score_vision")
        else:
            raise ValueError(f"unknown schedule {schedule!r}")
        self.select(stream)
        mark("select")
        if compact:
            self.compact(k, v, stream)
            mark("compact")
        return sched

    def decode(self, step, q, k_new, v_new, stream=None):
        tgvkv_decode_attn(self.problem, self.opts, self.kc, self.vc, self.budgets, self.seg_offsets,
                          self.decode_reserve, step, q, k_new, v_new, self.out, self.ws_decode, stream,
                          self.unit_order)
        return self.out


class PagedPool:
    """A pool of cache pages shared by the sequences in service (continuous batching).

    Owns k_pool / v_pool [n_pages][heads_kv][page_size][head_dim] and the list of free
    page ids.  admit() places a batch evicted into EvictionBuffers in the pool (page
    table, then paged compaction); release() returns a finished sequence's pages.
    Page assignment and every copy run in the library; this class only keeps the
    free list, which needs the number of pages a batch took (one device read).
    """

    def __init__(self, heads_kv: int, head_dim: int, page_size: int, n_pages: int, device="cuda"):
        import torch
        self.page_size, self.n_pages = int(page_size), int(n_pages)
        self.k_pool = torch.empty((n_pages, heads_kv, page_size, head_dim), dtype=torch.bfloat16, device=device)
        self.v_pool = torch.empty_like(self.k_pool)
        self.free = list(range(n_pages))
        self.device = device

    def admit(self, buf: "EvictionBuffers", k, v, stream=None):
        """Page table [B*L, max_pages] of an evicted batch, with its rows compacted into the pool."""
        import torch
        p, o = buf.problem, buf.opts
        width, pool = page_plan(p, o, buf.total_budget, buf.decode_reserve, self.page_size)
        if pool > len(self.free):
            raise MemoryError(f"pool has {len(self.free)} free pages, the batch may need {pool}")
        ids = torch.tensor(self.free[:pool], dtype=torch.int32, device=self.device)
        table = torch.empty((p.batch * p.layers, width), dtype=torch.int32, device=self.device)
        used = torch.zeros((1,), dtype=torch.int64, device=self.device)
        tgvkv_page_table(p, o, buf.budgets, buf.total_budget, buf.decode_reserve, self.page_size, ids, table, used,
                         stream)
        tgvkv_compact_paged(p, o, k, v, buf.idx, buf.budgets, buf.idx_offsets, buf.total_budget, table,
                            self.page_size, self.k_pool, self.v_pool, stream, buf.unit_order)
        n = int(used.item()) if p.batch > 0 else 0
        del self.free[:n]
        return table

    def release(self, table_rows):
        """Return the pages of finished sequences' table rows to the free list."""
        ids = table_rows.reshape(-1).cpu().tolist()
        self.free.extend(int(i) for i in ids if i >= 0)

    def decode(self, problem, opts, table, budgets, decode_reserve, steps, q, k_new, v_new, out, workspace,
               stream=None, unit_order=None):
        """One decode step of a continuous batch whose sequence b is at step steps[b]."""
        tgvkv_decode_attn_paged(problem, opts, self.k_pool, self.v_pool, self.page_size, table, budgets,
                                decode_reserve, steps, q, k_new, v_new, out, workspace, stream, unit_order)
        return out
