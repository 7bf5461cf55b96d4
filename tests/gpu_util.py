"""Helpers of the GPU parity tests: device upload, oracle runs per slice, and the acceptance rules.

Acceptance (GPU vs fp64 oracle on the same bf16 inputs):
* scores (lse, s^T, w~, s^V, TV mass): |g - o| <= 2e-3 |o| + 1e-12 (lse: + 1e-4 absolute);
* budgets: exact for the same masses; end to end, a +-1 trade between two layers is
  accepted only if the oracle's fractional parts of both layers lie within the
  score tolerance of each other (the rounding cut);
* retained sets: exact, except swaps at the k-th boundary whose oracle scores lie
  within 2e-3 relative of the oracle's k-th score;
* compacted K/V: bit-exact where the retained sets agree;
* decode outputs: |g - o| <= 1e-2 absolute.
"""

from __future__ import annotations

import sys

import numpy as np

import oracle.tgvkv_oracle as O
from workloads import bf16_bits_to_f32

SCORE_RTOL = 2e-3
DECODE_ATOL = 1e-2


def log(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def dev_bf16(bits: np.ndarray):
    import torch
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).cuda()


def host(t):
    return t.detach().cpu().numpy()


def bf16_host_bits(t) -> np.ndarray:
    import torch
    return t.detach().view(torch.int16).cpu().numpy().view(np.uint16)


def assert_close_rel(name, g, o, rtol=SCORE_RTOL, atol=1e-12):
    g = np.asarray(g, np.float64)
    o = np.asarray(o, np.float64)
    assert g.shape == o.shape, (name, g.shape, o.shape)
    if g.size == 0:
        return 0.0
    assert np.all(np.isfinite(g)), f"{name}: non-finite GPU values"
    err = np.abs(g - o)
    bound = rtol * np.abs(o) + atol
    bad = err > bound
    rel = float(np.max(err / (np.abs(o) + 1e-30)))
    assert not bad.any(), (f"{name}: {int(bad.sum())} of {g.size} outside tolerance; "
                           f"worst g={g[bad][0]!r} o={o[bad][0]!r} max rel {rel:.3e}")
    return rel


def oracle_scores(q_bits, k_bits, cfg, head_mode=0, fp32_inputs=None):
    """Oracle scores of one slice from bf16 bits ([H][N_t][d], [H_kv][N][d])."""
    q = bf16_bits_to_f32(q_bits) if fp32_inputs is None else fp32_inputs[0]
    k = bf16_bits_to_f32(k_bits) if fp32_inputs is None else fp32_inputs[1]
    r = O.score_slice(q, k, cfg.n_sys, cfg.n_vis, cfg.n_qst, None, head_mode)
    r.pop("P")
    return r


def budget_allowed(gpu_b, orc_b, masses, total, N, n_floor, tol=SCORE_RTOL):
    """True if gpu budgets equal the oracle's, or differ only by +-1 trades at the rounding cut."""
    gpu_b = np.asarray(gpu_b, np.int64)
    orc_b = np.asarray(orc_b, np.int64)
    if np.array_equal(gpu_b, orc_b):
        return True
    if gpu_b.sum() != total or np.abs(gpu_b - orc_b).max() > 1:
        return False
    _, det = O.layer_budgets(masses, total, N, n_floor, return_detail=True)
    x = det["x"]
    frac = det["frac"]
    diff = np.nonzero(gpu_b != orc_b)[0]
    # all flipped layers must sit at the cut: their fractional parts within the
    # score tolerance (relative to the real-valued share) of one another
    span = frac[diff].max() - frac[diff].min()
    return bool(span <= 2 * tol * max(1.0, float(np.max(x[diff]))))


def candidate_scores(s_vis, s_txt, budget, cfg, n_sink=0, n_recent=0, vis_scale=None):
    """Oracle view of one selection row: per-position score of the competing candidates and the k-th score.

    vis_scale: None for TPR (text first); a factor for the joint ranking without TPR.
    """
    N = cfg.n_tokens
    forced = set(O.forced_positions(N, n_sink, n_recent).tolist())
    tpos = O.text_positions(cfg.n_sys, cfg.n_vis, cfg.n_qst)
    vpos = O.vision_positions(cfg.n_sys, cfg.n_vis, cfg.n_qst)
    n_tf = sum(1 for p in tpos if p not in forced)
    rest = budget - len(forced)
    sc = {}
    if rest <= 0:
        return sc, None
    if vis_scale is not None:
        for i, p in enumerate(tpos):
            if p not in forced:
                sc[int(p)] = float(s_txt[i])
        for j, p in enumerate(vpos):
            if p not in forced:
                sc[int(p)] = float(vis_scale * s_vis[j])
        k = rest
    elif rest <= n_tf:
        for i, p in enumerate(tpos):
            if p not in forced:
                sc[int(p)] = float(s_txt[i])
        k = rest
    else:
        for j, p in enumerate(vpos):
            if p not in forced:
                sc[int(p)] = float(s_vis[j])
        k = rest - n_tf
    if k <= 0 or k > len(sc):
        return sc, None
    kth = sorted(sc.values(), reverse=True)[k - 1]
    return sc, kth


def idx_allowed(gpu_idx, orc_idx, s_vis, s_txt, budget, cfg, n_sink=0, n_recent=0, tol=SCORE_RTOL,
                vis_scale=None):
    """Number of boundary swaps; raises AssertionError if a difference is not a boundary tie."""
    g = set(int(x) for x in gpu_idx)
    o = set(int(x) for x in orc_idx)
    assert len(gpu_idx) == len(orc_idx) == budget
    assert list(gpu_idx) == sorted(gpu_idx), "retained positions not ascending"
    if g == o:
        return 0
    sc, kth = candidate_scores(s_vis, s_txt, budget, cfg, n_sink, n_recent, vis_scale)
    assert kth is not None, "sets differ but no top-k boundary exists"
    for p in g ^ o:
        assert p in sc, f"position {p} differs but is not a top-k candidate"
        assert abs(sc[p] - kth) <= tol * abs(kth) + 1e-30, f"position {p} score {sc[p]} not at the k-th {kth}"
    return len(g ^ o) // 2
