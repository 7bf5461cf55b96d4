"""Plain float64 CPU oracle for the TGV-KV eviction pass and pruned-cache decode.

TEST INFRASTRUCTURE ONLY.  Only the test suite, the package smoke check and the
benchmark's CPU-baseline leg may import or call this module.  The GPU library
never calls it and shares no code with it.

It restates, one (sequence, layer) slice at a time and in float64, what the
paper "TGV-KV: Text-Grounded KV Eviction for Vision-Language Models" defines:

* Sec. 3.1, Eq. (2): causal row softmax A = softmax(QK^T + M), restricted to the
  rows whose queries are text tokens (the only rows the method reads);
* Sec. 3.2, Eq. (5) and Sec. 3.3 "TVB", Eq. (6): per-layer budget share from the
  summed text->vision attention;
* Sec. 3.3 "TWR", Eq. (7)-(9): text weights, text-weighted vision scores and
  text scores;
* Sec. 3.3 "TPR", Eq. (10): text-first retention with top-k;
* Sec. 3.1, Eq. (3)-(4): decode appends one key/value per step and attends over
  the (pruned) cache.

Where the paper is silent the readings recorded in the design notes apply: a
1/sqrt(d) logit scale; heads averaged (one retained set per layer) or, as an
option, averaged per KV-head group; w normalised to sum 1; budgets as integer
shares of a global budget rho*N*L with a per-layer cap of N, largest-remainder
rounding and lower-layer tie-break; top-k ties broken toward the lower
position; retained positions emitted in ascending order.

Parity status: the numeric score values (lse, s^T, w~, s^V, TV mass) are pinned
only through invariants, closed forms and brute force -- the paper prints no
worked numeric example of any score.
"""

from __future__ import annotations

import math
from typing import Dict, List, Optional, Sequence

import numpy as np


# --------------------------------------------------------------------------- layout
def text_positions(n_sys: int, n_vis: int, n_qst: int) -> np.ndarray:
    """Positions pi(i) of the text tokens, in text order (system then question).

    The token layout is system text, then vision, then question text, so the
    text set T of Sec. 3.3 (Eq. (10)) is [0, n_sys) U [n_sys + n_vis, N).
    """
    return np.concatenate([np.arange(n_sys), n_sys + n_vis + np.arange(n_qst)]).astype(np.int64)


def vision_positions(n_sys: int, n_vis: int, n_qst: int) -> np.ndarray:
    """Positions of the vision tokens (the set V of Eq. (10))."""
    return (n_sys + np.arange(n_vis)).astype(np.int64)


def forced_positions(n_tokens: int, n_sink: int, n_recent: int) -> np.ndarray:
    """First n_sink and last n_recent positions, kept by every method (App. A.2)."""
    s = set(range(min(max(n_sink, 0), n_tokens)))
    s |= set(range(max(n_tokens - max(n_recent, 0), 0), n_tokens))
    return np.array(sorted(s), dtype=np.int64)


def default_scale(head_dim: int) -> float:
    return 1.0 / math.sqrt(head_dim)


# --------------------------------------------------------------------------- scores
def text_row_softmax(q_text: np.ndarray, k: np.ndarray, n_sys: int, n_vis: int, n_qst: int,
                     sm_scale: float):
    """Text-query rows of the causal attention of Sec. 3.1, Eq. (2).

    q_text [H][N_t][d] (text order), k [H_kv][N][d]; query head h reads KV head
    h // (H / H_kv).  Row i sees keys j <= pi(i) (the mask M is -inf strictly
    above the diagonal).  Returns P [H][N_t][N] (zero where masked) and the row
    log-sum-exp lse [H][N_t] of the scaled logits.
    """
    q_text = np.asarray(q_text, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    H, n_text, _ = q_text.shape
    H_kv, N, _ = k.shape
    G = H // H_kv
    pi = text_positions(n_sys, n_vis, n_qst)
    masked = np.arange(N)[None, :] > pi[:, None]          # [N_t][N]
    P = np.zeros((H, n_text, N))
    lse = np.zeros((H, n_text))
    for h in range(H):
        z = sm_scale * (q_text[h] @ k[h // G].T)
        z[masked] = -np.inf
        zmax = z.max(axis=1, keepdims=True) if n_text else np.zeros((0, 1))
        e = np.exp(z - zmax)
        e[masked] = 0.0
        s = e.sum(axis=1, keepdims=True)
        P[h] = e / s
        lse[h] = zmax[:, 0] + np.log(s[:, 0])
    return P, lse


def head_average(P: np.ndarray, heads_kv: int, head_mode: int) -> np.ndarray:
    """Attention averaged over heads, per selection group: [g][N_t][N].

    head_mode 0: one group, the mean over all query heads (the paper's maps are
    head averages, Fig. 2, and the retained set I_l is per layer, Eq. (10)).
    head_mode 1: one group per KV head, the mean over the query heads sharing it.
    """
    H = P.shape[0]
    if head_mode == 0:
        return P.mean(axis=0)[None]
    G = H // heads_kv
    return P.reshape(heads_kv, G, *P.shape[1:]).mean(axis=1)


def tv_mass(P: np.ndarray, n_sys: int, n_vis: int) -> float:
    """Sum of the text->vision slice of the head-averaged attention (Eq. (5) with Eq. (6))."""
    if P.shape[1] == 0 or n_vis == 0:
        return 0.0
    return float(P.mean(axis=0)[:, n_sys:n_sys + n_vis].sum())


def text_scores(Abar: np.ndarray, n_sys: int, n_vis: int, n_qst: int) -> np.ndarray:
    """Eq. (9): s^T_j = sum over text rows i >= j of A^TT_ij, per group: [g][N_t]."""
    pi = text_positions(n_sys, n_vis, n_qst)
    TT = Abar[:, :, pi]                       # rows i (text queries), columns j (text keys)
    return np.tril(TT).sum(axis=1)            # keep i >= j, sum over rows


def text_weights(s_txt: np.ndarray) -> np.ndarray:
    """Eq. (7) then normalisation: w_j = s^T_j / (number of text rows that see key j).

    With 0-based j that count is N_t - j (the paper's 1-based N_t - j + 1).
    The normalised weight w~ = w / sum(w) (sum 1 per group; all zero if sum(w) == 0).
    """
    n_text = s_txt.shape[-1]
    w = s_txt / (n_text - np.arange(n_text, dtype=np.float64))
    tot = w.sum(axis=-1, keepdims=True)
    return np.where(tot > 0, w / np.where(tot > 0, tot, 1.0), 0.0)


def vision_scores(Abar: np.ndarray, w_tilde: np.ndarray, n_sys: int, n_vis: int) -> np.ndarray:
    """Eq. (8): s^V_j = sum_i w~_i A^TV_ij, per group: [g][N_v]."""
    TV = Abar[:, :, n_sys:n_sys + n_vis]       # [g][N_t][N_v]
    return np.einsum("gi,gij->gj", w_tilde, TV)


def score_slice(q_text, k, n_sys, n_vis, n_qst, sm_scale=None, head_mode=0,
                vision_rank: int = 0) -> Dict[str, np.ndarray]:
    """All scores of one (sequence, layer): lse, s_txt, w_txt (= w~), tv_mass, s_vis.

    vision_rank 1 is the ablation's plain attention sum in place of TWR (Table 5):
    every text row weighs 1, so s^V_j = sum_i A^TV_ij, and w_txt is all ones.
    """
    H_kv, _, d = np.shape(k)
    if sm_scale is None:
        sm_scale = default_scale(d)
    P, lse = text_row_softmax(q_text, k, n_sys, n_vis, n_qst, sm_scale)
    Abar = head_average(P, H_kv, head_mode)
    s_txt = text_scores(Abar, n_sys, n_vis, n_qst)
    w_til = text_weights(s_txt) if vision_rank == 0 else np.ones_like(s_txt)
    s_vis = vision_scores(Abar, w_til, n_sys, n_vis)
    return {"lse": lse, "s_txt": s_txt, "w_txt": w_til, "tv_mass": tv_mass(P, n_sys, n_vis),
            "s_vis": s_vis, "P": P}


# --------------------------------------------------------------------------- budgets
def budget_masses(tv_masses: Sequence[float], rule: int, n_text: int) -> List[float]:
    """Per-layer masses that share out the budget (Table 1(a), Eq. (5) over other slices).

    rule 0: the text->vision mass (TVB); 1: uniform (every layer 1); 2: the
    text->text mass.  Every text row's probabilities over its visible keys sum
    to 1, and its visible keys are text and vision tokens, so the head-averaged
    text->text mass of a layer is N_t minus its text->vision mass.  Non-finite
    or negative masses count as 0 first (as in layer_budgets).
    """
    out = []
    for x in tv_masses:
        x = float(x)
        x = x if (math.isfinite(x) and x > 0.0) else 0.0
        if rule == 0:
            out.append(x)
        elif rule == 1:
            out.append(1.0)
        elif rule == 2:
            out.append(max(float(n_text) - x, 0.0))
        else:
            raise ValueError("unknown budget rule")
    return out


def layer_budgets(masses: Sequence[float], total_budget: int, n_tokens: int, n_floor: int = 0,
                  return_detail: bool = False):
    """Integer per-layer budgets of one sequence (TVB, Eq. (5)-(6)).

    Each layer's share of the global budget is its text->vision mass over the
    sum across layers.  The paper gives the share as a fraction; the counts used
    by Eq. (10) are obtained by
      1. an optional floor of n_floor tokens per layer, given first;
      2. water-filling the rest, R = B_tot - L*floor, in proportion to the
         shares, with each layer capped at N - floor (capped layers are fixed
         and the remainder is re-shared among the others; with zero total mass
         the shares are uniform);
      3. largest-remainder rounding: floors of the real shares, then +1 to the
         layers with the largest fractional parts, ties to the lower layer.
    All arithmetic is float64 in this exact order.  Returns int64 [L].
    """
    L = len(masses)
    if L == 0:
        return (np.zeros(0, np.int64), {}) if return_detail else np.zeros(0, np.int64)
    if total_budget < 0 or total_budget > L * n_tokens:
        raise ValueError("total budget outside [0, L*N]")
    m = []
    for x in masses:
        x = float(x)
        m.append(x if (math.isfinite(x) and x > 0.0) else 0.0)
    F = min(int(n_floor), total_budget // L, n_tokens)
    cap = n_tokens - F
    R = total_budget - L * F
    S = 0.0
    for x in m:
        S += x
    f = [x / S for x in m] if S > 0.0 else [1.0 / L] * L
    x = [0.0] * L
    active = [True] * L
    n_active = L
    remaining = float(R)
    while n_active > 0:
        Fa = 0.0
        for l in range(L):
            if active[l]:
                Fa += f[l]
        for l in range(L):
            if active[l]:
                x[l] = (remaining * f[l]) / Fa if Fa > 0.0 else remaining / n_active
        over = [l for l in range(L) if active[l] and x[l] > cap]
        if not over:
            break
        for l in over:
            x[l] = float(cap)
            active[l] = False
            remaining -= cap
            n_active -= 1
    base = [min(int(math.floor(v)), cap) for v in x]
    frac = [v - math.floor(v) for v in x]
    b = [F + base[l] for l in range(L)]
    r = total_budget - sum(b)
    if r < 0:
        raise ArithmeticError("largest-remainder deficit is negative")
    order = sorted((l for l in range(L) if b[l] < n_tokens), key=lambda l: (-frac[l], l))
    if r > len(order):
        raise ArithmeticError("not enough layers below the cap")
    for l in order[:r]:
        b[l] += 1
    out = np.array(b, dtype=np.int64)
    if return_detail:
        return out, {"x": np.array(x), "frac": np.array(frac), "floor": F, "cap": cap, "R": R,
                     "order": order, "r": r}
    return out


def forced_vision_count(n_sys: int, n_vis: int, n_qst: int, n_sink: int = 0, n_recent: int = 0) -> int:
    """Number of forced positions (first n_sink, last n_recent) that are vision tokens."""
    f = forced_positions(n_sys + n_vis + n_qst, n_sink, n_recent)
    return int(np.count_nonzero((f >= n_sys) & (f < n_sys + n_vis)))


def vision_only_budgets(masses: Sequence[float], vision_budget: int, n_text: int, n_vis: int,
                        n_forced_vis: int = 0) -> np.ndarray:
    """Per-layer kept-token counts of vision-only eviction (App. B.3).

    In this mode every layer keeps all of its N_t text tokens and the retention
    ratio counts vision tokens only.  Forced positions that are vision tokens
    (App. A.2) are kept like the text, so the per-sequence vision budget V_tot
    counts the other n_vis - n_forced_vis vision tokens.  It is shared out over the
    layers by TVB exactly as the full budget is in layer_budgets (Eq. (5)-(6)),
    with that count as the per-layer cap, and layer l keeps
    b_l = N_t + n_forced_vis + v_l tokens.  Retention then always falls in the
    first case of Eq. (10).  Returns int64 [L].
    """
    cap = n_vis - n_forced_vis
    if vision_budget < 0 or vision_budget > len(masses) * cap:
        raise ValueError("vision budget outside [0, L*(n_vis - forced vision)]")
    return int(n_text) + int(n_forced_vis) + layer_budgets(masses, vision_budget, cap, 0)


# --------------------------------------------------------------------------- retention
def tpr_select(s_vis: np.ndarray, s_txt: np.ndarray, budget: int, n_sys: int, n_vis: int,
               n_qst: int, n_sink: int = 0, n_recent: int = 0) -> np.ndarray:
    """Retained positions of one (sequence, layer, group), ascending (TPR, Eq. (10)).

    Forced tokens (first n_sink, last n_recent; App. A.2) come first.  Then, if
    the rest of the budget does not cover the remaining text, the top text
    tokens by s^T; otherwise all text and the top vision tokens by s^V.  With no
    forced tokens this is exactly Eq. (10): T U TopK(s^V, b - N_t) if b > N_t,
    else TopK(s^T, b).  Ties in TopK go to the lower position.
    """
    N = n_sys + n_vis + n_qst
    tpos = text_positions(n_sys, n_vis, n_qst)
    vpos = vision_positions(n_sys, n_vis, n_qst)
    forced = forced_positions(N, n_sink, n_recent)
    fset = set(forced.tolist())
    if budget < 0 or budget > N:
        raise ValueError("budget outside [0, N]")
    if budget <= len(forced):
        return forced[:budget].copy()
    rest = budget - len(forced)
    t_keep = np.array([p not in fset for p in tpos], dtype=bool)
    v_keep = np.array([p not in fset for p in vpos], dtype=bool)
    t_cand, t_sc = tpos[t_keep], np.asarray(s_txt, np.float64)[t_keep]
    v_cand, v_sc = vpos[v_keep], np.asarray(s_vis, np.float64)[v_keep]
    if rest <= len(t_cand):
        order = np.lexsort((t_cand, -t_sc))
        chosen = t_cand[order[:rest]]
    else:
        order = np.lexsort((v_cand, -v_sc))
        chosen = np.concatenate([t_cand, v_cand[order[:rest - len(t_cand)]]])
    return np.sort(np.concatenate([forced, chosen])).astype(np.int64)


def joint_select(s_vis: np.ndarray, s_txt: np.ndarray, budget: int, n_sys: int, n_vis: int,
                 n_qst: int, n_sink: int = 0, n_recent: int = 0, vis_scale: float = 1.0) -> np.ndarray:
    """Retention without TPR (the ablation's TPR-off rows, Table 5), ascending.

    Forced tokens first, as in tpr_select; then the top (budget - |forced|) of all
    other positions ranked together: text token j by s^T_j, vision token j by
    vis_scale * s^V_j.  Under TWR (weights summing to 1) vis_scale = N_t puts s^V
    on the column-sum scale of s^T; under the plain attention sum it is 1.
    Ties go to the lower position.
    """
    N = n_sys + n_vis + n_qst
    tpos = text_positions(n_sys, n_vis, n_qst)
    vpos = vision_positions(n_sys, n_vis, n_qst)
    forced = forced_positions(N, n_sink, n_recent)
    if budget < 0 or budget > N:
        raise ValueError("budget outside [0, N]")
    if budget <= len(forced):
        return forced[:budget].copy()
    fset = set(forced.tolist())
    pos = np.concatenate([tpos, vpos])
    sc = np.concatenate([np.asarray(s_txt, np.float64), vis_scale * np.asarray(s_vis, np.float64)])
    keep = np.array([p not in fset for p in pos], dtype=bool)
    pos, sc = pos[keep], sc[keep]
    order = np.lexsort((pos, -sc))
    chosen = pos[order[:budget - len(forced)]]
    return np.sort(np.concatenate([forced, chosen])).astype(np.int64)


# --------------------------------------------------------------------------- cache
def compact_slice(k: np.ndarray, v: np.ndarray, idx_groups: Sequence[np.ndarray], head_mode: int):
    """Gather the retained rows of every KV head: Kc[h] = K[h][I], Vc[h] = V[h][I].

    idx_groups holds one index array (head_mode 0) or one per KV head (head_mode 1).
    Returns lists of arrays [b_l][d] per KV head, in the dtype given.
    """
    H_kv = k.shape[0]
    sel = [idx_groups[0 if head_mode == 0 else h] for h in range(H_kv)]
    return [k[h][sel[h]] for h in range(H_kv)], [v[h][sel[h]] for h in range(H_kv)]


def decode_attention(q: np.ndarray, Kc: Sequence[np.ndarray], Vc: Sequence[np.ndarray],
                     sm_scale: float) -> np.ndarray:
    """Single-query softmax attention per head over a (pruned + appended) cache.

    q [H][d]; Kc/Vc per KV head [n][d] (already holding the appended token of
    this step, Eq. (3)-(4)).  Returns out [H][d] in float64.
    """
    q = np.asarray(q, np.float64)
    H, d = q.shape
    H_kv = len(Kc)
    G = H // H_kv
    out = np.zeros((H, d))
    for h in range(H):
        K = np.asarray(Kc[h // G], np.float64)
        V = np.asarray(Vc[h // G], np.float64)
        z = sm_scale * (K @ q[h])
        z = z - z.max()
        p = np.exp(z)
        p /= p.sum()
        out[h] = p @ V
    return out


# --------------------------------------------------------------------------- whole slices
def evict_sequence(q_text_seq, k_seq, n_sys, n_vis, n_qst, total_budget_per_seq, sm_scale=None,
                   head_mode=0, n_sink=0, n_recent=0, layers: Optional[Sequence[int]] = None,
                   keep_P: bool = False, vision_only: bool = False, budget_rule: int = 0,
                   vision_rank: int = 0, joint_rank: bool = False):
    """Score, budget and select every layer of one sequence.

    q_text_seq [L][H][N_t][d], k_seq [L][H_kv][N][d] (any float dtype; used in float64).
    total_budget_per_seq is B_tot, or the vision budget V_tot with vision_only
    (App. B.3; see vision_only_budgets).  budget_rule / vision_rank / joint_rank
    select the paper's variants (budget_masses, score_slice, joint_select); all
    0 / False is TGV-KV.  Returns per-layer score dicts, the budgets [L] (tokens
    kept per layer) and the retained positions per layer and group.
    """
    if vision_only and joint_rank:
        raise ValueError("vision-only eviction keeps all text: no joint ranking")
    L = len(k_seq)
    H_kv, N, d = np.shape(k_seq[0])
    scale = default_scale(d) if sm_scale is None else sm_scale
    scores = []
    for l in range(L):
        sc = score_slice(q_text_seq[l], k_seq[l], n_sys, n_vis, n_qst, scale, head_mode, vision_rank)
        if not keep_P:
            sc.pop("P")
        scores.append(sc)
    masses = budget_masses([s["tv_mass"] for s in scores], budget_rule, n_sys + n_qst)
    if vision_only:
        nfv = forced_vision_count(n_sys, n_vis, n_qst, n_sink, n_recent)
        budgets = vision_only_budgets(masses, total_budget_per_seq, n_sys + n_qst, n_vis, nfv)
    else:
        nf = len(forced_positions(N, n_sink, n_recent))
        budgets = layer_budgets(masses, total_budget_per_seq, N, nf)
    idx = []
    for l in range(L):
        g = scores[l]["s_vis"].shape[0]
        if joint_rank:
            vis_scale = float(n_sys + n_qst) if vision_rank == 0 else 1.0
            idx.append([joint_select(scores[l]["s_vis"][gi], scores[l]["s_txt"][gi], int(budgets[l]),
                                     n_sys, n_vis, n_qst, n_sink, n_recent, vis_scale) for gi in range(g)])
        else:
            idx.append([tpr_select(scores[l]["s_vis"][gi], scores[l]["s_txt"][gi], int(budgets[l]),
                                   n_sys, n_vis, n_qst, n_sink, n_recent) for gi in range(g)])
    return scores, budgets, idx


def flat_offsets(counts: Sequence[int]) -> np.ndarray:
    """Exclusive prefix sum with a final total: [c0, c1, ...] -> [0, c0, c0+c1, ...]."""
    out = np.zeros(len(counts) + 1, dtype=np.int64)
    out[1:] = np.cumsum(np.asarray(counts, dtype=np.int64))
    return out


def decode_reference(q_steps, kn_steps, vn_steps, Kc: List[np.ndarray], Vc: List[np.ndarray],
                     sm_scale: float):
    """Run decode steps t = 0..T-1 for one (sequence, layer): append, then attend.

    q_steps [T][H][d], kn_steps/vn_steps [T][H_kv][d].  Returns outputs [T][H][d].
    """
    Kc = [np.asarray(x, np.float64) for x in Kc]
    Vc = [np.asarray(x, np.float64) for x in Vc]
    outs = []
    for t in range(len(q_steps)):
        Kc = [np.concatenate([Kc[h], np.asarray(kn_steps[t][h], np.float64)[None]]) for h in range(len(Kc))]
        Vc = [np.concatenate([Vc[h], np.asarray(vn_steps[t][h], np.float64)[None]]) for h in range(len(Vc))]
        outs.append(decode_attention(q_steps[t], Kc, Vc, sm_scale))
    return np.stack(outs) if outs else np.zeros((0,) + np.shape(q_steps)[1:])
