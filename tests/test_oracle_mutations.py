"""Plant plausible mistakes in the oracle (on the CPU) and confirm that some pin fails.

Each mutant replaces one step of the oracle module for the duration of a test;
the pins are the same checks the real oracle passes.
"""

import math

import numpy as np
import pytest

import oracle.tgvkv_oracle as O
from tests import oracle_pins as pins

_orig = {name: getattr(O, name) for name in
         ("text_row_softmax", "text_scores", "text_weights", "vision_scores", "tv_mass",
          "head_average", "layer_budgets", "tpr_select", "decode_attention", "vision_only_budgets",
          "budget_masses", "score_slice", "joint_select", "forced_positions", "evict_sequence")}


def _softmax_mask_off_by_one(q_text, k, n_sys, n_vis, n_qst, sm_scale):
    # a row no longer sees its own key
    P, lse = _orig["text_row_softmax"](q_text, k, n_sys, n_vis, n_qst + 0, sm_scale)
    pi = O.text_positions(n_sys, n_vis, n_qst)
    P = P.copy()
    for i, p in enumerate(pi):
        if p > 0:
            P[:, i, p] = 0.0
            P[:, i] /= P[:, i].sum(axis=-1, keepdims=True)
    return P, lse


def _softmax_wrong_kv_head(q_text, k, n_sys, n_vis, n_qst, sm_scale):
    H = q_text.shape[0]
    H_kv = k.shape[0]
    k2 = np.stack([k[h % H_kv] for h in range(H)])         # h % H_kv instead of h // G
    P, lse = _orig["text_row_softmax"](q_text, k2, n_sys, n_vis, n_qst, sm_scale)
    return P, lse


def _softmax_no_scale(q_text, k, n_sys, n_vis, n_qst, sm_scale):
    return _orig["text_row_softmax"](q_text, k, n_sys, n_vis, n_qst, 1.0)


def _text_scores_wrong_triangle(Abar, n_sys, n_vis, n_qst):
    pi = O.text_positions(n_sys, n_vis, n_qst)
    return np.triu(Abar[:, :, pi]).sum(axis=1)


def _text_scores_rows_not_cols(Abar, n_sys, n_vis, n_qst):
    pi = O.text_positions(n_sys, n_vis, n_qst)
    return np.tril(Abar[:, :, pi]).sum(axis=2)


def _text_weights_off_by_one(s_txt):
    n = s_txt.shape[-1]
    w = s_txt / (n - np.arange(n) + 1.0)
    return w / w.sum(axis=-1, keepdims=True)


def _text_weights_unnormalised(s_txt):
    n = s_txt.shape[-1]
    return s_txt / (n - np.arange(n, dtype=float))


def _vision_scores_reversed_weights(Abar, w_tilde, n_sys, n_vis):
    return _orig["vision_scores"](Abar, w_tilde[:, ::-1].copy(), n_sys, n_vis)


def _vision_scores_unweighted(Abar, w_tilde, n_sys, n_vis):
    return _orig["vision_scores"](Abar, np.ones_like(w_tilde) / w_tilde.shape[1], n_sys, n_vis)


def _tv_mass_sum_not_mean(P, n_sys, n_vis):
    return _orig["tv_mass"](P, n_sys, n_vis) * P.shape[0]


def _head_average_wrong_grouping(P, heads_kv, head_mode):
    if head_mode == 0:
        return P.mean(axis=0)[None]
    H = P.shape[0]
    G = H // heads_kv
    return P.reshape(G, heads_kv, *P.shape[1:]).mean(axis=0)


def _budgets_ties_to_higher_layer(masses, total_budget, n_tokens, n_floor=0, return_detail=False):
    b, det = _orig["layer_budgets"](masses, total_budget, n_tokens, n_floor, return_detail=True)
    L = len(masses)
    order = sorted((l for l in range(L) if b[l] - (1 if l in det["order"][:det["r"]] else 0) < n_tokens),
                   key=lambda l: (-det["frac"][l], -l))
    base = b.copy()
    for l in det["order"][:det["r"]]:
        base[l] -= 1
    for l in order[:det["r"]]:
        base[l] += 1
    return (base, det) if return_detail else base


def _budgets_floor_rounding(masses, total_budget, n_tokens, n_floor=0, return_detail=False):
    # nearest-integer rounding without the largest-remainder correction
    L = len(masses)
    m = np.asarray(masses, float)
    x = total_budget * (m / m.sum() if m.sum() > 0 else np.full(L, 1.0 / L))
    b = np.minimum(np.floor(x + 0.5), n_tokens).astype(np.int64)
    return (b, {}) if return_detail else b


def _tpr_ties_to_higher_position(s_vis, s_txt, budget, n_sys, n_vis, n_qst, n_sink=0, n_recent=0):
    N = n_sys + n_vis + n_qst
    # reverse the positions, select, map back: ties now go to the higher original position
    rs_t = np.asarray(s_txt, float)
    rs_v = np.asarray(s_vis, float)
    I = _orig["tpr_select"](rs_v[::-1].copy(), rs_t[::-1].copy(), budget, n_qst, n_vis, n_sys,
                            n_recent, n_sink)
    return np.sort(N - 1 - I)


def _tpr_vision_first(s_vis, s_txt, budget, n_sys, n_vis, n_qst, n_sink=0, n_recent=0):
    if budget <= n_vis:
        vpos = O.vision_positions(n_sys, n_vis, n_qst)
        order = np.lexsort((vpos, -np.asarray(s_vis, float)))
        return np.sort(vpos[order[:budget]])
    return _orig["tpr_select"](s_vis, s_txt, budget, n_sys, n_vis, n_qst, n_sink, n_recent)


def _decode_no_scale(q, Kc, Vc, sm_scale):
    return _orig["decode_attention"](q, Kc, Vc, 1.0)


def _vision_only_cap_at_sequence_length(masses, vision_budget, n_text, n_vis, n_forced_vis=0):
    # caps a layer's vision share at N (text + vision) instead of n_vis
    return int(n_text) + int(n_forced_vis) + O.layer_budgets(masses, vision_budget, n_vis + n_text, 0)


def _vision_only_drops_text(masses, vision_budget, n_text, n_vis, n_forced_vis=0):
    # forgets that every layer also keeps its text tokens
    return _orig["vision_only_budgets"](masses, vision_budget, 0, n_vis, n_forced_vis)


def _vision_only_forced_inside_budget(masses, vision_budget, n_text, n_vis, n_forced_vis=0):
    # counts the forced vision tokens inside the vision budget (as a floor) instead of beside it
    return int(n_text) + O.layer_budgets(masses, vision_budget, n_vis, n_forced_vis)


def _tt_mass_not_flipped(tv_masses, rule, n_text):
    # uses the text->vision mass for the text->text rule
    return _orig["budget_masses"](tv_masses, 0 if rule == 2 else rule, n_text)


def _attention_sum_still_weighted(q_text, k, n_sys, n_vis, n_qst, sm_scale=None, head_mode=0, vision_rank=0):
    # ignores the plain-attention-sum switch
    return _orig["score_slice"](q_text, k, n_sys, n_vis, n_qst, sm_scale, head_mode, 0)


def _joint_ties_to_higher_position(s_vis, s_txt, budget, n_sys, n_vis, n_qst, n_sink=0, n_recent=0,
                                   vis_scale=1.0):
    N = n_sys + n_vis + n_qst
    I = _orig["joint_select"](np.asarray(s_vis, float)[::-1].copy(), np.asarray(s_txt, float)[::-1].copy(),
                              budget, n_qst, n_vis, n_sys, n_recent, n_sink, vis_scale)
    return np.sort(N - 1 - I)


def _joint_without_scale(s_vis, s_txt, budget, n_sys, n_vis, n_qst, n_sink=0, n_recent=0, vis_scale=1.0):
    # ranks the vision scores unscaled
    return _orig["joint_select"](s_vis, s_txt, budget, n_sys, n_vis, n_qst, n_sink, n_recent, 1.0)


def _forced_drops_recent(n_tokens, n_sink, n_recent):
    # forgets the last n_recent tokens of App. A.2
    return _orig["forced_positions"](n_tokens, n_sink, 0)


def _forced_one_recent_too_many(n_tokens, n_sink, n_recent):
    # keeps n_recent + 1 trailing tokens
    return _orig["forced_positions"](n_tokens, n_sink, n_recent + 1 if n_recent > 0 else 0)


def _evict_sequence_no_floor(*args, **kwargs):
    # hands TVB no per-layer floor for the forced tokens
    real = O.layer_budgets

    def no_floor(masses, total_budget, n_tokens, n_floor=0, return_detail=False):
        return real(masses, total_budget, n_tokens, 0, return_detail)

    O.layer_budgets = no_floor
    try:
        return _orig["evict_sequence"](*args, **kwargs)
    finally:
        O.layer_budgets = real


MUTANTS = {
    "softmax_mask_off_by_one": ("text_row_softmax", _softmax_mask_off_by_one),
    "softmax_wrong_kv_head": ("text_row_softmax", _softmax_wrong_kv_head),
    "softmax_no_scale": ("text_row_softmax", _softmax_no_scale),
    "text_scores_wrong_triangle": ("text_scores", _text_scores_wrong_triangle),
    "text_scores_rows_not_cols": ("text_scores", _text_scores_rows_not_cols),
    "text_weights_off_by_one": ("text_weights", _text_weights_off_by_one),
    "text_weights_unnormalised": ("text_weights", _text_weights_unnormalised),
    "vision_scores_reversed_weights": ("vision_scores", _vision_scores_reversed_weights),
    "vision_scores_unweighted": ("vision_scores", _vision_scores_unweighted),
    "tv_mass_sum_not_mean": ("tv_mass", _tv_mass_sum_not_mean),
    "head_average_wrong_grouping": ("head_average", _head_average_wrong_grouping),
    "budgets_ties_to_higher_layer": ("layer_budgets", _budgets_ties_to_higher_layer),
    "budgets_plain_rounding": ("layer_budgets", _budgets_floor_rounding),
    "tpr_ties_to_higher_position": ("tpr_select", _tpr_ties_to_higher_position),
    "tpr_vision_first": ("tpr_select", _tpr_vision_first),
    "decode_no_scale": ("decode_attention", _decode_no_scale),
    "vision_only_cap_at_sequence_length": ("vision_only_budgets", _vision_only_cap_at_sequence_length),
    "vision_only_drops_text": ("vision_only_budgets", _vision_only_drops_text),
    "vision_only_forced_inside_budget": ("vision_only_budgets", _vision_only_forced_inside_budget),
    "tt_mass_not_flipped": ("budget_masses", _tt_mass_not_flipped),
    "attention_sum_still_weighted": ("score_slice", _attention_sum_still_weighted),
    "joint_ties_to_higher_position": ("joint_select", _joint_ties_to_higher_position),
    "joint_without_scale": ("joint_select", _joint_without_scale),
    "forced_drops_recent": ("forced_positions", _forced_drops_recent),
    "forced_one_recent_too_many": ("forced_positions", _forced_one_recent_too_many),
    "evict_sequence_no_floor": ("evict_sequence", _evict_sequence_no_floor),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_mistake_is_caught(name, monkeypatch):
    attr, fn = MUTANTS[name]
    monkeypatch.setattr(O, attr, fn)
    failed = []
    for check in pins.ALL_CHECKS:
        try:
            check(O)
        except (AssertionError, ValueError, ArithmeticError, IndexError):
            failed.append(check.__name__)
    assert failed, f"mutant {name} passed every pin"
