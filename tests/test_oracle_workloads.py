"""The oracle on the tiny workload: the paper's invariants hold on the synthetic data (CPU only)."""

import numpy as np

import oracle.tgvkv_oracle as O
from workloads import CONFIGS, bf16_bits_to_f32, make_prefill_tensors, total_budget


def test_tiny_workload_end_to_end():
    cfg = CONFIGS["tiny"]
    t = make_prefill_tensors(cfg, seed=0)
    for fp32 in (True, False):
        if fp32:  # the tiny case is specified in fp32: use the unrounded draws
            from workloads.gen import gen_k_slice, gen_qtext_slice
            q = gen_qtext_slice(cfg, 0, 0, 0)[None]
            k = gen_k_slice(cfg, 0, 0, 0)[None]
        else:
            q = bf16_bits_to_f32(t["q_text"][0])
            k = bf16_bits_to_f32(t["k"][0])
        for rho in cfg.rhos:
            tot = total_budget(rho, cfg.n_tokens, cfg.layers)
            scores, budgets, idx = O.evict_sequence(q, k, cfg.n_sys, cfg.n_vis, cfg.n_qst, tot)
            sc = scores[0]
            assert abs(sc["s_txt"].sum() + sc["tv_mass"] - cfg.n_text) < 1e-10
            assert budgets.sum() == tot
            I = idx[0][0]
            assert len(I) == tot
            text = set(O.text_positions(cfg.n_sys, cfg.n_vis, cfg.n_qst).tolist())
            if tot > cfg.n_text:
                assert text <= set(I.tolist())
            else:
                assert set(I.tolist()) <= text
            if rho == 1.0:
                assert list(I) == list(range(cfg.n_tokens))
