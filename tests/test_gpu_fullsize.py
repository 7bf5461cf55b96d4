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
from workloads.configs import CONFIGS

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


def test_llavanext_full(lib):
    """batch 4 x 32 layers x 32 heads, 35 + 2880 + 64 tokens, 5 % retention, 128 decode steps."""
    cfg = CONFIGS["llavanext"]
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
