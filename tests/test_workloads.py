"""The seeded input generator: bf16 rounding, slice addressability, recipes (CPU only)."""

import numpy as np
import torch

from workloads import (CONFIGS, bf16_bits_to_f32, f32_to_bf16_bits, gen_k_slice, gen_qtext_slice,
                       make_decode_tensors, make_prefill_tensors, total_budget)
from workloads.configs import custom_config, depth_profile


def test_bf16_rounding_matches_torch():
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.standard_normal(100000).astype(np.float32) * 10.0 ** rng.integers(-8, 8, 100000),
                        np.array([0.0, -0.0, 1.0, 1.00390625, 1.005859375, 65504.0, -3.0e38], np.float32)])
    # values exactly halfway between two bf16 numbers, to exercise ties-to-even
    halves = (np.arange(1, 2000, dtype=np.uint32) << np.uint32(16)) | np.uint32(0x8000)
    x = np.concatenate([x, halves.view(np.float32)]).astype(np.float32)
    ours = f32_to_bf16_bits(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(ours, ref)
    back = bf16_bits_to_f32(ours)
    assert np.array_equal(back, torch.from_numpy(x).to(torch.bfloat16).float().numpy())


def test_slices_regenerate_alone():
    cfg = custom_config(batch=2, layers=3, heads_q=4, heads_kv=2, head_dim=64, n_sys=3, n_vis=20, n_qst=5)
    full = make_prefill_tensors(cfg, seed=11, threads=4)
    for b in range(2):
        for l in range(3):
            assert np.array_equal(full["k"][b, l], f32_to_bf16_bits(gen_k_slice(cfg, 11, b, l)))
            assert np.array_equal(full["q_text"][b, l], f32_to_bf16_bits(gen_qtext_slice(cfg, 11, b, l)))
    again = make_prefill_tensors(cfg, seed=11, threads=1)
    for n in full:
        assert np.array_equal(full[n], again[n])
    other = make_prefill_tensors(cfg, seed=12, threads=2)
    assert not np.array_equal(full["k"], other["k"])
    dec = make_decode_tensors(cfg, seed=11, steps=3)
    assert dec["q"].shape == (3, 2, 3, 4, 64) and dec["k_new"].shape == (3, 2, 3, 2, 64)
    # the first steps do not depend on how many steps were drawn
    dec1 = make_decode_tensors(cfg, seed=11, steps=1)
    assert np.array_equal(dec1["q"][0], dec["q"][0])


def test_recipes():
    cfg = CONFIGS["tiny"]
    k = gen_k_slice(cfg, 0, 0, 0)
    assert k.shape == (4, 168, 64)
    vis = k[:, 8:152]
    # vision keys cluster around a shared mean: per-head spread ~ sigma, text keys ~ 1
    assert abs(vis.std(axis=1).mean() - 0.3) < 0.05
    assert abs(k[:, 152:].std() - 1.0) < 0.15
    # token 0 is an attention sink (x4)
    assert np.abs(k[:, 0]).mean() > 2.5
    # video frames have their own means
    vid = custom_config(n_sys=2, n_vis=64, n_qst=3, frames=4, heads_kv=1, heads_q=1)
    kv = gen_k_slice(vid, 0, 0, 0)[0, 2:66].reshape(4, 16, -1).mean(axis=1)
    assert np.abs(kv[0] - kv[3]).mean() > 0.05


def test_total_budget():
    assert total_budget(0.10, 168, 1) == 17
    assert total_budget(0.05, 2979, 32) == 4766
    assert total_budget(0.05, 8256, 28) == 11558
    assert total_budget(0.10, 8256, 28) == 23117
    assert total_budget(0.05, 3171, 40) == 6342
    assert total_budget(0.05, 651, 32) == 1042 and total_budget(0.2, 651, 32) == 4166
    assert total_budget(0.5, 3, 1) == 2   # halves round away from zero


def test_depth_profile_changes_only_question_queries():
    """The model shapes draw i.i.d. text queries; the depth profile shifts only the question rows."""
    for name in ("llava15", "llavanext", "qwen2vl_video", "stress13b"):
        assert CONFIGS[name].tv_gap == 0.0
    cfg = custom_config(batch=1, layers=4, heads_q=4, heads_kv=2, head_dim=64, n_sys=3, n_vis=40, n_qst=6)
    dp = depth_profile(cfg)
    for l in range(4):
        q0, q1 = gen_qtext_slice(cfg, 3, 0, l), gen_qtext_slice(dp, 3, 0, l)
        assert np.array_equal(q0[:, :3], q1[:, :3]) and not np.array_equal(q0[:, 3:], q1[:, 3:])
        assert np.array_equal(gen_k_slice(cfg, 3, 0, l), gen_k_slice(dp, 3, 0, l))
