"""Seeded, slice-addressable input generation.

Every tensor slice ``(name, b, l)`` has its own NumPy ``PCG64`` stream seeded by
``SeedSequence([seed, name_id, b, l])``, so any single slice can be regenerated
alone (the oracle checks sampled slices of the large workloads this way) and a
whole batch can be drawn in parallel threads.  Values are drawn in fp32 and
rounded once, round-to-nearest-even, to bf16; both the oracle and the GPU
library read exactly those bf16 values.

Recipes (per sequence b and layer l):

* text queries and text keys: i.i.d. N(0, 1);
* vision keys per KV head: a shared mean vector mu ~ N(0, I_d) plus
  ``sigma * N(0, 1)`` noise per token, which makes vision keys mutually similar
  and text keys diverse (the modality gap the paper describes in Sec. 1);
  with ``frames > 0`` each frame has its own mean, drawn as an AR(1) walk
  ``mu_f = sqrt(1 - a^2) mu_{f-1} + a eps_f`` whose marginals stay N(0, I);
* token 0's key is scaled by ``sink_scale`` (an attention sink);
* with ``tv_gap > 0``, the layers' text-to-vision attention differs by depth:
  each question-row query of layer l gets ``c * mu`` added (mu the mean vision
  key of its KV head, averaged over frames), with c chosen so that every vision
  logit of the row moves by ``s_l`` on average,
  ``s_l = -tv_gap * (1 - 0.85 exp(-x / 0.08) - 0.25 x) + 0.5 z``, x = l / (L - 1),
  z ~ N(0, 1) per (sequence, layer).  Shallow layers then put much of a
  question row's mass on the image and middle layers very little (the modality
  gap), so TVB's layer budgets spread out as the paper describes;
* values, decode queries and decode keys/values: i.i.d. N(0, 1).
"""

from __future__ import annotations

import concurrent.futures as _fut
import os
from typing import Dict, Optional, Sequence

import numpy as np

from .configs import WorkloadConfig, frame_size

_NAME_ID = {"k": 1, "v": 2, "q_text": 3, "vis_mean": 4, "dec_q": 5, "dec_k": 6, "dec_v": 7, "tv_shift": 8}


def _rng(seed: int, name: str, *idx: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, _NAME_ID[name], *idx])))


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round fp32 to bf16 (round to nearest, ties to even); returns the uint16 bit patterns."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    r = (u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)
    return r.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bit patterns to fp32."""
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def total_budget(rho: float, n_tokens: int, layers: int) -> int:
    """Global per-sequence KV budget: rho of all L*N cached tokens, rounded half away from zero."""
    x = float(rho) * float(n_tokens * layers)
    return int(np.floor(x + 0.5)) if x >= 0 else -int(np.floor(-x + 0.5))


def _vision_means(cfg: WorkloadConfig, seed: int, b: int, l: int) -> np.ndarray:
    """Vision key means, [H_kv][n_frames][d] (one frame unless the config has frames)."""
    rng = _rng(seed, "vis_mean", b, l)
    nf = max(cfg.frames, 1)
    eps = rng.standard_normal((cfg.heads_kv, nf, cfg.head_dim), dtype=np.float32)
    if nf == 1:
        return eps
    a = np.float32(cfg.frame_alpha)
    keep = np.float32(np.sqrt(np.float32(1.0) - a * a))
    mu = np.empty_like(eps)
    mu[:, 0] = eps[:, 0]
    for f in range(1, nf):
        mu[:, f] = keep * mu[:, f - 1] + a * eps[:, f]
    return mu


def gen_k_slice(cfg: WorkloadConfig, seed: int, b: int, l: int) -> np.ndarray:
    """Keys of one (sequence, layer): fp32 [H_kv][N][d], before bf16 rounding."""
    rng = _rng(seed, "k", b, l)
    k = rng.standard_normal((cfg.heads_kv, cfg.n_tokens, cfg.head_dim), dtype=np.float32)
    if cfg.n_vis > 0:
        mu = _vision_means(cfg, seed, b, l)
        v0, v1 = cfg.n_sys, cfg.n_sys + cfg.n_vis
        sigma = np.float32(cfg.vis_sigma)
        fs = frame_size(cfg)
        if fs is None:
            k[:, v0:v1] = mu[:, 0:1, :] + sigma * k[:, v0:v1]
        else:
            for f in range(cfg.frames):
                a0, a1 = v0 + f * fs, v0 + (f + 1) * fs
                k[:, a0:a1] = mu[:, f:f + 1, :] + sigma * k[:, a0:a1]
    if cfg.sink and cfg.n_tokens > 0:
        k[:, 0] *= np.float32(cfg.sink_scale)
    return k


def gen_v_slice(cfg: WorkloadConfig, seed: int, b: int, l: int) -> np.ndarray:
    rng = _rng(seed, "v", b, l)
    return rng.standard_normal((cfg.heads_kv, cfg.n_tokens, cfg.head_dim), dtype=np.float32)


def vision_logit_shift(cfg: WorkloadConfig, seed: int, b: int, l: int) -> float:
    """Mean shift s_l of the question rows' vision logits in layer l (0 unless tv_gap > 0)."""
    if cfg.tv_gap <= 0 or cfg.n_vis == 0:
        return 0.0
    x = l / max(cfg.layers - 1, 1)
    z = float(_rng(seed, "tv_shift", b, l).standard_normal())
    return -cfg.tv_gap * (1.0 - 0.85 * np.exp(-x / 0.08) - 0.25 * x) + 0.5 * z


def gen_qtext_slice(cfg: WorkloadConfig, seed: int, b: int, l: int) -> np.ndarray:
    """Text-row queries of one (sequence, layer): fp32 [H][N_t][d] in text order (system, then question)."""
    rng = _rng(seed, "q_text", b, l)
    q = rng.standard_normal((cfg.heads_q, cfg.n_text, cfg.head_dim), dtype=np.float32)
    shift = vision_logit_shift(cfg, seed, b, l)
    if shift != 0.0 and cfg.n_qst > 0:
        mu = _vision_means(cfg, seed, b, l).mean(axis=1)  # [H_kv][d]
        c = shift * np.sqrt(cfg.head_dim) / np.sum(mu * mu, axis=-1)  # q.mu / sqrt(d) moves by shift
        add = np.repeat((c[:, None] * mu).astype(np.float32), cfg.group, axis=0)  # query head h -> KV head h / G
        q[:, cfg.n_sys:] += add[:, None, :]
    return q


def gen_decode_slice(cfg: WorkloadConfig, seed: int, b: int, l: int, steps: int):
    """Decode inputs of one (sequence, layer) for ``steps`` steps: q [T][H][d], k_new/v_new [T][H_kv][d]."""
    q = _rng(seed, "dec_q", b, l).standard_normal((steps, cfg.heads_q, cfg.head_dim), dtype=np.float32)
    kn = _rng(seed, "dec_k", b, l).standard_normal((steps, cfg.heads_kv, cfg.head_dim), dtype=np.float32)
    vn = _rng(seed, "dec_v", b, l).standard_normal((steps, cfg.heads_kv, cfg.head_dim), dtype=np.float32)
    return q, kn, vn


def _threads(threads: Optional[int]) -> int:
    if threads:
        return threads
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def make_prefill_tensors(cfg: WorkloadConfig, seed: int = 0, threads: Optional[int] = None,
                         names=("q_text", "k", "v"), seqs: Optional[Sequence[int]] = None) -> Dict[str, np.ndarray]:
    """Whole-batch prefill inputs as bf16 bit patterns (uint16), in the library's layouts.

    q_text [B][L][H][N_t][d], k and v [B][L][H_kv][N][d].  With seqs, only those
    sequences of the batch are generated (leading dimension len(seqs), in that
    order); each is identical to its slice of the whole batch.
    """
    L = cfg.layers
    bs = list(range(cfg.batch)) if seqs is None else [int(b) for b in seqs]
    B = len(bs)
    shapes = {
        "q_text": (B, L, cfg.heads_q, cfg.n_text, cfg.head_dim),
        "k": (B, L, cfg.heads_kv, cfg.n_tokens, cfg.head_dim),
        "v": (B, L, cfg.heads_kv, cfg.n_tokens, cfg.head_dim),
    }
    fns = {"q_text": gen_qtext_slice, "k": gen_k_slice, "v": gen_v_slice}
    out = {n: np.empty(shapes[n], dtype=np.uint16) for n in names}

    def work(item):
        n, i, l = item
        out[n][i, l] = f32_to_bf16_bits(fns[n](cfg, seed, bs[i], l))

    items = [(n, i, l) for n in names for i in range(B) for l in range(L)]
    with _fut.ThreadPoolExecutor(_threads(threads)) as ex:
        list(ex.map(work, items))
    return out


def make_decode_tensors(cfg: WorkloadConfig, seed: int = 0, steps: Optional[int] = None,
                        threads: Optional[int] = None, seqs: Optional[Sequence[int]] = None) -> Dict[str, np.ndarray]:
    """Decode inputs as bf16 bits: q [T][B][L][H][d], k_new and v_new [T][B][L][H_kv][d].

    With seqs, only those sequences (second dimension len(seqs), in that order).
    """
    T = cfg.decode_steps if steps is None else steps
    L = cfg.layers
    bs = list(range(cfg.batch)) if seqs is None else [int(b) for b in seqs]
    B = len(bs)
    q = np.empty((T, B, L, cfg.heads_q, cfg.head_dim), np.uint16)
    kn = np.empty((T, B, L, cfg.heads_kv, cfg.head_dim), np.uint16)
    vn = np.empty_like(kn)

    def work(item):
        i, l = item
        a, c, e = gen_decode_slice(cfg, seed, bs[i], l, T)
        q[:, i, l] = f32_to_bf16_bits(a)
        kn[:, i, l] = f32_to_bf16_bits(c)
        vn[:, i, l] = f32_to_bf16_bits(e)

    with _fut.ThreadPoolExecutor(_threads(threads)) as ex:
        list(ex.map(work, [(i, l) for i in range(B) for l in range(L)]))
    return {"q": q, "k_new": kn, "v_new": vn}
