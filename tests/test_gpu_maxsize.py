"""Parity at the largest sequence the library takes: N = 2^24 tokens, head_dim 128.

Two layers hold the same keys, values and decode inputs, so the second layer's key rows
start 2^31 elements into the key tensor.  The oracle checks layer 0 in full (every vision
score, the budgets, the retained set, the compacted rows, two decode steps over that set);
layer 1 must give layer 0's results bit for bit.  Keys are random bf16 bit patterns (both
signs, magnitudes in [1/8, 2)), which at this size are far cheaper to draw than normal
values; values are the keys with the sign flipped, so a K/V mix-up cannot pass.  The
selection runs its global-memory key path here (rows longer than its LDS key buffer).
"""

import numpy as np
import pytest

import oracle.tgvkv_oracle as O
from paper_2606_03075_amd import binding as bd
from tests.gpu_util import DECODE_ATOL, assert_close_rel, bf16_host_bits, dev_bf16, host, idx_allowed, log
from workloads import bf16_bits_to_f32, f32_to_bf16_bits
from workloads.configs import custom_config

pytestmark = pytest.mark.gpu


def _bf16_bits(rng, shape):
    u = rng.integers(0, 1 << 16, size=shape, dtype=np.uint16)
    exp = np.uint16(124) + ((u >> np.uint16(7)) & np.uint16(3))
    return (u & np.uint16(0x807F)) | (exp << np.uint16(7))


def test_max_sequence(lib):
    import torch
    ns, nq, N, D = 5, 11, 1 << 24, 128
    cfg = custom_config(name="maxn", batch=1, layers=2, heads_q=2, heads_kv=1, head_dim=D, n_sys=ns,
                        n_vis=N - ns - nq, n_qst=nq)
    nv, nt, L = cfg.n_vis, cfg.n_text, cfg.layers
    steps, total = 2, 40000
    rng = np.random.default_rng(2024)
    log(f"max sequence: N={N} D={D} layers={L} total={total}")
    q = f32_to_bf16_bits(rng.standard_normal((2, nt, D)).astype(np.float32))
    k = _bf16_bits(rng, (1, N, D))
    v = k ^ np.uint16(0x8000)
    dq = f32_to_bf16_bits(rng.standard_normal((steps, 2, D)).astype(np.float32))
    dk = f32_to_bf16_bits(rng.standard_normal((steps, 1, D)).astype(np.float32))
    dv = f32_to_bf16_bits(rng.standard_normal((steps, 1, D)).astype(np.float32))

    # device tensors [B=1][L=2][...], both layers the same
    def two_layers(bits):
        one = dev_bf16(bits)
        out = torch.empty((1, L) + tuple(one.shape), dtype=one.dtype, device="cuda")
        for l in range(L):
            out[0, l].copy_(one)
        del one
        return out

    q_d, k_d, v_d = two_layers(q), two_layers(k), two_layers(v)
    p = bd.problem_from(cfg)
    buf = bd.EvictionBuffers(p, None, total, steps)
    buf.evict(q_d, k_d, v_d)
    outs = []
    for st in range(steps):
        buf.decode(st, two_layers(dq[st]), two_layers(dk[st]), two_layers(dv[st]))
        outs.append(host(buf.out).copy())
    torch.cuda.synchronize()
    del k_d, v_d
    budgets, io, so = host(buf.budgets), host(buf.idx_offsets), host(buf.seg_offsets)
    idx = host(buf.idx)
    log("  GPU done; oracle on layer 0")

    # layer 1 repeats layer 0 bit for bit
    for name in ("lse", "s_txt", "w_txt", "s_vis", "tv_mass"):
        a = host(getattr(buf, name))
        assert np.array_equal(a[0, 0], a[0, 1]), name
    assert budgets[0, 0] == budgets[0, 1]
    b0 = int(budgets[0, 0])
    assert np.array_equal(idx[io[0]:io[0] + b0], idx[io[1]:io[1] + b0])
    kc, vc = bf16_host_bits(buf.kc), bf16_host_bits(buf.vc)
    seg = lambda a, l: a[so[l] * D:(so[l] + b0 + steps) * D]
    assert np.array_equal(seg(kc, 0), seg(kc, 1)) and np.array_equal(seg(vc, 0), seg(vc, 1))
    for st in range(steps):
        assert np.array_equal(outs[st][0, 0], outs[st][0, 1])

    # layer 0 against the oracle
    sc = O.score_slice(bf16_bits_to_f32(q), bf16_bits_to_f32(k), ns, nv, nq)
    sc.pop("P")
    assert_close_rel("lse", host(buf.lse[0, 0]), sc["lse"], atol=1e-4)
    assert_close_rel("s_txt", host(buf.s_txt[0, 0]), sc["s_txt"])
    assert_close_rel("w_txt", host(buf.w_txt[0, 0]), sc["w_txt"])
    assert_close_rel("tv_mass", host(buf.tv_mass[0, 0]), sc["tv_mass"])
    assert_close_rel("s_vis", host(buf.s_vis[0, 0]), sc["s_vis"])
    ob = O.layer_budgets([sc["tv_mass"]] * L, total, N)
    assert np.array_equal(budgets[0], ob), (budgets[0], ob)
    oidx = O.tpr_select(sc["s_vis"][0], sc["s_txt"][0], b0, ns, nv, nq)
    gidx = idx[io[0]:io[0] + b0]
    swaps = idx_allowed(gidx, oidx, sc["s_vis"][0], sc["s_txt"][0], b0, cfg)
    log(f"  budgets {budgets[0].tolist()}, boundary swaps {swaps}")
    assert np.array_equal(seg(kc, 0)[:b0 * D].reshape(b0, D), k[0][gidx])
    assert np.array_equal(seg(vc, 0)[:b0 * D].reshape(b0, D), v[0][gidx])
    # decode over the retained set just validated (boundary swaps included) and compacted bit for bit
    Kc, Vc = [bf16_bits_to_f32(k[0][gidx])], [bf16_bits_to_f32(v[0][gidx])]
    ref = O.decode_reference(bf16_bits_to_f32(dq), bf16_bits_to_f32(dk), bf16_bits_to_f32(dv), Kc, Vc,
                             1.0 / np.sqrt(D))
    for st in range(steps):
        err = np.abs(outs[st][0, 0] - ref[st]).max()
        assert err <= DECODE_ATOL, (st, err)


@pytest.mark.parametrize("shape", [
    # one query head, 16384 text rows (8000 system + 8384 question), 100 vision tokens
    dict(heads_q=1, heads_kv=1, head_dim=64, n_sys=8000, n_vis=100, n_qst=8384),
    # 16 query heads per KV head, 1024 text rows each
    dict(heads_q=16, heads_kv=1, head_dim=128, n_sys=24, n_vis=500, n_qst=1000),
])
def test_max_text_rows(lib, shape):
    """16384 text rows per KV head (query heads x text tokens), the library's limit: the
    row normalisers of a KV head's text rows fill the text pass's LDS buffer."""
    from tests.test_gpu_e2e import run_and_check
    cfg = custom_config(name="maxtext", batch=1, layers=2, **shape)
    assert cfg.heads_q // cfg.heads_kv * cfg.n_text == 16384
    # a budget inside the text (top text tokens), then one that reaches into the vision tokens
    for rho in (0.3, 0.998):
        run_and_check(cfg, rho, steps=2, seed=5)


def test_max_layers(lib):
    """512 layers (the library's limit) end to end: budgets shared over every layer, decode's
    longest-first dispatch over 1024 (sequence, layer) segments."""
    from tests.test_gpu_e2e import run_and_check
    cfg = custom_config(name="maxlayers", batch=2, layers=512, heads_q=2, heads_kv=1, head_dim=64, n_sys=3,
                        n_vis=30, n_qst=4)
    run_and_check(cfg, 0.2, steps=2, seed=9)
