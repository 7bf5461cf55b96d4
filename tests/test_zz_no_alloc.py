"""tgvkv_decode_attn_noalloc (split partials in the library's static per-GPU buffer) against
tgvkv_decode_attn (split partials in a caller workspace), through the C ABI.

Two calls in a row on the same GPU, the second with a smaller problem: the static
buffer then still holds the first call's partials, and every value the second call
reads must be its own.  Both entry points run the same kernels, so outputs and the
appended cache rows must be equal bit for bit; the outputs are also checked against
the fp64 oracle's decode over the oracle's retained rows (decode tolerance 1e-2).
"""

import numpy as np
import pytest

import oracle.tgvkv_oracle as O
from paper_2606_03075_amd import binding as bd
from tests.gpu_util import DECODE_ATOL, dev_bf16, host, log
from workloads import bf16_bits_to_f32, make_decode_tensors, make_prefill_tensors, total_budget
from workloads.configs import custom_config

pytestmark = pytest.mark.gpu

# (name, shape, rho): the first uses the matrix-core decode (7 query heads per KV head), the
# second, smaller one the vector decode; both small enough that every unit's tokens are split
CASES = [
    ("gqa7", dict(batch=2, layers=3, heads_q=28, heads_kv=4, head_dim=128, n_sys=9, n_vis=300, n_qst=20), 0.3),
    ("mha", dict(batch=1, layers=2, heads_q=2, heads_kv=2, head_dim=64, n_sys=4, n_vis=90, n_qst=7), 0.5),
]


def _run_case(name, shape, rho, steps=3, seed=4):
    import torch
    cfg = custom_config(name=name, **shape)
    p = bd.problem_from(cfg)
    B, L, Hkv, D = cfg.batch, cfg.layers, cfg.heads_kv, cfg.head_dim
    ws_bytes = bd.workspace_size(p, None, bd.CALL_DECODE)
    assert 0 < ws_bytes <= 16 << 20, ws_bytes  # the token ranges are split: the scratch buffer is used
    t = make_prefill_tensors(cfg, seed=seed)
    dec = make_decode_tensors(cfg, seed=seed, steps=steps)
    tot = total_budget(rho, cfg.n_tokens, L)
    buf = bd.EvictionBuffers(p, None, tot, steps)
    buf.evict(dev_bf16(t["q_text"]), dev_bf16(t["k"]), dev_bf16(t["v"]))
    kc2, vc2 = buf.kc.clone(), buf.vc.clone()
    out2 = torch.full_like(buf.out, float("nan"))
    outs = []
    for st in range(steps):
        q, kn, vn = dev_bf16(dec["q"][st]), dev_bf16(dec["k_new"][st]), dev_bf16(dec["v_new"][st])
        buf.decode(st, q, kn, vn)
        bd.tgvkv_decode_attn_noalloc(p, None, kc2, vc2, buf.budgets, buf.seg_offsets, steps, st, q, kn, vn, out2,
                                     unit_order=buf.unit_order)
        torch.cuda.synchronize()
        assert torch.equal(out2, buf.out), (name, st)
        outs.append(host(out2).copy())
    assert torch.equal(kc2.view(torch.int16), buf.kc.view(torch.int16))
    assert torch.equal(vc2.view(torch.int16), buf.vc.view(torch.int16))
    # the oracle's decode over the oracle's retained rows
    tau = 1.0 / np.sqrt(D)
    worst = 0.0
    for b in range(B):
        _, ob, oidx = O.evict_sequence(bf16_bits_to_f32(t["q_text"][b]), bf16_bits_to_f32(t["k"][b]), cfg.n_sys,
                                       cfg.n_vis, cfg.n_qst, tot)
        for l in range(L):
            sel = oidx[l][0]
            Kc = [bf16_bits_to_f32(t["k"][b, l, h][sel]) for h in range(Hkv)]
            Vc = [bf16_bits_to_f32(t["v"][b, l, h][sel]) for h in range(Hkv)]
            ref = O.decode_reference(bf16_bits_to_f32(dec["q"][:, b, l]), bf16_bits_to_f32(dec["k_new"][:, b, l]),
                                     bf16_bits_to_f32(dec["v_new"][:, b, l]), Kc, Vc, tau)
            for st in range(steps):
                err = float(np.abs(outs[st][b, l] - ref[st]).max())
                worst = max(worst, err)
                assert err <= DECODE_ATOL, (name, b, l, st, err)
    log(f"  {name}: {steps} steps equal to tgvkv_decode_attn bit for bit, oracle max err {worst:.2e}")


def test_noalloc_decode_matches_workspace_decode(lib):
    for name, shape, rho in CASES:  # the second call is the smaller problem
        log(f"noalloc decode {name} {shape} rho={rho}")
        _run_case(name, shape, rho)


def test_noalloc_validates_before_any_launch(lib):
    """Invalid calls return their status and launch nothing, as tgvkv_decode_attn's do."""
    import torch
    p = bd.make_problem(1, 1, 2, 2, 64, 2, 10, 2)
    z = torch.zeros(64, dtype=torch.bfloat16, device="cuda")
    i32 = torch.zeros(1, dtype=torch.int32, device="cuda")
    i64 = torch.zeros(2, dtype=torch.int64, device="cuda")
    out = torch.full((256,), 7.0, dtype=torch.float32, device="cuda")
    with pytest.raises(bd.TgvkvError) as exc:
        bd.tgvkv_decode_attn_noalloc(p, None, z, z, i32, i64, 2, 2, z, z, z, out)  # step outside the reserve
    assert exc.value.status == bd.TGVKV_E_CAPACITY
    with pytest.raises(bd.TgvkvError) as exc:
        bd.tgvkv_decode_attn_noalloc(bd.make_problem(1, 1, 3, 2, 64, 2, 10, 2), None, z, z, i32, i64, 2, 0, z, z, z,
                                     out)  # heads_q not a multiple of heads_kv
    assert exc.value.status == bd.TGVKV_E_INVAL
    torch.cuda.synchronize()
    assert torch.all(out == 7.0)
