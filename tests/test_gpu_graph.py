"""The decode loop captured in a HIP graph (through torch.cuda.CUDAGraph) replays bit for bit.

Every library call is kernel launches on the caller's stream (no allocation, memset, copy or
synchronisation inside), so a serving loop can capture its decode steps once and replay them.
The graph here holds T decode steps, each followed by a copy of its output made by an
elementwise kernel.  It is replayed several times with eager library work and device
synchronisation between the replays, and every replay must equal the eager decode.
"""

import numpy as np
import pytest

from paper_2606_03075_amd import binding as bd
from tests.gpu_util import dev_bf16, log
from workloads import make_decode_tensors, make_prefill_tensors, total_budget
from workloads.configs import custom_config

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("heads_q,heads_kv", [(4, 4), (14, 2)])
def test_decode_graph_replays(lib, heads_q, heads_kv):
    import torch
    cfg = custom_config(name="graph", batch=2, layers=3, heads_q=heads_q, heads_kv=heads_kv, head_dim=128,
                        n_sys=6, n_vis=300, n_qst=21)
    T = 5
    log(f"graph decode H={heads_q} Hkv={heads_kv} T={T}")
    t = make_prefill_tensors(cfg, seed=4)
    dec = make_decode_tensors(cfg, seed=4, steps=T)
    q, k, v = (dev_bf16(t[n]) for n in ("q_text", "k", "v"))
    dq, dk, dv = ([dev_bf16(dec[n][s]) for s in range(T)] for n in ("q", "k_new", "v_new"))
    buf = bd.EvictionBuffers(bd.problem_from(cfg), None, total_budget(0.2, cfg.n_tokens, cfg.layers), T)
    buf.evict(q, k, v)

    eager = []
    for s in range(T):
        buf.decode(s, dq[s], dk[s], dv[s])
        eager.append(buf.out.clone())
    torch.cuda.synchronize()

    saved = [torch.empty_like(buf.out) for _ in range(T)]
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):  # warm the copy kernel outside the capture
        torch.add(buf.out, 0.0, out=saved[0])
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        for s in range(T):
            buf.decode(s, dq[s], dk[s], dv[s])
            torch.add(buf.out, 0.0, out=saved[s])
    torch.cuda.synchronize()

    for rep in range(3):
        for x in saved:
            x.fill_(float("nan"))
        buf.decode(0, dq[0], dk[0], dv[0])  # eager work between replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for s in range(T):
            assert torch.equal(saved[s], eager[s]), f"replay {rep}, step {s}"
    # the cache after the replays still gives the eager results
    buf.decode(T - 1, dq[T - 1], dk[T - 1], dv[T - 1])
    torch.cuda.synchronize()
    assert torch.equal(buf.out, eager[T - 1])


@pytest.mark.parametrize("schedule", ["two_step", "phases"])
def test_eviction_graph_replays(lib, schedule):
    """The whole eviction pass (scores, budgets, vision scores where needed, selection,
    compaction) captured once and replayed: every output equals the eager pass bit for bit."""
    import torch
    cfg = custom_config(name="graphev", batch=2, layers=4, heads_q=8, heads_kv=2, head_dim=128, n_sys=6,
                        n_vis=300, n_qst=21)
    log(f"graph eviction {schedule}")
    t = make_prefill_tensors(cfg, seed=8)
    q, k, v = (dev_bf16(t[n]) for n in ("q_text", "k", "v"))
    buf = bd.EvictionBuffers(bd.problem_from(cfg), None, total_budget(0.1, cfg.n_tokens, cfg.layers), 2)
    names = ("lse", "s_txt", "w_txt", "tv_mass", "s_vis", "budgets", "idx_offsets", "seg_offsets", "unit_order",
             "idx", "kc", "vc")
    # the decode-reserve slots of the cache are not written by the pass: zero them on both sides
    buf.kc.zero_()
    buf.vc.zero_()
    buf.evict(q, k, v, schedule=schedule)
    torch.cuda.synchronize()
    eager = {n: getattr(buf, n).clone() for n in names}
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        buf.evict(q, k, v, schedule=schedule)
    torch.cuda.synchronize()
    for rep in range(3):
        for n in ("s_vis", "idx", "kc", "vc"):
            getattr(buf, n).zero_()
        buf.score(q, k, bd.SCORE_STATS)  # eager work between replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for n in names:
            assert torch.equal(getattr(buf, n), eager[n]), f"replay {rep}: {n}"
