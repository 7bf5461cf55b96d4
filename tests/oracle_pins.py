"""Pins for the fp64 oracle: what the paper and the mathematics fix, independent of the oracle's code.

Each check takes the oracle module ``O`` as an argument, so the mutation tests
can run the same checks against copies of the oracle with a planted mistake and
confirm that some check fails.  Checks raise AssertionError on failure.

Sources of truth used here (never the oracle's own formulas):
* independent library routines (scipy.special.softmax / logsumexp, torch SDPA);
* closed forms: zero queries give uniform causal rows; orthogonal one-hot keys
  give a softmax known exactly;
* invariants: each text row's mass splits into text and vision parts, so
  sum_j s^T_j + m = N_t; the normalised weights sum to 1; budgets sum to the
  global budget;
* brute force on tiny inputs: enumeration for largest-remainder rounding,
  pairwise dominance for top-k;
* the printed KV-memory column of the paper's efficiency table.
"""

from __future__ import annotations

import itertools
import json
import math
import os

import numpy as np

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _tiny_inputs(rng, H=4, H_kv=2, d=8, n_sys=3, n_vis=7, n_qst=5, scale_q=1.0):
    N, n_text = n_sys + n_vis + n_qst, n_sys + n_qst
    q = rng.standard_normal((H, n_text, d)) * scale_q
    k = rng.standard_normal((H_kv, N, d))
    return q, k


def _positions(n_sys, n_vis, n_qst):
    return list(range(n_sys)) + [n_sys + n_vis + i for i in range(n_qst)]


def _first_and_last(n, n_first, n_last):
    """App. A.2 spelled out by hand: positions 0..n_first-1 and n-n_last..n-1, clipped to [0, n)."""
    out = set()
    for p in range(n):
        if p < n_first or p >= n - n_last:
            out.add(p)
    return out


# ----------------------------------------------------------------------------- softmax rows
def check_softmax_rows(O, seed=0):
    """Rows of Eq. (2) restricted to text queries: sums, causal zeros, library softmax."""
    from scipy.special import logsumexp, softmax
    rng = np.random.default_rng(seed)
    for (H, H_kv, d, ns, nv, nq) in [(4, 2, 8, 3, 7, 5), (3, 3, 4, 0, 4, 3), (2, 1, 8, 4, 0, 2)]:
        q, k = _tiny_inputs(rng, H, H_kv, d, ns, nv, nq)
        tau = 1.0 / math.sqrt(d)
        P, lse = O.text_row_softmax(q, k, ns, nv, nq, tau)
        pi = _positions(ns, nv, nq)
        N = ns + nv + nq
        G = H // H_kv
        for h in range(H):
            for i, p in enumerate(pi):
                z = [tau * sum(float(q[h, i, t]) * float(k[h // G, j, t]) for t in range(d))
                     for j in range(p + 1)]
                ref = softmax(np.array(z))
                assert np.allclose(P[h, i, :p + 1], ref, rtol=1e-12, atol=1e-15)
                assert np.all(P[h, i, p + 1:] == 0.0)
                assert abs(P[h, i].sum() - 1.0) < 1e-12
                assert abs(lse[h, i] - logsumexp(np.array(z))) < 1e-12
        assert P.shape == (H, ns + nq, N)


# ----------------------------------------------------------------------------- invariants
def check_mass_split(O, seed=1):
    """Every text row sums to 1 and splits into text and vision parts: sum_j s^T_j + m = N_t."""
    rng = np.random.default_rng(seed)
    for (H, H_kv, d, ns, nv, nq) in [(4, 2, 8, 3, 7, 5), (6, 3, 16, 2, 11, 6), (2, 2, 8, 0, 5, 4)]:
        q, k = _tiny_inputs(rng, H, H_kv, d, ns, nv, nq, scale_q=2.0)
        n_text = ns + nq
        r1 = O.score_slice(q, k, ns, nv, nq, None, 0)
        assert r1["s_txt"].shape == (1, n_text)
        assert abs(r1["s_txt"].sum() + r1["tv_mass"] - n_text) < 1e-10
        # per KV-head groups: each group's text rows still sum to 1
        r2 = O.score_slice(q, k, ns, nv, nq, None, 1)
        P = r2["P"]
        G = H // H_kv
        for g in range(H_kv):
            grp_vis = P[g * G:(g + 1) * G, :, ns:ns + nv].mean(axis=0).sum()
            assert abs(r2["s_txt"][g].sum() + grp_vis - n_text) < 1e-10
        # system rows never see vision keys (causal mask)
        assert np.all(P[:, :ns, ns:] == 0.0)


def check_weights_and_vision_sum(O, seed=2):
    """w~ sums to 1 and is proportional to s^T_j / (N_t - j); sum_j s^V_j = sum_i w~_i vm_i."""
    rng = np.random.default_rng(seed)
    for mode in (0, 1):
        H, H_kv, d, ns, nv, nq = 4, 2, 8, 3, 9, 6
        q, k = _tiny_inputs(rng, H, H_kv, d, ns, nv, nq, scale_q=1.5)
        r = O.score_slice(q, k, ns, nv, nq, None, mode)
        n_text = ns + nq
        P = r["P"]
        G = H // H_kv
        groups = [list(range(H))] if mode == 0 else [list(range(g * G, (g + 1) * G)) for g in range(H_kv)]
        for gi, heads in enumerate(groups):
            wt = r["w_txt"][gi]
            assert abs(wt.sum() - 1.0) < 1e-12
            with np.errstate(divide="ignore", invalid="ignore"):  # a broken oracle may give 0 / 0
                ratio = np.array([r["s_txt"][gi][j] / (n_text - j) / wt[j] for j in range(n_text)])
            assert np.all(np.isfinite(ratio)) and ratio.max() - ratio.min() < 1e-9 * ratio.max()
            vm = [sum(P[h, i, ns + j] for h in heads for j in range(nv)) / len(heads) for i in range(n_text)]
            lhs = r["s_vis"][gi].sum()
            rhs = sum(wt[i] * vm[i] for i in range(n_text))
            assert abs(lhs - rhs) < 1e-12


# ----------------------------------------------------------------------------- closed forms
def check_zero_query(O):
    """q = 0: every visible key gets 1/(pi(i)+1); s^T, w, m and s^V follow in closed form."""
    ns, nv, nq, d = 4, 10, 6, 8
    H, H_kv = 4, 2
    rng = np.random.default_rng(3)
    q = np.zeros((H, ns + nq, d))
    k = rng.standard_normal((H_kv, ns + nv + nq, d))
    pi = _positions(ns, nv, nq)
    n_text = ns + nq
    for mode in (0, 1):
        r = O.score_slice(q, k, ns, nv, nq, None, mode)
        sT = [sum(1.0 / (pi[i] + 1) for i in range(j, n_text)) for j in range(n_text)]
        w = [sT[j] / (n_text - j) for j in range(n_text)]
        wt = [x / sum(w) for x in w]
        m = sum(nv / (pi[i] + 1) for i in range(ns, n_text))
        sV = sum(wt[i] / (pi[i] + 1) for i in range(ns, n_text))
        for g in range(r["s_txt"].shape[0]):
            assert np.allclose(r["s_txt"][g], sT, rtol=1e-13, atol=0)
            assert np.allclose(r["w_txt"][g], wt, rtol=1e-13, atol=0)
            assert np.allclose(r["s_vis"][g], sV, rtol=1e-13, atol=0)
        assert abs(r["tv_mass"] - m) < 1e-12
        lse_ref = np.log(np.array([pi[i] + 1.0 for i in range(n_text)]))
        assert np.allclose(r["lse"], lse_ref[None, :], rtol=0, atol=1e-13)


def planted_case(H=4, H_kv=2, ns=3, nv=6, nq=4, a=2.0, seed=4):
    """Orthogonal one-hot keys and one-hot queries aimed at chosen targets.

    Key j is c*e_j and query (h, i) is c*e_t(h,i) with t(h,i) <= pi(i), so the
    scaled logit is a = tau*c^2 on the target and 0 elsewhere; the softmax of
    row (h, i) is exactly e^a / (e^a + pi(i)) on the target and 1 / (e^a + pi(i))
    on every other visible key.
    """
    rng = np.random.default_rng(seed)
    N, n_text = ns + nv + nq, ns + nq
    d = N + 3
    tau = 1.0 / math.sqrt(d)
    c = math.sqrt(a / tau)
    pi = _positions(ns, nv, nq)
    k = np.zeros((H_kv, N, d))
    for g in range(H_kv):
        for j in range(N):
            k[g, j, j] = c
    tgt = np.zeros((H, n_text), dtype=int)
    q = np.zeros((H, n_text, d))
    for h in range(H):
        for i in range(n_text):
            tgt[h, i] = int(rng.integers(0, pi[i] + 1))
            q[h, i, tgt[h, i]] = c
    P = np.zeros((H, n_text, N))
    for h in range(H):
        for i in range(n_text):
            den = math.exp(a) + pi[i]
            for j in range(pi[i] + 1):
                P[h, i, j] = (math.exp(a) if j == tgt[h, i] else 1.0) / den
    return q, k, P, (ns, nv, nq)


def check_planted(O):
    """Closed-form softmax with distinct targets per head and row pins every index."""
    H, H_kv = 4, 2
    q, k, P, (ns, nv, nq) = planted_case(H, H_kv)
    n_text = ns + nq
    pi = _positions(ns, nv, nq)
    G = H // H_kv
    for mode in (0, 1):
        r = O.score_slice(q, k, ns, nv, nq, None, mode)
        groups = [list(range(H))] if mode == 0 else [list(range(g * G, (g + 1) * G)) for g in range(H_kv)]
        for gi, heads in enumerate(groups):
            Ab = [[sum(P[h, i, j] for h in heads) / len(heads) for j in range(P.shape[2])] for i in range(n_text)]
            sT = [sum(Ab[i][pi[j]] for i in range(j, n_text)) for j in range(n_text)]
            w = [sT[j] / (n_text - j) for j in range(n_text)]
            wt = [x / sum(w) for x in w]
            sV = [sum(wt[i] * Ab[i][ns + j] for i in range(n_text)) for j in range(nv)]
            assert np.allclose(r["s_txt"][gi], sT, rtol=1e-12, atol=1e-15)
            assert np.allclose(r["w_txt"][gi], wt, rtol=1e-12, atol=1e-15)
            assert np.allclose(r["s_vis"][gi], sV, rtol=1e-12, atol=1e-15)
        m = sum(P[h, i, ns + j] for h in range(H) for i in range(n_text) for j in range(nv)) / H
        assert abs(r["tv_mass"] - m) < 1e-12
        assert np.allclose(r["P"], P, rtol=1e-12, atol=1e-15)


# ----------------------------------------------------------------------------- budgets
def _brute_round(x, total):
    """Integer vector with entries floor/ceil of x summing to total that minimises sum (b - x)^2;
    among equal costs the one giving the +1 to lower layers (lexicographically largest)."""
    lo = [math.floor(v) for v in x]
    best = None
    for bits in itertools.product((0, 1), repeat=len(x)):
        b = [lo[i] + bits[i] for i in range(len(x))]
        if sum(b) != total:
            continue
        cost = sum((b[i] - x[i]) ** 2 for i in range(len(x)))
        key = (round(cost, 9), tuple(-v for v in b))
        if best is None or key < best[0]:
            best = (key, b)
    return best[1]


def check_budgets(O, seed=5):
    rng = np.random.default_rng(seed)
    # sums, bounds, rho = 1 keeps everything
    for L, N in [(1, 10), (4, 7), (32, 651), (7, 1)]:
        for _ in range(6):
            m = rng.random(L) * rng.choice([1e-3, 1.0, 50.0])
            for tot in sorted({0, 1, L * N // 3, L * N // 2, L * N - 1, L * N}):
                if tot < 0:
                    continue
                b = O.layer_budgets(m, tot, N)
                assert b.sum() == tot and b.min() >= 0 and b.max() <= N
        b = O.layer_budgets(rng.random(L), L * N, N)
        assert np.all(b == N)
    # a single layer takes the whole budget
    assert list(O.layer_budgets([0.3], 17, 168)) == [17]
    # equal masses: budgets differ by at most one and the extras go to the lowest layers
    for L, N, tot in [(32, 2979, 4766), (5, 100, 13), (28, 8256, 11558)]:
        b = O.layer_budgets([0.7] * L, tot, N)
        q, r = divmod(tot, L)
        assert list(b) == [q + 1] * r + [q] * (L - r)
    # zero total mass falls back to uniform shares
    assert list(O.layer_budgets([0.0, 0.0, 0.0], 10, 9)) == [4, 3, 3]
    # brute-force largest remainder when no cap binds
    for _ in range(40):
        L = int(rng.integers(1, 6))
        N = 1000
        m = rng.random(L) + 1e-3
        tot = int(rng.integers(0, 60))
        x = [tot * v / m.sum() for v in m]
        b = O.layer_budgets(m, tot, N)
        assert list(b) == _brute_round(x, tot), (m, tot)
    # the cap is water-filled: one dominant layer stops at N, the rest share the remainder
    assert list(O.layer_budgets([100.0, 1.0, 1.0, 1.0], 20, 10)) == [10, 4, 3, 3]
    assert list(O.layer_budgets([100.0, 100.0, 1.0, 2.0], 25, 10)) == [10, 10, 2, 3]
    # a floor is given first to every layer
    assert list(O.layer_budgets([1.0, 0.0, 0.0, 0.0], 20, 30, n_floor=5)) == [5, 5, 5, 5]
    b = O.layer_budgets([1.0, 0.0, 0.0, 0.0], 20, 30, n_floor=3)
    assert list(b) == [3 + 8, 3, 3, 3]
    # monotone: raising one layer's mass never lowers its budget
    for _ in range(30):
        L, N = 8, 200
        m = rng.random(L) + 0.01
        tot = int(rng.integers(1, L * N))
        l = int(rng.integers(0, L))
        b0 = O.layer_budgets(m, tot, N)[l]
        m2 = m.copy()
        m2[l] *= 1.0 + rng.random() * 3
        assert O.layer_budgets(m2, tot, N)[l] >= b0


def check_efficiency_memory(O):
    """KV memory of the paper's efficiency table equals rho x the full cache (per-sequence budget)."""
    with open(os.path.join(GOLDEN, "efficiency_memory.json")) as f:
        gold = json.load(f)
    from workloads import total_budget
    L = gold["layers"]
    row_bytes = 2 * gold["kv_width"] * gold["bytes_per_elem"]      # K and V rows of one token
    for ctx in gold["contexts"]:
        n = ctx["tokens"]
        for rho_s, printed in ctx["memory_gb"].items():
            rho = float(rho_s)
            tot = total_budget(rho, n, L)
            b = O.layer_budgets(np.ones(L), tot, n)
            gib = int(b.sum()) * row_bytes / 2 ** 30
            assert round(gib, 2) == printed, (n, rho, gib, printed)


# ----------------------------------------------------------------------------- retention
def _rank_key(p, sc_t, sc_v, ns, nv, forced):
    """Ordering of Eq. (10) with forced tokens first: (class, -score, position)."""
    if p in forced:
        return (0, 0.0, p)
    if ns <= p < ns + nv:
        return (2, -sc_v[p - ns], p)
    ti = p if p < ns else p - nv
    return (1, -sc_t[ti], p)


def check_tpr(O, seed=6):
    rng = np.random.default_rng(seed)
    for _ in range(200):
        ns, nv, nq = (int(x) for x in rng.integers(0, 9, size=3))
        N = ns + nv + nq
        if N == 0:
            continue
        n_text = ns + nq
        # ties are common: draw from a small set of values
        sv = rng.integers(0, 4, size=nv).astype(float) / 4
        st = rng.integers(0, 4, size=n_text).astype(float) / 4
        n_sink, n_recent = (0, 0) if rng.random() < 0.5 else (int(rng.integers(0, 5)), int(rng.integers(0, 3)))
        forced = _first_and_last(N, n_sink, n_recent)
        for b in range(0, N + 1):
            I = O.tpr_select(sv, st, b, ns, nv, nq, n_sink, n_recent)
            I = list(I)
            assert len(I) == b and len(set(I)) == b
            assert I == sorted(I)
            tset = set(_positions(ns, nv, nq))
            if not forced:
                if b > n_text:
                    assert tset <= set(I)
                else:
                    assert set(I) <= tset
            dropped = [p for p in range(N) if p not in set(I)]
            if b >= len(forced):
                assert forced <= set(I)
            for a in I:
                for c in dropped:
                    assert _rank_key(a, st, sv, ns, nv, forced) < _rank_key(c, st, sv, ns, nv, forced)
        # keeping everything
        assert list(O.tpr_select(sv, st, N, ns, nv, nq)) == list(range(N))


# ----------------------------------------------------------------------------- cache and decode
def check_compact_and_decode(O, seed=7):
    import torch
    rng = np.random.default_rng(seed)
    H, H_kv, d, N = 4, 2, 16, 23
    k = rng.standard_normal((H_kv, N, d))
    v = rng.standard_normal((H_kv, N, d))
    allidx = [np.arange(N)]
    Kc, Vc = O.compact_slice(k, v, allidx, 0)
    for h in range(H_kv):
        assert np.array_equal(Kc[h], k[h]) and np.array_equal(Vc[h], v[h])
    sel = [np.array([0, 3, 4, 9, 22]), np.array([1, 2, 5, 6, 7])]
    Kc, Vc = O.compact_slice(k, v, sel, 1)
    for h in range(H_kv):
        for n, p in enumerate(sel[h]):
            assert np.array_equal(Kc[h][n], k[h][p]) and np.array_equal(Vc[h][n], v[h][p])
    # full cache plus two appended tokens equals a textbook attention routine
    T = 2
    qs = rng.standard_normal((T, H, d))
    kn = rng.standard_normal((T, H_kv, d))
    vn = rng.standard_normal((T, H_kv, d))
    tau = 1.0 / math.sqrt(d)
    Kc, Vc = O.compact_slice(k, v, allidx, 0)
    outs = O.decode_reference(qs, kn, vn, Kc, Vc, tau)
    G = H // H_kv
    for t in range(T):
        K = np.concatenate([k, kn[:t + 1].transpose(1, 0, 2)], axis=1)
        V = np.concatenate([v, vn[:t + 1].transpose(1, 0, 2)], axis=1)
        qt = torch.tensor(qs[t][:, None, :], dtype=torch.float64)              # [H][1][d]
        Kt = torch.tensor(np.repeat(K, G, axis=0), dtype=torch.float64)
        Vt = torch.tensor(np.repeat(V, G, axis=0), dtype=torch.float64)
        ref = torch.nn.functional.scaled_dot_product_attention(qt, Kt, Vt, scale=tau)[:, 0, :].numpy()
        assert np.allclose(outs[t], ref, rtol=1e-12, atol=1e-12)
    # an empty retained set at the first step attends only to the appended token
    Kc0 = [np.zeros((0, d)) for _ in range(H_kv)]
    out0 = O.decode_reference(qs[:1], kn[:1], vn[:1], Kc0, Kc0, tau)
    for h in range(H):
        assert np.array_equal(out0[0][h], vn[0][h // G])


def check_vision_only(O, seed=8):
    """Vision-only eviction (App. B.3): all text kept, the budget counts vision tokens."""
    rng = np.random.default_rng(seed)
    for L, nt, nv in [(1, 4, 10), (4, 3, 7), (32, 75, 576), (5, 0, 9)]:
        for _ in range(4):
            m = rng.random(L) * rng.choice([1e-3, 1.0, 50.0])
            for V in sorted({0, 1, L * nv // 3, L * nv - 1, L * nv}):
                b = O.vision_only_budgets(m, V, nt, nv)
                # every layer keeps its text, the vision part respects the vision cap, sums add up
                assert b.sum() == L * nt + V and b.min() >= nt and (b - nt).max() <= nv, (L, nt, nv, V, b)
        # rho = 1 keeps every token, rho = 0 keeps exactly the text
        assert np.all(O.vision_only_budgets(rng.random(L), L * nv, nt, nv) == nt + nv)
        assert np.all(O.vision_only_budgets(rng.random(L), 0, nt, nv) == nt)
    # equal masses: vision shares differ by at most one, extras on the lowest layers
    L, nt, nv, V = 32, 99, 2880, 4608 + 7
    b = O.vision_only_budgets([0.5] * L, V, nt, nv)
    q, r = divmod(V, L)
    assert list(b - nt) == [q + 1] * r + [q] * (L - r)
    # the cap is the vision count, not the sequence length: a dominant layer stops at n_vis
    assert list(O.vision_only_budgets([100.0, 1.0, 1.0, 1.0], 20, 5, 10)) == [15, 9, 8, 8]
    # forced vision positions (a sink at position 0 with no system text) are kept like the text;
    # the budget shares out the other vision tokens
    assert O.forced_vision_count(0, 12, 3, n_sink=4, n_recent=1) == 4
    assert O.forced_vision_count(2, 12, 3, n_sink=4, n_recent=1) == 2
    assert O.forced_vision_count(5, 12, 3, n_sink=4, n_recent=1) == 0
    b = O.vision_only_budgets([1.0, 0.0, 0.0, 0.0], 20, 3, 12, n_forced_vis=4)
    assert list(b) == [3 + 4 + 8, 3 + 4 + 4, 3 + 4 + 4, 3 + 4 + 4]
    assert np.all(O.vision_only_budgets([1.0, 2.0], 0, 3, 12, n_forced_vis=4) == 7)
    # retention: all text, then exactly b_l - N_t vision tokens, the top ones by s^V (brute force)
    for _ in range(100):
        ns, nv, nq = int(rng.integers(0, 4)), int(rng.integers(1, 12)), int(rng.integers(0, 4))
        n = ns + nv + nq
        sv = np.round(rng.standard_normal(nv), 1)        # coarse grid: many ties
        st = np.round(rng.random(ns + nq), 1)
        v = int(rng.integers(0, nv + 1))
        keep = O.tpr_select(sv, st, ns + nq + v, ns, nv, nq)
        text = set(range(ns)) | set(range(ns + nv, n))
        assert text <= set(keep.tolist()) and len(keep) == ns + nq + v
        best = sorted(range(nv), key=lambda j: (-sv[j], j))[:v]
        assert sorted(set(keep.tolist()) - text) == sorted(ns + j for j in best)
    # whole sequence: budgets and sets of every layer
    ns, nv, nq, L = 3, 20, 4, 3
    q, k = [], []
    for _ in range(L):
        qq, kk = _tiny_inputs(rng, n_sys=ns, n_vis=nv, n_qst=nq)
        q.append(qq)
        k.append(kk)
    V = 17
    scores, b, idx = O.evict_sequence(q, k, ns, nv, nq, V, vision_only=True)
    assert b.sum() == L * (ns + nq) + V
    text = set(range(ns)) | set(range(ns + nv, ns + nv + nq))
    for l in range(L):
        assert text <= set(idx[l][0].tolist()) and len(idx[l][0]) == b[l]


def check_variants(O, seed=9):
    """Budget rules, the plain attention sum and ranking without TPR (Table 1(a), Table 5)."""
    rng = np.random.default_rng(seed)
    # uniform budgets ignore the masses: the closed form of an equal split
    for L, N, tot in [(32, 2979, 4766), (5, 100, 13), (7, 40, 0)]:
        m = rng.random(L) * 10
        b = O.layer_budgets(O.budget_masses(m, 1, 99), tot, N)
        q, r = divmod(tot, L)
        assert list(b) == [q + 1] * r + [q] * (L - r)
    # the text->text rule: N_t minus the text->vision mass, clamped at 0, non-finite masses as 0
    tt = O.budget_masses([0.25, 0.875, 0.5, 3.0, float("nan")], 2, 1)
    assert tt == [0.75, 0.125, 0.5, 0.0, 1.0]
    assert list(O.layer_budgets(tt[:3], 11, 100)) == [6, 1, 4]  # shares 0.75 : 0.125 : 0.5 of 11
    # ... and the identity behind it, from the oracle's own softmax: the head-averaged mass of
    # the text x text block plus the text->vision mass is N_t
    for head_mode in (0, 1):
        q, k = _tiny_inputs(rng, n_sys=3, n_vis=7, n_qst=5)
        P, _ = O.text_row_softmax(q, k, 3, 7, 5, 0.4)
        tpos = _positions(3, 7, 5)
        tt_direct = P[:, :, tpos].sum(axis=(1, 2)).mean()
        assert abs(tt_direct + O.tv_mass(P, 3, 7) - 8) < 1e-9
    # plain attention sum: unit weights, and the vision scores add up to the layer's TV mass
    for head_mode in (0, 1):
        q, k = _tiny_inputs(rng, n_sys=2, n_vis=9, n_qst=4)
        sc = O.score_slice(q, k, 2, 9, 4, 0.5, head_mode, vision_rank=1)
        assert np.all(sc["w_txt"] == 1.0)
        if head_mode == 0:
            assert abs(sc["s_vis"].sum() - sc["tv_mass"]) < 1e-9
        tw = O.score_slice(q, k, 2, 9, 4, 0.5, head_mode)
        assert np.allclose(tw["s_txt"], sc["s_txt"]) and not np.allclose(tw["s_vis"], sc["s_vis"])
    # ranking without TPR: forced first, then every other token on one scale (pairwise dominance)
    for _ in range(200):
        ns, nv, nq = int(rng.integers(0, 4)), int(rng.integers(0, 10)), int(rng.integers(0, 4))
        n = ns + nv + nq
        if n == 0:
            continue
        fs, fr = int(rng.integers(0, 3)), int(rng.integers(0, 2))
        sv = np.round(rng.random(nv), 1)
        st = np.round(rng.random(ns + nq) * 3, 1)
        scale = float(rng.choice([1.0, ns + nq if ns + nq else 1.0]))
        b = int(rng.integers(0, n + 1))
        keep = O.joint_select(sv, st, b, ns, nv, nq, fs, fr, scale)
        assert len(keep) == b and np.all(np.diff(keep) > 0)
        forced = _first_and_last(n, fs, fr)
        score = {}
        for i, p_ in enumerate(_positions(ns, nv, nq)):
            score[p_] = st[i]
        for j in range(nv):
            score[ns + j] = scale * sv[j]
        kept = set(keep.tolist())
        if b >= len(forced):
            assert forced <= kept
            for p_ in kept - forced:
                for q_ in set(range(n)) - kept - forced:
                    assert score[p_] > score[q_] or (score[p_] == score[q_] and p_ < q_), (p_, q_)
    # a dominant vision token beats the text without TPR, and never with it
    assert list(O.joint_select([5.0, 0.0], [1.0, 1.0], 1, 1, 2, 1)) == [1]
    assert list(O.tpr_select([5.0, 0.0], [1.0, 1.0], 1, 1, 2, 1)) == [0]


# ----------------------------------------------------------------------------- forced tokens
def _vision_blind_layer(rng, H, H_kv, d, ns, nv, nq, blind):
    """One layer's q/k whose question rows put exactly zero float64 mass on vision keys if blind.

    Every key is +-c u for one unit direction u and every question query is +c u, so a
    question row's logits are +c^2/sqrt(d) on text keys and -c^2/sqrt(d) on vision keys.
    With c^2/sqrt(d) = 400 the vision probabilities are exp(-800) relative to the text ones,
    which is 0 in float64.  System rows never see vision keys (causal mask).  A layer that is
    not blind gets random keys, so its mass is positive.
    """
    N, n_text = ns + nv + nq, ns + nq
    u = np.zeros(d)
    u[0] = 1.0
    c = math.sqrt(400.0 * math.sqrt(d))
    if not blind:
        return rng.standard_normal((H, n_text, d)), rng.standard_normal((H_kv, N, d))
    k = np.tile(c * u, (H_kv, N, 1))
    k[:, ns:ns + nv] = -c * u
    q = np.tile(c * u, (H, n_text, 1))
    return q, k


def check_forced(O, seed=10):
    """App. A.2 keeps the first 4 and the last 1 tokens: closed forms, and the per-layer floor of TVB.

    The floor: with forced tokens every layer first gets F = min(|forced|, B_tot // L, N) of
    the budget and the rest R = B_tot - L*F is shared by mass, so masses (m, 0, 0, 0) give
    budgets (F + R, F, F, F) and the three zero-mass layers keep exactly the forced positions.
    """
    # closed forms of the forced set
    assert list(O.forced_positions(10, 4, 1)) == [0, 1, 2, 3, 9]
    assert list(O.forced_positions(10, 4, 0)) == [0, 1, 2, 3]
    assert list(O.forced_positions(10, 0, 1)) == [9]
    assert list(O.forced_positions(10, 0, 3)) == [7, 8, 9]
    assert list(O.forced_positions(10, 0, 0)) == []
    assert list(O.forced_positions(5, 4, 1)) == [0, 1, 2, 3, 4]       # n_sink + n_recent == N
    assert list(O.forced_positions(4, 4, 1)) == [0, 1, 2, 3]          # overlap: the last token is a sink
    assert list(O.forced_positions(3, 4, 2)) == [0, 1, 2]             # both larger than N
    assert list(O.forced_positions(1, 0, 1)) == [0]
    assert list(O.forced_positions(0, 4, 1)) == []
    for n in range(0, 12):
        for a in range(0, 6):
            for r in range(0, 4):
                f = O.forced_positions(n, a, r)
                assert set(f.tolist()) == _first_and_last(n, a, r) and list(f) == sorted(f), (n, a, r)
    # the forced set is what a budget of |forced| keeps, whatever the scores
    ns, nv, nq = 3, 12, 5
    st = np.linspace(1.0, 0.0, ns + nq)
    sv = np.linspace(0.0, 1.0, nv)
    assert list(O.tpr_select(sv, st, 5, ns, nv, nq, 4, 1)) == [0, 1, 2, 3, ns + nv + nq - 1]
    assert list(O.joint_select(sv, st, 5, ns, nv, nq, 4, 1)) == [0, 1, 2, 3, ns + nv + nq - 1]
    # whole sequence: layer 0 sees vision, layers 1..3 put zero mass on it
    rng = np.random.default_rng(seed)
    H, H_kv, d, L = 4, 2, 16, 4
    N = ns + nv + nq
    q, k = [], []
    for l in range(L):
        ql, kl = _vision_blind_layer(rng, H, H_kv, d, ns, nv, nq, blind=l > 0)
        q.append(ql)
        k.append(kl)
    for tot in (24, 30, 35):
        scores, b, idx = O.evict_sequence(q, k, ns, nv, nq, tot, n_sink=4, n_recent=1)
        assert scores[0]["tv_mass"] > 0.0
        for l in range(1, L):
            assert scores[l]["tv_mass"] == 0.0
        F = min(5, tot // L, N)
        assert list(b) == [F + tot - L * F, F, F, F], (tot, list(b))
        for l in range(1, L):
            assert list(idx[l][0]) == [0, 1, 2, 3, N - 1]
        assert {0, 1, 2, 3, N - 1} <= set(idx[0][0].tolist())
    # past the cap N the dominant layer stops at N and the rest is shared evenly, lower layers first
    scores, b, idx = O.evict_sequence(q, k, ns, nv, nq, 37, n_sink=4, n_recent=1)
    assert list(b) == [N, 5 + 1, 5 + 1, 5]
    # a budget below L*|forced| floors at B_tot // L and keeps the first forced positions
    scores, b, idx = O.evict_sequence(q, k, ns, nv, nq, 13, n_sink=4, n_recent=1)
    assert list(b) == [3 + 1, 3, 3, 3]
    for l in range(1, L):
        assert list(idx[l][0]) == [0, 1, 2]
    # without forced tokens the same masses give everything to layer 0
    scores, b, idx = O.evict_sequence(q, k, ns, nv, nq, 18, n_sink=0, n_recent=0)
    assert list(b) == [18, 0, 0, 0]


ALL_CHECKS = [
    check_softmax_rows,
    check_mass_split,
    check_weights_and_vision_sum,
    check_zero_query,
    check_planted,
    check_budgets,
    check_efficiency_memory,
    check_tpr,
    check_compact_and_decode,
    check_vision_only,
    check_variants,
    check_forced,
]
