"""Pins for the CPU oracle (runs without a GPU).

The oracle is checked against things other than itself: hand-derived golden
cases, the brute-force definitions in tests/brute.py (a different route),
closed forms, invariants and reductions to textbook/library routines. The
mutation tests at the end plant plausible mistakes in a temporary copy of
the oracle's C source and check that these pins catch every one of them.
"""
import ctypes
import dataclasses
import json
import math
import os
import shutil
import subprocess
from fractions import Fraction

import numpy as np
import pytest
import scipy.special

import brute
import oracle
from paper_2607_27952_amd import workloads as W

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _load(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def _orc_scores(wl, **kw):
    return oracle.scores(wl.R, wl.G, wl.Hq, wl.Hkv, wl.Dh, wl.q, wl.k, wl.cu_seqlens, wl.vis_start,
                         wl.cu_vis, oracle.BF16 if wl.qk_dtype == W.BF16 else oracle.F32,
                         scale=wl.scale, **kw)


def _fcode(dtype):
    return oracle.BF16 if dtype == W.BF16 else oracle.F32


def _make_wl(q, k, cu_seqlens, vis_start, cu_vis, Hq, Hkv, scale, dtype=W.F32, feats=None, Dv=1):
    q = np.asarray(q, np.float32)
    k = np.asarray(k, np.float32)
    R = len(cu_seqlens) - 1
    N = int(cu_vis[-1])
    if feats is None:
        feats = np.ones((N, Dv), np.float32)
    return W.Workload(name="handmade", R=R, G=q.shape[0], Hq=Hq, Hkv=Hkv, Dh=q.shape[-1],
                      qk_dtype=dtype, scale=scale, cu_seqlens=np.asarray(cu_seqlens, np.int32),
                      vis_start=np.asarray(vis_start, np.int32), cu_vis=np.asarray(cu_vis, np.int32),
                      q=W.to_bf16_bits(q) if dtype == W.BF16 else q,
                      k=W.to_bf16_bits(k) if dtype == W.BF16 else k,
                      Dv=feats.shape[1], f_dtype=W.F32, feats=feats,
                      cu_keep=np.asarray([0] + [1] * R, np.int32).cumsum().astype(np.int32))


# ---------------------------------------------------------------- scores (Eq. 6-8)

def test_scores_golden_two_heads():
    g = _load("scores_two_heads.json")
    wl = _make_wl(g["q"], g["k"], g["cu_seqlens"], g["vis_start"], g["cu_vis"], g["Hq"], g["Hkv"], g["scale"])
    w, rows = _orc_scores(wl, want_rows=True)
    np.testing.assert_allclose(w, g["w"], rtol=g["rel_tol"])
    np.testing.assert_allclose(rows, np.asarray(g["rows"]), rtol=g["rel_tol"])


@pytest.mark.parametrize("seed", range(12))
def test_scores_match_bruteforce(seed):
    rng = np.random.default_rng(seed)
    Hkv = int(rng.choice([1, 2, 3]))
    g = int(rng.choice([1, 2, 3, 7]))
    wl = W.tiny(seed, R=int(rng.integers(1, 4)), G=int(rng.integers(1, 4)), Hq=Hkv * g, Hkv=Hkv,
                Dh=int(rng.choice([4, 8, 16])), n_range=(1, 24), t_range=(1, 12),
                qk_dtype=[W.F32, W.BF16][seed % 2])
    w, rows = _orc_scores(wl, want_rows=True)
    wb, rows_b = brute.scores(wl, rng=np.random.default_rng(seed + 100), want_rows=True)
    np.testing.assert_allclose(w, wb, rtol=1e-12, atol=0)
    np.testing.assert_allclose(rows, rows_b, rtol=1e-11, atol=1e-300)


def test_scores_rows_sum_to_one_and_w_normalised():
    wl = W.tiny(5, R=3, G=2, Hq=6, Hkv=2, Dh=16, n_range=(5, 40), t_range=(2, 20))
    w, rows = _orc_scores(wl, want_rows=True)
    for r in range(wl.R):
        a, b = wl.cu_seqlens[r], wl.cu_seqlens[r + 1]
        np.testing.assert_allclose(rows[:, :, a:b].sum(axis=2), 1.0, atol=1e-12)
        seg = w[wl.cu_vis[r]:wl.cu_vis[r + 1]]
        assert abs(seg.sum() - 1.0) < 1e-12 and (seg >= 0).all()


def test_scores_uniform_keys_closed_form():
    """All keys equal: every row is uniform, so w_i = 1/N for any G, Hq."""
    rng = np.random.default_rng(1)
    N, T, G, Hq, Hkv, Dh = 37, 11, 3, 6, 3, 8
    P = N + T
    q = rng.standard_normal((G, 1, Hq, Dh))
    k = np.broadcast_to(rng.standard_normal((1, 1, Hkv, Dh)), (G, P, Hkv, Dh)).copy()
    wl = _make_wl(q, k, [0, P], [T // 4], [0, N], Hq, Hkv, 0.3)
    np.testing.assert_allclose(_orc_scores(wl), 1.0 / N, rtol=1e-13)


@pytest.mark.parametrize("delta", [0.5, 3.0, 9.0])
def test_scores_planted_key_closed_form(delta):
    """Zero keys except one visual key with scaled logit delta in every head:
    w_planted = e^delta / (N - 1 + e^delta), whatever G and Hq."""
    rng = np.random.default_rng(2)
    N, T, G, Hkv, g, Dh, scale = 29, 7, 2, 2, 3, 8, 0.25
    Hq = Hkv * g
    P = N + T
    v0, planted = 3, 11
    q = np.zeros((G, 1, Hq, Dh))
    k = np.zeros((G, P, Hkv, Dh))
    for l in range(G):
        for kv in range(Hkv):
            u = rng.standard_normal(Dh)
            q[l, 0, kv * g:(kv + 1) * g] = u           # heads of one group share a query
            k[l, v0 + planted, kv] = (delta / scale) * u / np.dot(u, u)
    wl = _make_wl(q.astype(np.float32), k, [0, P], [v0], [0, N], Hq, Hkv, scale)
    # the fp32 rounding of q and k moves the planted logit by ~1e-7 relative
    qq = W.as_f32(wl.q, W.F32).astype(np.float64)
    kk = W.as_f32(wl.k, W.F32).astype(np.float64)
    w = _orc_scores(wl)
    # exact expectation from the rounded inputs, per head (closed form per row)
    s = np.zeros(N)
    for l in range(G):
        for h in range(Hq):
            d = scale * np.dot(qq[l, 0, h], kk[l, v0 + planted, h // g])
            e = math.exp(d)
            row_vis = np.full(N, 1.0 / (P - 1 + e))
            row_vis[planted] = e / (P - 1 + e)
            s += row_vis
    np.testing.assert_allclose(w, s / s.sum(), rtol=1e-13)
    assert abs(w[planted] - math.exp(delta) / (N - 1 + math.exp(delta))) < 1e-5


def test_scores_single_head_is_softmax_over_visual_logits():
    """G = Hq = 1: the text mass cancels in Eq. 8, leaving softmax over the visual logits."""
    wl = W.tiny(9, R=2, G=1, Hq=1, Hkv=1, Dh=16, n_range=(10, 30), t_range=(3, 9), qk_dtype=W.F32)
    w = _orc_scores(wl)
    q = W.as_f32(wl.q, W.F32).astype(np.float64)
    k = W.as_f32(wl.k, W.F32).astype(np.float64)
    for r in range(wl.R):
        a = int(wl.cu_seqlens[r]) + int(wl.vis_start[r])
        logits = wl.scale * k[0, a:a + wl.n(r), 0] @ q[0, r, 0]
        np.testing.assert_allclose(w[wl.cu_vis[r]:wl.cu_vis[r + 1]], scipy.special.softmax(logits), rtol=1e-13)


def test_scores_two_token_row_is_logistic():
    """P = 2: the last row is (expit(l0 - l1), expit(l1 - l0))."""
    q = np.array([[[[0.3, -1.2, 0.7, 2.0]]]])
    k = np.array([[[[1.0, 0.5, -0.25, 0.125]]], [[[-2.0, 1.0, 0.5, 0.75]]]]).reshape(1, 2, 1, 4)
    wl = _make_wl(q, k, [0, 2], [0], [0, 1], 1, 1, 0.5)
    w, rows = _orc_scores(wl, want_rows=True)
    qf = W.as_f32(wl.q, W.F32).astype(np.float64)[0, 0, 0]
    kf = W.as_f32(wl.k, W.F32).astype(np.float64)[0, :, 0]
    l0, l1 = 0.5 * kf[0] @ qf, 0.5 * kf[1] @ qf
    np.testing.assert_allclose(rows[0, 0], [scipy.special.expit(l0 - l1), scipy.special.expit(l1 - l0)], rtol=1e-13)
    assert w[0] == 1.0


@pytest.mark.parametrize("c", [-80.0, 80.0])
def test_scores_logit_shift_invariance(c):
    """Adding c to every logit of a row (k_j += c q / (sigma |q|^2)) leaves w unchanged."""
    wl = W.tiny(4, R=2, G=2, Hq=3, Hkv=3, Dh=8, n_range=(6, 20), t_range=(2, 8), qk_dtype=W.F32)
    w0 = _orc_scores(wl)
    k = W.as_f32(wl.k, W.F32).astype(np.float64).copy()
    q = W.as_f32(wl.q, W.F32).astype(np.float64)
    for l in range(wl.G):
        for r in range(wl.R):
            a, b = wl.cu_seqlens[r], wl.cu_seqlens[r + 1]
            for h in range(wl.Hq):
                u = q[l, r, h]
                k[l, a:b, h] += c * u / (wl.scale * np.dot(u, u))
    wl2 = _make_wl(wl.q, k, wl.cu_seqlens, wl.vis_start, wl.cu_vis, wl.Hq, wl.Hkv, wl.scale)
    w1 = _orc_scores(wl2)
    assert np.all(np.isfinite(w1))
    np.testing.assert_allclose(w1, w0, rtol=2e-5)   # the shifted keys are rounded to fp32


def test_scores_permuting_visual_keys_permutes_w():
    wl = W.tiny(6, R=1, G=2, Hq=4, Hkv=2, Dh=8, n_range=(12, 12), t_range=(5, 5), qk_dtype=W.F32)
    w0 = _orc_scores(wl)
    perm = np.random.default_rng(0).permutation(12)
    k = wl.k.copy()
    v0 = int(wl.vis_start[0])
    k[:, v0:v0 + 12] = wl.k[:, v0 + perm]
    wl2 = _make_wl(wl.q, k, wl.cu_seqlens, wl.vis_start, wl.cu_vis, wl.Hq, wl.Hkv, wl.scale)
    np.testing.assert_allclose(_orc_scores(wl2), w0[perm], rtol=1e-14)


# ---------------------------------------------------------------- selection (Eq. 9-12)

def _sel(w, X, K, mode=oracle.KCENTER, dtype=W.F32):
    X = np.asarray(X)
    N = X.shape[0]
    return oracle.select(1, X.shape[1], np.asarray(w, np.float32), X, [0, N], [0, K],
                         _fcode(dtype), mode=mode)


def test_select_golden_cases():
    for case in _load("select_four_tokens.json")["cases"]:
        X = np.asarray(case["feats"], np.float32)
        kept, order, gains = _sel(case["w"], X, case["K"])
        assert list(order) == case["order"], case["name"]
        assert list(kept) == case["kept"], case["name"]
        np.testing.assert_allclose(gains, case["gains"], rtol=max(case["gain_rel_tol"], 1e-12), atol=1e-12)
        kept, order, _ = _sel(case["w"], X, case["K"], mode=oracle.TOPK)
        assert list(kept) == case["topk_kept"] and list(order) == case["topk_order"], case["name"]


@pytest.mark.parametrize("seed", range(16))
def test_select_matches_bruteforce(seed):
    rng = np.random.default_rng(seed)
    N = int(rng.integers(2, 64))
    Dv = int(rng.choice([3, 8, 32]))
    X = rng.standard_normal((N, Dv)).astype(np.float32)
    distinct = N
    if seed % 3 == 0:                               # some exact duplicates
        X[N // 2:] = X[:N - N // 2]
        distinct = N // 2
    w = rng.dirichlet(np.ones(N)).astype(np.float32)
    # beyond the distinct rows every objective is a rounding-level zero, where the
    # two routes may legitimately differ; that regime is pinned by exact cases instead
    K = int(rng.integers(1, max(1, distinct) + 1))
    kept, order, gains = _sel(w, X, K)
    ob, gb = brute.select(w, X, K)
    assert list(order) == list(ob)
    np.testing.assert_allclose(gains, gb, rtol=1e-12, atol=1e-15)
    assert list(kept) == sorted(ob)


def test_select_bf16_features_match_bruteforce():
    wl = W.tiny(21, R=3, n_range=(20, 60), Dv=48, comps=5)
    w = np.random.default_rng(0).dirichlet(np.ones(wl.N_total)).astype(np.float32)
    kept, order, _ = oracle.select(wl.R, wl.Dv, w, wl.feats, wl.cu_vis, wl.cu_keep, oracle.BF16)
    X = W.as_f32(wl.feats, W.BF16)
    for r in range(wl.R):
        a, b = wl.cu_vis[r], wl.cu_vis[r + 1]
        ob, _ = brute.select(w[a:b], X[a:b], wl.kk(r))
        assert list(order[wl.cu_keep[r]:wl.cu_keep[r + 1]]) == list(ob)


def test_select_orthogonal_features_is_topk():
    """One-hot features: every coverage distance is 1, so the greedy is top-K by w."""
    rng = np.random.default_rng(3)
    N = 40
    X = np.eye(N, dtype=np.float32) * rng.uniform(0.5, 3.0, size=(N, 1)).astype(np.float32)
    w = rng.dirichlet(np.ones(N)).astype(np.float32)
    w[7] = w[19]                                        # an exact tie
    K = 17
    _, order, _ = _sel(w, X, K)
    expect = np.argsort(-w.astype(np.float64), kind="stable")[:K]
    assert list(order) == list(expect)


def test_select_uniform_weights_is_farthest_point():
    rng = np.random.default_rng(4)
    X = rng.standard_normal((50, 6)).astype(np.float32)
    w = np.full(50, 1.0 / 50, np.float32)
    _, order, _ = _sel(w, X, 12)
    assert list(order) == list(brute.gonzalez(X.astype(np.float64), 12))


def test_select_identical_features():
    """delta is 0 after the first pick, so the rest are the lowest remaining indices."""
    rng = np.random.default_rng(5)
    X = np.tile(rng.standard_normal((1, 9)).astype(np.float32), (30, 1))
    w = rng.dirichlet(np.ones(30)).astype(np.float32)
    K = 8
    kept, order, gains = _sel(w, X, K)
    j1 = int(np.argmax(w))
    rest = [i for i in range(30) if i != j1][:K - 1]
    assert list(order) == [j1] + rest
    assert np.all(gains[1:] == 0.0)


def test_select_orthogonal_clusters_one_pick_each():
    """Exact-duplicate clusters on orthogonal axes: one pick per cluster while any is uncovered."""
    rng = np.random.default_rng(6)
    C, per = 6, 5
    X = np.repeat(np.eye(C, 8, dtype=np.float32), per, axis=0) * 2.0
    w = rng.dirichlet(np.ones(C * per)).astype(np.float32)
    _, order, _ = _sel(w, X, C)
    assert sorted(set(int(i) // per for i in order)) == list(range(C))
    # and within each cluster, the pick is that cluster's most relevant token
    for i in order:
        c = int(i) // per
        assert w[i] == w[c * per:(c + 1) * per].max()


def test_select_k_equals_one_and_n():
    rng = np.random.default_rng(7)
    X = rng.standard_normal((25, 4)).astype(np.float32)
    w = rng.dirichlet(np.ones(25)).astype(np.float32)
    kept, order, _ = _sel(w, X, 1)
    assert list(order) == [int(np.argmax(w))]
    kept, order, _ = _sel(w, X, 25)
    assert list(kept) == list(range(25)) and sorted(order) == list(range(25))


@pytest.mark.parametrize("seed", range(4))
def test_select_invariants(seed):
    wl = W.tiny(30 + seed, R=3, n_range=(30, 120), Dv=40, comps=6)
    w = np.random.default_rng(seed).dirichlet(np.ones(wl.N_total)).astype(np.float32)
    kept, order, gains = oracle.select(wl.R, wl.Dv, w, wl.feats, wl.cu_vis, wl.cu_keep, oracle.BF16)
    for r in range(wl.R):
        a, b = wl.cu_keep[r], wl.cu_keep[r + 1]
        kr, orr, gr = kept[a:b], order[a:b], gains[a:b]
        assert len(set(orr)) == wl.kk(r)
        assert np.all(np.diff(kr) > 0) and kr[0] >= 0 and kr[-1] < wl.n(r)
        assert sorted(orr) == list(kr)
        wr = w[wl.cu_vis[r]:wl.cu_vis[r + 1]]
        assert orr[0] == int(np.argmax(wr))
        assert np.all(np.diff(gr[1:]) <= 0)          # objective never grows after t = 1


def test_select_power_of_two_scaling_invariant():
    wl = W.tiny(40, R=2, n_range=(40, 80), Dv=24, comps=5, f_dtype=W.F32)
    w = np.random.default_rng(1).dirichlet(np.ones(wl.N_total)).astype(np.float32)
    _, o0, _ = oracle.select(wl.R, wl.Dv, w, wl.feats, wl.cu_vis, wl.cu_keep, oracle.F32)
    scale = (2.0 ** np.random.default_rng(2).integers(-6, 7, size=(wl.N_total, 1))).astype(np.float32)
    _, o1, _ = oracle.select(wl.R, wl.Dv, w, wl.feats * scale, wl.cu_vis, wl.cu_keep, oracle.F32)
    assert list(o0) == list(o1)


def test_topk_is_stable_sort():
    rng = np.random.default_rng(8)
    N = 300
    w = rng.integers(0, 40, size=N).astype(np.float32) / 40   # many ties
    X = rng.standard_normal((N, 3)).astype(np.float32)
    kept, order, gains = _sel(w, X, 77, mode=oracle.TOPK)
    expect = np.argsort(-w.astype(np.float64), kind="stable")[:77]
    assert list(order) == list(expect)
    assert list(kept) == sorted(expect)
    np.testing.assert_array_equal(gains, w[expect])


def _golden_float(v):
    return float(v)  # json carries "inf" / "nan" as strings; float() reads both


def test_select_clamp_golden():
    """Reading 10: a coverage term that rounds below 0 is clamped, so the tie at 0 goes to the lower index."""
    c = _load("select_clamp_replay.json")["clamp"]
    X = np.array([[float.fromhex(v) for v in row] for row in c["feats_hex"]], np.float32)
    assert X[0, 2] != X[1, 2] and np.array_equal(X[0], X[2])
    kept, order, gains = _sel(c["w"], X, c["K"])
    assert list(order) == c["order"]
    np.testing.assert_array_equal(gains, c["gains"])      # exactly 0, never negative


def test_select_gains_never_negative_on_near_parallel_rows():
    """Eq. 10 with the clamp: every objective is >= 0 even where 1 - cos rounds below 0."""
    rng = np.random.default_rng(11)
    base = rng.standard_normal((8, 3)).astype(np.float32)
    base[:, 2] *= np.float32(1e-4)
    X = np.repeat(base, 4, axis=0)
    for k in range(X.shape[0]):                      # one-ulp nudges of the small component
        X[k, 2] = np.nextafter(X[k, 2], np.float32(np.inf)) if k % 2 else X[k, 2]
    w = rng.dirichlet(np.ones(X.shape[0])).astype(np.float32)
    _, order, gains = _sel(w, X, X.shape[0])
    assert np.all(gains >= 0.0)
    assert sorted(order) == list(range(X.shape[0]))


def test_select_edge_values_golden():
    g = _load("select_edge_values.json")
    for case in g["cases"]:
        X = np.asarray(case["feats"], np.float32)
        w = np.array([_golden_float(v) for v in case["w"]], np.float32)
        _, order, gains = _sel(w, X, case["K"])
        assert list(order) == case["order"], case["name"]
        # every delta here is exactly 0 or 1, so each gain is an fp32 relevance value or 0
        expect = np.array([_golden_float(v) for v in case["gains"]], np.float32).astype(np.float64)
        np.testing.assert_array_equal(gains, expect, err_msg=case["name"])
    t = g["topk"]
    w = np.array([_golden_float(v) for v in t["w"]], np.float32)
    kept, order, gains = _sel(w, np.eye(len(w), dtype=np.float32), t["K"], mode=oracle.TOPK)
    assert list(order) == t["order"] and list(kept) == t["kept"]
    np.testing.assert_array_equal(gains, np.array(t["gains"], np.float32).astype(np.float64))


# ---------------------------------------------------------------- replay, gather, budget

def test_replay_classifies_steps():
    wl = W.tiny(50, R=2, n_range=(30, 60), Dv=16, comps=4, k_frac=0.5)
    w = np.random.default_rng(3).dirichlet(np.ones(wl.N_total)).astype(np.float32)
    _, order, _ = oracle.select(wl.R, wl.Dv, w, wl.feats, wl.cu_vis, wl.cu_keep, oracle.BF16)
    st, mg = oracle.replay(wl.R, wl.Dv, w, wl.feats, wl.cu_vis, wl.cu_keep, order, oracle.BF16)
    assert np.all(st == 0) and np.all(mg == 0)
    bad = order.copy()
    t = int(wl.cu_keep[0]) + 3
    bad[t], bad[t + 1] = bad[t + 1], bad[t]            # swap two distinct-valued picks
    st, mg = oracle.replay(wl.R, wl.Dv, w, wl.feats, wl.cu_vis, wl.cu_keep, bad, oracle.BF16)
    assert st[t] == 2 and mg[t] > 1e-6
    dup = order.copy()
    dup[t] = dup[t - 1]
    st, _ = oracle.replay(wl.R, wl.Dv, w, wl.feats, wl.cu_vis, wl.cu_keep, dup, oracle.BF16)
    assert np.all(st[t:wl.cu_keep[1]] == 2)


def test_replay_excuses_near_ties():
    X = np.eye(4, dtype=np.float32)
    w = np.array([0.5, 0.25, 0.25 * (1 - 2 ** -22), 0.0], np.float32)   # 2.4e-7 relative gap
    st, mg = oracle.replay(1, 4, w, X, [0, 4], [0, 3], np.array([0, 2, 1], np.int32), oracle.F32)
    assert list(st) == [0, 1, 0] and 0 < mg[1] < 1e-6


def test_replay_folds_the_candidates_pick_golden():
    """Eq. 10-11 under teacher forcing: after an excused pick the replay folds the candidate's pick."""
    c = _load("select_clamp_replay.json")["replay"]
    X = np.asarray(c["feats"], np.float32)
    st, mg = oracle.replay(1, X.shape[1], np.asarray(c["w"], np.float32), X, [0, X.shape[0]],
                           [0, c["K"]], np.asarray(c["picks"], np.int32), oracle.F32)
    assert list(st) == c["status"]
    np.testing.assert_array_equal(mg, c["margin"])


def test_gather_is_byte_copy():
    rng = np.random.default_rng(9)
    feats = rng.integers(0, 2 ** 16, size=(50, 7), dtype=np.uint16)   # includes NaN patterns
    cu_vis = np.array([0, 20, 50], np.int32)
    cu_keep = np.array([0, 4, 9], np.int32)
    kept = np.array([1, 5, 6, 19, 0, 3, 4, 28, 29], np.int32)
    out = oracle.gather(2, feats, cu_vis, kept, cu_keep)
    expect = np.concatenate([feats[0:20][kept[:4]], feats[20:50][kept[4:]]])
    assert out.tobytes() == expect.tobytes()


def test_budget_golden_and_exact():
    for n, num, den, k in _load("budgets.json")["cases"]:
        assert oracle.budget(n, num, den) == k
    for n in range(1, 300):
        for num, den in [(1, 8), (3, 8), (5, 8), (1, 3), (7, 9)]:
            assert oracle.budget(n, num, den) == math.ceil(Fraction(n * num, den))



# ------------------------------------------------- attention sources (Table 4)

def _orc_rows(wl, cu_rows, row_pos, q_rows, **kw):
    return oracle.rows_scores(wl.R, wl.G, wl.Hq, wl.Hkv, wl.Dh, q_rows, wl.k, wl.cu_seqlens,
                              wl.vis_start, wl.cu_vis, cu_rows, row_pos, _fcode(wl.qk_dtype),
                              scale=wl.scale, **kw)


def _random_rows(wl, rng, max_rows=4):
    """Random row sets per request: positions anywhere from the visual span's start
    to the last token, with queries drawn fresh (sharp, so the rows differ)."""
    counts, pos = [], []
    for r in range(wl.R):
        lo, hi = int(wl.vis_start[r]), wl.p(r)
        m = int(rng.integers(1, min(max_rows, hi - lo) + 1))
        pos.extend(sorted(rng.choice(np.arange(lo, hi), size=m, replace=False).tolist()))
        counts.append(m)
    cu_rows = np.concatenate([[0], np.cumsum(counts)]).astype(np.int32)
    q = rng.standard_normal((wl.G, int(cu_rows[-1]), wl.Hq, wl.Dh)).astype(np.float32)
    q = W.to_bf16_bits(q) if wl.qk_dtype == W.BF16 else q
    return cu_rows, np.asarray(pos, np.int32), q


@pytest.mark.parametrize("seed", range(8))
def test_rows_scores_match_bruteforce(seed):
    wl = W.tiny(300 + seed, R=3, G=1 + seed % 2, Hq=4, Hkv=1 + seed % 2 * 1, Dh=8 if seed % 2 else 16,
                n_range=(1, 20), t_range=(2, 12), qk_dtype=W.BF16 if seed % 3 else W.F32)
    rng = np.random.default_rng(seed)
    cu_rows, pos, q = _random_rows(wl, rng)
    w, s = _orc_rows(wl, cu_rows, pos, q, want_sums=True)
    wb, sb = brute.rows_scores(wl, cu_rows, pos, q, want_sums=True)
    np.testing.assert_allclose(w, wb, rtol=1e-10, atol=1e-15)
    np.testing.assert_allclose(s, sb, rtol=1e-10, atol=1e-15)


def test_rows_golden_causal():
    gold = _load("rows_causal.json")
    P, v0, N, Dh = gold["P"], gold["vis_start"], gold["N"], gold["Dh"]
    k = np.ones((1, P, 1, Dh), np.float32)
    wl = _make_wl(np.zeros((1, 1, 1, Dh)), k, [0, P], [v0], [0, N], 1, 1, 0.5)
    for case in gold["cases"]:
        rows = np.asarray(case["rows"], np.int32)
        q = np.random.default_rng(len(rows)).standard_normal((1, len(rows), 1, Dh)).astype(np.float32)
        w = _orc_rows(wl, [0, len(rows)], rows, q)
        exp = np.array([float(Fraction(x)) for x in case["w"]])
        np.testing.assert_allclose(w, exp, rtol=1e-13, atol=1e-15)


def test_rows_of_last_token_is_token_scores():
    for seed in range(4):
        wl = W.tiny(320 + seed, R=3, G=2, Hq=4, Hkv=2, Dh=16, n_range=(1, 30), t_range=(1, 10))
        cu_rows = np.arange(wl.R + 1, dtype=np.int32)
        pos = np.array([wl.p(r) - 1 for r in range(wl.R)], np.int32)
        np.testing.assert_allclose(_orc_rows(wl, cu_rows, pos, wl.q), _orc_scores(wl), rtol=1e-13)


def test_rows_keys_after_the_rows_are_invisible():
    wl = W.tiny(330, R=2, G=1, Hq=2, Hkv=1, Dh=16, n_range=(8, 20), t_range=(8, 12), qk_dtype=W.F32)
    rng = np.random.default_rng(3)
    # rows end before the last few tokens; keys after the last row get huge values
    counts, pos = [], []
    for r in range(wl.R):
        lo, hi = int(wl.vis_start[r]) + 2, wl.p(r) - 3
        pos.extend([lo, (lo + hi) // 2, hi])
        counts.append(3)
    cu_rows = np.concatenate([[0], np.cumsum(counts)]).astype(np.int32)
    q = rng.standard_normal((1, 6, 2, 16)).astype(np.float32)
    w0 = _orc_rows(wl, cu_rows, pos, q)
    k2 = wl.k.copy()
    for r in range(wl.R):
        a = int(wl.cu_seqlens[r])
        k2[:, a + int(pos[3 * r + 2]) + 1:int(wl.cu_seqlens[r + 1])] = 50.0
    w1 = _orc_rows(dataclasses.replace(wl, k=k2), cu_rows, pos, q)
    assert np.array_equal(w0, w1)


def test_rows_sums_add_over_row_sets():
    """Eq. 7 sums rows: the unnormalised sums of a union are the sums of the parts."""
    wl = W.tiny(340, R=3, G=2, Hq=4, Hkv=2, Dh=16, n_range=(4, 25), t_range=(4, 12))
    rng = np.random.default_rng(7)
    cu_a, pos_a, q_a = _random_rows(wl, rng, 3)
    cu_b, pos_b, q_b = _random_rows(wl, rng, 3)
    _, sa = _orc_rows(wl, cu_a, pos_a, q_a, want_sums=True)
    _, sb = _orc_rows(wl, cu_b, pos_b, q_b, want_sums=True)
    pos, qs, cnt = [], [], []
    for r in range(wl.R):
        ia = slice(int(cu_a[r]), int(cu_a[r + 1]))
        ib = slice(int(cu_b[r]), int(cu_b[r + 1]))
        pos.extend(list(pos_a[ia]) + list(pos_b[ib]))
        qs.append(np.concatenate([q_a[:, ia], q_b[:, ib]], axis=1))
        cnt.append(int(cu_a[r + 1] - cu_a[r] + cu_b[r + 1] - cu_b[r]))
    cu = np.concatenate([[0], np.cumsum(cnt)]).astype(np.int32)
    _, s = _orc_rows(wl, cu, np.asarray(pos, np.int32), np.concatenate(qs, axis=1), want_sums=True)
    np.testing.assert_allclose(s, sa + sb, rtol=1e-12)


def test_rows_reject_invisible_or_out_of_range_rows():
    wl = W.tiny(350, R=1, n_range=(5, 5), t_range=(8, 8))
    q = wl.q[:, :1]
    with pytest.raises(RuntimeError):
        _orc_rows(wl, [0, 1], [wl.p(0)], q)           # past the last token
    with pytest.raises(RuntimeError):
        _orc_rows(wl, [0, 1], [int(wl.vis_start[0]) - 1], q) if wl.vis_start[0] > 0 else \
            _orc_rows(wl, [0, 1], [-1], q)             # sees no visual token / negative


def test_source_rows_golden():
    gold = _load("source_rows.json")
    for case in gold["cases"]:
        for name, code in gold["sources"].items():
            got = oracle.source_rows(code, case["q_begin"], case["q_end"])
            assert got.tolist() == case[name], (name, case)
    with pytest.raises(ValueError):
        oracle.source_rows(0, 5, 5)



# ------------------------------------------------- prefill attention (Sec. 3.3)

def _orc_prefill(wl, pi):
    return oracle.prefill(wl.R, wl.G, wl.Hq, wl.Hkv, wl.Dh, pi.q, wl.k, pi.v, wl.cu_seqlens,
                          _fcode(wl.qk_dtype), scale=wl.scale)


@pytest.mark.parametrize("seed", range(6))
def test_prefill_matches_bruteforce(seed):
    wl = W.tiny(400 + seed, R=2 + seed % 2, G=1 + seed % 2, Hq=4, Hkv=1 + seed % 2 * 1, Dh=8 if seed % 2 else 16,
                n_range=(1, 20), t_range=(2, 12), qk_dtype=W.BF16 if seed % 3 else W.F32)
    pi = W.prefill_inputs(wl, seed)
    np.testing.assert_allclose(_orc_prefill(wl, pi), brute.prefill(wl, pi.q, pi.v), rtol=1e-10, atol=1e-13)


def test_prefill_equal_keys_give_prefix_means():
    wl = W.tiny(410, R=2, G=1, Hq=2, Hkv=1, Dh=8, n_range=(3, 9), t_range=(2, 6), qk_dtype=W.F32)
    wl = dataclasses.replace(wl, k=np.ones_like(wl.k))
    pi = W.prefill_inputs(wl)
    out = _orc_prefill(wl, pi)
    v = pi.v.astype(np.float64)
    for r in range(wl.R):
        a, b = int(wl.cu_seqlens[r]), int(wl.cu_seqlens[r + 1])
        prefix = np.cumsum(v[0, a:b, 0], axis=0) / np.arange(1, b - a + 1)[:, None]
        for h in range(wl.Hq):
            np.testing.assert_allclose(out[0, a:b, h], prefix, rtol=1e-13, atol=1e-15)
        # the first position sees only itself
        np.testing.assert_array_equal(out[0, a, 0], v[0, a, 0])


def test_prefill_last_row_weights_are_the_token_scores_rows():
    """With one-hot values the last row's output is its attention row, which the
    last-token scores see as well (Sec. 3.3 reads row p* of the same map)."""
    wl = W.tiny(420, R=2, G=1, Hq=2, Hkv=2, Dh=64, n_range=(5, 20), t_range=(3, 20), qk_dtype=W.F32)
    assert int(np.diff(wl.cu_seqlens).max()) <= wl.Dh
    pi = W.prefill_inputs(wl)
    v = np.zeros_like(pi.v)
    for r in range(wl.R):
        a, b = int(wl.cu_seqlens[r]), int(wl.cu_seqlens[r + 1])
        for j in range(b - a):
            v[0, a + j, :, j] = 1.0
    out = _orc_prefill(wl, W.PrefillInputs(q=pi.q, v=v))
    _, rows = _orc_scores(wl, want_rows=True)
    for r in range(wl.R):
        a, b = int(wl.cu_seqlens[r]), int(wl.cu_seqlens[r + 1])
        for h in range(wl.Hq):
            np.testing.assert_allclose(out[0, b - 1, h, :b - a], rows[0, h, a:b], rtol=1e-12, atol=1e-15)



# ------------------------------------- cloud connector (Sec. 3.2, 3.4 after Eq. 12)

def _orc_connector(x, cw, eps=1e-5, **kw):
    return oracle.connector(x, cw.gamma, cw.beta, cw.w1, cw.b1, cw.w2, cw.b2, _fcode(cw.dtype), eps=eps, **kw)


def _np_connector(x, cw, eps=1e-5):
    """LayerNorm, GELU (erf) and the two products in NumPy/SciPy matrix form."""
    X = W.as_f32(x, cw.dtype).astype(np.float64)
    W1 = W.as_f32(cw.w1, cw.dtype).astype(np.float64)
    W2 = W.as_f32(cw.w2, cw.dtype).astype(np.float64)
    mu = X.mean(axis=1, keepdims=True)
    var = X.var(axis=1, keepdims=True)
    xh = (X - mu) / np.sqrt(var + eps) * cw.gamma.astype(np.float64) + cw.beta.astype(np.float64)
    h = xh @ W1.T + cw.b1.astype(np.float64)
    g = 0.5 * h * (1.0 + scipy.special.erf(h / np.sqrt(2.0)))
    return g @ W2.T + cw.b2.astype(np.float64)


@pytest.mark.parametrize("dtype", [W.BF16, W.F32])
def test_connector_matches_matrix_form(dtype):
    rng = np.random.default_rng(5)
    cw = W.connector_weights(48, 80, 32, dtype, seed=1)
    x = rng.standard_normal((37, 48)).astype(np.float32)
    x = W.to_bf16_bits(x) if dtype == W.BF16 else x
    np.testing.assert_allclose(_orc_connector(x, cw), _np_connector(x, cw), rtol=1e-11, atol=1e-12)


def test_connector_identity_weights_give_gelu_of_layernorm():
    n = 16
    eye = np.eye(n, dtype=np.float32)
    cw = W.ConnectorWeights(gamma=np.ones(n, np.float32), beta=np.zeros(n, np.float32), w1=eye,
                            b1=np.zeros(n, np.float32), w2=eye, b2=np.zeros(n, np.float32), dtype=W.F32)
    # a row with mean 0 and variance 1 is its own LayerNorm (eps aside)
    base = np.array([1.0, -1.0] * (n // 2), np.float32)
    y = _orc_connector(base[None], cw, eps=0.0)
    # GELU(1) = Phi(1), GELU(-1) = -Phi(-1)
    phi1 = 0.5 * (1 + math.erf(1 / math.sqrt(2)))
    np.testing.assert_allclose(y[0], [phi1, -(1 - phi1)] * (n // 2), rtol=1e-14)
    # a constant row normalises to 0 and GELU(0) = 0
    np.testing.assert_array_equal(_orc_connector(np.full((1, n), 3.0, np.float32), cw), np.zeros((1, n)))


def test_connector_layernorm_is_shift_and_scale_invariant():
    rng = np.random.default_rng(6)
    cw = W.connector_weights(32, 24, 16, W.F32, seed=2)
    # multiples of 2^-10, so that x + 4 and 8 x are exact in fp32
    x = (np.round(rng.standard_normal((9, 32)) * 1024) / 1024).astype(np.float32)
    y = _orc_connector(x, cw, eps=0.0)
    np.testing.assert_allclose(_orc_connector(x + np.float32(4.0), cw, eps=0.0), y, rtol=1e-9, atol=1e-11)
    np.testing.assert_allclose(_orc_connector(x * np.float32(8.0), cw, eps=0.0), y, rtol=1e-12, atol=1e-14)


def test_connector_one_hot_weights_closed_form():
    """Hand-derived: x = (3, 1, -1, -3) has mean 0 and variance 5, so eps = 4
    gives rstd = 1/3; beta shifts the last feature by 1/2. One-hot rows of W1
    (not symmetric, Dh != Dv) pick features, b1 biases one hidden unit, and
    W2 (Do != Dh) picks, scales and adds hidden units; b2 shifts one output."""
    f32 = lambda a: np.asarray(a, np.float32)
    gelu = lambda u: 0.5 * u * (1 + math.erf(u / math.sqrt(2)))
    w1 = np.zeros((5, 4), np.float32)
    for j, src in enumerate([1, 3, 0, 2, 1]):
        w1[j, src] = 1.0
    w2 = f32([[0, 0, 0, 0, 2], [-1, 0, 0, 0, 0], [0, 1, 1, 0, 0]])
    cw = W.ConnectorWeights(gamma=f32([1, 1, 1, 1]), beta=f32([0, 0, 0, 0.5]), w1=w1,
                            b1=f32([0, 0, 0, 0, 0.25]), w2=w2, b2=f32([0, 0.125, 0]), dtype=W.F32)
    y, xh, h = _orc_connector(f32([[3, 1, -1, -3]]), cw, eps=4.0, want_intermediate=True)
    np.testing.assert_allclose(xh[0], [1, 1 / 3, -1 / 3, -0.5], rtol=1e-15)
    np.testing.assert_allclose(h[0], [1 / 3, -0.5, 1, -1 / 3, 7 / 12], rtol=1e-15)
    np.testing.assert_allclose(y[0], [2 * gelu(7 / 12), -gelu(1 / 3) + 0.125, gelu(1) + gelu(-0.5)], rtol=1e-14)


# ---------------------------------------------------------------- planted mistakes

MUTANTS = {
    # dropped term: the last layer is never summed (Eq. 7)
    "drop_layer": ("for (int l = 0; l < G; ++l) {\n      for (int h = 0; h < Hq; ++h) {\n        const int kv = h / g;\n        const int64_t qoff",
                   "for (int l = 0; l < G - 1 + (G == 1); ++l) {\n      for (int h = 0; h < Hq; ++h) {\n        const int kv = h / g;\n        const int64_t qoff"),
    # wrong index: query head h reads KV head h % Hkv instead of h / g
    "kv_index": ("const int kv = h / g;\n        const int64_t qoff", "const int kv = h % Hkv;\n        const int64_t qoff"),
    # softmax over the visual span only instead of the whole row (Eq. 6)
    "visual_softmax": ("for (int64_t j = 0; j < P; ++j) Z += exp(logit[j] - m);",
                       "for (int64_t j = v0; j < v0 + N; ++j) Z += exp(logit[j] - m);"),
    # wrong sign in the coverage distance (Eq. 10)
    "cover_sign": ("const double t = 1.0 - dot / sqrt(f->nn[i] * f->nn[j]);",
                   "const double t = 1.0 + dot / sqrt(f->nn[i] * f->nn[j]);"),
    # unnormalised features in Eq. 10
    "no_normalise": ("const double t = 1.0 - dot / sqrt(f->nn[i] * f->nn[j]);",
                     "const double t = 1.0 - dot;"),
    # ties broken towards the highest index
    "tie_high": ("if (best < 0 || o[i] > o[best]) best = i;", "if (best < 0 || o[i] >= o[best]) best = i;"),
    # additive instead of multiplicative objective (Eq. 11)
    "additive": ("o[i] = orc_obj(orc_rel(w[row0 + i]) * delta[i]);\n      }\n      /* Eq. 11 */",
                 "o[i] = orc_obj(orc_rel(w[row0 + i]) + delta[i]);\n      }\n      /* Eq. 11 */"),
    # coverage from the first pick only (delta not folded with later picks)
    "no_min": ("if (c < delta[i]) delta[i] = c;\n        o[i] = orc_obj(orc_rel(w[row0 + i]) * delta[i]);\n      }\n      /* Eq. 11 */",
               "if (t == 1) delta[i] = c;\n        o[i] = orc_obj(orc_rel(w[row0 + i]) * delta[i]);\n      }\n      /* Eq. 11 */"),
    # max instead of min over the selected set in Eq. 10 (coverage by the farthest pick)
    "max_not_min": ("if (c < delta[i]) delta[i] = c;\n        o[i] = orc_obj(orc_rel(w[row0 + i]) * delta[i]);\n      }\n      /* Eq. 11 */",
                    "if (delta[i] == INFINITY || c > delta[i]) delta[i] = c;\n        o[i] = orc_obj(orc_rel(w[row0 + i]) * delta[i]);\n      }\n      /* Eq. 11 */"),
    # the replay folds max instead of min as well
    "replay_max_not_min": ("if (c < delta[i]) delta[i] = c;\n        o[i] = orc_obj(orc_rel(w[row0 + i]) * delta[i]);\n      }\n    }\n    orc_free_feats",
                           "if (delta[i] == INFINITY || c > delta[i]) delta[i] = c;\n        o[i] = orc_obj(orc_rel(w[row0 + i]) * delta[i]);\n      }\n    }\n    orc_free_feats"),
    # Eq. 10's coverage term left unclamped (1 - cos may round below 0)
    "unclamped": ("return t > 0.0 ? t : 0.0;", "return t;"),
    # the replay folds the oracle's own argmax instead of the candidate's pick
    "replay_fold_best": ("const double c = orc_cover(&xf, i, gp);", "const double c = orc_cover(&xf, i, best);"),
    # a NaN objective (+inf relevance on a covered token) kept as is instead of counting as 0
    "raw_objective": ("static double orc_obj(double v) { return v == v ? v : 0.0; }",
                      "static double orc_obj(double v) { return v; }"),
    # negative relevance kept as is instead of counting as 0
    "raw_relevance": ("static double orc_rel(float w) { return (double)w > 0.0 ? (double)w : 0.0; }",
                      "static double orc_rel(float w) { return (double)w; }"),
    # zero-norm rows treated as covered (delta 0) instead of cosine 0 (delta 1)
    "zero_norm": ("if (f->nn[i] <= 0.0 || f->nn[j] <= 0.0) return 1.0;",
                  "if (f->nn[i] <= 0.0 || f->nn[j] <= 0.0) return 0.0;"),
    # kept indices left in pick order instead of ascending (Eq. 12)
    "unsorted_kept": ("if (sel[i]) kept[out0 + c++] = (int32_t)i;",
                      "if (sel[i]) { kept[out0 + c] = order[out0 + c]; ++c; }"),
    # Table 4 rows scored as if they were the last token (causal mask ignored)
    "rows_no_causal": ("const int64_t p = row_pos[m];", "const int64_t p = P - 1; (void)row_pos;"),
    # off by one in the causal softmax: the row's own key left out of Z
    "rows_off_by_one": ("for (int64_t j = 0; j <= p; ++j) Z += exp(logit[j] - mx);",
                        "for (int64_t j = 0; j < p; ++j) Z += exp(logit[j] - mx);"),
    # every row renormalised over the visual tokens it sees
    "rows_renormalise": ("for (int64_t j = 0; j <= p; ++j) Z += exp(logit[j] - mx);",
                         "for (int64_t j = v0; j <= p && j < v0 + N; ++j) Z += exp(logit[j] - mx);"),
    # prefill rows that see the whole request (no causal mask)
    "prefill_no_mask": ("const int64_t seen = p;", "const int64_t seen = P - 1; (void)p;"),
    # prefill values read from the wrong KV head
    "prefill_v_head": ("vx[j * Dh + d] = orc_widen(v, off, qk_dtype);",
                       "vx[j * Dh + d] = orc_widen(v, off + (Hkv > 1 ? Dh : 0) * (kv + 1 < Hkv ? 1 : -1), qk_dtype);"),
    # connector: GELU's tanh approximation instead of erf
    "gelu_tanh": ("g[j] = 0.5 * acc * (1.0 + erf(acc / sqrt(2.0)));",
                  "g[j] = 0.5 * acc * (1.0 + tanh(0.7978845608 * (acc + 0.044715 * acc * acc * acc)));"),
    # connector: LayerNorm without its mean
    "ln_no_mean": ("mean /= Dv;", "mean = 0.0;"),
    # connector: first bias dropped
    "no_b1": ("double acc = b1[j];", "double acc = 0.0 * b1[j];"),
    # connector: first weight matrix read transposed
    "w1_transposed": ("orc_widen(w1, (int64_t)j * Dv + d, dtype)", "orc_widen(w1, (int64_t)d * Dh + j, dtype)"),
    # connector: eps added outside the square root
    "eps_outside_sqrt": ("const double rstd = 1.0 / sqrt(var + eps);", "const double rstd = 1.0 / (sqrt(var) + eps);"),
    # Middle taken as q_(floor(M/2)+1) instead of q_ceil(M/2)
    "middle_floor": ("case 2: pos[0] = qb + (M + 1) / 2 - 1; return 1;", "case 2: pos[0] = qb + M / 2; return 1;"),
}


def _build_mutant(tmp_path, name):
    src = open(os.path.join(os.path.dirname(oracle.__file__), "oracle.c")).read()
    old, new = MUTANTS[name]
    assert src.count(old) == 1, f"mutation site for {name} not found exactly once"
    d = tmp_path / name
    d.mkdir()
    (d / "oracle.c").write_text(src.replace(old, new))
    subprocess.run(["gcc", "-O1", "-std=c11", "-fopenmp", "-fPIC", "-shared", "-o", str(d / "liboracle.so"),
                    str(d / "oracle.c"), "-lm"], check=True)
    (d / "__init__.py").write_text(open(oracle.__file__).read())
    return d


def _pins_pass():
    """Run the cheap pins against the currently bound oracle library; True if all pass."""
    checks = [test_scores_golden_two_heads, lambda: test_scores_match_bruteforce(1),
              lambda: test_scores_match_bruteforce(2), lambda: test_scores_planted_key_closed_form(3.0),
              test_select_golden_cases, lambda: test_select_matches_bruteforce(0),
              test_select_clamp_golden, test_select_edge_values_golden,
              test_replay_classifies_steps, test_replay_excuses_near_ties,
              test_replay_folds_the_candidates_pick_golden,
              lambda: test_select_matches_bruteforce(5), test_select_orthogonal_features_is_topk,
              test_select_uniform_weights_is_farthest_point, lambda: test_select_invariants(0),
              lambda: test_rows_scores_match_bruteforce(1), lambda: test_rows_scores_match_bruteforce(2),
              test_rows_golden_causal, test_source_rows_golden,
              lambda: test_prefill_matches_bruteforce(1), test_prefill_equal_keys_give_prefix_means,
              test_connector_one_hot_weights_closed_form, test_connector_identity_weights_give_gelu_of_layernorm,
              test_connector_layernorm_is_shift_and_scale_invariant]
    for c in checks:
        try:
            c()
        except AssertionError:
            return False
    return True


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_catch_planted_mistake(tmp_path, name):
    d = _build_mutant(tmp_path, name)
    saved = oracle._lib
    try:
        oracle._lib = None
        path = oracle.LIB_PATH
        oracle.LIB_PATH = str(d / "liboracle.so")
        oracle.lib()
        assert not _pins_pass(), f"planted mistake {name} went unnoticed"
    finally:
        oracle.LIB_PATH = path
        oracle._lib = saved


def test_replay_objective_is_the_free_runs_gain():
    """On the oracle's own pick sequence the replay's objective of each pick is
    the gain the free run recorded (w at t = 1, then w * delta)."""
    wl = W.tiny(52, R=2, n_range=(40, 90), Dv=24, comps=5, k_frac=0.3)
    w = np.random.default_rng(4).dirichlet(np.ones(wl.N_total)).astype(np.float32)
    _, order, gains = oracle.select(wl.R, wl.Dv, w, wl.feats, wl.cu_vis, wl.cu_keep, oracle.BF16)
    st, _, obj = oracle.replay(wl.R, wl.Dv, w, wl.feats, wl.cu_vis, wl.cu_keep, order, oracle.BF16,
                               want_objective=True)
    assert np.all(st == 0)
    np.testing.assert_array_equal(obj, gains)
