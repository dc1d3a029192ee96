"""HIP path vs the CPU oracle, on the same seeded inputs (needs an MI355X).

Bars (the oracle is fp64; the library computes in fp32 with exact bf16 widening):
  * scores   element-wise |gpu - oracle| <= 1e-5 * oracle (+ FLT_MIN floor);
  * select   every GPU pick is replayed against the oracle (teacher forcing,
             oracle.replay): it must be the oracle's own lowest-index argmax,
             or within 1e-6 relative of the oracle's best objective (an
             excused near-tie); zero failed steps. Kept sets are compared as
             sets and must match exactly unless the replay excused a step;
  * top-k    identical set and order (both sides rank the same fp32 values);
  * gather   byte-identical rows.
Small cases span several chunks/tiles with ragged tails; every request of
the five named workloads is checked in tests/test_gpu_fullsize.py.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2607_27952_amd import last
from paper_2607_27952_amd import workloads as W

pytestmark = pytest.mark.gpu

FLT_MIN = np.finfo(np.float32).tiny
SCORE_RTOL = 1e-5
TIE_RTOL = 1e-6


def _fd(dtype):
    return oracle.BF16 if dtype == W.BF16 else oracle.F32


def orc_scores(wl, want_rows=False):
    return oracle.scores(wl.R, wl.G, wl.Hq, wl.Hkv, wl.Dh, wl.q, wl.k, wl.cu_seqlens, wl.vis_start,
                         wl.cu_vis, _fd(wl.qk_dtype), scale=wl.scale, want_rows=want_rows)


def gpu_scores(dw, want_rows=False):
    out = last.token_scores(dw.batch, dw.q, dw.k, want_rows=want_rows)
    torch.cuda.synchronize()
    if want_rows:
        return out[0].cpu().numpy(), out[1].cpu().numpy()
    return out.cpu().numpy()


def assert_scores(g, o, what=""):
    g = np.asarray(g, np.float64)
    err = np.abs(g - o)
    bad = err > SCORE_RTOL * np.abs(o) + FLT_MIN
    assert not bad.any(), (f"{what}: {bad.sum()} of {bad.size} scores off; worst rel "
                           f"{np.max(err / np.maximum(np.abs(o), FLT_MIN)):.3g}")


def gpu_select(dw_feats, scores_t, cu_vis, cu_keep, mode=last.KCENTER):
    kept, order, gains = last.diverse_select(scores_t, dw_feats, cu_vis, cu_keep, mode=mode)
    torch.cuda.synchronize()
    return kept.cpu().numpy(), order.cpu().numpy(), gains.cpu().numpy()


def check_selection(wl, w32, kept, order, tag="", same_sets=None):
    """Replay the GPU pick sequence on the oracle; returns (exact, excused) step
    counts. With `same_sets` (a list), appends per request whether the kept set
    equals the oracle's own free run."""
    R = wl.R
    st, mg = oracle.replay(R, wl.Dv, w32, wl.feats, wl.cu_vis, wl.cu_keep, order, _fd(wl.f_dtype),
                           rel_tol=TIE_RTOL)
    failed = np.flatnonzero(st == 2)
    assert failed.size == 0, f"{tag}: {failed.size} failed steps, first at {failed[:5]}, margins {mg[failed[:5]]}"
    okept, _, _ = oracle.select(R, wl.Dv, w32, wl.feats, wl.cu_vis, wl.cu_keep, _fd(wl.f_dtype))
    for r in range(R):
        a, b = wl.cu_keep[r], wl.cu_keep[r + 1]
        kr = kept[a:b]
        assert np.all(np.diff(kr) > 0) and kr[0] >= 0 and kr[-1] < wl.n(r), f"{tag}: kept not ascending/in range"
        assert sorted(order[a:b]) == list(kr), f"{tag}: kept is not the sorted pick set"
        if np.all(st[a:b] == 0):
            assert list(kr) == list(okept[a:b]), f"{tag}: request {r} set differs without any near-tie"
        if same_sets is not None:
            same_sets.append(list(kr) == list(okept[a:b]))
    return int((st == 0).sum()), int((st == 1).sum())


# ------------------------------------------------------------------ scores

SCORE_CASES = [
    # seed, R, G, Hq, Hkv, Dh, qk dtype, n_range, t_range
    (0, 3, 1, 4, 4, 128, W.BF16, (1, 700), (1, 90)),
    (1, 4, 2, 8, 2, 128, W.BF16, (200, 1500), (5, 300)),
    (2, 2, 3, 14, 2, 64, W.BF16, (100, 900), (2, 40)),
    (3, 5, 1, 16, 16, 64, W.F32, (1, 600), (1, 50)),
    (4, 2, 2, 28, 4, 128, W.BF16, (1000, 3000), (20, 130)),
    (5, 3, 1, 12, 2, 128, W.BF16, (256, 2000), (32, 256)),
    (6, 2, 1, 32, 2, 128, W.F32, (50, 400), (3, 20)),         # g = 16: two head groups
    (7, 6, 2, 6, 3, 64, W.F32, (1, 5), (1, 3)),               # tiny requests, P down to 2
]


@pytest.mark.parametrize("case", SCORE_CASES, ids=lambda c: f"s{c[0]}")
def test_scores_parity_small(case):
    seed, R, G, Hq, Hkv, Dh, dt, nr, tr = case
    for sharp in (False, True):
        wl = W.tiny(seed, R=R, G=G, Hq=Hq, Hkv=Hkv, Dh=Dh, n_range=nr, t_range=tr, qk_dtype=dt, sharp=sharp)
        dw = last.DeviceWorkload.upload(wl)
        assert_scores(gpu_scores(dw), orc_scores(wl), f"case {seed} sharp={sharp}")


def test_scores_rows_debug_output():
    wl = W.tiny(11, R=3, G=2, Hq=8, Hkv=2, Dh=128, n_range=(300, 900), t_range=(10, 80))
    dw = last.DeviceWorkload.upload(wl)
    s, rows = gpu_scores(dw, want_rows=True)
    w, orows = orc_scores(wl, want_rows=True)
    assert_scores(s, w, "scores")
    for r in range(wl.R):
        a, b = wl.cu_seqlens[r], wl.cu_seqlens[r + 1]
        np.testing.assert_allclose(rows[:, :, a:b].astype(np.float64).sum(axis=2), 1.0, atol=1e-6)
    assert_scores(rows.ravel(), orows.ravel(), "rows")


@pytest.mark.parametrize("c", [-80.0, 80.0])
def test_scores_large_logit_shift(c):
    """Adding c to every logit of each row must not overflow or change w."""
    wl = W.tiny(12, R=2, G=1, Hq=4, Hkv=4, Dh=64, n_range=(200, 600), t_range=(5, 40), qk_dtype=W.F32)
    k = wl.k.astype(np.float64)
    q = wl.q.astype(np.float64)
    for r in range(wl.R):
        a, b = wl.cu_seqlens[r], wl.cu_seqlens[r + 1]
        for h in range(wl.Hq):
            u = q[0, r, h]
            k[0, a:b, h] += c * u / (wl.scale * np.dot(u, u))
    wl.k = k.astype(np.float32)
    g = gpu_scores(last.DeviceWorkload.upload(wl))
    assert np.all(np.isfinite(g))
    assert_scores(g, orc_scores(wl), f"shift {c}")


def test_scores_deterministic():
    wl = W.tiny(13, R=4, G=2, Hq=28, Hkv=4, Dh=128, n_range=(500, 2500), t_range=(10, 100))
    dw = last.DeviceWorkload.upload(wl)
    a = gpu_scores(dw)
    b = gpu_scores(dw)
    assert a.tobytes() == b.tobytes()


# ------------------------------------------------------------------ selection

SELECT_CASES = [
    # seed, R, n_range, Dv, dtype, k_frac, comps
    (20, 3, (1, 300), 64, W.BF16, None, 4),
    (21, 2, (129, 700), 256, W.BF16, 0.25, 8),
    (22, 4, (100, 400), 1024, W.BF16, 0.125, 16),
    (23, 2, (300, 640), 136, W.BF16, 0.5, 5),      # Dv not a multiple of 64
    (24, 3, (50, 500), 96, W.F32, 0.2, 6),
    (25, 1, (1500, 2100), 512, W.BF16, 0.1, 24),
    (26, 7, (1, 260), 256, W.BF16, 0.3, 3),        # four 64-column stages only; one-block requests
    (27, 2, (1025, 1100), 768, W.BF16, None, 12),  # greedy blocks of 256 threads
    (28, 1, (8193, 8300), 256, W.BF16, 0.05, 32),  # multi-block greedy (a small batch)
    (29, 5, (1, 200), 32, W.F32, 0.5, 3),          # fp32 rows shorter than one staged chunk
    (32, 1, (16385, 16600), 256, W.BF16, 0.03, 32),  # multi-block greedy, 9 slices
    (33, 2, (30000, 32767), 64, W.BF16, 0.02, 16),   # up to the 32768-token limit, staged Gram
    (34, 1, (20000, 24000), 48, W.F32, 0.02, 8),     # fp32 Gram beyond 16384 tokens
    (36, 3, (840, 896), 128, W.BF16, 0.1, 8),        # one-wave greedy, 14 tokens a lane
    (37, 2, (513, 576), 256, W.BF16, 0.15, 6),       # one-wave greedy, 9 tokens a lane
]


@pytest.mark.parametrize("case", SELECT_CASES, ids=lambda c: f"k{c[0]}")
def test_select_parity_small(case):
    seed, R, nr, Dv, dt, kf, comps = case
    wl = W.tiny(seed, R=R, n_range=nr, Dv=Dv, f_dtype=dt, k_frac=kf, comps=comps)
    rng = np.random.default_rng(seed)
    w32 = np.concatenate([rng.dirichlet(np.ones(wl.n(r)) * 0.7) for r in range(R)]).astype(np.float32)
    dw = last.DeviceWorkload.upload(wl)
    kept, order, gains = gpu_select(dw.feats, torch.from_numpy(w32).cuda(), wl.cu_vis, wl.cu_keep)
    check_selection(wl, w32, kept, order, f"case {seed}")
    # gains: w at the first pick, then the objective at each pick, never increasing
    for r in range(R):
        a, b = wl.cu_keep[r], wl.cu_keep[r + 1]
        assert gains[a] == w32[wl.cu_vis[r] + order[a]]
        assert np.all(np.diff(gains[a + 1:b]) <= 0)


def _select_handmade(X, w, K, dtype=W.F32):
    X = np.asarray(X, np.float32)
    N, Dv = X.shape
    wl = W.Workload(name="hand", R=1, G=1, Hq=1, Hkv=1, Dh=64, qk_dtype=W.F32, scale=0.125,
                    cu_seqlens=np.array([0, N + 1], np.int32), vis_start=np.array([0], np.int32),
                    cu_vis=np.array([0, N], np.int32), q=None, k=None, Dv=Dv, f_dtype=dtype,
                    feats=W.to_bf16_bits(X) if dtype == W.BF16 else X,
                    cu_keep=np.array([0, K], np.int32))
    feats = last.to_torch(wl.feats, dtype, "cuda")
    w32 = np.asarray(w, np.float32)
    kept, order, gains = gpu_select(feats, torch.from_numpy(w32).cuda(), wl.cu_vis, wl.cu_keep)
    return wl, w32, kept, order, gains


@pytest.mark.parametrize("dtype", [W.F32, W.BF16])
def test_select_edge_cases(dtype):
    rng = np.random.default_rng(30)
    Dv = 64
    # K = 1 and K = N
    X = rng.standard_normal((150, Dv))
    w = rng.dirichlet(np.ones(150))
    for K in (1, 150):
        wl, w32, kept, order, _ = _select_handmade(X, w, K, dtype)
        check_selection(wl, w32, kept, order, f"K={K}")
    # N = 1
    wl, w32, kept, order, gains = _select_handmade(X[:1], [1.0], 1, dtype)
    assert list(kept) == [0] and list(order) == [0] and gains[0] == 1.0
    # identical features: the rest are the lowest remaining indices, objective exactly 0
    Xi = np.tile(X[:1], (200, 1))
    wl, w32, kept, order, gains = _select_handmade(Xi, w[:150].tolist() + [0.001] * 50, 20, dtype)
    j1 = int(np.argmax(w32))
    assert list(order) == [j1] + [i for i in range(200) if i != j1][:19]
    assert np.all(gains[1:] == 0.0)
    # exact duplicates spread over several tiles, plus zero rows
    Xd = rng.standard_normal((300, Dv))
    Xd[150:] = Xd[:150]
    Xd[[7, 77, 277]] = 0.0
    wd = rng.dirichlet(np.ones(300))
    wl, w32, kept, order, _ = _select_handmade(Xd, wd, 200, dtype)
    check_selection(wl, w32, kept, order, "duplicates")
    # one-hot rows: top-K by weight
    Xo = np.eye(256, Dv * 4)[:, :Dv * 4]
    wl, w32, kept, order, _ = _select_handmade(Xo, rng.dirichlet(np.ones(256)), 40, dtype)
    assert list(order) == list(np.argsort(-w32.astype(np.float64), kind="stable")[:40])


@pytest.mark.parametrize("dtype", [W.F32, W.BF16])
def test_select_edge_values_golden(dtype):
    """Relevance that is not a probability (+inf, NaN, negative): the same pick
    sequence and gains as the oracle's golden cases (a non-positive relevance
    counts as 0; a NaN objective, +inf on a covered duplicate, counts as 0)."""
    import json, os
    g = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "select_edge_values.json")))
    for case in g["cases"]:
        w = np.array([float(v) for v in case["w"]], np.float32)
        X = np.asarray(case["feats"], np.float32)
        X = np.pad(X, ((0, 0), (0, 8 - X.shape[1])))   # zero columns change no norm or dot
        _, _, kept, order, gains = _select_handmade(X, w, case["K"], dtype)
        assert list(order) == case["order"], case["name"]
        assert list(kept) == sorted(case["order"]), case["name"]
        expect = np.array([float(v) for v in case["gains"]], np.float32)
        np.testing.assert_array_equal(gains, expect, err_msg=case["name"])
    t = g["topk"]
    w = np.array([float(v) for v in t["w"]], np.float32)
    X = np.eye(len(w), 8, dtype=np.float32)
    feats = last.to_torch(W.to_bf16_bits(X) if dtype == W.BF16 else X, dtype, "cuda")
    kept, order, gains = gpu_select(feats, torch.from_numpy(w).cuda(), [0, len(w)], [0, t["K"]], mode=last.TOPK)
    assert list(order) == t["order"] and list(kept) == t["kept"]
    np.testing.assert_array_equal(gains, np.array(t["gains"], np.float32))


@pytest.mark.parametrize("N,nth", [(700, "one wave"), (3000, "several waves")])
def test_select_infinite_relevance_on_duplicates(N, nth):
    """+inf relevance on clusters of exact duplicates: once every uncovered token
    is gone, the remaining objectives are 0 or NaN (+inf * 0), all counting as 0,
    so the greedy takes the lowest remaining indices, as the oracle does."""
    rng = np.random.default_rng(N)
    C = 6
    base = rng.standard_normal((C, 64)).astype(np.float32)
    X = base[rng.integers(0, C, size=N)]
    w = rng.dirichlet(np.ones(N)).astype(np.float32)
    w[rng.choice(N, 40, replace=False)] = np.inf
    K = 60
    wl, w32, kept, order, gains = _select_handmade(X, w, K, W.F32)
    okept, oorder, ogains = oracle.select(1, 64, w32, wl.feats, wl.cu_vis, wl.cu_keep, oracle.F32)
    assert list(order) == list(oorder)
    assert list(kept) == list(okept)
    np.testing.assert_array_equal(gains, ogains.astype(np.float32))


def test_select_largest_request():
    """A request of exactly 32768 tokens (the register-resident greedy's limit)."""
    rng = np.random.default_rng(35)
    N, Dv = 32768, 64
    centers = rng.standard_normal((64, Dv))
    X = centers[rng.integers(0, 64, N)] + 0.4 * rng.standard_normal((N, Dv))
    wl, w32, kept, order, _ = _select_handmade(X, rng.dirichlet(np.ones(N) * 0.5), 512, W.BF16)
    check_selection(wl, w32, kept, order, "N=32768")


# Long requests: the greedy on several compute units (slices of 2048 tokens,
# 4096 past 32768, 8192 past 65536), one candidate exchange per step.
MC_CASES = [
    # seed, R, n_range, Dv, dtype, k_frac, comps
    (50, 2, (32769, 40000), 32, W.BF16, 0.02, 16),   # 9-10 slices of 4096, ragged last slice
    (51, 1, (63000, 65536), 16, W.BF16, 0.01, 24),   # up to 16 slices of 4096
    (52, 1, (65537, 70000), 16, W.BF16, 0.01, 24),   # slices of 8192
    (53, 2, (16385, 18000), 24, W.F32, 0.05, 12),    # fp32 features, 9 slices of 2048
    (56, 3, (8193, 12000), 64, W.BF16, 0.05, 12),    # from 8193 tokens (a small batch)
]


@pytest.mark.parametrize("case", MC_CASES, ids=lambda c: f"mc{c[0]}")
def test_select_parity_multiblock(case):
    seed, R, nr, Dv, dt, kf, comps = case
    wl = W.tiny(seed, R=R, n_range=nr, Dv=Dv, f_dtype=dt, k_frac=kf, comps=comps)
    rng = np.random.default_rng(seed)
    w32 = np.concatenate([rng.dirichlet(np.ones(wl.n(r)) * 0.7) for r in range(R)]).astype(np.float32)
    dw = last.DeviceWorkload.upload(wl)
    print(f"multi-block case {seed}: N = {np.diff(wl.cu_vis).tolist()}", flush=True)
    kept, order, gains = gpu_select(dw.feats, torch.from_numpy(w32).cuda(), wl.cu_vis, wl.cu_keep)
    check_selection(wl, w32, kept, order, f"case {seed}")
    # gains against the oracle's fp64 objective of the same picks: 1e-6 relative
    # plus w * 2^-20 (the cosine's fp32 partial sums)
    obj = oracle.replay(R, wl.Dv, w32, wl.feats, wl.cu_vis, wl.cu_keep, order, _fd(wl.f_dtype),
                        rel_tol=TIE_RTOL, want_objective=True)[2]
    wpick = np.concatenate([w32[wl.cu_vis[r] + order[wl.cu_keep[r]:wl.cu_keep[r + 1]]] for r in range(R)])
    gerr = np.abs(gains.astype(np.float64) - obj)
    assert np.all(gerr <= 1e-6 * np.abs(obj) + 2.0 ** -20 * wpick.astype(np.float64)), f"gain off by {gerr.max():.3g}"


def _select_batch(Xs, ws, Ks, dtype):
    """Selection over handmade requests (feature rows Xs[r], relevance ws[r], budget Ks[r])."""
    X = np.concatenate([np.asarray(x, np.float32) for x in Xs])
    cu_vis = np.concatenate([[0], np.cumsum([len(x) for x in Xs])]).astype(np.int32)
    cu_keep = np.concatenate([[0], np.cumsum(Ks)]).astype(np.int32)
    R = len(Xs)
    wl = W.Workload(name="hand", R=R, G=1, Hq=1, Hkv=1, Dh=64, qk_dtype=W.F32, scale=0.125,
                    cu_seqlens=cu_vis + np.arange(R + 1, dtype=np.int32), vis_start=np.zeros(R, np.int32),
                    cu_vis=cu_vis, q=None, k=None, Dv=X.shape[1], f_dtype=dtype,
                    feats=W.to_bf16_bits(X) if dtype == W.BF16 else X, cu_keep=cu_keep)
    w32 = np.concatenate([np.asarray(w, np.float32) for w in ws])
    feats = last.to_torch(wl.feats, dtype, "cuda")
    kept, order, gains = gpu_select(feats, torch.from_numpy(w32).cuda(), wl.cu_vis, wl.cu_keep)
    return wl, w32, kept, order, gains


@pytest.mark.parametrize("dtype", [W.F32, W.BF16])
def test_select_mixed_batch_multiblock(dtype):
    """One request past 16384 tokens puts the whole batch on the multi-block
    greedy: a request of one token (every other slice empty), one of exactly
    one slice, one kept whole (K = N, the last picks at objective 0), one with
    a ragged last slice, and one of 40000 tokens, in one launch."""
    rng = np.random.default_rng(54)
    Dv = 32
    centres = rng.standard_normal((20, Dv))
    centres /= np.linalg.norm(centres, axis=1, keepdims=True)
    sizes, Ks = [1, 2048, 600, 17000, 40000], [1, 100, 600, 170, 400]
    Xs = [centres[rng.integers(0, 20, n)] + 0.3 / np.sqrt(Dv) * rng.standard_normal((n, Dv)) for n in sizes]
    Xs[2][100:] = Xs[2][:500]   # duplicates, so that the whole-request budget reaches objective 0
    ws = [rng.dirichlet(np.ones(n) * 0.7) for n in sizes]
    wl, w32, kept, order, gains = _select_batch(Xs, ws, Ks, dtype)
    check_selection(wl, w32, kept, order, "mixed multi-block batch")
    assert list(kept[:1]) == [0] and list(order[:1]) == [0] and gains[0] == w32[0]
    a = wl.cu_keep[2]
    assert sorted(order[a:a + 600]) == list(range(600)) and gains[a + 599] == 0.0


@pytest.mark.parametrize("n_long", [9000, 20000])
def test_select_large_batch_one_block_per_request(n_long):
    """A batch whose long request would need more blocks than the device has
    compute units once every request gets its slices: every request then runs
    on one block (512 threads up to 16384 tokens, 1024 threads beyond)."""
    rng = np.random.default_rng(n_long)
    Dv = 64
    sizes = [n_long] + [int(x) for x in rng.integers(50, 400, size=63)]
    centres = rng.standard_normal((16, Dv))
    centres /= np.linalg.norm(centres, axis=1, keepdims=True)
    Xs = [centres[rng.integers(0, 16, n)] + 0.3 / np.sqrt(Dv) * rng.standard_normal((n, Dv)) for n in sizes]
    ws = [rng.dirichlet(np.ones(n) * 0.7) for n in sizes]
    Ks = [max(1, n // 16) for n in sizes]
    wl, w32, kept, order, _ = _select_batch(Xs, ws, Ks, W.BF16)
    check_selection(wl, w32, kept, order, f"64 requests, the longest {n_long}")


def test_select_largest_request_multiblock():
    """A request of 131072 tokens, the largest diverse_select takes (16 slices
    of 8192; 69 GB of coverage distances)."""
    rng = np.random.default_rng(55)
    N, Dv = 131072, 8
    centres = rng.standard_normal((32, Dv))
    centres /= np.linalg.norm(centres, axis=1, keepdims=True)
    X = centres[rng.integers(0, 32, N)] + 0.3 / np.sqrt(Dv) * rng.standard_normal((N, Dv))
    print("N = 131072", flush=True)
    wl, w32, kept, order, _ = _select_batch([X], [rng.dirichlet(np.ones(N) * 0.5)], [256], W.BF16)
    check_selection(wl, w32, kept, order, "N=131072")
    torch.cuda.empty_cache()


def test_select_deterministic():
    wl = W.tiny(31, R=3, n_range=(400, 1200), Dv=512, k_frac=0.2, comps=12)
    w32 = np.random.default_rng(1).dirichlet(np.ones(wl.N_total)).astype(np.float32)
    dw = last.DeviceWorkload.upload(wl)
    s = torch.from_numpy(w32).cuda()
    a = gpu_select(dw.feats, s, wl.cu_vis, wl.cu_keep)
    b = gpu_select(dw.feats, s, wl.cu_vis, wl.cu_keep)
    for x, y in zip(a, b):
        assert x.tobytes() == y.tobytes()


@pytest.mark.parametrize("seed,R,nr", [(40, 4, (1, 5000)), (41, 4, (1, 5000)), (42, 2, (16385, 32768)),
                                       (43, 3, (32769, 131072)), (44, 5, (1, 40000))])
def test_topk_parity(seed, R, nr):
    wl = W.tiny(seed, R=R, n_range=nr, Dv=64, k_frac=0.125)
    rng = np.random.default_rng(seed)
    w32 = (rng.integers(0, 50, size=wl.N_total) / 50.0).astype(np.float32)   # many ties
    dw = last.DeviceWorkload.upload(wl)
    kept, order, gains = gpu_select(dw.feats, torch.from_numpy(w32).cuda(), wl.cu_vis, wl.cu_keep,
                                    mode=last.TOPK)
    ok, oo, og = oracle.select(wl.R, wl.Dv, w32, wl.feats, wl.cu_vis, wl.cu_keep, oracle.BF16, mode=oracle.TOPK)
    assert list(kept) == list(ok)
    assert list(order) == list(oo)
    np.testing.assert_array_equal(gains.astype(np.float64), og)


# ------------------------------------------------------------------ gather

@pytest.mark.parametrize("Dv,dtype", [(4096, np.uint16), (1536, np.uint16), (1024, np.float32), (77, np.uint16), (5, np.uint8)])
def test_gather_bit_exact(Dv, dtype):
    rng = np.random.default_rng(Dv)
    cu_vis = np.array([0, 300, 301, 1000], np.int32)
    cu_keep = np.array([0, 40, 41, 141], np.int32)
    itemsize = np.dtype(dtype).itemsize
    feats = rng.integers(0, 256, size=(1000, Dv * itemsize), dtype=np.uint8).view(dtype)   # NaN payloads too
    kept = np.concatenate([np.sort(rng.choice(300, 40, replace=False)), [0],
                           np.sort(rng.choice(699, 100, replace=False))]).astype(np.int32)
    ft = torch.from_numpy(feats.view(np.int16) if dtype == np.uint16 else feats).cuda()
    out = last.gather_kept(ft, cu_vis, torch.from_numpy(kept).cuda(), cu_keep)
    torch.cuda.synchronize()
    expect = oracle.gather(3, feats, cu_vis, kept, cu_keep)
    assert out.cpu().numpy().tobytes() == expect.tobytes()


def test_gather_out_of_range_index_gives_zero_row():
    feats = torch.arange(40 * 16, dtype=torch.float32).reshape(40, 16).cuda()
    out = last.gather_kept(feats, [0, 10, 40], torch.tensor([3, 10, 29, -1], dtype=torch.int32).cuda(), [0, 2, 4])
    torch.cuda.synchronize()
    o = out.cpu().numpy()
    np.testing.assert_array_equal(o[0], feats[3].cpu().numpy())
    assert np.all(o[1] == 0) and np.all(o[3] == 0)
    np.testing.assert_array_equal(o[2], feats[39].cpu().numpy())


# ------------------------------------------------------------------ full-size workloads

@pytest.fixture(scope="module")
def workloads():
    cache = {}

    def get(name, budget=None):
        key = (name, budget)
        if key not in cache:
            wl = W.make(name, budget=budget)
            cache[key] = (wl, last.DeviceWorkload.upload(wl))
        return cache[key]
    return get


def _two_phase(dw_feats, cu_vis_h, cu_keep_h, make_scores):
    """The k-center as diverse_select_similarity on a side stream, overlapped with
    `make_scores()` on the current stream, then diverse_select_pick after a join."""
    main = torch.cuda.current_stream()
    side = torch.cuda.Stream()
    ws = torch.empty(last.select_workspace(cu_vis_h, dw_feats.shape[-1], dw_feats.dtype, pair=True),
                     dtype=torch.uint8, device="cuda")
    cu_vis = torch.from_numpy(np.asarray(cu_vis_h, np.int32)).cuda()   # made on the main stream
    side.wait_stream(main)
    last.diverse_select_similarity(dw_feats, cu_vis_h, ws, cu_vis=cu_vis, stream=side)
    scores = make_scores()
    main.wait_stream(side)
    kept, order, gains = last.diverse_select_pick(scores, cu_vis_h, cu_keep_h, ws, dw_feats.shape[-1],
                                                  dw_feats.dtype, cu_vis=cu_vis)
    torch.cuda.synchronize()
    return scores, kept.cpu().numpy(), order.cpu().numpy(), gains.cpu().numpy()


@pytest.mark.parametrize("case", [c for c in SELECT_CASES if c[0] in (20, 23, 24, 27)], ids=lambda c: f"k{c[0]}")
def test_two_phase_select_small(case):
    """Split k-center (bf16 streamed and staged Gram, fp32 Gram, 256-thread greedy):
    the oracle replay accepts it, and it is bit-identical to one diverse_select call."""
    seed, R, nr, Dv, dt, kf, comps = case
    wl = W.tiny(seed, R=R, n_range=nr, Dv=Dv, f_dtype=dt, k_frac=kf, comps=comps)
    rng = np.random.default_rng(seed)
    w32 = np.concatenate([rng.dirichlet(np.ones(wl.n(r)) * 0.7) for r in range(R)]).astype(np.float32)
    dw = last.DeviceWorkload.upload(wl)
    st = torch.from_numpy(w32).cuda()
    _, kept, order, gains = _two_phase(dw.feats, wl.cu_vis, wl.cu_keep, lambda: st)
    check_selection(wl, w32, kept, order, f"two-phase case {seed}")
    one = gpu_select(dw.feats, st, wl.cu_vis, wl.cu_keep)
    for x, y in zip((kept, order, gains), one):
        assert x.tobytes() == y.tobytes()


@pytest.mark.parametrize("name", W.CONFIGS)
def test_config_two_phase_overlapped(name, workloads):
    """The bench's overlapped schedule (distances on a side stream while the scores
    run) gives bit-identical scores, kept, order and gains to the serial calls."""
    wl, dw = workloads(name)
    g, kept, order, gains = _two_phase(dw.feats, wl.cu_vis, dw.cu_keep_h,
                                       lambda: last.token_scores(dw.batch, dw.q, dw.k))
    g1 = last.token_scores(dw.batch, dw.q, dw.k)
    one = gpu_select(dw.feats, g1, wl.cu_vis, dw.cu_keep_h)
    assert g.cpu().numpy().tobytes() == g1.cpu().numpy().tobytes()
    for x, y in zip((kept, order, gains), one):
        assert x.tobytes() == y.tobytes()


def test_long_requests_x1(workloads):
    """Two requests of 32768 tokens (past the 512-thread greedy): the scores of
    both requests against the oracle; the whole selection's invariants; and
    the first 64 picks of each request replayed on the oracle (a full replay
    costs about 1 TFLOP of fp64 per request), stage-isolated and end to end."""
    wl, dw = workloads("x1_long_video")
    g = last.token_scores(dw.batch, dw.q, dw.k)
    gs = g.cpu().numpy()
    assert_scores(gs, orc_scores(wl), "x1, both requests")
    kept, order, gains = gpu_select(dw.feats, g, wl.cu_vis, dw.cu_keep_h)
    P = 64
    for r in range(wl.R):
        a, b = wl.cu_keep[r], wl.cu_keep[r + 1]
        kr = kept[a:b]
        assert b - a == 4096 and np.all(np.diff(kr) > 0) and kr[0] >= 0 and kr[-1] < wl.n(r)
        assert sorted(order[a:b]) == list(kr)
        assert np.all(np.diff(gains[a + 1:b]) <= 0)
        sub = wl.subset([r])
        w_orc = orc_scores(sub).astype(np.float32)
        _, o2, _ = gpu_select(last.to_torch(sub.feats, sub.f_dtype, "cuda"), torch.from_numpy(w_orc).cuda(),
                              sub.cu_vis, sub.cu_keep)
        cu_p = np.array([0, P], np.int32)
        for what, picks in (("oracle scores", o2[:P]), ("end to end", order[a:a + P])):
            st, mg = oracle.replay(1, wl.Dv, w_orc, sub.feats, sub.cu_vis, cu_p, np.ascontiguousarray(picks),
                                   _fd(wl.f_dtype), rel_tol=TIE_RTOL)
            assert not np.any(st == 2), f"x1 request {r} ({what}): failed steps {np.flatnonzero(st == 2)[:5]}"


@pytest.mark.parametrize("profile", [False, True])
def test_two_host_threads_two_streams(profile):
    """Two host threads, each on its own stream with its own workspaces, run the
    whole path on different batches at the same time (with kernel timing on or
    off): every result is bit-identical to the same call made alone."""
    import threading
    wls = [W.tiny(81, R=4, G=2, Hq=8, Hkv=2, Dh=128, n_range=(200, 900), t_range=(10, 60), Dv=256, k_frac=0.1),
           W.tiny(82, R=3, G=1, Hq=16, Hkv=16, Dh=64, n_range=(100, 1300), t_range=(5, 40), Dv=512, k_frac=0.2)]
    dws = [last.DeviceWorkload.upload(wl) for wl in wls]

    def run(dw, wl, stream, ws_s, ws_k):
        s = last.token_scores(dw.batch, dw.q, dw.k, ws=ws_s, stream=stream)
        kept, order, gains = last.diverse_select(s, dw.feats, wl.cu_vis, wl.cu_keep, cu_vis=dw.batch.cu_vis,
                                                 cu_keep=dw.cu_keep, ws=ws_k, stream=stream)
        out = last.gather_kept(dw.feats, wl.cu_vis, kept, wl.cu_keep, cu_vis=dw.batch.cu_vis, cu_keep=dw.cu_keep,
                               stream=stream)
        return s, kept, order, gains, out

    def host(x):
        return [t.cpu().view(torch.uint8).numpy().tobytes() if t.dtype == torch.bfloat16 else t.cpu().numpy().tobytes()
                for t in x]

    alone = []
    for dw, wl in zip(dws, wls):
        ws_s = torch.empty(last.token_scores_workspace(dw.batch, dw.q.dtype), dtype=torch.uint8, device="cuda")
        ws_k = torch.empty(last.select_workspace(wl.cu_vis, wl.Dv, dw.feats.dtype), dtype=torch.uint8, device="cuda")
        r = run(dw, wl, None, ws_s, ws_k)
        torch.cuda.synchronize()
        alone.append(host(r))

    results = [[], []]
    errors = []

    def worker(i):
        try:
            dw, wl = dws[i], wls[i]
            stream = torch.cuda.Stream()
            with torch.cuda.stream(stream):
                ws_s = torch.empty(last.token_scores_workspace(dw.batch, dw.q.dtype), dtype=torch.uint8, device="cuda")
                ws_k = torch.empty(last.select_workspace(wl.cu_vis, wl.Dv, dw.feats.dtype), dtype=torch.uint8,
                                   device="cuda")
            for _ in range(6):
                r = run(dw, wl, stream, ws_s, ws_k)
                stream.synchronize()
                results[i].append(host(r))
        except Exception as e:   # reported below, in the main thread
            errors.append(repr(e))

    last.profile_reset()
    last.profile_enable(profile)
    try:
        th = [threading.Thread(target=worker, args=(i,)) for i in range(2)]
        for t in th:
            t.start()
        for t in th:
            t.join(timeout=120)
        assert not any(t.is_alive() for t in th), "a worker thread did not finish"
    finally:
        last.profile_enable(False)
    torch.cuda.synchronize()
    assert not errors, errors
    for i in range(2):
        assert len(results[i]) == 6
        for rep in results[i]:
            assert rep == alone[i], f"thread {i}: a result differs from the call made alone"
    if profile:
        prof = last.profile_collect()
        assert prof.get("score_stream", (0, 0))[0] >= 12 and prof.get("gather", (0, 0))[0] >= 12


@pytest.mark.parametrize("sizes,div", [([700, 12000, 500, 9000, 400, 600, 300, 650], 8),
                                       ([700, 40000, 500, 9000, 400, 600, 300, 650], 32)],
                         ids=["12000", "40000"])
def test_ragged_batch_pipelined_greedy(sizes, div):
    """A ragged batch (long requests among short ones) takes the pipelined
    schedule: the off-diagonal Gram in groups of decreasing request size, each
    group's greedy on a side stream beside the later groups' Gram (with a
    40000-token request, the multi-block greedy). The result is bit-identical to
    the two-call form (the whole Gram, then every greedy) and passes the oracle
    replay."""
    rng = np.random.default_rng(91)
    R, Dv = len(sizes), 256
    cu_vis = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int32)
    cu_keep = np.concatenate([[0], np.cumsum([(n + div - 1) // div for n in sizes])]).astype(np.int32)
    # a 24-component mixture like the workloads': unit-norm centres, noise of norm 0.3
    centres = rng.standard_normal((24, Dv)).astype(np.float32)
    centres /= np.linalg.norm(centres, axis=1, keepdims=True)
    X = (centres[rng.integers(0, 24, size=int(cu_vis[-1]))] + 0.3 / np.sqrt(Dv) * rng.standard_normal(
        (int(cu_vis[-1]), Dv))).astype(np.float32)
    w32 = np.concatenate([rng.dirichlet(np.ones(n) * 0.7) for n in sizes]).astype(np.float32)
    feats_bits = W.to_bf16_bits(X)
    feats = last.to_torch(feats_bits, W.BF16, "cuda")
    st = torch.from_numpy(w32).cuda()
    last.profile_enable(True)
    last.profile_reset()
    one = gpu_select(feats, st, cu_vis, cu_keep)
    prof = last.profile_collect()
    last.profile_enable(False)
    assert prof.get("greedy_side", (0, 0))[0] >= 2, f"no pipelined greedy launches: {sorted(prof)}"
    _, kept, order, gains = _two_phase(feats, cu_vis, cu_keep, lambda: st)
    for x, y in zip(one, (kept, order, gains)):
        assert x.tobytes() == y.tobytes()
    wl = W.Workload(name="ragged", R=R, G=1, Hq=1, Hkv=1, Dh=64, qk_dtype=W.F32, scale=0.125,
                    cu_seqlens=cu_vis + np.arange(R + 1, dtype=np.int32), vis_start=np.zeros(R, np.int32),
                    cu_vis=cu_vis, q=None, k=None, Dv=Dv, f_dtype=W.BF16, feats=feats_bits, cu_keep=cu_keep)
    check_selection(wl, w32, one[0], one[1], "ragged pipelined batch")


def test_multiblock_wait_timeout_marks_request_invalid():
    """The multi-block greedy's bounded waits, forced to time out from the host
    (LAST_MC_WAIT_US=0, read by the library at every launch): every wave still
    finishes, each request's outputs are either the normal ones or marked
    invalid (-1 / NaN), and the next call with the normal limit is exact again."""
    import os
    rng = np.random.default_rng(57)
    Dv, sizes = 32, [20000, 9000, 30000]
    Xs = [rng.standard_normal((n, Dv)) for n in sizes]
    ws = [rng.dirichlet(np.ones(n)) for n in sizes]
    Ks = [n // 50 for n in sizes]
    wl, w32, kept0, order0, gains0 = _select_batch(Xs, ws, Ks, W.BF16)
    os.environ["LAST_MC_WAIT_US"] = "0"
    try:
        _, _, kept1, order1, gains1 = _select_batch(Xs, ws, Ks, W.BF16)
    finally:
        del os.environ["LAST_MC_WAIT_US"]
    n_marked = 0
    for r in range(wl.R):
        a, b = wl.cu_keep[r], wl.cu_keep[r + 1]
        same = (np.array_equal(kept1[a:b], kept0[a:b]) and np.array_equal(order1[a:b], order0[a:b])
                and np.array_equal(gains1[a:b], gains0[a:b]))
        marked = np.any(kept1[a:b] == -1) and np.any(order1[a:b] == -1) and np.any(np.isnan(gains1[a:b]))
        assert same or marked, f"request {r}: neither the normal result nor marked invalid"
        n_marked += int(marked)
    # with no wait allowed, a block that polls before its request's last block
    # has published times out: the timeout path did run
    assert n_marked >= 1
    _, _, kept2, order2, gains2 = _select_batch(Xs, ws, Ks, W.BF16)
    for x, y in zip((kept0, order0, gains0), (kept2, order2, gains2)):
        assert x.tobytes() == y.tobytes()
