"""The k-center in rounds (no N x N coverage matrix; Sec. 3.4's incremental
form) against the matrix form and the fp64 oracle (needs an MI355X).

Both forms compute every coverage distance of Eq. 10 with the same
arithmetic (the same 128-column chunks on the matrix cores, the same fp64
folding, the same operand order for each pair), and the rounds certify each
pick as the exact argmax of Eq. 11, so kept, order and gains must agree bit
for bit. The rounds' own picks are also replayed on the oracle (teacher
forcing, near-ties within 1e-6 excused, no failed step), and the kept sets
compared with the oracle's free run. LAST_KCENTER_FORM selects the form.
"""
import contextlib
import json
import os
import threading

import numpy as np
import pytest
import torch

import oracle
from paper_2607_27952_amd import last
from paper_2607_27952_amd import workloads as W

pytestmark = pytest.mark.gpu

TIE_RTOL = 1e-6


@contextlib.contextmanager
def env(**kw):
    old = {k: os.environ.get(k) for k in kw}
    os.environ.update({k: str(v) for k, v in kw.items()})
    try:
        yield
    finally:
        for k, v in old.items():
            if v is None:
                os.environ.pop(k, None)
            else:
                os.environ[k] = v


def select(form, feats, w, cu_vis, cu_keep):
    with env(LAST_KCENTER_FORM=form):
        k, o, g = last.diverse_select(w, feats, cu_vis, cu_keep)
        torch.cuda.synchronize()
    return k.cpu().numpy(), o.cpu().numpy(), g.cpu().numpy()


def both(feats, w, cu_vis, cu_keep, tag):
    """Both forms on the same inputs; asserts bit-identical outputs, returns the rounds'."""
    g = select("gram", feats, w, cu_vis, cu_keep)
    r = select("rounds", feats, w, cu_vis, cu_keep)
    for nm, a, b in zip(("kept", "order", "gains"), g, r):
        d = np.flatnonzero(a.view(np.uint32) != b.view(np.uint32))
        assert d.size == 0, f"{tag}: {nm} differs at {d[:5]}: {a[d[:5]]} vs {b[d[:5]]}"
    return r


def replay(wl, w32, kept, order, tag):
    """The rounds' picks on the oracle: no failed step; kept equals the oracle's
    free run wherever no step was excused."""
    fd = oracle.BF16 if wl.f_dtype == W.BF16 else oracle.F32
    st, mg = oracle.replay(wl.R, wl.Dv, w32, wl.feats, wl.cu_vis, wl.cu_keep, order, fd, rel_tol=TIE_RTOL)
    failed = np.flatnonzero(st == 2)
    assert failed.size == 0, f"{tag}: {failed.size} failed steps, first at {failed[:5]}, margins {mg[failed[:5]]}"
    okept, _, _ = oracle.select(wl.R, wl.Dv, w32, wl.feats, wl.cu_vis, wl.cu_keep, fd)
    for r in range(wl.R):
        a, b = wl.cu_keep[r], wl.cu_keep[r + 1]
        assert np.all(np.diff(kept[a:b]) > 0), f"{tag}: kept of request {r} not ascending"
        assert sorted(order[a:b]) == list(kept[a:b]), f"{tag}: kept of request {r} is not the pick set"
        if np.all(st[a:b] == 0):
            assert list(kept[a:b]) == list(okept[a:b]), f"{tag}: request {r} differs without a near-tie"


SMALL = [
    # seed, R, n_range, Dv, k_frac, comps
    (20, 3, (1, 300), 256, None, 4),
    (21, 2, (129, 700), 256, 0.25, 8),
    (22, 4, (100, 400), 1024, 0.125, 16),
    (25, 1, (1500, 2100), 512, 0.1, 24),
    (26, 7, (1, 260), 256, 0.3, 3),          # one-token requests, partial fold tiles
    (27, 2, (1025, 1100), 768, None, 12),
    (28, 1, (8193, 8300), 256, 0.05, 32),
    (38, 5, (300, 3000), 4096, 0.2, 6),     # the widest features the rounds take
    (39, 3, (2000, 3000), 256, 0.5, 2),     # many picks a round (few clusters)
]


@pytest.mark.parametrize("case", SMALL, ids=lambda c: f"r{c[0]}")
def test_rounds_small(case):
    seed, R, nr, Dv, kf, comps = case
    wl = W.tiny(seed, R=R, n_range=nr, Dv=Dv, f_dtype=W.BF16, k_frac=kf, comps=comps)
    rng = np.random.default_rng(seed)
    w32 = np.concatenate([rng.dirichlet(np.ones(wl.n(r)) * 0.7) for r in range(R)]).astype(np.float32)
    dw = last.DeviceWorkload.upload(wl)
    kept, order, _ = both(dw.feats, torch.from_numpy(w32).cuda(), wl.cu_vis, wl.cu_keep, f"case {seed}")
    replay(wl, w32, kept, order, f"case {seed}")


def test_rounds_many_requests():
    """2100 requests: past the 2048 whose fold-tile prefixes the rounds keep
    in LDS, so the task decode reads them from the workspace, and the prefix
    kernel takes several passes. Bit-identical to the matrix form; a few
    requests replayed on the oracle."""
    R = 2100
    wl = W.tiny(41, R=R, n_range=(1, 64), t_range=(1, 4), Hq=2, Hkv=1, Dh=64, Dv=256, f_dtype=W.BF16,
                k_frac=0.3, comps=3)
    rng = np.random.default_rng(41)
    w32 = np.concatenate([rng.dirichlet(np.ones(wl.n(r)) * 0.7) for r in range(R)]).astype(np.float32)
    dw = last.DeviceWorkload.upload(wl)
    kept, order, _ = both(dw.feats, torch.from_numpy(w32).cuda(), wl.cu_vis, wl.cu_keep, "2100 requests")
    sub = [0, 1, 1023, 2047, 2048, 2099]
    idx = np.concatenate([np.arange(wl.cu_keep[r], wl.cu_keep[r + 1]) for r in sub])
    vis = np.concatenate([np.arange(wl.cu_vis[r], wl.cu_vis[r + 1]) for r in sub])
    replay(wl.subset(sub), w32[vis], kept[idx], order[idx], "2100 requests, sampled")


def _hand(X, w, K):
    X = np.asarray(X, np.float32)
    X = np.pad(X, ((0, 0), (0, (-X.shape[1]) % 256)))   # zero columns change no norm or dot
    feats = last.to_torch(W.to_bf16_bits(X), W.BF16, "cuda")
    cv, ck = np.array([0, X.shape[0]], np.int32), np.array([0, K], np.int32)
    return both(feats, torch.from_numpy(np.asarray(w, np.float32)).cuda(), cv, ck, f"hand K={K}")


def test_rounds_edge_cases():
    rng = np.random.default_rng(30)
    X = rng.standard_normal((150, 64))
    w = rng.dirichlet(np.ones(150))
    for K in (1, 2, 150):
        _hand(X, w, K)
    kept, order, gains = _hand(X[:1], [1.0], 1)
    assert list(kept) == [0] and gains[0] == 1.0
    # identical features: one pick, then the lowest remaining indices at objective 0
    Xi = np.tile(X[:1], (400, 1))
    wi = np.concatenate([w, np.full(250, 0.001)])
    kept, order, gains = _hand(Xi, wi, 300)
    j1 = int(np.argmax(wi.astype(np.float32)))
    assert list(order) == [j1] + [i for i in range(400) if i != j1][:299]
    assert np.all(gains[1:] == 0.0)
    # duplicates across 32-row blocks and fold tiles, plus zero rows
    Xd = rng.standard_normal((700, 64))
    Xd[350:] = Xd[:350]
    Xd[[7, 77, 277, 600]] = 0.0
    _hand(Xd, rng.dirichlet(np.ones(700)), 500)
    # one-hot rows: every distance is 1, so the picks follow the relevance
    kept, order, _ = _hand(np.eye(300, 512), rng.dirichlet(np.ones(300)), 260)
    # all tokens of a request picked
    _hand(rng.standard_normal((3000, 128)), rng.dirichlet(np.ones(3000)), 3000)


def test_rounds_edge_values_golden():
    """Relevance that is not a probability (+inf, NaN, negative): the golden
    pick sequences and gains of the oracle's cases, through the rounds."""
    g = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "select_edge_values.json")))
    for case in g["cases"]:
        w = np.array([float(v) for v in case["w"]], np.float32)
        _, order, gains = _hand(np.asarray(case["feats"], np.float32), w, case["K"])
        assert list(order) == case["order"], case["name"]
        want = np.array([float(v) for v in case["gains"]], np.float32)
        assert np.array_equal(gains, want, equal_nan=True), case["name"]


@pytest.mark.parametrize("N", [700, 3000])
def test_rounds_infinite_relevance_on_duplicates(N):
    """+inf relevance on clusters of exact duplicates: after the uncovered tokens
    run out, every objective is 0 or NaN and the rest of the budget goes to the
    lowest remaining indices, in both forms; the sequence is the oracle's."""
    rng = np.random.default_rng(N)
    base = rng.standard_normal((6, 64)).astype(np.float32)
    X = base[rng.integers(0, 6, size=N)]
    w = rng.dirichlet(np.ones(N)).astype(np.float32)
    w[rng.choice(N, 40, replace=False)] = np.inf
    kept, order, gains = _hand(X, w, 60)
    Xp = np.pad(X, ((0, 0), (0, 192)))
    okept, oorder, ogains = oracle.select(1, 256, w, W.to_bf16_bits(Xp), np.array([0, N], np.int32),
                                          np.array([0, 60], np.int32), oracle.BF16)
    assert list(order) == list(oorder) and list(kept) == list(okept)
    np.testing.assert_array_equal(gains, ogains.astype(np.float32))


@pytest.mark.parametrize("name,sharp", [("c2_llava15", False), ("c3_llava_next", False), ("c4_dynres", False),
                                        ("c5_video", False), ("c5_video", True), ("x1_long_video", False)])
def test_rounds_workloads(name, sharp):
    """Every request of the paper-shaped batches (scores from the score pass):
    the rounds and the matrix pick the same tokens, bit for bit."""
    wl = W.make(name, sharp=sharp)
    dw = last.DeviceWorkload.upload(wl)
    s = last.token_scores(dw.batch, dw.q, dw.k)
    both(dw.feats, s, wl.cu_vis, wl.cu_keep, name)
    del dw, s
    torch.cuda.empty_cache()


def test_rounds_timeout_marks_requests_invalid():
    """A wait limit of 0 (forced from the host) stops the rounds at their first
    wait: each request is then either complete and exact or marked invalid
    (kept and order -1, gains NaN), and the next call on the same workspace is
    exact again."""
    wl = W.tiny(40, R=6, n_range=(500, 2500), Dv=256, f_dtype=W.BF16, k_frac=0.2, comps=8)
    rng = np.random.default_rng(40)
    w32 = np.concatenate([rng.dirichlet(np.ones(wl.n(r))) for r in range(wl.R)]).astype(np.float32)
    dw = last.DeviceWorkload.upload(wl)
    wt = torch.from_numpy(w32).cuda()
    ref = select("gram", dw.feats, wt, wl.cu_vis, wl.cu_keep)
    with env(LAST_KCENTER_FORM="rounds"):
        ws = torch.empty(last.select_workspace(wl.cu_vis, wl.Dv, dw.feats.dtype), dtype=torch.uint8, device="cuda")
    for limit, again in (("0", False), ("10000000", True)):
        with env(LAST_KCENTER_FORM="rounds", LAST_MC_WAIT_US=limit):
            k, o, g = last.diverse_select(wt, dw.feats, wl.cu_vis, wl.cu_keep, ws=ws)
            torch.cuda.synchronize()
        k, o, g = k.cpu().numpy(), o.cpu().numpy(), g.cpu().numpy()
        for r in range(wl.R):
            a, b = wl.cu_keep[r], wl.cu_keep[r + 1]
            exact = (np.array_equal(k[a:b], ref[0][a:b]) and np.array_equal(o[a:b], ref[1][a:b])
                     and np.array_equal(g[a:b].view(np.uint32), ref[2][a:b].view(np.uint32)))
            invalid = np.all(k[a:b] == -1) and np.all(o[a:b] == -1) and np.all(np.isnan(g[a:b]))
            assert exact or (invalid and not again), f"limit {limit}: request {r} neither exact nor marked invalid"


def test_rounds_two_host_threads():
    """Two rounds calls at once, on two streams from two host threads: each
    result is bit-identical to the call made alone (the task queues of the two
    grids need no co-residency)."""
    wls = [W.tiny(41, R=3, n_range=(3000, 9000), Dv=512, f_dtype=W.BF16, k_frac=0.1, comps=16),
           W.tiny(42, R=5, n_range=(1000, 6000), Dv=256, f_dtype=W.BF16, k_frac=0.15, comps=8)]
    dws = [last.DeviceWorkload.upload(wl) for wl in wls]
    ws_ = [torch.from_numpy(np.concatenate([np.random.default_rng(43 + i).dirichlet(np.ones(wl.n(r)))
                                            for r in range(wl.R)]).astype(np.float32)).cuda()
           for i, wl in enumerate(wls)]
    with env(LAST_KCENTER_FORM="rounds"):
        alone = [tuple(x.cpu().numpy().tobytes() for x in last.diverse_select(w, dw.feats, wl.cu_vis, wl.cu_keep))
                 for w, dw, wl in zip(ws_, dws, wls)]
        torch.cuda.synchronize()
        results, errors = [[], []], []

        def worker(i):
            try:
                stream = torch.cuda.Stream()
                for _ in range(4):
                    out = last.diverse_select(ws_[i], dws[i].feats, wls[i].cu_vis, wls[i].cu_keep, stream=stream)
                    stream.synchronize()
                    results[i].append(tuple(x.cpu().numpy().tobytes() for x in out))
            except Exception as e:   # reported below, in the main thread
                errors.append(repr(e))

        th = [threading.Thread(target=worker, args=(i,)) for i in range(2)]
        for t in th:
            t.start()
        for t in th:
            t.join(timeout=120)
    assert not any(t.is_alive() for t in th), "a worker thread did not finish"
    assert not errors, errors
    for i in range(2):
        assert len(results[i]) == 4 and all(x == alone[i] for x in results[i]), f"thread {i} differs"
