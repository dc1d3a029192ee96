"""Attention sources of Table 4 on the HIP path vs the CPU oracle (needs an MI355X).

last_rows_scores takes any set of causal query rows per request: one row per
request (Last, First, Middle) runs the streamed single-row kernels, several
rows (All Mean) the two matrix-core passes. Scores must match the fp64
oracle element-wise within 1e-5 relative (FLT_MIN floor), as for the
last-token path. Small cases span several row groups (more than 128 query
rows per KV head), several key chunks (more than 1024 keys) and ragged
tails; the five named workloads run at full size with every source and are
checked on sampled requests.
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
SOURCES = {"last": oracle.SRC_LAST, "first": oracle.SRC_FIRST, "middle": oracle.SRC_MIDDLE,
           "all_mean": oracle.SRC_ALL_MEAN}


def _fd(dtype):
    return oracle.BF16 if dtype == W.BF16 else oracle.F32


def assert_scores(g, o, what=""):
    g = np.asarray(g, np.float64)
    err = np.abs(g - o)
    bad = err > SCORE_RTOL * np.abs(o) + FLT_MIN
    assert not bad.any(), (f"{what}: {bad.sum()} of {bad.size} scores off; worst rel "
                           f"{np.max(err / np.maximum(np.abs(o), FLT_MIN)):.3g}")


def orc_rows(wl, cu_rows, row_pos, q):
    return oracle.rows_scores(wl.R, wl.G, wl.Hq, wl.Hkv, wl.Dh, q, wl.k, wl.cu_seqlens, wl.vis_start,
                              wl.cu_vis, cu_rows, row_pos, _fd(wl.qk_dtype), scale=wl.scale)


def gpu_rows(wl, dw, cu_rows, row_pos, q):
    rows = last.Rows.make(cu_rows, row_pos)
    qt = last.to_torch(q, wl.qk_dtype, "cuda")
    out = last.rows_scores(dw.batch, rows, qt, dw.k)
    torch.cuda.synchronize()
    return out.cpu().numpy()


def source_set(qr, src, lib_side):
    """Row positions and queries of source `src` for every request; the library's
    helper picks them on the GPU side, the oracle's on the oracle side."""
    pick = last.source_rows if lib_side else oracle.source_rows
    counts, pos, qs = [], [], []
    for r in range(len(qr.q_begin)):
        p = pick(src, int(qr.q_begin[r]), int(qr.q_end[r]))
        counts.append(len(p))
        pos.extend(p.tolist())
        qs.append(qr.rows(r)[:, p - int(qr.q_begin[r])])
    cu = np.concatenate([[0], np.cumsum(counts)]).astype(np.int32)
    return cu, np.asarray(pos, np.int32), np.ascontiguousarray(np.concatenate(qs, axis=1))


def random_rows(wl, rng, lo_frac=0.0, max_rows=300):
    """Random row sets: positions between the visual span's start and the last token."""
    counts, pos = [], []
    for r in range(wl.R):
        lo = int(wl.vis_start[r]) + int(lo_frac * wl.n(r))
        hi = wl.p(r)
        m = int(rng.integers(1, min(max_rows, hi - lo) + 1))
        pos.extend(sorted(rng.choice(np.arange(lo, hi), size=m, replace=False).tolist()))
        counts.append(m)
    cu = np.concatenate([[0], np.cumsum(counts)]).astype(np.int32)
    q = rng.standard_normal((wl.G, int(cu[-1]), wl.Hq, wl.Dh)).astype(np.float32)
    q *= np.float32(wl.qk_std if wl.qk_std > 0 else 1.0 / np.sqrt(wl.Dh))
    q = W.to_bf16_bits(q) if wl.qk_dtype == W.BF16 else q
    return cu, np.asarray(pos, np.int32), q


ROW_CASES = [
    # seed, R, G, Hq, Hkv, Dh, qk dtype, n_range, t_range, max_rows, lo_frac
    (60, 3, 1, 4, 4, 128, W.BF16, (1, 700), (2, 90), 40, 0.0),
    (61, 2, 2, 8, 2, 128, W.BF16, (1100, 2500), (5, 300), 70, 0.0),      # several key / visual chunks
    (62, 2, 1, 28, 4, 128, W.BF16, (300, 900), (60, 130), 120, 0.5),     # 7 x 120 rows: several row groups
    (63, 4, 1, 16, 16, 64, W.F32, (1, 600), (2, 50), 12, 0.0),
    (64, 3, 2, 12, 2, 64, W.BF16, (200, 1500), (10, 256), 200, 0.3),
    (65, 2, 1, 6, 3, 128, W.F32, (1030, 1100), (3, 40), 30, 0.9),        # rows inside the visual span
    (66, 5, 1, 4, 2, 64, W.BF16, (1, 5), (2, 4), 8, 0.0),                # tiny requests
]


@pytest.mark.parametrize("case", ROW_CASES, ids=lambda c: f"r{c[0]}")
def test_rows_parity_small(case):
    seed, R, G, Hq, Hkv, Dh, dt, nr, tr, mx, lo = case
    for sharp in (False, True):
        wl = W.tiny(seed, R=R, G=G, Hq=Hq, Hkv=Hkv, Dh=Dh, n_range=nr, t_range=tr, qk_dtype=dt, sharp=sharp)
        rng = np.random.default_rng(seed)
        cu, pos, q = random_rows(wl, rng, lo, mx)
        dw = last.DeviceWorkload.upload(wl)
        g = gpu_rows(wl, dw, cu, pos, q)
        assert_scores(g, orc_rows(wl, cu, pos, q), f"case {seed} sharp={sharp}")
        for r in range(wl.R):
            seg = g[wl.cu_vis[r]:wl.cu_vis[r + 1]].astype(np.float64)
            assert np.all(seg >= 0) and abs(seg.sum() - 1.0) < 1e-5


@pytest.mark.parametrize("src", sorted(SOURCES))
def test_sources_small(src):
    wl = W.tiny(70, R=4, G=2, Hq=8, Hkv=2, Dh=128, n_range=(100, 1500), t_range=(8, 200))
    qr = W.query_rows(wl)
    cu_g, pos_g, q_g = source_set(qr, SOURCES[src], lib_side=True)
    cu_o, pos_o, q_o = source_set(qr, SOURCES[src], lib_side=False)
    dw = last.DeviceWorkload.upload(wl)
    assert_scores(gpu_rows(wl, dw, cu_g, pos_g, q_g), orc_rows(wl, cu_o, pos_o, q_o), src)


def test_last_source_equals_token_scores():
    wl = W.tiny(71, R=3, G=2, Hq=28, Hkv=4, Dh=128, n_range=(500, 2500), t_range=(10, 100))
    qr = W.query_rows(wl)
    cu, pos, q = source_set(qr, oracle.SRC_LAST, lib_side=True)
    dw = last.DeviceWorkload.upload(wl)
    a = gpu_rows(wl, dw, cu, pos, q)
    b = last.token_scores(dw.batch, dw.q, dw.k).cpu().numpy()
    assert a.tobytes() == b.tobytes()


def test_rows_deterministic():
    wl = W.tiny(72, R=3, G=1, Hq=12, Hkv=2, Dh=128, n_range=(900, 2000), t_range=(30, 200))
    cu, pos, q = random_rows(wl, np.random.default_rng(2), 0.0, 150)
    dw = last.DeviceWorkload.upload(wl)
    assert gpu_rows(wl, dw, cu, pos, q).tobytes() == gpu_rows(wl, dw, cu, pos, q).tobytes()


def test_rows_rejects_invisible_rows():
    wl = W.tiny(73, R=2, n_range=(20, 30), t_range=(8, 12))
    dw = last.DeviceWorkload.upload(wl)
    q = last.to_torch(wl.q, wl.qk_dtype, "cuda")
    bad = last.Rows.make([0, 1, 2], [int(wl.vis_start[0]) - 1 if wl.vis_start[0] > 0 else -1, wl.p(1) - 1])
    with pytest.raises(last.LastError) as e:
        last.rows_scores(dw.batch, bad, q, dw.k)
    assert e.value.status == last.LAST_ERR_INVALID


# ------------------------------------------------------------------ full-size workloads

SAMPLES = {"c1_single_fp32": [0], "c2_llava15": [0, 63], "c3_llava_next": [9],
           "c4_dynres": None, "c5_video": [2]}


@pytest.fixture(scope="module")
def full():
    cache = {}

    def get(name):
        if name not in cache:
            wl = W.make(name)
            cache[name] = (wl, last.DeviceWorkload.upload(wl), W.query_rows(wl))
        return cache[name]
    return get


@pytest.mark.parametrize("src", sorted(SOURCES))
@pytest.mark.parametrize("name", W.CONFIGS)
def test_config_sources(name, src, full):
    wl, dw, qr = full(name)
    cu, pos, q = source_set(qr, SOURCES[src], lib_side=True)
    g = gpu_rows(wl, dw, cu, pos, q)
    for r in range(wl.R):
        seg = g[wl.cu_vis[r]:wl.cu_vis[r + 1]].astype(np.float64)
        assert np.all(seg >= 0) and abs(seg.sum() - 1.0) < 1e-5, f"{name} {src} request {r}"
    samples = SAMPLES[name]
    if samples is None:
        order = np.argsort(np.diff(wl.cu_vis))
        samples = [int(order[0]), int(order[len(order) // 2])]
    sub = wl.subset(samples)
    cu_o, pos_o, q_o = source_set(qr.subset(samples), SOURCES[src], lib_side=False)
    w = orc_rows(sub, cu_o, pos_o, q_o)
    got = np.concatenate([g[wl.cu_vis[r]:wl.cu_vis[r + 1]] for r in samples])
    assert_scores(got, w, f"{name} {src} requests {samples}")
