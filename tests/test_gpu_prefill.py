"""Prefill attention with the LAST scores from its last rows (Sec. 3.3) on the
HIP path vs the CPU oracle (needs an MI355X).

Bars:
  * scores: element-wise within 1e-5 relative of the oracle (FLT_MIN floor),
    as for last_token_scores;
  * out: the kernel rounds every probability to bf16 before the value
    product (relative error <= 2^-8 each) and rounds the output to bf16
    (<= 2^-8 relative). The matrix cores accumulate in fp32 without a
    round-to-nearest guarantee per addition; allow 2 ulps of the running
    magnitude per key (2^-22 (p + 1) max |v_jd|). So for row p and
    dimension d, with V = max_{j<=p} |v_jd|:
      |out - oracle| <= 2^-8 (V + |oracle|) + 2^-22 (p + 1) V + 1e-5 V,
    the last term for the fp32 logits and exponentials.
Small cases span several 128-position query blocks and 64-key stages with
ragged tails; the workloads run at full size, checked on sampled requests
(C4 and C5 on a prefix of one request, which its causal rows make
self-contained, and one KV group of heads).
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
U = 2.0 ** -8   # unit roundoff of bf16 (8 significant bits)


def bf16_to_f64(t):
    return t.cpu().view(torch.int16).numpy().view(np.uint16).astype(np.uint32).__lshift__(16).view(np.float32).astype(np.float64)


def assert_scores(g, o, what=""):
    g = np.asarray(g, np.float64)
    err = np.abs(g - o)
    bad = err > SCORE_RTOL * np.abs(o) + FLT_MIN
    assert not bad.any(), (f"{what}: {bad.sum()} of {bad.size} scores off; worst rel "
                           f"{np.max(err / np.maximum(np.abs(o), FLT_MIN)):.3g}")


def assert_out(wl, v_bits, got, exp, what=""):
    """The bound of the module docstring, row by row, per request and KV head."""
    v = W.as_f32(v_bits, wl.qk_dtype).astype(np.float64)
    g = wl.Hq // wl.Hkv
    for r in range(wl.R):
        a, b = int(wl.cu_seqlens[r]), int(wl.cu_seqlens[r + 1])
        vmax = np.maximum.accumulate(np.abs(v[:, a:b]), axis=1)          # [G][P][Hkv][Dh], prefix max
        vmax = np.repeat(vmax, g, axis=2)                                # per query head
        e = exp[:, a:b]
        keys = np.arange(1, b - a + 1, dtype=np.float64)[None, :, None, None]
        bound = U * (vmax + np.abs(e)) + (2.0 ** -22 * keys + 1e-5) * vmax
        err = np.abs(got[:, a:b] - e)
        bad = err > bound
        assert not bad.any(), (f"{what} request {r}: {bad.sum()} of {bad.size} outputs off; worst "
                               f"{np.max(err - bound):.3g} over the bound")


def run(wl, pi, convert=True):
    dw = last.DeviceWorkload.upload(wl)
    q = last.to_torch(pi.q, wl.qk_dtype, "cuda")
    v = last.to_torch(pi.v, wl.qk_dtype, "cuda")
    out, scores = last.prefill_attention(dw.batch, q, dw.k, v)
    torch.cuda.synchronize()
    return (bf16_to_f64(out) if convert else out), scores.cpu().numpy(), dw


def orc_scores(wl):
    return oracle.scores(wl.R, wl.G, wl.Hq, wl.Hkv, wl.Dh, wl.q, wl.k, wl.cu_seqlens, wl.vis_start,
                         wl.cu_vis, oracle.BF16, scale=wl.scale)


def orc_prefill(wl, pi):
    return oracle.prefill(wl.R, wl.G, wl.Hq, wl.Hkv, wl.Dh, pi.q, wl.k, pi.v, wl.cu_seqlens, oracle.BF16,
                          scale=wl.scale)


PREFILL_CASES = [
    # seed, R, G, Hq, Hkv, Dh, n_range, t_range
    (80, 3, 1, 4, 4, 128, (1, 300), (2, 60)),
    (81, 2, 2, 8, 2, 128, (200, 700), (5, 200)),      # several 128-query blocks, 64-key stages
    (82, 4, 1, 6, 3, 64, (1, 40), (2, 30)),           # short requests, P below one wave's 32 rows
    (83, 2, 1, 28, 4, 128, (400, 900), (30, 130)),    # g = 7
    (84, 5, 1, 2, 1, 64, (1, 3), (2, 4)),             # P down to 3
]


@pytest.mark.parametrize("case", PREFILL_CASES, ids=lambda c: f"p{c[0]}")
def test_prefill_parity_small(case):
    seed, R, G, Hq, Hkv, Dh, nr, tr = case
    for sharp in (False, True):
        wl = W.tiny(seed, R=R, G=G, Hq=Hq, Hkv=Hkv, Dh=Dh, n_range=nr, t_range=tr, qk_dtype=W.BF16, sharp=sharp)
        pi = W.prefill_inputs(wl, seed)
        out, scores, _ = run(wl, pi)
        assert_out(wl, pi.v, out, orc_prefill(wl, pi), f"case {seed} sharp={sharp}")
        assert_scores(scores, orc_scores(wl), f"case {seed} sharp={sharp} scores")


def test_prefill_scores_match_token_scores_and_deterministic():
    wl = W.tiny(85, R=3, G=2, Hq=8, Hkv=2, Dh=128, n_range=(300, 1200), t_range=(10, 100))
    pi = W.prefill_inputs(wl)
    out1, s1, dw = run(wl, pi)
    out2, s2, _ = run(wl, pi)
    assert out1.tobytes() == out2.tobytes() and s1.tobytes() == s2.tobytes()
    t = last.token_scores(dw.batch, dw.q, dw.k).cpu().numpy().astype(np.float64)
    np.testing.assert_allclose(s1, t, rtol=2e-5, atol=FLT_MIN)


def test_prefill_rejects_fp32():
    wl = W.tiny(86, R=1, qk_dtype=W.F32)
    dw = last.DeviceWorkload.upload(wl)
    pi = W.prefill_inputs(wl)
    q = last.to_torch(pi.q, wl.qk_dtype, "cuda")
    with pytest.raises(last.LastError) as e:
        last.prefill_attention(dw.batch, q, dw.k, last.to_torch(pi.v, wl.qk_dtype, "cuda"))
    assert e.value.status == last.LAST_ERR_UNSUPPORTED


# ------------------------------------------------------------------ full-size workloads

def _group(wl, pi, kv, T=None):
    """One KV group of heads (and, with T, the first T tokens of a one-request
    batch, which causal rows make self-contained) as a batch of its own."""
    g = wl.Hq // wl.Hkv
    hs = slice(kv * g, (kv + 1) * g)
    k = wl.k[:, :, kv:kv + 1]
    q = pi.q[:, :, hs]
    v = pi.v[:, :, kv:kv + 1]
    cu = wl.cu_seqlens
    if T is not None:
        k, q, v = k[:, :T], q[:, :T], v[:, :T]
        cu = np.array([0, T], np.int32)
    sub = W.Workload(name=wl.name + "-group", R=len(cu) - 1, G=wl.G, Hq=g, Hkv=1, Dh=wl.Dh,
                     qk_dtype=wl.qk_dtype, scale=wl.scale, cu_seqlens=cu, vis_start=wl.vis_start[:len(cu) - 1],
                     cu_vis=np.array([0, 1], np.int32) if T is not None else wl.cu_vis, q=None,
                     k=np.ascontiguousarray(k), Dv=wl.Dv, f_dtype=wl.f_dtype, feats=None, cu_keep=wl.cu_keep,
                     qk_std=wl.qk_std)
    return sub, W.PrefillInputs(q=np.ascontiguousarray(q), v=np.ascontiguousarray(v)), hs


FULL = {"c2_llava15": ([0, 63], None), "c3_llava_next": ([7], None), "c4_dynres": (None, 1024),
        "c5_video": ([5], 1024)}


@pytest.mark.parametrize("name", sorted(FULL))
def test_config_prefill(name):
    wl = W.make(name)
    reqs, T = FULL[name]
    if reqs is None:                      # the largest request of the ragged batch
        reqs = [int(np.argmax(np.diff(wl.cu_seqlens)))]
    pi = W.prefill_inputs(wl)
    out, scores, _ = run(wl, pi, convert=False)
    # scores of the sampled requests, from all heads and layers
    sub = wl.subset(reqs)
    got = np.concatenate([scores[wl.cu_vis[r]:wl.cu_vis[r + 1]] for r in reqs])
    assert_scores(got, orc_scores(sub), f"{name} scores {reqs}")
    # outputs of one KV group of heads, whole requests or a prefix of one
    for r in reqs[:1] if T is not None else reqs:
        a, b = int(wl.cu_seqlens[r]), int(wl.cu_seqlens[r + 1])
        one = wl.subset([r])
        pone = W.PrefillInputs(q=pi.q[:, a:b], v=pi.v[:, a:b])
        kv = wl.Hkv - 1
        grp, pg, hs = _group(one, pone, kv, T)
        n = grp.T_total
        expect = orc_prefill(grp, pg)
        got = bf16_to_f64(out[:, a:a + n, hs].contiguous())
        assert_out(grp, pg.v, got, expect, f"{name} request {r} heads {hs}")
