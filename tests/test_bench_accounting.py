"""The bench's algorithmic work figures (no GPU): the Gram's diagonal and
off-diagonal blocks together count every unordered pair of a request once,
diagonal included, and the score pass counts every key row once."""
import os
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402
from paper_2607_27952_amd import workloads as W  # noqa: E402


def test_gram_flops_cover_each_pair_once():
    for n in [1, 5, 127, 128, 129, 576, 1000, 2880]:
        d, o = bench.gram_flops(np.array([n]), 16)
        assert d + o == n * (n + 1) * 16          # N(N+1)/2 pairs x 2 flops x Dv
        if n <= 128:
            assert o == 0


def test_kernel_work_matches_shapes():
    wl = W.tiny(3, R=3, G=2, Hq=8, Hkv=2, Dh=64, n_range=(100, 300), t_range=(5, 40), Dv=256)
    work = bench.kernel_work(wl)
    elt = 2 if wl.qk_dtype == W.BF16 else 4
    assert work["score_stream"] == ("hbm", wl.G * wl.T_total * wl.Hkv * wl.Dh * elt + wl.G * wl.R * wl.Hq * wl.Dh * elt)
    n = np.diff(wl.cu_vis)
    d, o = bench.gram_flops(n, wl.Dv)
    assert d + o == float(np.sum(n * (n + 1))) * wl.Dv
    felt = 2 if wl.f_dtype == W.BF16 else 4
    assert work["gather"] == ("hbm", 2 * wl.K_total * wl.Dv * felt)


def test_gram_bound_is_the_slower_resource():
    """Each Gram launch is priced by whichever of its algorithmic bytes (the
    features it must read once; the coverage blocks it writes are this design's,
    not the method's) and its flops takes longer at the published peaks."""
    wl = W.make("c2_llava15")
    n = np.diff(wl.cu_vis)
    work = bench.gram_work(wl)
    d, o = bench.gram_flops(n, wl.Dv)
    b = wl.N_total * wl.Dv * 2
    # C2's 576-token requests: 7.6 flops a byte on the diagonal, 282 off it, both
    # under the 312 that the peaks balance at, so both launches are HBM-bound
    assert work["gram_diag"] == ("hbm", b)
    assert work["gram"] == ("hbm", b)
    assert d / b < 312 and o / b < 312
    # long requests make the off-diagonal launch a contraction bound by the matrix cores
    wl5 = W.tiny(5, R=1, n_range=(4000, 4000), Dv=2048, k_frac=0.1)
    w5 = bench.gram_work(wl5)
    assert w5["gram"] == ("mfma", bench.gram_flops(np.diff(wl5.cu_vis), 2048)[1])


def test_multi_gpu_request_exits():
    import subprocess
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True, text=True)
    assert r.returncode == 2 and "one GPU" in r.stderr


def test_rows_work_counts_causal_prefixes():
    wl = W.tiny(4, R=2, G=2, Hq=8, Hkv=2, Dh=64, n_range=(50, 80), t_range=(10, 20), Dv=64)
    elt = 2 if wl.qk_dtype == W.BF16 else 4
    # one row at the last token per request: pass 1 reads every key, pass 2 every visual key
    cu = np.arange(wl.R + 1)
    pos = np.array([wl.p(r) - 1 for r in range(wl.R)])
    w = bench.rows_work(wl, cu, pos)
    q_bytes = wl.G * wl.R * wl.Hq * wl.Dh * elt
    assert w["rows_stats_bytes"] == wl.G * wl.T_total * wl.Hkv * wl.Dh * elt + q_bytes
    assert w["rows_visual_bytes"] == wl.G * wl.N_total * wl.Hkv * wl.Dh * elt + q_bytes
    assert w["rows_stats_flops"] == 2.0 * wl.G * wl.Hq * wl.T_total * wl.Dh
    # a row at the first visual token sees that token and everything before it
    pos2 = np.array([[int(wl.vis_start[r]), wl.p(r) - 1] for r in range(wl.R)]).ravel()
    w2 = bench.rows_work(wl, np.arange(0, 2 * wl.R + 1, 2), pos2)
    assert w2["rows_visual_flops"] == 2.0 * wl.G * wl.Hq * (wl.N_total + wl.R) * wl.Dh
    assert w2["rows_stats_flops"] == 2.0 * wl.G * wl.Hq * (wl.T_total + int(np.sum(wl.vis_start + 1))) * wl.Dh
    # single-row sources: the score pass reads each request's causal prefix
    kw = bench.kernel_work(wl, pos - 3)
    assert kw["score_stream"][1] == wl.G * (wl.T_total - wl.R * 3) * wl.Hkv * wl.Dh * elt + q_bytes


def test_prefill_flops_count_causal_rows():
    wl = W.tiny(5, R=3, G=2, Hq=4, Hkv=2, Dh=64, n_range=(10, 40), t_range=(2, 9), Dv=64)
    P = np.diff(wl.cu_seqlens)
    expect = sum(4 * wl.Dh * wl.G * wl.Hq * sum(p + 1 for p in range(n)) for n in P)
    assert bench.prefill_flops(wl) == expect


def test_connector_work_counts_two_products_and_one_norm_pass():
    wl = W.tiny(4, R=2, n_range=(40, 90), t_range=(3, 9), Dv=256)
    work = bench.connector_work(wl)
    K, D = wl.K_total, wl.Dv
    assert W.connector_dims(wl) == (D, D)
    assert work["connector_gemm1"] == ("mfma", 2.0 * K * D * D)
    assert work["connector_gemm2"] == ("mfma", 2.0 * K * D * D)
    # bf16 rows read and normalised rows written, plus gamma and beta in fp32
    assert work["connector_layernorm"] == ("hbm", 2 * K * D * 2 + 2 * D * 4)


def test_prefill_bound_is_the_slower_resource():
    """C2's short MHA requests move more bytes than the matrix cores need time
    for (q, k, v and the output, 2.7 GB against 430 GFLOP); long grouped-query
    requests are bound by the products."""
    wl = W.make("c2_llava15")
    b = wl.G * wl.T_total * (2 * wl.Hq + 2 * wl.Hkv) * wl.Dh * 2
    assert bench.prefill_work(wl) == ("hbm", b)
    wl5 = W.tiny(6, R=1, Hq=8, Hkv=1, Dh=128, n_range=(6000, 6000), t_range=(10, 10))
    assert bench.prefill_work(wl5) == ("mfma", bench.prefill_flops(wl5))


def test_stage_work_follows_the_papers_costs():
    """Scores: every key row and query read once (Eq. 6-8, O(L H N)); similarity:
    features read once and 2 K N Dv flops (Sec. 3.4, one x_j^T X product per
    pick, no N x N matrix); gather: the kept rows read and written."""
    wl = W.make("c2_llava15")
    sw = bench.stage_work(wl)
    assert sw["scores"] == bench.kernel_work(wl)["score_stream"]
    assert sw["similarity_bytes"] == 64 * 576 * 4096 * 2
    assert sw["similarity_flops"] == 2.0 * 64 * 64 * 576 * 4096
    # 302 MB at 8 TB/s (37.7 us) outlasts 19.3 GFLOP at 2.5 PFLOP/s (7.7 us)
    assert sw["similarity"] == ("hbm", sw["similarity_bytes"])
    assert sw["gather"] == ("hbm", 2 * 64 * 64 * 4096 * 2)
    c1 = W.make("c1_single_fp32")
    s1 = bench.stage_work(c1)
    # fp32 features: the flops run on the fp64 vector ALUs (78.6 TFLOP/s)
    assert s1["similarity"][0] == "alu" and s1["similarity_flops"] == 2.0 * 64 * 576 * 1024


def test_similarity_summary_reports_flops_not_bytes():
    wl = W.make("c2_llava15")
    kernels = {"gram_diag": {"ms_per_step": 0.05}, "gram": {"ms_per_step": 0.15}}
    sm = bench.similarity_summary(wl, kernels)
    d, o = bench.gram_flops(np.diff(wl.cu_vis), wl.Dv)
    assert sm["gram_unique_flops"] == d + o == 64 * 576 * 577 * 4096
    assert sm["paper_flops"] == 2.0 * 64 * 64 * 576 * 4096
    assert abs(sm["tflops_on_gram_work"] - (d + o) / 0.2e-3 / 1e12) < 0.01
    assert abs(sm["gram_work_over_paper_work"] - 577 / 128) < 0.01


def test_rounds_kernels_accounting():
    """The rounds form (kernels norms and rounds): the norms read the features
    once; the rounds are priced on the paper's similarity work (2 K N Dv flops
    against the features read once), and the summary reports that form."""
    wl = W.make("c5_video")
    kw = bench.kernel_work(wl)
    sw = bench.stage_work(wl)
    assert kw["norms"] == ("hbm", wl.N_total * wl.Dv * 2)
    assert kw["rounds"] == sw["similarity"]
    assert sw["similarity_flops"] == 2.0 * 8 * 1024 * 16384 * 3584
    kernels = {"norms": {"ms_per_step": 0.2}, "rounds": {"ms_per_step": 6.2}}
    sm = bench.similarity_summary(wl, kernels)
    assert sm["form"] == "rounds" and abs(sm["rounds_ms_per_step"] - 6.4) < 1e-9
    assert abs(sm["tflops_on_paper_work"] - sw["similarity_flops"] / 6.4e-3 / 1e12) < 0.01
    assert bench.kcenter_form(kernels) == "rounds"
    assert bench.kcenter_form({"gram": {}}) == "matrix" and bench.kcenter_form({"topk": {}}) is None
