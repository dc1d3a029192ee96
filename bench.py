"""Benchmark of the LAST token-selection path on one MI355X.

A step is one pass of the whole path over one batch that is already resident
in HBM: last_token_scores -> diverse_select (k-center) -> gather_kept. With
--source first|middle|all_mean the scores come from those query rows instead
(last_rows_scores, the attention sources of the paper's Table 4).

Default workload: the LLaVA-1.5-shaped batch (64 requests of 576 visual +
64 text tokens, 2 guidance layers of 32 heads, head_dim 128, bf16; budget
B = 64 of 576; 576 x 4096 encoder features per request).

Prints ONE JSON line on stdout. Per-kernel times come from HIP events that
the library records on the launch stream around each kernel during the timed
steps. The CPU oracle is timed on this host on a bounded sample of the same
workload (cpu_baseline). Other lines go to stderr.
"""
import argparse
import hashlib
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0        # MI355X HBM3E
MFMA_BF16_PEAK_TFLOPS = 2500.0
FP64_VECTOR_PEAK_TFLOPS = 78.6   # fp32 features: the Gram runs fp64 FMAs on the vector ALUs
PROFILES = os.path.join(ROOT, "profiles")


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="c2_llava15")
    ap.add_argument("--budget", type=int, default=None)
    ap.add_argument("--source", default="last", choices=("last", "first", "middle", "all_mean"),
                    help="attention rows the scores come from (Table 4)")
    ap.add_argument("--prefill", action="store_true",
                    help="take the scores from the guidance model's causal prefill attention of every "
                         "position (last_prefill_attention) instead of recomputing the last row")
    ap.add_argument("--connector", action="store_true",
                    help="apply the cloud connector (last_connector: LayerNorm, Linear, GELU, Linear, "
                         "Dv -> Dv -> Dv, seeded weights) to the gathered rows in every step")
    ap.add_argument("--overlap", action="store_true",
                    help="run the k-center's distances (diverse_select_similarity) on a second stream "
                         "beside the score pass, then diverse_select_pick; by default every call runs "
                         "in order on one stream")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-configs", action="store_true",
                    help="time only the chosen workload (by default the other paper-shaped batches and the "
                         "LLaVA-1.5 batch's other budgets are timed too and reported under \"configs\")")
    ap.add_argument("--cpu-seconds", type=float, default=12.0,
                    help="target CPU time for the oracle sample")
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="before warmup, run one plain device copy of this many MiB, so that a "
                         "counter run sees a kernel of known traffic beside the path's kernels")
    return ap.parse_args()


def describe(wl, budget):
    n = np.diff(wl.cu_vis)
    t = np.diff(wl.cu_seqlens) - n
    ks = np.diff(wl.cu_keep)
    return (f"{wl.name}: {wl.R} requests x ({int(n.mean()) if n.min() == n.max() else 'ragged'} visual + "
            f"{int(t.mean()) if t.min() == t.max() else 'ragged'} text tokens), {wl.G} guidance layers, "
            f"{wl.Hq}/{wl.Hkv} heads, head_dim {wl.Dh}, {wl.qk_dtype}; features {wl.Dv}-d {wl.f_dtype}; "
            f"budget {int(ks[0]) if ks.min() == ks.max() else 'ceil(N/8)'}")


GRAM_TILE = 128   # rows per side of one Gram tile block


def gram_flops(n, dv):
    """Unique multiply-adds (x2) of each request's symmetric Gram, split into the
    diagonal tile blocks (upper triangle with the diagonal) and the off-diagonal
    tile blocks (full rectangles above the diagonal)."""
    diag = off = 0.0
    for nr in n:
        sizes = [min(GRAM_TILE, nr - s) for s in range(0, nr, GRAM_TILE)]
        diag += sum(m * (m + 1) / 2 for m in sizes) * 2 * dv
        tot = nr * (nr + 1) / 2 * 2 * dv
        off += tot - sum(m * (m + 1) / 2 for m in sizes) * 2 * dv
    return diag, off


HBM_BYTES_PER_S = HBM_PEAK_GBS * 1e9
MFMA_FLOPS_PER_S = MFMA_BF16_PEAK_TFLOPS * 1e12


def rows_work(wl, cu_rows, row_pos):
    """Algorithmic work of the attention-source passes. Pass 1 reads every key up
    to the last row of its request once and forms one logit per (row, head, key
    the row sees); pass 2 reads the visual keys the rows see and forms their
    logits again. A pass is bound by whichever of HBM bytes and MFMA flops takes
    longer at the peaks."""
    elt = 2 if wl.qk_dtype == "bf16" else 4
    keys1 = keys2 = logits1 = logits2 = 0
    for r in range(wl.R):
        pos = np.asarray(row_pos[int(cu_rows[r]):int(cu_rows[r + 1])], np.int64)
        v0, n = int(wl.vis_start[r]), wl.n(r)
        keys1 += int(pos.max()) + 1
        keys2 += min(n, int(pos.max()) - v0 + 1)
        logits1 += int(np.sum(pos + 1))
        logits2 += int(np.sum(np.clip(pos - v0 + 1, 0, n)))
    q_bytes = wl.G * int(cu_rows[-1]) * wl.Hq * wl.Dh * elt
    b1 = wl.G * keys1 * wl.Hkv * wl.Dh * elt + q_bytes
    b2 = wl.G * keys2 * wl.Hkv * wl.Dh * elt + q_bytes
    f1 = 2.0 * wl.G * wl.Hq * logits1 * wl.Dh
    f2 = 2.0 * wl.G * wl.Hq * logits2 * wl.Dh

    def bound(b, f):
        return ("hbm", b) if b / HBM_BYTES_PER_S >= f / MFMA_FLOPS_PER_S else ("mfma", f)
    return {"rows_stats": bound(b1, f1), "rows_visual": bound(b2, f2),
            "rows_stats_bytes": b1, "rows_stats_flops": f1, "rows_visual_bytes": b2, "rows_visual_flops": f2}


def gram_work(wl):
    """The two Gram launches, each bound by whichever of its algorithmic bytes and
    matrix-core (bf16) or fp64-vector (fp32 features) flops takes longer at the
    peaks. Algorithmic bytes are the features the launch must read once: every
    row for the diagonal launch, the rows of every request with more than one
    row block for the off-diagonal one. The coverage blocks both launches write
    are a product of this design (the paper's method keeps no N x N matrix), so
    they count as measured traffic, not as algorithmic work. Flops are the
    launch's share of each request's symmetric Gram."""
    felt = 2 if wl.f_dtype == "bf16" else 4
    n = np.diff(wl.cu_vis).astype(np.int64)
    nb = (n + GRAM_TILE - 1) // GRAM_TILE
    f_diag, f_off = gram_flops(n, wl.Dv)
    b_diag = wl.N_total * wl.Dv * felt
    b_off = int(np.sum(n[nb > 1])) * wl.Dv * felt
    peak, kind = (MFMA_FLOPS_PER_S, "mfma") if felt == 2 else (FP64_VECTOR_PEAK_TFLOPS * 1e12, "alu")

    def bound(b, f):
        return ("hbm", b) if b / HBM_BYTES_PER_S >= f / peak else (kind, f)
    if felt == 4:
        # fp32 features: one launch covers every sub-tile (its blocks compute their own norms)
        return {"gram": bound(b_diag, f_diag + f_off)}
    return {"gram_diag": bound(b_diag, f_diag), "gram": bound(b_off, f_off)}


def prefill_flops(wl):
    """Causal attention of every position: row p takes p + 1 keys, 2 Dh flops
    each for the logits and 2 Dh for the value product."""
    P = np.diff(wl.cu_seqlens).astype(np.float64)
    return 4.0 * wl.Dh * wl.G * wl.Hq * float(np.sum(P * (P + 1) / 2))


def prefill_work(wl):
    """The prefill attention, bound by whichever of its flops and its bytes (q,
    k, v read once, the output written once) takes longer at the peaks."""
    elt = 2
    b = wl.G * wl.T_total * (2 * wl.Hq + 2 * wl.Hkv) * wl.Dh * elt
    f = prefill_flops(wl)
    return ("hbm", b) if b / HBM_BYTES_PER_S >= f / MFMA_FLOPS_PER_S else ("mfma", f)


def connector_work(wl):
    """The cloud connector on the K_total kept rows: LayerNorm reads and writes
    K Dv bf16 values; the two products take 2 K Dv Dh and 2 K Dh Do flops."""
    Dh, Do = wl.Dv, wl.Dv
    K = wl.K_total
    return {"connector_layernorm": ("hbm", 4 * K * wl.Dv + 8 * wl.Dv),
            "connector_gemm1": ("mfma", 2.0 * K * wl.Dv * Dh),
            "connector_gemm2": ("mfma", 2.0 * K * Dh * Do)}


def kernel_work(wl, row_pos=None):
    """Algorithmic bytes / flops per launch of each kernel, and its bound.
    row_pos: one scored row per request (a single-row attention source), whose
    causal prefix is what the score pass reads; None for the last token."""
    elt = 2 if wl.qk_dtype == "bf16" else 4
    felt = 2 if wl.f_dtype == "bf16" else 4
    n = np.diff(wl.cu_vis).astype(np.int64)
    kk = np.diff(wl.cu_keep).astype(np.int64)
    tokens = wl.T_total if row_pos is None else int(np.sum(np.asarray(row_pos, np.int64) + 1))
    k_bytes = wl.G * tokens * wl.Hkv * wl.Dh * elt
    q_bytes = wl.G * wl.R * wl.Hq * wl.Dh * elt
    vlog = wl.G * wl.Hq * wl.N_total * 4
    gw = gram_work(wl)
    return {
        # key rows of every guidance layer + the last-token queries, each read once
        "score_stream": ("hbm", k_bytes + q_bytes),
        "score_partial": ("hbm", k_bytes + q_bytes),
        # visual logits in, scores out
        "score_finalize": ("hbm", vlog + wl.N_total * 4),
        # features read once
        "sqnorm": ("hbm", wl.N_total * wl.Dv * felt),
        **gw,
        # the k-center in rounds (no N x N matrix): the norms read the features
        # once; the rounds do the paper's own similarity work, one x_j^T X per
        # pick (2 K N Dv flops), against the features read once
        "norms": ("hbm", wl.N_total * wl.Dv * felt),
        "rounds": stage_work(wl, row_pos)["similarity"],
        # one coverage row of N_r floats per pick, plus the weights
        "greedy": ("hbm", float(np.sum(kk * n)) * 4 + wl.N_total * 4),
        "topk": ("hbm", wl.N_total * 4 + wl.K_total * 4),
        # kept rows read and written
        "gather": ("hbm", 2 * wl.K_total * wl.Dv * felt),
        "prefill": prefill_work(wl) if wl.qk_dtype == "bf16" else ("mfma", prefill_flops(wl)),
    }


def stage_work(wl, row_pos=None):
    """Algorithmic work of each stage of the path, as the paper defines the stage:
    - scores (Eq. 6-8, O(L H N)): every key row of every guidance layer and the
      scored query rows read once (HBM);
    - similarity (Sec. 3.4, O(K N d_v), no N x N matrix): the features read once,
      and one x_j^T X product per pick, 2 K N Dv flops; bound by whichever takes
      longer at the peaks (matrix cores for bf16 features, the fp64 vector ALUs
      that the fp32-feature path runs on);
    - gather (Eq. 12): the kept rows read and written once (HBM)."""
    elt = 2 if wl.qk_dtype == "bf16" else 4
    felt = 2 if wl.f_dtype == "bf16" else 4
    tokens = wl.T_total if row_pos is None else int(np.sum(np.asarray(row_pos, np.int64) + 1))
    score_bytes = wl.G * tokens * wl.Hkv * wl.Dh * elt + wl.G * wl.R * wl.Hq * wl.Dh * elt
    kk = np.diff(wl.cu_keep).astype(np.float64)
    nv = np.diff(wl.cu_vis).astype(np.float64)
    sim_flops = float(np.sum(2 * kk * nv)) * wl.Dv
    sim_bytes = wl.N_total * wl.Dv * felt
    peak, kind = (MFMA_FLOPS_PER_S, "mfma") if felt == 2 else (FP64_VECTOR_PEAK_TFLOPS * 1e12, "alu")
    sim = ("hbm", sim_bytes) if sim_bytes / HBM_BYTES_PER_S >= sim_flops / peak else (kind, sim_flops)
    return {"scores": ("hbm", score_bytes), "similarity": sim,
            "gather": ("hbm", 2 * wl.K_total * wl.Dv * felt),
            "similarity_bytes": sim_bytes, "similarity_flops": sim_flops}


SCORE_KERNELS = ("score_prefix", "score_stream", "score_partial", "score_merge", "score_finalize")
SIMILARITY_KERNELS = ("select_plan", "gram_diag", "gram", "norms", "rounds")


def similarity_summary(wl, kernels):
    """The k-center's distance stage against the paper's work and, for the
    matrix form, against the Gram's own executed work (each request's symmetric
    Gram, diagonal included). The rounds form (no matrix; kernels norms and
    rounds, which also run the greedy) is reported against the paper's work."""
    sw = stage_work(wl)
    rounds_ms = sum(kernels[k]["ms_per_step"] for k in ("norms", "rounds") if k in kernels)
    if "rounds" in kernels and rounds_ms > 0:
        return {"form": "rounds", "paper_flops": sw["similarity_flops"],
                "rounds_ms_per_step": round(rounds_ms, 4),
                "tflops_on_paper_work": round(sw["similarity_flops"] / (rounds_ms * 1e-3) / 1e12, 2)}
    gram_ms = sum(kernels[k]["ms_per_step"] for k in ("gram_diag", "gram") if k in kernels)
    if gram_ms <= 0:
        return None
    d, o = gram_flops(np.diff(wl.cu_vis), wl.Dv)
    unique = d + o
    return {"form": "matrix", "paper_flops": sw["similarity_flops"], "gram_unique_flops": unique,
            "gram_ms_per_step": round(gram_ms, 4),
            "tflops_on_paper_work": round(sw["similarity_flops"] / (gram_ms * 1e-3) / 1e12, 2),
            "tflops_on_gram_work": round(unique / (gram_ms * 1e-3) / 1e12, 2),
            "gram_work_over_paper_work": round(unique / sw["similarity_flops"], 2)}


def cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def roofline_entry(name, bound, work, avg_ms):
    if bound == "hbm":
        ach = work / (avg_ms * 1e-3) / 1e9
        return {"kernel": name, "bound": "hbm", "achieved": round(ach, 1), "peak": HBM_PEAK_GBS,
                "unit": "GB/s", "frac": round(ach / HBM_PEAK_GBS, 4), "bytes_per_launch": int(work)}
    ach = work / (avg_ms * 1e-3) / 1e12
    peak = MFMA_BF16_PEAK_TFLOPS if bound == "mfma" else FP64_VECTOR_PEAK_TFLOPS
    return {"kernel": name, "bound": bound, "achieved": round(ach, 2), "peak": peak,
            "unit": "TFLOP/s", "frac": round(ach / peak, 4), "flops_per_launch": int(work)}


def traffic_for(kernel, workload):
    """HBM bytes per launch measured by rocprofv3 counters, if a summary for this
    kernel and workload exists and the kernel source is unchanged since."""
    path = os.path.join(PROFILES, f"{kernel}_{workload}_traffic.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f)
    src = os.path.join(ROOT, rec["source"])
    if not os.path.exists(src):
        return None
    if hashlib.sha256(open(src, "rb").read()).hexdigest() != rec["source_sha256"]:
        return None
    return rec.get("bytes_per_launch")


def cpu_baseline(wl, target_s):
    import oracle
    fd = oracle.BF16 if wl.f_dtype == "bf16" else oracle.F32
    qd = oracle.BF16 if wl.qk_dtype == "bf16" else oracle.F32
    threads = len(os.sched_getaffinity(0))

    def run(sub, nth=threads):
        t0 = time.perf_counter()
        w = oracle.scores(sub.R, sub.G, sub.Hq, sub.Hkv, sub.Dh, sub.q, sub.k, sub.cu_seqlens,
                          sub.vis_start, sub.cu_vis, qd, scale=sub.scale, nthreads=nth)
        kept, _, _ = oracle.select(sub.R, sub.Dv, w.astype(np.float32), sub.feats, sub.cu_vis,
                                   sub.cu_keep, fd, nthreads=nth)
        oracle.gather(sub.R, sub.feats, sub.cu_vis, kept, sub.cu_keep)
        return time.perf_counter() - t0

    t_one = run(wl.subset([0]))
    n = int(min(wl.R, max(1, math.ceil(target_s / max(t_one, 1e-6)))))
    sub = wl if n == wl.R else wl.subset(list(range(n)))
    passes, dt = 0, 0.0
    while dt < target_s and passes < 100:      # the whole batch is repeated when it is quick
        dt += run(sub)
        passes += 1
    what = f"all {wl.R} requests" if n == wl.R else f"first {n} of {wl.R} requests"
    # the same path on one thread, over requests taken in order for about a quarter of the time
    n1, dt1 = 0, 0.0
    while dt1 < target_s / 4 and n1 < wl.R:
        dt1 += run(wl.subset([n1]), 1)
        n1 += 1
    return {"value": round(n * passes / dt, 3), "unit": "requests/s", "cores": threads, "kind": "oracle",
            "cpu_model": cpu_model(),
            "sample": f"{what} x {passes} pass(es), whole path (scores, k-center, gather) in fp64, "
                      f"{dt:.1f} s on {threads} threads",
            "single_thread": {"value": round(n1 / dt1, 3), "unit": "requests/s",
                              "sample": f"first {n1} request(s) one at a time, {dt1:.1f} s on 1 thread"}}


def measure(args, name, budget, steps, warmup, source="last", prefill=False, connector=False, overlap=False,
            copy_mib=0):
    """Time `steps` steps of the path on one workload (after `warmup` steps) and
    return the per-workload record: throughput, p50/p90 step latency, per-kernel
    times (HIP events the library records around each kernel, in a second timed
    pass), per-kernel and per-stage rooflines, and the workload object."""
    import torch
    from paper_2607_27952_amd import last
    from paper_2607_27952_amd import workloads as W

    dev = torch.device("cuda:0")
    t0 = time.time()
    wl = W.make(name, budget=budget)
    log(f"[bench] generated {wl.name} (budget {budget}) in {time.time() - t0:.1f}s")
    dw = last.DeviceWorkload.upload(wl, device=dev)
    b = dw.batch
    stream = torch.cuda.current_stream()

    # every buffer allocated once, outside the timed region
    scores = torch.empty(wl.N_total, dtype=torch.float32, device=dev)
    kept = torch.empty(wl.K_total, dtype=torch.int32, device=dev)
    order = torch.empty(wl.K_total, dtype=torch.int32, device=dev)
    gains = torch.empty(wl.K_total, dtype=torch.float32, device=dev)
    out = torch.empty((wl.K_total, wl.Dv), dtype=dw.feats.dtype, device=dev)
    rows = q_rows = None
    pre = None
    if prefill:
        if source != "last":
            raise SystemExit("--prefill takes the scores from the last rows; --source must be last")
        pin = W.prefill_inputs(wl)
        pre = (last.to_torch(pin.q, wl.qk_dtype, dev), last.to_torch(pin.v, wl.qk_dtype, dev))
        pre_out = torch.empty(pre[0].shape, dtype=pre[0].dtype, device=dev)
        del pin
        log(f"[bench] scores from the causal prefill attention of all {wl.T_total} positions")
    if source != "last":
        qr = W.query_rows(wl)
        src = {"first": last.SRC_FIRST, "middle": last.SRC_MIDDLE, "all_mean": last.SRC_ALL_MEAN}[source]
        counts, pos, qs = [], [], []
        for r in range(wl.R):
            p = last.source_rows(src, int(qr.q_begin[r]), int(qr.q_end[r]))
            counts.append(len(p))
            pos.extend(p.tolist())
            qs.append(qr.rows(r)[:, p - int(qr.q_begin[r])])
        rows = last.Rows.make(np.concatenate([[0], np.cumsum(counts)]), pos, device=dev)
        q_rows = last.to_torch(np.ascontiguousarray(np.concatenate(qs, axis=1)), wl.qk_dtype, dev)
        ws_s = torch.empty(last.rows_scores_workspace(b, rows, dw.q.dtype), dtype=torch.uint8, device=dev)
        log(f"[bench] scores from the {source} rows: {int(rows.cu_rows_h[-1])} query rows")
    elif pre is not None:
        ws_s = torch.empty(last.prefill_attention_workspace(b), dtype=torch.uint8, device=dev)
    else:
        ws_s = torch.empty(last.token_scores_workspace(b, dw.q.dtype), dtype=torch.uint8, device=dev)
    ws_k = torch.empty(last.select_workspace(wl.cu_vis, wl.Dv, dw.feats.dtype, pair=overlap), dtype=torch.uint8,
                       device=dev)

    conn = None
    if connector:
        if wl.f_dtype != "bf16":
            raise SystemExit("--connector runs on bf16 features")
        Dh, Do = W.connector_dims(wl)
        cw = W.connector_weights(wl.Dv, Dh, Do, W.BF16)
        f32 = lambda a: torch.from_numpy(np.ascontiguousarray(a, np.float32)).to(dev)
        conn = dict(gamma=f32(cw.gamma), beta=f32(cw.beta), w1=last.to_torch(cw.w1, W.BF16, dev), b1=f32(cw.b1),
                    w2=last.to_torch(cw.w2, W.BF16, dev), b2=f32(cw.b2))
        conn_out = torch.empty((wl.K_total, Do), dtype=torch.bfloat16, device=dev)
        ws_c = torch.empty(max(256, last.connector_workspace(wl.K_total, wl.Dv, Dh)), dtype=torch.uint8, device=dev)
        del cw
        log(f"[bench] cloud connector {wl.Dv} -> {Dh} -> {Do} on the {wl.K_total} kept rows")

    if copy_mib > 0:
        nbytes = copy_mib << 20
        src_t = torch.ones(nbytes // 4, dtype=torch.int32, device=dev)
        dst_t = torch.empty_like(src_t)
        torch.cuda.synchronize()
        dst_t.copy_(src_t)
        torch.cuda.synchronize()
        log(f"[bench] calibration copy: {nbytes} bytes read, {nbytes} bytes written")
        del src_t, dst_t

    # The distances of Eq. 10 need only the features: on a second stream (default
    # priority) they overlap the score pass; the pick waits for both streams.
    side = torch.cuda.Stream(device=dev)

    def step(marks=None):
        # marks: events recorded on the stream around each call (the score call,
        # the selection, the gather, the connector)
        mark = (lambda i: marks[i].record(stream)) if marks is not None else (lambda i: None)
        if overlap:
            side.wait_stream(stream)
            last.diverse_select_similarity(dw.feats, wl.cu_vis, ws_k, cu_vis=b.cu_vis, stream=side)
        mark(0)
        if pre is not None:
            last.prefill_attention(b, pre[0], dw.k, pre[1], out=pre_out, scores=scores, ws=ws_s)
        elif rows is None:
            last.token_scores(b, dw.q, dw.k, scores=scores, ws=ws_s)
        else:
            last.rows_scores(b, rows, q_rows, dw.k, scores=scores, ws=ws_s)
        mark(1)
        if overlap:
            stream.wait_stream(side)
            last.diverse_select_pick(scores, wl.cu_vis, dw.cu_keep_h, ws_k, wl.Dv, dw.feats.dtype, cu_vis=b.cu_vis,
                                     cu_keep=dw.cu_keep, kept=kept, order=order, gains=gains)
        else:
            last.diverse_select(scores, dw.feats, wl.cu_vis, dw.cu_keep_h, cu_vis=b.cu_vis, cu_keep=dw.cu_keep,
                                kept=kept, order=order, gains=gains, ws=ws_k)
        mark(2)
        last.gather_kept(dw.feats, wl.cu_vis, kept, dw.cu_keep_h, cu_vis=b.cu_vis, cu_keep=dw.cu_keep, out=out)
        mark(3)
        if conn is not None:
            last.connector(out, conn["gamma"], conn["beta"], conn["w1"], conn["b1"], conn["w2"], conn["b2"],
                           out=conn_out, ws=ws_c)
        mark(4)

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()

    def timed(profile):
        """`steps` steps bracketed by synchronisation; per-step HIP events on the launch stream.
        With `profile`, the library also records events around each of its kernels."""
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(steps)]
        last.profile_reset()
        last.profile_enable(profile)
        torch.cuda.synchronize()
        t_a = time.perf_counter()
        for i in range(steps):
            ev[i][0].record(stream)
            step()
            ev[i][1].record(stream)
        torch.cuda.synchronize()
        t_b = time.perf_counter()
        last.profile_enable(False)
        prof = last.profile_collect() if profile else {}
        return t_b - t_a, np.array([x.elapsed_time(y) for x, y in ev]), prof

    def timed_calls():
        """`steps` steps with events between the calls: each call's time on the
        stream, inter-kernel gaps included (what a caller of that call waits)."""
        ev = [[torch.cuda.Event(enable_timing=True) for _ in range(5)] for _ in range(steps)]
        torch.cuda.synchronize()
        for i in range(steps):
            step(ev[i])
        torch.cuda.synchronize()
        t = np.array([[ev[i][j].elapsed_time(ev[i][j + 1]) for j in range(4)] for i in range(steps)])
        return t.mean(axis=0)

    # throughput: the path alone; per-kernel times: a second timed pass with the
    # library's kernel events (they add a little time between kernels); per-call
    # times: a third pass with events between the calls only
    elapsed, step_ms, _ = timed(False)
    elapsed_prof, _, prof = timed(True)
    call_ms = timed_calls()

    single = rows is not None and int(rows.cu_rows_h[-1]) == wl.R
    row_pos = rows.row_pos_h if single else None
    work = kernel_work(wl, row_pos)
    if rows is not None and not single:
        work.update({k: v for k, v in rows_work(wl, rows.cu_rows_h, rows.row_pos_h).items()
                     if k in ("rows_stats", "rows_visual")})
    if conn is not None:
        work.update(connector_work(wl))
    kernels = {}
    for kname, (launches, total_ms) in prof.items():
        if launches == 0:   # timed in an earlier workload of this process, not in this one
            continue
        kernels[kname] = {"launches": launches, "avg_ms": round(total_ms / max(launches, 1), 5),
                          "ms_per_step": round(total_ms / steps, 5)}
    # work figures are per step; a kernel launched several times a step (the Gram
    # of a ragged batch, in groups) does its share per launch
    rooflines = [roofline_entry(k, bd, w / max(1.0, kernels[k]["launches"] / steps), kernels[k]["avg_ms"])
                 for k, (bd, w) in work.items() if k in kernels and kernels[k]["avg_ms"] > 0]
    # greedies launched on the library's side streams overlap the Gram; they are
    # reported but neither counted in the stage sums nor taken as the dominant kernel
    dominant = max((kv for kv in kernels.items() if kv[0] != "greedy_side"), key=lambda kv: kv[1]["ms_per_step"])[0]
    main_roof = next((r for r in rooflines if r["kernel"] == dominant), None)
    if main_roof is not None:
        tr = traffic_for(dominant, name if source == "last" and pre is None else
                         f"{name}_{'prefill' if pre is not None else source}")
        main_roof = {k: main_roof[k] for k in ("bound", "achieved", "peak", "unit", "frac")} | {
            "traffic": tr, "kernel": dominant}

    score_ms = sum(kernels[k]["ms_per_step"] for k in kernels
                   if k.startswith("score") or k.startswith("rows") or k.startswith("prefill"))
    similarity_ms = sum(kernels[k]["ms_per_step"] for k in SIMILARITY_KERNELS if k in kernels)
    select_ms = similarity_ms + sum(kernels[k]["ms_per_step"] for k in ("greedy", "topk") if k in kernels)
    gather_ms = kernels.get("gather", {}).get("ms_per_step", 0.0)
    if "greedy_side" in kernels:
        # the overlapped greedies end after the Gram: the select stage is what the
        # step leaves after the score and gather kernels
        select_ms = max(select_ms, elapsed_prof / steps * 1e3 - score_ms - gather_ms)
    conn_ms = sum(kernels[k]["ms_per_step"] for k in kernels if k.startswith("connector"))
    sw = stage_work(wl, row_pos)
    stage_roof = {}
    calls = {"scores": float(call_ms[0]), "select": float(call_ms[1]), "gather": float(call_ms[2])}
    if conn is not None:
        calls["connector"] = float(call_ms[3])
    if rows is None and pre is None and score_ms > 0:
        # the whole last_token_scores call, as a caller waits for it (events
        # between the calls; its kernels and the gaps between them)
        stage_roof["scores"] = roofline_entry("scores: the last_token_scores call (" +
                                              "+".join(k for k in kernels if k in SCORE_KERNELS) + ")",
                                              *sw["scores"], calls["scores"])
        stage_roof["scores_kernels"] = roofline_entry("scores: sum of the score kernels' own event times",
                                                      *sw["scores"], score_ms)
    if similarity_ms > 0:
        e = roofline_entry("similarity: " + "+".join(k for k in SIMILARITY_KERNELS if k in kernels),
                           *sw["similarity"], similarity_ms)
        e["paper_work"] = "features read once; 2 K N Dv flops (one x_j^T X product per pick)"
        stage_roof["similarity"] = e
    if gather_ms > 0:
        stage_roof["gather"] = roofline_entry("gather", *sw["gather"], gather_ms)
    if "greedy" in kernels and "greedy_side" not in kernels:
        kk = np.diff(wl.cu_keep)
        stage_roof["greedy"] = {"bound": "latency", "steps_longest_request": int(kk.max()),
                                "us_per_step_longest_request": round(kernels["greedy"]["ms_per_step"] * 1e3 / int(kk.max()), 3)}
    ms_per_step = elapsed / steps * 1e3
    return {
        "wl": wl,
        "value": round(wl.R * steps / elapsed, 2),
        "ms_per_step": round(ms_per_step, 4),
        "visual_tokens_scored_per_s": round(wl.N_total / (score_ms * 1e-3), 1) if score_ms > 0 else None,
        "p50_select_latency_ms": round(float(np.median(step_ms)), 4),
        "p90_select_latency_ms": round(float(np.percentile(step_ms, 90)), 4),
        "ms_per_step_with_kernel_events": round(elapsed_prof / steps * 1e3, 4),
        "stage_ms_per_step": {"scores": round(score_ms, 4), "select": round(select_ms, 4),
                              "gather": round(gather_ms, 4)} | ({"connector": round(conn_ms, 4)} if conn else {}),
        "call_ms_per_step": {k: round(v, 4) for k, v in calls.items()},
        "kernels": kernels,
        "roofline": main_roof,
        "rooflines": rooflines,
        "stage_rooflines": stage_roof,
        "similarity": similarity_summary(wl, kernels),
        "rows": rows,
        "pre": pre,
        "conn": conn,
    }


# The other workloads timed beside the headline one (each of the paper-shaped
# batches, and the LLaVA-1.5 batch at its other two budgets): name, budget, steps.
CONFIG_RUNS = (("c1_single_fp32", None, 50), ("c2_llava15", 128, 30), ("c2_llava15", 192, 30),
               ("c3_llava_next", None, 20), ("c4_dynres", None, 10), ("c5_video", None, 10))


def kcenter_form(kernels):
    """Which form of the k-center ran: the rounds (no N x N matrix) or the matrix."""
    return "rounds" if "rounds" in kernels else "matrix" if "gram" in kernels or "gram_diag" in kernels else None


def config_summary(m, budget):
    wl = m["wl"]
    ks = np.diff(wl.cu_keep)
    return {"workload": describe(wl, budget), "requests": wl.R, "visual_tokens": wl.N_total,
            "kept_tokens": wl.K_total, "budget": int(ks[0]) if ks.min() == ks.max() else "ceil(N/8)",
            "requests_per_s": m["value"], "ms_per_step": m["ms_per_step"],
            "visual_tokens_scored_per_s": m["visual_tokens_scored_per_s"],
            "p50_select_latency_ms": m["p50_select_latency_ms"], "stage_ms_per_step": m["stage_ms_per_step"],
            "call_ms_per_step": m["call_ms_per_step"],
            "kernels_ms_per_step": {k: v["ms_per_step"] for k, v in m["kernels"].items()},
            "kcenter_form": kcenter_form(m["kernels"]),
            "roofline": m["roofline"], "stage_rooflines": m["stage_rooflines"], "similarity": m["similarity"]}


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (this build has no multi-GPU path); got --gpus {args.gpus}",
              file=sys.stderr)
        sys.exit(2)
    import torch

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    m = measure(args, args.workload, args.budget, args.steps, args.warmup, source=args.source,
                prefill=args.prefill, connector=args.connector, overlap=args.overlap,
                copy_mib=args.copy_calibration_mib)
    wl = m["wl"]
    res = {
        "metric": "requests/sec and visual tokens scored/sec per GPU; p50 select latency",
        "value": m["value"],
        "unit": "requests/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": m["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": describe(wl, args.budget) + ("" if args.source == "last" else
                                                             f"; scores from the {args.source} query rows")
                   + ("; scores from the causal prefill attention of every position" if m["pre"] is not None else "")
                   + (f"; cloud connector {wl.Dv}->{wl.Dv}->{wl.Dv} on the kept rows" if m["conn"] is not None else ""),
                   "schedule": ("one stream" if not args.overlap else
                                "distances (plan, Gram) on a second stream beside the score pass; "
                                "greedy and gather after both"),
                   "requests": wl.R, "visual_tokens": wl.N_total,
                   "kept_tokens": wl.K_total, "arithmetic": (
                       "bf16 inputs, " + ("fp32 FMA score pass" if args.source != "all_mean" else
                                          "bf16 MFMA score passes with fp32 accumulation")
                       + ", bf16 MFMA coverage dot products with fp32 partial sums folded into fp64"
                       + ", fp32 objective"),
                   "kcenter_form": kcenter_form(m["kernels"])},
        "visual_tokens_scored_per_s": m["visual_tokens_scored_per_s"],
        "p50_select_latency_ms": m["p50_select_latency_ms"],
        "p90_select_latency_ms": m["p90_select_latency_ms"],
        "ms_per_step_with_kernel_events": m["ms_per_step_with_kernel_events"],
        "stage_ms_per_step": m["stage_ms_per_step"],
        "call_ms_per_step": m["call_ms_per_step"],
        "kernels": m["kernels"],
        "roofline": m["roofline"],
        "rooflines": m["rooflines"],
        "stage_rooflines": m["stage_rooflines"],
        "similarity": m["similarity"],
        "configs": None,
        "cpu_baseline": None,
        "device": torch.cuda.get_device_name(0),
    }
    default_mode = not (args.prefill or args.connector or args.overlap or args.source != "last")
    if default_mode and not args.no_configs:
        res["configs"] = {}
        del m
        for name, budget, steps in CONFIG_RUNS:
            if name == args.workload and budget == args.budget:
                continue
            torch.cuda.empty_cache()
            t0 = time.time()
            mc = measure(args, name, budget, steps, 3)
            res["configs"][name if budget is None else f"{name}_b{budget}"] = config_summary(mc, budget)
            log(f"[bench] {name} (budget {budget}): {mc['ms_per_step']} ms per step, {time.time() - t0:.1f}s")
            del mc
    if not args.no_cpu_baseline:
        t0 = time.time()
        from paper_2607_27952_amd import workloads as W
        res["cpu_baseline"] = cpu_baseline(W.make(args.workload, budget=args.budget), args.cpu_seconds)
        log(f"[bench] cpu baseline took {time.time() - t0:.1f}s")
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
