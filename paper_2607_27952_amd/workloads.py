"""Seeded synthetic inputs for the LAST token-selection path.

This module only *draws* inputs: shapes, CSR offsets, query/key tensors,
encoder features and budgets. It contains none of the method's arithmetic
(no attention, no softmax, no selection); both the HIP library's tests and
the CPU oracle consume what it produces.

Five named workloads mirror the shapes of the paper's settings:

  c1_single_fp32  one request, fp32, 1 guidance layer, 16 heads (MHA),
                  head_dim 64, 576 visual + 40 text tokens, B=64, 8-cluster
                  features of width 1024, 5 planted relevant tokens.
  c2_llava15      64 requests shaped like LLaVA-1.5 (24x24 = 576 visual
                  tokens, 64 text), 32 heads MHA, head_dim 128, bf16, scores
                  from 2 guidance layers, B in {64,128,192}, 32-cluster
                  features of width 4096, 2% planted relevant tokens.
  c3_llava_next   32 requests of 5 crops x 576 = 2880 visual + 96 text
                  tokens, 32/8 heads (GQA), bf16, B=320, 64-cluster
                  features of width 4096, 30% near-duplicates per crop.
  c4_dynres       128 ragged requests, visual count log-uniform in
                  [256, 16384], 32-256 text tokens, 12/2 heads, bf16,
                  B = ceil(N/8), 128-cluster features of width 1536.
  c5_video        8 requests of 64 frames x 256 = 16384 visual + 128 text
                  tokens, 28/4 heads, 4 guidance layers, B=1024, width-3584
                  features with frame-to-frame redundancy and scene cuts
                  every 16 frames.

One more, beyond the paper's settings, measures requests past 16384 tokens:

  x1_long_video   2 requests of 128 frames x 256 = 32768 visual + 128 text
                  tokens, otherwise shaped like c5_video; B=4096 (12.5%).

Conventions (shared with the C-ABI):
  q     [G][R][Hq][Dh]         the last query token of each request
  k     [G][T_total][Hkv][Dh]  keys of every prefill token, CSR by cu_seqlens
  feats [N_total][Dv]          encoder features of the visual tokens, CSR by cu_vis
  bf16 arrays are numpy uint16 bit patterns (round-to-nearest-even from fp32).
  Each request's visual span starts at floor(T_r / 4) (a system-prompt-like
  prefix), the rest of the text follows, and the last token is text.
"""
from __future__ import annotations

import concurrent.futures
import dataclasses
import hashlib
import math
import os
from typing import Dict, List, Optional

import numpy as np

F32 = "f32"
BF16 = "bf16"

CONFIGS = ("c1_single_fp32", "c2_llava15", "c3_llava_next", "c4_dynres", "c5_video")
EXTRA = ("x1_long_video",)
_CONFIG_IDS = {name: i for i, name in enumerate(CONFIGS + EXTRA)}


def to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """fp32 -> bf16 bit patterns, round to nearest, ties to even (finite inputs)."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    r = (u >> 16) & 1
    r += 0x7FFF
    r += u
    r >>= 16
    return r.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """bf16 bit patterns -> fp32 values (exact)."""
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def as_f32(x: np.ndarray, dtype: str) -> np.ndarray:
    return bf16_bits_to_f32(x) if dtype == BF16 else np.asarray(x, dtype=np.float32)


def _store(x: np.ndarray, dtype: str) -> np.ndarray:
    return to_bf16_bits(x) if dtype == BF16 else np.ascontiguousarray(x, dtype=np.float32)


@dataclasses.dataclass
class Workload:
    name: str
    R: int
    G: int
    Hq: int
    Hkv: int
    Dh: int
    qk_dtype: str
    scale: float
    cu_seqlens: np.ndarray
    vis_start: np.ndarray
    cu_vis: np.ndarray
    q: np.ndarray
    k: np.ndarray
    Dv: int
    f_dtype: str
    feats: np.ndarray
    cu_keep: np.ndarray
    planted: Optional[List[np.ndarray]] = None
    notes: str = ""
    qk_std: float = 0.0          # element std of q and k as drawn (0: 1/sqrt(Dh))

    @property
    def T_total(self) -> int:
        return int(self.cu_seqlens[-1])

    @property
    def N_total(self) -> int:
        return int(self.cu_vis[-1])

    @property
    def K_total(self) -> int:
        return int(self.cu_keep[-1])

    def n(self, r: int) -> int:
        return int(self.cu_vis[r + 1] - self.cu_vis[r])

    def p(self, r: int) -> int:
        return int(self.cu_seqlens[r + 1] - self.cu_seqlens[r])

    def kk(self, r: int) -> int:
        return int(self.cu_keep[r + 1] - self.cu_keep[r])

    def with_budgets(self, budgets) -> "Workload":
        """Same inputs with new per-request budgets (an int, or one per request)."""
        b = np.broadcast_to(np.asarray(budgets, dtype=np.int64), (self.R,))
        cu_keep = np.zeros(self.R + 1, np.int32)
        cu_keep[1:] = np.cumsum(b)
        return dataclasses.replace(self, cu_keep=cu_keep)

    def subset(self, reqs) -> "Workload":
        """A batch made of the listed requests, with every CSR offset re-based."""
        reqs = [int(r) for r in reqs]
        ks, qs, fs, P, N, K, vs = [], [], [], [], [], [], []
        for r in reqs:
            a, b = int(self.cu_seqlens[r]), int(self.cu_seqlens[r + 1])
            ks.append(self.k[:, a:b])
            qs.append(self.q[:, r:r + 1])
            fs.append(self.feats[int(self.cu_vis[r]):int(self.cu_vis[r + 1])])
            P.append(b - a)
            N.append(self.n(r))
            K.append(self.kk(r))
            vs.append(int(self.vis_start[r]))

        def cu(v):
            out = np.zeros(len(v) + 1, np.int32)
            out[1:] = np.cumsum(v)
            return out

        return dataclasses.replace(
            self, name=f"{self.name}[{','.join(map(str, reqs))}]", R=len(reqs),
            cu_seqlens=cu(P), vis_start=np.asarray(vs, np.int32), cu_vis=cu(N),
            q=np.ascontiguousarray(np.concatenate(qs, axis=1)),
            k=np.ascontiguousarray(np.concatenate(ks, axis=1)),
            feats=np.ascontiguousarray(np.concatenate(fs, axis=0)), cu_keep=cu(K),
            planted=None)

    def manifest(self) -> Dict[str, object]:
        def h(a):
            return hashlib.sha256(np.ascontiguousarray(a).tobytes()).hexdigest()
        return {
            "name": self.name, "R": self.R, "G": self.G, "Hq": self.Hq, "Hkv": self.Hkv,
            "Dh": self.Dh, "qk_dtype": self.qk_dtype, "scale": self.scale, "Dv": self.Dv,
            "f_dtype": self.f_dtype, "T_total": self.T_total, "N_total": self.N_total,
            "K_total": self.K_total,
            "sha256": {n: h(getattr(self, n)) for n in
                       ("cu_seqlens", "vis_start", "cu_vis", "q", "k", "feats", "cu_keep")},
        }

    def score_bytes(self) -> int:
        """Bytes the score pass must read at least once: every key row plus q."""
        elt = 2 if self.qk_dtype == BF16 else 4
        return (self.G * self.T_total * self.Hkv * self.Dh + self.G * self.R * self.Hq * self.Dh) * elt


def _cu(v) -> np.ndarray:
    out = np.zeros(len(v) + 1, np.int32)
    out[1:] = np.cumsum(np.asarray(v, dtype=np.int64))
    return out


def _layout(N: np.ndarray, T: np.ndarray):
    P = N + T
    vis_start = (T // 4).astype(np.int32)
    return _cu(P), vis_start, _cu(N)


def _mixture(rng, n: int, dv: int, comps: int, sigma: float) -> np.ndarray:
    """n points around `comps` random unit-norm centres; the noise has norm ~sigma."""
    centres = rng.standard_normal((comps, dv), dtype=np.float32)
    centres /= np.linalg.norm(centres, axis=1, keepdims=True)
    z = rng.integers(0, comps, size=n)
    x = centres[z]
    x += rng.standard_normal((n, dv), dtype=np.float32) * np.float32(sigma / math.sqrt(dv))
    return x


def _qk(rng_q, rng_k, G, R, Hq, Hkv, Dh, T_total, std):
    q = rng_q.standard_normal((G, R, Hq, Dh), dtype=np.float32) * np.float32(std)
    k = rng_k.standard_normal((G, T_total, Hkv, Dh), dtype=np.float32) * np.float32(std)
    return q, k


def _pool_map(fn, items):
    """Run fn over items on a few threads (numpy's samplers release the GIL);
    every item owns its seed, so the result does not depend on the thread count."""
    items = list(items)
    workers = max(1, min(8, os.cpu_count() or 1, len(items)))
    if workers == 1:
        return [fn(i) for i in items]
    with concurrent.futures.ThreadPoolExecutor(workers) as ex:
        return list(ex.map(fn, items))


def _features_c3(rng, n, dv):
    x = _mixture(rng, n, dv, 64, 0.3)
    for c in range(n // 576):
        crop = np.arange(c * 576, (c + 1) * 576)
        dst = rng.choice(crop, size=173, replace=False)
        keep = np.setdiff1d(crop, dst)
        src = rng.choice(keep, size=173, replace=True)
        eps = rng.standard_normal((173, dv), dtype=np.float32)
        eps *= (0.1 * np.linalg.norm(x[src], axis=1, keepdims=True)
                / np.linalg.norm(eps, axis=1, keepdims=True))
        x[dst] = x[src] + eps
    return x


def _features_c5(rng, n, dv):
    x = np.empty((n // 256, 256, dv), dtype=np.float32)
    for f in range(n // 256):
        if f % 16 == 0:
            x[f] = rng.standard_normal((256, dv), dtype=np.float32)
        else:
            x[f] = x[f - 1] + rng.standard_normal((256, dv), dtype=np.float32) * np.float32(0.05)
    return x.reshape(n, dv)


def make(name: str, budget: Optional[int] = None, sharp: bool = False, seed: int = 0) -> Workload:
    """Build one of the named workloads. `sharp` draws q and k with unit element std
    instead of 1/sqrt(Dh), which spreads the logits over a realistic range.

    Seeds: SeedSequence([2607, 27952, config id, seed]) spawns, in this order,
    the streams for sizes, q, k, planted tokens and features; the k and feature
    streams spawn one child per request (per layer and request for k)."""
    if name not in _CONFIG_IDS:
        raise ValueError(f"unknown workload {name!r}; expected one of {CONFIGS + EXTRA}")
    ss = np.random.SeedSequence([2607, 27952, _CONFIG_IDS[name], seed])
    ss_sizes, ss_q, ss_k, ss_plant, ss_feat = ss.spawn(5)
    s_sizes = np.random.default_rng(ss_sizes)
    s_plant = np.random.default_rng(ss_plant)
    planted = None

    if name == "c1_single_fp32":
        R, G, Hq, Hkv, Dh, Dv = 1, 1, 16, 16, 64, 1024
        N = np.array([576]); T = np.array([40])
        qkd, fd = F32, F32
        K = 64 if budget is None else budget
    elif name == "c2_llava15":
        R, G, Hq, Hkv, Dh, Dv = 64, 2, 32, 32, 128, 4096
        N = np.full(R, 576); T = np.full(R, 64)
        qkd, fd = BF16, BF16
        K = 64 if budget is None else budget
    elif name == "c3_llava_next":
        R, G, Hq, Hkv, Dh, Dv = 32, 1, 32, 8, 128, 4096
        N = np.full(R, 2880); T = np.full(R, 96)
        qkd, fd = BF16, BF16
        K = 320 if budget is None else budget
    elif name == "c4_dynres":
        R, G, Hq, Hkv, Dh, Dv = 128, 1, 12, 2, 128, 1536
        N = np.clip(np.rint(np.exp(s_sizes.uniform(math.log(256), math.log(16384), R))), 256, 16384).astype(np.int64)
        T = s_sizes.integers(32, 257, size=R)
        qkd, fd = BF16, BF16
        K = None if budget is None else budget
    elif name == "c5_video":
        R, G, Hq, Hkv, Dh, Dv = 8, 4, 28, 4, 128, 3584
        N = np.full(R, 64 * 256); T = np.full(R, 128)
        qkd, fd = BF16, BF16
        K = 1024 if budget is None else budget
    else:  # x1_long_video
        R, G, Hq, Hkv, Dh, Dv = 2, 4, 28, 4, 128, 3584
        N = np.full(R, 128 * 256); T = np.full(R, 128)
        qkd, fd = BF16, BF16
        K = 4096 if budget is None else budget

    N = N.astype(np.int64)
    T = T.astype(np.int64)
    cu_seqlens, vis_start, cu_vis = _layout(N, T)
    T_total = int(cu_seqlens[-1])
    scale = 1.0 / math.sqrt(Dh)
    std = np.float32(1.0 if sharp else 1.0 / math.sqrt(Dh))
    g = Hq // Hkv
    q32 = np.random.default_rng(ss_q).standard_normal((G, R, Hq, Dh), dtype=np.float32) * std

    if name in ("c1_single_fp32", "c2_llava15"):
        n_plant = 5 if name == "c1_single_fp32" else int(round(0.02 * 576))
        planted = [np.sort(s_plant.choice(int(N[r]), size=n_plant, replace=False)) for r in range(R)]

    kdt = np.uint16 if qkd == BF16 else np.float32
    k_out = np.empty((G, T_total, Hkv, Dh), dtype=kdt)
    k_seeds = ss_k.spawn(G * R)

    def fill_k(item):
        l, r = item
        a, b = int(cu_seqlens[r]), int(cu_seqlens[r + 1])
        blk = np.random.default_rng(k_seeds[l * R + r]).standard_normal((b - a, Hkv, Dh), dtype=np.float32)
        blk *= std
        if planted is not None:
            for kv in range(Hkv):
                u = q32[l, r, kv * g:(kv + 1) * g].mean(axis=0)
                step = (3.0 / scale) * u / float(np.dot(u, u))
                for i in planted[r]:
                    blk[int(vis_start[r]) + int(i), kv] += step
        k_out[l, a:b] = _store(blk, qkd)

    _pool_map(fill_k, [(l, r) for l in range(G) for r in range(R)])

    fdt = np.uint16 if fd == BF16 else np.float32
    f_out = np.empty((int(cu_vis[-1]), Dv), dtype=fdt)
    f_seeds = ss_feat.spawn(R)

    def fill_f(r):
        rng = np.random.default_rng(f_seeds[r])
        n = int(N[r])
        if name == "c1_single_fp32":
            x = _mixture(rng, n, Dv, 8, 0.3)
        elif name == "c2_llava15":
            x = _mixture(rng, n, Dv, 32, 0.3)
        elif name == "c3_llava_next":
            x = _features_c3(rng, n, Dv)
        elif name == "c4_dynres":
            x = _mixture(rng, n, Dv, 128, 0.3)
        else:   # c5_video, x1_long_video
            x = _features_c5(rng, n, Dv)
        f_out[int(cu_vis[r]):int(cu_vis[r + 1])] = _store(x, fd)

    _pool_map(fill_f, range(R))

    if K is None:
        Kr = (N + 7) // 8
    else:
        Kr = np.full(R, int(K))
    cu_keep = _cu(Kr)
    return Workload(name=name + ("_sharp" if sharp else ""), R=R, G=G, Hq=Hq, Hkv=Hkv, Dh=Dh,
                    qk_dtype=qkd, scale=scale, cu_seqlens=cu_seqlens, vis_start=vis_start,
                    cu_vis=cu_vis, q=_store(q32, qkd), k=k_out, Dv=Dv, f_dtype=fd,
                    feats=f_out, cu_keep=cu_keep, planted=planted, qk_std=float(std))


def tiny(seed: int, R: int = 2, G: int = 1, Hq: int = 4, Hkv: int = 2, Dh: int = 64,
         n_range=(1, 48), t_range=(1, 16), Dv: int = 32, qk_dtype: str = BF16,
         f_dtype: str = BF16, sharp: bool = True, comps: int = 4, k_frac=None) -> Workload:
    """Small random batch for oracle/brute-force and parity tests.

    Visual and text counts are drawn per request from the inclusive ranges; the
    budget is drawn uniformly in [1, N_r] unless k_frac fixes K_r = ceil(k_frac*N_r).
    """
    rng = np.random.default_rng(np.random.SeedSequence([2607, 27952, 99, seed]))
    N = rng.integers(n_range[0], n_range[1] + 1, size=R)
    T = rng.integers(max(1, t_range[0]), t_range[1] + 1, size=R)
    cu_seqlens, vis_start, cu_vis = _layout(N, T)
    std = 1.0 if sharp else 1.0 / math.sqrt(Dh)
    q32, k32 = _qk(rng, rng, G, R, Hq, Hkv, Dh, int(cu_seqlens[-1]), std)
    feats = np.concatenate([_mixture(rng, int(n), Dv, comps, 0.5) for n in N])
    if k_frac is None:
        Kr = np.array([rng.integers(1, int(n) + 1) for n in N])
    else:
        Kr = np.array([max(1, min(int(n), math.ceil(k_frac * int(n)))) for n in N])
    return Workload(name=f"tiny{seed}", R=R, G=G, Hq=Hq, Hkv=Hkv, Dh=Dh, qk_dtype=qk_dtype,
                    scale=1.0 / math.sqrt(Dh), cu_seqlens=cu_seqlens, vis_start=vis_start,
                    cu_vis=cu_vis, q=_store(q32, qk_dtype), k=_store(k32, qk_dtype), Dv=Dv,
                    f_dtype=f_dtype, feats=_store(feats, f_dtype), cu_keep=_cu(Kr), qk_std=float(std))


@dataclasses.dataclass
class QueryRows:
    """Queries of every text-query token of a batch: the tokens after each
    request's visual span, positions [q_begin[r], q_end[r]) with
    q_end[r] = P_r (the last of them is the last query token).

      q_begin, q_end  [R] request-local positions
      cu_q            [R+1] CSR offsets of the rows in q
      q               [G][Q_total][Hq][Dh], the workload's storage dtype
    """
    q_begin: np.ndarray
    q_end: np.ndarray
    cu_q: np.ndarray
    q: np.ndarray

    def rows(self, r: int) -> np.ndarray:
        """q of request r's query tokens: [G][M_r][Hq][Dh]."""
        return self.q[:, int(self.cu_q[r]):int(self.cu_q[r + 1])]

    def subset(self, reqs) -> "QueryRows":
        reqs = [int(r) for r in reqs]
        return QueryRows(q_begin=self.q_begin[reqs].copy(), q_end=self.q_end[reqs].copy(),
                         cu_q=_cu([int(self.cu_q[r + 1] - self.cu_q[r]) for r in reqs]),
                         q=np.ascontiguousarray(np.concatenate([self.rows(r) for r in reqs], axis=1)))


def query_rows(wl: Workload, seed: int = 0) -> QueryRows:
    """Queries for every text token after the visual span of each request.

    The row of the last token is the workload's own q (so a source made of
    that row alone is the last-token path); the others are fresh draws with
    the same element distribution, from SeedSequence([2607, 27952, 1000 +
    seed, r]) for request r. Nothing here depends on how rows are chosen."""
    N = np.diff(wl.cu_vis).astype(np.int64)
    P = np.diff(wl.cu_seqlens).astype(np.int64)
    qb = (wl.vis_start.astype(np.int64) + N).astype(np.int32)
    qe = P.astype(np.int32)
    M = (qe - qb).astype(np.int64)
    if np.any(M < 1):
        raise ValueError("every request needs at least one text token after its visual span")
    cu_q = _cu(M)
    std = np.float32(wl.qk_std if wl.qk_std > 0 else 1.0 / math.sqrt(wl.Dh))
    dt = np.uint16 if wl.qk_dtype == BF16 else np.float32
    out = np.empty((wl.G, int(cu_q[-1]), wl.Hq, wl.Dh), dtype=dt)
    for r in range(wl.R):
        rng = np.random.default_rng(np.random.SeedSequence([2607, 27952, 1000 + seed, r]))
        x = rng.standard_normal((wl.G, int(M[r]), wl.Hq, wl.Dh), dtype=np.float32) * std
        a = int(cu_q[r])
        out[:, a:a + int(M[r]) - 1] = _store(x[:, :-1], wl.qk_dtype)
        out[:, a + int(M[r]) - 1] = wl.q[:, r]
    return QueryRows(q_begin=qb, q_end=qe, cu_q=cu_q, q=out)


@dataclasses.dataclass
class PrefillInputs:
    """Queries and values of every prefill position, for the guidance model's
    causal prefill attention.

      q  [G][T_total][Hq][Dh]   queries of every position; each request's last
                                position holds the workload's own last query
      v  [G][T_total][Hkv][Dh]  values, drawn N(0, 1)
    Both in the workload's storage dtype."""
    q: np.ndarray
    v: np.ndarray


def prefill_inputs(wl: Workload, seed: int = 0, ids=None) -> PrefillInputs:
    """Draw prefill queries and values. Request r draws from SeedSequence([2607,
    27952, 2000 + seed, ids[r], layer]) (ids defaults to 0..R-1, so that a
    subset can reproduce the rows of the batch it came from)."""
    ids = list(range(wl.R)) if ids is None else [int(i) for i in ids]
    std = np.float32(wl.qk_std if wl.qk_std > 0 else 1.0 / math.sqrt(wl.Dh))
    dt = np.uint16 if wl.qk_dtype == BF16 else np.float32
    T = wl.T_total
    q_out = np.empty((wl.G, T, wl.Hq, wl.Dh), dtype=dt)
    v_out = np.empty((wl.G, T, wl.Hkv, wl.Dh), dtype=dt)

    def fill(item):
        l, r = item
        a, b = int(wl.cu_seqlens[r]), int(wl.cu_seqlens[r + 1])
        rng = np.random.default_rng(np.random.SeedSequence([2607, 27952, 2000 + seed, ids[r], l]))
        qq = rng.standard_normal((b - a, wl.Hq, wl.Dh), dtype=np.float32) * std
        vv = rng.standard_normal((b - a, wl.Hkv, wl.Dh), dtype=np.float32)
        q_out[l, a:b - 1] = _store(qq[:-1], wl.qk_dtype)
        q_out[l, b - 1] = wl.q[l, r]
        v_out[l, a:b] = _store(vv, wl.qk_dtype)

    _pool_map(fill, [(l, r) for l in range(wl.G) for r in range(wl.R)])
    return PrefillInputs(q=q_out, v=v_out)


@dataclasses.dataclass
class ConnectorWeights:
    """Synthetic weights of a token-wise connector: LayerNorm(Dv) -> Linear(Dv, Dh)
    -> GELU -> Linear(Dh, Do). w1 [Dh][Dv] and w2 [Do][Dh] in the storage dtype
    (one output feature per row), the rest fp32."""
    gamma: np.ndarray
    beta: np.ndarray
    w1: np.ndarray
    b1: np.ndarray
    w2: np.ndarray
    b2: np.ndarray
    dtype: str


def connector_weights(Dv: int, Dh: int, Do: int, dtype: str = BF16, seed: int = 0) -> ConnectorWeights:
    """Draw from SeedSequence([2607, 27952, 3000 + seed]): weights N(0, 1/fan_in),
    biases N(0, 0.02^2), gamma 1 + N(0, 0.1^2), beta N(0, 0.1^2)."""
    rng = np.random.default_rng(np.random.SeedSequence([2607, 27952, 3000 + seed]))
    f32 = np.float32
    gamma = (1.0 + 0.1 * rng.standard_normal(Dv, dtype=f32)).astype(f32)
    beta = (0.1 * rng.standard_normal(Dv, dtype=f32)).astype(f32)
    w1 = rng.standard_normal((Dh, Dv), dtype=f32) * f32(1.0 / math.sqrt(Dv))
    b1 = (0.02 * rng.standard_normal(Dh, dtype=f32)).astype(f32)
    w2 = rng.standard_normal((Do, Dh), dtype=f32) * f32(1.0 / math.sqrt(Dh))
    b2 = (0.02 * rng.standard_normal(Do, dtype=f32)).astype(f32)
    return ConnectorWeights(gamma=gamma, beta=beta, w1=_store(w1, dtype), b1=b1, w2=_store(w2, dtype), b2=b2,
                            dtype=dtype)


def connector_dims(wl: Workload):
    """(Dh, Do) of the cloud connector for a workload: a square token-wise MLP
    at the feature width (Dv -> Dv -> Dv), the shape of a connector whose
    encoder width already matches the language model's."""
    return wl.Dv, wl.Dv

