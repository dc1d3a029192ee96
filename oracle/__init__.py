"""CPU oracle for the LAST token-selection path -- TEST INFRASTRUCTURE ONLY.

Thin numpy/ctypes wrapper over ``oracle/oracle.c`` (fp64, plain loops). Only
the tests, the smoke check and the benchmark's CPU-baseline leg use it; the
product library never imports it, and it imports nothing from the product.

Each function names the paper passage it follows (arXiv 2607.27952, Sec. 3):
  scores  -- Eq. 6-8 (last-query-token attention row, sum over layers and
             heads, normalisation over the visual tokens)
  select  -- Eq. 9-12 (importance-weighted greedy k-center, ascending kept
             indices) and the Table 5 Top-k ablation
  replay  -- teacher-forced check of a candidate pick sequence under Eq. 9-11
  gather  -- Eq. 12 (rows of X in ascending kept order)
  budget  -- Eq. 2 (K = ceil(rho * N))
  rows_scores -- Table 4 attention sources: Eq. 6-8 over any set of causal
             query rows per request (first / middle / every query token)
  source_rows -- the row positions of each Table 4 attention source
  connector -- Sec. 3.4 (after Eq. 12), Sec. 3.2: the cloud's token-wise connector on X_S
  prefill -- Sec. 3.3: the guidance model's causal prefill attention
             (every query row), whose last row Eq. 7 reads
"""
import ctypes
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "liboracle.so")

F32, BF16 = 0, 1
KCENTER, TOPK = 0, 1

_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            from . import build as _b
            _b.build()
        L = ctypes.CDLL(LIB_PATH)
        P, I, I64, D = ctypes.c_void_p, ctypes.c_int, ctypes.c_int64, ctypes.c_double
        L.oracle_scores.argtypes = [I, I, I, I, I, I, D, P, P, P, P, P, P, P, I]
        L.oracle_scores.restype = I
        L.oracle_select.argtypes = [I, I, I, I, P, P, P, P, P, P, P, I]
        L.oracle_select.restype = I
        L.oracle_replay.argtypes = [I, I, I, P, P, P, P, P, D, P, P, P, I]
        L.oracle_replay.restype = I
        L.oracle_gather.argtypes = [I, I64, P, P, P, P, P]
        L.oracle_gather.restype = I
        L.oracle_budget.argtypes = [I64, I64, I64]
        L.oracle_budget.restype = I64
        L.oracle_rows_scores.argtypes = [I, I, I, I, I, I, D, P, P, P, P, P, P, P, P, P, I]
        L.oracle_rows_scores.restype = I
        L.oracle_source_rows.argtypes = [I, ctypes.c_int32, ctypes.c_int32, P]
        L.oracle_source_rows.restype = I
        L.oracle_prefill.argtypes = [I, I, I, I, I, I, D, P, P, P, P, P, I]
        L.oracle_prefill.restype = I
        L.oracle_connector.argtypes = [I64, I, I, I, I, D, P, P, P, P, P, P, P, P, P, P, I]
        L.oracle_connector.restype = I
        L.oracle_max_threads.argtypes = []
        L.oracle_max_threads.restype = I
        _lib = L
    return _lib


def _ptr(a):
    return ctypes.c_void_p(a.ctypes.data) if a is not None else None


def _i32(a):
    return np.ascontiguousarray(a, dtype=np.int32)


def _storage(x, dtype):
    """Return (contiguous array, dtype code). bf16 data is passed as uint16 bit patterns."""
    if dtype == BF16:
        x = np.ascontiguousarray(x)
        assert x.dtype == np.uint16, "bf16 inputs are passed as uint16 bit patterns"
        return x, BF16
    x = np.ascontiguousarray(x, dtype=np.float32)
    return x, F32


def max_threads():
    return lib().oracle_max_threads()


def scores(R, G, Hq, Hkv, Dh, q, k, cu_seqlens, vis_start, cu_vis, dtype,
           scale=0.0, want_rows=False, nthreads=0):
    """Eq. 6-8 in fp64. Returns w [N_total] (fp64) and, if asked, rows [G][Hq][T_total]."""
    cu_seqlens, vis_start, cu_vis = _i32(cu_seqlens), _i32(vis_start), _i32(cu_vis)
    q, qd = _storage(q, dtype)
    k, _ = _storage(k, dtype)
    T = int(cu_seqlens[R])
    w = np.zeros(int(cu_vis[R]), dtype=np.float64)
    rows = np.zeros((G, Hq, T), dtype=np.float64) if want_rows else None
    rc = lib().oracle_scores(R, G, Hq, Hkv, Dh, qd, float(scale), _ptr(cu_seqlens),
                             _ptr(vis_start), _ptr(cu_vis), _ptr(q), _ptr(k), _ptr(w),
                             _ptr(rows), nthreads)
    if rc != 0:
        raise RuntimeError(f"oracle_scores failed ({rc})")
    return (w, rows) if want_rows else w


def rows_scores(R, G, Hq, Hkv, Dh, q, k, cu_seqlens, vis_start, cu_vis, cu_rows, row_pos, dtype,
                scale=0.0, want_sums=False, nthreads=0):
    """Table 4 sources: Eq. 6-8 summed over the causal rows at row_pos (CSR by cu_rows).

    q is [G][M_total][Hq][Dh]. Returns w [N_total] (fp64) and, if asked, the
    unnormalised sums s [N_total].
    """
    cu_seqlens, vis_start, cu_vis = _i32(cu_seqlens), _i32(vis_start), _i32(cu_vis)
    cu_rows, row_pos = _i32(cu_rows), _i32(row_pos)
    q, qd = _storage(q, dtype)
    k, _ = _storage(k, dtype)
    w = np.zeros(int(cu_vis[R]), dtype=np.float64)
    s = np.zeros(int(cu_vis[R]), dtype=np.float64) if want_sums else None
    rc = lib().oracle_rows_scores(R, G, Hq, Hkv, Dh, qd, float(scale), _ptr(cu_seqlens),
                                  _ptr(vis_start), _ptr(cu_vis), _ptr(cu_rows), _ptr(row_pos),
                                  _ptr(q), _ptr(k), _ptr(w), _ptr(s), nthreads)
    if rc != 0:
        raise RuntimeError(f"oracle_rows_scores failed ({rc})")
    return (w, s) if want_sums else w


SRC_LAST, SRC_FIRST, SRC_MIDDLE, SRC_ALL_MEAN = 0, 1, 2, 3


def connector(x, gamma, beta, w1, b1, w2, b2, dtype, eps=1e-5, want_intermediate=False, nthreads=0):
    """phi_c of Sec. 3.2 / 3.4 on X_S (Eq. 12) in fp64: y [K][Do] (and xhat [K][Dv], h [K][Dh] if asked)."""
    x, xd = _storage(x, dtype)
    w1, _ = _storage(w1, dtype)
    w2, _ = _storage(w2, dtype)
    K, Dv = x.shape
    Dh, Do = w1.shape[0], w2.shape[0]
    f = lambda a: np.ascontiguousarray(a, dtype=np.float32)
    gamma, beta, b1, b2 = f(gamma), f(beta), f(b1), f(b2)
    y = np.zeros((K, Do))
    xh = np.zeros((K, Dv)) if want_intermediate else None
    h = np.zeros((K, Dh)) if want_intermediate else None
    rc = lib().oracle_connector(K, Dv, Dh, Do, xd, float(eps), _ptr(x), _ptr(gamma), _ptr(beta), _ptr(w1),
                                _ptr(b1), _ptr(w2), _ptr(b2), _ptr(y), _ptr(xh), _ptr(h), nthreads)
    if rc != 0:
        raise RuntimeError(f"oracle_connector failed ({rc})")
    return (y, xh, h) if want_intermediate else y


def prefill(R, G, Hq, Hkv, Dh, q, k, v, cu_seqlens, dtype, scale=0.0, nthreads=0):
    """Causal prefill attention (Eq. 6, every row) in fp64: out [G][T_total][Hq][Dh]."""
    cu_seqlens = _i32(cu_seqlens)
    q, qd = _storage(q, dtype)
    k, _ = _storage(k, dtype)
    v, _ = _storage(v, dtype)
    T = int(cu_seqlens[R])
    out = np.zeros((G, T, Hq, Dh), dtype=np.float64)
    rc = lib().oracle_prefill(R, G, Hq, Hkv, Dh, qd, float(scale), _ptr(cu_seqlens), _ptr(q), _ptr(k),
                              _ptr(v), _ptr(out), nthreads)
    if rc != 0:
        raise RuntimeError(f"oracle_prefill failed ({rc})")
    return out


def source_rows(src, qb, qe):
    """Table 4: positions of the rows of attention source `src` for a query at [qb, qe)."""
    pos = np.zeros(max(1, qe - qb), np.int32)
    n = lib().oracle_source_rows(int(src), int(qb), int(qe), _ptr(pos))
    if n < 0:
        raise ValueError("empty query or unknown source")
    return pos[:n].copy()


def select(R, Dv, w32, feats, cu_vis, cu_keep, dtype, mode=KCENTER, nthreads=0):
    """Eq. 9-12 (mode KCENTER) or Table 5 Top-k (mode TOPK). w32 is the fp32 relevance."""
    cu_vis, cu_keep = _i32(cu_vis), _i32(cu_keep)
    w32 = np.ascontiguousarray(w32, dtype=np.float32)
    feats, fd = _storage(feats, dtype)
    Kt = int(cu_keep[R])
    kept = np.zeros(Kt, np.int32)
    order = np.zeros(Kt, np.int32)
    gains = np.zeros(Kt, np.float64)
    rc = lib().oracle_select(R, Dv, fd, mode, _ptr(w32), _ptr(feats), _ptr(cu_vis),
                             _ptr(cu_keep), _ptr(kept), _ptr(order), _ptr(gains), nthreads)
    if rc != 0:
        raise RuntimeError(f"oracle_select failed ({rc})")
    return kept, order, gains


def replay(R, Dv, w32, feats, cu_vis, cu_keep, picks, dtype, rel_tol=1e-6, nthreads=0, want_objective=False):
    """Teacher-forced replay of `picks` under Eq. 9-11.

    Returns (status, margin): status 0 exact / 1 excused near-tie / 2 failed per step;
    with want_objective also the oracle's fp64 objective of each pick.
    """
    cu_vis, cu_keep, picks = _i32(cu_vis), _i32(cu_keep), _i32(picks)
    w32 = np.ascontiguousarray(w32, dtype=np.float32)
    feats, fd = _storage(feats, dtype)
    Kt = int(cu_keep[R])
    status = np.zeros(Kt, np.int32)
    margin = np.zeros(Kt, np.float64)
    obj = np.zeros(Kt, np.float64) if want_objective else None
    rc = lib().oracle_replay(R, Dv, fd, _ptr(w32), _ptr(feats), _ptr(cu_vis), _ptr(cu_keep),
                             _ptr(picks), float(rel_tol), _ptr(status), _ptr(margin), _ptr(obj), nthreads)
    if rc != 0:
        raise RuntimeError(f"oracle_replay failed ({rc})")
    return (status, margin, obj) if want_objective else (status, margin)


def gather(R, feats, cu_vis, kept, cu_keep):
    """Eq. 12: rows of feats in the order of `kept`, request by request (byte copy)."""
    cu_vis, cu_keep, kept = _i32(cu_vis), _i32(cu_keep), _i32(kept)
    feats = np.ascontiguousarray(feats)
    row_bytes = feats.strides[0] if feats.ndim == 2 else feats.itemsize
    out = np.zeros((int(cu_keep[R]),) + feats.shape[1:], dtype=feats.dtype)
    rc = lib().oracle_gather(R, int(row_bytes), _ptr(feats), _ptr(cu_vis), _ptr(kept),
                             _ptr(cu_keep), _ptr(out))
    if rc != 0:
        raise RuntimeError(f"oracle_gather failed ({rc})")
    return out


def budget(n, num, den):
    """Eq. 2: ceil(n * num / den), integer-exact."""
    return int(lib().oracle_budget(int(n), int(num), int(den)))
