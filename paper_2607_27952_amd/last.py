"""ctypes binding over liblast.so (include/last.h). Argument marshalling only:
every step of the path runs in the library's HIP kernels; PyTorch provides
device memory and the current stream.

The library must be built (``python -m paper_2607_27952_amd._build`` or
``__graft_entry__.build()``); loading fails loudly if it is missing.
"""
from __future__ import annotations

import contextlib
import ctypes
import os
from dataclasses import dataclass
from typing import Optional

import numpy as np
import torch  # imported before the library so that both share torch's HIP runtime

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "liblast.so")

LAST_OK, LAST_ERR_INVALID, LAST_ERR_UNSUPPORTED, LAST_ERR_WORKSPACE, LAST_ERR_DEVICE = range(5)
LAST_F32, LAST_BF16 = 0, 1
KCENTER, TOPK = 0, 1
SRC_LAST, SRC_FIRST, SRC_MIDDLE, SRC_ALL_MEAN = 0, 1, 2, 3

EXPORTS = ("last_token_scores_workspace", "last_token_scores", "last_token_scores_static", "last_source_rows",
           "last_rows_scores_workspace", "last_rows_scores", "last_prefill_attention_workspace",
           "last_prefill_attention", "diverse_select_workspace", "diverse_select_similarity_workspace",
           "diverse_select", "diverse_select_similarity", "diverse_select_pick", "gather_kept", "last_connector_workspace", "last_connector", "last_budget", "last_status_string", "last_version",
           "last_profile_enable", "last_profile_collect", "last_profile_reset",
           "last_profile_count", "last_profile_kernel")


class LastError(RuntimeError):
    def __init__(self, status: int, what: str):
        self.status = status
        super().__init__(f"{what}: {status_string(status)} (status {status})")


class _Batch(ctypes.Structure):
    _fields_ = [("R", ctypes.c_int32), ("G", ctypes.c_int32), ("Hq", ctypes.c_int32),
                ("Hkv", ctypes.c_int32), ("Dh", ctypes.c_int32), ("qk_dtype", ctypes.c_int32),
                ("softmax_scale", ctypes.c_float),
                ("cu_seqlens", ctypes.c_void_p), ("cu_seqlens_h", ctypes.c_void_p),
                ("vis_start", ctypes.c_void_p), ("vis_start_h", ctypes.c_void_p),
                ("cu_vis", ctypes.c_void_p), ("cu_vis_h", ctypes.c_void_p)]


_lib = None


def lib():
    """Load liblast.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with __graft_entry__.build() "
                               "or python -m paper_2607_27952_amd._build")
        L = ctypes.CDLL(LIB_PATH)
        P, I32, SZ = ctypes.c_void_p, ctypes.c_int32, ctypes.c_size_t
        L.last_token_scores_workspace.argtypes = [ctypes.POINTER(_Batch)]
        L.last_token_scores_workspace.restype = SZ
        L.last_token_scores.argtypes = [ctypes.POINTER(_Batch), P, P, P, P, P, SZ, P]
        L.last_token_scores.restype = I32
        L.last_token_scores_static.argtypes = [ctypes.POINTER(_Batch), P, P, P, P, P]
        L.last_token_scores_static.restype = I32
        L.last_source_rows.argtypes = [I32, I32, I32, P]
        L.last_source_rows.restype = I32
        L.last_rows_scores_workspace.argtypes = [ctypes.POINTER(_Batch), P, P]
        L.last_rows_scores_workspace.restype = SZ
        L.last_rows_scores.argtypes = [ctypes.POINTER(_Batch), P, P, P, P, P, P, P, P, SZ, P]
        L.last_rows_scores.restype = I32
        L.last_prefill_attention_workspace.argtypes = [ctypes.POINTER(_Batch)]
        L.last_prefill_attention_workspace.restype = SZ
        L.last_prefill_attention.argtypes = [ctypes.POINTER(_Batch), P, P, P, P, P, P, SZ, P]
        L.last_prefill_attention.restype = I32
        L.diverse_select_workspace.argtypes = [I32, P, I32, I32, I32]
        L.diverse_select_workspace.restype = SZ
        L.diverse_select_similarity_workspace.argtypes = [I32, P, I32, I32]
        L.diverse_select_similarity_workspace.restype = SZ
        L.diverse_select.argtypes = [I32, I32, I32, I32, P, P, P, P, P, P, P, P, P, P, SZ, P]
        L.diverse_select.restype = I32
        L.diverse_select_similarity.argtypes = [I32, I32, I32, P, P, P, P, SZ, P]
        L.diverse_select_similarity.restype = I32
        L.diverse_select_pick.argtypes = [I32, I32, I32, P, P, P, P, P, P, P, P, P, SZ, P]
        L.diverse_select_pick.restype = I32
        L.gather_kept.argtypes = [I32, I32, SZ, P, P, P, P, P, P, P, P]
        L.gather_kept.restype = I32
        I64 = ctypes.c_int64
        L.last_connector_workspace.argtypes = [I64, I32, I32]
        L.last_connector_workspace.restype = SZ
        L.last_connector.argtypes = [I32, I64, I32, I32, I32, ctypes.c_float, P, P, P, P, P, P, P, P, P, SZ, P]
        L.last_connector.restype = I32
        L.last_budget.argtypes = [I32, I32, I32]
        L.last_budget.restype = I32
        L.last_status_string.argtypes = [I32]
        L.last_status_string.restype = ctypes.c_char_p
        L.last_version.argtypes = []
        L.last_version.restype = I32
        L.last_profile_enable.argtypes = [I32]
        L.last_profile_enable.restype = I32
        L.last_profile_collect.argtypes = []
        L.last_profile_collect.restype = I32
        L.last_profile_reset.argtypes = []
        L.last_profile_reset.restype = None
        L.last_profile_count.argtypes = []
        L.last_profile_count.restype = I32
        L.last_profile_kernel.argtypes = [I32, ctypes.POINTER(ctypes.c_char_p),
                                          ctypes.POINTER(ctypes.c_int64), ctypes.POINTER(ctypes.c_double)]
        L.last_profile_kernel.restype = I32
        _lib = L
    return _lib


def status_string(status: int) -> str:
    return lib().last_status_string(int(status)).decode()


def _ptr(t) -> Optional[int]:
    if t is None:
        return None
    if isinstance(t, np.ndarray):
        return t.ctypes.data
    return t.data_ptr()


def _stream(stream) -> int:
    s = stream if stream is not None else torch.cuda.current_stream()
    return s.cuda_stream


def _on(stream):
    """Allocate a call's temporaries (device CSR copies, outputs, workspace) on
    the stream the call enqueues on. torch's caching allocator then frees them
    in that stream's order, so a block cannot be handed to another stream's
    allocation while the library's kernels still read it."""
    return torch.cuda.stream(stream) if stream is not None else contextlib.nullcontext()


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.bfloat16:
        return LAST_BF16
    if t.dtype == torch.float32:
        return LAST_F32
    raise TypeError(f"unsupported dtype {t.dtype}; expected bfloat16 or float32")


def _i32_host(a) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a, dtype=np.int32))


def _i32_dev(a: np.ndarray, device) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).to(device)


def _workspace(nbytes: int, device) -> torch.Tensor:
    # torch's caching allocator hands out 512-byte aligned blocks
    return torch.empty(max(int(nbytes), 256), dtype=torch.uint8, device=device)


@dataclass
class Batch:
    """A ragged batch of requests: host and device copies of the CSR arrays."""
    R: int
    G: int
    Hq: int
    Hkv: int
    Dh: int
    scale: float
    cu_seqlens_h: np.ndarray
    vis_start_h: np.ndarray
    cu_vis_h: np.ndarray
    cu_seqlens: torch.Tensor
    vis_start: torch.Tensor
    cu_vis: torch.Tensor

    @staticmethod
    def make(G, Hq, Hkv, Dh, cu_seqlens, vis_start, cu_vis, scale=0.0, device="cuda"):
        cs, vs, cv = _i32_host(cu_seqlens), _i32_host(vis_start), _i32_host(cu_vis)
        return Batch(R=len(cs) - 1, G=G, Hq=Hq, Hkv=Hkv, Dh=Dh, scale=float(scale),
                     cu_seqlens_h=cs, vis_start_h=vs, cu_vis_h=cv, cu_seqlens=_i32_dev(cs, device),
                     vis_start=_i32_dev(vs, device), cu_vis=_i32_dev(cv, device))

    def struct(self, qk_dtype: int) -> _Batch:
        return _Batch(self.R, self.G, self.Hq, self.Hkv, self.Dh, qk_dtype, self.scale,
                      _ptr(self.cu_seqlens), _ptr(self.cu_seqlens_h), _ptr(self.vis_start),
                      _ptr(self.vis_start_h), _ptr(self.cu_vis), _ptr(self.cu_vis_h))

    @property
    def T_total(self) -> int:
        return int(self.cu_seqlens_h[-1])

    @property
    def N_total(self) -> int:
        return int(self.cu_vis_h[-1])


def token_scores_workspace(batch: Batch, qk_dtype=torch.bfloat16) -> int:
    code = LAST_BF16 if qk_dtype == torch.bfloat16 else LAST_F32
    b = batch.struct(code)
    return int(lib().last_token_scores_workspace(ctypes.byref(b)))


def token_scores(batch: Batch, q: torch.Tensor, k: torch.Tensor, scores=None, attn_rows=None,
                 want_rows=False, ws=None, stream=None):
    """last_token_scores (Eq. 6-8): returns scores [N_total] fp32 (and rows if asked)."""
    with _on(stream):
        code = _dtype_code(q)
        if k.dtype != q.dtype:
            raise TypeError("q and k must share a dtype")
        b = batch.struct(code)
        if scores is None:
            scores = torch.empty(batch.N_total, dtype=torch.float32, device=q.device)
        if want_rows and attn_rows is None:
            attn_rows = torch.empty((batch.G, batch.Hq, batch.T_total), dtype=torch.float32, device=q.device)
        need = int(lib().last_token_scores_workspace(ctypes.byref(b)))
        if ws is None:
            ws = _workspace(need, q.device)
        st = lib().last_token_scores(ctypes.byref(b), _ptr(q), _ptr(k), _ptr(scores), _ptr(attn_rows),
                                     _ptr(ws), ws.numel(), _stream(stream))
        if st != LAST_OK:
            raise LastError(st, "last_token_scores")
        return (scores, attn_rows) if want_rows else scores


STATIC_SCRATCH_BYTES = 64 << 20   # LAST_STATIC_SCRATCH_BYTES


def token_scores_static(batch: Batch, q: torch.Tensor, k: torch.Tensor, scores=None, attn_rows=None,
                        want_rows=False, stream=None):
    """last_token_scores_static: last_token_scores on the library's static per-device
    scratch (no workspace). Allocates nothing when `scores` (and `attn_rows`) are given."""
    code = _dtype_code(q)
    if k.dtype != q.dtype:
        raise TypeError("q and k must share a dtype")
    b = batch.struct(code)
    with _on(stream):
        if scores is None:
            scores = torch.empty(batch.N_total, dtype=torch.float32, device=q.device)
        if want_rows and attn_rows is None:
            attn_rows = torch.empty((batch.G, batch.Hq, batch.T_total), dtype=torch.float32, device=q.device)
        st = lib().last_token_scores_static(ctypes.byref(b), _ptr(q), _ptr(k), _ptr(scores), _ptr(attn_rows),
                                            _stream(stream))
    if st != LAST_OK:
        raise LastError(st, "last_token_scores_static")
    return (scores, attn_rows) if want_rows else scores


def source_rows(src: int, q_begin: int, q_end: int) -> np.ndarray:
    """last_source_rows (Table 4): positions of the rows of attention source `src`."""
    pos = np.zeros(max(1, int(q_end) - int(q_begin)), np.int32)
    n = lib().last_source_rows(int(src), int(q_begin), int(q_end), _ptr(pos))
    if n < 0:
        raise ValueError("empty query or unknown attention source")
    return pos[:n].copy()


@dataclass
class Rows:
    """Query rows per request (CSR): host and device copies."""
    cu_rows_h: np.ndarray
    row_pos_h: np.ndarray
    cu_rows: torch.Tensor
    row_pos: torch.Tensor

    @staticmethod
    def make(cu_rows, row_pos, device="cuda") -> "Rows":
        cr, rp = _i32_host(cu_rows), _i32_host(row_pos)
        return Rows(cu_rows_h=cr, row_pos_h=rp, cu_rows=_i32_dev(cr, device), row_pos=_i32_dev(rp, device))


def rows_scores_workspace(batch: Batch, rows: Rows, qk_dtype=torch.bfloat16) -> int:
    code = LAST_BF16 if qk_dtype == torch.bfloat16 else LAST_F32
    b = batch.struct(code)
    return int(lib().last_rows_scores_workspace(ctypes.byref(b), _ptr(rows.cu_rows_h), _ptr(rows.row_pos_h)))


def rows_scores(batch: Batch, rows: Rows, q: torch.Tensor, k: torch.Tensor, scores=None, ws=None,
                stream=None):
    """last_rows_scores (Table 4 sources): scores [N_total] fp32 from the causal rows
    at rows.row_pos; q is [G][M_total][Hq][Dh]."""
    with _on(stream):
        code = _dtype_code(q)
        if k.dtype != q.dtype:
            raise TypeError("q and k must share a dtype")
        b = batch.struct(code)
        if scores is None:
            scores = torch.empty(batch.N_total, dtype=torch.float32, device=q.device)
        need = int(lib().last_rows_scores_workspace(ctypes.byref(b), _ptr(rows.cu_rows_h), _ptr(rows.row_pos_h)))
        if ws is None:
            ws = _workspace(need, q.device)
        st = lib().last_rows_scores(ctypes.byref(b), _ptr(rows.cu_rows), _ptr(rows.cu_rows_h), _ptr(rows.row_pos),
                                    _ptr(rows.row_pos_h), _ptr(q), _ptr(k), _ptr(scores), _ptr(ws), ws.numel(),
                                    _stream(stream))
        if st != LAST_OK:
            raise LastError(st, "last_rows_scores")
        return scores


def prefill_attention_workspace(batch: Batch) -> int:
    b = batch.struct(LAST_BF16)
    return int(lib().last_prefill_attention_workspace(ctypes.byref(b)))


def prefill_attention(batch: Batch, q: torch.Tensor, k: torch.Tensor, v: torch.Tensor, out=None, scores=None,
                      ws=None, stream=None):
    """last_prefill_attention (Sec. 3.3): causal attention of every position,
    out [G][T_total][Hq][Dh] bf16, and the last-row scores [N_total] fp32."""
    with _on(stream):
        code = _dtype_code(q)
        if k.dtype != q.dtype or v.dtype != q.dtype:
            raise TypeError("q, k and v must share a dtype")
        b = batch.struct(code)
        if out is None:
            out = torch.empty(q.shape, dtype=q.dtype, device=q.device)
        if scores is None:
            scores = torch.empty(batch.N_total, dtype=torch.float32, device=q.device)
        if ws is None:
            ws = _workspace(lib().last_prefill_attention_workspace(ctypes.byref(b)), q.device)
        st = lib().last_prefill_attention(ctypes.byref(b), _ptr(q), _ptr(k), _ptr(v), _ptr(out), _ptr(scores),
                                          _ptr(ws), ws.numel(), _stream(stream))
        if st != LAST_OK:
            raise LastError(st, "last_prefill_attention")
        return out, scores


def select_workspace(cu_vis_h, Dv: int, f_dtype=torch.bfloat16, mode: int = KCENTER, pair: bool = False) -> int:
    """Workspace bytes of diverse_select, or (pair=True) of the two-call form
    diverse_select_similarity + diverse_select_pick."""
    cv = _i32_host(cu_vis_h)
    code = LAST_BF16 if f_dtype == torch.bfloat16 else LAST_F32
    if pair:
        return int(lib().diverse_select_similarity_workspace(len(cv) - 1, _ptr(cv), Dv, code))
    return int(lib().diverse_select_workspace(len(cv) - 1, _ptr(cv), Dv, code, mode))


def diverse_select(scores: torch.Tensor, feats: torch.Tensor, cu_vis_h, cu_keep_h, cu_vis=None,
                   cu_keep=None, mode: int = KCENTER, kept=None, order=None, gains=None,
                   want_order=True, ws=None, stream=None):
    """diverse_select (Eq. 9-12 or the Top-k ablation): returns (kept, order, gains)."""
    with _on(stream):
        dev = feats.device
        cv, ck = _i32_host(cu_vis_h), _i32_host(cu_keep_h)
        R = len(cv) - 1
        Dv = feats.shape[-1]
        code = _dtype_code(feats)
        if cu_vis is None:
            cu_vis = _i32_dev(cv, dev)
        if cu_keep is None:
            cu_keep = _i32_dev(ck, dev)
        Kt = int(ck[-1])
        if kept is None:
            kept = torch.empty(Kt, dtype=torch.int32, device=dev)
        if want_order and order is None:
            order = torch.empty(Kt, dtype=torch.int32, device=dev)
        if want_order and gains is None:
            gains = torch.empty(Kt, dtype=torch.float32, device=dev)
        if ws is None:
            ws = _workspace(lib().diverse_select_workspace(R, _ptr(cv), Dv, code, mode), dev)
        st = lib().diverse_select(R, Dv, code, mode, _ptr(scores), _ptr(feats), _ptr(cu_vis), _ptr(cv),
                                  _ptr(cu_keep), _ptr(ck), _ptr(kept), _ptr(order), _ptr(gains),
                                  _ptr(ws), ws.numel(), _stream(stream))
        if st != LAST_OK:
            raise LastError(st, "diverse_select")
        return kept, order, gains


def diverse_select_similarity(feats: torch.Tensor, cu_vis_h, ws: torch.Tensor, cu_vis=None, stream=None):
    """diverse_select_similarity (Eq. 10): the coverage distances of every request into ws."""
    with _on(stream):
        dev = feats.device
        cv = _i32_host(cu_vis_h)
        if cu_vis is None:
            cu_vis = _i32_dev(cv, dev)
        st = lib().diverse_select_similarity(len(cv) - 1, feats.shape[-1], _dtype_code(feats), _ptr(feats),
                                             _ptr(cu_vis), _ptr(cv), _ptr(ws), ws.numel(), _stream(stream))
        if st != LAST_OK:
            raise LastError(st, "diverse_select_similarity")
        return ws


def diverse_select_pick(scores: torch.Tensor, cu_vis_h, cu_keep_h, ws: torch.Tensor, Dv: int,
                        f_dtype=torch.bfloat16, cu_vis=None, cu_keep=None, kept=None, order=None,
                        gains=None, want_order=True, stream=None):
    """diverse_select_pick (Eq. 9-12) on the distances diverse_select_similarity left in ws:
    returns (kept, order, gains)."""
    with _on(stream):
        dev = scores.device
        cv, ck = _i32_host(cu_vis_h), _i32_host(cu_keep_h)
        code = LAST_BF16 if f_dtype == torch.bfloat16 else LAST_F32
        if cu_vis is None:
            cu_vis = _i32_dev(cv, dev)
        if cu_keep is None:
            cu_keep = _i32_dev(ck, dev)
        Kt = int(ck[-1])
        if kept is None:
            kept = torch.empty(Kt, dtype=torch.int32, device=dev)
        if want_order and order is None:
            order = torch.empty(Kt, dtype=torch.int32, device=dev)
        if want_order and gains is None:
            gains = torch.empty(Kt, dtype=torch.float32, device=dev)
        st = lib().diverse_select_pick(len(cv) - 1, Dv, code, _ptr(scores), _ptr(cu_vis), _ptr(cv), _ptr(cu_keep),
                                       _ptr(ck), _ptr(kept), _ptr(order), _ptr(gains), _ptr(ws), ws.numel(),
                                       _stream(stream))
        if st != LAST_OK:
            raise LastError(st, "diverse_select_pick")
        return kept, order, gains


def gather_kept(feats: torch.Tensor, cu_vis_h, kept: torch.Tensor, cu_keep_h, cu_vis=None,
                cu_keep=None, out=None, stream=None):
    """gather_kept (Eq. 12): the kept rows of feats, byte for byte."""
    with _on(stream):
        dev = feats.device
        cv, ck = _i32_host(cu_vis_h), _i32_host(cu_keep_h)
        R = len(cv) - 1
        Dv = feats.shape[-1]
        if cu_vis is None:
            cu_vis = _i32_dev(cv, dev)
        if cu_keep is None:
            cu_keep = _i32_dev(ck, dev)
        if out is None:
            out = torch.empty((int(ck[-1]), Dv), dtype=feats.dtype, device=dev)
        st = lib().gather_kept(R, Dv, feats.element_size(), _ptr(feats), _ptr(cu_vis), _ptr(cv),
                               _ptr(kept), _ptr(cu_keep), _ptr(ck), _ptr(out), _stream(stream))
        if st != LAST_OK:
            raise LastError(st, "gather_kept")
        return out


def connector_workspace(K: int, Dv: int, Dh: int) -> int:
    return int(lib().last_connector_workspace(int(K), int(Dv), int(Dh)))


def connector(x: torch.Tensor, gamma: torch.Tensor, beta: torch.Tensor, w1: torch.Tensor, b1: torch.Tensor,
              w2: torch.Tensor, b2: torch.Tensor, eps: float = 1e-5, out=None, ws=None, stream=None):
    """last_connector (Sec. 3.4 after Eq. 12, the cloud side): LayerNorm, Linear, GELU, Linear
    on every row of x [K][Dv]; returns out [K][Do] in x's dtype."""
    with _on(stream):
        code = _dtype_code(x)
        if w1.dtype != x.dtype or w2.dtype != x.dtype:
            raise TypeError("x, w1 and w2 must share a dtype")
        K, Dv = x.shape
        Dh, Do = w1.shape[0], w2.shape[0]
        if w1.shape[1] != Dv or w2.shape[1] != Dh:
            raise ValueError("w1 must be [Dh][Dv] and w2 [Do][Dh]")
        for t in (gamma, beta, b1, b2):
            if t.dtype != torch.float32:
                raise TypeError("gamma, beta, b1 and b2 must be float32")
        if gamma.numel() != Dv or beta.numel() != Dv or b1.numel() != Dh or b2.numel() != Do:
            raise ValueError("gamma and beta need Dv entries, b1 Dh and b2 Do")
        if out is None:
            out = torch.empty((K, Do), dtype=x.dtype, device=x.device)
        if ws is None:
            ws = _workspace(lib().last_connector_workspace(K, Dv, Dh), x.device)
        st = lib().last_connector(code, K, Dv, Dh, Do, float(eps), _ptr(x), _ptr(gamma), _ptr(beta), _ptr(w1),
                                  _ptr(b1), _ptr(w2), _ptr(b2), _ptr(out), _ptr(ws), ws.numel(), _stream(stream))
        if st != LAST_OK:
            raise LastError(st, "last_connector")
        return out


def budget(n: int, num: int, den: int) -> int:
    return int(lib().last_budget(int(n), int(num), int(den)))


# ------------------------------------------------------------------ profiling
def profile_enable(on: bool = True) -> None:
    lib().last_profile_enable(1 if on else 0)


def profile_reset() -> None:
    lib().last_profile_reset()


def profile_collect() -> dict:
    """Fold finished kernel timings (call after synchronising). Returns
    {kernel: (launches, total_ms)}."""
    L = lib()
    L.last_profile_collect()
    out = {}
    name = ctypes.c_char_p()
    n = ctypes.c_int64()
    ms = ctypes.c_double()
    for i in range(L.last_profile_count()):
        if L.last_profile_kernel(i, ctypes.byref(name), ctypes.byref(n), ctypes.byref(ms)):
            out[name.value.decode()] = (int(n.value), float(ms.value))
    return out


# ------------------------------------------------------------------ workloads
def to_torch(x: np.ndarray, dtype: str, device) -> torch.Tensor:
    """Upload a workload array (bf16 as uint16 bit patterns, or fp32)."""
    if dtype == "bf16":
        t = torch.from_numpy(np.ascontiguousarray(x).view(np.int16)).view(torch.bfloat16)
    else:
        t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32))
    return t.to(device)


@dataclass
class DeviceWorkload:
    batch: Batch
    q: torch.Tensor
    k: torch.Tensor
    feats: torch.Tensor
    cu_keep_h: np.ndarray
    cu_keep: torch.Tensor
    Dv: int

    @staticmethod
    def upload(wl, device="cuda") -> "DeviceWorkload":
        batch = Batch.make(wl.G, wl.Hq, wl.Hkv, wl.Dh, wl.cu_seqlens, wl.vis_start, wl.cu_vis,
                           scale=wl.scale, device=device)
        return DeviceWorkload(batch=batch, q=to_torch(wl.q, wl.qk_dtype, device),
                              k=to_torch(wl.k, wl.qk_dtype, device),
                              feats=to_torch(wl.feats, wl.f_dtype, device),
                              cu_keep_h=_i32_host(wl.cu_keep), cu_keep=_i32_dev(wl.cu_keep, device),
                              Dv=wl.Dv)
