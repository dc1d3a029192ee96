"""last_token_scores_static, the scores entry point that allocates nothing (its
scratch is a static per-device array): the same results as last_token_scores,
bit for bit, on consecutive calls of different sizes through the C ABI; and
host-side rejection of a batch whose workspace exceeds the array."""
import ctypes

import numpy as np
import pytest
import torch

from paper_2607_27952_amd import last
from paper_2607_27952_amd import workloads as W


class _Sentinel:
    """A host buffer standing in for a device pointer; a rejected call must not touch it."""
    def __init__(self, n=64):
        self.a = np.full(n, 0x5A, np.uint8)
        self.p = self.a.ctypes.data

    def untouched(self):
        return bool(np.all(self.a == 0x5A))


def test_static_scores_reject_oversize_batch_on_the_host():
    # G * Hq * N_total * 4 bytes of visual logits alone exceed the 64 MiB scratch
    R, G, Hq, Hkv, Dh, N = 1, 4, 32, 8, 128, 140000
    cs = np.array([0, N + 2], np.int32)
    cv = np.array([0, N], np.int32)
    vs = np.array([1], np.int32)
    dev = _Sentinel()
    b = last._Batch(R, G, Hq, Hkv, Dh, last.LAST_BF16, 0.0, dev.p, cs.ctypes.data, dev.p, vs.ctypes.data,
                    dev.p, cv.ctypes.data)
    L = last.lib()
    assert L.last_token_scores_workspace(ctypes.byref(b)) > last.STATIC_SCRATCH_BYTES
    q, k, out = _Sentinel(), _Sentinel(), _Sentinel()
    assert L.last_token_scores_static(ctypes.byref(b), q.p, k.p, out.p, None, None) == last.LAST_ERR_WORKSPACE
    # malformed calls are rejected the same way as by last_token_scores
    assert L.last_token_scores_static(ctypes.byref(b), None, k.p, out.p, None, None) == last.LAST_ERR_INVALID
    b.Hq = 30
    assert L.last_token_scores_static(ctypes.byref(b), q.p, k.p, out.p, None, None) == last.LAST_ERR_INVALID
    assert q.untouched() and k.untouched() and out.untouched() and dev.untouched()


def _pair(wl, want_rows):
    dw = last.DeviceWorkload.upload(wl)
    ref = last.token_scores(dw.batch, dw.q, dw.k, want_rows=want_rows)
    got = last.token_scores_static(dw.batch, dw.q, dw.k, want_rows=want_rows)
    torch.cuda.synchronize()
    if want_rows:
        return (ref[0].cpu().numpy(), ref[1].cpu().numpy()), (got[0].cpu().numpy(), got[1].cpu().numpy())
    return (ref.cpu().numpy(),), (got.cpu().numpy(),)


@pytest.mark.gpu
def test_static_scores_match_workspace_scores_on_consecutive_calls():
    """Two calls in a row, the second smaller: each is bit-identical to
    last_token_scores with a caller workspace (the same kernels), and the
    scratch left by the first call does not leak into the second."""
    assert torch.cuda.is_available()
    big = W.tiny(71, R=5, G=2, Hq=8, Hkv=2, Dh=128, n_range=(300, 1500), t_range=(10, 90))
    small = W.tiny(72, R=2, G=1, Hq=4, Hkv=4, Dh=64, n_range=(20, 90), t_range=(3, 9), qk_dtype=W.F32)
    for wl, rows in ((big, False), (small, True)):
        ref, got = _pair(wl, rows)
        for a, b in zip(ref, got):
            assert a.tobytes() == b.tobytes(), f"{wl.name}: static scratch result differs"
        s = ref[0]
        for r in range(wl.R):
            assert abs(s[wl.cu_vis[r]:wl.cu_vis[r + 1]].astype(np.float64).sum() - 1.0) < 1e-5


@pytest.mark.gpu
def test_static_scores_full_size_batch():
    """The 64-request LLaVA-1.5-shaped batch (about 12 MiB of scratch), then a
    one-request call: both bit-identical to the workspace entry point."""
    wl = W.make("c2_llava15")
    ref, got = _pair(wl, False)
    assert ref[0].tobytes() == got[0].tobytes()
    one = wl.subset([5])
    ref, got = _pair(one, False)
    assert ref[0].tobytes() == got[0].tobytes()
