"""MI355X-native LAST token-selection path (arXiv 2607.27952).

The compute lives in ``liblast.so`` (hand-written gfx950 HIP kernels behind a
C ABI, declared in ``include/last.h``). ``paper_2607_27952_amd.last`` is the
thin ctypes binding over it; ``paper_2607_27952_amd.workloads`` draws seeded
synthetic inputs. Nothing is loaded at import time.
"""
__all__ = ["last", "workloads"]
