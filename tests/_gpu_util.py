"""Helpers for GPU tests: torch transfers and the element-wise tolerance."""
import numpy as np

ATOL = 2e-3      # O max-abs bound
RTOL = 1e-2      # O max-rel bound (|gpu - ref| <= ATOL + RTOL*|ref|)
LSE_ATOL = 2e-3


def to_gpu(a):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def to_np(t):
    return t.detach().cpu().numpy()


def check_close(got, ref, atol=ATOL, rtol=RTOL, what="O"):
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    err = np.abs(got - ref)
    bad = err > atol + rtol * np.abs(ref)
    assert not bad.any(), (f"{what}: {bad.sum()} elements out of tolerance; max abs err "
                           f"{err.max():.3e} at ref {ref.ravel()[err.argmax()]:.4f}")
    return float(err.max())
