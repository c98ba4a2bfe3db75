"""Comparison helpers for GPU-vs-oracle parity tests (test infrastructure)."""
import numpy as np
import torch

# spec tolerance for fp32 outputs (log-probs, scores, log-likelihoods):
#   |gpu - oracle| <= 1e-5 * max(1, |oracle|)
RTOL = 1e-5


def to_np(t):
    if isinstance(t, torch.Tensor):
        t = t.detach().cpu()
        if t.dtype == torch.bfloat16:
            return t.view(torch.int16).numpy().view(np.uint16)
        return t.numpy()
    return np.asarray(t)


def assert_close(gpu, ref, what, tol=RTOL):
    gpu = np.asarray(gpu, np.float64)
    ref = np.asarray(ref, np.float64)
    assert gpu.shape == ref.shape, f"{what}: shape {gpu.shape} vs {ref.shape}"
    both_inf = np.isinf(gpu) & np.isinf(ref) & (np.sign(gpu) == np.sign(ref))
    with np.errstate(invalid="ignore"):
        err = np.where(both_inf, 0.0, np.abs(gpu - ref))
    bound = tol * np.maximum(1.0, np.where(np.isinf(ref), 1.0, np.abs(ref)))
    bad = ~(err <= bound)
    if bad.any():
        i = np.argwhere(bad)[0]
        raise AssertionError(f"{what}: {bad.sum()} of {bad.size} outside tolerance; first at "
                             f"{tuple(i)}: gpu {gpu[tuple(i)]!r} oracle {ref[tuple(i)]!r}; "
                             f"max err {np.nanmax(err):.3e}")


def assert_equal(gpu, ref, what):
    gpu = np.asarray(gpu)
    ref = np.asarray(ref)
    assert gpu.shape == ref.shape, f"{what}: shape {gpu.shape} vs {ref.shape}"
    bad = gpu != ref
    if bad.any():
        i = np.argwhere(bad)[0]
        raise AssertionError(f"{what}: {bad.sum()} of {bad.size} differ; first at {tuple(i)}: "
                             f"gpu {gpu[tuple(i)]!r} oracle {ref[tuple(i)]!r}")
