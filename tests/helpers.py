"""Shared helpers for the GPU parity tests: device conversion and the
tolerance rule for fp32 results against the fp64 oracle.

Tolerance.  The library computes in fp32 (MFMA with fp32 accumulation); the
oracle accumulates the same fp32 inputs in fp64.  A result that is a sum of
terms t_i carries an fp32 rounding error that grows with the size of the
terms, not with the size of the (possibly cancelling) sum, so the bound is
    |gpu - ref| <= ATOL + RTOL * max(|ref|, sigma),   sigma = sqrt(sum_i t_i^2),
with ATOL = 1e-5 and RTOL = 1e-4.  sigma is computed by the oracle itself: the
forward and backward maps are sums of products, and (a*b)^2 = a^2 * b^2, so
running the oracle on element-wise squared inputs (without ReLU, with the
ReLU mask already applied to the output gradient) returns sum_i t_i^2.
"""
from __future__ import annotations

import numpy as np
import torch

ATOL = 1e-5
RTOL = 1e-4


def dev(a, dtype=None) -> torch.Tensor:
    t = torch.from_numpy(np.ascontiguousarray(a))
    if dtype is not None:
        t = t.to(dtype)
    return t.to("cuda")


def host(t: torch.Tensor) -> np.ndarray:
    torch.cuda.synchronize()
    return t.detach().cpu().numpy()


def assert_close(name: str, gpu, ref, sigma=None, atol=ATOL, rtol=RTOL):
    gpu = np.asarray(gpu, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert gpu.shape == ref.shape, f"{name}: shape {gpu.shape} vs {ref.shape}"
    if gpu.size == 0:
        return
    scale = np.abs(ref) if sigma is None else np.maximum(np.abs(ref), np.asarray(sigma))
    err = np.abs(gpu - ref)
    bound = atol + rtol * scale
    bad = ~(err <= bound)
    plain = int(np.sum(~(err <= atol + rtol * np.abs(ref))))
    if bad.any():
        i = np.unravel_index(np.argmax(err - bound), err.shape)
        raise AssertionError(
            f"{name}: {int(bad.sum())}/{err.size} outside tolerance "
            f"(worst at {i}: gpu={gpu[i]!r} ref={ref[i]!r} bound={bound[i]:.3g}); "
            f"plain allclose failures {plain}")
    return plain


def keys_of(coords: np.ndarray, grid) -> np.ndarray:
    c = np.asarray(coords, dtype=np.int64)
    B, mx, my, mz = (int(v) for v in grid)
    return ((c[:, 0] * mz + c[:, 3]) * my + c[:, 2]) * mx + c[:, 1]
