"""Shared helpers for the GPU parity tests: device conversion and the
tolerance rules for fp32 results against the fp64 oracle.

Tolerance.  The library computes in fp32 (MFMA with fp32 accumulation); the
oracle accumulates the same fp32 inputs in fp64.  The bar is 1e-4 relative
and 1e-5 absolute:

* Per-site results (a row of y, dx, a pooling dx row, the ground state g_out)
  are compared with the plain rule  |gpu - ref| <= ATOL + RTOL * |ref|
  (``assert_site``).
* Reductions over every pair of a layer (dW, dbias, dg_in) are sums of up to
  millions of terms t_i.  Their fp32 rounding error grows with the terms, not
  with the (possibly cancelling) sum, so they are compared with
      |gpu - ref| <= ATOL + RTOL * max(|ref|, sigma),   sigma = sqrt(sum_i t_i^2)
  (``assert_reduction``).  sigma is computed by the oracle itself: these maps
  are sums of products, and (a*b)^2 = a^2 * b^2, so running the oracle on
  element-wise squared inputs (ReLU mask already applied to the output
  gradient) returns sum_i t_i^2.

Every comparison also counts its failures under the plain rule, whichever
rule it enforces, and records them in ``REPORT``; tests/conftest.py prints
the totals at the end of the session (and writes them as JSON to the file
named by $SCN_PARITY_REPORT).

ReLU.  The backward's ReLU mask is a decision taken in floating point.  The
parity tests give the library's backward the oracle's forward output
(rounded to fp32) as its post-activation input, so both sides take the mask
from the same value: y_ref > 0 in fp64 and fp32(y_ref) > 0 agree unless
0 < y_ref < 2^-149, which ``relu_inputs`` rules out for each case.
"""
from __future__ import annotations

import os

import numpy as np
import torch

ATOL = 1e-5
RTOL = 1e-4

# (test id, name, kind, elements, plain-rule failures, failures of the enforced rule)
REPORT: list = []


def _test_id() -> str:
    t = os.environ.get("PYTEST_CURRENT_TEST", "")
    return t.split(" ")[0]


def dev(a, dtype=None) -> torch.Tensor:
    t = torch.from_numpy(np.ascontiguousarray(a))
    if dtype is not None:
        t = t.to(dtype)
    return t.to("cuda")


def host(t: torch.Tensor) -> np.ndarray:
    torch.cuda.synchronize()
    return t.detach().cpu().numpy()


def _compare(name, kind, gpu, ref, sigma, atol, rtol):
    gpu = np.asarray(gpu, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert gpu.shape == ref.shape, f"{name}: shape {gpu.shape} vs {ref.shape}"
    if gpu.size == 0:
        REPORT.append((_test_id(), name, kind, 0, 0, 0))
        return 0
    err = np.abs(gpu - ref)
    plain_bound = atol + rtol * np.abs(ref)
    plain = int(np.sum(~(err <= plain_bound)))
    bound = plain_bound if sigma is None else atol + rtol * np.maximum(np.abs(ref),
                                                                       np.asarray(sigma))
    bad = ~(err <= bound)
    REPORT.append((_test_id(), name, kind, int(err.size), plain, int(bad.sum())))
    if bad.any():
        i = np.unravel_index(np.argmax(err - bound), err.shape)
        raise AssertionError(
            f"{name}: {int(bad.sum())}/{err.size} outside tolerance "
            f"(worst at {i}: gpu={gpu[i]!r} ref={ref[i]!r} bound={bound[i]:.3g}); "
            f"plain-rule failures {plain}")
    return plain


def assert_site(name: str, gpu, ref, atol=ATOL, rtol=RTOL) -> int:
    """Per-site result under the plain rule; returns its failure count (0)."""
    return _compare(name, "site", gpu, ref, None, atol, rtol)


def assert_reduction(name: str, gpu, ref, sigma, atol=ATOL, rtol=RTOL) -> int:
    """Reduction over pairs under the sigma rule; returns the plain-rule
    failure count (reported, not enforced)."""
    assert sigma is not None, name
    return _compare(name, "reduction", gpu, ref, sigma, atol, rtol)


def assert_exact(name: str, gpu, ref) -> None:
    """Bit-exact comparison (rulebooks, pooling values, argmax)."""
    gpu = np.asarray(gpu)
    ref = np.asarray(ref)
    assert gpu.shape == ref.shape, f"{name}: shape {gpu.shape} vs {ref.shape}"
    ok = np.array_equal(gpu, ref)
    REPORT.append((_test_id(), name, "exact", int(gpu.size), 0 if ok else 1, 0 if ok else 1))
    assert ok, f"{name}: not bit-exact ({int(np.sum(gpu != ref))} of {gpu.size} differ)"


def relu_inputs(y_ref, g_ref):
    """The oracle's post-activation y and g_out as fp32 device tensors, the
    ReLU-mask inputs of the library's backward (see the module docstring)."""
    y = np.asarray(y_ref, np.float64)
    g = np.asarray(g_ref, np.float64)
    tiny = 2.0 ** -149
    assert not np.any((y > 0) & (y < tiny)) and not np.any((g > 0) & (g < tiny))
    return dev(y.astype(np.float32)), dev(g.astype(np.float32))


def kink_flips(y_gpu, pre_ref) -> int:
    """Entries where the library's own forward and the oracle disagree on the
    ReLU decision (reported; the backward comparison does not depend on it)."""
    return int(np.sum((np.asarray(y_gpu) > 0) != (np.asarray(pre_ref) > 0)))


def keys_of(coords: np.ndarray, grid) -> np.ndarray:
    c = np.asarray(coords, dtype=np.int64)
    B, mx, my, mz = (int(v) for v in grid)
    return ((c[:, 0] * mz + c[:, 3]) * my + c[:, 2]) * mx + c[:, 1]


def sq(a):
    """Element-wise square in fp64 (inputs of the oracle's sigma runs)."""
    return None if a is None else np.asarray(a, np.float64) ** 2


def conv_parity(scn, g, o, x, g_in, W, bias, relu, seed):
    """One convolution layer, forward and backward, against the oracle on
    the same inputs: y and g_out, then dx (per-site), dW, dbias and dg_in
    (reductions) for a seeded dy ~ U[-1, 1] and dg_out ~ U[-1, 1].  Returns
    the oracle's (y, g_out)."""
    import oracle
    from gen import stream_rng

    Cout = W.shape[2]
    bd = None if bias is None else dev(bias)
    y_ref, go_ref = oracle.conv_fwd(o, x, g_in, W, bias, relu=relu)
    yd, god = scn.conv_fwd(g, dev(x), dev(g_in), dev(W), bd, relu=relu)
    assert_site("y", host(yd), y_ref)
    assert_site("g_out", host(god), go_ref)
    pre_ref, gpre_ref = (oracle.conv_fwd(o, x, g_in, W, bias, relu=False) if relu
                         else (y_ref, go_ref))
    if relu:
        assert kink_flips(host(yd), pre_ref) <= 1e-4 * pre_ref.size + 1
    rng = stream_rng(seed, 2)
    dy = rng.uniform(-1, 1, size=(g.a_out, Cout)).astype(np.float32)
    dg = rng.uniform(-1, 1, size=Cout).astype(np.float32)
    ref = oracle.conv_bwd(o, x, g_in, W, bias, dy, dg, relu=relu)
    dyb = dy * (pre_ref > 0) if relu else dy
    dgb = dg * (gpre_ref > 0) if relu else dg
    sig = {k: np.sqrt(v) for k, v in
           oracle.conv_bwd(o, sq(x), sq(g_in), sq(W), None, sq(dyb), sq(dgb)).items()}
    yr, gr = relu_inputs(y_ref, go_ref) if relu else (None, None)
    out = scn.conv_bwd(g, dev(x), dev(g_in), dev(W), yr, gr, dev(dy), dev(dg), relu=relu)
    assert_site("dx", host(out["dx"]), ref["dx"])
    for k in ("dW", "dbias", "dg_in"):
        assert_reduction(k, host(out[k]), ref[k], sig[k])
    return y_ref, go_ref


def pool_parity(scn, g, o, x, g_in, rng, overlapping):
    """One max-pooling layer against the oracle on the same inputs: values,
    argmax and (without overlapping windows) dx bit-exact; dx summed over
    overlapping windows per-site; dg_in a reduction."""
    import oracle

    C = x.shape[1]
    y_ref, go_ref, ak_ref, _ = oracle.maxpool_fwd(o, x, g_in)
    yd, god, am = scn.maxpool_fwd(g, dev(x), dev(g_in))
    assert_exact("pool y", host(yd), y_ref.astype(np.float32))
    assert_exact("pool g_out", host(god), go_ref.astype(np.float32))
    assert_exact("argmax", host(am).astype(np.int32), ak_ref)
    dy = rng.uniform(-1, 1, size=(g.a_out, C)).astype(np.float32)
    dg = rng.uniform(-1, 1, size=C).astype(np.float32)
    dx_ref, dgi_ref = oracle.maxpool_bwd(o, x, g_in, dy, dg)
    dxd, dgid = scn.maxpool_bwd(g, am, dev(dy), dev(dg))
    if not overlapping:
        # every input has at most one window: dx is a copy of dy entries
        assert_exact("pool dx", host(dxd), dx_ref.astype(np.float32))
    else:
        # an input sums dy over up to 8 windows (fp32, fixed order)
        assert_site("pool dx", host(dxd), dx_ref)
    sig = np.sqrt(oracle.maxpool_bwd(o, x, g_in, sq(dy), sq(dg))[1])
    assert_reduction("pool dg_in", host(dgid), dgi_ref, sig)


def definition_rulebook(coords, grid, f, s):
    """(out_coords in key order, offsets, in_rows, out_rows) of a cubic
    filter of size f and stride s, from the definition."""
    c = np.asarray(coords, np.int64)
    B, mx, my, mz = (int(v) for v in grid)
    ox, oy, oz = ((m - f) // s + 1 if m >= f else 0 for m in (mx, my, mz))
    K = f ** 3
    if min(ox, oy, oz) == 0:
        z = np.zeros(0, np.int32)
        return np.zeros((0, 4), np.int32), np.zeros(K + 1, np.int64), z, z
    row = np.full((B, mz, my, mx), -1, np.int32)
    row[c[:, 0], c[:, 3], c[:, 2], c[:, 1]] = np.arange(len(c), dtype=np.int32)
    offs = [(kx, ky, kz) for kz in range(f) for ky in range(f) for kx in range(f)]

    def window(kx, ky, kz):  # [b, oz, oy, ox] -> row of site s*o + k
        return row[:, kz:kz + s * (oz - 1) + 1:s, ky:ky + s * (oy - 1) + 1:s,
                   kx:kx + s * (ox - 1) + 1:s]

    active = np.zeros((B, oz, oy, ox), bool)
    for k in offs:
        active |= window(*k) >= 0
    b, z, y, x = np.nonzero(active)  # C order: ascending key
    out_coords = np.stack([b, x, y, z], axis=1).astype(np.int32)
    in_rows, out_rows, offsets = [], [], [0]
    for k in offs:
        r = window(*k)[active]
        hit = np.nonzero(r >= 0)[0]
        in_rows.append(r[hit])
        out_rows.append(hit.astype(np.int32))
        offsets.append(offsets[-1] + len(hit))
    return (out_coords, np.array(offsets, np.int64), np.concatenate(in_rows),
            np.concatenate(out_rows))
