"""CPU oracle for the sparse 3D convolution hot path (Graham, "Sparse 3D
convolutional neural networks", section 1.3).

TEST INFRASTRUCTURE ONLY: imported by ``tests/``, by the package smoke check
and by the benchmark's CPU-baseline leg, never by the GPU library or its Python
binding.  The arithmetic lives in ``scn_oracle.cpp`` (plain C++, std::map /
std::set, naive loops, double precision); this module only marshals numpy
arrays through ctypes.

Feature arrays are float64 and row-major with channels innermost; rulebook
arrays follow the GPU library's layout (int32 coordinates (b, x, y, z),
per-offset pair lists concatenated by offset, int64 offsets).
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass
from typing import Optional, Sequence

import numpy as np

from .build import LIB_PATH, build

STATUS = {0: "ok", 1: "invalid", 2: "range", 3: "duplicate", 4: "overflow"}

# section 1.2, Figure 2: the cubic and square lattices, and the tetrahedral
# and triangular lattices in skewed coordinates (grid x + y (+ z) < m, filter
# offsets kx + ky (+ kz) < f); the 2D lattices use grids with mz = 1
LATTICES = {"cubic": 0, "tetrahedral": 1, "square": 2, "triangular": 3}

_lib = None


class OracleError(RuntimeError):
    def __init__(self, code: int):
        super().__init__(f"oracle status {code} ({STATUS.get(code, '?')})")
        self.code = code
        self.status = STATUS.get(code, "?")


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            build()
        L = ctypes.CDLL(LIB_PATH)
        P = ctypes.c_void_p
        i64, i32 = ctypes.c_int64, ctypes.c_int32
        L.orc_rb_build.argtypes = [P, i64, P, i32, i32, ctypes.POINTER(P)]
        L.orc_rb_build.restype = ctypes.c_int
        L.orc_rb_build_lattice.argtypes = [P, i64, P, i32, i32, i32, ctypes.POINTER(P)]
        L.orc_rb_build_nd.restype = ctypes.c_int
        L.orc_rb_build_nd.argtypes = [P, i64, i32, P, i32, i32, ctypes.POINTER(P)]
        L.orc_rb_info_nd.argtypes = [P, P]
        L.orc_rb_build_lattice.restype = ctypes.c_int
        L.orc_rb_free.argtypes = [P]
        L.orc_rb_info.argtypes = [P, P]
        L.orc_rb_offsets.argtypes = [P, P]
        L.orc_rb_export.argtypes = [P, P, P, P]
        L.orc_conv_fwd.argtypes = [P, P, P, P, P, i32, i32, i32, P, i64, P, P]
        L.orc_conv_bwd.argtypes = [P, P, P, P, P, P, P, i32, i32, i32, P, P, P, P]
        L.orc_maxpool_fwd.argtypes = [P, P, P, i32, P, P, P, P]
        L.orc_maxpool_bwd.argtypes = [P, P, P, P, P, i32, P, P]
        for f in (L.orc_conv_fwd, L.orc_conv_bwd, L.orc_maxpool_fwd, L.orc_maxpool_bwd):
            f.restype = ctypes.c_int
        _lib = L
    return _lib


def _p(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _f64(a) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a, dtype=np.float64))


@dataclass
class RulebookArrays:
    a_in: int
    a_out: int
    n_pairs: int
    K: int
    out_grid: tuple            # (B, mx, my, mz) of the output layer ((B, m_1..m_d) in d dims)
    out_coords: np.ndarray     # int32[a_out][4] (int32[a_out][d + 1] in d dims)
    in_rows: np.ndarray        # int32[n_pairs]
    out_rows: np.ndarray       # int32[n_pairs]
    offsets: np.ndarray        # int64[K+1]


class Rulebook:
    """Owner of an oracle rulebook (H_in, H_out and the per-offset rule lists)
    on one of the lattices of Figure 2, or (``ndim`` given) on the hypercubic
    lattice over sites (b, x_1, .., x_ndim) with grid (B, m_1, .., m_ndim)."""

    def __init__(self, coords: np.ndarray, grid: Sequence[int], f: int, s: int,
                 lattice: str = "cubic", ndim: Optional[int] = None):
        g = np.ascontiguousarray(np.asarray(grid, dtype=np.int64))
        h = ctypes.c_void_p()
        if ndim is None:
            c = np.ascontiguousarray(np.asarray(coords, dtype=np.int32).reshape(-1, 4))
            rc = lib().orc_rb_build_lattice(_p(c), len(c), _p(g), int(f), int(s),
                                            LATTICES[lattice], ctypes.byref(h))
        else:
            if lattice != "cubic":
                raise ValueError("sites of ndim coordinates take the hypercubic lattice")
            c = np.ascontiguousarray(np.asarray(coords, dtype=np.int32).reshape(-1, ndim + 1))
            rc = lib().orc_rb_build_nd(_p(c), len(c), int(ndim), _p(g), int(f), int(s),
                                       ctypes.byref(h))
        if rc != 0:
            raise OracleError(rc)
        self._h = h
        self.f, self.s, self.lattice = int(f), int(s), lattice
        info = np.zeros(10, np.int64)
        lib().orc_rb_info_nd(self._h, _p(info))
        self.a_in, self.a_out, self.n_pairs, self.K = (int(v) for v in info[:4])
        self.ndim = int(info[4])
        self.out_grid = (int(info[5]),) + tuple(int(v) for v in info[6:6 + self.ndim])

    def __del__(self):
        h = getattr(self, "_h", None)
        if h is not None and _lib is not None:
            _lib.orc_rb_free(h)
            self._h = None

    def arrays(self) -> RulebookArrays:
        oc = np.zeros((self.a_out, self.ndim + 1), np.int32)
        ir = np.zeros(self.n_pairs, np.int32)
        orr = np.zeros(self.n_pairs, np.int32)
        off = np.zeros(self.K + 1, np.int64)
        lib().orc_rb_offsets(self._h, _p(off))
        lib().orc_rb_export(self._h, _p(oc), _p(ir), _p(orr))
        return RulebookArrays(self.a_in, self.a_out, self.n_pairs, self.K, self.out_grid,
                              oc, ir, orr, off)


def _check(rc: int):
    if rc != 0:
        raise OracleError(rc)


def conv_fwd(rb: Rulebook, x, g_in, W, bias, relu: bool = False, rows=None):
    """Returns (y, g_out) in float64.  ``rows`` restricts y to those output rows."""
    x, g_in, W = _f64(x), _f64(g_in), _f64(W)
    K, Cin, Cout = W.shape
    assert K == rb.K and x.shape[1] == Cin and g_in.shape == (Cin,)
    b = None if bias is None else _f64(bias)
    r = None if rows is None else np.ascontiguousarray(np.asarray(rows, np.int64))
    n = rb.a_out if r is None else len(r)
    y = np.zeros((n, Cout), np.float64)
    g = np.zeros(Cout, np.float64)
    _check(lib().orc_conv_fwd(rb._h, _p(x), _p(g_in), _p(W), _p(b), Cin, Cout, int(relu),
                              _p(r), 0 if r is None else len(r), _p(y), _p(g)))
    return y, g


def conv_bwd(rb: Rulebook, x, g_in, W, bias, dy, dg_out=None, relu: bool = False):
    """Returns dict(dx, dg_in, dW, dbias) in float64."""
    x, g_in, W, dy = _f64(x), _f64(g_in), _f64(W), _f64(dy)
    K, Cin, Cout = W.shape
    assert dy.shape == (rb.a_out, Cout)
    b = None if bias is None else _f64(bias)
    dg = None if dg_out is None else _f64(dg_out)
    out = dict(dx=np.zeros((rb.a_in, Cin)), dg_in=np.zeros(Cin), dW=np.zeros((K, Cin, Cout)),
               dbias=np.zeros(Cout))
    _check(lib().orc_conv_bwd(rb._h, _p(x), _p(g_in), _p(W), _p(b), _p(dy), _p(dg), Cin, Cout,
                              int(relu), _p(out["dx"]), _p(out["dg_in"]), _p(out["dW"]),
                              _p(out["dbias"])))
    return out


def maxpool_fwd(rb: Rulebook, x, g_in):
    """Returns (y, g_out, arg_k int32[a_out][C], arg_inactive uint8[a_out][C])."""
    x, g_in = _f64(x), _f64(g_in)
    C = x.shape[1]
    y = np.zeros((rb.a_out, C))
    g = np.zeros(C)
    ak = np.zeros((rb.a_out, C), np.int32)
    ai = np.zeros((rb.a_out, C), np.uint8)
    _check(lib().orc_maxpool_fwd(rb._h, _p(x), _p(g_in), C, _p(y), _p(g), _p(ak), _p(ai)))
    return y, g, ak, ai


def maxpool_bwd(rb: Rulebook, x, g_in, dy, dg_out=None):
    """Returns (dx, dg_in) in float64."""
    x, g_in, dy = _f64(x), _f64(g_in), _f64(dy)
    C = x.shape[1]
    dg = None if dg_out is None else _f64(dg_out)
    dx = np.zeros((rb.a_in, C))
    dgi = np.zeros(C)
    _check(lib().orc_maxpool_bwd(rb._h, _p(x), _p(g_in), _p(dy), _p(dg), C, _p(dx), _p(dgi)))
    return dx, dgi
