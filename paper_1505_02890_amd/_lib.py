"""ctypes binding of ``libscn.so`` (the C ABI declared in ``include/scn.h``).

This module only marshals arguments: it checks tensor shapes, dtypes and
devices, allocates the caller-owned outputs and workspaces with PyTorch, and
passes raw device pointers plus the current HIP stream to the library.  Every
step of the computation runs in the library's HIP kernels.  If the library has
not been built the first call raises; there is no fallback.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

import numpy as np
import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.environ.get("SCN_LIB") or os.path.join(HERE, "libscn.so")

SCN_RELU = 1
# section 1.2, Figure 2: the cubic and square lattices, and the tetrahedral and
# triangular lattices in skewed coordinates (2D lattices: grids with mz = 1)
LATTICES = {"cubic": 0, "tetrahedral": 1, "square": 2, "triangular": 3}
STATUS = {0: "ok", 1: "invalid", 2: "range", 3: "duplicate", 4: "overflow",
          5: "unsupported", 6: "workspace", 7: "hip", 8: "nomem"}

EXPORTED = (
    "scn_rulebook_build", "scn_rulebook_build_lattice", "scn_rulebook_build_nd",
    "scn_rulebook_build_next",
    "scn_rulebook_build_chain",
    "scn_rulebook_get_info", "scn_rulebook_out_coords",
    "scn_rulebook_in_rows", "scn_rulebook_out_rows", "scn_rulebook_offsets",
    "scn_rulebook_export", "scn_rulebook_free", "scn_conv_fwd",
    "scn_conv_bwd_workspace_bytes", "scn_conv_bwd", "scn_maxpool_fwd",
    "scn_maxpool_bwd_workspace_bytes", "scn_maxpool_bwd", "scn_set_allocator",
    "scn_set_dense_forward", "scn_last_error", "scn_version", "scn_conv_fwd_noalloc",
    "scn_conv_fwd_noalloc_max_bytes", "scn_set_kernel_timer", "scn_ceiling_copy",
    "scn_ceiling_mfma_f32",
)

_ALLOC_FN = ctypes.CFUNCTYPE(ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p, ctypes.c_void_p)
_FREE_FN = ctypes.CFUNCTYPE(None, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p)


class ScnError(RuntimeError):
    def __init__(self, code: int, where: str, message: str):
        super().__init__(f"{where}: status {code} ({STATUS.get(code, '?')}): {message}")
        self.code = code
        self.status = STATUS.get(code, "?")


class _Info(ctypes.Structure):
    _fields_ = [("a_in", ctypes.c_int64), ("a_out", ctypes.c_int64),
                ("n_pairs", ctypes.c_int64), ("K", ctypes.c_int32),
                ("filter", ctypes.c_int32), ("stride", ctypes.c_int32),
                ("input_sorted", ctypes.c_int32), ("in_grid", ctypes.c_int64 * 4),
                ("out_grid", ctypes.c_int64 * 4), ("lattice", ctypes.c_int32),
                ("dense_view", ctypes.c_int32), ("ndim", ctypes.c_int32),
                ("keyed", ctypes.c_int32), ("in_grid_nd", ctypes.c_int64 * 5),
                ("out_grid_nd", ctypes.c_int64 * 5)]


_lib = None


def lib() -> ctypes.CDLL:
    """Load libscn.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(
            f"HIP library {LIB_PATH} is missing: build it with "
            "`python -m paper_1505_02890_amd.build` (or __graft_entry__.build())")
    L = ctypes.CDLL(LIB_PATH)
    P, i32, i64, u32, sz = (ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_uint32,
                            ctypes.c_size_t)
    st = ctypes.c_int
    sig = {
        "scn_rulebook_build": (st, [P, i64, P, i32, i32, P, ctypes.POINTER(P)]),
        "scn_rulebook_build_lattice": (st, [P, i64, P, i32, i32, i32, P, ctypes.POINTER(P)]),
        "scn_rulebook_build_nd": (st, [P, i64, i32, P, i32, i32, P, ctypes.POINTER(P)]),
        "scn_rulebook_build_next": (st, [P, i32, i32, P, ctypes.POINTER(P)]),
        "scn_rulebook_build_chain": (st, [P, i64, P, i32, i32, P, P, P, ctypes.POINTER(P)]),
        "scn_rulebook_get_info": (st, [P, ctypes.POINTER(_Info)]),
        "scn_rulebook_out_coords": (P, [P]),
        "scn_rulebook_in_rows": (P, [P]),
        "scn_rulebook_out_rows": (P, [P]),
        "scn_rulebook_offsets": (ctypes.POINTER(ctypes.c_int64), [P]),
        "scn_rulebook_export": (st, [P, P, P, P, P]),
        "scn_rulebook_free": (None, [P]),
        "scn_conv_fwd": (st, [P, P, P, P, P, i32, i32, u32, P, P, P]),
        "scn_conv_fwd_noalloc": (st, [P, P, P, P, P, i32, i32, u32, P, P, P]),
        "scn_conv_fwd_noalloc_max_bytes": (sz, []),
        "scn_set_kernel_timer": (st, [P]),
        "scn_ceiling_copy": (st, [P, P, sz, P]),
        "scn_ceiling_mfma_f32": (st, [P, i64, i32, ctypes.POINTER(ctypes.c_double), P]),
        "scn_conv_bwd_workspace_bytes": (sz, [P, i32, i32, u32]),
        "scn_conv_bwd": (st, [P, P, P, P, P, P, P, P, i32, i32, u32, P, P, P, P, P, sz, P]),
        "scn_maxpool_fwd": (st, [P, P, P, i32, P, P, P, P]),
        "scn_maxpool_bwd_workspace_bytes": (sz, [P, i32]),
        "scn_maxpool_bwd": (st, [P, P, P, P, i32, P, P, P, sz, P]),
        "scn_set_allocator": (None, [_ALLOC_FN, _FREE_FN, P]),
        "scn_set_dense_forward": (st, [i64, i32]),
        "scn_last_error": (ctypes.c_char_p, []),
        "scn_version": (ctypes.c_char_p, []),
    }
    for name, (res, args) in sig.items():
        f = getattr(L, name)
        f.restype = res
        f.argtypes = args
    _lib = L
    return L


def _check(rc: int, where: str):
    if rc != 0:
        msg = lib().scn_last_error().decode(errors="replace")
        raise ScnError(rc, where, msg)


def _stream() -> int:
    return torch.cuda.current_stream().cuda_stream


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _dev_tensor(t: torch.Tensor, dtype, shape, name: str) -> torch.Tensor:
    if not isinstance(t, torch.Tensor) or t.device.type != "cuda":
        raise TypeError(f"{name} must be a CUDA (HIP) tensor")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return t


class Rulebook:
    """Owner of a device rulebook built by ``scn_rulebook_build_lattice``
    (or ``scn_rulebook_build_nd`` when ``ndim`` is given).

    ``coords`` is a device int32 [n, 4] tensor of (b, x, y, z) rows; ``grid``
    is (B, mx, my, mz); ``lattice`` is "cubic", "tetrahedral", "square" or
    "triangular".  With ``ndim``, coords is [n, ndim + 1] rows (b, x_1, ..)
    and grid (B, m_1, .., m_ndim) on the hypercubic lattice.  Attributes
    mirror ``scn_rulebook_info``.
    """

    def __init__(self, coords: Optional[torch.Tensor], grid: Sequence[int], filter: int,
                 stride: int, lattice: str = "cubic", prev: Optional["Rulebook"] = None,
                 ndim: Optional[int] = None):
        h = ctypes.c_void_p()
        if ndim is not None:
            n = int(coords.shape[0]) if coords.dim() == 2 else -1
            _dev_tensor(coords, torch.int32, (n, ndim + 1), "coords")
            if lattice != "cubic":
                raise ValueError("sites of ndim coordinates take the hypercubic lattice")
            g = np.ascontiguousarray(np.asarray(grid, dtype=np.int64).reshape(ndim + 1))
            _check(lib().scn_rulebook_build_nd(
                _ptr(coords), n, int(ndim), g.ctypes.data_as(ctypes.c_void_p), int(filter),
                int(stride), ctypes.c_void_p(_stream()), ctypes.byref(h)),
                "scn_rulebook_build_nd")
            device = coords.device
        elif prev is not None:
            # the layer after prev: its sites are prev's active outputs
            _check(lib().scn_rulebook_build_next(prev.handle, int(filter), int(stride),
                                                 ctypes.c_void_p(_stream()), ctypes.byref(h)),
                   "scn_rulebook_build_next")
            device = prev.device
        else:
            n = int(coords.shape[0]) if coords.dim() == 2 else -1
            _dev_tensor(coords, torch.int32, (n, 4), "coords")
            if lattice not in LATTICES:
                raise ValueError(f"lattice must be one of {sorted(LATTICES)}, got {lattice!r}")
            g = np.ascontiguousarray(np.asarray(grid, dtype=np.int64).reshape(4))
            _check(lib().scn_rulebook_build_lattice(
                _ptr(coords), n, g.ctypes.data_as(ctypes.c_void_p), int(filter), int(stride),
                LATTICES[lattice], ctypes.c_void_p(_stream()), ctypes.byref(h)),
                "scn_rulebook_build_lattice")
            device = coords.device
        self._adopt(h, device)

    @classmethod
    def _from_handle(cls, h: ctypes.c_void_p, device) -> "Rulebook":
        rb = cls.__new__(cls)
        rb._adopt(h, device)
        return rb

    def _adopt(self, h: ctypes.c_void_p, device) -> None:
        self._h = h
        self.device = device
        info = _Info()
        _check(lib().scn_rulebook_get_info(self._h, ctypes.byref(info)), "scn_rulebook_get_info")
        self.a_in, self.a_out, self.n_pairs = int(info.a_in), int(info.a_out), int(info.n_pairs)
        self.K, self.filter, self.stride = int(info.K), int(info.filter), int(info.stride)
        self.input_sorted = bool(info.input_sorted)
        self.dense_view = bool(info.dense_view)
        self.lattice = {v: k for k, v in LATTICES.items()}[int(info.lattice)]
        self.ndim, self.keyed = int(info.ndim), bool(info.keyed)
        self.in_grid = tuple(int(v) for v in info.in_grid_nd[:self.ndim + 1])
        self.out_grid = tuple(int(v) for v in info.out_grid_nd[:self.ndim + 1])
        off = lib().scn_rulebook_offsets(self._h)
        self.offsets = np.array([off[k] for k in range(self.K + 1)], dtype=np.int64)

    @property
    def handle(self):
        return self._h

    def close(self):
        h = getattr(self, "_h", None)
        if h is not None and h.value and _lib is not None:
            _lib.scn_rulebook_free(h)
        self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def export(self):
        """(out_coords int32[a_out, ndim+1], in_rows int32[P], out_rows int32[P]) on the
        device."""
        oc = torch.empty((self.a_out, self.ndim + 1), dtype=torch.int32, device=self.device)
        ir = torch.empty(self.n_pairs, dtype=torch.int32, device=self.device)
        orr = torch.empty(self.n_pairs, dtype=torch.int32, device=self.device)
        _check(lib().scn_rulebook_export(self._h, _ptr(oc), _ptr(ir), _ptr(orr),
                                         ctypes.c_void_p(_stream())), "scn_rulebook_export")
        return oc, ir, orr

    def out_coords(self) -> torch.Tensor:
        oc = torch.empty((self.a_out, self.ndim + 1), dtype=torch.int32, device=self.device)
        _check(lib().scn_rulebook_export(self._h, _ptr(oc), None, None,
                                         ctypes.c_void_p(_stream())), "scn_rulebook_export")
        return oc


def build_rulebook(coords: torch.Tensor, grid: Sequence[int], filter: int, stride: int,
                   lattice: str = "cubic") -> Rulebook:
    return Rulebook(coords, grid, filter, stride, lattice)


def build_rulebook_nd(coords: torch.Tensor, grid: Sequence[int], filter: int,
                      stride: int) -> Rulebook:
    """Hypercubic rulebook over sites of ndim = len(grid) - 1 coordinates
    (keyed builder: sorted keys and hash tables)."""
    return Rulebook(coords, grid, filter, stride, ndim=len(grid) - 1)


def next_rulebook(prev: Rulebook, filter: int, stride: int) -> Rulebook:
    """The rulebook of the layer after `prev` (its sites are prev's active
    outputs, on prev's output grid and lattice)."""
    return Rulebook(None, prev.out_grid, filter, stride, prev.lattice, prev=prev)


def conv_fwd(rb: Rulebook, x: torch.Tensor, g_in: torch.Tensor, W: torch.Tensor,
             bias: Optional[torch.Tensor] = None, relu: bool = False,
             y: Optional[torch.Tensor] = None, g_out: Optional[torch.Tensor] = None,
             noalloc: bool = False):
    """Returns (y [a_out, Cout], g_out [Cout]); y and g_out are allocated here
    unless given.  noalloc=True calls scn_conv_fwd_noalloc (the library then
    allocates nothing)."""
    K, Cin, Cout = (int(v) for v in W.shape)
    if K != rb.K:
        raise ValueError(f"W has {K} offsets, rulebook has {rb.K}")
    _dev_tensor(W, torch.float32, (K, Cin, Cout), "W")
    _dev_tensor(x, torch.float32, (rb.a_in, Cin), "x")
    _dev_tensor(g_in, torch.float32, (Cin,), "g_in")
    if bias is not None:
        _dev_tensor(bias, torch.float32, (Cout,), "bias")
    if y is None:
        y = torch.empty((rb.a_out, Cout), dtype=torch.float32, device=x.device)
    _dev_tensor(y, torch.float32, (rb.a_out, Cout), "y")
    if g_out is None:
        g_out = torch.empty(Cout, dtype=torch.float32, device=x.device)
    _dev_tensor(g_out, torch.float32, (Cout,), "g_out")
    name = "scn_conv_fwd_noalloc" if noalloc else "scn_conv_fwd"
    _check(getattr(lib(), name)(rb.handle, _ptr(x), _ptr(g_in), _ptr(W), _ptr(bias), Cin, Cout,
                                SCN_RELU if relu else 0, _ptr(y), _ptr(g_out),
                                ctypes.c_void_p(_stream())), name)
    return y, g_out


def conv_bwd_workspace(rb: Rulebook, Cin: int, Cout: int, relu: bool) -> torch.Tensor:
    n = lib().scn_conv_bwd_workspace_bytes(rb.handle, Cin, Cout, SCN_RELU if relu else 0)
    return torch.empty(max(int(n), 1), dtype=torch.uint8, device=rb.device)


def conv_bwd(rb: Rulebook, x: torch.Tensor, g_in: torch.Tensor, W: torch.Tensor,
             y: Optional[torch.Tensor], g_out: Optional[torch.Tensor], dy: torch.Tensor,
             dg_out: Optional[torch.Tensor] = None, relu: bool = False,
             need=("dx", "dg_in", "dW", "dbias"), ws: Optional[torch.Tensor] = None):
    """Returns a dict with the requested gradients among dx, dg_in, dW, dbias."""
    K, Cin, Cout = (int(v) for v in W.shape)
    _dev_tensor(W, torch.float32, (rb.K, Cin, Cout), "W")
    _dev_tensor(x, torch.float32, (rb.a_in, Cin), "x")
    _dev_tensor(g_in, torch.float32, (Cin,), "g_in")
    _dev_tensor(dy, torch.float32, (rb.a_out, Cout), "dy")
    if relu:
        _dev_tensor(y, torch.float32, (rb.a_out, Cout), "y")
        _dev_tensor(g_out, torch.float32, (Cout,), "g_out")
    if dg_out is not None:
        _dev_tensor(dg_out, torch.float32, (Cout,), "dg_out")
    dev = x.device
    out = {}
    if "dx" in need:
        out["dx"] = torch.empty((rb.a_in, Cin), dtype=torch.float32, device=dev)
    if "dg_in" in need:
        out["dg_in"] = torch.empty(Cin, dtype=torch.float32, device=dev)
    if "dW" in need:
        out["dW"] = torch.empty((K, Cin, Cout), dtype=torch.float32, device=dev)
    if "dbias" in need:
        out["dbias"] = torch.empty(Cout, dtype=torch.float32, device=dev)
    if ws is None:
        ws = conv_bwd_workspace(rb, Cin, Cout, relu)
    _check(lib().scn_conv_bwd(rb.handle, _ptr(x), _ptr(g_in), _ptr(W), _ptr(y), _ptr(g_out),
                              _ptr(dy), _ptr(dg_out), Cin, Cout, SCN_RELU if relu else 0,
                              _ptr(out.get("dx")), _ptr(out.get("dg_in")), _ptr(out.get("dW")),
                              _ptr(out.get("dbias")), _ptr(ws), ws.numel(),
                              ctypes.c_void_p(_stream())), "scn_conv_bwd")
    return out


def maxpool_fwd(rb: Rulebook, x: torch.Tensor, g_in: torch.Tensor):
    """Returns (y [a_out, C], g_out [C], argmax uint8 [a_out, C])."""
    C = int(x.shape[1]) if x.dim() == 2 else -1
    _dev_tensor(x, torch.float32, (rb.a_in, C), "x")
    _dev_tensor(g_in, torch.float32, (C,), "g_in")
    y = torch.empty((rb.a_out, C), dtype=torch.float32, device=x.device)
    g_out = torch.empty(C, dtype=torch.float32, device=x.device)
    am = torch.empty((rb.a_out, C), dtype=torch.uint8, device=x.device)
    _check(lib().scn_maxpool_fwd(rb.handle, _ptr(x), _ptr(g_in), C, _ptr(y), _ptr(g_out), _ptr(am),
                                 ctypes.c_void_p(_stream())), "scn_maxpool_fwd")
    return y, g_out, am


def maxpool_bwd(rb: Rulebook, argmax: torch.Tensor, dy: torch.Tensor,
                dg_out: Optional[torch.Tensor] = None, ws: Optional[torch.Tensor] = None):
    """Returns (dx [a_in, C], dg_in [C])."""
    C = int(dy.shape[1]) if dy.dim() == 2 else -1
    _dev_tensor(dy, torch.float32, (rb.a_out, C), "dy")
    _dev_tensor(argmax, torch.uint8, (rb.a_out, C), "argmax")
    if dg_out is not None:
        _dev_tensor(dg_out, torch.float32, (C,), "dg_out")
    dx = torch.empty((rb.a_in, C), dtype=torch.float32, device=dy.device)
    dg_in = torch.empty(C, dtype=torch.float32, device=dy.device)
    if ws is None:
        n = lib().scn_maxpool_bwd_workspace_bytes(rb.handle, C)
        ws = torch.empty(max(int(n), 1), dtype=torch.uint8, device=dy.device)
    _check(lib().scn_maxpool_bwd(rb.handle, _ptr(argmax), _ptr(dy), _ptr(dg_out), C, _ptr(dx),
                                 _ptr(dg_in), _ptr(ws), ws.numel(), ctypes.c_void_p(_stream())),
           "scn_maxpool_bwd")
    return dx, dg_in


def version() -> str:
    return lib().scn_version().decode()


# Every callback pair ever installed stays alive for the life of the process:
# a rulebook built under a pair frees its memory through it, also after the
# pair has been replaced.
_hooks_kept = []


def build_chain(coords: torch.Tensor, grid, layers, lattice: str = "cubic") -> list:
    """Rulebooks of a chain of layers (``scn_rulebook_build_chain``): layer 0
    from ``coords`` on ``grid``, each later layer from the previous layer's
    active outputs; ``layers`` is a sequence of (filter, stride).  The chain
    waits for the device twice in all."""
    n = int(coords.shape[0]) if coords.dim() == 2 else -1
    _dev_tensor(coords, torch.int32, (n, 4), "coords")
    if lattice not in LATTICES:
        raise ValueError(f"lattice must be one of {sorted(LATTICES)}, got {lattice!r}")
    nl = len(layers)
    g = np.ascontiguousarray(np.asarray(grid, dtype=np.int64).reshape(4))
    fs = np.ascontiguousarray([int(f) for f, _ in layers], dtype=np.int32)
    ss = np.ascontiguousarray([int(s) for _, s in layers], dtype=np.int32)
    hs = (ctypes.c_void_p * max(nl, 1))()
    _check(lib().scn_rulebook_build_chain(
        _ptr(coords), n, g.ctypes.data_as(ctypes.c_void_p), LATTICES[lattice], nl,
        fs.ctypes.data_as(ctypes.c_void_p), ss.ctypes.data_as(ctypes.c_void_p),
        ctypes.c_void_p(_stream()), hs), "scn_rulebook_build_chain")
    return [Rulebook._from_handle(ctypes.c_void_p(hs[i]), coords.device) for i in range(nl)]


def set_dense_forward(min_rows: int = -1, min_offsets: int = -1) -> None:
    """Stride-1 rulebooks built from now on carry the dense forward view when
    they have at least ``min_rows`` outputs and ``min_offsets`` offsets
    (``scn_set_dense_forward``; negative values restore the defaults)."""
    _check(lib().scn_set_dense_forward(int(min_rows), int(min_offsets)), "scn_set_dense_forward")


def set_allocator(alloc=None, free=None) -> None:
    """Route the library's own device allocations through alloc(bytes, stream)
    -> pointer and free(pointer, stream) (``scn_set_allocator``).  ``"torch"``
    installs PyTorch's caching allocator; no argument restores the library's
    default pool."""
    if alloc == "torch":
        def alloc(nbytes, stream):
            return torch.cuda.caching_allocator_alloc(int(nbytes), stream=int(stream))

        def free(ptr, stream):
            torch.cuda.caching_allocator_delete(int(ptr))
    if alloc is None or free is None:
        lib().scn_set_allocator(_ALLOC_FN(), _FREE_FN(), None)
        return

    def c_alloc(nbytes, stream, ctx):
        try:
            return int(alloc(nbytes, stream or 0)) or None
        except Exception:  # the library reports SCN_ERR_NOMEM
            return None

    def c_free(ptr, stream, ctx):
        try:
            free(ptr, stream or 0)
        except Exception:
            pass

    hooks = (_ALLOC_FN(c_alloc), _FREE_FN(c_free))
    _hooks_kept.append(hooks)
    lib().scn_set_allocator(hooks[0], hooks[1], None)
