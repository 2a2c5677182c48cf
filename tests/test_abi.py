"""CPU checks of the C ABI boundary: the built library loads and exports every
function declared in include/scn.h, and calls that fail before touching the GPU
report their status (no compute runs here)."""
from __future__ import annotations

import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "scn.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(scn_[a-z0-9_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def libscn():
    from paper_1505_02890_amd import _lib
    if not os.path.exists(_lib.LIB_PATH):
        from paper_1505_02890_amd.build import build
        build()
    return _lib.lib()


def test_header_declares_the_boundary():
    names = declared_functions()
    for n in ("scn_rulebook_build", "scn_conv_fwd", "scn_conv_bwd", "scn_maxpool_fwd",
              "scn_maxpool_bwd", "scn_rulebook_free"):
        assert n in names


def test_library_exports_every_declared_symbol(libscn):
    from paper_1505_02890_amd import EXPORTED
    names = declared_functions()
    for n in names:
        assert hasattr(libscn, n), f"{n} declared in scn.h but not exported"
    assert set(names) == set(EXPORTED), "binding and header disagree"


def test_host_side_argument_errors(libscn):
    # these fail in argument validation, before any device work
    out = ctypes.c_void_p(123)
    grid = (ctypes.c_int64 * 4)(1, 4, 4, 4)
    assert libscn.scn_rulebook_build(None, 5, grid, 2, 1, None, ctypes.byref(out)) == 1
    assert out.value is None
    assert libscn.scn_rulebook_build(None, 0, grid, 0, 1, None, ctypes.byref(out)) == 1
    assert libscn.scn_rulebook_build(None, 0, grid, 4, 1, None, ctypes.byref(out)) == 5
    assert b"filter" in libscn.scn_last_error()
    bad = (ctypes.c_int64 * 4)(1, 0, 4, 4)
    assert libscn.scn_rulebook_build(None, 0, bad, 2, 1, None, ctypes.byref(out)) == 1
    outs = (ctypes.c_void_p * 2)(123, 456)
    fs = (ctypes.c_int32 * 2)(2, 2)
    ss = (ctypes.c_int32 * 2)(1, 2)
    assert libscn.scn_rulebook_build_chain(None, 5, grid, 0, 2, fs, ss, None, outs) == 1
    assert outs[0] is None and outs[1] is None
    assert libscn.scn_rulebook_build_chain(None, 0, grid, 0, 0, fs, ss, None, outs) == 1
    assert libscn.scn_rulebook_build_chain(None, 0, grid, 0, 65, fs, ss, None, outs) == 1
    big = (ctypes.c_int32 * 2)(4, 2)
    assert libscn.scn_rulebook_build_chain(None, 0, grid, 0, 2, big, ss, None, outs) == 5
    assert libscn.scn_conv_fwd(None, None, None, None, None, 1, 1, 0, None, None, None) == 1
    assert libscn.scn_maxpool_fwd(None, None, None, 1, None, None, None, None) == 1
    assert libscn.scn_conv_bwd_workspace_bytes(None, 4, 4, 0) == 0
    libscn.scn_rulebook_free(None)
    assert libscn.scn_version().startswith(b"scn-mi355x")


def test_binding_fails_loudly_without_library(monkeypatch, tmp_path):
    from paper_1505_02890_amd import _lib
    monkeypatch.setattr(_lib, "_lib", None)
    monkeypatch.setattr(_lib, "LIB_PATH", str(tmp_path / "missing.so"))
    with pytest.raises(RuntimeError, match="missing"):
        _lib.lib()
