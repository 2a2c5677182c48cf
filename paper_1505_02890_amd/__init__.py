"""Sparse 3D convolution hot path (Graham, "Sparse 3D convolutional neural
networks", section 1.3) on AMD Instinct MI355X.

The computation lives in ``libscn.so`` (hand-written HIP for gfx950, C ABI in
``include/scn.h``); this package is its thin Python binding.
"""
from ._lib import (  # noqa: F401
    EXPORTED,
    LIB_PATH,
    SCN_RELU,
    Rulebook,
    ScnError,
    build_chain,
    build_rulebook,
    build_rulebook_nd,
    conv_bwd,
    conv_bwd_workspace,
    conv_fwd,
    lib,
    maxpool_bwd,
    maxpool_fwd,
    next_rulebook,
    set_allocator,
    set_dense_forward,
    version,
)
