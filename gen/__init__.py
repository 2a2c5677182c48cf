"""Seeded synthetic inputs shared by the oracle tests, the GPU parity tests and
the benchmark.

This package only draws coordinates and random numbers; it contains none of
the sparse-convolution arithmetic (no active-set rule, no rulebook, no
convolution), so both sides of a parity test can use it without sharing any
part of the method.
"""
from .synth import (  # noqa: F401
    SEED_BASE,
    CONFIGS,
    LayerSpec,
    ConfigInput,
    make_config,
    make_dy,
    make_dg,
    trefoil_walk,
    bridge_walk,
    shell_sites,
    random_sites,
    tetra_sites,
    tetra_random_sites,
    tetra_shell_sites,
    triangle_sites,
    image_patch_sites,
    tri_random_sites,
    stream_rng,
)
