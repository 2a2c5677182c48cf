"""Whole-network sparse CNN inference on the C ABI: the cubic networks of the
paper's 3D object-recognition experiment (section 2, "Object recognition"),

    32C2 - MP3/2 - 64C2 - MP3/2 - 96C2 - ... - output,

with L levels of 3x3x3 stride-2 max-pooling.  Every convolution has a 2x2x2
filter, stride 1, ReLU, and 32*(i+1) output channels at level i; "output" is a
1x1x1 convolution to the class scores on the single site that remains.

All padding is valid, so the input grid is the size the network reduces to one
site: working back from 1, a C2 adds 1 and an MP3/2 maps m to 2m + 1, which
gives 62, 126 and 254 for 4, 5 and 6 levels.

The same networks run on the tetrahedral lattice of section 1.2 (the rows
marked with a triangle in the experiment's table): a C2 filter then covers 4
sites, an MP3/2 region 10, and the grid of size m is the tetrahedron
x + y + z < m in skewed coordinates; the sizes above are unchanged.

The 2D networks of the square-versus-triangular comparison (section 2,
SquareNet and TriangLeNet) have pairs of C2 layers between the poolings,

    32C2 - 32C2 - MP3/2 - 64C2 - 64C2 - MP3/2 - ... - 192C2 - 192C2 - output,

i.e. five levels of two convolutions each; they run on the square and the
triangular lattice (grids with one z plane), with input size 189.

Every step runs in the library's kernels (rulebook build, contraction,
pooling); this module only sequences the calls and keeps the layer state.
"""
from __future__ import annotations

import math
from dataclasses import dataclass
from typing import List

import torch

from . import _lib as scn


def input_size(levels: int, convs: int = 1) -> int:
    """Grid size that `levels` x (convs x C2, MP3/2) followed by convs x C2
    reduce to 1."""
    m = 1 + convs  # each C2 adds one
    for _ in range(levels):
        m = 2 * m + 1  # MP3/2: (m_in - 3) / 2 + 1 = m
        m += convs     # the C2 layers before it
    return m


PLANAR = ("square", "triangular")


def window_size(f: int, lattice: str = "cubic") -> int:
    """Sites under a filter of size f on each lattice of Figure 2."""
    return {"cubic": f ** 3, "tetrahedral": math.comb(f + 2, 3), "square": f * f,
            "triangular": math.comb(f + 1, 2)}[lattice]


@dataclass
class Layer:
    kind: str            # "conv" or "pool"
    f: int
    s: int
    cin: int = 0
    cout: int = 0
    relu: bool = False


def architecture(levels: int, classes: int = 50, width: int = 32, cin: int = 1,
                 convs: int = 1) -> List[Layer]:
    """convs x nC2 then MP3/2 per level (n = width, 2*width, ...), convs last
    C2 layers, then the 1x1 class layer."""
    layers: List[Layer] = []
    c = cin
    for i in range(levels + 1):
        for _ in range(convs):
            layers.append(Layer("conv", 2, 1, c, width * (i + 1), True))
            c = width * (i + 1)
        if i < levels:
            layers.append(Layer("pool", 3, 2))
    layers.append(Layer("conv", 1, 1, c, classes, False))
    return layers


class SparseNet:
    """Random-initialised weights (He scaling) for `architecture(...)` on one
    of the lattices of Figure 2; the input ground state is 0 (an empty site
    holds no signal)."""

    def __init__(self, levels: int, classes: int = 50, width: int = 32, seed: int = 0,
                 device: str = "cuda", lattice: str = "cubic", convs: int = 1, cin: int = 1):
        if lattice not in ("cubic", "tetrahedral") + PLANAR:
            raise ValueError(f"unknown lattice {lattice!r}")
        self.levels = levels
        self.lattice = lattice
        self.layers = architecture(levels, classes, width, cin, convs)
        self.m = input_size(levels, convs)
        g = torch.Generator().manual_seed(seed)
        self.params = []
        for L in self.layers:
            if L.kind != "conv":
                self.params.append(None)
                continue
            K = window_size(L.f, lattice)
            W = torch.randn(K, L.cin, L.cout, generator=g) * math.sqrt(2.0 / (K * L.cin))
            b = torch.randn(L.cout, generator=g) * 0.05
            self.params.append((W.to(device), b.to(device)))
        self.device = device

    def forward(self, coords: torch.Tensor, x: torch.Tensor, batch: int):
        """coords int32 [n][4] (b, x, y, z) on the device (z = 0 on a 2D
        lattice), x [n][cin].  Returns (scores [a][classes], out_coords [a][4],
        per-layer records)."""
        grid = (batch, self.m, self.m, 1 if self.lattice in PLANAR else self.m)
        g = torch.zeros(x.shape[1], dtype=torch.float32, device=self.device)
        rec = []
        # Rulebooks depend only on the active sites, not on the features: build
        # the whole chain first, in one call that waits for the device twice,
        # then issue every convolution and pooling back to back.  The first
        # layer's sites are the input; each later layer's are the previous
        # layer's active outputs (its rank bitmap is reused).
        rbs = scn.build_chain(coords, grid, [(L.f, L.s) for L in self.layers],
                              lattice=self.lattice)
        for L, p, rb in zip(self.layers, self.params, rbs):
            if L.kind == "conv":
                W, b = p
                x, g = scn.conv_fwd(rb, x, g, W, b, relu=L.relu)
                rec.append(("conv", rb.a_in, rb.a_out, rb.n_pairs, L.cin, L.cout))
            else:
                x, g, _ = scn.maxpool_fwd(rb, x, g)
                rec.append(("pool", rb.a_in, rb.a_out, rb.n_pairs, x.shape[1], x.shape[1]))
        return x, rb.out_coords(), rec


def macs(records) -> int:
    """Multiply-accumulates of the convolutions (active pairs only)."""
    return int(sum(P * ci * co for kind, _, _, P, ci, co in records if kind == "conv"))
