"""A whole nC2-MP3/2 network (the object-recognition networks of section 2)
through the C ABI against the same chain of layers in the oracle.

The oracle builds every layer's rulebook from its own output sites, so the
two chains share only the seeded input and the weights."""
from __future__ import annotations

import os
import sys

import numpy as np
import pytest

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))

import oracle  # noqa: E402
from gen import image_patch_sites, shell_sites, stream_rng, tetra_shell_sites  # noqa: E402
from helpers import assert_exact, assert_site, dev, host  # noqa: E402

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def scn():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_1505_02890_amd as m
    m.lib()  # raises if the HIP library is missing
    return m


def _batch(batch, m, scale, seed, lattice="cubic"):
    rows = []
    for b in range(batch):
        rng = stream_rng(seed, b)
        semi = [0.5 * scale * float(rng.uniform(0.6, 1.0)) for _ in range(3)]
        power = (2, 4)[int(rng.integers(2))]
        if lattice == "cubic":
            s = shell_sites(rng, m, semi, [m / 2.0] * 3, power)
        else:
            s = tetra_shell_sites(rng, m, semi, power)
        rows.append(np.concatenate([np.full((len(s), 1), b, np.int64), s], axis=1))
    return np.ascontiguousarray(np.concatenate(rows).astype(np.int32))


@pytest.mark.parametrize("lattice,levels,width,scale", [
    ("cubic", 1, 4, 3.0), ("cubic", 2, 4, 6.0), ("cubic", 3, 3, 12.0),
    ("tetrahedral", 1, 4, 1.5), ("tetrahedral", 2, 4, 4.0), ("tetrahedral", 3, 3, 9.0)])
def test_network_matches_oracle_chain(scn, lattice, levels, width, scale):
    from paper_1505_02890_amd.network import SparseNet, input_size

    batch = 3
    m = input_size(levels)
    coords = _batch(batch, m, scale, 4242 + levels, lattice)
    net = SparseNet(levels, classes=5, width=width, seed=levels, lattice=lattice)
    x = np.ones((len(coords), 1), np.float32)
    out, oc, rec = net.forward(dev(coords, torch.int32), dev(x), batch)
    assert [r[0] for r in rec] == [L.kind for L in net.layers]

    c, grid, xr = coords, (batch, m, m, m), x.astype(np.float64)
    g = np.zeros(1)
    for L, p in zip(net.layers, net.params):
        o = oracle.Rulebook(c, grid, L.f, L.s, lattice=lattice)
        if L.kind == "conv":
            W, b = (host(t).astype(np.float64) for t in p)
            xr, g = oracle.conv_fwd(o, xr, g, W, b, relu=L.relu)
        else:
            xr, g, _, _ = oracle.maxpool_fwd(o, xr, g)
        c, grid = o.arrays().out_coords, tuple(o.out_grid)

    assert_exact("final sites", host(oc), c)
    # one final site per sample whose shell survives the network
    assert len(c) == batch and np.array_equal(c[:, 0], np.arange(batch))
    # every class score, elementwise (the chain carries fp32 rounding through
    # all layers on the library's side)
    assert_site("scores", host(out), xr)


@pytest.mark.parametrize("lattice,levels,patch", [("square", 1, 5), ("triangular", 1, 4),
                                                  ("square", 2, 9), ("triangular", 2, 8)])
def test_planar_network_matches_oracle_chain(scn, lattice, levels, patch):
    """The 2D SquareNet / TriangLeNet shape (two C2 per level) on an image
    patch with three channels, against the chain of oracle layers."""
    from paper_1505_02890_amd.network import SparseNet, input_size

    batch = 2
    m = input_size(levels, convs=2)
    cell = image_patch_sites(lattice, m, patch, patch)
    coords = np.ascontiguousarray(np.concatenate(
        [np.concatenate([np.full((len(cell), 1), b), cell], axis=1) for b in range(batch)]
    ).astype(np.int32))
    x = stream_rng(77, levels).standard_normal((len(coords), 3)).astype(np.float32)
    net = SparseNet(levels, classes=4, width=4, seed=levels, lattice=lattice, convs=2, cin=3)
    out, oc, rec = net.forward(dev(coords, torch.int32), dev(x), batch)
    c, grid, xr = coords, (batch, m, m, 1), x.astype(np.float64)
    g = np.zeros(3)
    for L, p in zip(net.layers, net.params):
        o = oracle.Rulebook(c, grid, L.f, L.s, lattice=lattice)
        if L.kind == "conv":
            W, b = (host(t).astype(np.float64) for t in p)
            xr, g = oracle.conv_fwd(o, xr, g, W, b, relu=L.relu)
        else:
            xr, g, _, _ = oracle.maxpool_fwd(o, xr, g)
        c, grid = o.arrays().out_coords, tuple(o.out_grid)
    assert_exact("final sites", host(oc), c)
    assert len(c) == batch
    assert_site("scores", host(out), xr)


@pytest.mark.timeout(900)
def test_scale80_cubic_network_at_batch_256(scn):
    """The scale-80 cubic network (six C2-MP3/2 levels, input grid 254^3) at
    batch 256: its first grids hold 256 * 255^2 * 8 bitmap words, past the
    occupancy bitmaps, so the chain's rulebooks come from the keyed builder.
    Samples do not interact: the final site and the class scores of sampled
    samples equal the oracle chain run on each sample alone."""
    from paper_1505_02890_amd.network import SparseNet, input_size

    batch, levels, scale = 256, 6, 80.0
    m = input_size(levels)
    assert batch * (m + 1) ** 2 * ((m + 1 + 31) // 32) > 1 << 26
    coords = _batch(batch, m, scale, 8080)
    net = SparseNet(levels, classes=10, seed=80)
    x = np.ones((len(coords), 1), np.float32)
    out, oc, rec = net.forward(dev(coords, torch.int32), dev(x), batch)
    out, oc = host(out), host(oc)
    assert len(oc) == batch and np.array_equal(oc[:, 0], np.arange(batch))
    for b in (0, 131, 255):
        cb = coords[coords[:, 0] == b].copy()
        cb[:, 0] = 0
        c, grid, xr, g = cb, (1, m, m, m), np.ones((len(cb), 1)), np.zeros(1)
        for L, p in zip(net.layers, net.params):
            o = oracle.Rulebook(c, grid, L.f, L.s)
            if L.kind == "conv":
                W, bias = (host(t).astype(np.float64) for t in p)
                xr, g = oracle.conv_fwd(o, xr, g, W, bias, relu=L.relu)
            else:
                xr, g, _, _ = oracle.maxpool_fwd(o, xr, g)
            c, grid = o.arrays().out_coords, tuple(o.out_grid)
        assert_exact(f"final site of sample {b}", oc[b, 1:], c[0, 1:])
        assert_site(f"scores of sample {b}", out[b:b + 1], xr)
