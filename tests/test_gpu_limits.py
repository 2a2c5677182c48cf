"""GPU parity at the library's stated limits: the largest grid the occupancy
bitmap accepts (B * my * mz * ceil(mx / 32) = 2^26 words), one word past it
(the keyed builder),
the widest convolution layers (256 channels) and pooling at 1024+ channels,
against the oracle."""
from __future__ import annotations

import numpy as np
import pytest

torch = pytest.importorskip("torch")

import oracle  # noqa: E402
from gen import random_sites, stream_rng  # noqa: E402

from helpers import conv_parity, dev, host, pool_parity  # noqa: E402

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def scn():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_1505_02890_amd as m
    m.lib()  # raises if the HIP library is missing
    return m


def _check(g, o):
    oa = o.arrays()
    assert (g.a_in, g.a_out, g.n_pairs, g.K) == (oa.a_in, oa.a_out, oa.n_pairs, oa.K)
    assert tuple(g.out_grid) == tuple(oa.out_grid)
    assert np.array_equal(g.offsets, oa.offsets)
    oc, ir, orr = g.export()
    assert np.array_equal(host(oc), oa.out_coords)
    assert np.array_equal(host(ir), oa.in_rows)
    assert np.array_equal(host(orr), oa.out_rows)


@pytest.mark.parametrize("grid,f,s", [((1, 2048, 2048, 512), 3, 1),   # exactly 2^26 words
                                      ((2, 1024, 2048, 512), 2, 2),   # 2^26 words over two samples
                                      ((1, 2048, 2048, 512), 3, 2)])
def test_largest_bitmap_grid(scn, grid, f, s):
    B, mx, my, mz = grid
    assert B * my * mz * ((mx + 31) // 32) == 1 << 26
    rng = stream_rng(81, f * 10 + s)
    coords = random_sites(rng, B, (mx, my, mz), 4000)
    # a few sites on the far corners of the grid
    corners = np.array([[B - 1, mx - 1, my - 1, mz - 1], [0, 0, 0, 0], [B - 1, mx - 1, 0, mz - 1]],
                       np.int32)
    keep = ~(coords[:, None, :] == corners[None]).all(axis=2).any(axis=1)
    coords = np.concatenate([coords[keep], corners]).astype(np.int32)
    g = scn.build_rulebook(dev(coords), grid, f, s)
    o = oracle.Rulebook(coords, grid, f, s)
    _check(g, o)


def test_one_word_past_the_bitmap_limit(scn):
    """One word past the bitmaps' limit the build goes to the keyed builder
    (sorted keys and hash tables), with the same result."""
    grid = (1, 2048, 2048, 513)
    rng = stream_rng(83, 0)
    coords = random_sites(rng, 1, grid[1:], 3000)
    corners = np.array([[0, 2047, 2047, 512], [0, 0, 0, 0]], np.int32)
    keep = ~(coords[:, None, :] == corners[None]).all(axis=2).any(axis=1)
    coords = np.concatenate([coords[keep], corners]).astype(np.int32)
    g = scn.build_rulebook(dev(coords), grid, 3, 1)
    assert g.keyed
    _check(g, oracle.Rulebook(coords, grid, 3, 1))


@pytest.mark.parametrize("f", [2, 3])
def test_widest_layers(scn, f):
    """256 input and 256 output channels (the largest the library takes)."""
    Cin = Cout = 256
    rng = stream_rng(82, f)
    coords = random_sites(rng, 1, (20, 18, 16), 700)
    K = f ** 3
    x = rng.standard_normal((len(coords), Cin)).astype(np.float32)
    g_in = (rng.standard_normal(Cin) * 0.5).astype(np.float32)
    W = (rng.standard_normal((K, Cin, Cout)) / np.sqrt(K * Cin)).astype(np.float32)
    bias = (rng.standard_normal(Cout) * 0.1).astype(np.float32)
    grid = (1, 20, 18, 16)
    g = scn.build_rulebook(dev(coords), grid, f, 1)
    o = oracle.Rulebook(coords, grid, f, 1)
    conv_parity(scn, g, o, x, g_in, W, bias, False, 83 + f)


def test_too_wide_layers_are_refused(scn):
    coords = random_sites(stream_rng(84, 0), 1, (8, 8, 8), 50)
    g = scn.build_rulebook(dev(coords), (1, 8, 8, 8), 2, 1)
    x = dev(np.ones((50, 257), np.float32))
    with pytest.raises(scn.ScnError) as e:
        scn.conv_fwd(g, x, dev(np.zeros(257, np.float32)), dev(np.ones((8, 257, 4), np.float32)))
    assert e.value.status == "unsupported"


@pytest.mark.parametrize("C", [1024, 1028, 3])
@pytest.mark.parametrize("f,s", [(2, 2), (3, 2)])
def test_pooling_channel_extremes(scn, C, f, s):
    """1024 channels (the widest four-channel path), 1028 (one channel per
    thread) and 3, against the oracle."""
    rng = stream_rng(85, C + f)
    coords = random_sites(rng, 1, (12, 11, 10), 300)
    x = rng.standard_normal((len(coords), C)).astype(np.float32)
    g_in = (np.abs(rng.standard_normal(C)) * 0.5).astype(np.float32)
    grid = (1, 12, 11, 10)
    g = scn.build_rulebook(dev(coords), grid, f, s)
    o = oracle.Rulebook(coords, grid, f, s)
    pool_parity(scn, g, o, x, g_in, rng, f > s)
