"""GPU parity of the keyed rulebook builder (sorted site keys and open-
addressing hash tables): hypercubic sites in 1 to 4 dimensions
(scn_rulebook_build_nd) and 3D grids past the occupancy bitmaps
(scn_rulebook_build falls back to it), against the oracle: rulebooks
bit-exact, convolution and pooling within the fp32 tolerance; in 3D also
against the bitmap builder."""
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


def random_sites_nd(rng, B, dims, n):
    total = B * int(np.prod(dims))
    idx = rng.choice(total, size=min(n, total), replace=False)
    cols, rest = [], idx
    for m in dims:
        cols.append(rest % m)
        rest = rest // m
    return np.stack([rest] + cols, axis=1).astype(np.int32)


def check_rulebook(g, o):
    oa = o.arrays()
    assert (g.a_in, g.a_out, g.n_pairs, g.K) == (oa.a_in, oa.a_out, oa.n_pairs, oa.K)
    assert tuple(g.out_grid) == tuple(oa.out_grid)
    assert np.array_equal(g.offsets, oa.offsets)
    oc, ir, orr = g.export()
    assert np.array_equal(host(oc), oa.out_coords)
    assert np.array_equal(host(ir), oa.in_rows)
    assert np.array_equal(host(orr), oa.out_rows)


ND_CASES = [  # (d, B, dims, n, f, s, sort)
    (4, 2, (9, 8, 7, 9), 700, 2, 1, False),
    (4, 1, (10, 9, 9, 8), 900, 2, 2, False),
    (4, 1, (12, 11, 10, 9), 1500, 2, 1, True),
    (4, 3, (6, 6, 6, 6), 300, 1, 2, False),
    (4, 1, (9, 9, 9, 9), 600, 2, 3, False),
    (2, 2, (40, 37), 500, 3, 1, False),
    (2, 1, (33, 31), 300, 3, 2, False),
    (1, 3, (300,), 200, 3, 1, False),
    (1, 2, (100,), 60, 2, 2, True),
    (3, 2, (20, 18, 17), 900, 3, 1, False),
    (3, 1, (21, 19, 18), 700, 3, 2, False),
    (3, 1, (16, 17, 15), 800, 2, 2, True),
]


@pytest.mark.parametrize("case", ND_CASES, ids=[str(i) for i in range(len(ND_CASES))])
def test_nd_rulebook_bit_exact(scn, case):
    d, B, dims, n, f, s, srt = case
    rng = stream_rng(600 + ND_CASES.index(case), 0)
    coords = random_sites_nd(rng, B, dims, n)
    if srt:  # rows already in key order (the builder's no-permutation path)
        key = coords[:, 0].astype(np.int64)
        for a in reversed(range(d)):
            key = key * dims[a] + coords[:, 1 + a]
        coords = coords[np.argsort(key)]
    grid = (B,) + dims
    g = scn.build_rulebook_nd(dev(coords), grid, f, s)
    assert g.ndim == d and g.keyed and g.input_sorted == srt
    check_rulebook(g, oracle.Rulebook(coords, grid, f, s, ndim=d))


@pytest.mark.parametrize("f,s", [(3, 1), (2, 2), (3, 2), (1, 1), (2, 3)])
def test_keyed_equals_bitmap_builder_in_3d(scn, f, s):
    rng = stream_rng(610, f * 10 + s)
    grid = (2, 30, 27, 25)
    coords = random_sites(rng, 2, grid[1:], 3000)
    a = scn.build_rulebook(dev(coords), grid, f, s)
    b = scn.build_rulebook_nd(dev(coords), grid, f, s)
    assert not a.keyed and b.keyed
    assert (a.a_out, a.n_pairs, a.input_sorted) == (b.a_out, b.n_pairs, b.input_sorted)
    assert np.array_equal(a.offsets, b.offsets)
    for x, y in zip(a.export(), b.export()):
        assert np.array_equal(host(x), host(y))


CONV_ND = [  # (d, B, dims, n, f, s, Cin, Cout, relu)
    (4, 2, (8, 7, 8, 7), 600, 2, 1, 16, 32, False),
    (4, 1, (9, 9, 8, 8), 700, 2, 2, 32, 16, True),
    (4, 1, (7, 7, 7, 7), 400, 1, 1, 8, 8, False),
    (2, 1, (30, 28), 300, 3, 1, 16, 16, True),
]


@pytest.mark.parametrize("case", CONV_ND, ids=[str(i) for i in range(len(CONV_ND))])
def test_nd_conv_parity(scn, case):
    d, B, dims, n, f, s, Cin, Cout, relu = case
    seed = 620 + CONV_ND.index(case)
    rng = stream_rng(seed, 0)
    coords = random_sites_nd(rng, B, dims, n)
    grid = (B,) + dims
    g = scn.build_rulebook_nd(dev(coords), grid, f, s)
    o = oracle.Rulebook(coords, grid, f, s, ndim=d)
    check_rulebook(g, o)
    x = rng.standard_normal((len(coords), Cin)).astype(np.float32)
    g_in = rng.standard_normal(Cin).astype(np.float32)
    W = (rng.standard_normal((f ** d, Cin, Cout)) / np.sqrt(f ** d * Cin)).astype(np.float32)
    bias = rng.standard_normal(Cout).astype(np.float32)
    conv_parity(scn, g, o, x, g_in, W, bias, relu, seed)


POOL_ND = [  # (d, B, dims, n, f, s, C)
    (4, 2, (10, 9, 8, 9), 900, 2, 2, 16),
    (4, 1, (9, 8, 9, 8), 700, 2, 2, 5),
    (4, 1, (8, 8, 8, 8), 500, 1, 2, 8),
    (2, 2, (31, 29), 400, 2, 2, 8),
    (2, 1, (30, 28), 300, 3, 3, 8),
    (1, 1, (200,), 90, 2, 2, 12),
]


@pytest.mark.parametrize("case", POOL_ND, ids=[str(i) for i in range(len(POOL_ND))])
def test_nd_pool_parity(scn, case):
    d, B, dims, n, f, s, C = case
    rng = stream_rng(640 + POOL_ND.index(case), 0)
    coords = random_sites_nd(rng, B, dims, n)
    grid = (B,) + dims
    g = scn.build_rulebook_nd(dev(coords), grid, f, s)
    o = oracle.Rulebook(coords, grid, f, s, ndim=d)
    check_rulebook(g, o)
    x = rng.standard_normal((len(coords), C)).astype(np.float32)
    x[rng.random(x.shape) < 0.2] = 0.0
    g_in = (np.abs(rng.standard_normal(C)) * 0.3).astype(np.float32)
    pool_parity(scn, g, o, x, g_in, rng, f > s)


# grids past the occupancy bitmaps (2^26 words per grid): the cubic build
# goes to the keyed builder
BIG = [((1, 1 << 20, 1 << 10, 1 << 10), 3, 1), ((1, 1 << 20, 1 << 10, 1 << 10), 2, 2),
       ((2, 4096, 4096, 1024), 3, 2), ((1, 2048, 2048, 513), 3, 1)]


@pytest.mark.parametrize("grid,f,s", BIG, ids=[str(i) for i in range(len(BIG))])
def test_grid_past_the_bitmaps(scn, grid, f, s):
    B, mx, my, mz = grid
    assert B * my * mz * ((mx + 31) // 32) > 1 << 26
    rng = stream_rng(650, BIG.index((grid, f, s)))
    # clustered sites (a window sees several), plus the far corners
    centres = np.stack([rng.integers(0, B, 60), rng.integers(0, mx - 8, 60),
                        rng.integers(0, my - 8, 60), rng.integers(0, mz - 8, 60)], 1)
    pts = centres[rng.integers(0, 60, 6000)] + np.concatenate(
        [np.zeros((6000, 1), np.int64), rng.integers(0, 8, (6000, 3))], 1)
    corners = np.array([[B - 1, mx - 1, my - 1, mz - 1], [0, 0, 0, 0], [B - 1, mx - 1, 0, mz - 1]])
    coords = np.unique(np.concatenate([pts, corners]), axis=0).astype(np.int32)
    coords = coords[rng.permutation(len(coords))]
    g = scn.build_rulebook(dev(coords), grid, f, s)
    assert g.keyed and g.ndim == 3
    o = oracle.Rulebook(coords, grid, f, s)
    check_rulebook(g, o)
    if s == 1:
        C = 16
        x = rng.standard_normal((len(coords), C)).astype(np.float32)
        g_in = rng.standard_normal(C).astype(np.float32)
        W = (rng.standard_normal((f ** 3, C, C)) / np.sqrt(f ** 3 * C)).astype(np.float32)
        conv_parity(scn, g, o, x, g_in, W, None, True, 660 + BIG.index((grid, f, s)))
    else:
        C = 8
        x = rng.standard_normal((len(coords), C)).astype(np.float32)
        pool_parity(scn, g, o, x, np.zeros(C, np.float32), rng, f > s)


def test_keyed_chain(scn):
    """next_rulebook and build_chain on a grid past the bitmaps: each layer
    from the previous one's outputs, as the oracle chain."""
    grid = (1, 1 << 19, 1 << 10, 1 << 10)
    rng = stream_rng(670, 0)
    centres = np.stack([np.zeros(40, np.int64), rng.integers(0, grid[1] - 16, 40),
                        rng.integers(0, grid[2] - 16, 40), rng.integers(0, grid[3] - 16, 40)], 1)
    pts = centres[rng.integers(0, 40, 3000)] + np.concatenate(
        [np.zeros((3000, 1), np.int64), rng.integers(0, 16, (3000, 3))], 1)
    coords = np.unique(pts, axis=0).astype(np.int32)
    layers = [(3, 1), (2, 2), (3, 1), (3, 2)]
    chain = scn.build_chain(dev(coords), grid, layers)
    g = None
    c, gr = coords, grid
    for i, (f, s) in enumerate(layers):
        g = scn.build_rulebook(dev(coords), grid, f, s) if i == 0 else scn.next_rulebook(g, f, s)
        o = oracle.Rulebook(c, gr, f, s)
        check_rulebook(g, o)
        check_rulebook(chain[i], o)
        oa = o.arrays()
        c, gr = oa.out_coords, tuple(oa.out_grid)


def test_nd_next_rulebook(scn):
    rng = stream_rng(671, 0)
    dims = (12, 11, 10, 12)
    coords = random_sites_nd(rng, 2, dims, 1200)
    g = scn.build_rulebook_nd(dev(coords), (2,) + dims, 2, 1)
    nxt = scn.next_rulebook(g, 2, 2)
    assert nxt.keyed and nxt.ndim == 4
    oa = oracle.Rulebook(coords, (2,) + dims, 2, 1, ndim=4).arrays()
    check_rulebook(nxt, oracle.Rulebook(oa.out_coords, oa.out_grid, 2, 2, ndim=4))


def test_nd_empty_and_errors(scn):
    e0 = scn.build_rulebook_nd(dev(np.zeros((0, 5), np.int32)), (1, 4, 4, 4, 4), 2, 1)
    assert (e0.a_in, e0.a_out, e0.n_pairs, e0.K) == (0, 0, 0, 16)
    dup = np.array([[0, 1, 2, 3, 1], [0, 1, 2, 3, 1]], np.int32)
    with pytest.raises(scn.ScnError) as e:
        scn.build_rulebook_nd(dev(dup), (1, 4, 4, 4, 4), 2, 1)
    assert e.value.status == "duplicate"
    with pytest.raises(scn.ScnError) as e:
        scn.build_rulebook_nd(dev(np.array([[0, 1, 2, 4, 1]], np.int32)), (1, 4, 4, 4, 4), 2, 1)
    assert e.value.status == "range"
    with pytest.raises(scn.ScnError) as e:  # 3^4 = 81 offsets
        scn.build_rulebook_nd(dev(np.array([[0, 1, 2, 3, 1]], np.int32)), (1, 4, 4, 4, 4), 3, 1)
    assert e.value.status == "unsupported"
    # windows wider than their stride off 3D: a convolution rulebook only
    c2 = np.array([[0, 1, 2], [0, 3, 3]], np.int32)
    g2 = scn.build_rulebook_nd(dev(c2), (1, 9, 9), 3, 2)
    with pytest.raises(scn.ScnError) as e:
        scn.maxpool_fwd(g2, dev(np.ones((2, 4), np.float32)), dev(np.zeros(4, np.float32)))
    assert e.value.status == "unsupported"


def test_keyed_chain_switches_to_the_bitmaps(scn):
    """A chain whose first grids are past the bitmaps and whose later grids fit
    them: the later layers come from the bitmap builder, with the same
    rulebooks as the oracle chain (and next_rulebook does the same)."""
    grid = (2, 4096, 4096, 1024)
    layers = [(3, 2), (3, 2), (2, 1), (3, 1)]
    rng = stream_rng(672, 0)
    centres = np.stack([rng.integers(0, 2, 50), rng.integers(0, grid[1] - 24, 50),
                        rng.integers(0, grid[2] - 24, 50), rng.integers(0, grid[3] - 24, 50)], 1)
    pts = centres[rng.integers(0, 50, 5000)] + np.concatenate(
        [np.zeros((5000, 1), np.int64), rng.integers(0, 24, (5000, 3))], 1)
    coords = np.unique(pts, axis=0).astype(np.int32)
    chain = scn.build_chain(dev(coords), grid, layers)
    assert [r.keyed for r in chain] == [True, True, False, False]
    g = None
    c, gr = coords, grid
    for i, (f, s) in enumerate(layers):
        g = scn.build_rulebook(dev(coords), grid, f, s) if i == 0 else scn.next_rulebook(g, f, s)
        assert g.keyed == (i < 2)
        o = oracle.Rulebook(c, gr, f, s)
        check_rulebook(g, o)
        check_rulebook(chain[i], o)
        oa = o.arrays()
        c, gr = oa.out_coords, tuple(oa.out_grid)
