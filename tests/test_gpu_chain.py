"""Chained rulebooks: scn_rulebook_build_next against a build from the
previous layer's exported output sites and against the oracle, through the C
ABI, on every lattice."""
from __future__ import annotations

import numpy as np
import pytest

torch = pytest.importorskip("torch")

import oracle  # noqa: E402
from gen import random_sites, stream_rng, tetra_random_sites, tri_random_sites  # noqa: E402

from helpers import dev, host  # noqa: E402

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def scn():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_1505_02890_amd as m
    m.lib()  # raises if the HIP library is missing
    return m


def _arrays(g):
    oc, ir, orr = g.export()
    return host(oc), host(ir), host(orr)


def _same(a, b, sorted_inputs=True):
    assert (a.a_in, a.a_out, a.n_pairs, a.K, a.lattice) == (b.a_in, b.a_out, b.n_pairs, b.K, b.lattice)
    assert tuple(a.out_grid) == tuple(b.out_grid) and a.input_sorted == b.input_sorted
    assert a.input_sorted or not sorted_inputs
    assert np.array_equal(a.offsets, b.offsets)
    for x, y in zip(_arrays(a), _arrays(b)):
        assert np.array_equal(x, y)


def _sites(lattice, rng, B, m, n):
    if lattice == "cubic":
        return random_sites(rng, B, (m, m, m), n), (B, m, m, m)
    if lattice == "tetrahedral":
        return tetra_random_sites(rng, B, m, n), (B, m, m, m)
    if lattice == "square":
        return random_sites(rng, B, (m, m, 1), n), (B, m, m, 1)
    return tri_random_sites(rng, B, m, n), (B, m, m, 1)


CHAINS = [
    # (lattice, B, m, n, [(f, s), ...])
    ("cubic", 2, 40, 3000, [(2, 1), (3, 2), (2, 1), (2, 2), (1, 1)]),
    ("cubic", 1, 70, 5000, [(3, 1), (3, 3), (2, 1)]),
    ("tetrahedral", 2, 40, 2500, [(2, 1), (3, 2), (2, 1), (3, 2)]),
    ("square", 3, 90, 4000, [(2, 1), (2, 1), (3, 2), (2, 2)]),
    ("triangular", 3, 90, 3000, [(2, 1), (3, 2), (2, 1), (3, 2)]),
]


@pytest.mark.parametrize("case", CHAINS, ids=[c[0] + str(i) for i, c in enumerate(CHAINS)])
def test_chain_matches_rebuild_and_oracle(scn, case):
    lattice, B, m, n, layers = case
    coords, grid = _sites(lattice, stream_rng(91, CHAINS.index(case)), B, m, n)
    f, s = layers[0]
    g = scn.build_rulebook(dev(coords), grid, f, s, lattice=lattice)
    o = oracle.Rulebook(coords, grid, f, s, lattice=lattice)
    for f, s in layers[1:]:
        nxt = scn.next_rulebook(g, f, s)
        ref = scn.build_rulebook(g.out_coords(), g.out_grid, f, s, lattice=lattice)
        _same(nxt, ref)
        oa = o.arrays()
        o = oracle.Rulebook(oa.out_coords, oa.out_grid, f, s, lattice=lattice)
        ob = o.arrays()
        oc, ir, orr = _arrays(nxt)
        assert np.array_equal(oc, ob.out_coords) and np.array_equal(ir, ob.in_rows)
        assert np.array_equal(orr, ob.out_rows) and np.array_equal(nxt.offsets, ob.offsets)
        g = nxt


def test_chain_from_empty_layer(scn):
    g = scn.build_rulebook(dev(np.zeros((0, 4), np.int32)), (2, 9, 9, 9), 2, 1)
    nxt = scn.next_rulebook(g, 3, 2)
    assert nxt.a_in == 0 and nxt.a_out == 0 and nxt.n_pairs == 0
    assert tuple(nxt.out_grid) == (2, 3, 3, 3)


def test_chain_from_empty_grid_is_refused(scn):
    coords = random_sites(stream_rng(92, 0), 1, (2, 9, 9), 20)
    g = scn.build_rulebook(dev(coords), (1, 2, 9, 9), 3, 1)   # mx < f: output grid empty
    assert g.out_grid[1] == 0
    with pytest.raises(scn.ScnError) as e:
        scn.next_rulebook(g, 2, 1)
    assert e.value.status == "invalid"


def test_chain_outlives_its_source(scn):
    """The previous rulebook may be freed once the next one is built."""
    coords, grid = _sites("cubic", stream_rng(93, 0), 1, 30, 1500)
    g = scn.build_rulebook(dev(coords), grid, 2, 1)
    ref = scn.build_rulebook(g.out_coords(), g.out_grid, 3, 2)
    nxt = scn.next_rulebook(g, 3, 2)
    g.close()
    torch.cuda.synchronize()
    _same(nxt, ref)


def test_chain_on_another_stream_outlives_its_source(scn):
    """The next rulebook built on another stream than its source's, then the
    source freed at once (its free is ordered on its own stream): the next
    build's last kernels, which read the source's output bitmap and sites,
    still run before that free, so the result equals a fresh build."""
    coords, grid = _sites("cubic", stream_rng(93, 1), 2, 40, 6000)
    g = scn.build_rulebook(dev(coords), grid, 2, 1)
    ref = scn.build_rulebook(g.out_coords(), g.out_grid, 3, 2)
    torch.cuda.synchronize()
    side = torch.cuda.Stream()
    with torch.cuda.stream(side):
        nxt = scn.next_rulebook(g, 3, 2)
        g.close()
    # a build on the source's stream right after the free may take the freed
    # memory from the pool and overwrite it
    other = scn.build_rulebook(dev(coords), grid, 3, 1)
    torch.cuda.synchronize()
    _same(nxt, ref)
    assert other.a_in == len(coords)


def test_use_on_another_stream_right_after_the_build(scn):
    """The build returns before its last kernels finish (emission, the mask
    sort); a call on another stream is ordered after them by the library."""
    rng = stream_rng(94, 0)
    coords, grid = _sites("cubic", rng, 1, 40, 6000)
    Cin, Cout = 16, 24
    x = dev(rng.standard_normal((len(coords), Cin)).astype(np.float32))
    g_in = dev(np.zeros(Cin, np.float32))
    W = dev((rng.standard_normal((27, Cin, Cout)) / 20).astype(np.float32))
    cd = dev(coords)
    torch.cuda.synchronize()
    scn.set_dense_forward(0, 1)
    try:
        g = scn.build_rulebook(cd, grid, 3, 1)
    finally:
        scn.set_dense_forward()
    side = torch.cuda.Stream()
    with torch.cuda.stream(side):
        y, _ = scn.conv_fwd(g, x, g_in, W, None)
        oc, ir, orr = g.export()
    side.synchronize()
    o = oracle.Rulebook(coords, grid, 3, 1)
    oa = o.arrays()
    assert np.array_equal(host(oc), oa.out_coords) and np.array_equal(host(ir), oa.in_rows)
    assert np.array_equal(host(orr), oa.out_rows)
    y_ref, _ = oracle.conv_fwd(o, host(x), host(g_in), host(W), None)
    assert np.allclose(host(y), y_ref, rtol=1e-4, atol=1e-4)


@pytest.mark.parametrize("case", CHAINS, ids=[c[0] + str(i) for i, c in enumerate(CHAINS)])
def test_chain_build_matches_layer_by_layer(scn, case):
    """scn_rulebook_build_chain (two waits for the whole chain) gives the
    rulebooks of the layer-by-layer builds."""
    lattice, B, m, n, layers = case
    coords, grid = _sites(lattice, stream_rng(91, CHAINS.index(case)), B, m, n)
    chain = scn.build_chain(dev(coords), grid, layers, lattice=lattice)
    assert len(chain) == len(layers)
    g = None
    for (f, s), c in zip(layers, chain):
        first = g is None
        g = (scn.build_rulebook(dev(coords), grid, f, s, lattice=lattice) if first
             else scn.next_rulebook(g, f, s))
        _same(c, g, sorted_inputs=not first)   # layer 0 takes the caller's order


def test_chain_build_errors(scn):
    coords = random_sites(stream_rng(92, 1), 1, (2, 9, 9), 20)
    with pytest.raises(scn.ScnError) as e:   # layer 0's output grid is empty (mx < f)
        scn.build_chain(dev(coords), (1, 2, 9, 9), [(3, 1), (2, 1)])
    assert e.value.status == "invalid"
    with pytest.raises(scn.ScnError) as e:
        scn.build_chain(dev(coords), (1, 2, 9, 9), [])
    assert e.value.status == "invalid"
    bad = np.array([[0, 1, 1, 1], [0, 1, 1, 1]], np.int32)   # duplicate site in layer 0
    with pytest.raises(scn.ScnError) as e:
        scn.build_chain(dev(bad), (1, 9, 9, 9), [(2, 1), (2, 2)])
    assert e.value.status == "duplicate"
