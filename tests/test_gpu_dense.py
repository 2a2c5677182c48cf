"""GPU parity of the dense-block forward (stride-1 rulebooks that carry the
mask-sorted view, scn_set_dense_forward) against the oracle, on every
lattice and across channel counts: one to sixteen 16-channel steps, one to
four 64-channel chunks (including last chunks of a single 16-channel step:
Cin = 80, 136, 200), several 64-column blocks, ragged last blocks, ReLU on and
off, sorted and shuffled inputs.  The same layers with the view switched off
(the per-offset pair-list forward) also match the oracle and give the same
rulebook; repeated calls are bitwise identical.  Single-channel layers with
the view (a network's first layer) are checked forward and backward."""
from __future__ import annotations

import math

import numpy as np
import pytest

torch = pytest.importorskip("torch")

import oracle  # noqa: E402
from gen import random_sites, stream_rng, tetra_random_sites, tri_random_sites  # noqa: E402

from helpers import assert_site, conv_parity, dev, host  # noqa: E402

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def scn():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_1505_02890_amd as m
    m.lib()  # raises if the HIP library is missing
    m.set_dense_forward(0, 1)  # every stride-1 rulebook with outputs
    yield m
    m.set_dense_forward()


def _K(lattice, f):
    return {"cubic": f ** 3, "tetrahedral": math.comb(f + 2, 3), "square": f * f,
            "triangular": math.comb(f + 1, 2)}[lattice]


def _sites(lattice, rng, B, m, n, shuffle=True):
    if lattice == "cubic":
        return random_sites(rng, B, (m, m, m), n, shuffle=shuffle), (B, m, m, m)
    if lattice == "tetrahedral":
        return tetra_random_sites(rng, B, m, n, shuffle=shuffle), (B, m, m, m)
    if lattice == "square":
        return random_sites(rng, B, (m, m, 1), n, shuffle=shuffle), (B, m, m, 1)
    return tri_random_sites(rng, B, m, n, shuffle=shuffle), (B, m, m, 1)


CASES = [
    # (lattice, f, B, m, n, Cin, Cout, relu, shuffle)
    ("cubic", 3, 2, 24, 3000, 64, 64, False, True),      # the benchmark's shape, small
    ("cubic", 3, 1, 30, 2500, 1, 16, True, True),        # one channel (non-vector loads)
    ("cubic", 2, 2, 20, 1800, 3, 32, True, False),       # sorted input
    ("cubic", 3, 1, 22, 1500, 17, 5, False, True),       # ragged channels and columns
    ("cubic", 2, 1, 18, 1200, 96, 96, True, True),       # two chunks, two column blocks
    ("cubic", 3, 1, 16, 700, 256, 72, False, True),      # four chunks
    ("cubic", 2, 1, 14, 2744, 32, 32, False, True),      # every site active
    ("tetrahedral", 3, 2, 30, 2000, 48, 40, True, True),
    ("tetrahedral", 2, 1, 26, 1500, 64, 64, False, False),
    ("square", 3, 3, 60, 2500, 32, 64, True, True),
    ("triangular", 3, 3, 70, 2400, 64, 32, False, True),
    ("triangular", 2, 1, 9, 45, 8, 8, False, True),       # one block, grid filled
    # last 64-channel chunk of one 16-channel step (Cin % 64 in 65..80)
    ("cubic", 3, 1, 18, 1200, 80, 40, True, True),
    ("cubic", 2, 1, 16, 1000, 136, 64, False, True),
    ("cubic", 3, 1, 14, 600, 200, 48, True, True),
    ("tetrahedral", 3, 1, 24, 1500, 80, 72, False, True),
    # one input channel: odd and wide column counts, every lattice's window
    ("cubic", 2, 2, 20, 1800, 1, 7, False, True),
    ("cubic", 3, 1, 20, 1500, 1, 130, True, False),
    ("tetrahedral", 3, 1, 24, 1500, 1, 33, True, True),
    ("square", 3, 2, 50, 2000, 1, 64, False, True),
    ("triangular", 2, 1, 40, 600, 1, 256, True, True),
]


@pytest.mark.parametrize("case", CASES, ids=[f"{c[0]}{i}" for i, c in enumerate(CASES)])
def test_dense_forward_parity(scn, case):
    lattice, f, B, m, n, Cin, Cout, relu, shuffle = case
    rng = stream_rng(170, CASES.index(case))
    coords, grid = _sites(lattice, rng, B, m, n, shuffle)
    K = _K(lattice, f)
    x = rng.standard_normal((len(coords), Cin)).astype(np.float32)
    g_in = (rng.standard_normal(Cin) * 0.5).astype(np.float32)
    W = (rng.standard_normal((K, Cin, Cout)) / np.sqrt(K * Cin)).astype(np.float32)
    bias = (rng.standard_normal(Cout) * 0.1).astype(np.float32)
    g = scn.build_rulebook(dev(coords), grid, f, 1, lattice=lattice)
    o = oracle.Rulebook(coords, grid, f, 1, lattice=lattice)
    assert g.a_out == o.arrays().a_out
    assert g.dense_view
    y_ref, go_ref = oracle.conv_fwd(o, x, g_in, W, bias, relu=relu)
    yd, god = scn.conv_fwd(g, dev(x), dev(g_in), dev(W), dev(bias), relu=relu)
    assert_site("y", host(yd), y_ref)
    assert_site("g_out", host(god), go_ref)
    # repeated calls: bitwise identical
    yd2, _ = scn.conv_fwd(g, dev(x), dev(g_in), dev(W), dev(bias), relu=relu)
    assert torch.equal(yd, yd2)


@pytest.mark.parametrize("lattice,f", [("cubic", 3), ("cubic", 2), ("tetrahedral", 3),
                                       ("triangular", 3)])
def test_dense_matches_pair_lists(scn, lattice, f):
    """The view leaves the rulebook unchanged, and the forward with and
    without it both match the oracle."""
    rng = stream_rng(171, _K(lattice, f))
    coords, grid = _sites(lattice, rng, 2, 28, 2500)
    Cin, Cout = 32, 48
    K = _K(lattice, f)
    x = rng.standard_normal((len(coords), Cin)).astype(np.float32)
    g_in = (rng.standard_normal(Cin) * 0.5).astype(np.float32)
    W = (rng.standard_normal((K, Cin, Cout)) / np.sqrt(K * Cin)).astype(np.float32)
    bias = (rng.standard_normal(Cout) * 0.1).astype(np.float32)
    gd = scn.build_rulebook(dev(coords), grid, f, 1, lattice=lattice)
    scn.set_dense_forward(1 << 62, 1)  # no view
    try:
        gp = scn.build_rulebook(dev(coords), grid, f, 1, lattice=lattice)
    finally:
        scn.set_dense_forward(0, 1)
    assert gd.dense_view and not gp.dense_view
    for a, b in zip(gd.export(), gp.export()):
        assert torch.equal(a, b)
    o = oracle.Rulebook(coords, grid, f, 1, lattice=lattice)
    y_ref, go_ref = oracle.conv_fwd(o, x, g_in, W, bias, relu=True)
    for name, g in (("dense view", gd), ("pair lists", gp)):
        yd, god = scn.conv_fwd(g, dev(x), dev(g_in), dev(W), dev(bias), relu=True)
        assert_site(f"y ({name})", host(yd), y_ref)
        assert_site(f"g_out ({name})", host(god), go_ref)


def test_dense_empty_and_strided(scn):
    """No outputs: nothing to launch.  Strided rulebooks never carry the view
    and still match the oracle."""
    g = scn.build_rulebook(dev(np.zeros((0, 4), np.int32)), (1, 8, 8, 8), 3, 1)
    y, go = scn.conv_fwd(g, dev(np.zeros((0, 4), np.float32)), dev(np.zeros(4, np.float32)),
                         dev(np.ones((27, 4, 8), np.float32)), None)
    assert y.shape == (0, 8)
    rng = stream_rng(172, 0)
    coords, grid = _sites("cubic", rng, 1, 25, 1500)
    x = rng.standard_normal((len(coords), 16)).astype(np.float32)
    g_in = (rng.standard_normal(16) * 0.5).astype(np.float32)
    W = (rng.standard_normal((8, 16, 24)) / 8).astype(np.float32)
    g = scn.build_rulebook(dev(coords), grid, 2, 2)
    o = oracle.Rulebook(coords, grid, 2, 2)
    assert not g.dense_view
    y_ref, _ = oracle.conv_fwd(o, x, g_in, W, None)
    yd, _ = scn.conv_fwd(g, dev(x), dev(g_in), dev(W), None)
    assert_site("y strided", host(yd), y_ref)


# single-channel layers with the view, forward and backward, across column
# counts (odd, under and over 64) and lattices
C1_CASES = [
    ("cubic", 3, 1, 22, 1500, 64, True, True),
    ("cubic", 2, 2, 18, 1600, 7, False, True),
    ("tetrahedral", 3, 1, 24, 1500, 33, True, True),
    ("square", 3, 2, 40, 1500, 64, False, False),
    ("triangular", 3, 1, 50, 900, 20, True, True),
    ("cubic", 3, 1, 20, 1200, 96, True, True),
]


@pytest.mark.parametrize("case", C1_CASES, ids=[f"{c[0]}{i}" for i, c in enumerate(C1_CASES)])
def test_single_channel_fwd_bwd(scn, case):
    lattice, f, B, m, n, Cout, relu, shuffle = case
    i = C1_CASES.index(case)
    rng = stream_rng(175, i)
    coords, grid = _sites(lattice, rng, B, m, n, shuffle)
    K = _K(lattice, f)
    x = rng.standard_normal((len(coords), 1)).astype(np.float32)
    g_in = (rng.standard_normal(1) * 0.5).astype(np.float32)
    W = (rng.standard_normal((K, 1, Cout)) / np.sqrt(K)).astype(np.float32)
    bias = (rng.standard_normal(Cout) * 0.1).astype(np.float32)
    g = scn.build_rulebook(dev(coords), grid, f, 1, lattice=lattice)
    o = oracle.Rulebook(coords, grid, f, 1, lattice=lattice)
    assert g.dense_view
    conv_parity(scn, g, o, x, g_in, W, bias, relu, 300 + i)
