"""GPU parity on the 2D lattices of Figure 2 (i) and (ii): rulebooks,
convolution and max-pooling on square and triangular rulebooks against the
oracle, through the C ABI.  Same bars as the 3D tests."""
from __future__ import annotations

import ctypes
import math

import numpy as np
import pytest

torch = pytest.importorskip("torch")

import oracle  # noqa: E402
from gen import random_sites, stream_rng, tri_random_sites  # noqa: E402

from helpers import conv_parity, dev, host, pool_parity  # noqa: E402

pytestmark = pytest.mark.gpu
SQ, TRI = "square", "triangular"


@pytest.fixture(scope="module")
def scn():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_1505_02890_amd as m
    m.lib()  # raises if the HIP library is missing
    return m


def _sites(lattice, rng, B, m, n, shuffle=True):
    if lattice == SQ:
        return random_sites(rng, B, (m, m, 1), n, shuffle=shuffle)
    return tri_random_sites(rng, B, m, n, shuffle=shuffle)


def _pair(scn, lattice, coords, grid, f, s):
    g = scn.build_rulebook(dev(coords, torch.int32), grid, f, s, lattice=lattice)
    o = oracle.Rulebook(coords, grid, f, s, lattice=lattice)
    return g, o


def _check_rulebook(g, o, lattice):
    oa = o.arrays()
    assert g.lattice == lattice
    assert (g.a_in, g.a_out, g.n_pairs, g.K) == (oa.a_in, oa.a_out, oa.n_pairs, oa.K)
    assert tuple(g.out_grid) == tuple(oa.out_grid) and g.out_grid[3] == 1
    assert np.array_equal(g.offsets, oa.offsets)
    oc, ir, orr = g.export()
    assert np.array_equal(host(oc), oa.out_coords)
    assert np.array_equal(host(ir), oa.in_rows)
    assert np.array_equal(host(orr), oa.out_rows)


RB_CASES = [
    # (lattice, B, m, n, f, s, shuffle)
    (SQ, 2, 20, 150, 2, 1, True),
    (SQ, 3, 70, 900, 3, 1, False),     # x-rows of three words
    (SQ, 2, 41, 500, 3, 2, True),
    (SQ, 1, 12, 144, 2, 2, True),      # every site active
    (SQ, 2, 30, 200, 2, 3, True),      # gaps
    (TRI, 2, 20, 120, 2, 1, True),
    (TRI, 3, 70, 900, 3, 1, False),
    (TRI, 2, 41, 500, 3, 2, True),
    (TRI, 1, 11, 66, 3, 2, True),      # every site active, MP3/2
    (TRI, 2, 9, 30, 1, 1, True),
    (TRI, 1, 2, 3, 3, 1, True),        # grid smaller than the filter
]


@pytest.mark.parametrize("case", RB_CASES, ids=[str(i) for i in range(len(RB_CASES))])
def test_rulebook_bit_exact(scn, case):
    lattice, B, m, n, f, s, shuf = case
    rng = stream_rng(71, RB_CASES.index(case))
    coords = _sites(lattice, rng, B, m, n, shuf)
    g, o = _pair(scn, lattice, coords, (B, m, m, 1), f, s)
    _check_rulebook(g, o, lattice)
    assert g.K == (f * f if lattice == SQ else math.comb(f + 1, 2))


def test_rulebook_errors(scn):
    ok = np.array([[0, 1, 1, 0]], np.int32)
    for lattice in (SQ, TRI):
        with pytest.raises(scn.ScnError) as e:          # a 2D grid has one plane
            scn.build_rulebook(dev(ok), (1, 6, 6, 2), 2, 1, lattice=lattice)
        assert e.value.status == "invalid"
        with pytest.raises(scn.ScnError) as e:          # z must be 0
            scn.build_rulebook(dev(np.array([[0, 1, 1, 1]], np.int32)), (1, 6, 6, 1), 2, 1,
                               lattice=lattice)
        assert e.value.status == "range"
    with pytest.raises(scn.ScnError) as e:              # 4 + 2 >= 6
        scn.build_rulebook(dev(np.array([[0, 4, 2, 0]], np.int32)), (1, 6, 6, 1), 2, 1,
                           lattice=TRI)
    assert e.value.status == "range"
    with pytest.raises(scn.ScnError) as e:
        scn.build_rulebook(dev(ok), (1, 6, 7, 1), 2, 1, lattice=TRI)
    assert e.value.status == "invalid"
    from paper_1505_02890_amd import _lib
    h = ctypes.c_void_p()
    g4 = np.array([1, 6, 6, 1], np.int64)
    d = dev(ok)
    rc = _lib.lib().scn_rulebook_build_lattice(
        ctypes.c_void_p(d.data_ptr()), 1, g4.ctypes.data_as(ctypes.c_void_p), 2, 1, 4,
        ctypes.c_void_p(torch.cuda.current_stream().cuda_stream), ctypes.byref(h))
    assert rc == 1 and not h.value                      # unknown lattice: invalid


CONV_CASES = [
    # (lattice, f, s, B, m, n, Cin, Cout, relu)
    (SQ, 2, 1, 2, 30, 400, 3, 32, True),
    (SQ, 3, 1, 1, 40, 700, 64, 64, False),
    (SQ, 2, 2, 2, 33, 500, 17, 5, True),
    (SQ, 2, 1, 1, 40, 1600, 96, 96, True),     # dense
    (TRI, 2, 1, 2, 30, 300, 3, 32, True),
    (TRI, 3, 1, 1, 50, 900, 64, 64, False),
    (TRI, 2, 2, 2, 33, 400, 17, 5, True),
    (TRI, 2, 1, 1, 50, 1275, 96, 96, True),    # dense
]


@pytest.mark.parametrize("case", CONV_CASES, ids=[str(i) for i in range(len(CONV_CASES))])
def test_conv_fwd_bwd_parity(scn, case):
    lattice, f, s, B, m, n, Cin, Cout, relu = case
    seed = 720 + CONV_CASES.index(case)
    rng = stream_rng(seed, 1)
    coords = _sites(lattice, rng, B, m, n)
    K = f * f if lattice == SQ else math.comb(f + 1, 2)
    x = rng.standard_normal((len(coords), Cin)).astype(np.float32)
    g_in = (rng.standard_normal(Cin) * 0.5).astype(np.float32)
    W = (rng.standard_normal((K, Cin, Cout)) / np.sqrt(K * Cin)).astype(np.float32)
    bias = (rng.standard_normal(Cout) * 0.1).astype(np.float32)
    g, o = _pair(scn, lattice, coords, (B, m, m, 1), f, s)
    _check_rulebook(g, o, lattice)
    conv_parity(scn, g, o, x, g_in, W, bias, relu, seed)


POOL_CASES = [
    # (lattice, f, s, B, m, n, C, zero_frac, g_scale)
    (SQ, 3, 2, 1, 41, 900, 16, 0.0, 0.5),     # MP3/2 (9-site regions)
    (SQ, 2, 2, 2, 30, 500, 5, 0.3, 0.0),
    (SQ, 3, 2, 1, 21, 441, 64, 0.2, 0.1),     # dense
    (TRI, 3, 2, 1, 41, 700, 16, 0.0, 0.5),    # MP3/2 (6-site regions)
    (TRI, 3, 2, 2, 31, 400, 5, 0.3, 0.0),     # one channel per thread, ties
    (TRI, 3, 2, 1, 21, 231, 64, 0.2, 0.1),    # dense
    (TRI, 2, 2, 2, 30, 400, 12, 0.0, 1.5),    # 3-site regions, gaps
]


@pytest.mark.parametrize("case", POOL_CASES, ids=[str(i) for i in range(len(POOL_CASES))])
def test_maxpool_parity(scn, case):
    lattice, f, s, B, m, n, C, zf, gs = case
    rng = stream_rng(740 + POOL_CASES.index(case), 0)
    coords = _sites(lattice, rng, B, m, n)
    x = rng.standard_normal((len(coords), C)).astype(np.float32)
    x[rng.random(x.shape) < zf] = 0.0
    g_in = (np.abs(rng.standard_normal(C)) * gs).astype(np.float32)
    g, o = _pair(scn, lattice, coords, (B, m, m, 1), f, s)
    _check_rulebook(g, o, lattice)
    pool_parity(scn, g, o, x, g_in, rng, f > s)
