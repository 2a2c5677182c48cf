"""The full-size parity tests check GPU rulebooks against a numpy evaluation
of the rulebook's definition on a dense occupancy grid
(helpers.definition_rulebook).  These CPU tests pin that evaluation to the
oracle's std::map rulebook, and to brute force over every output window, on
small inputs with every filter and stride the workloads use."""
from __future__ import annotations

import itertools

import numpy as np
import pytest

import oracle
from gen import random_sites, stream_rng
from helpers import definition_rulebook


@pytest.mark.parametrize("f,s", [(1, 1), (2, 1), (3, 1), (2, 2), (3, 2), (3, 3), (2, 3)])
def test_definition_matches_oracle(f, s):
    rng = stream_rng(61, 10 * f + s)
    grid = (3, 13, 11, 9)
    coords = random_sites(rng, grid[0], grid[1:], 400)
    oc, off, ir, orr = definition_rulebook(coords, grid, f, s)
    oa = oracle.Rulebook(coords, grid, f, s).arrays()
    assert np.array_equal(oc, oa.out_coords)
    assert np.array_equal(off, oa.offsets)
    assert np.array_equal(ir, oa.in_rows)
    assert np.array_equal(orr, oa.out_rows)


def test_definition_brute_force():
    """Every output window of a tiny grid, enumerated directly."""
    rng = stream_rng(62, 0)
    grid = (2, 6, 5, 7)
    coords = random_sites(rng, 2, grid[1:], 40)
    occ = {tuple(c): r for r, c in enumerate(coords.tolist())}
    for f, s in ((2, 1), (3, 2)):
        oc, off, ir, orr = definition_rulebook(coords, grid, f, s)
        outs = []
        for b in range(grid[0]):
            for z, y, x in itertools.product(*(range((m - f) // s + 1) for m in grid[:0:-1])):
                if any((b, s * x + kx, s * y + ky, s * z + kz) in occ
                       for kz in range(f) for ky in range(f) for kx in range(f)):
                    outs.append((b, x, y, z))
        assert oc.tolist() == [list(o) for o in outs]
        K = f ** 3
        for k in range(K):
            kx, ky, kz = k % f, (k // f) % f, k // (f * f)
            want = [(occ[(b, s * x + kx, s * y + ky, s * z + kz)], o)
                    for o, (b, x, y, z) in enumerate(outs)
                    if (b, s * x + kx, s * y + ky, s * z + kz) in occ]
            got = list(zip(ir[off[k]:off[k + 1]].tolist(), orr[off[k]:off[k + 1]].tolist()))
            assert got == want


def test_definition_empty_grid():
    oc, off, ir, orr = definition_rulebook(np.zeros((0, 4), np.int32), (1, 2, 5, 5), 3, 1)
    assert oc.shape == (0, 4) and len(ir) == 0 and np.all(off == 0)
