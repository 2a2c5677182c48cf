"""GPU parity: the HIP library (through its C ABI) against the CPU oracle on
seeded small inputs that span several tiles and ragged tails.

Bars: rulebooks, active sets, pooling outputs, argmax and pooling input
gradients bit-exact; fp32 features and gradients within 1e-5 absolute and
1e-4 relative (per-site results under the plain rule, reductions over pairs
relative to max(|ref|, rss of the summed terms); ``tests/helpers.py``).
"""
from __future__ import annotations

import numpy as np
import pytest

torch = pytest.importorskip("torch")

import oracle  # noqa: E402
from gen import random_sites, stream_rng  # noqa: E402

from helpers import (assert_reduction, assert_site, conv_parity, dev, host, keys_of,  # noqa: E402
                     pool_parity, sq)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def scn():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_1505_02890_amd as m
    m.lib()  # raises if the HIP library is missing
    return m


def _rb_pair(scn, coords, grid, f, s):
    g = scn.build_rulebook(dev(coords, torch.int32), grid, f, s)
    o = oracle.Rulebook(coords, grid, f, s)
    return g, o


def _check_rulebook(g, o):
    oa = o.arrays()
    assert (g.a_in, g.a_out, g.n_pairs, g.K) == (oa.a_in, oa.a_out, oa.n_pairs, oa.K)
    assert tuple(g.out_grid) == tuple(oa.out_grid)
    assert np.array_equal(g.offsets, oa.offsets)
    oc, ir, orr = g.export()
    assert np.array_equal(host(oc), oa.out_coords)
    assert np.array_equal(host(ir), oa.in_rows)
    assert np.array_equal(host(orr), oa.out_rows)


RB_CASES = [
    # (B, dims, n, f, s, shuffle)
    (1, (8, 8, 8), 60, 2, 1, True),
    (2, (8, 8, 8), 200, 3, 1, True),
    (3, (70, 5, 9), 400, 2, 1, False),
    (2, (33, 40, 3), 500, 3, 1, True),
    (2, (40, 3, 35), 300, 2, 2, True),
    (1, (65, 9, 10), 700, 3, 2, True),
    (2, (11, 10, 9), 250, 3, 3, True),
    (1, (7, 7, 7), 343, 2, 1, True),     # every site active
    (1, (7, 7, 7), 343, 2, 2, False),
    (2, (9, 6, 7), 100, 1, 1, True),
    (1, (100, 3, 3), 80, 2, 3, True),    # stride above filter (gaps)
    (4, (1, 1, 1), 4, 1, 1, True),       # one site per sample
    (1, (2, 9, 9), 50, 3, 1, True),      # an axis shorter than the filter: no outputs
    (1, (130, 4, 4), 600, 2, 2, True),   # x-rows spanning several words, odd extent
]


@pytest.mark.parametrize("case", RB_CASES, ids=[str(i) for i in range(len(RB_CASES))])
def test_rulebook_bit_exact(scn, case):
    B, dims, n, f, s, shuf = case
    rng = stream_rng(11, hash(case) & 0xFFFF)
    coords = random_sites(rng, B, dims, n, shuffle=shuf)
    g, o = _rb_pair(scn, coords, (B,) + tuple(dims), f, s)
    _check_rulebook(g, o)
    assert g.input_sorted == bool(np.all(np.diff(keys_of(coords, (B,) + tuple(dims))) > 0))


def test_rulebook_empty(scn):
    coords = np.zeros((0, 4), np.int32)
    g, o = _rb_pair(scn, coords, (2, 5, 5, 5), 2, 1)
    assert g.a_out == 0 and g.n_pairs == 0
    _check_rulebook(g, o)


def test_rulebook_figure3(scn):
    coords = np.array([[0, 2, 2, 0], [0, 3, 2, 0], [0, 4, 2, 0]], np.int32)
    g, o = _rb_pair(scn, coords, (1, 6, 6, 2), 2, 1)
    assert g.out_grid == (1, 5, 5, 1) and g.a_out == 8
    _check_rulebook(g, o)


def test_rulebook_errors(scn):
    grid = (2, 6, 6, 6)
    dup = np.array([[0, 1, 1, 1], [1, 2, 3, 4], [0, 1, 1, 1]], np.int32)
    with pytest.raises(scn.ScnError) as e:
        scn.build_rulebook(dev(dup), grid, 2, 1)
    assert e.value.status == "duplicate"
    for bad in ([2, 0, 0, 0], [0, 6, 0, 0], [0, 0, -1, 0], [0, 0, 0, 6], [-1, 0, 0, 0]):
        c = np.array([[0, 1, 1, 1], bad], np.int32)
        with pytest.raises(scn.ScnError) as e:
            scn.build_rulebook(dev(c), grid, 2, 1)
        assert e.value.status == "range", bad
    ok = np.array([[0, 1, 1, 1]], np.int32)
    with pytest.raises(scn.ScnError) as e:
        scn.build_rulebook(dev(ok), grid, 4, 1)
    assert e.value.status == "unsupported"
    with pytest.raises(scn.ScnError) as e:
        scn.build_rulebook(dev(ok), grid, 2, 0)
    assert e.value.status == "invalid"
    # a grid past the occupancy bitmaps builds through the keyed builder
    big = scn.build_rulebook(dev(ok), (1, 1 << 20, 1 << 10, 1 << 10), 2, 1)
    assert big.keyed and (big.a_in, big.a_out, big.n_pairs) == (1, 8, 8)
    # misaligned coordinate pointer (offset by one int32)
    flat = dev(np.zeros(9, np.int32))
    with pytest.raises(scn.ScnError) as e:
        scn.build_rulebook(flat[1:].view(2, 4), grid, 2, 1)
    assert e.value.status == "invalid"


# --------------------------------------------------------------------------
# convolution
# --------------------------------------------------------------------------

CONV_CASES = [
    # (f, s, B, dims, n, Cin, Cout, relu)
    (2, 1, 2, (10, 9, 11), 300, 1, 16, False),
    (2, 1, 1, (12, 12, 12), 500, 16, 32, True),
    (3, 1, 2, (9, 10, 8), 400, 17, 3, True),
    (3, 1, 1, (40, 12, 10), 900, 64, 64, False),
    (2, 2, 2, (11, 10, 9), 300, 32, 96, True),
    (3, 2, 1, (13, 12, 11), 400, 3, 160, False),
    (1, 1, 1, (6, 6, 6), 50, 5, 7, False),
    (3, 3, 1, (12, 9, 10), 300, 8, 8, True),
    (2, 1, 1, (70, 40, 3), 1500, 96, 128, True),
    (2, 1, 1, (40, 30, 2), 600, 224, 256, False),
    (2, 1, 3, (20, 20, 20), 2500, 64, 64, True),
]


def _conv_inputs(case, seed):
    f, s, B, dims, n, Cin, Cout, relu = case
    rng = stream_rng(seed, 1)
    coords = random_sites(rng, B, dims, n)
    K = f ** 3
    x = rng.standard_normal((len(coords), Cin)).astype(np.float32)
    g_in = (rng.standard_normal(Cin) * 0.5).astype(np.float32)
    W = (rng.standard_normal((K, Cin, Cout)) / np.sqrt(K * Cin)).astype(np.float32)
    bias = (rng.standard_normal(Cout) * 0.1).astype(np.float32)
    return coords, (B,) + tuple(dims), x, g_in, W, bias


def _conv_check(scn, case, inputs, seed):
    f, s, B, dims, n, Cin, Cout, relu = case
    coords, grid, x, g_in, W, bias = inputs
    g, o = _rb_pair(scn, coords, grid, f, s)
    _check_rulebook(g, o)
    conv_parity(scn, g, o, x, g_in, W, bias, relu, seed)
    return g


@pytest.mark.parametrize("case", CONV_CASES, ids=[str(i) for i in range(len(CONV_CASES))])
def test_conv_fwd_bwd_parity(scn, case):
    i = CONV_CASES.index(case)
    _conv_check(scn, case, _conv_inputs(case, 100 + i), 200 + i)


@pytest.mark.parametrize("case", [CONV_CASES[2], CONV_CASES[4], CONV_CASES[10]],
                         ids=["f3s1", "f2s2", "f2s1-64"])
def test_conv_sorted_input(scn, case):
    """Sites listed in key order: the rulebook keeps no rank-to-row table and
    the input gradient writes ranks directly."""
    coords, grid, x, g_in, W, bias = _conv_inputs(case, 400 + CONV_CASES.index(case))
    order = np.argsort(keys_of(coords, grid), kind="stable")
    g = _conv_check(scn, case, (coords[order], grid, x[order], g_in, W, bias),
                    500 + CONV_CASES.index(case))
    assert g.input_sorted


def test_conv_without_bias_and_partial_outputs(scn):
    case = (3, 1, 1, (10, 11, 12), 350, 12, 20, False)
    coords, grid, x, g_in, W, _ = _conv_inputs(case, 7)
    g, o = _rb_pair(scn, coords, grid, 3, 1)
    y_ref, go_ref = oracle.conv_fwd(o, x, g_in, W, None)
    yd, god = scn.conv_fwd(g, dev(x), dev(g_in), dev(W), None)
    assert_site("y", host(yd), y_ref)
    assert_site("g_out", host(god), go_ref)
    dy = stream_rng(8, 1).uniform(-1, 1, size=(g.a_out, 20)).astype(np.float32)
    ref = oracle.conv_bwd(o, x, g_in, W, None, dy, None)
    sig = {k: np.sqrt(v) for k, v in
           oracle.conv_bwd(o, sq(x), sq(g_in), sq(W), None, sq(dy), None).items()}
    for need in (("dx",), ("dW",), ("dg_in",), ("dbias", "dx")):
        out = scn.conv_bwd(g, dev(x), dev(g_in), dev(W), None, None, dev(dy), None, need=need)
        assert set(out) == set(need)
        for k in need:
            if k == "dx":
                assert_site(k, host(out[k]), ref[k])
            else:
                assert_reduction(k, host(out[k]), ref[k], sig[k])


def test_conv_empty_input_gives_ground_state(scn):
    coords = np.zeros((0, 4), np.int32)
    g, o = _rb_pair(scn, coords, (1, 6, 6, 6), 2, 1)
    rng = stream_rng(9, 0)
    g_in = rng.standard_normal(4).astype(np.float32)
    W = rng.standard_normal((8, 4, 6)).astype(np.float32)
    b = rng.standard_normal(6).astype(np.float32)
    x = np.zeros((0, 4), np.float32)
    for relu in (False, True):
        yd, god = scn.conv_fwd(g, dev(x), dev(g_in), dev(W), dev(b), relu=relu)
        _, go_ref = oracle.conv_fwd(o, x, g_in, W, b, relu=relu)
        assert yd.shape == (0, 6)
        assert_site("g_out", host(god), go_ref)


def test_conv_deterministic(scn):
    case = (3, 1, 2, (16, 14, 12), 1500, 64, 64, True)
    coords, grid, x, g_in, W, bias = _conv_inputs(case, 31)
    g = scn.build_rulebook(dev(coords), grid, 3, 1)
    dy = dev(stream_rng(32, 0).uniform(-1, 1, size=(g.a_out, 64)).astype(np.float32))
    res = []
    for _ in range(2):
        y, go = scn.conv_fwd(g, dev(x), dev(g_in), dev(W), dev(bias), relu=True)
        out = scn.conv_bwd(g, dev(x), dev(g_in), dev(W), y, go, dy, None, relu=True)
        res.append([host(t) for t in (y, go, out["dx"], out["dW"], out["dbias"], out["dg_in"])])
    for a, b in zip(*res):
        assert np.array_equal(a.view(np.uint32), b.view(np.uint32))


def test_conv_workspace_checked(scn):
    case = (2, 1, 1, (8, 8, 8), 100, 4, 4, False)
    coords, grid, x, g_in, W, bias = _conv_inputs(case, 5)
    g = scn.build_rulebook(dev(coords), grid, 2, 1)
    dy = dev(np.ones((g.a_out, 4), np.float32))
    small = torch.empty(16, dtype=torch.uint8, device="cuda")
    with pytest.raises(scn.ScnError) as e:
        scn.conv_bwd(g, dev(x), dev(g_in), dev(W), None, None, dy, ws=small)
    assert e.value.status == "workspace"


# --------------------------------------------------------------------------
# max-pooling
# --------------------------------------------------------------------------

POOL_CASES = [
    # (f, s, B, dims, n, C, zero_frac, g_scale)
    (2, 2, 2, (12, 11, 10), 500, 16, 0.0, 0.5),
    (2, 2, 1, (9, 9, 9), 400, 1, 0.5, 0.0),     # many exact ties with g = 0
    (2, 2, 3, (70, 6, 7), 900, 33, 0.3, 0.0),
    (3, 3, 1, (13, 14, 12), 600, 8, 0.0, 2.0),  # ground state often the maximum
    (2, 2, 1, (8, 8, 8), 512, 64, 0.2, -0.1),   # every site active
    (3, 2, 1, (13, 14, 12), 600, 16, 0.0, 0.5),  # overlapping windows (MP3/2)
    (3, 2, 2, (9, 11, 10), 500, 5, 0.3, 0.0),    # MP3/2, one channel per thread, ties
    (3, 2, 1, (7, 7, 7), 343, 64, 0.2, 0.1),     # MP3/2, every site active
    (3, 2, 2, (30, 9, 8), 900, 12, 0.0, 1.5),    # MP3/2, ground state often wins
    (2, 3, 1, (14, 13, 11), 500, 8, 0.0, 0.5),   # gaps between windows
    (1, 2, 2, (15, 12, 11), 700, 8, 0.0, 0.5),   # one-site windows (K = 1)
    (3, 2, 1, (40, 33, 30), 6000, 4, 0.1, 0.3),  # MP3/2 over many output waves, ragged last
]


@pytest.mark.parametrize("case", POOL_CASES, ids=[str(i) for i in range(len(POOL_CASES))])
def test_maxpool_parity(scn, case):
    f, s, B, dims, n, C, zf, gs = case
    rng = stream_rng(300 + POOL_CASES.index(case), 0)
    coords = random_sites(rng, B, dims, n)
    x = rng.standard_normal((len(coords), C)).astype(np.float32)
    x[rng.random(x.shape) < zf] = 0.0
    g_in = (np.abs(rng.standard_normal(C)) * gs).astype(np.float32)
    grid = (B,) + tuple(dims)
    g, o = _rb_pair(scn, coords, grid, f, s)
    _check_rulebook(g, o)
    pool_parity(scn, g, o, x, g_in, rng, f > s)


# Block counts around the runs of consecutive blocks that each XCD takes
# (3x3x3 windows: runs of up to 16 forward blocks and 32 cell-backward
# blocks; 2x2x2: 128 forward blocks; at most an eighth of the blocks; the
# launch is rounded up to whole rounds of 8 runs):
# fully active boxes give exact window counts.  (f, s, box edge, channels)
RUN_CASES = [
    (3, 2, 7, 64),    # 27 windows: 2 blocks, runs of 1
    (3, 2, 37, 64),   # 5832 windows: 365 blocks, runs of 16, a ragged last round
    (3, 2, 35, 4),    # 4913 windows, 256 a block: 20 blocks, runs of 2
    (2, 2, 32, 64),   # 4096 windows: 256 blocks, runs of 32, whole rounds
    (2, 2, 66, 64),   # 35937 windows: 2247 blocks, runs of 128, a ragged last round
]


@pytest.mark.parametrize("case", RUN_CASES, ids=[str(i) for i in range(len(RUN_CASES))])
def test_maxpool_block_runs(scn, case):
    f, s, m, C = case
    rng = stream_rng(420 + RUN_CASES.index(case), 0)
    g3 = np.stack(np.meshgrid(np.arange(m), np.arange(m), np.arange(m), indexing="ij"), -1)
    coords = np.concatenate([np.zeros((m ** 3, 1), np.int64), g3.reshape(-1, 3)], 1)
    coords = np.ascontiguousarray(coords[rng.permutation(len(coords))].astype(np.int32))
    x = rng.standard_normal((len(coords), C)).astype(np.float32)
    g_in = (np.abs(rng.standard_normal(C)) * 0.3).astype(np.float32)
    grid = (1, m, m, m)
    g, o = _rb_pair(scn, coords, grid, f, s)
    assert g.a_out == ((m - f) // s + 1) ** 3
    pool_parity(scn, g, o, x, g_in, rng, f > s)


def test_maxpool_needs_stride_two(scn):
    coords = random_sites(stream_rng(1, 1), 1, (8, 8, 8), 50)
    g = scn.build_rulebook(dev(coords), (1, 8, 8, 8), 2, 1)
    x = dev(np.ones((50, 4), np.float32))
    with pytest.raises(scn.ScnError) as e:
        scn.maxpool_fwd(g, x, dev(np.zeros(4, np.float32)))
    assert e.value.status == "unsupported"
