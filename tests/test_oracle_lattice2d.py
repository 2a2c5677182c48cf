"""Pins of the oracle's 2D lattices (Figure 2 (i) and (ii)) against things
other than itself (CPU only).

Reading: a 2D grid is a grid with mz = 1 whose sites have z = 0.  The square
lattice takes the f^2 offsets (kx, ky, 0); the triangular lattice is held in
skewed coordinates (sites x + y < m, mx = my = m) with the C(f+1, 2)
offsets kx + ky < f, numbered in the square scan order restricted to them.
An output exists where its whole window lies in the grid.

* counts the paper states: f^2 and C(f+1, 2) sites per filter; Figure 2 (i)
  and (ii); the worked example of Figure 3 in true 2D; triangular MP3/2
  regions of 6 sites that cover the grid and overlap by one site;
* dense equivalence: torch conv2d / max_pool2d (float64) of the field that
  holds M_in at active sites and g_in elsewhere, with the weights zero outside
  the triangle on the triangular lattice;
* brute-force active sets; dense autograd for the gradients.
"""
import math
import os

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import gen
import oracle

HERE = os.path.dirname(os.path.abspath(__file__))
SQ, TRI = "square", "triangular"


def offsets(f, lattice):
    return [(kx, ky) for ky in range(f) for kx in range(f) if lattice == SQ or kx + ky < f]


def out_size(m, f, s):
    return (m - f) // s + 1 if m >= f else 0


def valid_mask(B, mx, my, f, s, lattice):
    qx, qy = out_size(mx, f, s), out_size(my, f, s)
    v = np.zeros((B, qy, qx), bool)
    for oy in range(qy):
        for ox in range(qx):
            v[:, oy, ox] = lattice == SQ or s * (ox + oy) + f - 1 < mx
    return v


def field2d(coords, feats, g, B, mx, my):
    """[B, C, Y, X]: feats at active sites, g elsewhere (autograd to both)."""
    C = feats.shape[1]
    c = torch.as_tensor(np.asarray(coords, np.int64))
    vals = torch.zeros(B, my, mx, C, dtype=torch.float64)
    vals = vals.index_put((c[:, 0], c[:, 2], c[:, 1]), feats)
    mask = torch.zeros(B, my, mx, 1, dtype=torch.float64)
    mask[c[:, 0], c[:, 2], c[:, 1]] = 1.0
    return (mask * vals + (1.0 - mask) * g.view(1, 1, 1, C)).permute(0, 3, 1, 2)


def weight2d(W, f, lattice):
    K, Cin, Cout = W.shape
    Wc = torch.zeros(f, f, Cin, Cout, dtype=torch.float64)
    for k, (kx, ky) in enumerate(offsets(f, lattice)):
        Wc[ky, kx] = W[k]
    return Wc.permute(3, 2, 0, 1)


def sites(lattice, rng, B, m, n):
    if lattice == SQ:
        return gen.random_sites(rng, B, (m, m, 1), n)
    return gen.tri_random_sites(rng, B, m, n)


def full(lattice, m):
    cell = gen.triangle_sites(m) if lattice == TRI else \
        np.array([(x, y, 0) for y in range(m) for x in range(m)], np.int64)
    return np.concatenate([np.zeros((len(cell), 1), np.int64), cell], axis=1).astype(np.int32)


# ---------------------------------------------------------------- counts

@pytest.mark.parametrize("lattice", [SQ, TRI])
@pytest.mark.parametrize("f", [1, 2, 3, 4])
def test_filter_sizes(lattice, f):
    """f^2 sites per square filter, C(f+1, 2) per triangular one (3 for the
    smallest, 6 for MP3)."""
    coords = np.array([[0, f - 1, f - 1, 0]], np.int32)
    m = 3 * f
    rb = oracle.Rulebook(coords, (1, m, m, 1), f, 1, lattice=lattice)
    want = f * f if lattice == SQ else math.comb(f + 1, 2)
    assert rb.K == want == rb.a_out == rb.n_pairs
    assert rb.out_grid[3] == 1


@pytest.mark.parametrize("lattice,m,n_out", [(SQ, 4, 9), (TRI, 4, 6)])
def test_figure2_small_grids(lattice, m, n_out):
    """Figure 2 (i): a 4x4 square grid under a 2x2 filter (3x3 outputs, 4
    inputs each); (ii): a triangular grid of size 4 (10 sites) under a filter
    of size 2 (a grid of size 3, 6 outputs, 3 inputs each)."""
    coords = full(lattice, m)
    assert len(coords) == (16 if lattice == SQ else 10)
    rb = oracle.Rulebook(coords, (1, m, m, 1), 2, 1, lattice=lattice)
    assert rb.a_out == n_out
    assert rb.n_pairs == n_out * (4 if lattice == SQ else 3)


def test_figure3_in_two_dimensions():
    """The worked example of Figure 3 on the square lattice proper (the cubic
    pin embeds the same sites in a grid two planes deep)."""
    spec, pts = {}, []
    for line in open(os.path.join(HERE, "golden", "fig3_example.txt")):
        line = line.split("#")[0].split()
        if not line:
            continue
        if line[0] == "site":
            pts.append([int(v) for v in line[1:]])
        else:
            spec[line[0]] = [int(v) for v in line[1:]]
    grid = spec["grid"][:3] + [1]
    rb = oracle.Rulebook(np.array(pts, np.int32), grid, spec["filter"][0], spec["stride"][0],
                         lattice=SQ)
    assert list(rb.out_grid[1:3]) == spec["out_extent"][:2] and rb.out_grid[3] == 1
    assert rb.a_out == spec["active_out"][0]


def test_triangular_mp32_regions_cover_and_overlap_by_one():
    """Triangular MP3/2 on a full grid of size 2q + 1: every region holds 6
    sites, every site lies in some region, and regions at adjacent output
    sites share exactly one site."""
    m = 11
    coords = full(TRI, m)
    rb = oracle.Rulebook(coords, (1, m, m, 1), 3, 2, lattice=TRI)
    a = rb.arrays()
    members = [set() for _ in range(rb.a_out)]
    for i, o in zip(a.in_rows, a.out_rows):
        members[o].add(int(i))
    assert all(len(s) == 6 for s in members)
    assert set().union(*members) == set(range(len(coords)))
    pos = {tuple(c[1:3]): o for o, c in enumerate(a.out_coords.tolist())}
    n_adj = 0
    for p, o in pos.items():
        for d in ((1, 0), (0, 1), (1, -1)):
            q = (p[0] + d[0], p[1] + d[1])
            if q in pos:
                assert len(members[o] & members[pos[q]]) == 1
                n_adj += 1
    assert n_adj > 0


def test_statuses():
    with pytest.raises(oracle.OracleError) as e:      # a 2D grid has one plane
        oracle.Rulebook(np.array([[0, 1, 1, 0]], np.int32), (1, 5, 5, 2), 2, 1, lattice=SQ)
    assert e.value.status == "invalid"
    with pytest.raises(oracle.OracleError) as e:      # 3 + 2 >= 5
        oracle.Rulebook(np.array([[0, 3, 2, 0]], np.int32), (1, 5, 5, 1), 2, 1, lattice=TRI)
    assert e.value.status == "range"
    with pytest.raises(oracle.OracleError) as e:
        oracle.Rulebook(np.array([[0, 0, 0, 0]], np.int32), (1, 5, 6, 1), 2, 1, lattice=TRI)
    assert e.value.status == "invalid"
    with pytest.raises(oracle.OracleError) as e:      # z must be 0
        oracle.Rulebook(np.array([[0, 0, 0, 1]], np.int32), (1, 5, 5, 1), 2, 1, lattice=SQ)
    assert e.value.status == "range"


# ---------------------------------------------------------------- dense equivalence

CONV_CASES = [
    # (lattice, B, m, n, f, s, Cin, Cout)
    (SQ, 2, 9, 40, 2, 1, 3, 4),
    (SQ, 1, 10, 50, 3, 1, 2, 3),
    (SQ, 2, 11, 60, 2, 2, 3, 2),
    (SQ, 1, 12, 144, 3, 2, 2, 2),    # every site active
    (TRI, 2, 10, 30, 2, 1, 3, 4),
    (TRI, 1, 12, 40, 3, 1, 2, 3),
    (TRI, 2, 13, 50, 2, 2, 3, 2),
    (TRI, 1, 9, 45, 3, 2, 2, 2),     # every site active
    (TRI, 1, 2, 3, 3, 1, 2, 2),      # grid smaller than the filter
]


@pytest.mark.parametrize("case", CONV_CASES)
@pytest.mark.parametrize("relu", [False, True])
def test_conv_fwd_dense_equivalence(case, relu):
    lattice, B, m, n, f, s, Cin, Cout = case
    rng = np.random.default_rng(hash(("2d", case, relu)) % 2**32)
    coords = sites(lattice, rng, B, m, n)
    x = rng.standard_normal((len(coords), Cin))
    K = len(offsets(f, lattice))
    W = rng.standard_normal((K, Cin, Cout)) * 0.5
    bias = rng.standard_normal(Cout) * 0.3
    g_in = rng.standard_normal(Cin)
    rb = oracle.Rulebook(coords, (B, m, m, 1), f, s, lattice=lattice)
    assert rb.K == K
    y, g_out = oracle.conv_fwd(rb, x, g_in, W, bias, relu=relu)
    if out_size(m, f, s) == 0:
        assert rb.a_out == 0
        return
    X = field2d(coords, torch.tensor(x), torch.tensor(g_in), B, m, m)
    Y = F.conv2d(X, weight2d(torch.tensor(W), f, lattice), torch.tensor(bias), stride=s)
    if relu:
        Y = torch.relu(Y)
    Y = Y.permute(0, 2, 3, 1).numpy()
    oc = rb.arrays().out_coords
    assert (oc[:, 3] == 0).all()
    v = valid_mask(B, m, m, f, s, lattice)
    assert v[oc[:, 0], oc[:, 2], oc[:, 1]].all()
    np.testing.assert_allclose(y, Y[oc[:, 0], oc[:, 2], oc[:, 1]], rtol=1e-12, atol=1e-12)
    inactive = v.copy()
    inactive[oc[:, 0], oc[:, 2], oc[:, 1]] = False
    if inactive.any():
        np.testing.assert_allclose(Y[inactive], np.broadcast_to(g_out, Y[inactive].shape),
                                   rtol=1e-12, atol=1e-12)


def window_max(X, f, s, lattice, q):
    views = [X[:, :, ky:ky + s * (q - 1) + 1:s, kx:kx + s * (q - 1) + 1:s]
             for (kx, ky) in offsets(f, lattice)]
    V = torch.stack(views, 0)
    best, arg = V[0], torch.zeros_like(V[0], dtype=torch.long)
    for k in range(1, len(views)):
        up = V[k] > best
        best = torch.where(up, V[k], best)
        arg = torch.where(up, torch.full_like(arg, k), arg)
    return best, arg


POOL_CASES = [
    # (lattice, B, m, n, f, s, C)
    (SQ, 2, 12, 60, 2, 2, 3),
    (SQ, 1, 13, 70, 3, 2, 2),
    (TRI, 1, 15, 60, 3, 2, 3),
    (TRI, 2, 11, 66, 3, 2, 2),      # every site active
    (TRI, 1, 14, 50, 2, 2, 2),
]


@pytest.mark.parametrize("case", POOL_CASES)
def test_maxpool_dense_equivalence_and_gradients(case):
    lattice, B, m, n, f, s, C = case
    rng = np.random.default_rng(hash(("2dp", case)) % 2**32)
    coords = sites(lattice, rng, B, m, n)
    x = rng.standard_normal((len(coords), C))
    g_in = rng.standard_normal(C)
    rb = oracle.Rulebook(coords, (B, m, m, 1), f, s, lattice=lattice)
    y, g_out, ak, ai = oracle.maxpool_fwd(rb, x, g_in)
    q = out_size(m, f, s)
    tx, tg = torch.tensor(x, requires_grad=True), torch.tensor(g_in, requires_grad=True)
    Y, arg = window_max(field2d(coords, tx, tg, B, m, m), f, s, lattice, q)
    if lattice == SQ:  # the library routine agrees with the window maximum
        np.testing.assert_array_equal(
            Y.detach().numpy(),
            F.max_pool2d(field2d(coords, torch.tensor(x), torch.tensor(g_in), B, m, m), f, s).numpy())
    oc = rb.arrays().out_coords
    Yn = Y.detach().permute(0, 2, 3, 1).numpy()
    argn = arg.permute(0, 2, 3, 1).numpy()
    v = valid_mask(B, m, m, f, s, lattice)
    assert v[oc[:, 0], oc[:, 2], oc[:, 1]].all()
    np.testing.assert_array_equal(y, Yn[oc[:, 0], oc[:, 2], oc[:, 1]])
    won = ai == 0
    np.testing.assert_array_equal(ak[won], argn[oc[:, 0], oc[:, 2], oc[:, 1]][won])
    inactive = v.copy()
    inactive[oc[:, 0], oc[:, 2], oc[:, 1]] = False
    np.testing.assert_array_equal(Yn[inactive], np.broadcast_to(g_out, Yn[inactive].shape))
    # gradients through the same dense function
    dy = rng.uniform(-1, 1, (rb.a_out, C))
    dg = rng.uniform(-1, 1, C)
    dx, dgi = oracle.maxpool_bwd(rb, x, g_in, dy, dg)
    ot = torch.as_tensor(oc.astype(np.int64))
    L = (Y[ot[:, 0], :, ot[:, 2], ot[:, 1]] * torch.tensor(dy)).sum() + (tg * torch.tensor(dg)).sum()
    L.backward()
    np.testing.assert_allclose(dx, tx.grad.numpy(), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(dgi, tg.grad.numpy(), rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("case", CONV_CASES[:8:2] + CONV_CASES[1:8:2])
def test_conv_bwd_matches_dense_autograd(case):
    lattice, B, m, n, f, s, Cin, Cout = case
    rng = np.random.default_rng(hash(("2db", case)) % 2**32)
    coords = sites(lattice, rng, B, m, n)
    x = rng.standard_normal((len(coords), Cin))
    K = len(offsets(f, lattice))
    W = rng.standard_normal((K, Cin, Cout)) * 0.5
    bias = rng.standard_normal(Cout) * 0.3
    g_in = rng.standard_normal(Cin)
    rb = oracle.Rulebook(coords, (B, m, m, 1), f, s, lattice=lattice)
    dy = rng.uniform(-1, 1, (rb.a_out, Cout))
    dg = rng.uniform(-1, 1, Cout)
    got = oracle.conv_bwd(rb, x, g_in, W, bias, dy, dg, relu=True)
    tx, tg, tW, tb = (torch.tensor(v, requires_grad=True) for v in (x, g_in, W, bias))
    oc = torch.as_tensor(rb.arrays().out_coords.astype(np.int64))
    Y = torch.relu(F.conv2d(field2d(coords, tx, tg, B, m, m), weight2d(tW, f, lattice), tb,
                            stride=s))
    gpre = torch.relu(tb + (tW * tg.view(1, -1, 1)).sum((0, 1)))
    L = (Y[oc[:, 0], :, oc[:, 2], oc[:, 1]] * torch.tensor(dy)).sum() + \
        (gpre * torch.tensor(dg)).sum()
    L.backward()
    for name, t in (("dx", tx), ("dg_in", tg), ("dW", tW), ("dbias", tb)):
        np.testing.assert_allclose(got[name], t.grad.numpy(), rtol=1e-10, atol=1e-10,
                                   err_msg=name)


@pytest.mark.parametrize("lattice", [SQ, TRI])
@pytest.mark.parametrize("f,s", [(2, 1), (3, 1), (3, 2), (2, 3)])
def test_active_set_and_rules_brute_force(lattice, f, s):
    rng = np.random.default_rng(900 + 10 * f + s)
    B, m = 2, 11
    coords = sites(lattice, rng, B, m, 30)
    rb = oracle.Rulebook(coords, (B, m, m, 1), f, s, lattice=lattice)
    a = rb.arrays()
    row = {tuple(c): i for i, c in enumerate(coords.tolist())}
    offs = offsets(f, lattice)
    q = out_size(m, f, s)
    want_out, want_rules = [], [set() for _ in offs]
    for b in range(B):
        for oy in range(q):
            for ox in range(q):
                if lattice == TRI and s * (ox + oy) + f - 1 >= m:
                    continue
                hits = [(k, row.get((b, s * ox + kx, s * oy + ky, 0))) for k, (kx, ky) in
                        enumerate(offs)]
                hits = [(k, r) for k, r in hits if r is not None]
                if hits:
                    want_out.append((b, ox, oy, 0))
                    for k, r in hits:
                        want_rules[k].add((r, len(want_out) - 1))
    assert [tuple(c) for c in a.out_coords.tolist()] == want_out
    for k in range(rb.K):
        got = set(zip(a.in_rows[a.offsets[k]:a.offsets[k + 1]].tolist(),
                      a.out_rows[a.offsets[k]:a.offsets[k + 1]].tolist()))
        assert got == want_rules[k]
