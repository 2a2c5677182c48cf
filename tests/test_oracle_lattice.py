"""Pins of the oracle's tetrahedral lattice (section 1.2) against things other
than itself (CPU only).

Reading of section 1.2 in skewed integer coordinates: the grid of size m is
the sites x + y + z < m, a filter of size f covers the C(f+2, 3) offsets
kx + ky + kz < f (numbered in the cubic scan order restricted to them), and an
output exists where its whole window lies in the grid.

* counts the paper states: C(f+2, 3) sites per filter, 4 for size 2, 10 for
  size 3; Figure 2 (iv), a grid of size 3 under a filter of size 2; MP3/2
  regions of 10 sites, adjacent regions sharing exactly one site;
* dense equivalence: on the cube that holds the tetrahedral grid, a dense
  cross-correlation (torch conv3d, float64) whose weights are zero outside the
  tetrahedral offsets equals the sparse result at active outputs and g_out at
  inactive valid outputs; max-pooling likewise against a dense max over the
  window offsets;
* brute-force active sets over the valid output sites;
* gradients: dense autograd of the same dense functions, and central finite
  differences of the oracle's own forward.
"""
import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import gen
import oracle

T = "tetrahedral"


def tetra_offsets(f):
    """Offsets kx + ky + kz < f in the cube scan order (x fastest)."""
    return [(kx, ky, kz) for kz in range(f) for ky in range(f) for kx in range(f)
            if kx + ky + kz < f]


def out_size(m, f, s):
    return (m - f) // s + 1 if m >= f else 0


def valid_outputs(m, f, s):
    """Output sites whose whole window lies in the grid of size m."""
    q = out_size(m, f, s)
    return [(x, y, z) for z in range(q) for y in range(q) for x in range(q)
            if s * (x + y + z) + f - 1 < m]


def dense_field(coords, feats, g, B, m):
    """[B, C, Z, Y, X] over the cube [0, m)^3: feats at active sites, g
    elsewhere (keeps the autograd graph to feats and g)."""
    C = feats.shape[1]
    c = torch.as_tensor(np.asarray(coords, np.int64))
    vals = torch.zeros(B, m, m, m, C, dtype=torch.float64)
    vals = vals.index_put((c[:, 0], c[:, 3], c[:, 2], c[:, 1]), feats)
    mask = torch.zeros(B, m, m, m, 1, dtype=torch.float64)
    mask[c[:, 0], c[:, 3], c[:, 2], c[:, 1]] = 1.0
    return (mask * vals + (1.0 - mask) * g.view(1, 1, 1, 1, C)).permute(0, 4, 1, 2, 3)


def cube_weight(W, f):
    """Tetrahedral W[K][Cin][Cout] placed into a cube filter, zero elsewhere,
    in torch's [Cout][Cin][kz][ky][kx] layout."""
    K, Cin, Cout = W.shape
    Wc = torch.zeros(f, f, f, Cin, Cout, dtype=torch.float64)
    for k, (kx, ky, kz) in enumerate(tetra_offsets(f)):
        Wc[kz, ky, kx] = W[k]
    return Wc.permute(4, 3, 0, 1, 2)


def valid_mask(B, m, f, s):
    q = out_size(m, f, s)
    v = np.zeros((B, q, q, q), bool)
    for (x, y, z) in valid_outputs(m, f, s):
        v[:, z, y, x] = True
    return v


# ---------------------------------------------------------------- counts

@pytest.mark.parametrize("f", [1, 2, 3, 4, 5])
def test_filter_covers_binomial_sites(f):
    """C(f+2, 3) sites per filter: 4 for the smallest filter, 10 for MP3."""
    coords = np.array([[0, f - 1, f - 1, f - 1]], np.int32)   # one site, interior
    m = 4 * f
    rb = oracle.Rulebook(coords, (1, m, m, m), f, 1, lattice=T)
    assert rb.K == math.comb(f + 2, 3)
    # s = 1: the site is seen by one output per filter offset
    assert rb.a_out == rb.K == rb.n_pairs
    assert {2: 4, 3: 10}.get(f, rb.K) == rb.K


def test_figure2_iv_grid3_filter2():
    """Figure 2 (iv): a tetrahedral grid of size 3 under a filter of size 2
    gives a grid of size 2 (4 outputs), each seeing 4 input sites."""
    cell = gen.tetra_sites(3)
    assert len(cell) == 10
    coords = np.concatenate([np.zeros((10, 1), np.int64), cell], axis=1).astype(np.int32)
    rb = oracle.Rulebook(coords, (1, 3, 3, 3), 2, 1, lattice=T)
    a = rb.arrays()
    assert rb.a_out == 4 and rb.n_pairs == 16
    assert sorted(map(tuple, a.out_coords[:, 1:].tolist())) == sorted(
        [(0, 0, 0), (1, 0, 0), (0, 1, 0), (0, 0, 1)])


@pytest.mark.parametrize("m,f,s", [(5, 2, 1), (7, 3, 1), (7, 3, 2), (9, 2, 2), (11, 3, 3), (8, 1, 1)])
def test_full_grid_counts(m, f, s):
    cell = gen.tetra_sites(m)
    coords = np.concatenate([np.zeros((len(cell), 1), np.int64), cell], axis=1).astype(np.int32)
    rb = oracle.Rulebook(coords, (1, m, m, m), f, s, lattice=T)
    q = out_size(m, f, s)
    # the outputs form a tetrahedral grid of size q, all windows full
    assert rb.a_out == math.comb(q + 2, 3) == len(valid_outputs(m, f, s))
    assert rb.n_pairs == rb.a_out * math.comb(f + 2, 3)


def test_mp32_regions_have_ten_sites_and_neighbours_share_one():
    """MP3/2 on a full tetrahedral grid: every region holds 10 sites and two
    regions at adjacent output sites share exactly one site."""
    m = 11
    cell = gen.tetra_sites(m)
    coords = np.concatenate([np.zeros((len(cell), 1), np.int64), cell], axis=1).astype(np.int32)
    rb = oracle.Rulebook(coords, (1, m, m, m), 3, 2, lattice=T)
    a = rb.arrays()
    members = [set() for _ in range(rb.a_out)]
    for i, o in zip(a.in_rows, a.out_rows):
        members[o].add(int(i))
    assert all(len(s) == 10 for s in members)
    pos = {tuple(c[1:]): o for o, c in enumerate(a.out_coords.tolist())}
    steps = [(1, 0, 0), (0, 1, 0), (0, 0, 1), (1, -1, 0), (1, 0, -1), (0, 1, -1)]
    n_adj = 0
    for p, o in pos.items():
        for d in steps:
            q = tuple(p[i] + d[i] for i in range(3))
            if q in pos:
                assert len(members[o] & members[pos[q]]) == 1
                n_adj += 1
    assert n_adj > 0


def test_offset_order_is_restricted_cube_scan():
    """A single interior input p: output o = p - k sees it through offset k,
    so the list holding each pair names its offset."""
    f, m = 3, 9
    p = (2, 2, 2)
    coords = np.array([[0, *p]], np.int32)
    rb = oracle.Rulebook(coords, (1, m, m, m), f, 1, lattice=T)
    a = rb.arrays()
    offs = tetra_offsets(f)
    for k in range(rb.K):
        lo, hi = a.offsets[k], a.offsets[k + 1]
        assert hi - lo == 1
        o = a.out_coords[a.out_rows[lo]][1:]
        assert tuple(int(p[i] - o[i]) for i in range(3)) == offs[k]


def test_range_and_invalid_statuses():
    with pytest.raises(oracle.OracleError) as e:
        oracle.Rulebook(np.array([[0, 2, 2, 1]], np.int32), (1, 5, 5, 5), 2, 1, lattice=T)
    assert e.value.status == "range"                    # 2 + 2 + 1 >= 5
    with pytest.raises(oracle.OracleError) as e:
        oracle.Rulebook(np.array([[0, 0, 0, 0]], np.int32), (1, 5, 6, 5), 2, 1, lattice=T)
    assert e.value.status == "invalid"                  # unequal extents
    # the same site is fine on the cube
    oracle.Rulebook(np.array([[0, 2, 2, 1]], np.int32), (1, 5, 5, 5), 2, 1)


# ---------------------------------------------------------------- dense equivalence

CONV_CASES = [
    # (B, m, n, f, s, Cin, Cout)
    (1, 6, 25, 2, 1, 3, 4),
    (2, 7, 40, 3, 1, 2, 3),
    (2, 9, 50, 2, 2, 3, 2),
    (1, 9, 30, 3, 2, 2, 3),
    (1, 6, 56, 2, 1, 2, 2),     # every site active
    (1, 5, 12, 1, 1, 3, 3),
    (1, 4, 8, 4, 1, 2, 2),      # one output only
    (1, 2, 3, 3, 1, 2, 2),      # m < f: no outputs
]


def tetra_case(rng, B, m, n, C):
    coords = gen.tetra_random_sites(rng, B, m, n)
    return coords, rng.standard_normal((len(coords), C))


@pytest.mark.parametrize("case", CONV_CASES)
@pytest.mark.parametrize("relu", [False, True])
def test_conv_fwd_dense_equivalence(case, relu):
    B, m, n, f, s, Cin, Cout = case
    rng = np.random.default_rng(hash(("tetra", case, relu)) % 2**32)
    coords, x = tetra_case(rng, B, m, n, Cin)
    K = math.comb(f + 2, 3)
    W = rng.standard_normal((K, Cin, Cout)) * 0.5
    bias = rng.standard_normal(Cout) * 0.3
    g_in = rng.standard_normal(Cin)
    rb = oracle.Rulebook(coords, (B, m, m, m), f, s, lattice=T)
    assert rb.K == K
    y, g_out = oracle.conv_fwd(rb, x, g_in, W, bias, relu=relu)
    a = rb.arrays()
    if out_size(m, f, s) == 0:
        assert rb.a_out == 0 and y.shape == (0, Cout)
        return
    X = dense_field(coords, torch.tensor(x), torch.tensor(g_in), B, m)
    Y = F.conv3d(X, cube_weight(torch.tensor(W), f), torch.tensor(bias), stride=s)
    if relu:
        Y = torch.relu(Y)
    Y = Y.permute(0, 2, 3, 4, 1).numpy()
    oc = a.out_coords
    v = valid_mask(B, m, f, s)
    assert v[oc[:, 0], oc[:, 3], oc[:, 2], oc[:, 1]].all()
    np.testing.assert_allclose(y, Y[oc[:, 0], oc[:, 3], oc[:, 2], oc[:, 1]], rtol=1e-12, atol=1e-12)
    inactive = v.copy()
    inactive[oc[:, 0], oc[:, 3], oc[:, 2], oc[:, 1]] = False
    if inactive.any():
        np.testing.assert_allclose(Y[inactive], np.broadcast_to(g_out, Y[inactive].shape),
                                   rtol=1e-12, atol=1e-12)


def dense_window_max(X, f, s, m):
    """Max over the tetrahedral window offsets of a dense field [B, C, Z, Y, X]
    at every cube output site; returns (values, first arg offset)."""
    q = out_size(m, f, s)
    views = [X[:, :, kz:kz + s * (q - 1) + 1:s, ky:ky + s * (q - 1) + 1:s,
               kx:kx + s * (q - 1) + 1:s] for (kx, ky, kz) in tetra_offsets(f)]
    V = torch.stack(views, 0)                           # [K, B, C, q, q, q]
    best, arg = V[0], torch.zeros_like(V[0], dtype=torch.long)
    for k in range(1, len(views)):                      # first strict maximum wins
        up = V[k] > best
        best = torch.where(up, V[k], best)
        arg = torch.where(up, torch.full_like(arg, k), arg)
    return best, arg


POOL_CASES = [
    # (B, m, n, f, s, C)
    (1, 9, 40, 3, 2, 3),        # MP3/2
    (2, 11, 80, 3, 2, 2),
    (2, 8, 30, 2, 2, 2),        # MP2/2: disjoint regions with gaps
    (1, 10, 30, 3, 3, 2),
    (1, 7, 84, 3, 2, 2),        # every site active
]


@pytest.mark.parametrize("case", POOL_CASES)
def test_maxpool_fwd_dense_equivalence(case):
    B, m, n, f, s, C = case
    rng = np.random.default_rng(hash(("tetra", case)) % 2**32)
    coords, x = tetra_case(rng, B, m, n, C)
    g_in = rng.standard_normal(C)
    rb = oracle.Rulebook(coords, (B, m, m, m), f, s, lattice=T)
    y, g_out, ak, ai = oracle.maxpool_fwd(rb, x, g_in)
    np.testing.assert_array_equal(g_out, g_in)
    a = rb.arrays()
    Y, arg = dense_window_max(dense_field(coords, torch.tensor(x), torch.tensor(g_in), B, m), f, s, m)
    Y = Y.permute(0, 2, 3, 4, 1).numpy()
    arg = arg.permute(0, 2, 3, 4, 1).numpy()
    oc = a.out_coords
    v = valid_mask(B, m, f, s)
    assert v[oc[:, 0], oc[:, 3], oc[:, 2], oc[:, 1]].all()
    np.testing.assert_array_equal(y, Y[oc[:, 0], oc[:, 3], oc[:, 2], oc[:, 1]])
    inactive = v.copy()
    inactive[oc[:, 0], oc[:, 3], oc[:, 2], oc[:, 1]] = False
    np.testing.assert_array_equal(Y[inactive], np.broadcast_to(g_out, Y[inactive].shape))
    # the winner's offset agrees where the winner is an active site (ground
    # state ties between inactive positions carry no position)
    won = ai == 0
    np.testing.assert_array_equal(ak[won], arg[oc[:, 0], oc[:, 3], oc[:, 2], oc[:, 1]][won])


@pytest.mark.parametrize("f,s", [(2, 1), (3, 1), (2, 2), (3, 2), (4, 1)])
def test_active_set_and_rules_brute_force(f, s):
    rng = np.random.default_rng(700 + 10 * f + s)
    B, m = 2, 9
    coords = gen.tetra_random_sites(rng, B, m, 30)
    rb = oracle.Rulebook(coords, (B, m, m, m), f, s, lattice=T)
    a = rb.arrays()
    row = {tuple(c): i for i, c in enumerate(coords.tolist())}
    offs = tetra_offsets(f)
    want_out, want_rules = [], [set() for _ in offs]
    for b in range(B):
        for (ox, oy, oz) in sorted(valid_outputs(m, f, s), key=lambda p: (p[2], p[1], p[0])):
            hits = [(k, row.get((b, s * ox + kx, s * oy + ky, s * oz + kz)))
                    for k, (kx, ky, kz) in enumerate(offs)]
            hits = [(k, r) for k, r in hits if r is not None]
            if hits:
                want_out.append((b, ox, oy, oz))
                for k, r in hits:
                    want_rules[k].add((r, len(want_out) - 1))
    assert [tuple(c) for c in a.out_coords.tolist()] == want_out
    for k in range(rb.K):
        got = set(zip(a.in_rows[a.offsets[k]:a.offsets[k + 1]].tolist(),
                      a.out_rows[a.offsets[k]:a.offsets[k + 1]].tolist()))
        assert got == want_rules[k]


# ---------------------------------------------------------------- gradients

@pytest.mark.parametrize("case", CONV_CASES[:5])
@pytest.mark.parametrize("relu", [False, True])
def test_conv_bwd_matches_dense_autograd(case, relu):
    B, m, n, f, s, Cin, Cout = case
    rng = np.random.default_rng(3000 + hash(("tetra", case, relu)) % 2**32)
    coords, x = tetra_case(rng, B, m, n, Cin)
    K = math.comb(f + 2, 3)
    W = rng.standard_normal((K, Cin, Cout)) * 0.5
    bias = rng.standard_normal(Cout) * 0.3
    g_in = rng.standard_normal(Cin)
    rb = oracle.Rulebook(coords, (B, m, m, m), f, s, lattice=T)
    dy = rng.uniform(-1, 1, (rb.a_out, Cout))
    dg = rng.uniform(-1, 1, Cout)
    got = oracle.conv_bwd(rb, x, g_in, W, bias, dy, dg, relu=relu)
    tx, tg, tW, tb = (torch.tensor(v, requires_grad=True) for v in (x, g_in, W, bias))
    oc = torch.as_tensor(rb.arrays().out_coords.astype(np.int64))
    Y = F.conv3d(dense_field(coords, tx, tg, B, m), cube_weight(tW, f), tb, stride=s)
    gpre = tb + (tW * tg.view(1, -1, 1)).sum((0, 1))
    if relu:
        Y, gpre = torch.relu(Y), torch.relu(gpre)
    L = (Y[oc[:, 0], :, oc[:, 3], oc[:, 2], oc[:, 1]] * torch.tensor(dy)).sum() + \
        (gpre * torch.tensor(dg)).sum()
    L.backward()
    for name, t in (("dx", tx), ("dg_in", tg), ("dW", tW), ("dbias", tb)):
        np.testing.assert_allclose(got[name], t.grad.numpy(), rtol=1e-10, atol=1e-10,
                                   err_msg=name)


@pytest.mark.parametrize("case", POOL_CASES)
def test_maxpool_bwd_matches_dense_autograd(case):
    B, m, n, f, s, C = case
    rng = np.random.default_rng(4000 + hash(("tetra", case)) % 2**32)
    coords, x = tetra_case(rng, B, m, n, C)
    g_in = rng.standard_normal(C)
    rb = oracle.Rulebook(coords, (B, m, m, m), f, s, lattice=T)
    dy = rng.uniform(-1, 1, (rb.a_out, C))
    dg = rng.uniform(-1, 1, C)
    dx, dgi = oracle.maxpool_bwd(rb, x, g_in, dy, dg)
    tx, tg = torch.tensor(x, requires_grad=True), torch.tensor(g_in, requires_grad=True)
    oc = torch.as_tensor(rb.arrays().out_coords.astype(np.int64))
    Y, _ = dense_window_max(dense_field(coords, tx, tg, B, m), f, s, m)
    L = (Y[oc[:, 0], :, oc[:, 3], oc[:, 2], oc[:, 1]] * torch.tensor(dy)).sum() + \
        (tg * torch.tensor(dg)).sum()
    L.backward()
    np.testing.assert_allclose(dx, tx.grad.numpy(), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(dgi, tg.grad.numpy(), rtol=1e-12, atol=1e-12)


def test_conv_bwd_finite_differences():
    """Central differences of the oracle's own forward on the tetrahedral
    lattice (no torch involved)."""
    rng = np.random.default_rng(77)
    B, m, f, s, Cin, Cout = 1, 6, 2, 1, 2, 2
    coords, x = tetra_case(rng, B, m, 14, Cin)
    W = rng.standard_normal((4, Cin, Cout)) * 0.5
    bias = rng.standard_normal(Cout) * 0.3 + 0.2
    g_in = rng.standard_normal(Cin)
    rb = oracle.Rulebook(coords, (B, m, m, m), f, s, lattice=T)
    dy = rng.uniform(-1, 1, (rb.a_out, Cout))
    dg = rng.uniform(-1, 1, Cout)
    got = oracle.conv_bwd(rb, x, g_in, W, bias, dy, dg, relu=True)

    def loss(x_, g_, W_, b_):
        y, go = oracle.conv_fwd(rb, x_, g_, W_, b_, relu=True)
        return float((y * dy).sum() + (go * dg).sum())

    h = 1e-6
    params = dict(dx=x, dg_in=g_in, dW=W, dbias=bias)
    for name, arr in params.items():
        num = np.zeros_like(arr)
        for i in np.ndindex(arr.shape):
            p, q = arr.copy(), arr.copy()
            p[i] += h
            q[i] -= h
            num[i] = (loss(*[p if k == name else params[k] for k in params]) -
                      loss(*[q if k == name else params[k] for k in params])) / (2 * h)
        np.testing.assert_allclose(got[name], num, rtol=1e-6, atol=1e-7, err_msg=name)


def test_shell_generator_stays_in_grid():
    """The tetrahedral shell generator draws only grid sites, no duplicates."""
    rng = gen.stream_rng(5, 0)
    s = gen.tetra_shell_sites(rng, 30, [9.0, 7.0, 8.0], 2)
    assert len(s) > 0 and (s >= 0).all() and (s.sum(1) < 30).all()
    assert len(np.unique(s, axis=0)) == len(s)
