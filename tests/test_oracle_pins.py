"""Pins of the CPU oracle against things other than itself (CPU only).

* dense equivalence: the sparse result equals a dense 3D cross-correlation /
  max-pool (torch CPU, float64) of the field that holds M_in at active sites
  and g_in elsewhere, at active outputs; inactive dense outputs equal g_out
  (section 1.3: ground state, steps 2-3);
* brute-force active sets: an output is active iff any input in its window is
  (section 1.3, second active-site rule), enumerated over output sites;
* the worked example of Figure 3 and the trefoil behaviour of Figure 1;
* gradients: dense autograd through the same torch routines, and central
  finite differences of the oracle's own forward;
* counting invariants of the rule lists.
"""
import itertools
import os

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import gen
import oracle

HERE = os.path.dirname(os.path.abspath(__file__))


def keys_of(coords, grid):
    c = np.asarray(coords, np.int64)
    B, mx, my, mz = grid
    return ((c[:, 0] * mz + c[:, 3]) * my + c[:, 2]) * mx + c[:, 1]


def out_extent(m, f, s):
    return (m - f) // s + 1 if m >= f else 0


# ---------------------------------------------------------------- dense refs

def dense_input(coords, feats, g, grid):
    """Dense field [B, C, Z, Y, X]: feats at active sites, g elsewhere; keeps the
    autograd graph to feats and g."""
    B, mx, my, mz = grid
    C = feats.shape[1]
    c = torch.as_tensor(np.asarray(coords, np.int64))
    vals = torch.zeros(B, mz, my, mx, C, dtype=torch.float64)
    vals = vals.index_put((c[:, 0], c[:, 3], c[:, 2], c[:, 1]), feats)
    mask = torch.zeros(B, mz, my, mx, 1, dtype=torch.float64)
    mask[c[:, 0], c[:, 3], c[:, 2], c[:, 1]] = 1.0
    field = mask * vals + (1.0 - mask) * g.view(1, 1, 1, 1, C)
    return field.permute(0, 4, 1, 2, 3)


def torch_weight(W, f):
    K, Cin, Cout = W.shape
    return W.reshape(f, f, f, Cin, Cout).permute(4, 3, 0, 1, 2)


def random_case(rng, B, dims, n, Cin):
    coords = gen.random_sites(rng, B, dims, n)
    x = rng.standard_normal((len(coords), Cin))
    return coords, x


CONV_CASES = [
    # (B, dims, n, f, s, Cin, Cout)
    (1, (5, 4, 6), 20, 2, 1, 3, 4),
    (2, (6, 6, 5), 30, 3, 1, 2, 5),
    (2, (7, 5, 6), 40, 2, 2, 3, 2),
    (1, (7, 7, 7), 25, 3, 2, 1, 3),
    (2, (4, 5, 3), 60, 3, 1, 2, 2),   # dense-ish: most sites active
    (1, (5, 5, 5), 125, 2, 1, 2, 3),  # every site active
    (1, (6, 5, 4), 12, 1, 1, 3, 3),
    (1, (2, 6, 6), 10, 3, 1, 2, 2),   # mx < f: no outputs at all
]


@pytest.mark.parametrize("case", CONV_CASES)
@pytest.mark.parametrize("relu", [False, True])
def test_conv_fwd_dense_equivalence(case, relu):
    B, dims, n, f, s, Cin, Cout = case
    rng = np.random.default_rng(hash((case, relu)) % 2**32)
    coords, x = random_case(rng, B, dims, n, Cin)
    grid = (B,) + tuple(dims)
    K = f ** 3
    W = rng.standard_normal((K, Cin, Cout)) * 0.5
    bias = rng.standard_normal(Cout) * 0.3
    g_in = rng.standard_normal(Cin)
    rb = oracle.Rulebook(coords, grid, f, s)
    y, g_out = oracle.conv_fwd(rb, x, g_in, W, bias, relu=relu)
    a = rb.arrays()
    if min(out_extent(m, f, s) for m in dims) == 0:
        assert rb.a_out == 0 and rb.n_pairs == 0 and y.shape == (0, Cout)
        return
    X = dense_input(coords, torch.tensor(x), torch.tensor(g_in), grid)
    Y = F.conv3d(X, torch_weight(torch.tensor(W), f), torch.tensor(bias), stride=s)
    if relu:
        Y = torch.relu(Y)
    Y = Y.permute(0, 2, 3, 4, 1).numpy()          # [B, Z, Y, X, C]
    assert Y.shape[1:4] == tuple(out_extent(m, f, s) for m in (dims[2], dims[1], dims[0]))
    oc = a.out_coords
    np.testing.assert_allclose(y, Y[oc[:, 0], oc[:, 3], oc[:, 2], oc[:, 1]], rtol=1e-12, atol=1e-12)
    inactive = np.ones(Y.shape[:4], bool)
    inactive[oc[:, 0], oc[:, 3], oc[:, 2], oc[:, 1]] = False
    if inactive.any():
        np.testing.assert_allclose(Y[inactive], np.broadcast_to(g_out, Y[inactive].shape),
                                   rtol=1e-12, atol=1e-12)
    # rows restricted to a subset give the same values
    if rb.a_out:
        rows = rng.choice(rb.a_out, size=min(5, rb.a_out), replace=False)
        y2, _ = oracle.conv_fwd(rb, x, g_in, W, bias, relu=relu, rows=rows)
        np.testing.assert_array_equal(y2, y[rows])


POOL_CASES = [
    (1, (6, 6, 6), 40, 2, 2, 3),
    (2, (7, 5, 6), 50, 2, 2, 2),
    (2, (7, 7, 7), 60, 3, 2, 2),   # overlapping pooling MP3/2
    (1, (5, 6, 7), 30, 3, 3, 2),
    (1, (4, 4, 4), 64, 2, 2, 2),   # every site active
]


@pytest.mark.parametrize("case", POOL_CASES)
def test_maxpool_fwd_dense_equivalence(case):
    B, dims, n, f, s, C = case
    rng = np.random.default_rng(hash(case) % 2**32)
    coords, x = random_case(rng, B, dims, n, C)
    grid = (B,) + tuple(dims)
    g_in = rng.standard_normal(C)
    rb = oracle.Rulebook(coords, grid, f, s)
    y, g_out, ak, ai = oracle.maxpool_fwd(rb, x, g_in)
    np.testing.assert_array_equal(g_out, g_in)
    a = rb.arrays()
    X = dense_input(coords, torch.tensor(x), torch.tensor(g_in), grid)
    Y, idx = F.max_pool3d(X, f, s, return_indices=True)
    Y = Y.permute(0, 2, 3, 4, 1).numpy()
    idx = idx.permute(0, 2, 3, 4, 1).numpy()
    oc = a.out_coords
    np.testing.assert_array_equal(y, Y[oc[:, 0], oc[:, 3], oc[:, 2], oc[:, 1]])
    inactive = np.ones(Y.shape[:4], bool)
    inactive[oc[:, 0], oc[:, 3], oc[:, 2], oc[:, 1]] = False
    np.testing.assert_array_equal(Y[inactive], np.broadcast_to(g_out, Y[inactive].shape))
    # winning position: torch's flat index (z*H + y)*W + x -> window offset
    mx, my = dims[0], dims[1]
    fl = idx[oc[:, 0], oc[:, 3], oc[:, 2], oc[:, 1]]
    kx = fl % mx - s * oc[:, 1:2]
    ky = (fl // mx) % my - s * oc[:, 2:3]
    kz = fl // (mx * my) - s * oc[:, 3:4]
    np.testing.assert_array_equal(ak, (kz * f + ky) * f + kx)


def test_maxpool_tie_rule_matches_dense_scan_order():
    """Ties (exact zeros after ReLU, ground state 0) resolve to the first
    position in (z, y, x) scan order, as torch's CPU max_pool3d does."""
    rng = np.random.default_rng(7)
    B, dims, C = 1, (6, 6, 6), 4
    coords = gen.random_sites(rng, B, dims, 70)
    x = np.maximum(rng.standard_normal((len(coords), C)), 0.0)
    x[rng.random(x.shape) < 0.5] = 0.0
    g_in = np.zeros(C)
    rb = oracle.Rulebook(coords, (B,) + dims, 2, 2)
    y, _, ak, ai = oracle.maxpool_fwd(rb, x, g_in)
    a = rb.arrays()
    X = dense_input(coords, torch.tensor(x), torch.tensor(g_in), (B,) + dims)
    Y, idx = F.max_pool3d(X, 2, 2, return_indices=True)
    idx = idx.permute(0, 2, 3, 4, 1).numpy()
    oc = a.out_coords
    fl = idx[oc[:, 0], oc[:, 3], oc[:, 2], oc[:, 1]]
    s = 2
    kx = fl % 6 - s * oc[:, 1:2]
    ky = (fl // 6) % 6 - s * oc[:, 2:3]
    kz = fl // 36 - s * oc[:, 3:4]
    assert (y == 0).mean() > 0.2      # the case really has many ties
    np.testing.assert_array_equal(ak, (kz * 2 + ky) * 2 + kx)


# ---------------------------------------------------------------- gradients

def dense_conv_loss(coords, x, g_in, W, bias, dy, dg_out, grid, f, s, relu, oc):
    X = dense_input(coords, x, g_in, grid)
    Y = F.conv3d(X, torch_weight(W, f), bias, stride=s)
    gpre = bias + torch.einsum("kio,i->o", W, g_in)
    if relu:
        Y = torch.relu(Y)
        gpre = torch.relu(gpre)
    Yo = Y[oc[:, 0], :, oc[:, 3], oc[:, 2], oc[:, 1]]
    return (Yo * dy).sum() + (gpre * dg_out).sum()


@pytest.mark.parametrize("case", CONV_CASES[:6])
@pytest.mark.parametrize("relu", [False, True])
def test_conv_bwd_matches_dense_autograd(case, relu):
    B, dims, n, f, s, Cin, Cout = case
    rng = np.random.default_rng(1000 + hash((case, relu)) % 2**32)
    coords, x = random_case(rng, B, dims, n, Cin)
    grid = (B,) + tuple(dims)
    K = f ** 3
    W = rng.standard_normal((K, Cin, Cout)) * 0.5
    bias = rng.standard_normal(Cout) * 0.3
    g_in = rng.standard_normal(Cin)
    rb = oracle.Rulebook(coords, grid, f, s)
    dy = rng.uniform(-1, 1, (rb.a_out, Cout))
    dg = rng.uniform(-1, 1, Cout)
    got = oracle.conv_bwd(rb, x, g_in, W, bias, dy, dg, relu=relu)
    tx, tg, tW, tb = (torch.tensor(v, requires_grad=True) for v in (x, g_in, W, bias))
    oc = torch.as_tensor(rb.arrays().out_coords.astype(np.int64))
    L = dense_conv_loss(coords, tx, tg, tW, tb, torch.tensor(dy), torch.tensor(dg), grid, f, s,
                        relu, oc)
    L.backward()
    for name, t in (("dx", tx), ("dg_in", tg), ("dW", tW), ("dbias", tb)):
        np.testing.assert_allclose(got[name], t.grad.numpy(), rtol=1e-10, atol=1e-10,
                                   err_msg=name)


@pytest.mark.parametrize("case", POOL_CASES)
def test_maxpool_bwd_matches_dense_autograd(case):
    B, dims, n, f, s, C = case
    rng = np.random.default_rng(2000 + hash(case) % 2**32)
    coords, x = random_case(rng, B, dims, n, C)
    grid = (B,) + tuple(dims)
    g_in = rng.standard_normal(C)
    rb = oracle.Rulebook(coords, grid, f, s)
    dy = rng.uniform(-1, 1, (rb.a_out, C))
    dg = rng.uniform(-1, 1, C)
    dx, dgi = oracle.maxpool_bwd(rb, x, g_in, dy, dg)
    tx, tg = torch.tensor(x, requires_grad=True), torch.tensor(g_in, requires_grad=True)
    oc = torch.as_tensor(rb.arrays().out_coords.astype(np.int64))
    Y = F.max_pool3d(dense_input(coords, tx, tg, grid), f, s)
    L = (Y[oc[:, 0], :, oc[:, 3], oc[:, 2], oc[:, 1]] * torch.tensor(dy)).sum() + (tg * torch.tensor(dg)).sum()
    L.backward()
    np.testing.assert_allclose(dx, tx.grad.numpy(), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(dgi, tg.grad.numpy(), rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("relu", [False, True])
def test_conv_bwd_finite_differences(relu):
    """Central differences of the oracle's own forward (no torch involved)."""
    rng = np.random.default_rng(31 + relu)
    B, dims, f, s, Cin, Cout = 1, (4, 5, 4), 2, 1, 2, 3
    coords, x = random_case(rng, B, dims, 14, Cin)
    grid = (B,) + dims
    W = rng.standard_normal((8, Cin, Cout)) * 0.5
    bias = rng.standard_normal(Cout) * 0.3 + 0.2
    g_in = rng.standard_normal(Cin)
    rb = oracle.Rulebook(coords, grid, f, s)
    dy = rng.uniform(-1, 1, (rb.a_out, Cout))
    dg = rng.uniform(-1, 1, Cout)
    got = oracle.conv_bwd(rb, x, g_in, W, bias, dy, dg, relu=relu)

    def loss(x_, g_, W_, b_):
        y, go = oracle.conv_fwd(rb, x_, g_, W_, b_, relu=relu)
        return float((y * dy).sum() + (go * dg).sum())

    h = 1e-6
    params = dict(dx=x, dg_in=g_in, dW=W, dbias=bias)
    for name, arr in params.items():
        num = np.zeros_like(arr)
        for i in np.ndindex(arr.shape):
            p, m = arr.copy(), arr.copy()
            p[i] += h
            m[i] -= h
            args = [params[k] if k != name else p for k in params]
            argm = [params[k] if k != name else m for k in params]
            num[i] = (loss(*args) - loss(*argm)) / (2 * h)
        np.testing.assert_allclose(got[name], num, rtol=1e-6, atol=1e-7, err_msg=name)


def test_maxpool_bwd_finite_differences():
    rng = np.random.default_rng(44)
    B, dims, C = 1, (5, 6, 5), 2
    coords, x = random_case(rng, B, dims, 30, C)
    g_in = rng.standard_normal(C)
    rb = oracle.Rulebook(coords, (B,) + dims, 3, 2)
    dy = rng.uniform(-1, 1, (rb.a_out, C))
    dg = rng.uniform(-1, 1, C)
    dx, dgi = oracle.maxpool_bwd(rb, x, g_in, dy, dg)

    def loss(x_, g_):
        y, go, _, _ = oracle.maxpool_fwd(rb, x_, g_)
        return float((y * dy).sum() + (go * dg).sum())

    h = 1e-7
    for arr, got, is_x in ((x, dx, True), (g_in, dgi, False)):
        num = np.zeros_like(arr)
        for i in np.ndindex(arr.shape):
            p, m = arr.copy(), arr.copy()
            p[i] += h
            m[i] -= h
            num[i] = ((loss(p, g_in) - loss(m, g_in)) if is_x else (loss(x, p) - loss(x, m))) / (2 * h)
        np.testing.assert_allclose(got, num, rtol=1e-6, atol=1e-7)


# ---------------------------------------------------------------- active sets

@pytest.mark.parametrize("f,s", [(2, 1), (3, 1), (2, 2), (3, 2), (1, 1), (3, 3)])
def test_active_set_and_rules_brute_force(f, s):
    rng = np.random.default_rng(f * 10 + s)
    B, dims = 2, (6, 5, 7)
    coords = gen.random_sites(rng, B, dims, 25)
    grid = (B,) + dims
    rb = oracle.Rulebook(coords, grid, f, s)
    a = rb.arrays()
    row_of = {tuple(c): r for r, c in enumerate(coords.tolist())}
    mo = [out_extent(m, f, s) for m in dims]
    expect_out = []
    expect_pairs = {k: [] for k in range(f ** 3)}
    for b in range(B):
        for z in range(mo[2]):
            for y in range(mo[1]):
                for x in range(mo[0]):
                    hits = []
                    for kz, ky, kx in itertools.product(range(f), repeat=3):
                        r = row_of.get((b, s * x + kx, s * y + ky, s * z + kz))
                        if r is not None:
                            hits.append(((kz * f + ky) * f + kx, r))
                    if hits:
                        o = len(expect_out)
                        expect_out.append((b, x, y, z))
                        for k, r in hits:
                            expect_pairs[k].append((r, o))
    assert rb.out_grid == (B, *mo)
    np.testing.assert_array_equal(a.out_coords, np.array(expect_out, np.int32).reshape(-1, 4))
    for k in range(f ** 3):
        seg = slice(a.offsets[k], a.offsets[k + 1])
        got = list(zip(a.in_rows[seg].tolist(), a.out_rows[seg].tolist()))
        assert got == expect_pairs[k]


def test_figure3_worked_example():
    spec = {}
    sites = []
    for line in open(os.path.join(HERE, "golden", "fig3_example.txt")):
        line = line.split("#")[0].split()
        if not line:
            continue
        if line[0] == "site":
            sites.append([int(v) for v in line[1:]])
        else:
            spec[line[0]] = [int(v) for v in line[1:]]
    rb = oracle.Rulebook(np.array(sites, np.int32), spec["grid"], spec["filter"][0],
                         spec["stride"][0])
    assert rb.a_in == 3
    assert list(rb.out_grid[1:]) == spec["out_extent"]
    assert rb.a_out == spec["active_out"][0]


def test_trefoil_grows_under_conv_and_shrinks_under_pool():
    """Figure 1: a 2x2x2 convolution increases the number of active sites of the
    trefoil; a 2x2x2 pooling decreases it."""
    c = gen.make_config(0)
    conv = oracle.Rulebook(c.coords, c.grid, 2, 1)
    assert conv.a_out > conv.a_in
    pool = oracle.Rulebook(conv.arrays().out_coords, conv.out_grid, 2, 2)
    assert pool.a_out < pool.a_in


# ---------------------------------------------------------------- invariants

def _per_input_pair_count(coords, dims, f, s):
    """I1: the number of rules an input takes part in is the product over axes
    of #{k in [0,f): (c-k) divisible by s and 0 <= (c-k)/s < m_out}."""
    tot = np.ones(len(coords), np.int64)
    for ax, m in zip((1, 2, 3), dims):
        mo = out_extent(m, f, s)
        c = coords[:, ax].astype(np.int64)
        cnt = np.zeros(len(coords), np.int64)
        for k in range(f):
            d = c - k
            cnt += (d >= 0) & (d % s == 0) & (d // s < mo)
        tot *= cnt
    return tot


@pytest.mark.parametrize("f,s", [(2, 1), (3, 1), (2, 2), (3, 2)])
def test_rule_invariants(f, s):
    rng = np.random.default_rng(99 + f + 7 * s)
    B, dims = 2, (9, 8, 10)
    coords = gen.random_sites(rng, B, dims, 120)
    rb = oracle.Rulebook(coords, (B,) + dims, f, s)
    a = rb.arrays()
    # I1: per-input incidence counts
    cnt = np.bincount(a.in_rows, minlength=len(coords))
    np.testing.assert_array_equal(cnt, _per_input_pair_count(coords, dims, f, s))
    for k in range(rb.K):
        seg = slice(a.offsets[k], a.offsets[k + 1])
        ir, orr = a.in_rows[seg], a.out_rows[seg]
        # I5/I6: strictly increasing outputs and, with them, input keys
        assert np.all(np.diff(orr) > 0)
        kin = keys_of(coords[ir], (B,) + dims)
        assert np.all(np.diff(kin) > 0)
    # outputs sorted strictly by key
    ko = keys_of(a.out_coords, rb.out_grid)
    assert np.all(np.diff(ko) > 0)
    if f == s:
        # I2: non-overlapping pooling partitions the inputs it keeps
        assert np.all(cnt <= 1)
        assert rb.a_out <= rb.a_in


def test_counts_line_plane_single():
    """I7: one interior site -> f^3 outputs; a straight n-site line along x ->
    4(n+1) outputs for f=2; an n x n plane -> 2(n+1)^2 for f=2."""
    g = (1, 12, 12, 12)
    one = np.array([[0, 5, 5, 5]], np.int32)
    for f in (2, 3):
        assert oracle.Rulebook(one, g, f, 1).a_out == f ** 3
    n = 6
    line = np.array([[0, 2 + i, 5, 5] for i in range(n)], np.int32)
    assert oracle.Rulebook(line, g, 2, 1).a_out == 4 * (n + 1)
    plane = np.array([[0, 2 + i, 2 + j, 5] for i in range(n) for j in range(n)], np.int32)
    assert oracle.Rulebook(plane, g, 2, 1).a_out == 2 * (n + 1) ** 2


def test_translation_equivariance():
    """I8: shifting the input by a multiple of s shifts the outputs by the
    quotient and keeps the rule lists."""
    rng = np.random.default_rng(5)
    dims = (8, 8, 8)
    coords = gen.random_sites(rng, 1, dims, 30)
    coords[:, 1:] += 4                  # away from every border of the big grid
    big = (1, 24, 24, 24)
    for f, s in ((2, 1), (3, 1), (2, 2)):
        a = oracle.Rulebook(coords, big, f, s).arrays()
        sh = coords.copy()
        sh[:, 1:] += np.array([2, 4, 6], np.int32)
        b = oracle.Rulebook(sh, big, f, s).arrays()
        exp = a.out_coords.copy()
        exp[:, 1:] += np.array([2, 4, 6], np.int32) // s
        np.testing.assert_array_equal(b.out_coords, exp)
        np.testing.assert_array_equal(b.in_rows, a.in_rows)
        np.testing.assert_array_equal(b.out_rows, a.out_rows)


def test_f1_is_elementwise_affine():
    rng = np.random.default_rng(3)
    coords = gen.random_sites(rng, 1, (5, 5, 5), 20)
    x = rng.standard_normal((20, 1))
    W = np.array([[[1.7]]])
    b = np.array([-0.4])
    rb = oracle.Rulebook(coords, (1, 5, 5, 5), 1, 1)
    y, g = oracle.conv_fwd(rb, x, np.zeros(1), W, b)
    order = np.argsort(keys_of(coords, (1, 5, 5, 5)))
    np.testing.assert_allclose(y[:, 0], 1.7 * x[order, 0] - 0.4, rtol=1e-14)
    assert g[0] == pytest.approx(-0.4)


def test_empty_input_gives_ground_state_only():
    rb = oracle.Rulebook(np.zeros((0, 4), np.int32), (1, 4, 4, 4), 2, 1)
    assert rb.a_out == 0 and rb.n_pairs == 0
    W = np.full((8, 2, 3), 0.25)
    y, g = oracle.conv_fwd(rb, np.zeros((0, 2)), np.array([1.0, -2.0]), W, np.array([0.5, 0, 1]))
    assert y.shape == (0, 3)
    np.testing.assert_allclose(g, np.array([0.5, 0.0, 1.0]) + 8 * 0.25 * (1.0 - 2.0))


def test_error_statuses():
    g = (2, 4, 4, 4)
    with pytest.raises(oracle.OracleError) as e:
        oracle.Rulebook(np.array([[0, 1, 1, 1], [0, 1, 1, 1]], np.int32), g, 2, 1)
    assert e.value.status == "duplicate"
    for bad in ([2, 0, 0, 0], [0, 4, 0, 0], [0, 0, -1, 0], [-1, 0, 0, 0], [0, 0, 0, 4]):
        with pytest.raises(oracle.OracleError) as e:
            oracle.Rulebook(np.array([bad], np.int32), g, 2, 1)
        assert e.value.status == "range"
    with pytest.raises(oracle.OracleError) as e:
        oracle.Rulebook(np.zeros((1, 4), np.int32), g, 0, 1)
    assert e.value.status == "invalid"
