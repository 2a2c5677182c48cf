"""Pins of the oracle's hypercubic lattice in d = 1..4 dimensions (section 1.2:
the construction is the same in any dimension; the smallest filter has 2^d
sites), against things other than the oracle itself (CPU only):

* offset counts f^d;
* brute-force active sets and rule lists, enumerating every output site of
  the grid and every offset of its window (section 1.3, second active-site
  rule, and the rules of Q);
* dense equivalence: a naive dense d-dimensional cross-correlation and
  max-pool, loops written here over offsets with numpy slicing, over the
  field that holds M_in at active sites and g_in elsewhere, equal the
  sparse results at active outputs; inactive dense outputs equal g_out;
* central finite differences of the d = 4 forward for the gradients;
* the 3D path of this construction equals the oracle's cubic lattice, and
  the 2D one its square lattice (Figure 2 (i), (iii));
* error statuses.
"""
import itertools

import numpy as np
import pytest

import oracle


def out_extent(m, f, s):
    return (m - f) // s + 1 if m >= f else 0


def random_sites_nd(rng, B, dims, n):
    """n distinct sites (b, x_1..x_d), in random order."""
    total = B * int(np.prod(dims))
    idx = rng.choice(total, size=min(n, total), replace=False)
    cols = []
    rest = idx
    for m in dims:  # x_1 fastest
        cols.append(rest % m)
        rest = rest // m
    return np.stack([rest] + cols, axis=1).astype(np.int32)


def offsets_nd(f, d):
    """offset k -> (k_1, .., k_d), k = sum_a k_a f^(a-1), written out by enumeration"""
    out = []
    for k in range(f ** d):
        out.append(tuple((k // f ** a) % f for a in range(d)))
    return out


@pytest.mark.parametrize("d", [1, 2, 3, 4])
@pytest.mark.parametrize("f", [1, 2, 3])
def test_offset_count_is_f_to_the_d(d, f):
    rng = np.random.default_rng(d * 10 + f)
    dims = (5,) * d
    coords = random_sites_nd(rng, 1, dims, 6)
    rb = oracle.Rulebook(coords, (1,) + dims, f, 1, ndim=d)
    assert rb.K == f ** d
    assert rb.ndim == d and rb.out_grid == (1,) + tuple(out_extent(m, f, 1) for m in dims)


CASES = [  # (d, B, dims, n, f, s)
    (4, 2, (5, 4, 6, 5), 60, 2, 1),
    (4, 1, (6, 5, 5, 6), 90, 2, 2),
    (4, 1, (5, 5, 4, 5), 40, 3, 1),
    (4, 2, (7, 6, 5, 6), 70, 3, 2),
    (4, 1, (6, 6, 6, 6), 50, 1, 2),
    (2, 3, (9, 8), 30, 3, 2),
    (1, 2, (17,), 9, 2, 1),
    (1, 1, (20,), 12, 3, 3),
]


@pytest.mark.parametrize("case", CASES, ids=[str(i) for i in range(len(CASES))])
def test_active_set_and_rules_brute_force(case):
    d, B, dims, n, f, s = case
    rng = np.random.default_rng(7 + CASES.index(case))
    coords = random_sites_nd(rng, B, dims, n)
    rb = oracle.Rulebook(coords, (B,) + dims, f, s, ndim=d)
    a = rb.arrays()
    row_of = {tuple(c): r for r, c in enumerate(coords.tolist())}
    mo = [out_extent(m, f, s) for m in dims]
    offs = offsets_nd(f, d)
    expect_out, expect_pairs = [], {k: [] for k in range(len(offs))}
    # every output site in key order: b slowest, then x_d .. x_1 (x_1 fastest)
    for b in range(B):
        for rev in itertools.product(*[range(m) for m in reversed(mo)]):
            o = tuple(reversed(rev))
            hits = []
            for k, kk in enumerate(offs):
                r = row_of.get((b,) + tuple(s * o[a] + kk[a] for a in range(d)))
                if r is not None:
                    hits.append((k, r))
            if hits:
                row = len(expect_out)
                expect_out.append((b,) + o)
                for k, r in hits:
                    expect_pairs[k].append((r, row))
    assert rb.out_grid == (B, *mo)
    np.testing.assert_array_equal(a.out_coords,
                                  np.array(expect_out, np.int32).reshape(-1, d + 1))
    for k in range(len(offs)):
        seg = slice(a.offsets[k], a.offsets[k + 1])
        got = list(zip(a.in_rows[seg].tolist(), a.out_rows[seg].tolist()))
        assert got == expect_pairs[k]


def dense_field(coords, x, g_in, B, dims):
    """[B, m_1, .., m_d, C]: x at active sites, g_in elsewhere."""
    C = x.shape[1]
    F = np.empty((B,) + tuple(dims) + (C,), np.float64)
    F[...] = g_in
    for r, c in enumerate(coords.tolist()):
        F[tuple(c)] = x[r]
    return F


def dense_conv(F, W, bias, f, s, d):
    """Valid d-dimensional cross-correlation with stride s: out[o] = bias +
    sum_k F[s*o + k] W_k, a loop over offsets."""
    B = F.shape[0]
    dims = F.shape[1:1 + d]
    mo = [out_extent(m, f, s) for m in dims]
    Cout = W.shape[2]
    out = np.zeros((B,) + tuple(mo) + (Cout,)) + bias
    for k, kk in enumerate(offsets_nd(f, d)):
        sl = (slice(None),) + tuple(slice(kk[a], kk[a] + s * (mo[a] - 1) + 1, s) for a in range(d))
        out += F[sl] @ W[k]
    return out


def dense_maxpool(F, f, s, d):
    """max over the window, and the first offset (k ascending) reaching it"""
    B = F.shape[0]
    dims = F.shape[1:1 + d]
    mo = [out_extent(m, f, s) for m in dims]
    best = None
    arg = None
    for k, kk in enumerate(offsets_nd(f, d)):
        sl = (slice(None),) + tuple(slice(kk[a], kk[a] + s * (mo[a] - 1) + 1, s) for a in range(d))
        v = F[sl]
        if best is None:
            best, arg = v.copy(), np.zeros(v.shape, np.int64)
        else:
            upd = v > best
            best = np.where(upd, v, best)
            arg = np.where(upd, k, arg)
    return best, arg


@pytest.mark.parametrize("case", CASES[:5], ids=[str(i) for i in range(5)])
def test_conv_dense_equivalence(case):
    d, B, dims, n, f, s = case
    rng = np.random.default_rng(100 + CASES.index(case))
    coords = random_sites_nd(rng, B, dims, n)
    Cin, Cout = 3, 4
    x = rng.standard_normal((len(coords), Cin))
    g_in = rng.standard_normal(Cin)
    W = rng.standard_normal((f ** d, Cin, Cout))
    bias = rng.standard_normal(Cout)
    rb = oracle.Rulebook(coords, (B,) + dims, f, s, ndim=d)
    y, g_out = oracle.conv_fwd(rb, x, g_in, W, bias)
    dense = dense_conv(dense_field(coords, x, g_in, B, dims), W, bias, f, s, d)
    oc = rb.arrays().out_coords
    np.testing.assert_allclose(y, dense[tuple(oc.T)], rtol=1e-12, atol=1e-12)
    inactive = np.ones(dense.shape[:-1], bool)
    inactive[tuple(oc.T)] = False
    np.testing.assert_allclose(dense[inactive], np.broadcast_to(g_out, dense[inactive].shape),
                               rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("case", [c for c in CASES if c[5] >= 2],
                         ids=[str(i) for i, c in enumerate(CASES) if c[5] >= 2])
def test_maxpool_dense_equivalence(case):
    d, B, dims, n, f, s = case
    rng = np.random.default_rng(200 + CASES.index(case))
    coords = random_sites_nd(rng, B, dims, n)
    C = 3
    x = rng.standard_normal((len(coords), C))
    x[rng.random(x.shape) < 0.2] = 0.0  # ties with g = 0
    g_in = np.zeros(C)
    rb = oracle.Rulebook(coords, (B,) + dims, f, s, ndim=d)
    y, g_out, ak, _ = oracle.maxpool_fwd(rb, x, g_in)
    best, arg = dense_maxpool(dense_field(coords, x, g_in, B, dims), f, s, d)
    oc = rb.arrays().out_coords
    np.testing.assert_array_equal(y, best[tuple(oc.T)])
    np.testing.assert_array_equal(ak, arg[tuple(oc.T)])
    np.testing.assert_array_equal(g_out, g_in)


def test_conv_bwd_finite_differences_4d():
    rng = np.random.default_rng(9)
    d, B, dims, f, s, Cin, Cout = 4, 1, (3, 4, 3, 3), 2, 1, 2, 2
    coords = random_sites_nd(rng, B, dims, 12)
    x = rng.standard_normal((len(coords), Cin))
    g_in = rng.standard_normal(Cin)
    W = rng.standard_normal((f ** d, Cin, Cout)) * 0.5
    bias = rng.standard_normal(Cout)
    rb = oracle.Rulebook(coords, (B,) + dims, f, s, ndim=d)
    dy = rng.uniform(-1, 1, (rb.a_out, Cout))
    dg = rng.uniform(-1, 1, Cout)
    got = oracle.conv_bwd(rb, x, g_in, W, bias, dy, dg)

    def loss(x_, g_, W_, b_):
        y, go = oracle.conv_fwd(rb, x_, g_, W_, b_)
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


@pytest.mark.parametrize("f,s", [(3, 1), (2, 2), (3, 2)])
def test_three_and_two_dims_match_the_cubic_and_square_lattices(f, s):
    rng = np.random.default_rng(f * 3 + s)
    c3 = random_sites_nd(rng, 2, (7, 6, 8), 60)
    a = oracle.Rulebook(c3, (2, 7, 6, 8), f, s).arrays()
    b = oracle.Rulebook(c3, (2, 7, 6, 8), f, s, ndim=3).arrays()
    for name in ("out_coords", "in_rows", "out_rows", "offsets"):
        np.testing.assert_array_equal(getattr(a, name), getattr(b, name), err_msg=name)
    c2 = random_sites_nd(rng, 2, (9, 7), 30)
    sq = oracle.Rulebook(np.concatenate([c2, np.zeros((len(c2), 1), np.int32)], 1),
                         (2, 9, 7, 1), f, s, lattice="square").arrays()
    nd = oracle.Rulebook(c2, (2, 9, 7), f, s, ndim=2).arrays()
    np.testing.assert_array_equal(sq.out_coords[:, :3], nd.out_coords)
    for name in ("in_rows", "out_rows", "offsets"):
        np.testing.assert_array_equal(getattr(sq, name), getattr(nd, name), err_msg=name)


def test_error_statuses():
    c = np.array([[0, 1, 1, 1, 1], [0, 1, 1, 1, 1]], np.int32)
    with pytest.raises(oracle.OracleError) as e:
        oracle.Rulebook(c, (1, 3, 3, 3, 3), 2, 1, ndim=4)
    assert e.value.code == 3  # duplicate
    grid = (2, 3, 4, 5, 6)
    for col in range(5):  # b and every axis, one past each end
        for v in (-1, grid[col]):
            site = np.array([[1, 2, 3, 4, 5]], np.int32)
            site[0, col] = v
            with pytest.raises(oracle.OracleError) as e:
                oracle.Rulebook(site, grid, 2, 1, ndim=4)
            assert e.value.code == 2  # range
    # the largest site is in range
    assert oracle.Rulebook(np.array([[1, 2, 3, 4, 5]], np.int32), grid, 2, 1, ndim=4).a_in == 1
    with pytest.raises(oracle.OracleError) as e:
        oracle.Rulebook(np.zeros((0, 6), np.int32), (1, 3, 3, 3, 3, 3), 2, 1, ndim=5)
    assert e.value.code == 1  # invalid
