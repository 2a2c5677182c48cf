"""GPU parity on the five synthetic workloads, at their full sizes.

* Small stacks run through the oracle layer by layer: every layer of the GPU
  sees the same fp32 input as the oracle (the oracle's previous output rounded
  to fp32) and is compared in isolation, forward and backward.
* Large layers run at full size, in the launch configuration the benchmark
  times, and are compared inside an interior sub-box: the oracle runs on the
  active sites inside a cube; an output whose whole window lies inside the
  cube sees exactly the same inputs as in the full problem, and so does an
  input whose every output lies inside.  The weight gradient is compared with
  an output gradient that is zero outside the interior outputs, on both sides.
* Every layer of the two deep stacks (the surfaces, five conv + pool levels;
  the deep step, a 3x3x3 conv and six conv + pool levels) runs this way on
  its own full-size input: the active sites the definition gives for the
  layers below it, with seeded features.
* Full-size rulebooks are checked against their definition, computed here
  with numpy on a dense occupancy grid: output o is active iff some site
  s*o + k of its window is active, and pair (r, o) of offset k exists iff
  site s*o + k is active with row r.

Tolerances follow tests/helpers.py: rulebooks, pooling values, argmax and
(disjoint-window) pooling input gradients bit-exact; per-site results under
the plain 1e-4 / 1e-5 rule; reductions over pairs relative to the rss of
their terms.
"""
from __future__ import annotations

import numpy as np
import pytest

torch = pytest.importorskip("torch")

import oracle  # noqa: E402
from gen import make_config, make_dy, stream_rng  # noqa: E402

from helpers import (assert_exact, assert_reduction, assert_site, definition_rulebook,  # noqa: E402
                     dev, host, keys_of, kink_flips, sq)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def scn():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_1505_02890_amd as m
    m.lib()
    return m


def _f32(a):
    a = np.asarray(a)
    return a if a.dtype == np.float32 else a.astype(np.float32)


def step(msg):
    print(f"[configs] {msg}", flush=True)


# --------------------------------------------------------------------------
# rulebook against its definition (helpers.definition_rulebook)
# --------------------------------------------------------------------------

def check_rulebook_definition(g, defn):
    """The GPU rulebook equals the definition, bit for bit."""
    oc, off, ir, orr = defn
    assert g.a_out == len(oc)
    assert_exact("offsets", np.asarray(g.offsets), off)
    goc, gir, gorr = g.export()
    assert_exact("out_coords", host(goc), oc)
    assert_exact("in_rows", host(gir), ir)
    assert_exact("out_rows", host(gorr), orr)


# --------------------------------------------------------------------------
# interior sub-box comparison of one layer
# --------------------------------------------------------------------------

def subbox(coords, n_target, seed):
    """Sites of one sample inside a cube around a random active site, grown
    until it holds about n_target sites.  Returns (mask, b, lo, hi)."""
    rng = stream_rng(seed, 7)
    c = np.asarray(coords, np.int64)
    centre = c[int(rng.integers(len(c)))]
    same = c[:, 0] == centre[0]
    d = np.max(np.abs(c[:, 1:4] - centre[1:4]), axis=1)
    dd = np.sort(d[same])
    h = int(dd[min(n_target, len(dd)) - 1])
    lo, hi = centre[1:4] - h, centre[1:4] + h
    mask = same & (d <= h)
    return mask, int(centre[0]), lo, hi


def inside(coords, b, lo, hi):
    c = np.asarray(coords, np.int64)
    return (c[:, 0] == b) & np.all((c[:, 1:4] >= lo) & (c[:, 1:4] <= hi), axis=1)


def find_rows(sorted_coords, grid_out, query_coords):
    """Rows of query sites in a key-sorted coordinate list (all present)."""
    ks = keys_of(sorted_coords, grid_out)
    q = keys_of(query_coords, grid_out)
    pos = np.searchsorted(ks, q)
    assert np.all(ks[np.minimum(pos, len(ks) - 1)] == q)
    return pos


def conv_layer_interior(scn, coords, grid, x, g_in, W, bias, f, s, relu, seed, n_sub=6000,
                        defn=None):
    """Full-size GPU layer vs oracle on an interior sub-box: y, g_out, dx (per
    site), dW, dbias, dg_in (reductions).  Returns the definition's output
    sites and grid (or the GPU's, when defn is None and the rulebook was
    checked elsewhere)."""
    x = _f32(x)
    g_in = _f32(g_in)
    K, Cin, Cout = W.shape
    g = scn.build_rulebook(dev(np.ascontiguousarray(coords, np.int32)), grid, f, s)
    if defn is not None:
        check_rulebook_definition(g, defn)
        out_sites = defn[0]
    else:
        out_sites = host(g.out_coords())
    xd = dev(x)
    yd, god = scn.conv_fwd(g, xd, dev(g_in), dev(W), dev(bias), relu=relu)
    m, b, lo, hi = subbox(coords, n_sub, seed)
    sub = np.ascontiguousarray(np.asarray(coords)[m], np.int32)
    o = oracle.Rulebook(sub, grid, f, s)
    oc = o.arrays().out_coords.astype(np.int64)
    # interior outputs: window s*o + [0, f) inside the cube
    io = (oc[:, 0] == b) & np.all((s * oc[:, 1:4] >= lo) & (s * oc[:, 1:4] + f - 1 <= hi), axis=1)
    assert io.sum() > 0
    y_ref, go_ref = oracle.conv_fwd(o, x[m], g_in, W, bias, relu=relu)
    gr = find_rows(out_sites, g.out_grid, oc[io])
    y_gpu = host(yd)[gr]
    assert_site("y", y_gpu, y_ref[io])
    assert_site("g_out", host(god), go_ref)
    pre_ref = oracle.conv_fwd(o, x[m], g_in, W, bias, relu=False)[0] if relu else y_ref
    if relu:
        assert kink_flips(y_gpu, pre_ref[io]) <= 1e-4 * y_gpu.size + 1
    # backward: interior outputs carry the gradient, the others zero; the
    # ReLU mask of the interior rows is the oracle's forward on both sides
    dy_o = make_dy(seed, len(oc), Cout)
    dy_o[~io] = 0.0
    gr_t = torch.from_numpy(gr).cuda()
    dy_full = torch.zeros((g.a_out, Cout), dtype=torch.float32, device="cuda")
    dy_full[gr_t] = dev(dy_o[io])
    dg = np.zeros(Cout, np.float32)
    if relu:
        yd[gr_t] = dev(_f32(y_ref[io]))
        god = dev(_f32(go_ref))
    ref = oracle.conv_bwd(o, x[m], g_in, W, bias, dy_o, dg, relu=relu)
    dyb = dy_o * (pre_ref > 0) if relu else dy_o
    sig = {k: np.sqrt(v) for k, v in
           oracle.conv_bwd(o, sq(x[m]), sq(g_in), sq(W), None, sq(dyb), None).items()}
    out = scn.conv_bwd(g, xd, dev(g_in), dev(W), yd, god, dy_full, dev(dg), relu=relu)
    for k in ("dW", "dbias", "dg_in"):
        assert_reduction(k, host(out[k]), ref[k], sig[k])
    # dx at inputs whose outputs all lie inside: coordinates in [lo+f-1, hi-f+1]
    ii = inside(sub, b, lo + f - 1, hi - f + 1)
    rows_full = np.nonzero(m)[0][ii]
    assert_site("dx", host(out["dx"])[rows_full], ref["dx"][ii])
    del yd, dy_full, out
    return out_sites, g.out_grid


def pool_layer_interior(scn, coords, grid, x, g_in, f, seed, n_sub=6000, s=None, defn=None):
    """Max-pool (filter f, stride s, default s = f) at full size; outputs whose
    window lies in an interior sub-box are compared with the oracle run on the
    sub-box alone."""
    s = f if s is None else s
    x = _f32(x)
    g_in = _f32(g_in)
    g = scn.build_rulebook(dev(np.ascontiguousarray(coords, np.int32)), grid, f, s)
    if defn is not None:
        check_rulebook_definition(g, defn)
        out_sites = defn[0]
    else:
        out_sites = host(g.out_coords())
    yd, god, am = scn.maxpool_fwd(g, dev(x), dev(g_in))
    m, b, lo, hi = subbox(coords, n_sub, seed)
    sub = np.ascontiguousarray(np.asarray(coords)[m], np.int32)
    o = oracle.Rulebook(sub, grid, f, s)
    oc = o.arrays().out_coords.astype(np.int64)
    io = (oc[:, 0] == b) & np.all((s * oc[:, 1:4] >= lo) & (s * oc[:, 1:4] + f - 1 <= hi), axis=1)
    y_ref, _, ak_ref, _ = oracle.maxpool_fwd(o, x[m], g_in)
    gr = find_rows(out_sites, g.out_grid, oc[io])
    assert_exact("pool y", host(yd)[gr], y_ref[io].astype(np.float32))
    assert_exact("argmax", host(am)[gr].astype(np.int32), ak_ref[io])
    assert_exact("pool g_out", host(god), g_in)
    C = x.shape[1]
    dy_o = np.zeros((len(oc), C), np.float32)
    dy_o[io] = make_dy(seed, int(io.sum()), C)
    dy_full = torch.zeros((g.a_out, C), dtype=torch.float32, device="cuda")
    dy_full[torch.from_numpy(gr).cuda()] = dev(dy_o[io])
    dx_ref, dg_ref = oracle.maxpool_bwd(o, x[m], g_in, dy_o, None)
    dxd, dgd = scn.maxpool_bwd(g, am, dy_full)
    # every input of the cube: each of its windows is interior (same argmax on
    # both sides) or carries a zero output gradient on both sides
    rows = np.nonzero(m)[0]
    if f <= s:
        assert_exact("pool dx", host(dxd)[rows], dx_ref.astype(np.float32))
    else:
        assert_site("pool dx", host(dxd)[rows], dx_ref)
    sig = np.sqrt(oracle.maxpool_bwd(o, x[m], g_in, sq(dy_o), None)[1])
    assert_reduction("pool dg_in", host(dgd), dg_ref, sig)
    del yd, am, dy_full, dxd
    return out_sites, g.out_grid


# --------------------------------------------------------------------------
# per-layer inputs of the deep stacks
# --------------------------------------------------------------------------

class StackChain:
    """The input sites of every layer of a workload's stack, from the
    definition (each layer's active outputs are the next layer's inputs), and
    each layer's definition rulebook; computed on first use."""

    def __init__(self, cfg):
        self.cfg = cfg
        self.sites = {0: (cfg.coords, tuple(cfg.grid))}
        self.defs = {}

    def defn(self, li):
        if li not in self.defs:
            coords, grid = self.inputs(li)
            L = self.cfg.layers[li]
            step(f"definition of layer {li} ({L.kind} f={L.f} s={L.s}) on {len(coords)} sites")
            self.defs[li] = definition_rulebook(coords, grid, L.f, L.s)
        return self.defs[li]

    def inputs(self, li):
        if li not in self.sites:
            prev_coords, prev_grid = self.inputs(li - 1)
            L = self.cfg.layers[li - 1]
            oc = self.defn(li - 1)[0]
            og = (prev_grid[0],) + tuple((m - L.f) // L.s + 1 for m in prev_grid[1:])
            self.sites[li] = (oc, og)
        return self.sites[li]


def layer_features(cfg, li, n, C):
    """Seeded input features of layer li of a stack: the workload's own input
    for layer 0, else ReLU-like values (about half exact zeros) and a
    non-negative ground state, as a ReLU layer below would give."""
    if li == 0:
        return cfg.features, cfg.g0
    rng = stream_rng(cfg.seed, 100 + li)
    x = rng.standard_normal((n, C), dtype=np.float32)
    np.maximum(x, 0.0, out=x)
    g = np.abs(rng.standard_normal(C)).astype(np.float32) * 0.3
    g[rng.random(C) < 0.3] = 0.0
    return x, g


def run_stack_layer(scn, cfg, chain, li, n_sub):
    L = cfg.layers[li]
    coords, grid = chain.inputs(li)
    defn = chain.defn(li)
    C = L.cin if L.kind == "conv" else cfg.layers[li - 1].cout
    x, g_in = layer_features(cfg, li, len(coords), C)
    step(f"layer {li}: {L.kind} f={L.f} s={L.s} C={C}->{L.cout or C} on {len(coords)} sites")
    if L.kind == "conv":
        conv_layer_interior(scn, coords, grid, x, g_in, cfg.weights[li], cfg.biases[li], L.f,
                            L.s, L.relu, seed=cfg.seed + 1000 + li, n_sub=n_sub, defn=defn)
    else:
        pool_layer_interior(scn, coords, grid, x, g_in, L.f, seed=cfg.seed + 1000 + li,
                            n_sub=n_sub, s=L.s, defn=defn)
    torch.cuda.empty_cache()


def _sub_for(L, base):
    """Sub-box size that keeps the oracle's work per layer to seconds."""
    if L.kind != "conv":
        return base
    macs = L.f ** 3 * L.cin * max(L.cout, 1)
    return int(max(800, min(base, 3e8 / max(macs, 1) / 3)))


# --------------------------------------------------------------------------
# the workloads
# --------------------------------------------------------------------------

def test_trefoil_forward_chain(scn):
    """One knotted curve in 32^3: 2x2x2 conv 1->16 then 2x2x2/2 max-pool, forward."""
    cfg = make_config(0)
    conv, pool = cfg.layers
    g = scn.build_rulebook(dev(cfg.coords), cfg.grid, conv.f, conv.s)
    o = oracle.Rulebook(cfg.coords, cfg.grid, conv.f, conv.s)
    oa = o.arrays()
    oc, ir, orr = g.export()
    assert_exact("out_coords", host(oc), oa.out_coords)
    assert_exact("in_rows", host(ir), oa.in_rows)
    assert_exact("out_rows", host(orr), oa.out_rows)
    assert g.a_out > g.a_in  # growth (Figure 1)
    y, g1 = scn.conv_fwd(g, dev(cfg.features), dev(cfg.g0), dev(cfg.weights[0]),
                         dev(cfg.biases[0]))
    y_ref, g1_ref = oracle.conv_fwd(o, cfg.features, cfg.g0, cfg.weights[0], cfg.biases[0])
    assert_site("y", host(y), y_ref)
    assert_site("g_out", host(g1), g1_ref)
    x2, g2 = _f32(y_ref), _f32(g1_ref)
    pg = scn.build_rulebook(dev(oa.out_coords), oa.out_grid, pool.f, pool.s)
    po = oracle.Rulebook(oa.out_coords, oa.out_grid, pool.f, pool.s)
    yp, gp, am = scn.maxpool_fwd(pg, dev(x2), dev(g2))
    yp_ref, gp_ref, ak_ref, _ = oracle.maxpool_fwd(po, x2, g2)
    assert pg.a_out < pg.a_in  # shrinkage (Figure 1)
    assert_exact("pool y", host(yp), yp_ref.astype(np.float32))
    assert_exact("argmax", host(am).astype(np.int32), ak_ref)


def test_curve_batch_stack_layerwise(scn):
    """16 closed walks in 64^3; 4 x [2x2x2 conv + ReLU, 2x2x2/2 max-pool],
    channels 32/64/96/128; every layer forward and backward in isolation,
    the backward chained through the oracle's gradients."""
    cfg = make_config(1)
    coords, grid = cfg.coords, cfg.grid
    x, g = _f32(cfg.features), _f32(cfg.g0)
    saved = []
    # forward chain through the oracle; each GPU layer sees the same input
    for li, L in enumerate(cfg.layers):
        o = oracle.Rulebook(coords, grid, L.f, L.s)
        oa = o.arrays()
        gr = scn.build_rulebook(dev(np.ascontiguousarray(coords)), grid, L.f, L.s)
        goc, gir, gorr = gr.export()
        assert_exact(f"layer {li} out_coords", host(goc), oa.out_coords)
        assert_exact(f"layer {li} in_rows", host(gir), oa.in_rows)
        assert_exact(f"layer {li} out_rows", host(gorr), oa.out_rows)
        if L.kind == "conv":
            W, b = cfg.weights[li], cfg.biases[li]
            y_ref, go_ref = oracle.conv_fwd(o, x, g, W, b, relu=L.relu)
            pre_ref, gpre_ref = oracle.conv_fwd(o, x, g, W, b, relu=False)
            yd, god = scn.conv_fwd(gr, dev(x), dev(g), dev(W), dev(b), relu=L.relu)
            assert_site(f"layer {li} y", host(yd), y_ref)
            assert_site(f"layer {li} g", host(god), go_ref)
            saved.append(dict(o=o, g=gr, x=x, gin=g, y=y_ref, go=go_ref, pre=pre_ref,
                              gpre=gpre_ref, W=W, b=b, L=L))
        else:
            y_ref, go_ref, ak_ref, _ = oracle.maxpool_fwd(o, x, g)
            yd, god, am = scn.maxpool_fwd(gr, dev(x), dev(g))
            assert_exact(f"layer {li} pool y", host(yd), y_ref.astype(np.float32))
            assert_exact(f"layer {li} argmax", host(am).astype(np.int32), ak_ref)
            saved.append(dict(o=o, g=gr, x=x, gin=g, am=am, L=L))
        coords, grid = oa.out_coords, oa.out_grid
        x, g = _f32(y_ref), _f32(go_ref)
    # backward chain: dy U[-1, 1] on the top layer's rows, dg = 0 at the top
    dy = make_dy(cfg.seed, len(coords), x.shape[1])
    dg = np.zeros(x.shape[1], np.float32)
    for li in range(len(saved) - 1, -1, -1):
        S = saved[li]
        L, o, gr = S["L"], S["o"], S["g"]
        if L.kind == "pool":
            dx_ref, dgi_ref = oracle.maxpool_bwd(o, S["x"], S["gin"], dy, dg)
            dxd, dgid = scn.maxpool_bwd(gr, S["am"], dev(dy), dev(dg))
            assert_exact(f"layer {li} pool dx", host(dxd), dx_ref.astype(np.float32))
            sg = np.sqrt(oracle.maxpool_bwd(o, S["x"], S["gin"], sq(dy), sq(dg))[1])
            assert_reduction(f"layer {li} dg_in", host(dgid), dgi_ref, sg)
        else:
            # the ReLU mask comes from the oracle's forward on both sides
            ref = oracle.conv_bwd(o, S["x"], S["gin"], S["W"], S["b"], dy, dg, relu=True)
            dyb = dy * (S["pre"] > 0)
            dgb = dg * (S["gpre"] > 0)
            sig = {k: np.sqrt(v) for k, v in oracle.conv_bwd(
                o, sq(S["x"]), sq(S["gin"]), sq(S["W"]), None, sq(dyb), sq(dgb)).items()}
            out = scn.conv_bwd(gr, dev(S["x"]), dev(S["gin"]), dev(S["W"]), dev(_f32(S["y"])),
                               dev(_f32(S["go"])), dev(dy), dev(dg), relu=True)
            assert_site(f"layer {li} dx", host(out["dx"]), ref["dx"])
            for k in ("dW", "dbias", "dg_in"):
                assert_reduction(f"layer {li} {k}", host(out[k]), ref[k], sig[k])
            dx_ref, dgi_ref = ref["dx"], ref["dg_in"]
        dy, dg = _f32(dx_ref), _f32(dgi_ref)


@pytest.fixture(scope="module")
def surfaces():
    cfg = make_config(2)
    return cfg, StackChain(cfg)


@pytest.mark.parametrize("li", list(range(10)))
def test_surfaces_layer(scn, surfaces, li):
    """32 voxelised shells in 128^3, 5 x [2x2x2 conv + ReLU, 2x2x2/2
    max-pool], channels 32..160: layer li at full size on the definition's
    sites, forward and backward, against the oracle in a sub-box; the
    rulebook against its definition."""
    cfg, chain = surfaces
    run_stack_layer(scn, cfg, chain, li, _sub_for(cfg.layers[li], 6000))


def test_surfaces_overlapping_pool(scn, surfaces):
    """The paper's overlapping 3x3x3 stride-2 pooling on the first level's
    active set (ReLU-like features, many ties with the zero ground state)."""
    cfg, chain = surfaces
    oc, og = chain.inputs(1)
    xp = stream_rng(cfg.seed, 9).standard_normal((len(oc), 32)).astype(np.float32)
    xp[xp < 0] = 0.0
    pool_layer_interior(scn, oc, og, xp, np.zeros(32, np.float32), 3, seed=cfg.seed + 2, s=2,
                        defn=definition_rulebook(oc, og, 3, 2))


def test_microbenchmark_interior(scn):
    """1,000,000 shell sites in 512^3, one 3x3x3 conv 64->64: full-size
    rulebook against its definition; y, dx, dW, dbias, dg_in in sub-boxes."""
    cfg = make_config(3)
    L = cfg.layers[0]
    defn = definition_rulebook(cfg.coords, cfg.grid, L.f, L.s)
    for i in range(2):
        conv_layer_interior(scn, cfg.coords, cfg.grid, cfg.features, cfg.g0, cfg.weights[0],
                            cfg.biases[0], L.f, L.s, L.relu, seed=cfg.seed + 10 * i,
                            n_sub=3000, defn=defn if i == 0 else None)


def test_default_dense_view_wide_input(scn):
    """The 1M-site geometry with 80 input channels (a last 64-channel chunk of
    one 16-channel step) under the default dense-view policy, which picks the
    mask-sorted forward for this 3x3x3 layer of 4.4M outputs."""
    cfg = make_config(3)
    rng = stream_rng(cfg.seed, 300)
    Cin, Cout = 80, 48
    x = rng.standard_normal((len(cfg.coords), Cin), dtype=np.float32)
    g_in = (rng.standard_normal(Cin) * 0.3).astype(np.float32)
    W = (rng.standard_normal((27, Cin, Cout)) / np.sqrt(27 * Cin)).astype(np.float32)
    bias = (rng.standard_normal(Cout) * 0.1).astype(np.float32)
    g = scn.build_rulebook(dev(cfg.coords), cfg.grid, 3, 1)
    assert g.dense_view
    del g
    conv_layer_interior(scn, cfg.coords, cfg.grid, x, g_in, W, bias, 3, 1, True,
                        seed=cfg.seed + 30, n_sub=2500)


@pytest.fixture(scope="module")
def deep():
    cfg = make_config(4)
    assert 2_000_000 <= len(cfg.coords) <= 4_000_000
    return cfg, StackChain(cfg)


@pytest.mark.parametrize("li", list(range(13)))
def test_deep_step_layer(scn, deep, li):
    """8 samples of curve bundles and shells in 256^3 (2-4M sites): the
    3x3x3 conv (1->64, ReLU) and 6 x [2x2x2 conv + ReLU, 2x2x2/2 max-pool],
    channels 96..256: layer li at full size on the definition's sites,
    forward and backward, against the oracle in a sub-box."""
    cfg, chain = deep
    run_stack_layer(scn, cfg, chain, li, _sub_for(cfg.layers[li], 4000))
