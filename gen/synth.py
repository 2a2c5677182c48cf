"""Seeded synthetic sparse inputs shaped like the paper's workloads.

The paper (Section 2) trains on datasets that are not available here: pen
strokes (1D curves in 2+1D space-time), mesh surfaces rendered into a cubic
grid (SHREC2015, Section 2.2) and thresholded video differences.  The
generators below stand in for them with the same geometry: closed lattice
curves, including a knot-like curve as in Figure 1, and one-voxel-thick closed
surfaces (ellipsoids and even-exponent superquadrics under a random rotation).

Nothing here implements the method.  The functions only produce coordinate
lists, feature values, weights and output gradients, all from numpy
``default_rng`` streams derived from ``SEED_BASE + config_index``.

Reproducibility across hosts: only integer arithmetic and IEEE-exact
floating-point operations (+, -, *, /, sqrt) are applied to generated data,
except in the trefoil rasterisation, which uses Python's ``math.sin``/``cos``
on a fixed parameter grid.

Coordinate layout everywhere: ``int32[n][4]`` rows of (b, x, y, z).
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import List, Optional, Sequence, Tuple

import numpy as np

SEED_BASE = 150502890

# stream ids inside a config's SeedSequence
_S_COORDS, _S_FEATS, _S_WEIGHTS, _S_DY, _S_DG, _S_EXTRA = 0, 1, 2, 3, 4, 5


def stream_rng(seed: int, stream: int) -> np.random.Generator:
    """An independent generator for (seed, stream)."""
    return np.random.default_rng(np.random.SeedSequence([int(seed), int(stream)]))


# --------------------------------------------------------------------------
# curves
# --------------------------------------------------------------------------

_UNIT = np.array([[1, 0, 0], [-1, 0, 0], [0, 1, 0], [0, -1, 0], [0, 0, 1], [0, 0, -1]],
                 dtype=np.int64)


def _connect(points: Sequence[Tuple[int, int, int]]) -> List[Tuple[int, int, int]]:
    """Join consecutive lattice points of a closed polygon with unit steps
    (x first, then y, then z).  Returns the visited sites of the closed walk,
    without repeating the start."""
    out: List[Tuple[int, int, int]] = []
    n = len(points)
    for j in range(n):
        p = list(points[j])
        q = points[(j + 1) % n]
        out.append(tuple(p))
        for ax in range(3):
            while p[ax] != q[ax]:
                p[ax] += 1 if q[ax] > p[ax] else -1
                if tuple(p) != tuple(q):
                    out.append(tuple(p))
    return out


def _erase_loops(walk: List[Tuple[int, int, int]]) -> List[Tuple[int, int, int]]:
    """Chronological loop erasure: whenever a site is revisited, drop the loop
    in between.  A closed walk stays closed (consecutive sites stay adjacent)."""
    out: List[Tuple[int, int, int]] = []
    pos = {}
    for s in walk:
        if s in pos:
            cut = pos[s]
            for t in out[cut + 1:]:
                del pos[t]
            out = out[: cut + 1]
        else:
            pos[s] = len(out)
            out.append(s)
    # the closing step from out[-1] back to out[0] must be a unit step
    while len(out) > 2 and sum(abs(a - b) for a, b in zip(out[-1], out[0])) != 1:
        out.pop()
    return out


def trefoil_walk(rng: np.random.Generator, m: int = 32, target_steps: int = 400,
                 extent: int = 26) -> np.ndarray:
    """Closed self-avoiding 6-connected lattice walk that follows a trefoil
    knot (the curve of Figure 1), lengthened to about ``target_steps`` steps by
    seeded local detours.  Returns int64[n][3] sites (x, y, z), n = steps."""
    # parametric trefoil (sin t + 2 sin 2t, cos t - 2 cos 2t, -sin 3t)
    nt = 2000
    raw = []
    for j in range(nt):
        t = 2.0 * math.pi * j / nt
        raw.append((math.sin(t) + 2.0 * math.sin(2.0 * t),
                    math.cos(t) - 2.0 * math.cos(2.0 * t),
                    -math.sin(3.0 * t)))
    lo = [min(r[a] for r in raw) for a in range(3)]
    hi = [max(r[a] for r in raw) for a in range(3)]
    scale = extent / max(hi[a] - lo[a] for a in range(3))
    off = [(m - 1) / 2.0 - scale * (lo[a] + hi[a]) / 2.0 for a in range(3)]
    pts: List[Tuple[int, int, int]] = []
    for r in raw:
        q = tuple(int(math.floor(scale * r[a] + off[a] + 0.5)) for a in range(3))
        if not pts or q != pts[-1]:
            pts.append(q)
    while len(pts) > 1 and pts[-1] == pts[0]:
        pts.pop()
    walk = _erase_loops(_connect(pts))
    visited = set(walk)
    # seeded detours: replace the step a->b by a -> a+u -> b+u -> b
    tries = 0
    while len(walk) < target_steps and tries < 100000:
        tries += 1
        j = int(rng.integers(len(walk)))
        a = walk[j]
        b = walk[(j + 1) % len(walk)]
        e = tuple(bb - aa for aa, bb in zip(a, b))
        perp = [tuple(int(v) for v in u) for u in _UNIT if int(np.dot(u, e)) == 0]
        u = perp[int(rng.integers(len(perp)))]
        a2 = tuple(x + y for x, y in zip(a, u))
        b2 = tuple(x + y for x, y in zip(b, u))
        if a2 in visited or b2 in visited:
            continue
        if not all(0 <= c < m for c in a2 + b2):
            continue
        walk[j + 1:j + 1] = [a2, b2]
        visited.add(a2)
        visited.add(b2)
    return np.array(walk, dtype=np.int64)


def bridge_walk(rng: np.random.Generator, nsteps: int, m: int, *, centred: bool = True,
                redraws: int = 50) -> np.ndarray:
    """Closed lattice walk ("bridge"): nsteps/6 copies of each of the six unit
    steps in a seeded order.  With ``centred`` the walk is redrawn until its
    extent fits in m-3 and then centred in the box (after ``redraws`` failed
    draws the last one is centred and clipped).  Without ``centred`` it starts
    at a uniform random site and is clipped to the box.  Returns the distinct
    visited sites inside [0, m)^3 as int64[n][3]."""
    assert nsteps % 6 == 0
    steps = np.repeat(_UNIT, nsteps // 6, axis=0)
    for attempt in range(redraws if centred else 1):
        pos = np.cumsum(steps[rng.permutation(nsteps)], axis=0)
        lo, hi = pos.min(axis=0), pos.max(axis=0)
        if not centred or np.all(hi - lo <= m - 3):
            break
    if centred:
        pos = pos - lo + ((m - 1) - (hi - lo)) // 2
    else:
        pos = pos + rng.integers(0, m, size=3)
    keep = np.all((pos >= 0) & (pos < m), axis=1)
    return np.unique(pos[keep], axis=0)


# --------------------------------------------------------------------------
# surfaces
# --------------------------------------------------------------------------

def _rotation(rng: np.random.Generator) -> np.ndarray:
    """Uniform random rotation from a normalised 4-vector of normals."""
    q = rng.standard_normal(4)
    n = math.sqrt(q[0] * q[0] + q[1] * q[1] + q[2] * q[2] + q[3] * q[3])
    w, x, y, z = (float(v) / n for v in q)
    return np.array([
        [1 - 2 * (y * y + z * z), 2 * (x * y - z * w), 2 * (x * z + y * w)],
        [2 * (x * y + z * w), 1 - 2 * (x * x + z * z), 2 * (y * z - x * w)],
        [2 * (x * z - y * w), 2 * (y * z + x * w), 1 - 2 * (x * x + y * y)],
    ])


def shell_sites(rng: np.random.Generator, m: int, semi: Sequence[float],
                centre: Sequence[float], power: int = 2) -> np.ndarray:
    """One-voxel-thick closed surface: voxel p is on the shell iff
    F(p) <= 0 and some 6-neighbour has F > 0, where
    F(p) = sum_i (u_i / semi_i)^power - 1 and u = R^T (p + 0.5 - centre) for a
    seeded rotation R.  power 2 is an ellipsoid, 4 a rounded-box superquadric.
    Sites outside [0, m)^3 are dropped.  Returns int64[n][3] (x, y, z)."""
    assert power % 2 == 0 and power >= 2
    R = _rotation(rng)
    a = [float(v) for v in semi]
    c = [float(v) for v in centre]
    # farthest surface point from the centre: max(a) * 3^(1/2 - 1/power)
    reach = max(a) * (3.0 ** (0.5 - 1.0 / power)) + 2.0
    lo = [max(-1, int(math.floor(c[i] - reach))) for i in range(3)]
    hi = [min(m, int(math.ceil(c[i] + reach))) for i in range(3)]
    xs = [np.arange(lo[i], hi[i] + 1, dtype=np.float64) for i in range(3)]
    qx = (xs[0] + 0.5 - c[0])[:, None, None]
    qy = (xs[1] + 0.5 - c[1])[None, :, None]

    def inside_slab(z0: int, z1: int) -> np.ndarray:
        # inside-test for z-indices [z0, z1) of the box (out-of-box slices: False)
        zz = np.arange(z0, z1)
        ok = (zz >= 0) & (zz < len(xs[2]))
        res = np.zeros((len(xs[0]), len(xs[1]), len(zz)), dtype=bool)
        if not ok.any():
            return res
        qz = (xs[2][zz[ok]] + 0.5 - c[2])[None, None, :]
        F = np.full((len(xs[0]), len(xs[1]), int(ok.sum())), -1.0)
        for j in range(3):
            u = (qx * R[0][j] + qy * R[1][j]) + qz * R[2][j]
            t = u / a[j]
            t2 = t * t
            tp = t2
            for _ in range(power // 2 - 1):
                tp = tp * t2
            F = F + tp
        res[:, :, ok] = F <= 0.0
        return res

    out = []
    nz = len(xs[2])
    step = 24
    for z0 in range(0, nz, step):
        z1 = min(nz, z0 + step)
        ins = inside_slab(z0 - 1, z1 + 1)          # one halo slice each side
        core = ins[:, :, 1:-1]
        pad = np.pad(~ins, ((1, 1), (1, 1), (0, 0)), constant_values=True)
        nb = pad[:-2, 1:-1, 1:-1] | pad[2:, 1:-1, 1:-1]
        nb |= pad[1:-1, :-2, 1:-1] | pad[1:-1, 2:, 1:-1]
        nb |= pad[1:-1, 1:-1, :-2] | pad[1:-1, 1:-1, 2:]
        idx = np.argwhere(core & nb).astype(np.int64)
        idx[:, 2] += z0
        out.append(idx)
    idx = np.concatenate(out, axis=0) + np.array(lo, dtype=np.int64)
    keep = np.all((idx >= 0) & (idx < m), axis=1)
    return idx[keep]


# --------------------------------------------------------------------------
# small random inputs for tests
# --------------------------------------------------------------------------

def random_sites(rng: np.random.Generator, batch: int, dims: Sequence[int], n: int,
                 shuffle: bool = True) -> np.ndarray:
    """n distinct uniformly random sites of a (batch, mx, my, mz) grid as
    int32[n][4] rows (b, x, y, z), in seeded random order."""
    mx, my, mz = (int(d) for d in dims)
    vol = batch * mx * my * mz
    n = min(int(n), vol)
    flat = rng.choice(vol, size=n, replace=False)
    if not shuffle:
        flat = np.sort(flat)
    x = flat % mx
    y = (flat // mx) % my
    z = (flat // (mx * my)) % mz
    b = flat // (mx * my * mz)
    return np.stack([b, x, y, z], axis=1).astype(np.int32)


# --------------------------------------------------------------------------
# tetrahedral lattice (skewed coordinates: the grid of size m is the sites
# x + y + z < m; site (x, y, z) sits at x*e1 + y*e2 + z*e3 for unit vectors
# at 60 degrees to each other, so the grid is a regular tetrahedron)
# --------------------------------------------------------------------------

_SQ3 = math.sqrt(3.0)
_TETRA_BASIS = np.array([[1.0, 0.0, 0.0],
                         [0.5, _SQ3 / 2.0, 0.0],
                         [0.5, _SQ3 / 6.0, math.sqrt(2.0 / 3.0)]])   # rows e1, e2, e3
# the twelve nearest neighbours of a site, in skewed coordinates
_TETRA_NBRS = np.array([[1, 0, 0], [-1, 0, 0], [0, 1, 0], [0, -1, 0], [0, 0, 1], [0, 0, -1],
                        [1, -1, 0], [-1, 1, 0], [1, 0, -1], [-1, 0, 1], [0, 1, -1], [0, -1, 1]],
                       dtype=np.int64)


def tetra_sites(m: int) -> np.ndarray:
    """All sites x + y + z < m as int64[C(m+2, 3)][3] (x, y, z), z slowest."""
    r = np.arange(max(int(m), 0))
    z, y, x = np.meshgrid(r, r, r, indexing="ij")
    keep = (x + y + z) < m
    return np.stack([x[keep], y[keep], z[keep]], axis=1).astype(np.int64)


def tetra_random_sites(rng: np.random.Generator, batch: int, m: int, n: int,
                       shuffle: bool = True) -> np.ndarray:
    """n distinct uniformly random sites of `batch` tetrahedral grids of size m
    as int32[n][4] rows (b, x, y, z)."""
    cell = tetra_sites(m)
    vol = batch * len(cell)
    n = min(int(n), vol)
    flat = rng.choice(vol, size=n, replace=False)
    if not shuffle:
        flat = np.sort(flat)
    b, i = flat // max(len(cell), 1), flat % max(len(cell), 1)
    return np.concatenate([b[:, None], cell[i]], axis=1).astype(np.int32)


def triangle_sites(m: int) -> np.ndarray:
    """All sites x + y < m of a triangular grid of size m as int64[C(m+1, 2)][3]
    (x, y, 0), y slowest."""
    r = np.arange(max(int(m), 0))
    y, x = np.meshgrid(r, r, indexing="ij")
    keep = (x + y) < m
    return np.stack([x[keep], y[keep], np.zeros(int(keep.sum()), np.int64)], axis=1).astype(np.int64)


def tri_random_sites(rng: np.random.Generator, batch: int, m: int, n: int,
                     shuffle: bool = True) -> np.ndarray:
    """n distinct uniformly random sites of `batch` triangular grids of size m
    as int32[n][4] rows (b, x, y, 0)."""
    cell = triangle_sites(m)
    vol = batch * len(cell)
    n = min(int(n), vol)
    flat = rng.choice(vol, size=n, replace=False)
    if not shuffle:
        flat = np.sort(flat)
    b, i = flat // max(len(cell), 1), flat % max(len(cell), 1)
    return np.concatenate([b[:, None], cell[i]], axis=1).astype(np.int32)


def image_patch_sites(lattice: str, m: int, h: int, w: int) -> np.ndarray:
    """The sites of an h x w image placed in a 2D grid of size m as int64[h*w][3]
    (x, y, 0), row-major: on the square lattice a centred h x w rectangle, on
    the triangular lattice its affine image in skewed coordinates (a rhombus)
    centred on the triangle's centroid."""
    if lattice == "square":
        x0, y0 = (m - w) // 2, (m - h) // 2
    else:
        x0, y0 = m // 3 - w // 2, m // 3 - h // 2
    yy, xx = np.meshgrid(np.arange(h), np.arange(w), indexing="ij")
    pts = np.stack([xx.ravel() + x0, yy.ravel() + y0, np.zeros(h * w, np.int64)], axis=1)
    assert (pts[:, :2] >= 0).all() and (pts[:, :2] < m).all()
    assert lattice == "square" or (pts[:, 0] + pts[:, 1] < m).all()
    return pts.astype(np.int64)


def tetra_shell_sites(rng: np.random.Generator, m: int, semi: Sequence[float],
                      power: int = 2) -> np.ndarray:
    """The shell of `shell_sites` drawn on the tetrahedral grid of size m:
    site p is on it iff F(p) <= 0 and one of its twelve neighbours has F > 0,
    with F as there, evaluated at the site's position and centred on the
    grid's centroid.  Sites outside the grid are dropped.  Returns
    int64[n][3] (x, y, z) in skewed coordinates."""
    assert power % 2 == 0 and power >= 2
    R = _rotation(rng)
    a = [float(v) for v in semi]
    cs = (m - 1) / 4.0                       # centroid, skewed coordinates
    reach = max(a) * (3.0 ** (0.5 - 1.0 / power)) + 2.0
    # a skewed coordinate moves by at most sqrt(3/2) per unit of distance
    h = int(math.ceil(reach * math.sqrt(1.5))) + 1
    lo, hi = max(-1, int(math.floor(cs)) - h), min(m, int(math.ceil(cs)) + h)
    r = np.arange(lo, hi + 1, dtype=np.int64)
    E = _TETRA_BASIS

    def F(pts: np.ndarray) -> np.ndarray:
        d = pts.astype(np.float64) - cs
        ph = [d[:, 0] * E[0][j] + d[:, 1] * E[1][j] + d[:, 2] * E[2][j] for j in range(3)]
        out = np.full(len(pts), -1.0)
        for j in range(3):
            u = ph[0] * R[0][j] + ph[1] * R[1][j] + ph[2] * R[2][j]
            t = u / a[j]
            t2 = t * t
            tp = t2
            for _ in range(power // 2 - 1):
                tp = tp * t2
            out = out + tp
        return out

    found = []
    for z in r:
        yy, xx = np.meshgrid(r, r, indexing="ij")
        pts = np.stack([xx.ravel(), yy.ravel(), np.full(xx.size, z)], axis=1)
        pts = pts[(pts.min(axis=1) >= 0) & (pts.sum(axis=1) < m)]
        if len(pts) == 0:
            continue
        pts = pts[F(pts) <= 0.0]
        if len(pts) == 0:
            continue
        edge = np.zeros(len(pts), bool)
        for d in _TETRA_NBRS:
            edge |= F(pts + d) > 0.0
        found.append(pts[edge])
    if not found:
        return np.zeros((0, 3), np.int64)
    return np.concatenate(found, axis=0)


def _to_coords(per_sample: List[np.ndarray], rng: Optional[np.random.Generator]) -> np.ndarray:
    rows = []
    for b, s in enumerate(per_sample):
        s = np.unique(np.asarray(s, dtype=np.int64).reshape(-1, 3), axis=0)
        rows.append(np.concatenate([np.full((len(s), 1), b, np.int64), s], axis=1))
    c = np.concatenate(rows, axis=0) if rows else np.zeros((0, 4), np.int64)
    if rng is not None:
        c = c[rng.permutation(len(c))]
    return np.ascontiguousarray(c.astype(np.int32))


# --------------------------------------------------------------------------
# the five workloads
# --------------------------------------------------------------------------

@dataclass
class LayerSpec:
    kind: str            # "conv" or "pool"
    f: int               # filter / pooling size (linear)
    s: int               # stride
    cin: int = 0
    cout: int = 0
    relu: bool = False


@dataclass
class ConfigInput:
    index: int
    name: str
    seed: int
    grid: Tuple[int, int, int, int]       # (B, mx, my, mz)
    coords: np.ndarray                    # int32[n][4] (b, x, y, z)
    features: np.ndarray                  # float32[n][Cin]
    g0: np.ndarray                        # float32[Cin] input ground state (zero)
    layers: List[LayerSpec]
    weights: List[Optional[np.ndarray]]   # float32[K][Cin][Cout] per conv layer
    biases: List[Optional[np.ndarray]]    # float32[Cout] per conv layer
    backward: bool
    notes: dict = field(default_factory=dict)


CONFIGS = {
    0: "trefoil: B=1 m=32, C2 1->16 (no ReLU) -> MP2/2, forward only",
    1: "curves: B=16 m=64, 4x[C2+ReLU -> MP2/2] ch 32/64/96/128, fwd+bwd",
    2: "surfaces: B=32 m=128, 5x[C2+ReLU -> MP2/2] ch 32..160, fwd+bwd",
    3: "microbench: B=1 m=512, 1M shell sites, one C3 64->64, fwd+dX+dW",
    4: "deep: B=8 m=256, curves+shells ~2-4M sites, C3 1->64+ReLU, "
       "6x[C2+ReLU -> MP2/2] ch 96..256, fwd+bwd",
}


def _stack(ch: Sequence[int], cin: int = 1) -> List[LayerSpec]:
    out = []
    for c in ch:
        out.append(LayerSpec("conv", 2, 1, cin, c, True))
        out.append(LayerSpec("pool", 2, 2))
        cin = c
    return out


def _weights(rng: np.random.Generator, layers: List[LayerSpec], w_std, b_std):
    ws, bs = [], []
    for L in layers:
        if L.kind != "conv":
            ws.append(None)
            bs.append(None)
            continue
        K = L.f ** 3
        sd = w_std(L) if callable(w_std) else w_std
        ws.append((rng.standard_normal((K, L.cin, L.cout)) * sd).astype(np.float32))
        if b_std:
            bs.append((rng.standard_normal(L.cout) * b_std).astype(np.float32))
        else:
            bs.append(np.zeros(L.cout, np.float32))
    return ws, bs


def _he(L: LayerSpec) -> float:
    return math.sqrt(2.0 / (L.f ** 3 * L.cin))


def make_config(index: int, *, scale: float = 1.0) -> ConfigInput:
    """Build workload ``index`` (0-4).  ``scale`` < 1 shrinks the number of
    curves/shells for quick tests where noted (the grid and layers stay)."""
    seed = SEED_BASE + index
    rc = stream_rng(seed, _S_COORDS)
    rw = stream_rng(seed, _S_WEIGHTS)
    notes = {}
    if index == 0:
        m, B = 32, 1
        walk = trefoil_walk(rc, m=m, target_steps=400)
        coords = _to_coords([walk], rc)
        layers = [LayerSpec("conv", 2, 1, 1, 16, False), LayerSpec("pool", 2, 2)]
        ws, bs = _weights(rw, layers, 0.1, 0.0)
        backward = False
    elif index == 1:
        m, B = 64, 16
        samples = []
        for b in range(B):
            nsteps = 6 * int(rc.integers(1000 // 6, 3000 // 6 + 1))
            samples.append(bridge_walk(rc, nsteps, m))
        coords = _to_coords(samples, rc)
        layers = _stack([32, 64, 96, 128])
        ws, bs = _weights(rw, layers, _he, 0.1)
        backward = True
    elif index == 2:
        m, B = 128, 32
        samples = []
        for b in range(B):
            semi = rc.uniform(0.2, 0.45, size=3) * m
            power = 2 if rc.random() < 0.5 else 4
            samples.append(shell_sites(rc, m, semi, (m / 2.0,) * 3, power))
        coords = _to_coords(samples, rc)
        layers = _stack([32, 64, 96, 128, 160])
        ws, bs = _weights(rw, layers, _he, 0.1)
        backward = True
    elif index == 3:
        m, B = 512, 1
        target = int(round(1_000_000 * scale))
        keys = np.zeros(0, np.int64)
        nshell = 0
        while len(keys) < target:
            semi = rc.uniform(0.05, 0.2, size=3) * m
            power = 2 if rc.random() < 0.5 else 4
            reach = float(max(semi)) * (math.sqrt(3.0) if power > 2 else 1.0) + 2.0
            centre = rc.uniform(reach, m - reach, size=3)
            s = shell_sites(rc, m, semi, centre, power)
            k = (s[:, 2] * m + s[:, 1]) * m + s[:, 0]
            new = np.setdiff1d(k, keys)
            need = target - len(keys)
            if len(new) > need:
                new = np.sort(rc.choice(new, size=need, replace=False))
            keys = np.union1d(keys, new)
            nshell += 1
        notes["shells"] = nshell
        site = np.stack([keys % m, (keys // m) % m, keys // (m * m)], axis=1)
        coords = _to_coords([site], rc)
        layers = [LayerSpec("conv", 3, 1, 64, 64, False)]
        ws, bs = _weights(rw, layers, 1.0 / math.sqrt(27 * 64), 0.0)
        backward = True
    elif index == 4:
        m, B = 256, 8
        samples = []
        for b in range(B):
            nb = int(rc.integers(8, 33))
            ns = int(rc.integers(3, 7))
            nb = max(1, int(round(nb * scale)))
            ns = max(1, int(round(ns * scale)))
            parts = [bridge_walk(rc, 1998, m, centred=False) for _ in range(nb)]
            for _ in range(ns):
                semi = rc.uniform(0.2, 0.4, size=3) * m
                centre = rc.uniform(0.4, 0.6, size=3) * m
                power = 2 if rc.random() < 0.5 else 4
                parts.append(shell_sites(rc, m, semi, centre, power))
            samples.append(np.concatenate(parts, axis=0))
        coords = _to_coords(samples, rc)
        layers = [LayerSpec("conv", 3, 1, 1, 64, True)] + _stack([96, 128, 160, 192, 224, 256], 64)
        ws, bs = _weights(rw, layers, _he, 0.1)
        backward = True
    else:
        raise ValueError(f"no workload {index}")
    cin = layers[0].cin
    rf = stream_rng(seed, _S_FEATS)
    if index == 3:
        feats = rf.standard_normal((len(coords), cin)).astype(np.float32)
    else:
        feats = np.ones((len(coords), cin), np.float32)
    return ConfigInput(index=index, name=CONFIGS[index], seed=seed, grid=(B, m, m, m),
                       coords=coords, features=feats, g0=np.zeros(cin, np.float32),
                       layers=layers, weights=ws, biases=bs, backward=backward, notes=notes)


def make_dy(seed: int, rows: int, channels: int, stream: int = _S_DY) -> np.ndarray:
    """Output gradient U[-1, 1] float32[rows][channels]."""
    r = stream_rng(seed, stream)
    return r.uniform(-1.0, 1.0, size=(int(rows), int(channels))).astype(np.float32)


def make_dg(seed: int, channels: int, stream: int = _S_DG) -> np.ndarray:
    """Ground-state gradient U[-1, 1] float32[channels] (tests only: the loss
    of the workloads is on active rows, so their top-level dg is zero)."""
    r = stream_rng(seed, stream)
    return r.uniform(-1.0, 1.0, size=int(channels)).astype(np.float32)
