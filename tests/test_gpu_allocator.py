"""The caller's allocator hooks (scn_set_allocator): every device allocation
the library makes for itself goes through them and comes back through them,
and the results equal those with the library's own pool."""
from __future__ import annotations

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from gen import random_sites, stream_rng  # noqa: E402

from helpers import dev, host  # noqa: E402

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def scn():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_1505_02890_amd as m
    m.lib()  # raises if the HIP library is missing
    yield m
    m.set_allocator()


def _run(scn, coords, grid, x, g_in, W, b, dy):
    rb = scn.build_rulebook(dev(coords), grid, 3, 1)
    y, g = scn.conv_fwd(rb, dev(x), dev(g_in), dev(W), dev(b), relu=True)
    out = scn.conv_bwd(rb, dev(x), dev(g_in), dev(W), y, g, dev(dy), None, relu=True)
    nxt = scn.next_rulebook(rb, 2, 2)
    yp, gp, am = scn.maxpool_fwd(nxt, y, g)
    res = [host(t).copy() for t in (rb.out_coords(), y, g, out["dx"], out["dW"], out["dbias"],
                                   out["dg_in"], yp, am)]
    rb.close()
    nxt.close()
    torch.cuda.synchronize()
    return res


def test_caller_allocator_round_trip(scn):
    rng = stream_rng(95, 0)
    grid = (2, 24, 20, 18)
    coords = random_sites(rng, 2, grid[1:], 2500)
    x = rng.standard_normal((len(coords), 32)).astype(np.float32)
    g_in = (rng.standard_normal(32) * 0.3).astype(np.float32)
    W = (rng.standard_normal((27, 32, 48)) / np.sqrt(27 * 32)).astype(np.float32)
    b = (rng.standard_normal(48) * 0.1).astype(np.float32)
    a_out = scn.build_rulebook(dev(coords), grid, 3, 1).a_out
    dy = rng.uniform(-1, 1, (a_out, 48)).astype(np.float32)

    scn.set_allocator()
    want = _run(scn, coords, grid, x, g_in, W, b, dy)

    live, counts = {}, {"alloc": 0, "free": 0}

    def alloc(nbytes, stream):
        p = torch.cuda.caching_allocator_alloc(int(nbytes), stream=int(stream))
        live[p] = nbytes
        counts["alloc"] += 1
        return p

    def free(ptr, stream):
        assert ptr in live, "freed a block the hook did not allocate"
        del live[ptr]
        counts["free"] += 1
        torch.cuda.caching_allocator_delete(ptr)

    scn.set_allocator(alloc, free)
    try:
        got = _run(scn, coords, grid, x, g_in, W, b, dy)
    finally:
        scn.set_allocator()
    assert counts["alloc"] > 0 and counts["alloc"] == counts["free"] and not live
    for a, w in zip(got, want):
        assert np.array_equal(a, w)

    # a rulebook built under the hooks is freed through them after the reset
    scn.set_allocator(alloc, free)
    rb = scn.build_rulebook(dev(coords), grid, 2, 1)
    scn.set_allocator()
    assert live
    rb.close()
    torch.cuda.synchronize()
    assert not live and counts["alloc"] == counts["free"]


def test_allocator_failure_is_nomem(scn):
    coords = random_sites(stream_rng(96, 0), 1, (10, 10, 10), 100)
    scn.set_allocator(lambda n, s: 0, lambda p, s: None)
    try:
        with pytest.raises(scn.ScnError) as e:
            scn.build_rulebook(dev(coords), (1, 10, 10, 10), 2, 1)
        assert e.value.status == "nomem"
    finally:
        scn.set_allocator()
    scn.build_rulebook(dev(coords), (1, 10, 10, 10), 2, 1)   # the default pool again
