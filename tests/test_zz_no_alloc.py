"""scn_conv_fwd_noalloc (the forward for callers that cannot allocate)
against scn_conv_fwd through the C ABI: two calls in a row, the second with a
smaller input, each bit-identical to the allocating entry point and within
the per-site tolerance of the oracle; the library's allocator hook sees no
allocation during the no-alloc calls; shapes past the static scratch are
refused before any device work."""
from __future__ import annotations

import numpy as np
import pytest

torch = pytest.importorskip("torch")

import oracle  # noqa: E402
from gen import random_sites, stream_rng  # noqa: E402

from helpers import assert_site, dev, host  # noqa: E402

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def scn():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_1505_02890_amd as m
    m.lib()  # raises if the HIP library is missing
    return m


CASES = [
    # (f, B, dims, n, Cin, Cout, relu): the first large, the second smaller
    (3, 2, (30, 28, 26), 6000, 64, 64, True),
    (2, 1, (12, 10, 9), 300, 17, 24, False),
]


def _inputs(i, case):
    f, B, dims, n, Cin, Cout, relu = case
    rng = stream_rng(880, i)
    coords = random_sites(rng, B, dims, n)
    K = f ** 3
    x = rng.standard_normal((len(coords), Cin)).astype(np.float32)
    g_in = (rng.standard_normal(Cin) * 0.5).astype(np.float32)
    W = (rng.standard_normal((K, Cin, Cout)) / np.sqrt(K * Cin)).astype(np.float32)
    bias = (rng.standard_normal(Cout) * 0.1).astype(np.float32)
    return coords, (B,) + tuple(dims), x, g_in, W, bias


def test_noalloc_matches_conv_fwd_twice(scn):
    counted = []

    def alloc(nbytes, stream):
        counted.append(int(nbytes))
        return torch.cuda.caching_allocator_alloc(int(nbytes), stream=int(stream))

    def free(ptr, stream):
        torch.cuda.caching_allocator_delete(int(ptr))

    for i, case in enumerate(CASES):
        f, B, dims, n, Cin, Cout, relu = case
        coords, grid, x, g_in, W, bias = _inputs(i, case)
        g = scn.build_rulebook(dev(coords), grid, f, 1)
        xd, gd, Wd, bd = dev(x), dev(g_in), dev(W), dev(bias)
        y_a, go_a = scn.conv_fwd(g, xd, gd, Wd, bd, relu=relu)
        # outputs allocated before the call: the library itself allocates nothing
        y_n = torch.full_like(y_a, float("nan"))
        go_n = torch.full_like(go_a, float("nan"))
        torch.cuda.synchronize()
        scn.set_allocator(alloc, free)
        try:
            scn.conv_fwd(g, xd, gd, Wd, bd, relu=relu, y=y_n, g_out=go_n, noalloc=True)
            torch.cuda.synchronize()
        finally:
            scn.set_allocator()
        assert counted == [], f"call {i}: the library allocated {counted}"
        assert torch.equal(y_n, y_a) and torch.equal(go_n, go_a), f"call {i}"
        o = oracle.Rulebook(coords, grid, f, 1)
        y_ref, go_ref = oracle.conv_fwd(o, x, g_in, W, bias, relu=relu)
        assert_site(f"noalloc y (call {i})", host(y_n), y_ref)
        assert_site(f"noalloc g_out (call {i})", host(go_n), go_ref)


def test_noalloc_refuses_shapes_past_its_scratch(scn):
    cap = int(scn.lib().scn_conv_fwd_noalloc_max_bytes())
    assert cap == 8 << 20
    coords = random_sites(stream_rng(881, 0), 1, (8, 8, 8), 40)
    g = scn.build_rulebook(dev(coords), (1, 8, 8, 8), 3, 1)
    Cin, Cout = 256, 320  # 27 * 320 * 256 floats of packed weights: past 8 MiB
    x = torch.zeros((len(coords), Cin), dtype=torch.float32, device="cuda")
    with pytest.raises(scn.ScnError) as e:
        scn.conv_fwd(g, x, torch.zeros(Cin, device="cuda"),
                     torch.zeros((27, Cin, Cout), device="cuda"), noalloc=True)
    assert e.value.status == "workspace"
