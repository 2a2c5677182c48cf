"""One training step (forward, then backward) of a stack of sparse
convolutions and max-poolings on the C ABI: the layer sequences of the
synthetic workloads (a 2x2x2 convolution + ReLU and a 2x2x2 stride-2
max-pooling per level, optionally after a 3x3x3 convolution).

The step builds every layer's rulebook first, in one chain call (section 1.3:
the active output sites of a layer are the next layer's active input sites,
and rulebooks depend on sites only), then runs the forward layer by layer,
keeping each layer's input, output, ground states and argmax, then the
backward from an output gradient on the top layer's active rows (the loss is
on active rows only, so the top ground-state gradient is zero).  The input
layer's own gradients (dx, dg_in) are not computed: nothing consumes them.

Every step runs in the library's kernels; this module only sequences the
calls and keeps the layer state.
"""
from __future__ import annotations

from typing import Callable, Optional, Sequence

import torch

from . import _lib as scn


def conv_flops(records, backward: bool) -> float:
    """Flops of the convolutions' contractions over active pairs only:
    2*P*Cin*Cout for the forward, and for the backward the same for the
    weight gradient and (all but the first layer) the input gradient."""
    tot = 0.0
    for i, (kind, a_in, a_out, P, ci, co) in enumerate(records):
        if kind != "conv":
            continue
        passes = 1 + ((2 if i > 0 else 1) if backward else 0)
        tot += passes * 2.0 * P * ci * co
    return tot


class StackStep:
    """layers: objects with kind ("conv" / "pool"), f, s, cin, cout, relu;
    weights / biases: device tensors per conv layer (None for pools)."""

    def __init__(self, layers: Sequence, weights: Sequence, biases: Sequence):
        self.layers = list(layers)
        self.weights = list(weights)
        self.biases = list(biases)

    def run(self, coords: torch.Tensor, grid, x: torch.Tensor,
            dy_top: Optional[Callable[[int, int], torch.Tensor]] = None,
            marks: Optional[Callable[[str], None]] = None):
        """coords int32 [n][4] and x [n][cin] on the device.  dy_top(rows,
        channels) gives the output gradient of the top layer (no backward if
        None).  marks(name) is called after the rulebooks ("rulebook"), the
        forward ("fwd") and the backward ("bwd") are queued.  Returns
        (top output, per-layer records, weight gradients)."""
        mark = marks or (lambda name: None)
        rbs = scn.build_chain(coords, grid, [(L.f, L.s) for L in self.layers])
        mark("rulebook")
        g = torch.zeros(x.shape[1], dtype=torch.float32, device=x.device)
        saved, records = [], []
        for L, W, b, rb in zip(self.layers, self.weights, self.biases, rbs):
            if L.kind == "conv":
                y, go = scn.conv_fwd(rb, x, g, W, b, relu=L.relu)
                saved.append((x, g, y, go, None))
                records.append(("conv", rb.a_in, rb.a_out, rb.n_pairs, L.cin, L.cout))
            else:
                y, go, am = scn.maxpool_fwd(rb, x, g)
                saved.append((x, g, y, go, am))
                records.append(("pool", rb.a_in, rb.a_out, rb.n_pairs, x.shape[1], x.shape[1]))
            x, g = y, go
        mark("fwd")
        grads = {}
        if dy_top is not None:
            dy, dg = dy_top(x.shape[0], x.shape[1]), None
            for i in range(len(self.layers) - 1, -1, -1):
                L, rb = self.layers[i], rbs[i]
                xi, gi, y, go, am = saved[i]
                if L.kind == "conv":
                    need = ("dx", "dg_in", "dW", "dbias") if i > 0 else ("dW", "dbias")
                    out = scn.conv_bwd(rb, xi, gi, self.weights[i], y, go, dy, dg, relu=L.relu,
                                       need=need)
                    grads[i] = (out["dW"], out["dbias"])
                    dy, dg = out.get("dx"), out.get("dg_in")
                else:
                    dy, dg = scn.maxpool_bwd(rb, am, dy, dg)
            mark("bwd")
        return x, records, grads
