"""Throughput of the sparse-convolution hot path on one MI355X.

Workload: 1,000,000 active sites sampled from the union of seeded random
surface shells in a 512^3 grid, one 3x3x3 stride-1 sparse convolution with
Cin = Cout = 64, fp32, features N(0, 1), weights N(0, 1/sqrt(27*64)), output
gradients U[-1, 1].  One step = rulebook build (input map, active output set,
per-offset pair lists) + forward + input gradient + weight/bias/ground-state
gradients, with all inputs already resident in device memory.

Printed (one JSON line): effective GFLOP/s counting active pairs only
(3 contractions of 2*P*Cin*Cout flops per step), rulebook Msites/s and its
HBM fraction, per-phase times, the fraction of the fp32 MFMA peak of each
contraction (the input and weight gradients also timed alone) and of the
step's forward and backward together, the roofline of the dominant kernel
(the forward dense-block contraction, timed with HIP events on its stream),
max-pooling phases on the
convolution's output, and the CPU oracle timed on a bounded sample of the
same workload.

    python bench.py [--gpus 1] [--steps 10] [--warmup 3] [--no-cpu]

With --network it instead times whole-network inference of the paper's
networks (the nC2-MP3/2 object-recognition networks at scales 20/40/80 on the
cubic and the tetrahedral lattice; SquareNet and TriangLeNet on 32 x 32
images) and prints one JSON line per network.
"""
from __future__ import annotations

import argparse
import statistics
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

MFMA_FP32_PEAK_TFLOPS = 157.3
HBM_PEAK_GBS = 8000.0


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=10)
    p.add_argument("--warmup", type=int, default=3)
    p.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    p.add_argument("--cpu-sites", type=int, default=60000,
                   help="input sites of the bounded CPU-oracle sample")
    p.add_argument("--network", action="store_true",
                   help="instead: whole-network inference throughput of the paper's "
                        "networks (3D object recognition on the cubic and tetrahedral "
                        "lattices; 2D SquareNet / TriangLeNet), one JSON line each")
    p.add_argument("--batch", type=int, default=256,
                   help="samples per batch for --network (capped per network by the "
                        "rulebook's grid limit)")
    return p.parse_args()


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def measured_traffic():
    """HBM bytes per launch of the forward contraction from the committed
    rocprofv3 counter summary (FETCH_SIZE + WRITE_SIZE, each scaled by the
    same counter's reading for a device copy of known size), or None when the
    kernel source has changed since the counters were taken."""
    import hashlib
    path = os.path.join(ROOT, "profiles", "dense_fwd_1M_traffic.txt")
    src = os.path.join(ROOT, "paper_1505_02890_amd", "csrc", "conv.hip")
    if not os.path.exists(path):
        return None
    kv = {}
    for line in open(path):
        if line.startswith("#") or ":" not in line:
            continue
        k, v = line.split(":", 1)
        kv[k.strip()] = v.strip()
    sha = hashlib.sha256(open(src, "rb").read()).hexdigest()
    if kv.get("conv_hip_sha256") != sha:
        return None
    return float(kv["traffic_bytes"])


def cpu_baseline(cfg, n_sites: int):
    """The oracle (single-threaded, fp64, naive loops) on the sites of the
    workload inside a sub-box holding about n_sites sites: rulebook + forward
    + backward, reported in the same unit as the GPU value."""
    import oracle
    from gen import make_dy

    c = cfg.coords
    m = cfg.grid[1]
    # grow a centred cube until it holds enough sites
    centre = np.median(c[:, 1:4], axis=0)
    lo_h, hi_h = 1, m
    while lo_h < hi_h:
        h = (lo_h + hi_h) // 2
        sel = np.all(np.abs(c[:, 1:4] - centre) <= h, axis=1)
        if sel.sum() >= n_sites:
            hi_h = h
        else:
            lo_h = h + 1
    sel = np.all(np.abs(c[:, 1:4] - centre) <= lo_h, axis=1)
    coords = c[sel]
    x = cfg.features[sel]
    W = cfg.weights[0]
    L = cfg.layers[0]
    t0 = time.perf_counter()
    rb = oracle.Rulebook(coords, cfg.grid, L.f, L.s)
    t1 = time.perf_counter()
    y, g = oracle.conv_fwd(rb, x, cfg.g0, W, cfg.biases[0])
    t2 = time.perf_counter()
    dy = make_dy(cfg.seed + 1000, rb.a_out, L.cout)
    oracle.conv_bwd(rb, x, cfg.g0, W, cfg.biases[0], dy, None)
    t3 = time.perf_counter()
    flops = 3 * 2.0 * rb.n_pairs * L.cin * L.cout
    return {
        "value": round(flops / (t3 - t0) / 1e9, 4),
        "unit": "GFLOP/s",
        "cores": 1,
        "kind": "oracle",
        "sample": (f"{len(coords)} of the {len(c)} input sites (those in a centred "
                   f"cube of half-width {lo_h}), a_out={rb.a_out}, pairs={rb.n_pairs}; "
                   f"rulebook {t1 - t0:.2f}s, forward {t2 - t1:.2f}s, backward {t3 - t2:.2f}s"),
        "rulebook_msites_per_s": round(len(coords) / (t1 - t0) / 1e6, 4),
    }


def _time_net(net, cd, xd, batch_n, reps, warmup):
    import torch

    for _ in range(warmup):
        net.forward(cd, xd, batch_n)
    torch.cuda.synchronize()
    times = []
    for _ in range(reps):
        t0 = time.perf_counter()
        out, oc, rec = net.forward(cd, xd, batch_n)
        torch.cuda.synchronize()
        times.append(time.perf_counter() - t0)
    return float(np.median(times)), out, rec


def network_bench(batch: int, reps: int, warmup: int) -> None:
    """Inference throughput of the paper's networks, each batch timed end to
    end (every rulebook build, convolution and pooling, inputs resident in
    HBM; median over `reps`), random He-scaled weights:
      - the nC2-MP3/2 object-recognition networks of section 2 on the cubic
        and the tetrahedral lattice: each sample one seeded shell (ellipsoid
        or rounded-box superquadric, random rotation, semi-axes
        scale/2 * U(0.6, 1.0)) centred in the input grid, features 1.0;
      - SquareNet and TriangLeNet (the 2D comparison of section 2) on the
        square and the triangular lattice: each sample a 32 x 32 three-channel
        image (seeded N(0, 1) pixels) in the size-189 input grid, on the
        triangular lattice as its affine image (a rhombus)."""
    import torch

    from gen import image_patch_sites, shell_sites, stream_rng, tetra_shell_sites
    from paper_1505_02890_amd.network import PLANAR, SparseNet, input_size, macs

    # the paper's figures for these networks (GTX 780), context only
    paper = {"cubic": {20: (36, 1190), 40: (126, 794), 80: (406, 310)},
             "tetrahedral": {20: (9, 1133), 40: (35, 675), 80: (143, 286)},
             "square": {32: (41, None)}, "triangular": {32: (30, None)}}
    nets = [(lat, sc, lv) for lat in ("cubic", "tetrahedral")
            for sc, lv in ((20, 4), (40, 5), (80, 6))]
    nets += [("square", 32, 5), ("triangular", 32, 5)]
    for lattice, scale, levels in nets:
        planar = lattice in PLANAR
        convs = 2 if planar else 1
        m = input_size(levels, convs)
        # the rulebook's occupancy bitmap holds at most 2^26 words per grid
        # (the largest grid is the first convolution's output, m + 1 per axis)
        words = (m + 1) * (1 if planar else m + 1) * ((m + 1 + 31) // 32)
        batch_n = min(batch, (1 << 26) // words)
        rows = []
        for b in range(batch_n):
            rng = stream_rng(150502890 + scale, b)
            if planar:
                sh = image_patch_sites(lattice, m, scale, scale)
            else:
                semi = [0.5 * scale * float(rng.uniform(0.6, 1.0)) for _ in range(3)]
                power = (2, 4)[int(rng.integers(2))]
                if lattice == "cubic":
                    sh = shell_sites(rng, m, semi, [m / 2.0] * 3, power)
                else:
                    sh = tetra_shell_sites(rng, m, semi, power)
            rows.append(np.concatenate([np.full((len(sh), 1), b, np.int64), sh], axis=1))
        c = np.ascontiguousarray(np.concatenate(rows).astype(np.int32))
        cd = torch.from_numpy(c).cuda()
        if planar:
            x = stream_rng(150502890 + scale, 1 << 20).standard_normal((len(c), 3))
            xd = torch.from_numpy(x.astype(np.float32)).cuda()
            net = SparseNet(levels, classes=10, seed=scale, lattice=lattice, convs=2, cin=3)
            name, data = ("SquareNet" if lattice == "square" else "TriangLeNet"), \
                "synthetic (seeded 32x32 three-channel images)"
        else:
            xd = torch.ones((len(c), 1), dtype=torch.float32, device="cuda")
            net = SparseNet(levels, seed=scale, lattice=lattice)
            name, data = f"nC2-MP3/2 {lattice} network", "synthetic (seeded shells)"
        t, out, rec = _time_net(net, cd, xd, batch_n, reps, warmup)
        ops, tps = paper[lattice][scale]
        print(json.dumps({
            "metric": f"sparse CNN inference throughput ({name})",
            "value": round(batch_n / t, 1), "unit": "tests/s", "higher_is_better": True,
            "lattice": lattice, "scale": scale, "levels": levels, "input_grid": m,
            "batch": batch_n, "active_input_sites_per_sample": round(len(c) / batch_n, 1),
            "macs_per_sample_millions": round(macs(rec) / batch_n / 1e6, 2),
            "ms_per_batch": round(t * 1e3, 3), "final_sites": int(out.shape[0]),
            "paper_gtx780": {"million_operations": ops, "tests_per_s": tps,
                             "note": "context only"},
            "dtype": "f32", "data": data,
        }), flush=True)


def main():
    args = parse()
    if args.gpus != 1:
        print(json.dumps({"error": "this build runs on one GPU only; --gpus must be 1"}))
        sys.exit(2)
    if args.network:
        network_bench(args.batch, max(args.steps, 5), args.warmup)
        return
    import torch

    import paper_1505_02890_amd as scn
    from gen import make_config, make_dy

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    log("generating the 1M-site workload")
    cfg = make_config(3)
    L = cfg.layers[0]
    Cin, Cout = L.cin, L.cout
    d = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)  # noqa: E731
    coords, x, g0 = d(cfg.coords), d(cfg.features), d(cfg.g0)
    W, b = d(cfg.weights[0]), d(cfg.biases[0])

    rb = scn.build_rulebook(coords, cfg.grid, L.f, L.s)
    a_in, a_out, P = rb.a_in, rb.a_out, rb.n_pairs
    dy = d(make_dy(cfg.seed, a_out, Cout))
    ws = scn.conv_bwd_workspace(rb, Cin, Cout, False)
    del rb
    log(f"a_in={a_in} a_out={a_out} pairs={P}")

    stream = torch.cuda.current_stream()
    ev = lambda: torch.cuda.Event(enable_timing=True)  # noqa: E731
    phases = ("rulebook", "fwd", "bwd")

    def step(rec):
        e = [ev() for _ in range(4)]
        e[0].record(stream)
        r = scn.build_rulebook(coords, cfg.grid, L.f, L.s)
        e[1].record(stream)
        y, g = scn.conv_fwd(r, x, g0, W, b)
        e[2].record(stream)
        scn.conv_bwd(r, x, g0, W, None, None, dy, None, ws=ws)
        e[3].record(stream)
        if rec is not None:
            rec.append(e)
        return r, y, g

    log(f"warmup {args.warmup}")
    for _ in range(args.warmup):
        step(None)
    torch.cuda.synchronize()
    log(f"timing {args.steps} steps")
    recs = []
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step(recs)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ph = {p: [] for p in phases}
    for e in recs:
        for i, p in enumerate(phases):
            ph[p].append(e[i].elapsed_time(e[i + 1]))
    med = {p: float(np.median(v)) for p, v in ph.items()}
    ms_per_step = wall * 1e3 / args.steps
    flop_pass = 2.0 * P * Cin * Cout
    value = 3 * flop_pass / (ms_per_step / 1e3) / 1e9

    # dominant kernel: the forward contraction (dense blocks of mask-sorted
    # output rows: gather -> MFMA -> one store per row)
    fwd_ms = med["fwd"]
    achieved = flop_pass / (fwd_ms / 1e3) / 1e12
    log(f"ms/step={ms_per_step:.3f} phases(ms)={ {k: round(v, 4) for k, v in med.items()} }")

    # the two backward contractions timed on their own (outside the timed
    # steps): input gradient alone, weight gradient alone; median of 10
    r, y, g = step(None)

    def time_need(need):
        for _ in range(2):
            scn.conv_bwd(r, x, g0, W, None, None, dy, None, need=need, ws=ws)
        ts = []
        for _ in range(10):
            pe = [ev(), ev()]
            pe[0].record(stream)
            scn.conv_bwd(r, x, g0, W, None, None, dy, None, need=need, ws=ws)
            pe[1].record(stream)
            torch.cuda.synchronize()
            ts.append(pe[0].elapsed_time(pe[1]))
        return statistics.median(ts)

    dx_ms, dw_ms = time_need(("dx",)), time_need(("dW",))
    # the GEMM phase of a step: its forward and its backward call (one call
    # computes dx, dW, dbias and dg_in; the column sums of dy are counted once)
    gemm_ms = med["fwd"] + med["bwd"]

    # max-pooling on the convolution output: 2x2x2 stride 2 (windows partition
    # the inputs) and 3x3x3 stride 2 (overlapping windows), median of 5 runs
    C = Cout

    def time_pool(f, s):
        prb = scn.build_rulebook(r.out_coords(), r.out_grid, f, s)
        for _ in range(2):
            yp, gp, am = scn.maxpool_fwd(prb, y, g)
            scn.maxpool_bwd(prb, am, yp)
        fw, bw = [], []
        for _ in range(5):
            pe = [ev() for _ in range(3)]
            pe[0].record(stream)
            yp, gp, am = scn.maxpool_fwd(prb, y, g)
            pe[1].record(stream)
            scn.maxpool_bwd(prb, am, yp)
            pe[2].record(stream)
            torch.cuda.synchronize()
            fw.append(pe[0].elapsed_time(pe[1]))
            bw.append(pe[1].elapsed_time(pe[2]))
        fms, bms = statistics.median(fw), statistics.median(bw)
        fwd_bytes = 4.0 * prb.a_in * C + 8.0 * prb.n_pairs + 5.0 * prb.a_out * C
        bwd_bytes = 5.0 * prb.a_out * C + 4.0 * prb.a_in * C + 8.0 * prb.n_pairs
        return {
            "filter": f, "stride": s, "a_in": prb.a_in, "a_out": prb.a_out,
            "pairs": prb.n_pairs, "channels": C,
            "fwd_ms": round(fms, 4), "bwd_ms": round(bms, 4),
            "fwd_alg_gbs": round(fwd_bytes / (fms / 1e3) / 1e9, 1),
            "bwd_alg_gbs": round(bwd_bytes / (bms / 1e3) / 1e9, 1),
            "fwd_hbm_frac": round(fwd_bytes / (fms / 1e3) / 1e9 / HBM_PEAK_GBS, 3),
            "bwd_hbm_frac": round(bwd_bytes / (bms / 1e3) / 1e9 / HBM_PEAK_GBS, 3),
        }

    pool22 = time_pool(2, 2)
    pool32 = time_pool(3, 2)

    # a plain device copy of known size (calibrates the HBM byte counters)
    cal = torch.full((64 << 20,), 1.0, dtype=torch.float32, device=dev)
    cal2 = torch.empty_like(cal)
    cal2.copy_(cal)
    torch.cuda.synchronize()

    rb_bytes = 16.0 * a_in + 16.0 * a_out + 8.0 * P
    result = {
        "metric": "sparse-conv effective GFLOP/s (active sites only) + rulebook Msites/s, 1 GPU",
        "value": round(value, 2),
        "unit": "GFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic (seeded surface shells)",
        "config": {
            "workload": "1M active sites (surface shells, 512^3 grid), one 3x3x3 stride-1 sparse "
                        "conv 64->64; step = rulebook + forward + input grad + weight grad",
            "a_in": a_in, "a_out": a_out, "pairs": P, "cin": Cin, "cout": Cout,
        },
        "rulebook_msites_per_s": round(a_in / (med["rulebook"] / 1e3) / 1e6, 2),
        "phases_ms": {k: round(v, 4) for k, v in med.items()},
        "phase_gflops": {
            "fwd": round(flop_pass / (med["fwd"] / 1e3) / 1e9, 1),
            "bwd_dx_dw": round(2 * flop_pass / (med["bwd"] / 1e3) / 1e9, 1),
            "dx_alone": round(flop_pass / (dx_ms / 1e3) / 1e9, 1),
            "dw_alone": round(flop_pass / (dw_ms / 1e3) / 1e9, 1),
        },
        # fraction of the fp32 MFMA peak per contraction (the two backward
        # ones timed alone), and over the step's forward and backward calls
        "mfma_frac": {
            "fwd": round(flop_pass / (fwd_ms / 1e3) / 1e12 / MFMA_FP32_PEAK_TFLOPS, 4),
            "dx": round(flop_pass / (dx_ms / 1e3) / 1e12 / MFMA_FP32_PEAK_TFLOPS, 4),
            "dw": round(flop_pass / (dw_ms / 1e3) / 1e12 / MFMA_FP32_PEAK_TFLOPS, 4),
            "gemm_phase": round(3 * flop_pass / (gemm_ms / 1e3) / 1e12 / MFMA_FP32_PEAK_TFLOPS, 4),
        },
        "rulebook_alg_gbs": round(rb_bytes / (med["rulebook"] / 1e3) / 1e9, 1),
        "rulebook_hbm_frac": round(rb_bytes / (med["rulebook"] / 1e3) / 1e9 / HBM_PEAK_GBS, 3),
        "roofline": {
            "kernel": "dense_fwd_kernel (forward)",
            "bound": "mfma",
            "achieved": round(achieved, 3),
            "peak": MFMA_FP32_PEAK_TFLOPS,
            "unit": "TFLOP/s",
            "frac": round(achieved / MFMA_FP32_PEAK_TFLOPS, 4),
            "traffic": measured_traffic(),
        },
        "pool": pool22,
        "pool_overlapping": pool32,
        "cpu_baseline": None,
    }
    if not args.no_cpu:
        log("timing the CPU oracle on a bounded sample")
        result["cpu_baseline"] = cpu_baseline(cfg, args.cpu_sites)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
