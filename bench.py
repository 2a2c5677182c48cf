"""Throughput of the sparse-convolution hot path on one MI355X.

Workload: 1,000,000 active sites sampled from the union of seeded random
surface shells in a 512^3 grid, one 3x3x3 stride-1 sparse convolution with
Cin = Cout = 64, fp32, features N(0, 1), weights N(0, 1/sqrt(27*64)), output
gradients U[-1, 1].  One step = rulebook build (input map, active output set,
per-offset pair lists) + forward + input gradient + weight/bias/ground-state
gradients, with all inputs already resident in device memory.

Printed (one JSON line): effective GFLOP/s counting active pairs only
(3 contractions of 2*P*Cin*Cout flops per step), rulebook Msites/s and its
HBM fraction, per-phase times, each contraction kernel's own duration
(HIP events the library records around it on its stream, scn_set_kernel_timer)
and its fraction of the fp32 MFMA peak, the roofline of the dominant kernel
(the forward dense-block contraction), measured ceilings (a streaming copy,
a register-only MFMA loop), max-pooling phases on the convolution's output,
whole-step timings of the other four workloads (the trefoil forward; the
curve, surface and deep stacks forward + backward), and the CPU oracle timed
on bounded samples of the same workload on one core and on all cores.

    python bench.py [--gpus 1] [--steps 10] [--warmup 3] [--no-cpu] [--no-configs]

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
                   help="input sites of the bounded one-core CPU-oracle sample")
    p.add_argument("--cpu-sites-each", type=int, default=25000,
                   help="input sites per process of the all-core CPU-oracle sample")
    p.add_argument("--no-configs", action="store_true",
                   help="skip the whole-step timings of the other four workloads")
    p.add_argument("--network", action="store_true",
                   help="instead: whole-network inference throughput of the paper's "
                        "networks (3D object recognition on the cubic and tetrahedral "
                        "lattices; 2D SquareNet / TriangLeNet), one JSON line each")
    p.add_argument("--batch", type=int, default=256,
                   help="samples per batch for --network (the tetrahedral networks are "
                        "capped by the occupancy bitmaps' grid limit)")
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


def _centred_sample(c, m, n_sites, centre):
    """Sites in the smallest cube around `centre` that holds >= n_sites."""
    lo_h, hi_h = 1, m
    while lo_h < hi_h:
        h = (lo_h + hi_h) // 2
        if np.all(np.abs(c[:, 1:4] - centre) <= h, axis=1).sum() >= n_sites:
            hi_h = h
        else:
            lo_h = h + 1
    return np.all(np.abs(c[:, 1:4] - centre) <= lo_h, axis=1), lo_h


def _oracle_step(coords, grid, x, g0, W, bias, f, s, dy_seed):
    """The oracle (fp64, naive loops) on one sample: rulebook, forward,
    backward.  Returns (flops, rulebook s, forward s, backward s, a_out, P)."""
    import oracle
    from gen import make_dy

    t0 = time.perf_counter()
    rb = oracle.Rulebook(coords, grid, f, s)
    t1 = time.perf_counter()
    oracle.conv_fwd(rb, x, g0, W, bias)
    t2 = time.perf_counter()
    dy = make_dy(dy_seed, rb.a_out, W.shape[2])
    oracle.conv_bwd(rb, x, g0, W, bias, dy, None)
    t3 = time.perf_counter()
    flops = 3 * 2.0 * rb.n_pairs * W.shape[1] * W.shape[2]
    return flops, t1 - t0, t2 - t1, t3 - t2, rb.a_out, rb.n_pairs


def _cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(cfg, n_sites: int, n_sites_each: int):
    """The oracle, as it stands, on the host: (1) one thread on the sites of
    the workload inside a centred cube of about n_sites sites; (2) every
    available core (one process each, at most 16) on disjoint cubes of about
    n_sites_each sites around different centres, timed together.  Each runs
    rulebook + forward + backward; the value is in the GPU's unit."""
    import multiprocessing
    from concurrent.futures import ProcessPoolExecutor

    c = cfg.coords
    m = cfg.grid[1]
    L = cfg.layers[0]
    args = (cfg.g0, cfg.weights[0], cfg.biases[0], L.f, L.s)
    sel, h = _centred_sample(c, m, n_sites, np.median(c[:, 1:4], axis=0))
    fl, trb, tf, tb, a_out, P = _oracle_step(c[sel], cfg.grid, cfg.features[sel], *args[:3],
                                             L.f, L.s, cfg.seed + 1000)
    single = {
        "value": round(fl / (trb + tf + tb) / 1e9, 4), "unit": "GFLOP/s", "cores": 1,
        "kind": "oracle",
        "sample": (f"{int(sel.sum())} of the {len(c)} input sites (a centred cube of half-width "
                   f"{h}), a_out={a_out}, pairs={P}; rulebook {trb:.2f}s, forward {tf:.2f}s, "
                   f"backward {tb:.2f}s"),
        "rulebook_msites_per_s": round(int(sel.sum()) / trb / 1e6, 4),
    }
    # all cores: disjoint cubes around well-separated active sites
    try:
        ncpu = len(os.sched_getaffinity(0))
    except AttributeError:
        ncpu = os.cpu_count() or 1
    workers = max(1, min(16, ncpu))
    rng = np.random.default_rng(cfg.seed + 77)
    jobs, taken = [], np.zeros(len(c), bool)
    for i in rng.permutation(len(c)):
        if len(jobs) == workers:
            break
        if taken[i]:
            continue
        s_i, _ = _centred_sample(c, m, n_sites_each, c[i, 1:4])
        if np.any(s_i & taken):
            continue
        taken |= s_i
        jobs.append((np.ascontiguousarray(c[s_i]), tuple(cfg.grid),
                     np.ascontiguousarray(cfg.features[s_i])) + args + (cfg.seed + 2000 + i,))
    ctx = multiprocessing.get_context("spawn")
    with ProcessPoolExecutor(max_workers=len(jobs), mp_context=ctx) as ex:
        # the workers' start-up (interpreter, numpy, oracle library) stays
        # outside the timed region
        list(ex.map(_warm, range(len(jobs))))
        t0 = time.perf_counter()
        res = list(ex.map(_oracle_job, jobs))
        wall = time.perf_counter() - t0
    tot = sum(r[0] for r in res)
    sites = sum(len(j[0]) for j in jobs)
    allcore = {
        "value": round(tot / wall / 1e9, 4), "unit": "GFLOP/s", "cores": len(jobs),
        "kind": "oracle",
        "sample": (f"{len(jobs)} disjoint cubes of about {n_sites_each} input sites each "
                   f"({sites} sites, {sum(r[5] for r in res)} pairs), one process per core, "
                   f"wall {wall:.2f}s"),
        "host_cpus": ncpu, "cpu_model": _cpu_model(),
    }
    return single, allcore


def _warm(_):
    import oracle  # noqa: F401
    return 0


def _oracle_job(job):
    coords, grid, x, g0, W, bias, f, s, seed = job
    return _oracle_step(coords, grid, x, g0, W, bias, f, s, seed)


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
        # the occupancy bitmaps hold at most 2^26 32-bit words per grid (the
        # largest grid is the input, m per axis, rows padded to 32 sites);
        # past them the cubic lattice builds with sorted keys and hash
        # tables, the other lattices cap the batch
        words = m * (1 if planar else m) * ((m + 31) // 32)
        batch_n = batch if lattice == "cubic" else min(batch, (1 << 26) // words)
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


class KernelTimer:
    """Pairs of HIP events the library records around its contraction
    kernels (scn_set_kernel_timer): forward, input gradient, weight
    gradient, one set per timed step."""

    def __init__(self, scn, stream, n):
        import torch

        self.scn, self.stream = scn, stream
        self.sets = []
        for _ in range(n):
            ev = [torch.cuda.Event(enable_timing=True) for _ in range(6)]
            for e in ev:
                e.record(stream)  # creates the HIP event
            self.sets.append(ev)
        torch.cuda.synchronize()
        self.i = 0

    def arm(self):
        import ctypes

        ev = self.sets[self.i]
        self.i += 1
        arr = (ctypes.c_void_p * 6)(*[e.cuda_event for e in ev])
        self.scn.lib().scn_set_kernel_timer(arr)

    def disarm(self):
        self.scn.lib().scn_set_kernel_timer(None)

    def ms(self, which):
        j = {"fwd": 0, "dx": 2, "dw": 4}[which]
        return [ev[j].elapsed_time(ev[j + 1]) for ev in self.sets[:self.i]]


def ceilings(scn, dev):
    """Measured ceilings: a 1 GiB streaming copy (HBM) and a register-only
    loop of fp32 MFMA products (matrix cores), median of 10 each."""
    import ctypes

    import torch

    stream = torch.cuda.current_stream()
    nbytes = 1 << 30
    a = torch.ones(nbytes // 4, dtype=torch.float32, device=dev)
    b = torch.empty_like(a)
    L = scn.lib()
    sp = ctypes.c_void_p(stream.cuda_stream)

    def timed(fn, reps=10):
        fn()
        torch.cuda.synchronize()
        ts = []
        for _ in range(reps):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            fn()
            e1.record(stream)
            torch.cuda.synchronize()
            ts.append(e0.elapsed_time(e1))
        return statistics.median(ts)

    def copy():
        assert L.scn_ceiling_copy(ctypes.c_void_p(a.data_ptr()), ctypes.c_void_p(b.data_ptr()),
                                  nbytes, sp) == 0

    copy_ms = timed(copy)
    assert torch.equal(a[:1024], b[:1024])
    out = torch.empty(4 * 2048, dtype=torch.float32, device=dev)
    flops = ctypes.c_double()

    def mfma():
        assert L.scn_ceiling_mfma_f32(ctypes.c_void_p(out.data_ptr()), 2048, 4096,
                                      ctypes.byref(flops), sp) == 0

    mfma_ms = timed(mfma)
    copy_gbs = 2.0 * nbytes / (copy_ms / 1e3) / 1e9
    mfma_tf = flops.value / (mfma_ms / 1e3) / 1e12
    return {
        "hbm_copy": {"bytes_moved": 2 * nbytes, "ms": round(copy_ms, 4),
                     "gbs": round(copy_gbs, 1), "frac_of_peak": round(copy_gbs / HBM_PEAK_GBS, 4)},
        "mfma_f32_loop": {"flops": flops.value, "ms": round(mfma_ms, 4),
                          "tflops": round(mfma_tf, 2),
                          "frac_of_peak": round(mfma_tf / MFMA_FP32_PEAK_TFLOPS, 4)},
    }


CONFIG_WORKLOADS = {
    0: "one knotted closed lattice walk (400 steps) in 32^3; C2 1->16 -> MP2/2; forward",
    1: "16 closed lattice walks in 64^3; 4 x [C2 + ReLU -> MP2/2], ch 32/64/96/128; fwd + bwd",
    2: "32 voxelised superquadric shells in 128^3; 5 x [C2 + ReLU -> MP2/2], ch 32..160; "
       "fwd + bwd",
    4: "8 samples of curve bundles + shells in 256^3; C3 1->64 + ReLU, 6 x [C2 + ReLU -> "
       "MP2/2], ch 96..256; fwd + bwd",
}


def config_bench(scn, index, reps, warmup):
    """Whole step of workload `index` (chain of rulebooks, forward and, for
    the trained stacks, backward from U[-1, 1] output gradients), inputs in
    HBM; median of `reps` steps."""
    import torch

    from gen import make_config, make_dy
    from paper_1505_02890_amd.stack import StackStep, conv_flops

    cfg = make_config(index)
    dev = torch.device("cuda:0")
    d = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)  # noqa: E731
    coords, x = d(cfg.coords), d(cfg.features)
    Ws = [None if w is None else d(w) for w in cfg.weights]
    Bs = [None if b is None else d(b) for b in cfg.biases]
    st = StackStep(cfg.layers, Ws, Bs)
    dy_cache = {}

    def dy_top(rows, ch):
        if (rows, ch) not in dy_cache:
            dy_cache[(rows, ch)] = d(make_dy(cfg.seed, rows, ch))
        return dy_cache[(rows, ch)]

    stream = torch.cuda.current_stream()
    names = ("rulebook", "fwd", "bwd") if cfg.backward else ("rulebook", "fwd")

    def one():
        ev = {"start": torch.cuda.Event(enable_timing=True)}
        ev["start"].record(stream)

        def mark(name):
            ev[name] = torch.cuda.Event(enable_timing=True)
            ev[name].record(stream)

        out, rec, _ = st.run(coords, cfg.grid, x, dy_top if cfg.backward else None, mark)
        return ev, rec

    for _ in range(warmup):
        one()
    torch.cuda.synchronize()
    walls, evs = [], []
    rec = None
    for _ in range(reps):
        t0 = time.perf_counter()
        ev, rec = one()
        torch.cuda.synchronize()
        walls.append((time.perf_counter() - t0) * 1e3)
        evs.append(ev)
    ph = {}
    prev = "start"
    for nme in names:
        ph[nme] = statistics.median(e[prev].elapsed_time(e[nme]) for e in evs)
        prev = nme
    ms = statistics.median(walls)
    flops = conv_flops(rec, cfg.backward)
    a_in = len(cfg.coords)
    return {
        "workload": CONFIG_WORKLOADS[index],
        "a_in": a_in, "layers": len(cfg.layers),
        "step": "fwd + bwd" if cfg.backward else "fwd",
        "ms_per_step": round(ms, 4),
        "phases_ms": {k: round(v, 4) for k, v in ph.items()},
        "gflop_per_step": round(flops / 1e9, 3),
        "gflops": round(flops / (ms / 1e3) / 1e9, 1),
        "rulebook_chain_msites_per_s": round(a_in / (ph["rulebook"] / 1e3) / 1e6, 2),
        "first_layer": {"a_out": rec[0][2], "pairs": rec[0][3]},
        "reps": reps,
    }


def main():
    args = parse()
    if args.gpus != 1:
        print(json.dumps({"error": "this build runs on one GPU only; --gpus must be 1"}))
        sys.exit(2)
    if args.network:
        network_bench(args.batch, max(args.steps, 5), args.warmup)
        return
    from gen import make_config, make_dy

    log("generating the 1M-site workload")
    cfg = make_config(3)
    cpu = None
    if not args.no_cpu:
        # the CPU legs run before the GPU is touched (their worker processes
        # start from a process without a GPU context)
        log("timing the CPU oracle on bounded samples (one core, then all cores)")
        cpu = cpu_baseline(cfg, args.cpu_sites, args.cpu_sites_each)

    import torch

    import paper_1505_02890_amd as scn

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    L = cfg.layers[0]
    Cin, Cout = L.cin, L.cout
    d = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)  # noqa: E731
    coords, x, g0 = d(cfg.coords), d(cfg.features), d(cfg.g0)
    W, b = d(cfg.weights[0]), d(cfg.biases[0])

    rb = scn.build_rulebook(coords, cfg.grid, L.f, L.s)
    a_in, a_out, P = rb.a_in, rb.a_out, rb.n_pairs
    dense_view = rb.dense_view
    dy = d(make_dy(cfg.seed, a_out, Cout))
    ws = scn.conv_bwd_workspace(rb, Cin, Cout, False)
    del rb
    log(f"a_in={a_in} a_out={a_out} pairs={P}")

    stream = torch.cuda.current_stream()
    ev = lambda: torch.cuda.Event(enable_timing=True)  # noqa: E731
    phases = ("rulebook", "fwd", "bwd")
    timer = KernelTimer(scn, stream, args.steps)

    def step(rec):
        e = [ev() for _ in range(4)]
        if rec is not None:
            timer.arm()
        e[0].record(stream)
        r = scn.build_rulebook(coords, cfg.grid, L.f, L.s)
        e[1].record(stream)
        y, g = scn.conv_fwd(r, x, g0, W, b)
        e[2].record(stream)
        scn.conv_bwd(r, x, g0, W, None, None, dy, None, ws=ws)
        e[3].record(stream)
        if rec is not None:
            timer.disarm()
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
    # the contraction kernels' own durations over the timed steps (HIP events
    # the library records on the stream the kernels run on)
    kern = {k: float(np.mean(timer.ms(k))) for k in ("fwd", "dx", "dw")}
    log(f"ms/step={ms_per_step:.3f} phases(ms)={ {k: round(v, 4) for k, v in med.items()} } "
        f"kernels(ms)={ {k: round(v, 4) for k, v in kern.items()} }")

    # dominant kernel: the forward contraction (dense blocks of mask-sorted
    # output rows: gather -> MFMA -> one store per row)
    achieved = flop_pass / (kern["fwd"] / 1e3) / 1e12

    # max-pooling on the convolution output: 2x2x2 stride 2 (windows partition
    # the inputs) and 3x3x3 stride 2 (overlapping windows): mean of 10 back-to-back
    # calls, median of 3 such runs
    r, y, g = step(None)
    C = Cout

    def time_pool(f, s):
        prb = scn.build_rulebook(r.out_coords(), r.out_grid, f, s)
        for _ in range(2):
            yp, gp, am = scn.maxpool_fwd(prb, y, g)
            scn.maxpool_bwd(prb, am, yp)
        # back-to-back calls, so the host's per-call work overlaps the device's
        reps = 10
        fw, bw = [], []
        for _ in range(3):
            pe = [ev() for _ in range(3)]
            pe[0].record(stream)
            for _ in range(reps):
                yp, gp, am = scn.maxpool_fwd(prb, y, g)
            pe[1].record(stream)
            for _ in range(reps):
                scn.maxpool_bwd(prb, am, yp)
            pe[2].record(stream)
            torch.cuda.synchronize()
            fw.append(pe[0].elapsed_time(pe[1]) / reps)
            bw.append(pe[1].elapsed_time(pe[2]) / reps)
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
    del r, y, g, ws, dy
    torch.cuda.empty_cache()

    # the same rulebook from the keyed builder (sorted keys and open-
    # addressing hash tables: the path of grids past the bitmaps and of
    # sites of other dimensions), median of 5 builds, each one call
    log("keyed rulebook")
    kt = []
    for i in range(7):
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        rk = scn.build_rulebook_nd(coords, cfg.grid, L.f, L.s)
        torch.cuda.synchronize()
        if i >= 2:
            kt.append(time.perf_counter() - t0)
        assert (rk.a_out, rk.n_pairs) == (a_out, P)
        del rk
    keyed_ms = statistics.median(kt) * 1e3

    log("ceilings")
    ceil = ceilings(scn, dev)
    # a plain device copy of known size (calibrates the HBM byte counters)
    cal = torch.full((64 << 20,), 1.0, dtype=torch.float32, device=dev)
    cal2 = torch.empty_like(cal)
    import ctypes
    assert scn.lib().scn_ceiling_copy(ctypes.c_void_p(cal.data_ptr()),
                                      ctypes.c_void_p(cal2.data_ptr()), 256 << 20,
                                      ctypes.c_void_p(stream.cuda_stream)) == 0
    torch.cuda.synchronize()
    del cal, cal2

    configs = {}
    if not args.no_configs:
        for i, reps in ((0, 20), (1, 10), (2, 10), (4, 5)):
            log(f"workload {i}")
            configs[str(i)] = config_bench(scn, i, reps, 2)
            torch.cuda.empty_cache()

    rb_bytes = 16.0 * a_in + 16.0 * a_out + 8.0 * P
    mf = lambda ms: round(flop_pass / (ms / 1e3) / 1e12 / MFMA_FP32_PEAK_TFLOPS, 4)  # noqa: E731
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
            "dense_forward_view": dense_view,
        },
        "rulebook_msites_per_s": round(a_in / (med["rulebook"] / 1e3) / 1e6, 2),
        "rulebook_keyed": {"ms": round(keyed_ms, 4),
                           "msites_per_s": round(a_in / (keyed_ms / 1e3) / 1e6, 2)},
        "phases_ms": {k: round(v, 4) for k, v in med.items()},
        "kernels_ms": {k: round(v, 4) for k, v in kern.items()},
        "phase_gflops": {
            "fwd": round(flop_pass / (med["fwd"] / 1e3) / 1e9, 1),
            "bwd_dx_dw": round(2 * flop_pass / (med["bwd"] / 1e3) / 1e9, 1),
        },
        # fraction of the fp32 MFMA peak of each contraction kernel (its own
        # duration), of the forward call, and of the step's forward and
        # backward calls together (the GEMM phase)
        "mfma_frac": {
            "fwd_kernel": mf(kern["fwd"]), "dx_kernel": mf(kern["dx"]),
            "dw_kernel": mf(kern["dw"]), "fwd_call": mf(med["fwd"]),
            "gemm_phase": round(3 * flop_pass / ((med["fwd"] + med["bwd"]) / 1e3) / 1e12
                                / MFMA_FP32_PEAK_TFLOPS, 4),
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
            "frac_of_measured_ceiling": round(achieved / ceil["mfma_f32_loop"]["tflops"], 4),
        },
        "ceilings": ceil,
        "pool": pool22,
        "pool_overlapping": pool32,
        "configs": configs,
        "cpu_baseline": cpu[0] if cpu else None,
        "cpu_baseline_all_cores": cpu[1] if cpu else None,
    }
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
