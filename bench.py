"""Benchmark: edges/s of the sparse DNN forward pass on one MI355X.

Default workload (the very wide network, n = 2^20, L = 8, batch 8192, the largest configuration): one step
is one forward pass of all L layers from the CSR input batch Y_0 to the CSR output Y_L through
sdnn_forward_csr; value = batch * sum_k nnz(W_k) / step time.  Inputs are resident in HBM before timing
starts.  The line also carries the roofline of the dominant kernel (per-launch GPU time from the library's
profiling events over the timed steps), its achieved HBM bandwidth (compulsory bytes and, when the committed
rocprofv3 counters match the kernel's sources, counter bytes), the per-kernel time split, the density sweep
with the sparse-versus-dense crossover (the paper's Sec. V comparison) as extra keys, and the CPU oracle on
a bounded sample as a baseline.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--config 1..5] [--no-sweep]
"""

from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import re
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "edges/sec (batch × nnz(W_k) × L / time) at 1 MI355X; achieved HBM GB/s"
HBM_PEAK_GBS = 8000.0
FP64_VECTOR_TFLOPS = 78.6  # MI355X fp64 vector peak: the sparse kernels multiply-add in fp64
FP64_MATRIX_TFLOPS = 78.6  # MI355X fp64 matrix-core peak (dense-W arm)
FP32_MATRIX_TFLOPS = 157.3  # MI355X fp32 matrix-core peak (fp32 dense-W arm)
DENSE_BOTH = 3  # SDNN_ARENA_DENSE_F64 | SDNN_ARENA_DENSE_F32
PROFILES = os.path.join(ROOT, "profiles")


def log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


def _code_only(text: str) -> str:
    """Source text without comments and with whitespace runs collapsed, so that an edit of comments alone does
    not mark counters taken on the same code as stale."""
    text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
    text = re.sub(r"//[^\n]*", " ", text)
    return " ".join(text.split())


def _src_hash(*names):
    h = hashlib.sha256()
    for nm in names:
        with open(os.path.join(ROOT, "paper_1708_02937_amd", "csrc", nm), encoding="utf-8") as f:
            h.update(_code_only(f.read()).encode())
    return h.hexdigest()[:16]


def _pmc_traffic(kernel_tag: str, src_names):
    """HBM bytes per launch from the committed rocprofv3 --pmc summary, or None when the kernel source
    changed since the counters were taken (the summary records a hash of the sources it measured)."""
    path = os.path.join(PROFILES, f"{kernel_tag}_pmc.txt")
    if not os.path.exists(path):
        return None
    rec = {}
    with open(path) as f:
        for line in f:
            if ":" in line and not line.startswith((" ", "#")):
                k, v = line.split(":", 1)
                rec[k.strip()] = v.strip()
    if rec.get("source_hash") != _src_hash(*src_names):
        return None
    return int(rec["hbm_bytes_per_launch"]) if "hbm_bytes_per_launch" in rec else None


# ----------------------------------------------------------------------------------- timing helpers


def _events(torch):
    return torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)


def time_steps(torch, fn, steps: int):
    """Time exactly `steps` calls of fn() back to back on the current stream, with one HIP event between
    consecutive calls; returns (mean, median, min) milliseconds per call.  The mean is the span from the
    first event to the last over `steps`."""
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
    torch.cuda.synchronize()
    ev[0].record()
    for i in range(steps):
        fn()
        ev[i + 1].record()
    torch.cuda.synchronize()
    per = sorted(ev[i].elapsed_time(ev[i + 1]) for i in range(steps))
    mid = steps // 2
    median = per[mid] if steps % 2 else 0.5 * (per[mid - 1] + per[mid])
    return ev[0].elapsed_time(ev[-1]) / steps, median, per[0]


def time_calls(torch, fn, reps: int) -> float:
    """Average milliseconds per call of fn(), timed with HIP events on the current stream."""
    a, b = _events(torch)
    torch.cuda.synchronize()
    a.record()
    for _ in range(reps):
        fn()
    b.record()
    torch.cuda.synchronize()
    return a.elapsed_time(b) / reps


def kernel_split(records):
    """Per kernel name: launches, total and average ms, from profiling-log records (layer, name, ms)."""
    out = {}
    for layer, name, ms in records:
        r = out.setdefault(name, {"launches": 0, "total_ms": 0.0, "layers": []})
        r["launches"] += 1
        r["total_ms"] += ms
        r["layers"].append((layer, ms))
    for r in out.values():
        r["avg_ms"] = r["total_ms"] / r["launches"]
    return out


SPMM_KERNELS = ("spmm_fanin_kernel", "spmm_narrow_kernel", "spmm_slots_kernel", "spmm_tiled_kernel", "spmm_blocked_kernel")


def kernel_sources(kernel):
    """The library sources a kernel's counters depend on (their hash marks a counter summary as current)."""
    if kernel.startswith("spmm_blocked"):
        return ["blocked.hip", "common.h"]
    if kernel.startswith("gemm"):
        return ["gemm.hip", "common.h"]
    if kernel.startswith("spgemm"):
        return ["spgemm.hip", "common.h"]
    return ["spmm.hip", "common.h"]


def kernel_roofline(name, rec, p, trace=None):
    """Roofline of one profiled kernel over its launches: algorithmic bytes (flops) per launch, averaged over
    the launches, divided by the average launch time.  trace: (nnz per Y_k, products per layer) for the
    sparse-Y product."""
    launches = rec["layers"]
    byt = flops = 0.0
    for layer, _ in launches:
        nnz = p.layers[layer].nnz if layer >= 0 else 0
        if name in SPMM_KERNELS:
            b, f = spmm_algorithmic(p.n, p.batch, nnz)
        elif name == "gemm_dense_layer_kernel":
            b, f = 8 * p.n * p.n + 8 * p.n * p.batch, 2.0 * p.batch * p.n * p.n
        elif name == "spgemm_layer" and trace is not None:
            ny, prods = trace
            b = 8 * ny[layer] + 8 * ny[layer + 1] + 8 * p.batch + 8 * nnz + 8 * (p.n + 1) + 4 * p.n
            f = 2.0 * prods[layer]
        else:
            return None
        byt += b
        flops += f
    byt /= len(launches)
    flops /= len(launches)
    t_s = rec["avg_ms"] / 1e3
    if name == "gemm_dense_layer_kernel":
        roof = {"bound": "mfma", "achieved": round(flops / t_s / 1e12, 3), "peak": FP64_MATRIX_TFLOPS,
                "unit": "TFLOP/s"}
    elif flops / byt > FP64_VECTOR_TFLOPS * 1e12 / (HBM_PEAK_GBS * 1e9):
        roof = {"bound": "alu", "achieved": round(flops / t_s / 1e12, 3), "peak": FP64_VECTOR_TFLOPS,
                "unit": "TFLOP/s"}
    else:
        roof = {"bound": "hbm", "achieved": round(byt / t_s / 1e9, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s"}
    roof["frac"] = round(roof["achieved"] / roof["peak"], 4)
    roof.update({"kernel": name, "launches": len(launches), "avg_launch_ms": round(rec["avg_ms"], 5),
                 "algorithmic_bytes_per_launch": int(byt), "algorithmic_flops_per_launch": flops})
    return roof


def hbm_fields(roof, traffic):
    """Achieved HBM bandwidth of the dominant kernel: compulsory bytes per launch / average launch time, and
    counter bytes (rocprofv3 FETCH_SIZE + WRITE_SIZE, scaled) / the same time when the counters are current."""
    t_s = roof["avg_launch_ms"] / 1e3
    eff = roof["algorithmic_bytes_per_launch"] / t_s / 1e9
    out = {"kernel": roof["kernel"], "effective": round(eff, 1), "effective_frac": round(eff / HBM_PEAK_GBS, 4),
           "counter": None, "counter_frac": None}
    if traffic:
        cnt = traffic / t_s / 1e9
        out.update({"counter": round(cnt, 1), "counter_frac": round(cnt / HBM_PEAK_GBS, 4),
                    "counter_bytes_per_launch": traffic})
    return out


# ----------------------------------------------------------------------------------- the sweep


def spmm_algorithmic(n, batch, nnz):
    """Algorithmic bytes and flops of one dense-Y CSR layer launch (one layer, all samples).

    bytes: read Y^T (4 n batch) + fan-in lists (8 nnz) + list pointers (8 (n+1)) + bias (4 n),
    write Y_{k+1}^T (4 n batch).  flops: 2 per product, batch * nnz products.
    """
    return 8 * n * batch + 8 * nnz + 8 * (n + 1) + 4 * n, 2.0 * batch * nnz


def run_sweep(args, torch, sd):
    from workloads import make_config

    densities = [float(x) for x in args.densities.split(",")]
    nets, ys, outs, probs = [], [], [], []
    for d in densities:
        t0 = time.time()
        p = make_config(2, d)
        net = sd.net_from_problem(p, dense=0 if args.no_dense else DENSE_BOTH)
        nets.append(net)
        probs.append(p)
        ys.append(torch.from_numpy(p.y0_dense).cuda())
        outs.append(torch.empty_like(ys[-1]))
        net.workspace(p.batch, 0)
        log(f"density {d}: nnz/layer {p.layers[0].nnz}, set-up {time.time() - t0:.1f}s")

    def step():
        for net, y, o in zip(nets, ys, outs):
            net.forward_dense(y, out=o)

    for _ in range(args.warmup):
        step()
    for net in nets:
        net.set_profiling(True)
    t_wall = time.perf_counter()
    ms_step, ms_med, ms_min = time_steps(torch, step, args.steps)
    t_wall = time.perf_counter() - t_wall
    splits = []
    for net in nets:
        net.set_profiling(False)
        splits.append(kernel_split(net.read_profile()))
    edges = sum(p.edges() for p in probs)
    value = edges / (ms_step / 1e3)
    log(f"step {ms_step:.3f} ms (wall {1e3 * t_wall / args.steps:.3f} ms), {value:.4g} edges/s")

    # per-density forward time, and the average launch time of the layer kernel over the timed steps
    sweep = {}
    reps = max(3, args.steps)
    for d, net, y, o, p, sp in zip(densities, nets, ys, outs, probs, splits):
        t_full = time_calls(torch, lambda: net.forward_dense(y, out=o), reps)
        kname = next(k for k in sp if k != "transpose_kernel")
        sweep[f"{d:g}"] = {"sparse_ms": round(t_full, 4), "sparse_edges_per_s": p.edges() / (t_full / 1e3),
                           "layer_kernel": kname, "layer_launch_ms": round(sp[kname]["avg_ms"], 5),
                           "nnz_per_layer": int(p.layers[0].nnz)}

    # dense-W arms at every density: fp64 matrix cores (the sparse paths' arithmetic) and fp32 matrix cores (an
    # sgemm's arithmetic, the paper's comparison)
    if not args.no_dense:
        for d, net, y, o, p in zip(densities, nets, ys, outs, probs):
            for key, arm in (("dense_ms", sd.SDNN_ARM_DENSE), ("dense32_ms", sd.SDNN_ARM_DENSE_F32)):
                net.forward_dense(y, out=o, arm=arm)
                t_dense = time_calls(torch, lambda: net.forward_dense(y, out=o, arm=arm), max(2, reps // 2))
                sweep[f"{d:g}"][key] = round(t_dense, 4)
            torch.cuda.synchronize()

    def find_crossover(key="dense_ms"):
        pts = sorted((d, v["sparse_ms"], v.get(key)) for d, v in
                     ((float(k), v) for k, v in sweep.items()) if v.get(key))
        for (d0, s0, q0), (d1, s1, q1) in zip(pts, pts[1:]):
            r0, r1 = math.log(s0 / q0), math.log(s1 / q1)
            if r0 <= 0 <= r1 and r1 != r0:  # sparse faster at d0, slower at d1
                t = -r0 / (r1 - r0)
                return math.exp(math.log(d0) + t * (math.log(d1) - math.log(d0)))
        return None

    crossover = find_crossover()
    if (crossover is None or find_crossover("dense32_ms") is None) and not args.no_dense and max(densities) < 1.0:
        # the sparse arm wins at every sweep density: bracket the crossover with denser weights (same recipe,
        # same L); these points inform the crossover only and are not part of the step
        for d in (0.75, 1.0):
            if d <= max(densities):
                continue
            q = make_config(2, d)
            net = sd.net_from_problem(q, dense=DENSE_BOTH)
            y = torch.from_numpy(q.y0_dense).cuda()
            o = torch.empty_like(y)
            net.workspace(q.batch, 0)
            t_sp = time_calls(torch, lambda: net.forward_dense(y, out=o), max(2, reps // 2))
            t_dn = time_calls(torch, lambda: net.forward_dense(y, out=o, arm=sd.SDNN_ARM_DENSE), max(2, reps // 2))
            t_d32 = time_calls(torch, lambda: net.forward_dense(y, out=o, arm=sd.SDNN_ARM_DENSE_F32), max(2, reps // 2))
            net.free()
            sweep[f"{d:g}"] = {"sparse_ms": round(t_sp, 4), "dense_ms": round(t_dn, 4), "dense32_ms": round(t_d32, 4),
                               "nnz_per_layer": int(q.layers[0].nnz), "bracket": True}
            log(f"bracket density {d}: sparse {t_sp:.3f} ms, dense fp64 {t_dn:.3f} ms, fp32 {t_d32:.3f} ms")
            del q
            crossover = find_crossover()
            if crossover is not None and find_crossover("dense32_ms") is not None:
                break
    crossover32 = find_crossover("dense32_ms")
    # dominant kernel: the layer kernel with the largest share of the step
    best = None
    for d, sp in zip(densities, splits):
        for k, v in sp.items():
            if k != "transpose_kernel" and (best is None or v["total_ms"] > best[2]["total_ms"]):
                best = (d, k, v)
    dom, kernel, rec = best
    p = probs[densities.index(dom)]
    roof = kernel_roofline(kernel, rec, p)
    roof["traffic"] = _pmc_traffic(f"{kernel}_d{dom:g}", kernel_sources(kernel))
    roof["density"] = dom
    hbm = hbm_fields(roof, roof["traffic"])
    for net in nets:
        net.free()
    cfg = {"workload": "density-sweep n=4096 L=16 batch=1024 d=" + "/".join(f"{d:g}" for d in densities)
                       + " (CSR sparse-W path; fp32 storage, fp64 accumulate)",
           "n": 4096, "L": 16, "batch": 1024, "densities": densities}
    return dict(value=value, ms_step=ms_step, ms_median=ms_med, ms_min=ms_min, edges=edges, sweep=sweep,
                crossover=crossover, crossover32=crossover32, roofline=roof, hbm=hbm, config=cfg, probs=probs,
                densities=densities)


# oracle sample per workload (rows of the batch): all-core rate, and single-thread rate where the density-sweep
# and tiny-MLP workloads set one beside the paper's single-thread measurements
CPU_ROWS = {1: 64, 2: 1024, 3: 256, 4: 1024, 5: 16}
CPU_ROWS_SINGLE = {1: 64, 2: 8}


def _oracle_rate(probs, rows, threads, min_seconds):
    """Whole passes of the oracle over the first `rows` samples of every problem, all layers, until at least
    min_seconds of CPU work; returns (edges/s, seconds, passes)."""
    import oracle
    from workloads import csr_rows

    ys = [csr_rows(p.y0_as_csr(), np.arange(rows)) for p in probs]
    edges = 0
    t_total = 0.0
    passes = 0
    while passes == 0 or t_total < min_seconds:
        for y, p in zip(ys, probs):
            t0 = time.perf_counter()
            oracle.forward(p.n, p.layers, p.ymax, y, threads=threads)
            t_total += time.perf_counter() - t0
            edges += rows * sum(l.nnz for l in p.layers)
        passes += 1
    return edges / t_total, t_total, passes


def cpu_baseline(args, probs, config):
    """Oracle on the host cores: the first R samples of the workload (of every density for the sweep), all
    L layers; whole passes repeated until at least 10 s of CPU work."""
    import oracle

    rows = min(args.cpu_rows or CPU_ROWS[config], probs[0].batch)
    threads = oracle.default_threads()
    where = " at each density" if len(probs) > 1 else ""
    rate, secs, passes = _oracle_rate(probs, rows, threads, 10.0)
    rec = {"value": rate, "unit": "edges/s", "cores": threads, "kind": "oracle",
           "sample": f"first {rows} of {probs[0].batch} samples{where}, all {probs[0].L} layers, "
                     f"{passes} passes ({secs:.1f} s of CPU work)", "seconds": round(secs, 2), "cpu": _cpu_model()}
    if config in CPU_ROWS_SINGLE:
        r1 = min(CPU_ROWS_SINGLE[config], probs[0].batch)
        rate1, secs1, passes1 = _oracle_rate(probs, r1, 1, 3.0)
        rec["single_thread"] = {"value": rate1, "unit": "edges/s", "cores": 1,
                                "sample": f"first {r1} samples{where}, all {probs[0].L} layers, {passes1} passes",
                                "seconds": round(secs1, 2)}
    return rec


def _cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


# ----------------------------------------------------------------------------------- other workloads


def _crossover(points):
    """Log-log interpolation of the x where t_sparse = t_dense, from sorted (x, t_sparse, t_dense);
    x grows as W gets sparser, so the sparse arm is slower before the crossover and faster after it."""
    for (x0, s0, q0), (x1, s1, q1) in zip(points, points[1:]):
        r0, r1 = math.log(s0 / q0), math.log(s1 / q1)
        if r0 >= 0 >= r1 and r1 != r0:
            t = r0 / (r0 - r1)
            return math.exp(math.log(x0) + t * (math.log(x1) - math.log(x0)))
    return None


def run_paper_grid(args, torch, sd):
    """The paper's own experiment (Sec. V.B-D) on one MI355X: one layer of m x m weights with inverse
    sparsity S (Bernoulli pattern, values U[-1,3)) applied to 64 dense samples, through the CSR arm and the
    dense-W arm.  Per-layer time = (T(L identical layers) - T(1 layer)) / (L - 1), so the entry and exit
    transposes cancel (the paper times one iteration of its layer loop); L = 17 below m = 8192, then 9, 5
    and 3 (the dense copies take m^2 x 12 bytes per layer), so that the GPU time, not the host's launch
    time, is what remains.  Also the analogues
    of the paper's scaling parameters (Fig. 7), each normalised to m = 4096: dense time per element,
    sparse/dense ratio at S = 1, sparse slope per nonzero between S = 1 and S = 4, and the saturation time
    per row at S = 262144."""
    from workloads import PAPER_GRID_INV_SPARSITY, PAPER_GRID_SIZES, paper_grid

    sizes = [int(x) for x in args.grid_sizes.split(",")] if args.grid_sizes else list(PAPER_GRID_SIZES)
    invs = [int(x) for x in args.grid_inv.split(",")] if args.grid_inv else list(PAPER_GRID_INV_SPARSITY)
    reps = max(3, args.steps)
    grid = {}
    for m in sizes:
        grid[m] = {}
        for S in invs:
            t0 = time.time()
            # enough identical layers that GPU time, not host launch time, dominates the difference, within the
            # memory the dense copies take (m^2 x 12 bytes per layer)
            L = 17 if m < 8192 else {8192: 9, 16384: 5}.get(m, 3)
            p = paper_grid(m, S, L=L)
            l0 = p.layers[0]
            net = sd.Net(m, L, nnz_per_layer=int(l0.nnz), dense=0 if args.no_dense else DENSE_BOTH)
            dev = [torch.from_numpy(a).cuda() for a in (l0.row_ptr, l0.col, l0.val, l0.bias)]
            del p.layers[:]
            for k in range(L):
                net.set_layer(k, *dev)  # every layer references the same device arrays
            y = torch.from_numpy(p.y0_dense).cuda()
            o = torch.empty_like(y)
            rec = {"nnz": int(l0.nnz)}
            arms = [("sparse", sd.SDNN_ARM_SPARSE)]
            if not args.no_dense:
                net.build_dense()
                arms += [("dense", sd.SDNN_ARM_DENSE), ("dense32", sd.SDNN_ARM_DENSE_F32)]
            for name, arm in arms:
                for k1 in (1, L):
                    net.forward_dense(y, k1=k1, arm=arm, out=o)
                tl = time_calls(torch, lambda: net.forward_dense(y, k1=L, arm=arm, out=o), reps)
                t1 = time_calls(torch, lambda: net.forward_dense(y, k1=1, arm=arm, out=o), reps)
                rec[f"{name}_ms"] = round(max(tl - t1, 0.0) / (L - 1), 5)
            grid[m][S] = rec
            net.free()
            del net, dev, y, o, l0, p
            torch.cuda.empty_cache()
            log(f"m {m} S {S}: nnz {rec['nnz']}, sparse {rec['sparse_ms']:.4f} ms, dense {rec.get('dense_ms')}, "
                f"{time.time() - t0:.1f}s")
    # scaling parameters, as in the paper's Fig. 7
    params = {}
    for m in sizes:
        g = grid[m]
        q = {}
        if 1 in g and "dense_ms" in g[1]:
            q["dense_per_element"] = g[1]["dense_ms"] / (m * m)
            q["sparse_over_dense_at_S1"] = g[1]["sparse_ms"] / g[1]["dense_ms"] if g[1]["dense_ms"] > 0 else None
        if 1 in g and 4 in g:
            q["sparse_slope_per_nnz"] = (g[1]["sparse_ms"] - g[4]["sparse_ms"]) / (0.75 * m * m)
        if 262144 in g:
            q["saturation_per_row"] = g[262144]["sparse_ms"] / m
        for key, dk in (("crossover_inv_sparsity", "dense_ms"), ("crossover_inv_sparsity_f32", "dense32_ms")):
            pts = [(S, v["sparse_ms"], v[dk]) for S, v in sorted(g.items()) if v.get(dk) and v["sparse_ms"] > 0]
            q[key] = _crossover(pts)
        params[m] = q
    if 4096 in params:
        ref = params[4096]
        for m in sizes:
            for key in ("dense_per_element", "sparse_over_dense_at_S1", "sparse_slope_per_nnz", "saturation_per_row"):
                if params[m].get(key) is not None and ref.get(key):
                    params[m][key + "_rel4096"] = params[m][key] / ref[key]
    return grid, params



def run_semiring(args, torch, sd):
    """Matrix multiply over each semiring of Sec. II (sdnn_mxm_dense) on the density-sweep shape
    (n = 4096, batch = 1024): time per call (two transposes included) and edges/s."""
    from workloads import make_config

    names = ["plus_times", "max_plus", "max_min", "min_max", "xor_and"]
    densities = [float(x) for x in args.densities.split(",")]
    reps = max(3, args.steps)
    out = {}
    for d in densities:
        p = make_config(2, d, L=1)
        net = sd.net_from_problem(p)
        y = torch.from_numpy(p.y0_dense).cuda()
        z = torch.empty_like(y)
        out[f"{d:g}"] = {}
        # a CSR batch of the same shape with 10% of its entries stored (the rest are the 0-element)
        yc = p.y0_dense.copy()
        yc[np.random.default_rng(11).random(yc.shape) >= 0.1] = 0.0
        from workloads import dense_to_csr
        crs = [torch.from_numpy(a).cuda() for a in dense_to_csr(yc)]
        for sr, name in enumerate(names):
            net.mxm(0, sr, y, out=z)
            ms = time_calls(torch, lambda: net.mxm(0, sr, y, out=z), reps)
            net.mxm_csr(0, sr, *crs)
            ms_csr = time_calls(torch, lambda: net.mxm_csr(0, sr, *crs), reps)
            out[f"{d:g}"][name] = {"ms": round(ms, 5), "edges_per_s": p.edges() / (ms / 1e3),
                                   "csr_10pct_ms": round(ms_csr, 5)}
            log(f"semiring {name} d {d}: {ms:.4f} ms dense input, {ms_csr:.4f} ms CSR input (10% stored)")
        net.free()
    return out



def layer_trace(torch, net, p, y):
    """nnz of Y_0 .. Y_L and the products of each layer (sum over the stored entries (r, i) of Y_k of the
    fan-out of neuron i in W_k), from the same forward run one layer at a time (not timed)."""
    rp, c, v = y
    nnz = [int(c.numel())]
    products = []
    for k, l in enumerate(p.layers):
        fanout = torch.from_numpy(np.diff(l.row_ptr)).cuda()
        products.append(int(fanout[c.long()].sum().item()) if c.numel() else 0)
        rp, c, v = (t.clone() for t in net.forward_csr(rp, c, v, k0=k, k1=k + 1))
        nnz.append(int(c.numel()))
    return nnz, products


PMC_TAGS = {1: "tiny-mlp", 3: "sparse-activation", 4: "deep-sparse", 5: "very-wide"}


def run_csr_config(args, torch, sd):
    """Configs 3-5 (CSR input through sdnn_forward_csr) and config 1 (dense batch), one forward per step.
    The library's profiling log is on during the timed steps (config 1: during an extra pass of the same
    steps, so the event records do not weigh on a 30 us forward)."""
    from workloads import make_config

    t0 = time.time()
    p = make_config(args.config)
    log(f"generated {p.name} in {time.time() - t0:.1f}s")
    t0 = time.time()
    net = sd.net_from_problem(p)
    if p.y0_csr is not None:
        y = tuple(torch.from_numpy(a).cuda() for a in p.y0_csr)
        fn = lambda: net.forward_csr(*y)
    else:
        y = torch.from_numpy(p.y0_dense).cuda()
        o = torch.empty_like(y)
        fn = lambda: net.forward_dense(y, out=o)
    fn()
    torch.cuda.synchronize()
    log(f"set-up and first forward {time.time() - t0:.1f}s")
    for _ in range(args.warmup):
        fn()
    profiled_inline = p.y0_csr is not None
    if profiled_inline:
        net.set_profiling(True)
    ms, ms_med, ms_min = time_steps(torch, fn, args.steps)
    if not profiled_inline:
        net.set_profiling(True)
        time_steps(torch, fn, args.steps)
    net.set_profiling(False)
    split = kernel_split(net.read_profile())
    log(f"step {ms:.3f} ms; " + ", ".join(f"{k} {v['launches']} x {v['avg_ms']:.4f} ms" for k, v in split.items()))
    extra = {}
    if p.y0_csr is None:
        # a dense batch: the same forward replayed from a HIP graph (launch-bound at small sizes)
        g = net.capture_forward_dense(y, o)
        for _ in range(args.warmup):
            g.replay()
        timed = time_steps(torch, g.replay, args.steps)
        # the graph holds the net's buffers: release it, with its work finished, before the net is freed
        torch.cuda.synchronize()
        del g
        extra = {"eager_ms_per_step": round(ms, 4), "graph_ms_per_step": round(timed[0], 4)}
        log(f"eager {ms:.4f} ms, graph replay {timed[0]:.4f} ms per forward")
        if timed[0] < ms:
            ms, ms_med, ms_min = timed
    trace = None
    if args.config in (3, 4) and not args.no_layer_trace:
        nnz, products = layer_trace(torch, net, p, y)
        trace = (nnz, products)
        extra.update({"nnz_trace": nnz, "products_per_layer": products,
                      "products_per_s": sum(products) / (ms / 1e3)})
        log(f"nnz trace {nnz[:4]} ..., {sum(products):.4g} products per forward")
    net.free()
    torch.cuda.synchronize()
    per_step = {k: round(v["total_ms"] / args.steps, 4) for k, v in split.items()}
    dom = max(split, key=lambda k: split[k]["total_ms"])
    roof = kernel_roofline(dom, split[dom], p, trace)
    hbm = None
    if roof is not None:
        roof["traffic"] = _pmc_traffic(f"{dom}_{PMC_TAGS.get(args.config, p.name)}", kernel_sources(dom)) \
            if dom in SPMM_KERNELS else None
        hbm = hbm_fields(roof, roof["traffic"])
    cfg = {"workload": f"{p.name} n={p.n} L={p.L} batch={p.batch}", "n": p.n, "L": p.L, "batch": p.batch,
           "nnz_per_layer": int(p.layers[0].nnz), **extra}
    return dict(value=p.edges() / (ms / 1e3), ms_step=ms, ms_median=ms_med, ms_min=ms_min, config=cfg,
                roofline=roof, hbm=hbm, kernel_ms_per_step=per_step, sweep=None, crossover=None, probs=[p])


# ----------------------------------------------------------------------------- profile summaries (no GPU)


def _short_name(kname):
    base = kname.replace("sdnn::(anonymous namespace)::", "").replace("sdnn::", "").replace("void ", "")
    return base.split("(")[0].strip()


def summarize_stats(csv_dir, title, command, out):
    """Markdown table of a rocprofv3 --kernel-trace --stats run (the *kernel_stats.csv it wrote)."""
    import csv
    import glob

    path = sorted(glob.glob(os.path.join(csv_dir, "**", "*kernel_stats.csv"), recursive=True))[0]
    rows = list(csv.DictReader(open(path)))
    lines = ["# rocprofv3 kernel statistics", "", "command (from the repository root on the MI355X box):", "",
             f"    {command}", "", title, "", "| kernel | calls | avg us | min us | max us | share % |",
             "|---|---|---|---|---|---|"]
    for r in rows:
        lines.append(f"| {_short_name(r['Name'])} | {r['Calls']} | {float(r['AverageNs']) / 1e3:.2f} | "
                     f"{float(r['MinNs']) / 1e3:.2f} | {float(r['MaxNs']) / 1e3:.2f} | {float(r['Percentage']):.2f} |")
    with open(out, "w") as f:
        f.write("\n".join(lines) + "\n")


def _pmc_avg(csv_dir, counter, kernel):
    import csv
    import glob

    path = sorted(glob.glob(os.path.join(csv_dir, "**", "*counter_collection.csv"), recursive=True))[0]
    vals = [float(r["Counter_Value"]) for r in csv.DictReader(open(path))
            if r["Counter_Name"] == counter and _short_name(r["Kernel_Name"]).startswith(kernel)]
    assert vals, f"no {counter} records for {kernel} in {path}"
    return sum(vals) / len(vals), len(vals)


def summarize_pmc(kernel, tag, dirs, copy_bytes, commands, out, src_names):
    """HBM traffic per launch of `kernel` from FETCH_SIZE / WRITE_SIZE runs, each scaled by what the same
    counter reads for a plain device copy of copy_bytes bytes (dirs: fetch, write, copy-fetch, copy-write)."""
    fetch, nf = _pmc_avg(dirs[0], "FETCH_SIZE", kernel)
    write, nw = _pmc_avg(dirs[1], "WRITE_SIZE", kernel)
    cfetch, _ = _pmc_avg(dirs[2], "FETCH_SIZE", "__amd_rocclr_copyBuffer")
    cwrite, _ = _pmc_avg(dirs[3], "WRITE_SIZE", "__amd_rocclr_copyBuffer")
    fs, ws = copy_bytes / 1024 / cfetch, copy_bytes / 1024 / cwrite
    hbm = int(round((fetch * fs + write * ws) * 1024))
    lines = [f"# rocprofv3 HBM traffic counters: {kernel}", "",
             f"FETCH_SIZE and WRITE_SIZE (KiB per dispatch), averaged over {nf} / {nw} dispatches of the kernel,",
             f"each scaled by what the same counter reads for a plain device copy of {copy_bytes} bytes",
             f"(rocclr copyBuffer: FETCH_SIZE {cfetch:.1f} KiB -> scale {fs:.3f}; WRITE_SIZE {cwrite:.1f} KiB -> "
             f"scale {ws:.3f}).", "", "commands (from the repository root on the MI355X box):", ""]
    lines += [f"    {c}" for c in commands]
    lines += ["", f"workload: {tag}", f"fetch_kib_per_dispatch: {fetch:.1f}", f"write_kib_per_dispatch: {write:.1f}",
              f"fetch_scale: {fs:.4f}", f"write_scale: {ws:.4f}", f"hbm_bytes_per_launch: {hbm}",
              f"source_hash: {_src_hash(*src_names)}"]
    with open(out, "w") as f:
        f.write("\n".join(lines) + "\n")


def summarize_counters(dirs, title, commands, out, longest=False):
    """Per kernel, the mean of every counter over its dispatches, from rocprofv3 --pmc runs (counter_collection
    CSVs under each of dirs; runs of the same command, merged by kernel name), with busy fractions against the
    dispatch's cycles (GRBM_GUI_ACTIVE, summed over the 8 XCDs): VALU issue (4 cycles per wave64 instruction
    on a 16-lane SIMD, 1024 SIMDs), MFMA busy (per SIMD) and TA / TD busy (per CU)."""
    import csv
    import glob
    from collections import defaultdict

    agg = defaultdict(lambda: defaultdict(list))
    for d in dirs:
        for path in glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True):
            rows = [r for r in csv.DictReader(open(path)) if not _short_name(r["Kernel_Name"]).startswith(("at::", "__amd"))]
            if longest:
                # only each kernel's longest dispatch of this run (e.g. the one layer that does the work)
                dur = {}
                for r in rows:
                    k = _short_name(r["Kernel_Name"])
                    t = int(r["End_Timestamp"]) - int(r["Start_Timestamp"])
                    if t > dur.get(k, (-1, None))[0]:
                        dur[k] = (t, r["Dispatch_Id"])
                rows = [r for r in rows if dur[_short_name(r["Kernel_Name"])][1] == r["Dispatch_Id"]]
            for r in rows:
                agg[_short_name(r["Kernel_Name"])][r["Counter_Name"]].append(float(r["Counter_Value"]))
    lines = [f"# rocprofv3 counters: {title}", "", "commands (from the repository root on the MI355X box):", ""]
    lines += [f"    {c}" for c in commands]
    lines += ["", "| kernel | counter | dispatches | mean per dispatch |", "|---|---|---|---|"]
    derived = []
    for k in sorted(agg):
        m = {c: sum(v) / len(v) for c, v in agg[k].items()}
        for c in sorted(m):
            lines.append(f"| {k} | {c} | {len(agg[k][c])} | {m[c]:.6g} |")
        cyc = m.get("GRBM_GUI_ACTIVE", 0) / 8  # GUI-active cycles are summed over the 8 XCDs
        if cyc <= 0:
            continue
        if "SQ_INSTS_VALU" in m:  # a wave64 VALU instruction occupies its 16-lane SIMD for 4 cycles
            derived.append(f"| {k} | VALU issue: SQ_INSTS_VALU x 4 / (1024 SIMDs x cycles) | "
                           f"{m['SQ_INSTS_VALU'] * 4 / (1024 * cyc):.3f} |")
        if m.get("SQ_VALU_MFMA_BUSY_CYCLES"):
            derived.append(f"| {k} | MFMA busy: SQ_VALU_MFMA_BUSY_CYCLES / (1024 SIMDs x cycles) | "
                           f"{m['SQ_VALU_MFMA_BUSY_CYCLES'] / (1024 * cyc):.3f} |")
        for c in ("TA_TA_BUSY_sum", "TD_TD_BUSY_sum"):
            if c in m:
                derived.append(f"| {k} | {c} / (256 CUs x cycles) | {m[c] / (256 * cyc):.3f} |")
        derived.append(f"| {k} | dispatch cycles (GRBM_GUI_ACTIVE / 8 XCDs) | {cyc:.4g} |")
    if derived:
        lines += ["", "derived (busy fractions; 1.0 = every unit busy for the whole dispatch):", "",
                  "| kernel | ratio | value |", "|---|---|---|"] + derived
    with open(out, "w") as f:
        f.write("\n".join(lines) + "\n")


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--config", type=int, default=5)
    ap.add_argument("--no-sweep", action="store_true",
                    help="skip the density sweep (and its crossover) that the default run adds as extra keys")
    ap.add_argument("--densities", default="0.5,0.1,0.01,0.001")
    ap.add_argument("--no-dense", action="store_true", help="skip the dense-W arm")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-layer-trace", action="store_true",
                    help="skip the untimed layer-by-layer run that gives the nnz trace (for profiling runs)")
    ap.add_argument("--cpu-rows", type=int, default=0, help="oracle sample rows (0: per-workload default)")
    ap.add_argument("--paper-grid", action="store_true",
                    help="time the paper's own grid (m x m weights, inverse sparsity 1..262144, batch 64)")
    ap.add_argument("--grid-sizes", default="", help="comma-separated m values for --paper-grid")
    ap.add_argument("--semiring", action="store_true",
                    help="time matrix multiply over each semiring of Sec. II on the density-sweep shape")
    ap.add_argument("--grid-inv", default="", help="comma-separated inverse sparsities for --paper-grid")
    ap.add_argument("--copy-probe", type=int, default=0, metavar="BYTES",
                    help="only run a plain device copy of BYTES bytes 5 times (counter calibration)")
    ap.add_argument("--summarize-stats", nargs=4, metavar=("CSV_DIR", "TITLE", "COMMAND", "OUT"),
                    help="write a profiles/ table from a rocprofv3 --stats run (no GPU needed)")
    ap.add_argument("--summarize-counters", nargs=4, metavar=("DIRS", "TITLE", "COMMANDS", "OUT"),
                    help="write a profiles/ table of per-kernel counter means from rocprofv3 --pmc runs "
                         "('|'-separated directories and commands)")
    ap.add_argument("--longest-dispatch", action="store_true",
                    help="with --summarize-counters: only each kernel's longest dispatch of every run")
    ap.add_argument("--summarize-pmc", nargs=9,
                    metavar=("KERNEL", "WORKLOAD", "FETCH_DIR", "WRITE_DIR", "COPY_FETCH_DIR", "COPY_WRITE_DIR",
                             "COPY_BYTES", "COMMANDS", "OUT"),
                    help="write a profiles/ HBM-traffic summary from rocprofv3 --pmc runs ('|'-separated commands)")
    args = ap.parse_args()
    if args.summarize_stats:
        summarize_stats(*args.summarize_stats)
        return
    if args.summarize_counters:
        a = args.summarize_counters
        summarize_counters(a[0].split("|"), a[1], a[2].split("|"), a[3], longest=args.longest_dispatch)
        return
    if args.summarize_pmc:
        a = args.summarize_pmc
        summarize_pmc(a[0], a[1], a[2:6], int(a[6]), a[7].split("|"), a[8], kernel_sources(a[0]))
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py runs on one GPU only: the library has no multi-GPU path (batch rows would shard "
              "across GPUs with no per-layer exchange; see the design notes). Use --gpus 1.", file=sys.stderr)
        sys.exit(2)

    import torch

    import paper_1708_02937_amd as sd

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    if args.copy_probe:
        src = torch.ones(args.copy_probe // 4, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_probe_bytes": args.copy_probe}), flush=True)
        return
    if args.paper_grid:
        grid, params = run_paper_grid(args, torch, sd)
        print(json.dumps({
            "metric": "per-layer time (ms) of the CSR arm and the dense-W arm on the paper's grid, 1 MI355X",
            "unit": "ms", "higher_is_better": False, "n_gpus": 1, "steps": max(3, args.steps), "dtype": "f64",
            "data": "synthetic",
            "config": {"workload": "paper-grid: m x m W, Bernoulli(1/S) pattern, U[-1,3) values, batch 64, b = 0"},
            "grid": {str(m): {str(S): v for S, v in g.items()} for m, g in grid.items()},
            "scaling_params": {str(m): v for m, v in params.items()},
        }), flush=True)
        return
    if args.semiring:
        res = run_semiring(args, torch, sd)
        print(json.dumps({
            "metric": "time per sdnn_mxm_dense call (ms) and edges/s, one MI355X", "unit": "ms",
            "higher_is_better": False, "n_gpus": 1, "dtype": "f64", "data": "synthetic",
            "config": {"workload": "density-sweep shape n=4096 batch=1024, one layer, each semiring"},
            "semiring": res}), flush=True)
        return
    if args.config == 2:
        r = run_sweep(args, torch, sd)
    else:
        r = run_csr_config(args, torch, sd)
    out = {
        "metric": METRIC, "value": r["value"], "unit": "edges/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(r["ms_step"], 4), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "f64", "data": "synthetic", "config": r["config"],
        "roofline": r["roofline"], "achieved_hbm_gbs": r.get("hbm"), "ms_per_step_median": round(r["ms_median"], 4),
        "ms_per_step_min": round(r["ms_min"], 4),
    }
    if r.get("kernel_ms_per_step"):
        out["kernel_ms_per_step"] = r["kernel_ms_per_step"]
    if r.get("sweep"):
        out["sweep"] = r["sweep"]
        out["crossover_density"] = r["crossover"]
        out["crossover_density_f32"] = r.get("crossover32")
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(args, r["probs"], args.config)
    if args.config != 2 and not args.no_sweep:
        # the paper's sparse-versus-dense comparison on the density-sweep workload, as extra keys
        probs = r.pop("probs")
        del probs
        sw_args = argparse.Namespace(**{**vars(args), "steps": min(args.steps, 10), "warmup": min(args.warmup, 2)})
        t0 = time.time()
        sw = run_sweep(sw_args, torch, sd)
        out["density_sweep"] = {"workload": sw["config"]["workload"], "ms_per_step": round(sw["ms_step"], 4),
                                "value": sw["value"], "unit": "edges/s", "steps": sw_args.steps,
                                "roofline": sw["roofline"], "achieved_hbm_gbs": sw["hbm"], "sweep": sw["sweep"],
                                "crossover_density": sw["crossover"], "crossover_density_f32": sw["crossover32"]}
        log(f"density sweep {time.time() - t0:.1f}s")
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
