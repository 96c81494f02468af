"""Benchmark of the sparse linear hot path on one MI355X.

Default workload (the headline line): the full Llama-2-7B linear stack, 32
decoder layers x 7 matrices (q, k, v, o: 4096x4096; gate, up: 11008x4096;
down: 4096x11008), distinct seeds, bf16, weights N(0, 0.02) magnitude-pruned to
70% per matrix and stored in the bitmask expansion format (4.7 GB, beyond the
256 MB Infinity Cache), activations N(0, 1), decode batch sizes 1, 2, 4, 8, 16
and 32.

One step = the whole stack at every batch size (63 tokens).  Within a batch
size the layers run in order with a decoder's data dependencies: q|k|v in one
grouped launch (they share their input), o, gate|up in one grouped launch,
down - 4 launches per layer, 128 per batch size, one HIP graph per batch size.
Inputs are resident in HBM before timing starts; `value` is tokens/s over the
wall time of the timed steps.

Printed (one JSON line): tokens/s of the whole step; per batch size the step
time, tokens/s and achieved HBM rate, the same kernels on dense weights and
the vendor GEMM library (torch linear) on the same dense weights; the
roofline of the dominant kernel (sparse decode: algorithmic bytes = stored
values + bitmask + tile offsets + X + Y per launch, over its mean launch
duration = GPU time of the timed replays from HIP events / launches), against
the nominal 8 TB/s and the read rate this device sustains (spl_read_probe);
the CPU oracle timed on this host's cores on a bounded sample.

`--workload` selects the other rows' lines (one layer, one matrix, prefill,
int8, gated MLP half, pruning, training step, int4, the stack with one launch
per layer).
"""
from __future__ import annotations

import argparse
import concurrent.futures as cf
import ctypes
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import synth  # noqa: E402

METRIC = "sparse-linear tokens/s + achieved HBM GB/s, Llama-2-7B shapes at 70% sparsity"
HBM_PEAK_GBS = 8000.0


def _gen_matrix(args):
    layer, j, N, K, dtype, sparsity = args
    W, mask = synth.weight(synth.weight_seed(layer, j), N, K, dtype, sparsity)
    return layer, j, W, mask


def _to_dev(bits, dtype, torch):
    t = torch.from_numpy(np.ascontiguousarray(bits).view(np.int16))
    return t.view(torch.bfloat16 if dtype == "bf16" else torch.float16).cuda()


def generate_layers(nlayers: int, dtype: str, sparsity: float, workers: int):
    """Host-side generation of `nlayers` distinct layers (process pool; runs
    before anything touches the GPU)."""
    jobs = [(l, j, N, K, dtype, sparsity) for l in range(nlayers)
            for j, (_, N, K) in enumerate(synth.LLAMA2_7B_LINEARS)]
    host = [[None] * len(synth.LLAMA2_7B_LINEARS) for _ in range(nlayers)]
    with cf.ProcessPoolExecutor(max_workers=workers) as ex:
        for layer, j, W, mask in ex.map(_gen_matrix, jobs):
            host[layer][j] = (W, mask)
    return host


def upload_layers(host, dtype: str, keep_dense: bool):
    """Copy to HBM and pack on the GPU (pack_sparse)."""
    import torch

    import paper_2405_03594_amd as spl

    layers = []
    for hl in host:
        row = []
        for W, mask in hl:
            Wd = _to_dev(W, dtype, torch)
            Wc = spl.pack_sparse(Wd, torch.from_numpy(mask).cuda())
            row.append((Wc, Wd if keep_dense else None))
        layers.append(row)
    torch.cuda.synchronize()
    return layers


def make_activations(dtype: str, mmax: int):
    import torch

    xs = []
    for j, (_, N, K) in enumerate(synth.LLAMA2_7B_LINEARS):
        xs.append(_to_dev(synth.activations(synth.activation_seed(j), mmax, K, dtype), dtype, torch))
    return xs


TRAFFIC_FILE = os.path.join(ROOT, "profiles", "k_sparse_decode_llama7b_stack_traffic.txt")
KERNEL_SOURCES = [os.path.join(ROOT, "paper_2405_03594_amd", "csrc", f) for f in ("k_decode.hip", "spl_common.h")]


def measured_traffic():
    """HBM bytes per launch of the sparse decode kernel from the committed
    rocprofv3 FETCH_SIZE / WRITE_SIZE summary, or None when the kernel source
    has changed since the counters were taken (or there is no summary)."""
    import hashlib

    try:
        fields = dict(line.split(": ", 1) for line in open(TRAFFIC_FILE).read().splitlines()
                      if line and not line.startswith("#"))
        h = hashlib.sha256(b"".join(open(f, "rb").read() for f in KERNEL_SOURCES)).hexdigest()
        if fields.get("source_sha256") != h:
            return None
        return int(float(fields["traffic_bytes_per_launch"]))
    except (OSError, KeyError, ValueError):
        return None


# launch units of one decoder layer (indices into synth.LLAMA2_7B_LINEARS)
GROUPED = [(0, 1, 2), (3,), (4, 5), (6,)]
SINGLE = [(j,) for j in range(7)]


def algorithmic_bytes(Wc, M: int, K: int, N: int, esz: int = 2) -> int:
    return Wc.compressed_bytes() + M * K * esz + M * N * esz


def capture_graphs(layers, units, batches, fn):
    """One HIP graph per layer: fn(layer_index, unit, M) launched for every (M, unit)."""
    import torch

    graphs = []
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        for li in range(len(layers)):          # warm the launch path once outside capture
            for M in batches:
                for u in units:
                    fn(li, u, M)
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    for li in range(len(layers)):
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            for M in batches:
                for u in units:
                    fn(li, u, M)
        graphs.append(g)
    torch.cuda.synchronize()
    return graphs


def time_graphs(graphs, steps: int, warmup: int):
    """Warm up, then time exactly `steps` graph replays (rotating layers).
    Returns (wall seconds, list of per-step GPU milliseconds from events)."""
    import torch

    for i in range(warmup):
        graphs[i % len(graphs)].replay()
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(steps):
        ev[i][0].record(stream)
        graphs[i % len(graphs)].replay()
        ev[i][1].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    return wall, [a.elapsed_time(b) for a, b in ev]


def cpu_baseline(dtype: str, sparsity: float, batches, min_seconds: float = 10.0, max_reps: int = 200):
    """The oracle (fp64, plain C, OpenMP) on one layer's seven matrices at every
    batch size, repeated until at least `min_seconds` have passed (a bounded
    sample of the workload)."""
    import oracle

    packs, xs = [], []
    for j, (_, N, K) in enumerate(synth.LLAMA2_7B_LINEARS):
        W, mask = synth.weight(synth.weight_seed(0, j), N, K, dtype, sparsity)
        packs.append(oracle.pack(W, dtype, mask))
        xs.append(synth.activations(synth.activation_seed(j), max(batches), K, dtype))
    threads = oracle.max_threads()
    reps = 0
    t0 = time.perf_counter()
    while reps < max_reps and (reps == 0 or time.perf_counter() - t0 < min_seconds):
        for M in batches:
            for p, X in zip(packs, xs):
                oracle.linear_f64(X[:M], p, nthreads=threads)
        reps += 1
    dt = time.perf_counter() - t0
    return {"value": round(reps * sum(batches) / dt, 3), "unit": "tokens/s", "cores": threads, "kind": "oracle",
            "sample": f"one decoder layer (7 matrices, layer seed 0) at batches {list(batches)}, repeated {reps} "
                      f"times: fp64 product on the decoded weights, {dt:.1f} s on {threads} threads"}


# ---------------------------------------------------------------- other workloads

MFMA_BF16_PEAK_TFLOPS = 2500.0


def _need_gpu():
    import torch

    import paper_2405_03594_amd as spl

    spl.lib()
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    return torch, spl


def _line(args, metric, value, unit, ms, workload, roofline, cpu, extra=None, dtype="bf16", higher=True):
    out = {"metric": metric, "value": value, "unit": unit, "n_gpus": 1, "steps": args.steps,
           "warmup": args.warmup, "ms_per_step": round(ms, 4), "higher_is_better": higher, "scaling": "weak",
           "vs_baseline": None, "dtype": dtype, "data": "synthetic", "config": {"workload": workload}}
    if extra:
        out["config"].update(extra)
    out["roofline"] = roofline
    if cpu is not None:
        out["cpu_baseline"] = cpu
    return out


def _timed(units, fn, steps, warmup, keys):
    """One graph per key; time `steps` replays rotating over the keys.  Returns
    (wall ms per step, GPU ms per step)."""
    graphs = []
    for k in keys:
        graphs += capture_graphs([k], units, [None], lambda li, u, M, k=k: fn(k, u))
    wall, ms = time_graphs(graphs, steps, warmup)
    return wall * 1e3 / steps, float(np.mean(ms))


def _oracle_repeat(fn, min_seconds=10.0, max_reps=5000):
    reps, t0 = 0, time.perf_counter()
    while reps < max_reps and (reps == 0 or time.perf_counter() - t0 < min_seconds):
        fn()
        reps += 1
    return reps, time.perf_counter() - t0


def _sweep(fn, copies, steps, warmup):
    """One graph of `copies` launches (one per device copy, back to back);
    `steps` replays timed.  Returns (wall ms per launch, GPU ms per launch):
    a graph of a single short launch would time the graph's own start-up."""
    graphs = capture_graphs([0], list(range(copies)), [None], lambda li, u, M: fn(u))
    wall, ms = time_graphs(graphs, steps, warmup)
    return wall * 1e3 / (steps * copies), float(np.mean(ms)) / copies


def run_single(args):
    """One 4096x4096 fp16 matrix at 50% magnitude sparsity (W seed 0), one
    activation row (X seed 1); device copies of the packed (and of the dense)
    matrix rotated, at least 1.25 GB of each, far past the 256 MB Infinity
    Cache.  A step is one sweep over the copies: one graph of back-to-back
    products, one per copy; tokens/s counts products."""
    torch, spl = _need_gpu()
    N = K = 4096
    W, mask = synth.weight(0, N, K, "f16", 0.5)
    X = synth.activations(1, 1, K, "f16")
    Wd = _to_dev(W, "f16", torch)
    Wc = spl.pack_sparse(Wd, torch.from_numpy(mask).cuda())
    copies = max(8, -(-int(1.25e9) // Wc.compressed_bytes()))
    mats = [spl.SparseMatrix(Wc.bitmask.clone(), Wc.values.clone(), None, Wc.tile_offsets.clone(), N, K, Wc.nnz,
                             "tile16") for _ in range(copies)]
    dens = [Wd.clone() for _ in range(copies)]
    Xd = _to_dev(X, "f16", torch)
    Y = torch.empty((1, N), dtype=torch.float16, device="cuda")
    # a step is one sweep: the graph's `copies` products, each on its own copy
    sp_wall, sp_gpu = _sweep(lambda i: spl.sparse_linear(Xd, mats[i], out=Y), copies, args.steps, args.warmup)
    dn_wall, dn_gpu = _sweep(lambda i: spl.dense_linear(Xd, dens[i], out=Y), copies, args.steps, args.warmup)
    nbytes = Wc.compressed_bytes() + 2 * K + 2 * N
    achieved = nbytes / (sp_gpu * 1e-3) / 1e9
    cpu = None
    if not args.no_cpu_baseline:
        import oracle

        p = oracle.pack(W, "f16", mask)
        threads = oracle.max_threads()
        reps, dt = _oracle_repeat(lambda: oracle.linear_f64(X, p, nthreads=threads))
        cpu = {"value": round(reps / dt, 3), "unit": "tokens/s", "cores": threads, "kind": "oracle",
               "sample": f"the same matrix and activation row, fp64 product on the decoded weights, repeated "
                         f"{reps} times ({dt:.1f} s on {threads} threads)"}
    return _line(args, "sparse-linear tokens/s + achieved HBM GB/s, 4096x4096 fp16 at 50% sparsity, batch 1",
                 round(1.0 / (sp_wall * 1e-3), 1), "tokens/s", sp_wall * copies,
                 "one 4096x4096 fp16 matrix, 50% unstructured magnitude sparsity (seed 0), batch 1 (seed 1), "
                 f"{copies} device copies rotated ({copies * Wc.compressed_bytes() / 1e9:.2f} GB packed, "
                 f"{copies * 2 * N * K / 1e9:.2f} GB dense); a step is one graph of {copies} back-to-back "
                 f"products, one per copy",
                 {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                  "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": None, "kernel": "k_sparse_decode",
                  "bytes_per_launch": int(nbytes), "avg_launch_us": round(sp_gpu * 1e3, 3)},
                 cpu, {"gpu_us": round(sp_gpu * 1e3, 3), "dense_gpu_us": round(dn_gpu * 1e3, 3),
                       "speedup_vs_dense": round(dn_gpu / sp_gpu, 3)}, dtype="f16")


def _library_linear_ms(torch, pairs, reps: int) -> float:
    """Cross-check of the dense comparator: torch.nn.functional.linear (the
    vendor GEMM library) over the same (X, W) pairs, eager, timed with events
    around `reps` passes; GPU ms per pass."""
    import torch.nn.functional as F

    for _ in range(2):
        for x, w in pairs:
            F.linear(x, w)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        for x, w in pairs:
            F.linear(x, w)
    e1.record()
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / reps


def run_prefill(args):
    """One layer's seven matrices at M = 512 and 2048 (prefill kernels)."""
    torch, spl = _need_gpu()
    host = generate_layers(1, "bf16", args.sparsity, args.workers)
    layers = upload_layers(host, "bf16", keep_dense=not args.no_dense)
    del host
    Ms = [512, 2048]
    xs = make_activations("bf16", max(Ms))
    shapes = synth.LLAMA2_7B_LINEARS
    ys = {(M, j): torch.empty((M, N), dtype=torch.bfloat16, device="cuda") for M in Ms for j, (_, N, _) in
          enumerate(shapes)}
    xsl = {(M, j): xs[j][:M].contiguous() for M in Ms for j in range(len(shapes))}
    units = [(M, j) for M in Ms for j in range(len(shapes))]

    def sparse_fn(li, u):
        spl.sparse_linear(xsl[u], layers[0][u[1]][0], out=ys[u], algo="prefill")

    def dense_fn(li, u):
        spl.dense_linear(xsl[u], layers[0][u[1]][1], out=ys[u], algo="prefill")

    # the decoded-copy path: one workspace for the largest matrix, reused by every launch on the stream
    ws = torch.empty((max(spl.lib().spl_sparse_linear_expanded_workspace_bytes(ctypes.byref(layers[0][j][0].view()))
                          for j in range(len(shapes))),), dtype=torch.uint8, device="cuda")

    def expanded_fn(li, u):
        spl.sparse_linear_expanded(xsl[u], layers[0][u[1]][0], out=ys[u], workspace=ws)

    sp_wall, sp_gpu = _timed(units, sparse_fn, args.steps, args.warmup, [0])
    flops = sum(2.0 * M * N * K for M in Ms for (_, N, K) in shapes)
    launch_ms = sp_gpu / len(units)
    achieved = flops / len(units) / (launch_ms * 1e-3) / 1e12
    per_M = {}
    for M in Ms:
        uM = [u for u in units if u[0] == M]
        _, g = _timed(uM, sparse_fn, max(10, args.steps // 4), 2, [0])
        f = sum(2.0 * M * N * K for (_, N, K) in shapes)
        d = {"layer_us": round(g * 1e3, 2), "dense_equiv_tflops": round(f / (g * 1e-3) / 1e12, 1)}
        _, ge = _timed(uM, expanded_fn, max(10, args.steps // 4), 2, [0])
        d.update({"expanded_layer_us": round(ge * 1e3, 2), "expanded_tflops": round(f / (ge * 1e-3) / 1e12, 1)})
        if not args.no_dense:
            _, gd = _timed(uM, dense_fn, max(10, args.steps // 4), 2, [0])
            d.update({"dense_layer_us": round(gd * 1e3, 2), "dense_tflops": round(f / (gd * 1e-3) / 1e12, 1),
                      "speedup_vs_dense": round(gd / g, 3), "expanded_speedup_vs_dense": round(gd / ge, 3)})
            gl = _library_linear_ms(torch, [(xsl[u], layers[0][u[1]][1]) for u in uM], max(10, args.steps // 4))
            d.update({"library_dense_layer_us": round(gl * 1e3, 2),
                      "library_dense_tflops": round(f / (gl * 1e-3) / 1e12, 1)})
        per_M[str(M)] = d
    cpu = None
    if not args.no_cpu_baseline:
        import oracle

        W, mask = synth.weight(synth.weight_seed(0, 0), 4096, 4096, "bf16", args.sparsity)
        p = oracle.pack(W, "bf16", mask)
        X = synth.activations(synth.activation_seed(0), 64, 4096, "bf16")
        threads = oracle.max_threads()
        reps, dt = _oracle_repeat(lambda: oracle.linear_f64(X, p, nthreads=threads))
        # tokens/s of the whole layer at this rate: 64 rows of q per repetition, scaled by the layer's work
        layer_over_q = sum(N * K for (_, N, K) in shapes) / (4096 * 4096)
        cpu = {"value": round(reps * 64 / dt / layer_over_q, 3), "unit": "tokens/s", "cores": threads,
               "kind": "oracle",
               "sample": f"64 activation rows through the q matrix (4096x4096), fp64, repeated {reps} times "
                         f"({dt:.1f} s on {threads} threads), scaled to the layer's seven matrices by their "
                         f"element count ({layer_over_q:.2f}x q)"}
    return _line(args, "sparse-linear prefill tokens/s, Llama-2-7B layer shapes", round(sum(Ms) / (sp_wall * 1e-3), 1),
                 "tokens/s", sp_wall,
                 f"Llama-2-7B decoder layer, 7 linears, bf16, {int(args.sparsity * 100)}% unstructured magnitude "
                 f"sparsity, prefill M = 512 and 2048",
                 {"bound": "mfma", "achieved": round(achieved, 1), "peak": MFMA_BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                  "frac": round(achieved / MFMA_BF16_PEAK_TFLOPS, 4), "traffic": None, "kernel": "k_sparse_prefill",
                  "flops_per_launch": "dense-equivalent 2*M*N*K", "avg_launch_us": round(launch_ms * 1e3, 3)},
                 cpu, {"per_M": per_M, "sparsity": args.sparsity})


def _gen_int8(args):
    layer, j, N, K = args[:4]
    sparsity = args[4] if len(args) > 4 else 0.7
    Wq, mask, sw = synth.int8_weight(synth.weight_seed(layer, j), N, K, sparsity)
    return layer, j, Wq, mask, sw


def run_int8(args):
    """One layer's seven matrices, int8 weights and activations at 70%, batches 1, 16, 64; 4 layers rotated."""
    torch, spl = _need_gpu()
    nl = 4
    shapes = synth.LLAMA2_7B_LINEARS
    jobs = [(l, j, N, K) for l in range(nl) for j, (_, N, K) in enumerate(shapes)]
    host = [[None] * len(shapes) for _ in range(nl)]
    with cf.ProcessPoolExecutor(max_workers=args.workers) as ex:
        for l, j, Wq, mask, sw in ex.map(_gen_int8, jobs):
            host[l][j] = (Wq, mask, sw)
    layers = []
    for hl in host:
        row = []
        for Wq, mask, sw in hl:
            Wd = torch.from_numpy(Wq).cuda()
            Wc = spl.pack_sparse(Wd, torch.from_numpy(mask).cuda())
            row.append((Wc, Wd if not args.no_dense else None, torch.from_numpy(sw).cuda()))
        layers.append(row)
    Ms = [1, 16, 64]
    xq, sx = [], []
    for j, (_, N, K) in enumerate(shapes):
        q, s_ = synth.int8_activations(synth.activation_seed(j), max(Ms), K)
        xq.append(torch.from_numpy(q).cuda())
        sx.append(torch.from_numpy(s_).cuda())
    ys = {(M, j): torch.empty((M, N), dtype=torch.float16, device="cuda") for M in Ms for j, (_, N, _) in
          enumerate(shapes)}
    xs = {(M, j): (xq[j][:M].contiguous(), sx[j][:M].contiguous()) for M in Ms for j in range(len(shapes))}
    # grouped launches as in the decode driver: q|k|v, o, gate|up, down
    units = [(M, grp) for M in Ms for grp in GROUPED]

    def sparse_fn(li, u):
        M, grp = u
        spl.sparse_linear_int8_group([xs[(M, j)][0] for j in grp], [xs[(M, j)][1] for j in grp],
                                     [layers[li][j][0] for j in grp], [layers[li][j][2] for j in grp],
                                     outs=[ys[(M, j)] for j in grp])

    def dense_fn(li, u):
        M, grp = u
        spl.dense_linear_int8_group([xs[(M, j)][0] for j in grp], [xs[(M, j)][1] for j in grp],
                                    [layers[li][j][1] for j in grp], [layers[li][j][2] for j in grp],
                                    outs=[ys[(M, j)] for j in grp])

    sp_wall, sp_gpu = _timed(units, sparse_fn, args.steps, args.warmup, range(nl))

    def nbytes(M, grp):
        total = 0
        for j in grp:
            N, K = shapes[j][1], shapes[j][2]
            total += layers[0][j][0].compressed_bytes() + 4 * N + M * K + 4 * M + 2 * M * N
        return total

    step_bytes = sum(nbytes(M, grp) for (M, grp) in units)
    launch_ms = sp_gpu / len(units)
    achieved = step_bytes / len(units) / (launch_ms * 1e-3) / 1e9
    per_M = {}
    for M in Ms:
        uM = [u for u in units if u[0] == M]
        _, g = _timed(uM, sparse_fn, max(20, args.steps // 4), 3, range(nl))
        b = sum(nbytes(M, grp) for (_, grp) in uM)
        d = {"layer_us": round(g * 1e3, 2), "hbm_gbs": round(b / (g * 1e-3) / 1e9, 1)}
        if not args.no_dense:
            _, gd = _timed(uM, dense_fn, max(20, args.steps // 4), 3, range(nl))
            d.update({"dense_layer_us": round(gd * 1e3, 2), "speedup_vs_dense": round(gd / g, 3)})
        per_M[str(M)] = d
    cpu = None
    if not args.no_cpu_baseline:
        import oracle

        packs = [oracle.pack(host[0][j][0], "i8", host[0][j][1]) for j in range(len(shapes))]
        xh = [synth.int8_activations(synth.activation_seed(j), max(Ms), K) for j, (_, N, K) in enumerate(shapes)]
        threads = oracle.max_threads()

        def one():
            for M in Ms:
                for j in range(len(shapes)):
                    oracle.linear_i8(xh[j][0][:M], xh[j][1][:M], packs[j], host[0][j][2], nthreads=threads)

        reps, dt = _oracle_repeat(one)
        cpu = {"value": round(reps * sum(Ms) / dt, 3), "unit": "tokens/s", "cores": threads, "kind": "oracle",
               "sample": f"layer 0's seven int8 matrices at batches {Ms}, int64 sums and the fp16 epilogue, "
                         f"repeated {reps} times ({dt:.1f} s on {threads} threads)"}
    return _line(args, "sparse-quantized linear tokens/s + achieved HBM GB/s, Llama-2-7B layer at 70%",
                 round(sum(Ms) / (sp_wall * 1e-3), 1), "tokens/s", sp_wall,
                 "Llama-2-7B decoder layer, 7 linears (grouped launches q|k|v, o, gate|up, down), int8 weights "
                 "(per-row scales) and int8 activations (per-token scales), 70% sparsity, batches 1, 16, 64, "
                 "4 layers rotated",
                 {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                  "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": None, "kernel": "k_sparse_int8",
                  "bytes_per_launch": int(step_bytes / len(units)), "avg_launch_us": round(launch_ms * 1e3, 3)},
                 cpu, {"per_M": per_M}, dtype="i8")


MFMA_I8_PEAK_TOPS = 5000.0
# the four distinct inputs of a decoder layer's linears: q|k|v share one, gate|up share one
INPUT_OF_GROUP = {(0, 1, 2): 0, (3,): 3, (4, 5): 4, (6,): 6}


def run_int8_prefill(args):
    """One layer's seven matrices with int8 weights at prefill batch sizes M =
    512 and 2048: each step quantizes the layer's four distinct bf16 inputs per
    token, then runs the seven sparse int8 linears (grouped as q|k|v, o,
    gate|up, down)."""
    torch, spl = _need_gpu()
    shapes = synth.LLAMA2_7B_LINEARS
    jobs = [(0, j, N, K, args.sparsity) for j, (_, N, K) in enumerate(shapes)]
    host = [None] * len(shapes)
    with cf.ProcessPoolExecutor(max_workers=min(args.workers, len(jobs))) as ex:
        for _, j, Wq, mask, sw in ex.map(_gen_int8, jobs):
            host[j] = (Wq, mask, sw)
    mats = []
    for Wq, mask, sw in host:
        Wd = torch.from_numpy(Wq).cuda()
        mats.append((spl.pack_sparse(Wd, torch.from_numpy(mask).cuda()), Wd if not args.no_dense else None,
                     torch.from_numpy(sw).cuda()))
    Ms = [512, 2048]
    xb = {j: _to_dev(synth.activations(synth.activation_seed(j), max(Ms), shapes[j][2], "bf16"), "bf16", torch)
          for j in INPUT_OF_GROUP.values()}
    xin = {(M, j): xb[j][:M].contiguous() for M in Ms for j in xb}
    xq = {(M, j): torch.empty((M, shapes[j][2]), dtype=torch.int8, device="cuda") for M in Ms for j in xb}
    sx = {(M, j): torch.empty((M,), dtype=torch.float32, device="cuda") for M in Ms for j in xb}
    ys = {(M, j): torch.empty((M, N), dtype=torch.float16, device="cuda") for M in Ms for j, (_, N, _) in
          enumerate(shapes)}
    units = [(M, grp) for M in Ms for grp in GROUPED]

    def quantize(M, grp):
        i = INPUT_OF_GROUP[grp]
        spl.quantize_rows_i8(xin[(M, i)], out=xq[(M, i)], scales=sx[(M, i)])

    def linears(M, grp, dense=False):
        i = INPUT_OF_GROUP[grp]
        call = spl.dense_linear_int8_group if dense else spl.sparse_linear_int8_group
        call([xq[(M, i)]] * len(grp), [sx[(M, i)]] * len(grp), [mats[j][1 if dense else 0] for j in grp],
             [mats[j][2] for j in grp], outs=[ys[(M, j)] for j in grp])

    def step_fn(li, u):
        quantize(*u)
        linears(*u)

    # the decoded-copy path: one workspace for the largest matrix, reused by every launch on the stream
    ws = torch.empty((max(spl.lib().spl_sparse_linear_expanded_workspace_bytes(ctypes.byref(m[0].view()))
                          for m in mats),), dtype=torch.uint8, device="cuda")

    def linears_expanded(M, grp):
        i = INPUT_OF_GROUP[grp]
        for j in grp:
            spl.sparse_linear_int8_expanded(xq[(M, i)], sx[(M, i)], mats[j][0], mats[j][2], out=ys[(M, j)],
                                            workspace=ws)

    for u in units:                                     # quantized inputs in place before linears-only timing
        quantize(*u)
    torch.cuda.synchronize()
    sp_wall, sp_gpu = _timed(units, step_fn, args.steps, args.warmup, [0])
    _, lin_gpu = _timed(units, lambda li, u: linears(*u), args.steps, args.warmup, [0])
    launches = len(Ms) * len(shapes)
    launch_ms = lin_gpu / launches
    ops = sum(2.0 * M * N * K for M in Ms for (_, N, K) in shapes)
    achieved = ops / launches / (launch_ms * 1e-3) / 1e12
    per_M = {}
    for M in Ms:
        uM = [u for u in units if u[0] == M]
        reps = max(10, args.steps // 4)
        _, g = _timed(uM, step_fn, reps, 2, [0])
        _, gl = _timed(uM, lambda li, u: linears(*u), reps, 2, [0])
        _, gq = _timed(uM, lambda li, u: quantize(*u), reps, 2, [0])
        f = sum(2.0 * M * N * K for (_, N, K) in shapes)
        qbytes = sum(3 * M * shapes[j][2] + 4 * M for j in xb)
        d = {"layer_us": round(g * 1e3, 2), "linears_us": round(gl * 1e3, 2),
             "linears_dense_equiv_tops": round(f / (gl * 1e-3) / 1e12, 1), "quantize_us": round(gq * 1e3, 2),
             "quantize_hbm_gbs": round(qbytes / (gq * 1e-3) / 1e9, 1)}
        _, ge = _timed(uM, lambda li, u: linears_expanded(*u), reps, 2, [0])
        d.update({"expanded_linears_us": round(ge * 1e3, 2), "expanded_tops": round(f / (ge * 1e-3) / 1e12, 1)})
        if not args.no_dense:
            _, gd = _timed(uM, lambda li, u: linears(*u, dense=True), reps, 2, [0])
            d.update({"dense_linears_us": round(gd * 1e3, 2), "dense_tops": round(f / (gd * 1e-3) / 1e12, 1),
                      "speedup_vs_dense": round(gd / gl, 3), "expanded_speedup_vs_dense": round(gd / ge, 3)})
        per_M[str(M)] = d
    cpu = None
    if not args.no_cpu_baseline:
        import oracle

        threads = oracle.max_threads()
        rows = 64
        packs = [oracle.pack(Wq, "i8", mask) for Wq, mask, _ in host]
        xh = {j: synth.activations(synth.activation_seed(j), rows, shapes[j][2], "bf16") for j in xb}

        def one():
            q = {j: oracle.quantize_rows_i8(xh[j], "bf16") for j in xh}
            for grp, i in INPUT_OF_GROUP.items():
                for j in grp:
                    oracle.linear_i8(q[i][0], q[i][1], packs[j], host[j][2], nthreads=threads)

        reps, dt = _oracle_repeat(one)
        cpu = {"value": round(reps * rows / dt, 3), "unit": "tokens/s", "cores": threads, "kind": "oracle",
               "sample": f"{rows} tokens through the whole step (the four inputs quantized per token, the seven "
                         f"int8 matrices with int64 sums and the fp16 epilogue), repeated {reps} times "
                         f"({dt:.1f} s on {threads} threads)"}
    return _line(args, "sparse-quantized prefill tokens/s, Llama-2-7B layer shapes",
                 round(sum(Ms) / (sp_wall * 1e-3), 1), "tokens/s", sp_wall,
                 f"Llama-2-7B decoder layer, 7 linears (q|k|v, o, gate|up, down), int8 weights (per-row scales), "
                 f"bf16 activations quantized per token in the step, {int(args.sparsity * 100)}% unstructured "
                 f"magnitude sparsity, prefill M = 512 and 2048",
                 {"bound": "mfma", "achieved": round(achieved, 1), "peak": MFMA_I8_PEAK_TOPS, "unit": "TOP/s",
                  "frac": round(achieved / MFMA_I8_PEAK_TOPS, 4), "traffic": None,
                  "kernel": "k_sparse_prefill<int8>", "ops_per_launch": "dense-equivalent 2*M*N*K",
                  "avg_launch_us": round(launch_ms * 1e3, 3)},
                 cpu, {"per_M": per_M, "sparsity": args.sparsity}, dtype="i8")


def run_gated(args):
    """The gated half of a Llama MLP, silu(X Wgate^T) * (X Wup^T), on 4
    generated layers' gate/up pairs (11008 x 4096, --sparsity), cloned into
    at least 1.25 GB of device copies: one step = one graph of the fused
    launch on every copy at decode batches 1, 4 and 16 (batch-major, so a
    copy is not re-read until the whole set has streamed past the 256 MB
    Infinity Cache).  Prefill batches 512 and 2048 and the unfused path
    (grouped gate|up launch, then torch's silu and product) are timed
    alongside, each as one graph of back-to-back launches."""
    nl = 4
    N, K = 11008, 4096
    jobs = [(l, j, N, K, "bf16", args.sparsity) for l in range(nl) for j in (4, 5)]
    host = {}
    with cf.ProcessPoolExecutor(max_workers=min(args.workers, len(jobs))) as ex:
        for layer, j, W, mask in ex.map(_gen_matrix, jobs):
            host[(layer, j)] = (W, mask)
    torch, spl = _need_gpu()
    import torch.nn.functional as F

    mats = [[spl.pack_sparse(_to_dev(host[(l, j)][0], "bf16", torch), torch.from_numpy(host[(l, j)][1]).cuda())
             for j in (4, 5)] for l in range(nl)]
    Ms = [1, 4, 16]
    Mp = [512, 2048]
    xb = _to_dev(synth.activations(synth.activation_seed(4), max(Mp), K, "bf16"), "bf16", torch)
    xs = {M: xb[:M].contiguous() for M in Ms + Mp}
    ys = {M: torch.empty((M, N), dtype=torch.bfloat16, device="cuda") for M in Ms + Mp}
    gs = {M: torch.empty((M, N), dtype=torch.bfloat16, device="cuda") for M in Ms + Mp}
    us = {M: torch.empty((M, N), dtype=torch.bfloat16, device="cuda") for M in Ms + Mp}

    pair_bytes = mats[0][0].compressed_bytes() + mats[0][1].compressed_bytes()
    ncopy = max(2 * nl, -(-int(1.25e9) // pair_bytes))
    pairs = mats + [[spl.SparseMatrix(m.bitmask.clone(), m.values.clone(), None, m.tile_offsets.clone(), m.rows,
                                      m.cols, m.nnz, "tile16") for m in mats[c % nl]] for c in range(nl, ncopy)]

    def fused(c, M):
        spl.sparse_linear_silu_mul(xs[M], pairs[c][0], pairs[c][1], out=ys[M])

    def unfused(c, M):
        spl.sparse_linear_group([xs[M], xs[M]], pairs[c], outs=[gs[M], us[M]])
        torch.mul(F.silu(gs[M]), us[M], out=ys[M])

    units = [(c, M) for M in Ms for c in range(ncopy)]
    graphs = capture_graphs([0], units, [None], lambda li, u, M: fused(*u))
    wall, ms = time_graphs(graphs, args.steps, args.warmup)
    sp_wall, sp_gpu = wall * 1e3 / args.steps, float(np.mean(ms))
    del graphs
    nbytes = {M: pair_bytes + 2 * M * K + 2 * M * N for M in Ms}
    launch_ms = sp_gpu / len(units)
    achieved = sum(nbytes.values()) * ncopy / (sp_gpu * 1e-3) / 1e9
    per_M = {}
    for M in Ms + Mp:
        reps = max(10, args.steps // 4) if M in Ms else 10
        n = ncopy if M in Ms else nl
        _, g = _sweep(lambda c: fused(c, M), n, reps, 2)
        _, gu = _sweep(lambda c: unfused(c, M), n, reps, 2)
        d = {"fused_us": round(g * 1e3, 2), "unfused_us": round(gu * 1e3, 2), "fused_speedup": round(gu / g, 3)}
        if M in Ms:
            d["hbm_gbs"] = round(nbytes[M] / (g * 1e-3) / 1e9, 1)
        else:
            d["dense_equiv_tflops"] = round(2.0 * 2 * M * N * K / (g * 1e-3) / 1e12, 1)
        per_M[str(M)] = d
    cpu = None
    if not args.no_cpu_baseline:
        import oracle

        threads = oracle.max_threads()
        pg = oracle.pack(host[(0, 4)][0], "bf16", host[(0, 4)][1])
        pu = oracle.pack(host[(0, 5)][0], "bf16", host[(0, 5)][1])
        X = synth.activations(synth.activation_seed(4), max(Ms), K, "bf16")

        def one():
            for M in Ms:
                oracle.silu_mul_f64(X[:M], pg, pu, nthreads=threads)

        reps, dt = _oracle_repeat(one)
        cpu = {"value": round(reps * sum(Ms) / dt, 3), "unit": "tokens/s", "cores": threads, "kind": "oracle",
               "sample": f"layer 0's gate/up pair at batches {Ms}, binary64 products and silu, repeated {reps} "
                         f"times ({dt:.1f} s on {threads} threads)"}
    return _line(args, "gated MLP half (silu(gate) * up) tokens/s + achieved HBM GB/s, Llama-2-7B gate/up",
                 round(ncopy * sum(Ms) / (sp_wall * 1e-3), 1), "tokens/s", sp_wall,
                 f"Llama-2-7B gate and up (11008x4096 each), bf16, {int(args.sparsity * 100)}% unstructured "
                 f"magnitude sparsity, fused silu(gate) * up, batches 1, 4, 16; {nl} generated layers cloned into "
                 f"{ncopy} device copies ({ncopy * pair_bytes / 1e9:.2f} GB packed), a step is one graph of "
                 f"{len(units)} launches (every copy at every batch)",
                 {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                  "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": None, "kernel": "k_sparse_decode2<gated>",
                  "bytes_per_launch": int(sum(nbytes.values()) / len(Ms)), "avg_launch_us": round(launch_ms * 1e3, 3)},
                 cpu, {"per_M": per_M, "sparsity": args.sparsity})


def run_prune(args):
    """Magnitude pruning of one Llama-2-7B layer's seven bf16 matrices on the
    GPU (keep-masks at --sparsity), then packing them (pack_sparse): one step
    = mask + pack for all seven; 2 layers rotated."""
    nl = 2
    shapes = synth.LLAMA2_7B_LINEARS
    torch, spl = _need_gpu()
    ws = torch.empty((spl.lib().spl_magnitude_mask_workspace_bytes(),), dtype=torch.uint8, device="cuda")
    num, den = synth.parse_sparsity(args.sparsity)
    Ws = [[_to_dev(synth.round_to(synth.normal_f32(synth.weight_seed(l, j), (N, K), synth.WEIGHT_STD), "bf16"),
                   "bf16", torch) for j, (_, N, K) in enumerate(shapes)] for l in range(nl)]
    masks = [torch.empty((N, K), dtype=torch.uint8, device="cuda") for (_, N, K) in shapes]
    prunes = [N * K * num // den for (_, N, K) in shapes]

    def mask_fn(li, j):
        spl.magnitude_mask(Ws[li][j], prunes[j], out=masks[j], workspace=ws)

    units = list(range(len(shapes)))
    sp_wall, sp_gpu = _timed(units, mask_fn, args.steps, args.warmup, range(nl))
    algo_bytes = sum(3 * N * K for (_, N, K) in shapes)          # read W (2 B) once, write the mask (1 B)
    launch_ms = sp_gpu / len(units)
    achieved = algo_bytes / len(units) / (launch_ms * 1e-3) / 1e9
    t0 = time.perf_counter()
    torch.cuda.synchronize()
    reps = 5
    for _ in range(reps):
        for j in units:
            spl.pack_sparse(Ws[0][j], masks[j])
    torch.cuda.synchronize()
    pack_ms = (time.perf_counter() - t0) * 1e3 / reps
    cpu = None
    if not args.no_cpu_baseline:
        import oracle

        W = synth.round_to(synth.normal_f32(synth.weight_seed(0, 0), (4096, 4096), synth.WEIGHT_STD), "bf16")
        reps_c, dt = _oracle_repeat(lambda: oracle.magnitude_mask(W, "bf16", prunes[0]), min_seconds=10.0)
        layer_over_q = sum(N * K for (_, N, K) in shapes) / (4096 * 4096)
        cpu = {"value": round(reps_c / dt / layer_over_q, 4), "unit": "layers/s", "cores": 1, "kind": "oracle",
               "sample": f"the q matrix (4096x4096) masked {reps_c} times ({dt:.1f} s, one thread: a stable sort), "
                         f"scaled to the layer's seven matrices by element count ({layer_over_q:.2f}x q)"}
    return _line(args, "magnitude-pruning masks per second, one Llama-2-7B layer (7 matrices)",
                 round(1.0 / (sp_wall * 1e-3), 2), "layers/s", sp_wall,
                 f"Llama-2-7B decoder layer's seven bf16 matrices, N(0, 0.02), masks at "
                 f"{int(args.sparsity * 100)}% (exact count per matrix, ties by index), 2 layers rotated",
                 {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                  "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": None, "kernel": "k_mag_* (5 launches)",
                  "bytes_per_launch": int(algo_bytes / len(units)), "avg_launch_us": round(launch_ms * 1e3, 3)},
                 cpu, {"pack_sparse_ms_per_layer": round(pack_ms, 3), "sparsity": args.sparsity}, dtype="bf16")


def run_train(args):
    """One sparse training step of a Llama-2-7B layer's seven linears with the
    mask held fixed (Algorithm 1), M = 2048 tokens, bf16: per matrix the
    forward product, the weight gradient in the packed value order (one
    grouped call for the matrices that share an input: q|k|v, gate|up), the
    SGD update of the stored values and the input gradient read from W's
    packed tiles.  The alternative input gradient through a packed transpose (its
    values refreshed by a permutation gather after the update) is timed
    alongside."""
    shapes = synth.LLAMA2_7B_LINEARS
    host = generate_layers(1, "bf16", args.sparsity, args.workers)[0]
    torch, spl = _need_gpu()
    M = 2048
    lr = 1e-3
    mats, mats_t, perms, ws, igws, grads, xs, dys, ys, dxs = [], [], [], [], [], [], [], [], [], []
    for j, (_, N, K) in enumerate(shapes):
        W, mask = host[j]
        Wd = _to_dev(W, "bf16", torch)
        md = torch.from_numpy(mask).cuda()
        Wc = spl.pack_sparse(Wd, md)
        Wt = spl.pack_sparse(spl.transpose16(spl.unpack(Wc)), md.t().contiguous())   # set-up: the transposed pattern
        mats.append(Wc)
        mats_t.append(Wt)
        perms.append(spl.transpose_perm(Wc, Wt))                          # set-up: Wt's values from Wc's
        ws.append(torch.empty((spl.lib().spl_sparse_weight_grad_workspace_bytes(M, N, K),), dtype=torch.uint8,
                              device="cuda"))
        nig = spl.lib().spl_sparse_input_grad_workspace_bytes(M, ctypes.byref(Wc.view()))
        igws.append(torch.empty((nig,), dtype=torch.uint8, device="cuda") if nig > 0 else None)
        grads.append(torch.empty_like(Wc.values))
        xs.append(_to_dev(synth.activations(synth.activation_seed(j), M, K, "bf16"), "bf16", torch))
        dys.append(_to_dev(synth.activations(700 + j, M, N, "bf16"), "bf16", torch))
        ys.append(torch.empty((M, N), dtype=torch.bfloat16, device="cuda"))
        dxs.append(torch.empty((M, K), dtype=torch.bfloat16, device="cuda"))
    del host
    # the weight gradients of the matrices that share an input (q|k|v, gate|up) in one grouped call
    unit_of = {j: grp for grp in GROUPED for j in grp}
    gws = {grp: max((ws[i] for i in grp), key=lambda t: t.numel()) for grp in GROUPED}

    def step(li, j, part="all"):
        if part in ("all", "fwd"):
            spl.sparse_linear(xs[j], mats[j], out=ys[j])
        if part in ("all", "wgrad") and j == unit_of[j][0]:       # one grouped call per same-input unit
            grp = unit_of[j]
            spl.sparse_weight_grad_group([dys[i] for i in grp], [xs[i] for i in grp], [mats[i] for i in grp],
                                         outs=[grads[i] for i in grp], workspace=gws[grp])
        if part in ("all", "update"):
            spl.sparse_sgd_update(mats[j], grads[j], lr)
        if part in ("all", "dgrad"):
            spl.sparse_input_grad(dys[j], mats[j], out=dxs[j], workspace=igws[j])
        if part == "dgrad_packed_transpose":
            spl.permute_values(mats[j].values, perms[j], mats[j].nnz, mats_t[j].values)
            spl.sparse_linear(dys[j], mats_t[j], out=dxs[j])

    units = list(range(len(shapes)))
    wall, gpu = _timed(units, lambda li, j: step(li, j), args.steps, args.warmup, [0])
    parts = {}
    for part in ("fwd", "wgrad", "update", "dgrad", "dgrad_packed_transpose"):
        _, g = _timed(units, lambda li, j, part=part: step(li, j, part), max(5, args.steps // 4), 2, [0])
        parts[part + "_us"] = round(g * 1e3, 1)
    flops = sum(2.0 * M * N * K for (_, N, K) in shapes)                # one dense-equivalent product
    wgrad_ms = parts["wgrad_us"] * 1e-3
    achieved = flops / (wgrad_ms * 1e-3) / 1e12
    # the weight gradient issues the dense product; only its kept entries (2 M nnz flops) are wanted
    kept_flops = sum(2.0 * M * Wc.nnz for Wc in mats)
    parts["wgrad_kept_tflops"] = round(kept_flops / (wgrad_ms * 1e-3) / 1e12, 1)
    parts["wgrad_issued_tflops"] = round(achieved, 1)
    parts["step_dense_equiv_tflops"] = round(3 * flops / (gpu * 1e-3) / 1e12, 1)
    cpu = None
    if not args.no_cpu_baseline:
        import oracle

        N, K = shapes[0][1], shapes[0][2]
        Wq, mq = synth.weight(synth.weight_seed(0, 0), N, K, "bf16", args.sparsity)
        p = oracle.pack(Wq, "bf16", mq)
        rows = 64
        X = synth.activations(synth.activation_seed(0), rows, K, "bf16")
        dY = synth.activations(700, rows, N, "bf16")
        threads = oracle.max_threads()

        def one():
            oracle.linear_f64(X, p, nthreads=threads)
            oracle.weight_grad_f64(dY, X, "bf16", p)
            oracle.input_grad_f64(dY, "bf16", p)

        reps, dt = _oracle_repeat(one)
        layer_over_q = sum(N_ * K_ for (_, N_, K_) in shapes) / (N * K)
        cpu = {"value": round(reps * rows / dt / layer_over_q, 3), "unit": "tokens/s", "cores": threads,
               "kind": "oracle",
               "sample": f"{rows} tokens through the q matrix (forward, weight and input gradients in binary64), "
                         f"repeated {reps} times ({dt:.1f} s), scaled to the layer's seven matrices by element "
                         f"count ({layer_over_q:.2f}x q)"}
    return _line(args, "sparse training step tokens/s (mask held fixed), Llama-2-7B layer's linears",
                 round(M / (wall * 1e-3), 1), "tokens/s", wall,
                 f"Llama-2-7B decoder layer, 7 linears, bf16, {int(args.sparsity * 100)}% magnitude sparsity, "
                 f"M = {M} tokens: forward, weight gradient, SGD on the packed values, input gradient from the "
                 f"packed tiles",
                 {"bound": "mfma", "achieved": round(achieved, 1), "peak": MFMA_BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                  "frac": round(achieved / MFMA_BF16_PEAK_TFLOPS, 4), "traffic": None,
                  "kernel": "weight gradient (k_dense_prefill_dma_tr: dY and X read as stored, gather epilogue; "
                            "q|k|v and gate|up grouped: 4 launches per layer)",
                  "flops_per_launch": "2*M*N*K summed over the launch's matrices",
                  "avg_launch_us": round(parts["wgrad_us"] / len(GROUPED), 3)},
                 cpu, {"parts_per_layer": parts, "sparsity": args.sparsity, "lr": lr})


def _gen_int4(args):
    layer, j, N, K = args
    Wq, mask, sw = synth.int4_weight(synth.weight_seed(layer, j), N, K, 0.7)
    return layer, j, Wq, mask, sw


def run_int4(args):
    """One layer's seven matrices with 4-bit weights (per-row scales) at 70%,
    int8 activations, batches 1 and 16, one launch per matrix, 4 layers
    rotated; the same codes run through the int8 path alongside."""
    torch, spl = _need_gpu()
    nl = 4
    shapes = synth.LLAMA2_7B_LINEARS
    jobs = [(l, j, N, K) for l in range(nl) for j, (_, N, K) in enumerate(shapes)]
    host = [[None] * len(shapes) for _ in range(nl)]
    with cf.ProcessPoolExecutor(max_workers=args.workers) as ex:
        for l, j, Wq, mask, sw in ex.map(_gen_int4, jobs):
            host[l][j] = (Wq, mask, sw)
    layers = []
    for hl in host:
        row = []
        for Wq, mask, sw in hl:
            W8 = spl.pack_sparse(torch.from_numpy(Wq).cuda(), torch.from_numpy(mask).cuda())
            row.append((spl.pack_int4(W8), W8, torch.from_numpy(sw).cuda()))
        layers.append(row)
    Ms = [1, 16]
    xq, sx = [], []
    for j, (_, N, K) in enumerate(shapes):
        q, s_ = synth.int8_activations(synth.activation_seed(j), max(Ms), K)
        xq.append(torch.from_numpy(q).cuda())
        sx.append(torch.from_numpy(s_).cuda())
    xs = {(M, j): (xq[j][:M].contiguous(), sx[j][:M].contiguous()) for M in Ms for j in range(len(shapes))}
    ys = {(M, j): torch.empty((M, N), dtype=torch.float16, device="cuda") for M in Ms for j, (_, N, _) in
          enumerate(shapes)}
    units = [(M, j) for M in Ms for j in range(len(shapes))]

    def i4_fn(li, u):
        M, j = u
        spl.sparse_linear_int4(xs[u][0], xs[u][1], layers[li][j][0], layers[li][j][2], out=ys[u])

    def i8_fn(li, u):
        M, j = u
        spl.sparse_linear_int8(xs[u][0], xs[u][1], layers[li][j][1], layers[li][j][2], out=ys[u])

    wall, gpu = _timed(units, i4_fn, args.steps, args.warmup, range(nl))

    def nbytes(M, j):
        N, K = shapes[j][1], shapes[j][2]
        return layers[0][j][0].compressed_bytes() + 4 * N + M * K + 4 * M + 2 * M * N

    launch_ms = gpu / len(units)
    achieved = sum(nbytes(*u) for u in units) / len(units) / (launch_ms * 1e-3) / 1e9
    per_M = {}
    for M in Ms:
        uM = [u for u in units if u[0] == M]
        _, g4 = _timed(uM, i4_fn, max(20, args.steps // 4), 3, range(nl))
        _, g8 = _timed(uM, i8_fn, max(20, args.steps // 4), 3, range(nl))
        b = sum(nbytes(*u) for u in uM)
        per_M[str(M)] = {"layer_us": round(g4 * 1e3, 2), "hbm_gbs": round(b / (g4 * 1e-3) / 1e9, 1),
                         "int8_path_layer_us": round(g8 * 1e3, 2), "vs_int8_path": round(g8 / g4, 3)}
    cpu = None
    if not args.no_cpu_baseline:
        import oracle

        packs = [oracle.pack(host[0][j][0], "i8", host[0][j][1]) for j in range(len(shapes))]
        xh = [synth.int8_activations(synth.activation_seed(j), max(Ms), K) for j, (_, N, K) in enumerate(shapes)]
        threads = oracle.max_threads()

        def one():
            for M in Ms:
                for j in range(len(shapes)):
                    oracle.linear_i8(xh[j][0][:M], xh[j][1][:M], packs[j], host[0][j][2], nthreads=threads)

        reps, dt = _oracle_repeat(one)
        cpu = {"value": round(reps * sum(Ms) / dt, 3), "unit": "tokens/s", "cores": threads, "kind": "oracle",
               "sample": f"layer 0's seven matrices' 4-bit codes at batches {Ms} (int64 sums, fp16 epilogue), "
                         f"repeated {reps} times ({dt:.1f} s on {threads} threads)"}
    return _line(args, "4-bit sparse linear tokens/s + achieved HBM GB/s, Llama-2-7B layer at 70%",
                 round(sum(Ms) / (wall * 1e-3), 1), "tokens/s", wall,
                 "Llama-2-7B decoder layer, 7 linears, 4-bit weights (per-row scales) and int8 activations "
                 "(per-token scales), 70% sparsity, batches 1 and 16, one launch per matrix, 4 layers rotated",
                 {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                  "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": None, "kernel": "k_sparse_i4",
                  "bytes_per_launch": int(sum(nbytes(*u) for u in units) / len(units)),
                  "avg_launch_us": round(launch_ms * 1e3, 3)},
                 cpu, {"per_M": per_M}, dtype="i8")


def _gen_weight_bits(job):
    """Worker: the bf16 bits of matrix j of layer l (the generator's draw and
    rounding; the mask is made on the GPU, bit-exact with the generator's)."""
    l, j, N, K = job
    return l, j, synth.round_to(synth.normal_f32(synth.weight_seed(l, j), (N, K), synth.WEIGHT_STD), "bf16")


STACK_MS = [1, 2, 4, 8, 16, 32]
STACK_LAYERS = 32


def load_stack(args, keep_dense: bool):
    """All 32 layers (224 matrices, distinct seeds) at 70%: weights drawn on the
    host by worker processes started before this process touches the GPU,
    magnitude masks and packing on the GPU.  Returns (torch, spl, layers) with
    layers[l][j] = (packed, dense or None)."""
    import multiprocessing as mp

    shapes = synth.LLAMA2_7B_LINEARS
    num, den = synth.parse_sparsity(args.sparsity)
    jobs = [(l, j, N, K) for l in range(STACK_LAYERS) for j, (_, N, K) in enumerate(shapes)]
    with cf.ProcessPoolExecutor(max_workers=args.workers, mp_context=mp.get_context("spawn")) as ex:
        futures = [ex.submit(_gen_weight_bits, job) for job in jobs]     # workers exist before the GPU is used
        torch, spl = _need_gpu()
        ws = torch.empty((spl.lib().spl_magnitude_mask_workspace_bytes(),), dtype=torch.uint8, device="cuda")
        layers = [[None] * len(shapes) for _ in range(STACK_LAYERS)]
        for f in futures:
            l, j, bits = f.result()
            N, K = bits.shape
            Wd = _to_dev(bits, "bf16", torch)
            mask = spl.magnitude_mask(Wd, N * K * num // den, workspace=ws)
            layers[l][j] = (spl.pack_sparse(Wd, mask), Wd if keep_dense else None)
            del mask
    torch.cuda.synchronize()
    return torch, spl, layers


def hbm_probe(torch, spl, nbytes: int = 4 << 30, reps: int = 10) -> float:
    """Best read rate (GB/s) of spl_read_probe over a buffer far larger than the
    Infinity Cache."""
    buf = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    sink = torch.zeros(1, dtype=torch.int32, device="cuda")
    best = 0.0
    for i in range(reps + 2):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        spl.read_probe(buf, sink)
        e1.record()
        torch.cuda.synchronize()
        if i >= 2:
            best = max(best, nbytes / (e0.elapsed_time(e1) * 1e-3) / 1e9)
    del buf
    return best


def _stack_fns(spl, layers, xsl, ys, units):
    def sparse_stack(M):
        for row in layers:
            for u in units:
                spl.sparse_linear_group([xsl[(M, j)] for j in u], [row[j][0] for j in u], outs=[ys[(M, j)] for j in u])

    def dense_stack(M):
        for row in layers:
            for u in units:
                spl.dense_linear_group([xsl[(M, j)] for j in u], [row[j][1] for j in u], outs=[ys[(M, j)] for j in u])
    return sparse_stack, dense_stack


def _graph(torch, fn):
    """fn() captured in one HIP graph (after one eager run that warms the launch path)."""
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        fn()
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        fn()
    torch.cuda.synchronize()
    return g


def _replay_ms(torch, g, reps: int, warmup: int = 2) -> float:
    for _ in range(warmup):
        g.replay()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        g.replay()
    e1.record()
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / reps


def run_stack(args):
    """Default workload: the full 32-layer Llama-2-7B linear stack (224
    matrices, distinct seeds) at 70%, bf16, decode batches 1, 2, 4, 8, 16, 32.
    One step = the whole stack at every batch size, each batch size layer after
    layer in a decoder's order with its data dependencies: q|k|v (one grouped
    launch: they share their input), o, gate|up (one grouped launch), down -
    4 launches per layer, 128 per batch size, one HIP graph per batch size."""
    torch, spl, layers = load_stack(args, keep_dense=not args.no_dense)
    shapes = synth.LLAMA2_7B_LINEARS
    Ms = STACK_MS
    xs = make_activations("bf16", max(Ms))
    xsl = {(M, j): xs[j][:M].contiguous() for M in Ms for j in range(len(shapes))}
    ys = {(M, j): torch.empty((M, N), dtype=torch.bfloat16, device="cuda") for M in Ms
          for j, (_, N, _) in enumerate(shapes)}
    sparse_stack, dense_stack = _stack_fns(spl, layers, xsl, ys, GROUPED)
    graphs = {M: _graph(torch, lambda M=M: sparse_stack(M)) for M in Ms}

    # timed region: `steps` steps, each the stack at every batch size; events per batch size
    for i in range(args.warmup):
        for M in Ms:
            graphs[M].replay()
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    ev = {M: [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
              for _ in range(args.steps)] for M in Ms}
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        for M in Ms:
            ev[M][i][0].record(stream)
            graphs[M].replay()
            ev[M][i][1].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    gpu_ms = {M: float(np.mean([a.elapsed_time(b) for a, b in ev[M]])) for M in Ms}
    del graphs

    nl = len(layers)
    launches = nl * len(GROUPED)
    weight_bytes = sum(layers[l][j][0].compressed_bytes() for l in range(nl) for j in range(len(shapes)))
    xy_bytes = {M: nl * sum(M * (K + N) * 2 for (_, N, K) in shapes) for M in Ms}
    dense_bytes = nl * sum(N * K * 2 for (_, N, K) in shapes)
    per_M = {}
    reps = max(5, args.steps // 4)
    for M in Ms:
        g = gpu_ms[M]
        d = {"step_us": round(g * 1e3, 1), "tokens_per_s": round(M / (g * 1e-3), 1),
             "hbm_gbs": round((weight_bytes + xy_bytes[M]) / (g * 1e-3) / 1e9, 1),
             "layer_us": round(g * 1e3 / nl, 2)}
        if not args.no_dense:
            gd_graph = _graph(torch, lambda M=M: dense_stack(M))
            gd = _replay_ms(torch, gd_graph, reps)
            del gd_graph
            d.update({"dense_step_us": round(gd * 1e3, 1),
                      "dense_hbm_gbs": round((dense_bytes + xy_bytes[M]) / (gd * 1e-3) / 1e9, 1),
                      "speedup_vs_dense": round(gd / g, 3)})
        per_M[str(M)] = d

    # the vendor library's dense GEMM (torch linear -> hipBLASLt / rocBLAS) on the same
    # dense weights, as a cross-check of the dense comparator
    vendor = {}
    if not args.no_dense:
        for M in (1, 4, 16):
            def vendor_stack(M=M):
                for row in layers:
                    for j in range(len(shapes)):
                        torch.nn.functional.linear(xsl[(M, j)], row[j][1], out=ys[(M, j)])
            vendor_stack()
            ref = ys[(M, 6)].clone()
            gv = _graph(torch, vendor_stack)
            us = _replay_ms(torch, gv, reps) * 1e3
            same = bool(torch.equal(ys[(M, 6)], ref))          # the graph replays what eager computes
            del gv
            vendor[str(M)] = {"step_us": round(us, 1),
                              "hbm_gbs": round((dense_bytes + xy_bytes[M]) / (us * 1e-6) / 1e9, 1),
                              "our_dense_vs_vendor": round(us / per_M[str(M)]["dense_step_us"], 3),
                              "graph_matches_eager": same}

    probe = hbm_probe(torch, spl)
    avg_launch_ms = sum(gpu_ms.values()) / (len(Ms) * launches)
    bytes_per_launch = sum(weight_bytes + xy_bytes[M] for M in Ms) / (len(Ms) * launches)
    achieved = bytes_per_launch / (avg_launch_ms * 1e-3) / 1e9
    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline("bf16", args.sparsity, [1])
        cpu["value"] = round(cpu["value"] / nl, 4)
        cpu["sample"] += f"; tokens/s of the {nl}-layer stack = that rate / {nl}"
    tokens = sum(Ms) * args.steps
    out = _line(args, METRIC, round(tokens / wall, 1), "tokens/s", wall * 1e3 / args.steps,
                "Llama-2-7B linear stack: 32 layers x 7 matrices (q,k,v,o 4096x4096; gate,up 11008x4096; down "
                "4096x11008), distinct seeds, bf16, 70% unstructured magnitude sparsity in bitmask format; one step "
                f"= the stack at decode batches {Ms} ({sum(Ms)} tokens), 4 dependent launches per layer",
                {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                 "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": measured_traffic(), "kernel": "k_sparse_decode",
                 "bytes_per_launch": int(bytes_per_launch), "avg_launch_us": round(avg_launch_ms * 1e3, 3),
                 "peak_measured": round(probe, 1), "frac_of_measured": round(achieved / probe, 4)},
                cpu,
                {"batches": Ms, "tokens_per_step": sum(Ms), "launches_per_batch": launches,
                 "compressed_weight_bytes": int(weight_bytes), "dense_weight_bytes": int(dense_bytes),
                 "per_M": per_M, "vendor_dense": vendor, "hbm_read_probe_gbs": round(probe, 1),
                 "gpu_ms_per_step": round(sum(gpu_ms.values()), 4)})
    return out


def run_stack_layer(args):
    """The same stack with the seven linears of a layer in ONE launch (the
    benchmark's inputs are not chained from matrix to matrix, so a layer's
    matrices are independent): 32 launches per batch size.  Shows the kernel
    without the fixed cost of four launches per layer."""
    torch, spl, layers = load_stack(args, keep_dense=False)
    shapes = synth.LLAMA2_7B_LINEARS
    Ms = STACK_MS
    xs = make_activations("bf16", max(Ms))
    xsl = {(M, j): xs[j][:M].contiguous() for M in Ms for j in range(len(shapes))}
    ys = {(M, j): torch.empty((M, N), dtype=torch.bfloat16, device="cuda") for M in Ms
          for j, (_, N, _) in enumerate(shapes)}
    order = [(6, 4, 5, 0, 1, 2, 3)]                 # the longest rows (down) first
    sparse_stack, _ = _stack_fns(spl, layers, xsl, ys, order)
    nl = len(layers)
    weight_bytes = sum(layers[l][j][0].compressed_bytes() for l in range(nl) for j in range(len(shapes)))
    per_M, wall_ms = {}, 0.0
    for M in Ms:
        g = _graph(torch, lambda M=M: sparse_stack(M))
        ms = _replay_ms(torch, g, args.steps, args.warmup)
        del g
        b = weight_bytes + nl * sum(M * (K + N) * 2 for (_, N, K) in shapes)
        per_M[str(M)] = {"step_us": round(ms * 1e3, 1), "tokens_per_s": round(M / (ms * 1e-3), 1),
                         "hbm_gbs": round(b / (ms * 1e-3) / 1e9, 1)}
        wall_ms += ms
    avg_launch_ms = wall_ms / (len(Ms) * nl)
    bpl = sum(weight_bytes + nl * sum(M * (K + N) * 2 for (_, N, K) in shapes) for M in Ms) / (len(Ms) * nl)
    achieved = bpl / (avg_launch_ms * 1e-3) / 1e9
    return _line(args, METRIC, round(sum(Ms) / (wall_ms * 1e-3), 1), "tokens/s", wall_ms,
                 "Llama-2-7B linear stack, 32 layers x 7 matrices, bf16, 70%; one launch per layer (its seven "
                 f"independent matrices), decode batches {Ms}",
                 {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                  "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": None, "kernel": "k_sparse_decode",
                  "bytes_per_launch": int(bpl), "avg_launch_us": round(avg_launch_ms * 1e3, 3)},
                 None, {"per_M": per_M})


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--layers", type=int, default=8, help="distinct layers rotated through (>= 8 defeats MALL)")
    ap.add_argument("--sparsity", type=float, default=0.7)
    ap.add_argument("--batches", type=str, default="1,4,16")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-dense", action="store_true")
    ap.add_argument("--workers", type=int, default=min(16, os.cpu_count() or 1))
    ap.add_argument("--driver", choices=["grouped", "single"], default="grouped",
                    help="grouped: q|k|v and gate|up share a launch (a decoder layer's independent projections)")
    ap.add_argument("--workload", choices=["stack", "stack-layer", "layer", "decode", "single", "prefill", "int8",
                                           "int8-prefill", "gated", "prune", "train", "int4"],
                    default="stack",
                    help="stack: the 32-layer Llama-2-7B linear stack at batches 1..32, 4 dependent launches per "
                         "layer (default, the headline); stack-layer: the same with one launch per layer; layer "
                         "(or decode): one layer at batches 1,4,16; single: one 4096x4096 "
                         "fp16 matrix at 50%%, batch 1; prefill: one layer at M=512 and 2048; int8: one layer, "
                         "int8 weights and activations, batches 1,16,64; int8-prefill: one layer, int8 weights, "
                         "activations quantized per token, M=512 and 2048; gated: fused silu(gate)*up "
                         "of gate/up at batches 1,4,16; prune: magnitude masks of one layer; train: a masked training step of one "
                         "layer at M=2048; int4: 4-bit weights at batches 1,16")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="BYTES",
                    help="only run a plain device-to-device copy of BYTES ten times (the reference kernel "
                         "for scaling rocprofv3 FETCH_SIZE / WRITE_SIZE to bytes) and exit")
    args = ap.parse_args()
    if args.copy_calibration:
        import torch

        src = torch.empty(args.copy_calibration, dtype=torch.uint8, device="cuda").fill_(1)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        for _ in range(10):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_calibration_bytes": args.copy_calibration}), flush=True)
        return
    if args.gpus != 1:
        print(f"bench.py: measures one GPU only; --gpus {args.gpus} is not supported "
              f"(the kernels run on a single GPU; sharding across GPUs is not implemented)", file=sys.stderr)
        sys.exit(2)

    if args.workload not in ("decode", "layer"):
        out = {"stack": run_stack, "stack-layer": run_stack_layer, "single": run_single, "prefill": run_prefill, "int8": run_int8, "int8-prefill": run_int8_prefill,
               "gated": run_gated, "prune": run_prune, "train": run_train, "int4": run_int4}[args.workload](args)
        print(json.dumps(out), flush=True)
        return

    dtype = "bf16"
    batches = [int(b) for b in args.batches.split(",")]
    mmax = max(batches)
    t_gen = time.perf_counter()
    host = generate_layers(args.layers, dtype, args.sparsity, args.workers)

    import torch

    import paper_2405_03594_amd as spl

    spl.lib()
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    layers = upload_layers(host, dtype, keep_dense=not args.no_dense)
    del host
    xs = make_activations(dtype, mmax)
    xsl = {(M, j): xs[j][:M].contiguous() for M in batches for j in range(len(xs))}
    ys = {(M, j): torch.empty((M, N), dtype=torch.bfloat16, device="cuda")
          for M in batches for j, (_, N, _) in enumerate(synth.LLAMA2_7B_LINEARS)}
    t_gen = time.perf_counter() - t_gen
    print(f"# generated and packed {args.layers} layers in {t_gen:.1f} s", file=sys.stderr, flush=True)

    units = GROUPED if args.driver == "grouped" else SINGLE

    def sparse_fn(li, u, M):
        spl.sparse_linear_group([xsl[(M, j)] for j in u], [layers[li][j][0] for j in u],
                                outs=[ys[(M, j)] for j in u])

    def dense_fn(li, u, M):
        spl.dense_linear_group([xsl[(M, j)] for j in u], [layers[li][j][1] for j in u],
                               outs=[ys[(M, j)] for j in u])

    shapes = synth.LLAMA2_7B_LINEARS
    step_bytes = sum(algorithmic_bytes(layers[0][j][0], M, K, N) for M in batches for j, (_, N, K) in enumerate(shapes))
    launches = len(batches) * len(units)
    tokens_per_step = sum(batches)

    graphs = capture_graphs(layers, units, batches, sparse_fn)
    wall, step_ms = time_graphs(graphs, args.steps, args.warmup)
    ms_per_step = wall * 1e3 / args.steps
    gpu_step_ms = float(np.mean(step_ms))
    del graphs

    # roofline of the dominant kernel: mean algorithmic bytes per launch over its mean
    # launch duration = GPU time of the timed replays (events) / launches per step
    bytes_per_launch = step_bytes / launches
    launch_ms = gpu_step_ms / launches
    achieved = bytes_per_launch / (launch_ms * 1e-3) / 1e9

    # per batch size: one graph per layer and batch, sparse and dense, timed the same way
    per_batch = {}
    reps = max(20, args.steps // 4)
    for M in batches:
        g = capture_graphs(layers, units, [M], sparse_fn)
        _, ms = time_graphs(g, reps, 3)
        del g
        sp_us = float(np.mean(ms)) * 1e3
        b = sum(algorithmic_bytes(layers[0][j][0], M, K, N) for j, (_, N, K) in enumerate(shapes))
        d = {"layer_us": round(sp_us, 2), "tokens_per_s": round(M / (sp_us * 1e-6), 1),
             "hbm_gbs": round(b / (sp_us * 1e-6) / 1e9, 1)}
        if not args.no_dense:
            g = capture_graphs(layers, units, [M], dense_fn)
            _, ms = time_graphs(g, reps, 3)
            del g
            dn_us = float(np.mean(ms)) * 1e3
            db = sum(N * K * 2 + M * K * 2 + M * N * 2 for (_, N, K) in shapes)
            d.update({"dense_layer_us": round(dn_us, 2), "dense_hbm_gbs": round(db / (dn_us * 1e-6) / 1e9, 1),
                      "speedup_vs_dense": round(dn_us / sp_us, 3)})
        per_batch[str(M)] = d

    out = {
        "metric": METRIC,
        "value": round(tokens_per_step * args.steps / wall, 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {
            "workload": "Llama-2-7B decoder layer, 7 linears (q,k,v,o 4096x4096; gate,up 11008x4096; "
                        "down 4096x11008), bf16, 70% unstructured magnitude sparsity in bitmask format, "
                        f"decode batches {batches}",
            "batches": batches,
            "tokens_per_step": tokens_per_step,
            "layers_rotated": args.layers,
            "sparsity": args.sparsity,
            "graph_gpu_ms_per_step": round(gpu_step_ms, 4),
            "driver": args.driver,
            "launches_per_step": launches,
        },
        "roofline": {
            "bound": "hbm",
            "achieved": round(achieved, 1),
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": round(achieved / HBM_PEAK_GBS, 4),
            "traffic": None,                      # the committed counters cover the stack's launch mix
            "kernel": "k_sparse_decode",
            "bytes_per_launch": int(bytes_per_launch),
            "avg_launch_us": round(launch_ms * 1e3, 3),
        },
        "per_batch": per_batch,
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(dtype, args.sparsity, batches)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
