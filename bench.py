"""Benchmark of the sparse linear hot path on one MI355X.

Default workload: one Llama-2-7B decoder layer's seven linear layers (q, k, v,
o: 4096x4096; gate, up: 11008x4096; down: 4096x11008) in bf16, weights
N(0, 0.02) magnitude-pruned to 70% per matrix and stored in the bitmask
expansion format, activations N(0, 1) at decode batch sizes 1, 4 and 16.

One step = the seven sparse linears at each of the three batch sizes (1 + 4 +
16 = 21 tokens) in the order of a decoder layer.  The layer driver launches
the independent projections together, as a decoder layer allows: q|k|v in one
grouped launch, o, gate|up in one grouped launch, then down (4 launches per
batch size, 12 per step; `--driver single` launches the seven separately).
Each step is one HIP graph; steps rotate over `--layers` distinct layers (8 by
default, 1.18 GB of compressed weights) so that the 256 MB Infinity Cache
cannot hold the weights between steps.  Inputs are resident in HBM before
timing starts.

Printed (one JSON line): tokens/s of the whole step, the roofline of the
dominant kernel (sparse decode: algorithmic bytes = stored values + bitmask +
tile offsets + X + Y per launch; its mean launch duration = GPU time of the
timed graph replays over launches per step), the same kernels run on dense
weights (per batch size), and
the CPU oracle timed on this host's cores on a bounded sample.
"""
from __future__ import annotations

import argparse
import concurrent.futures as cf
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


TRAFFIC_FILE = os.path.join(ROOT, "profiles", "k_sparse_decode_llama7b_layer_traffic.txt")
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
        print(f"bench.py: this build measures one GPU; --gpus {args.gpus} is not supported "
              f"(multi-GPU sharding is a design note only)", file=sys.stderr)
        sys.exit(2)

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
            "traffic": measured_traffic(),
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
