"""Benchmark of the SparseInfer decode MLP path on one MI355X.

One step = one pass of the whole per-token path over one layer: x-sign
packing, sign-bit prediction (Eq. (2)), compaction, sparse gate/up with
actual sparsity and sparse down-projection, for the 7B-shaped layer
(d = 4096, k = 11008) with planted sparsity s = 0.9, alpha = 1.0, batch 1.
``--mlp relu`` times the non-gated ReLU MLP (no W_up) of an OPT-6.7B-shaped
layer (d = 4096, k = 16384) instead, same sparsity and alpha.
Steps cycle through a pool of independently seeded layers whose weights
(>= 4.4 GB) exceed the 256 MB Infinity Cache, so every step reads its bytes
from HBM.  The timed loop is replayed from a HIP graph (the per-call host
cost of Python would otherwise dominate a ~10 us step).

Prints one JSON line.  ``value`` is the effective HBM bandwidth on the
algorithmic bytes of a step (packed signs + x + the kept rows of W_gate,
W_up and W_down^T + y), divided by the measured time per step.
"""

from __future__ import annotations

import argparse
import json
import math
import os
import platform
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "µs per MLP layer (predict+sparse GEMV) at 7B shape, s=0.9; effective HBM GB/s"
D, K, S = 4096, 11008, 0.9
HBM_PEAK_GBS = 8000.0
# the non-gated workload (--mlp relu): OPT-6.7B's MLP shape
RELU_METRIC = "µs per non-gated ReLU MLP layer (predict+sparse GEMV) at OPT-6.7B shape, s=0.9; effective HBM GB/s"
RELU_D, RELU_K = 4096, 16384


def algorithmic_bytes(k, d, b, n_gate, n_up, n_down):
    """Bytes the method itself must move for one layer and one step."""
    return k * d // 8 + 2 * d * b + 2 * d * (n_gate + n_up + n_down) + 4 * d * b


COUNTERS_FILE = os.path.join(ROOT, "profiles", "k_owned_7b_s0.9_counters.txt")
RELU_COUNTERS_FILE = os.path.join(ROOT, "profiles", "k_owned_opt6.7b_relu_s0.9_counters.txt")
KERNEL_SOURCES = ("paper_2411_12692_amd/csrc/owned.hip", "paper_2411_12692_amd/csrc/layer_common.h",
                  "paper_2411_12692_amd/csrc/si_device.h")


def kernel_sources_sha256():
    import hashlib

    h = hashlib.sha256()
    for rel in KERNEL_SOURCES:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def measured_traffic(counters_file=COUNTERS_FILE):
    """HBM bytes per k_owned launch from the committed FETCH_SIZE/WRITE_SIZE
    summary, or None when that summary was taken on other kernel sources."""
    try:
        with open(counters_file) as f:
            fields = dict(line.split(":", 1) for line in f if ":" in line and not line.startswith((" ", "#", "|")))
    except OSError:
        return None
    fields = {k.strip(): v.strip() for k, v in fields.items()}
    if fields.get("sources_sha256") != kernel_sources_sha256():
        return None
    try:
        return int(fields["traffic_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def parse():
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=4096)
    ap.add_argument("--warmup", type=int, default=256)
    ap.add_argument("--layers", type=int, default=16, help="size of the rotating layer pool")
    ap.add_argument("--alpha", type=float, default=1.0)
    ap.add_argument("--mlp", choices=("gated", "relu"), default="gated",
                    help="gated: the 7B-shaped gated MLP (default); relu: the non-gated ReLU MLP of an "
                         "OPT-6.7B-shaped layer")
    ap.add_argument("--cpu-seconds", type=float, default=12.0, help="budget of the CPU-oracle baseline")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--launches", type=int, default=256, help="individually timed launches for the roofline")
    ap.add_argument("--profile-pass", action="store_true",
                    help="for hardware-counter runs: eager layer calls over the pool, then one plain 256 MiB "
                         "device copy whose counters calibrate the byte counters; prints no JSON")
    return ap.parse_args()


def profile_pass(layers, xs, ys, alpha, calls):
    """Eager launches only (counter collection serialises dispatches), then a
    plain copy of known size: 256 MiB read + 256 MiB written."""
    import torch

    for i in range(calls):
        layers[i % len(layers)](xs[i % len(xs)], alpha, y=ys[i % len(ys)])
    torch.cuda.synchronize()
    src = torch.empty(128 << 20, dtype=torch.float16, device=xs[0].device).fill_(1.0)
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(4):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(f"# profile pass: {calls} layer calls, 4 copies of {src.numel() * 2} bytes", file=sys.stderr, flush=True)


def cpu_baseline(layers_host, alpha, budget_s, k=K, d=D):
    """Time the CPU oracle (test infrastructure, never tuned) on a bounded
    sample of the same workload: predict + masked MLP on the first layers of
    the pool, repeated until the budget is spent, with one BLAS thread
    (``wu is None``: the non-gated MLP)."""
    import numpy as np
    from threadpoolctl import threadpool_limits

    import oracle

    total_bytes, total_s, calls = 0.0, 0.0, 0
    with threadpool_limits(limits=1):
        while total_s < budget_s:
            for wg, wu, wd, x, packed in layers_host:
                t0 = time.perf_counter()
                mask, _, _ = oracle.predict_rows(packed, x, alpha)
                if wu is None:
                    out = oracle.relu_mlp(wg, wd, x, mask)
                else:
                    out = oracle.sparse_mlp(wg, wu, wd, x, mask)
                total_s += time.perf_counter() - t0
                calls += 1
                total_bytes += algorithmic_bytes(k, d, x.shape[0], out["n_gate"], out["n_up"], out["n_down"])
                if total_s >= budget_s:
                    break
    return {
        "value": round(total_bytes / total_s / 1e9, 3),
        "unit": "GB/s",
        "us_per_layer": round(total_s / calls * 1e6, 1),
        "cores": 1,
        "kind": "oracle",
        "sample": f"{calls} layer calls over the first {len(layers_host)} layers of the pool "
                  f"(predict_rows + {'relu_mlp' if layers_host[0][1] is None else 'sparse_mlp'}, "
                  f"numpy float64, 1 thread, {total_s:.1f} s)",
        "cpu": platform.processor() or platform.machine(),
    }


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU only: the SparseInfer MLP path is built and timed on a single "
              "MI355X (a k-split over several GPUs would add one all-reduce of y per layer, which is not "
              "built); run it with --gpus 1.", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import paper_2411_12692_amd as si
    from paper_2411_12692_amd import synth

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    si._lib.load()  # fails loudly if the library is not built

    relu = args.mlp == "relu"
    D_, K_ = (RELU_D, RELU_K) if relu else (D, K)
    L = args.layers
    layers, xs, host = [], [], []
    for l in range(L):
        # the non-gated layer takes the planted W_gate as its W_fc1
        pl = synth.planted_layer(D_, K_, S, config=7 if relu else 2, layer=l, device=dev)
        layers.append(si.MLPLayer(pl.w_gate, None if relu else pl.w_up, pl.w_down))
        xs.append(pl.x)
        if not args.no_cpu_baseline and l < 2:
            def u16(t):
                return t.cpu().contiguous().view(torch.int16).numpy().view(np.uint16)
            wg, wd, xh = u16(pl.w_gate), u16(pl.w_down), u16(pl.x)
            wu = None if relu else u16(pl.w_up)
            import oracle
            host.append((wg, wu, wd, xh, oracle.pack_signs(wg)))
        del pl
    torch.cuda.synchronize()
    print(f"# pool of {L} layers ready", file=sys.stderr, flush=True)

    # per-layer work counters (deterministic per layer) -> algorithmic bytes
    ys = [torch.empty(1, D_, dtype=torch.float32, device=dev) for _ in range(L)]
    counts = []
    for l in range(L):
        _, (_, _, _, c) = layers[l](xs[l], args.alpha, outputs=True, y=ys[l])
        counts.append(c)
    torch.cuda.synchronize()
    counts = [c.tolist() for c in counts]
    if args.profile_pass:
        profile_pass(layers, xs, ys, args.alpha, max(args.launches, L))
        return
    bytes_per_layer = [algorithmic_bytes(K_, D_, 1, *c) for c in counts]
    mean_bytes = sum(bytes_per_layer) / L

    # graph of one pass over the pool, replayed
    stream = torch.cuda.Stream()
    per_graph = L * max(1, 64 // L)
    with torch.cuda.stream(stream):
        for i in range(per_graph):  # warm the path on the capture stream
            layers[i % L](xs[i % L], args.alpha, y=ys[i % L])
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=stream):
        for i in range(per_graph):
            layers[i % L](xs[i % L], args.alpha, y=ys[i % L])
    torch.cuda.synchronize()
    reps = max(1, math.ceil(args.steps / per_graph))
    wreps = max(1, math.ceil(args.warmup / per_graph))
    steps, warmup = reps * per_graph, wreps * per_graph
    for _ in range(wreps):
        graph.replay()
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    e0.record(stream)
    with torch.cuda.stream(stream):
        for _ in range(reps):
            graph.replay()
    e1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    gpu_ms = e0.elapsed_time(e1)
    us_per_layer = gpu_ms * 1e3 / steps
    print(f"# timed {steps} steps: {us_per_layer:.3f} us/layer (wall {wall * 1e6 / steps:.3f})",
          file=sys.stderr, flush=True)

    # The timed graph holds nothing but k_owned launches on `stream`, so the
    # per-step time above is that kernel's average launch duration.
    achieved = mean_bytes / us_per_layer / 1e3

    # For reference: individually timed launches (events around each call,
    # queued behind a spin kernel so that host enqueue time stays out).
    M = args.launches
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(M)]
    with torch.cuda.stream(stream):
        torch.cuda._sleep(int(2.4e9 * 0.02 * max(1, M / 256)))
        for i in range(M):
            a, b = evs[i]
            a.record(stream)
            layers[i % L](xs[i % L], args.alpha, y=ys[i % L])
            b.record(stream)
    torch.cuda.synchronize()
    isolated_us = sum(a.elapsed_time(b) * 1e3 for a, b in evs) / M

    result = {
        "metric": RELU_METRIC if relu else METRIC,
        "value": round(mean_bytes / us_per_layer / 1e3, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": steps,
        "warmup": warmup,
        "ms_per_step": round(us_per_layer / 1e3, 6),
        "us_per_layer": round(us_per_layer, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f16",
        "accumulate": "f32",
        "data": "synthetic",
        "config": {
            "workload": (f"OPT-6.7B-shaped non-gated ReLU MLP layer (no W_up) d={D_} k={K_}" if relu else
                         f"7B-shaped ReLU gated MLP layer d={D_} k={K_}") +
                        f", planted sparsity s={S}, alpha={args.alpha}, batch 1, rotating pool of {L} layers, "
                        f"HIP-graph replay",
            "d": D_, "k": K_, "batch": 1, "alpha": args.alpha, "layers_in_pool": L,
            "kept_rows": [c[0] for c in counts[:4]],
            "bytes_per_layer": int(mean_bytes),
        },
        "roofline": {
            "kernel": "k_owned (predict + group exchange + gate/up + down, one launch per layer)",
            "bound": "hbm",
            "achieved": round(achieved, 1),
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": round(achieved / HBM_PEAK_GBS, 4),
            "traffic": measured_traffic(RELU_COUNTERS_FILE if relu else COUNTERS_FILE),
            "launch_us": round(us_per_layer, 3),
            "isolated_launch_us": round(isolated_us, 3),
        },
    }
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(host, args.alpha, args.cpu_seconds, K_, D_)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
