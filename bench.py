"""Benchmark of the SparseInfer decode MLP path on one MI355X.

One step = one pass of the whole per-token path over one layer: x-sign
packing, sign-bit prediction (Eq. (2)), compaction, sparse gate/up with
actual sparsity and sparse down-projection, for the 7B-shaped layer
(d = 4096, k = 11008) with planted sparsity s = 0.9, alpha = 1.0, batch 1.
``--mlp relu`` times the non-gated ReLU MLP (no W_up) of an OPT-6.7B-shaped
layer (d = 4096, k = 16384) instead, same sparsity and alpha; ``--mlp block``
times the 7B layer as a decoder-block call (RMSNorm of the fp32 residual
stream and the residual add fused around the path) and, for comparison, the
plain call on the same layers; ``--mlp int8`` times the 7B layer with INT8
weights (symmetric, one scale per output channel, quantized on the device at
load; the predictor reads the MSBs of the INT8 W_gate).
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
INT8_METRIC = "µs per MLP layer with INT8 weights (predict+sparse GEMV) at 7B shape, s=0.9; effective HBM GB/s"
BLOCK_METRIC = ("µs per decoder-block MLP call (RMSNorm + predict + sparse GEMV + residual) at 7B shape, s=0.9; "
                "effective HBM GB/s")


def algorithmic_bytes(k, d, b, n_gate, n_up, n_down, block=False, int8=False):
    """Bytes the method itself must move for one layer and one step (the
    decoder-block call reads the fp32 residual stream and the norm weight
    instead of the fp16 x; INT8 rows are d bytes, plus the float scales of
    the kept W_gate / W_up rows and the d scales of the columns of y)."""
    x_bytes = 4 * d * b + 4 * d if block else 2 * d * b
    if int8:
        return k * d // 8 + x_bytes + d * (n_gate + n_up + n_down) + 4 * (n_gate + n_up) + 4 * d + 4 * d * b
    return k * d // 8 + x_bytes + 2 * d * (n_gate + n_up + n_down) + 4 * d * b


COUNTERS_FILE = os.path.join(ROOT, "profiles", "k_owned_7b_s0.9_counters.txt")
RELU_COUNTERS_FILE = os.path.join(ROOT, "profiles", "k_owned_opt6.7b_relu_s0.9_counters.txt")
INT8_COUNTERS_FILE = os.path.join(ROOT, "profiles", "k_owned_7b_int8_s0.9_counters.txt")
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
    ap.add_argument("--mlp", choices=("gated", "relu", "block", "int8"), default="gated",
                    help="gated: the 7B-shaped gated MLP (default); relu: the non-gated ReLU MLP of an "
                         "OPT-6.7B-shaped layer; block: the 7B layer with RMSNorm and residual fused; int8: the "
                         "7B layer with INT8 weights")
    ap.add_argument("--cpu-seconds", type=float, default=12.0, help="budget of the CPU-oracle baseline")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--launches", type=int, default=256, help="individually timed launches for the roofline")
    ap.add_argument("--profile-pass", action="store_true",
                    help="for hardware-counter runs: eager layer calls over the pool, then one plain 256 MiB "
                         "device copy whose counters calibrate the byte counters; prints no JSON")
    return ap.parse_args()


def profile_pass(step, n_layers, calls, dev):
    """Eager launches only (counter collection serialises dispatches), then a
    plain copy of known size: 256 MiB read + 256 MiB written."""
    import torch

    for i in range(calls):
        step(i)
    torch.cuda.synchronize()
    src = torch.empty(128 << 20, dtype=torch.float16, device=dev).fill_(1.0)
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(4):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(f"# profile pass: {calls} layer calls, 4 copies of {src.numel() * 2} bytes", file=sys.stderr, flush=True)


def cpu_baseline(layers_host, alpha, budget_s, k=K, d=D, block=None, int8=False):
    """Time the CPU oracle (test infrastructure, never tuned) on a bounded
    sample of the same workload: predict + masked MLP on the first layers of
    the pool, repeated until the budget is spent, with one BLAS thread
    (``wu is None``: the non-gated MLP; ``block`` = per-layer ``(h, norm_w,
    eps)``: the decoder-block form, RMSNorm and residual included; ``int8``:
    the entries hold the oracle's INT8 weights and scales, quantized beforehand,
    untimed, as at load)."""
    from threadpoolctl import threadpool_limits

    import oracle

    total_bytes, total_s, calls = 0.0, 0.0, 0
    with threadpool_limits(limits=1):
        while total_s < budget_s:
            for li, (wg, wu, wd, x, packed) in enumerate(layers_host):
                t0 = time.perf_counter()
                if int8:
                    mask, _, _ = oracle.predict_rows(packed, x, alpha)
                    (qg, sg), (qu, su), (qd, sd) = wg, wu, wd
                    out = oracle.int8_mlp(qg, sg, qu, su, qd, sd, x, mask)
                elif block is not None:
                    h, nw, eps = block[li]
                    out = oracle.mlp_block(h, nw, eps, packed, wg, wu, wd, alpha)
                else:
                    mask, _, _ = oracle.predict_rows(packed, x, alpha)
                    if wu is None:
                        out = oracle.relu_mlp(wg, wd, x, mask)
                    else:
                        out = oracle.sparse_mlp(wg, wu, wd, x, mask)
                total_s += time.perf_counter() - t0
                calls += 1
                total_bytes += algorithmic_bytes(k, d, x.shape[0], out["n_gate"], out["n_up"], out["n_down"],
                                                 block=block is not None, int8=int8)
                if total_s >= budget_s:
                    break
    what = ("rmsnorm_fp16 + predict_rows + sparse_mlp + residual" if block is not None else
            "predict_rows on pack_signs_int8 + int8_mlp" if int8 else
            f"predict_rows + {'relu_mlp' if layers_host[0][1] is None else 'sparse_mlp'}")
    return {
        "value": round(total_bytes / total_s / 1e9, 3),
        "unit": "GB/s",
        "us_per_layer": round(total_s / calls * 1e6, 1),
        "cores": 1,
        "kind": "oracle",
        "sample": f"{calls} layer calls over the first {len(layers_host)} layers of the pool "
                  f"({what}, numpy float64, 1 thread, {total_s:.1f} s)",
        "cpu": platform.processor() or platform.machine(),
    }


def time_graph(step, n_layers, steps_wanted, warmup_wanted):
    """Replay a HIP graph of back-to-back steps (one pass over the layer pool
    or more) and return (us per step, steps, warm-up steps, wall us per
    step); events on the replay stream bracket the timed replays."""
    import torch

    stream = torch.cuda.Stream()
    per_graph = n_layers * max(1, 64 // n_layers)
    with torch.cuda.stream(stream):
        for i in range(per_graph):  # warm the path on the capture stream
            step(i)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=stream):
        for i in range(per_graph):
            step(i)
    torch.cuda.synchronize()
    reps = max(1, math.ceil(steps_wanted / per_graph))
    wreps = max(1, math.ceil(warmup_wanted / per_graph))
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
    return e0.elapsed_time(e1) * 1e3 / steps, steps, warmup, wall * 1e6 / steps


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
    block = args.mlp == "block"
    int8 = args.mlp == "int8"
    D_, K_ = (RELU_D, RELU_K) if relu else (D, K)
    EPS = 1e-5
    L = args.layers
    layers, xs, hs, nws, host, host_block = [], [], [], [], [], []
    for l in range(L):
        # the non-gated layer takes the planted W_gate as its W_fc1
        pl = synth.planted_layer(D_, K_, S, config=7 if relu else 2, layer=l, device=dev)
        if int8:  # quantized on the device, as at load
            layers.append(si.Int8MLPLayer(pl.w_gate, pl.w_up, pl.w_down))
        else:
            layers.append(si.MLPLayer(pl.w_gate, None if relu else pl.w_up, pl.w_down))
        xs.append(pl.x)
        if block:
            # residual stream with the planted token's signs, positive norm weight
            hs.append(pl.x.float() * 3.0)
            g = torch.Generator(device="cpu").manual_seed(1000 + l)
            nws.append((0.5 + torch.rand(D_, generator=g)).to(dev))
        if not args.no_cpu_baseline and l < 2:
            def u16(t):
                return t.cpu().contiguous().view(torch.int16).numpy().view(np.uint16)
            wg, wd, xh = u16(pl.w_gate), u16(pl.w_down), u16(pl.x)
            wu = None if relu else u16(pl.w_up)
            import oracle
            if int8:
                qg = oracle.quantize_rows_int8(wg)
                host.append((qg, oracle.quantize_rows_int8(wu), oracle.quantize_rows_int8(wd), xh,
                             oracle.pack_signs_int8(qg[0])))
            else:
                host.append((wg, wu, wd, xh, oracle.pack_signs(wg)))
            if block:
                host_block.append((hs[-1].cpu().numpy(), nws[-1].cpu().numpy(), EPS))
        del pl
    torch.cuda.synchronize()
    print(f"# pool of {L} layers ready", file=sys.stderr, flush=True)

    ys = [torch.empty(1, D_, dtype=torch.float32, device=dev) for _ in range(L)]

    def step(i, outputs=False):
        l = i % L
        if block:
            return layers[l].block(hs[l], nws[l], EPS, args.alpha, outputs=outputs, y=ys[l])
        return layers[l](xs[l], args.alpha, outputs=outputs, y=ys[l])

    # per-layer work counters (deterministic per layer) -> algorithmic bytes
    counts = []
    for l in range(L):
        _, (_, _, _, c) = step(l, outputs=True)
        counts.append(c)
    torch.cuda.synchronize()
    counts = [c.tolist() for c in counts]
    if args.profile_pass:
        profile_pass(step, L, max(args.launches, L), dev)
        return
    bytes_per_layer = [algorithmic_bytes(K_, D_, 1, *c, block=block, int8=int8) for c in counts]
    mean_bytes = sum(bytes_per_layer) / L

    us_per_layer, steps, warmup, wall_us = time_graph(step, L, args.steps, args.warmup)
    print(f"# timed {steps} steps: {us_per_layer:.3f} us/layer (wall {wall_us:.3f})", file=sys.stderr, flush=True)
    plain_us = None
    if block:  # the same layers through the plain call (x given, no residual), for comparison
        plain_us, _, _, _ = time_graph(lambda i: layers[i % L](xs[i % L], args.alpha, y=ys[i % L]), L,
                                       args.steps, args.warmup)
        print(f"# plain call on the same layers: {plain_us:.3f} us/layer", file=sys.stderr, flush=True)

    # The timed graph holds nothing but k_owned launches on one stream, so the
    # per-step time above is that kernel's average launch duration.
    achieved = mean_bytes / us_per_layer / 1e3

    # For reference: individually timed launches (events around each call,
    # queued behind a spin kernel so that host enqueue time stays out).
    M = args.launches
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(M)]
    stream = torch.cuda.Stream()
    with torch.cuda.stream(stream):
        torch.cuda._sleep(int(2.4e9 * 0.02 * max(1, M / 256)))
        for i in range(M):
            a, b = evs[i]
            a.record(stream)
            step(i)
            b.record(stream)
    torch.cuda.synchronize()
    isolated_us = sum(a.elapsed_time(b) * 1e3 for a, b in evs) / M

    result = {
        "metric": RELU_METRIC if relu else BLOCK_METRIC if block else INT8_METRIC if int8 else METRIC,
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
        "dtype": "i8" if int8 else "f16",
        "accumulate": "f32",
        "data": "synthetic",
        "config": {
            "workload": (f"OPT-6.7B-shaped non-gated ReLU MLP layer (no W_up) d={D_} k={K_}" if relu else
                         f"7B-shaped ReLU gated MLP layer d={D_} k={K_} as a decoder-block call (RMSNorm of the "
                         f"fp32 residual stream, eps={EPS}, and the residual add fused)" if block else
                         f"7B-shaped ReLU gated MLP layer d={D_} k={K_} with INT8 weights (symmetric, one float "
                         f"scale per output channel, quantized on the device; fp16 x, fp32 accumulation)" if int8 else
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
            "traffic": None if block else measured_traffic(RELU_COUNTERS_FILE if relu else
                                                           INT8_COUNTERS_FILE if int8 else COUNTERS_FILE),
            "launch_us": round(us_per_layer, 3),
            "isolated_launch_us": round(isolated_us, 3),
        },
    }
    if plain_us is not None:
        result["plain_call_us"] = round(plain_us, 3)
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(host, args.alpha, args.cpu_seconds, K_, D_,
                                              block=host_block if block else None, int8=int8)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
