"""Phase timeline of the row-owning kernel (``k_owned``) on the benchmark's
workloads, from the trace build of the library.

Build it first with ``python -m paper_2411_12692_amd.build --trace`` (the
kernel compiled with ``-DSI_TRACE``, as ``libsparseinfer_trace.so``): every
block then stamps the 100 MHz real-time counter at numbered points of the
kernel, and every wave at points of its own, in LDS, written out once at the
kernel's end so that no store is in flight while it runs.  For the last
launch of each graph replay this prints, per point, the median, p10, p90
and maximum over blocks (or waves) of the time since the earliest block
started, each the median over several replays.

Usage: ``python -m paper_2411_12692_amd.phase_trace [--batch B] [--int8] [--shape 7b|13b] [--replays N]``

Workloads: one token: the fused call (predict + MLP) on 16 planted 7B-shaped
layers (d = 4096, k = 11008, s = 0.9, alpha = 1), as ``bench.py`` times it
(``--int8``: the same layers quantized to INT8, ``bench.py --mlp int8``;
``--shape 13b``: 13B-shaped layers, d = 5120, k = 13824, s = 0.88,
``bench.py --shape 13b``); B tokens: the mask call over the union of the
tokens' planted active sets of 8 7B-shaped layers (``bench.py --batch B``).
"""

from __future__ import annotations

import argparse
import ctypes
import os

import numpy as np

BLOCK_MARKS = {
    0: "block start",
    1: "tokens staged, x signs formed",
    2: "first popcount pass done",
    3: "own kept rows published",
    4: "group list formed",
    6: "wave 0's gate/up rows done",
    8: "down tile folded",
    9: "tile's zero flag seen",
    10: "block end (y atomics issued)",
}
WAVE_MARKS = {
    0: "last gate/up row requested",
    1: "gate/up rows done",
    2: "down started",
    3: "first down round/chunk: h3 in",
    4: "first down round/chunk done",
    5: "down rounds/chunks done",
}
SLOTS, WAVE_SLOTS, MAX_BLOCKS = 32, 8, 1024


def main() -> None:
    ap = argparse.ArgumentParser()
    ap.add_argument("--batch", type=int, default=1)
    ap.add_argument("--replays", type=int, default=8)
    ap.add_argument("--int8", action="store_true", help="INT8 weights (one token)")
    ap.add_argument("--shape", choices=("7b", "13b"), default="7b", help="layer shape (one token)")
    args = ap.parse_args()
    if args.shape != "7b" and args.batch != 1:
        raise SystemExit("--shape 13b is a one-token workload")

    import torch

    from . import _lib, build, synth

    if not os.path.exists(build.TRACE_LIB):
        raise SystemExit(f"{build.TRACE_LIB} is missing: run python -m paper_2411_12692_amd.build --trace")
    _lib.LIB_PATH = build.TRACE_LIB
    lib = _lib.load()
    import paper_2411_12692_amd as si

    dev = torch.device("cuda:0")
    D, K, S, cfg = (5120, 13824, 0.88, 4) if args.shape == "13b" else (4096, 11008, 0.9, 2)
    b = args.batch
    L = 16 if b == 1 else 8
    if b == 1:
        pls = [synth.planted_layer(D, K, S, config=cfg, layer=l, device=dev) for l in range(L)]
        if args.int8:
            layers = [si.Int8MLPLayer(p.w_gate, p.w_up, p.w_down) for p in pls]
        else:
            layers = [si.MLPLayer(p.w_gate, p.w_up, p.w_down) for p in pls]
        xs = [p.x for p in pls]
        y = torch.empty(1, D, dtype=torch.float32, device=dev)

        def call(i):
            layers[i % L](xs[i % L], 1.0, y=y)
        what = (f"fused call, {args.shape.upper()} layer (d={D}, k={K}){', INT8 weights' if args.int8 else ''}, "
                f"planted s={S}, alpha=1, 1 token, pool of {L} layers")
    else:
        pls = [synth.planted_layer(D, K, 0.9, config=5, layer=l, device=dev) for l in range(L)]
        layers = [si.MLPLayer(p.w_gate, p.w_up, p.w_down, max_batch=b) for p in pls]
        xs = [synth.batch_tokens(p, b, config=5, layer_id=l) for l, p in enumerate(pls)]
        ms = [synth.batch_union_mask(p, b, config=5, layer_id=l) for l, p in enumerate(pls)]

        def call(i):
            layers[i % L].sparse_mlp(xs[i % L], mask=ms[i % L])
        what = (f"mask call over the union of {b} tokens' planted active sets, 7B layer (d={D}, k={K}), s=0.9, "
                f"pool of {L} layers")

    stream = torch.cuda.Stream()
    n_calls = 2 * L
    with torch.cuda.stream(stream):
        for i in range(n_calls):
            call(i)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=stream):
        for i in range(n_calls):
            call(i)
    torch.cuda.synchronize()
    blocks, waves = [], []
    P = torch.cuda.get_device_properties(0).multi_processor_count
    for _ in range(args.replays):
        with torch.cuda.stream(stream):
            graph.replay()
        torch.cuda.synchronize()
        bt = np.zeros(MAX_BLOCKS * SLOTS, dtype=np.uint64)
        wt = np.zeros(MAX_BLOCKS * 16 * WAVE_SLOTS, dtype=np.uint64)
        if lib.si_trace_read(bt.ctypes.data_as(ctypes.c_void_p), ctypes.c_size_t(bt.nbytes)) != 0:
            raise SystemExit("si_trace_read failed")
        if lib.si_trace_wave_read(wt.ctypes.data_as(ctypes.c_void_p), ctypes.c_size_t(wt.nbytes)) != 0:
            raise SystemExit("si_trace_wave_read failed")
        t = bt[: P * SLOTS].reshape(P, SLOTS).astype(np.int64)
        w = wt[: P * 16 * WAVE_SLOTS].reshape(P, 16, WAVE_SLOTS)[:, :8, :].astype(np.int64)
        t0 = t[:, 0].min()
        blocks.append(np.where(t > 0, (t - t0) / 100.0, np.nan))
        waves.append(np.where(w > 0, (w - t0) / 100.0, np.nan))
    with np.errstate(all="ignore"):
        import warnings

        warnings.simplefilter("ignore")
        rel = np.nanmedian(np.stack(blocks), axis=0)
        wrel = np.nanmedian(np.stack(waves), axis=0)
    print(f"# k_owned phase trace: {what}; {P} blocks; us since the earliest block start, "
          f"median over {args.replays} graph replays of the last launch")
    print(f"{'point':40s} {'median':>8s} {'p10':>8s} {'p90':>8s} {'max':>8s} {'n':>6s}")
    for s, name in BLOCK_MARKS.items():
        c = rel[:, s]
        c = c[~np.isnan(c)]
        if c.size:
            print(f"{'block: ' + name:40s} {np.median(c):8.2f} {np.percentile(c, 10):8.2f} "
                  f"{np.percentile(c, 90):8.2f} {c.max():8.2f} {c.size:6d}")
    for s, name in WAVE_MARKS.items():
        c = wrel[:, :, s].ravel()
        c = c[~np.isnan(c)]
        if c.size:
            print(f"{'wave: ' + name:40s} {np.median(c):8.2f} {np.percentile(c, 10):8.2f} "
                  f"{np.percentile(c, 90):8.2f} {c.max():8.2f} {c.size:6d}")
    for s in (1, 5):
        med = [np.nanmedian(wrel[:, wv, s]) if np.any(~np.isnan(wrel[:, wv, s])) else float("nan") for wv in range(8)]
        print(f"wave index 0-7, {WAVE_MARKS[s]}: " + " ".join(f"{m:6.2f}" for m in med))


if __name__ == "__main__":
    main()
