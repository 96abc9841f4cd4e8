"""Per-layer conservativeness (alpha) schedules and their calibration.

Eq. (2) keeps a row unless ``alpha * N_pos < N_neg``; a larger alpha keeps
more rows (higher recall of the truly active rows, less sparsity, more
bytes).  The paper sets alpha slightly above 1 on the early layers, where a
missed active row costs the most accuracy (Section V), chooses the values by
test runs, and treats alpha as the knob of a design-space exploration
between time and accuracy.  This module provides that harness around the
per-call alpha of the library:

* :func:`early_layer_schedule` - alpha above 1 on the first layers only;
* :func:`calibrate` / :func:`calibrate_layer` / :func:`calibrate_stack` -
  per layer, the smallest alpha of a grid whose active-row recall over
  calibration tokens reaches a target;
* :func:`sweep` - per alpha: time per layer, recall and kept rows (the
  design-space exploration).

Predictions come from the library (``si_predict``); the truth (which gate
rows are positive) comes from a dense gate product on the device in fp32,
which is harness work, not part of the per-token path.
"""

from __future__ import annotations

import math
from typing import Callable, Iterable, List, Optional, Sequence

import torch

# alpha values tried by default (float32-exact decisions, Eq. (2))
DEFAULT_ALPHAS = (0.9, 0.95, 1.0, 1.01, 1.02, 1.03, 1.05, 1.1, 1.2, 1.35, 1.5)


def early_layer_schedule(n_layers: int, alpha: float = 1.0, early_alpha: float = 1.02,
                         early_layers: int = 20) -> List[float]:
    """``early_alpha`` on the first ``early_layers`` layers, ``alpha`` on the
    rest (the schedule shape of Section V: more conservative early layers)."""
    if n_layers < 0 or early_layers < 0:
        raise ValueError("layer counts must be >= 0")
    return [float(early_alpha) if l < early_layers else float(alpha) for l in range(n_layers)]


def gate_positive(w_gate: torch.Tensor, x: torch.Tensor) -> torch.Tensor:
    """``[b][k]`` bool: which gate pre-activations ``W_gate x_t`` are
    positive (fp32 accumulation of the fp16 products on the device)."""
    x2 = x.reshape(-1, w_gate.shape[1]).float()
    return (x2 @ w_gate.float().t()) > 0


def quality(kept: torch.Tensor, positive: torch.Tensor) -> dict:
    """Prediction quality of a kept mask ``[k]`` against the truly positive
    rows ``[b][k]`` of a batch (a row is needed if any token's gate value is
    positive).  ``active_recall`` = needed rows kept / needed rows;
    ``sparse_precision`` / ``sparse_recall`` are the paper's precision and
    recall of the predicted-sparse class (Section IV-A)."""
    kept = kept.reshape(-1).bool()
    needed = positive.reshape(-1, kept.numel()).any(dim=0)
    n_needed = int(needed.sum())
    n_kept_needed = int((kept & needed).sum())
    pred_sparse = ~kept
    truly_zero = ~needed
    ps = int(pred_sparse.sum())
    tz = int(truly_zero.sum())
    both = int((pred_sparse & truly_zero).sum())
    return {
        "active_recall": n_kept_needed / n_needed if n_needed else 1.0,
        "missed": n_needed - n_kept_needed,
        "kept": int(kept.sum()),
        "needed": n_needed,
        "sparse_precision": both / ps if ps else 1.0,
        "sparse_recall": both / tz if tz else 1.0,
    }


def calibrate(recall_at: Callable[[float], float], target: float,
              alphas: Sequence[float] = DEFAULT_ALPHAS) -> float:
    """Smallest alpha of ``alphas`` whose recall reaches ``target``
    (``recall_at(alpha)``), or ``+inf`` (keep every row) if none does.
    Recall does not decrease with alpha (the kept set only grows), so the
    grid is walked upwards and stops at the first hit."""
    if not 0.0 <= target <= 1.0:
        raise ValueError("target recall must be in [0, 1]")
    for a in sorted(float(v) for v in alphas):
        if recall_at(a) >= target:
            return a
    return math.inf


def _layer_recall_fn(layer, xs: Sequence[torch.Tensor], positives: Sequence[torch.Tensor]):
    def recall_at(alpha: float) -> float:
        needed = kept_needed = 0
        for x, pos in zip(xs, positives):
            mask, _, _ = layer.predict(x, alpha)
            q = quality(mask.bool(), pos)
            needed += q["needed"]
            kept_needed += q["needed"] - q["missed"]
        return kept_needed / needed if needed else 1.0
    return recall_at


def calibrate_layer(layer, xs: Sequence[torch.Tensor], target: float,
                    alphas: Sequence[float] = DEFAULT_ALPHAS,
                    positives: Optional[Sequence[torch.Tensor]] = None) -> float:
    """Calibrate one :class:`MLPLayer` on the token batches ``xs``
    (each ``[b][d]`` fp16 on the device): the smallest alpha whose
    active-row recall, pooled over the batches, reaches ``target``.
    ``positives`` overrides the truth (``[b][k]`` bool per batch)."""
    if positives is None:
        positives = [gate_positive(layer.w_gate, x) for x in xs]
    return calibrate(_layer_recall_fn(layer, xs, positives), target, alphas)


def calibrate_stack(layers, xs_per_layer: Sequence[Sequence[torch.Tensor]], target: float,
                    alphas: Sequence[float] = DEFAULT_ALPHAS) -> List[float]:
    """Per-layer alphas of a stack (one calibration per layer)."""
    return [calibrate_layer(layer, xs, target, alphas) for layer, xs in zip(layers, xs_per_layer)]


def _graph_time_us(fns: Sequence[Callable[[], None]], reps: int) -> float:
    stream = torch.cuda.Stream()
    with torch.cuda.stream(stream):
        for f in fns:
            f()
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=stream):
        for f in fns:
            f()
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    with torch.cuda.stream(stream):
        for _ in range(reps):
            graph.replay()
    e1.record(stream)
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) * 1e3 / (reps * len(fns))


def sweep(layers, xs: Sequence[torch.Tensor], alphas: Iterable[float] = DEFAULT_ALPHAS,
          reps: int = 8, positives: Optional[Sequence[torch.Tensor]] = None) -> List[dict]:
    """Design-space exploration over alpha: per alpha, the time per fused
    layer call (HIP-graph replay over the layers, one token batch each), the
    pooled active-row recall, the kept rows per layer and the paper's
    precision / recall of the sparse class."""
    if positives is None:
        positives = [gate_positive(l.w_gate, x) for l, x in zip(layers, xs)]
    out = []
    for a in alphas:
        a = float(a)
        ys = [torch.empty(x.reshape(-1, l.d).shape[0], l.d, dtype=torch.float32, device=x.device)
              for l, x in zip(layers, xs)]
        fns = [(lambda l=l, x=x, y=y: l(x, a, y=y)) for l, x, y in zip(layers, xs, ys)]
        us = _graph_time_us(fns, reps)
        qs = [quality(l.predict(x, a)[0].bool(), p) for l, x, p in zip(layers, xs, positives)]
        needed = sum(q["needed"] for q in qs)
        kept_needed = sum(q["needed"] - q["missed"] for q in qs)
        out.append({
            "alpha": a,
            "us_per_layer": us,
            "active_recall": kept_needed / needed if needed else 1.0,
            "kept_rows": sum(q["kept"] for q in qs) / len(qs),
            "sparse_precision": sum(q["sparse_precision"] for q in qs) / len(qs),
            "sparse_recall": sum(q["sparse_recall"] for q in qs) / len(qs),
        })
    return out


def main(argv=None) -> None:
    """``python -m paper_2411_12692_amd.schedule``: alpha sweep on planted
    7B-shaped layers whose prediction is uncertain (disagreement 0.47 on
    active rows, 0.53 on inactive rows, s = 0.9), plus a calibration of
    every layer to 99% active recall."""
    import argparse
    import json

    from . import MLPLayer, synth

    ap = argparse.ArgumentParser(description=main.__doc__.splitlines()[0])
    ap.add_argument("--d", type=int, default=4096)
    ap.add_argument("--k", type=int, default=11008)
    ap.add_argument("--layers", type=int, default=16)
    ap.add_argument("--p-active", type=float, default=0.47)
    ap.add_argument("--p-inactive", type=float, default=0.53)
    ap.add_argument("--target", type=float, default=0.99)
    args = ap.parse_args(argv)
    dev = torch.device("cuda:0")
    layers, xs = [], []
    for l in range(args.layers):
        pl = synth.planted_layer(args.d, args.k, 0.9, config=6, layer=l, device=dev,
                                 p_active=args.p_active, p_inactive=args.p_inactive)
        layers.append(MLPLayer(pl.w_gate, pl.w_up, pl.w_down))
        xs.append(pl.x)
    for row in sweep(layers, xs):
        print(json.dumps({k: (round(v, 4) if isinstance(v, float) else v) for k, v in row.items()}), flush=True)
    alphas = calibrate_stack(layers, [[x] for x in xs], args.target)
    print(json.dumps({"target_recall": args.target, "calibrated_alphas": alphas}), flush=True)


if __name__ == "__main__":
    main()
