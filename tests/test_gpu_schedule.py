"""The calibration harness on the GPU path: per-layer alphas of a small
planted stack equal the ones the oracle's prediction gives with the same
exact truth (the masks are bit-exact), and the alpha sweep behaves."""

import numpy as np
import pytest
import torch

import oracle
import paper_2411_12692_amd as si
from paper_2411_12692_amd import schedule, synth

pytestmark = pytest.mark.gpu
DEV = "cuda"


def u16(t: torch.Tensor) -> np.ndarray:
    return t.detach().cpu().contiguous().view(torch.int16).numpy().view(np.uint16)


def test_calibrated_alphas_match_oracle():
    layers, xs, truths, ref_alphas = [], [], [], []
    for l in range(4):
        pl = synth.planted_layer(512, 1376, 0.9, config=6, layer=l, p_active=0.47, p_inactive=0.53)
        wg, x = u16(pl.w_gate), u16(pl.x)
        packed = oracle.pack_signs(wg)
        truth = oracle.gate_truly_positive(wg, x)

        def recall_at(a, packed=packed, x=x, truth=truth):
            mask, _, _ = oracle.predict_rows(packed, x, a)
            return schedule.quality(torch.from_numpy(mask.astype(bool)), torch.from_numpy(truth))["active_recall"]

        ref_alphas.append(schedule.calibrate(recall_at, 0.99))
        layers.append(si.MLPLayer(pl.w_gate.to(DEV), pl.w_up.to(DEV), pl.w_down.to(DEV)))
        xs.append(pl.x.to(DEV))
        truths.append(torch.from_numpy(truth).to(DEV))
    got = [schedule.calibrate_layer(l, [x], 0.99, positives=[t]) for l, x, t in zip(layers, xs, truths)]
    assert got == ref_alphas
    # the device truth (fp32 accumulation) agrees with the exact one away from 0
    for l, x, t in zip(layers, xs, truths):
        dev_truth = schedule.gate_positive(l.w_gate, x)
        g = (x.float() @ l.w_gate.float().t())
        differ = dev_truth != t
        assert bool((g[differ].abs() < 1e-5).all())


def test_sweep_is_monotone():
    layers, xs = [], []
    for l in range(3):
        pl = synth.planted_layer(512, 1376, 0.9, config=6, layer=l, device=DEV, p_active=0.47, p_inactive=0.53)
        layers.append(si.MLPLayer(pl.w_gate, pl.w_up, pl.w_down))
        xs.append(pl.x)
    rows = schedule.sweep(layers, xs, alphas=(0.9, 1.0, 1.05, 1.2, float("inf")), reps=2)
    kept = [r["kept_rows"] for r in rows]
    recall = [r["active_recall"] for r in rows]
    assert all(b >= a for a, b in zip(kept, kept[1:]))
    assert all(b >= a for a, b in zip(recall, recall[1:]))
    assert kept[-1] == 1376 and recall[-1] == 1.0
    assert all(r["us_per_layer"] > 0 for r in rows)
