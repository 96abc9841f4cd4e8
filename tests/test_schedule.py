"""The alpha schedule / calibration harness (host logic), checked against
the oracle's prediction and exact truth on small planted layers."""

import math

import numpy as np
import pytest
import torch

import oracle
from paper_2411_12692_amd import schedule, synth


def u16(t: torch.Tensor) -> np.ndarray:
    return t.detach().cpu().contiguous().view(torch.int16).numpy().view(np.uint16)


def test_early_layer_schedule():
    s = schedule.early_layer_schedule(32, alpha=1.0, early_alpha=1.02, early_layers=20)
    assert s == [1.02] * 20 + [1.0] * 12
    assert schedule.early_layer_schedule(5, early_layers=20) == [1.02] * 5
    assert schedule.early_layer_schedule(0) == []
    with pytest.raises(ValueError):
        schedule.early_layer_schedule(-1)


def test_quality_hand_example():
    # 6 rows; truth (any token positive): rows 0, 1, 2; kept: rows 0, 2, 4
    positive = torch.tensor([[1, 0, 0, 0, 0, 0], [0, 1, 1, 0, 0, 0]], dtype=torch.bool)
    kept = torch.tensor([1, 0, 1, 0, 1, 0], dtype=torch.bool)
    q = schedule.quality(kept, positive)
    assert q["needed"] == 3 and q["kept"] == 3 and q["missed"] == 1
    assert q["active_recall"] == pytest.approx(2 / 3)
    # predicted sparse: rows 1, 3, 5; truly zero: rows 3, 4, 5
    assert q["sparse_precision"] == pytest.approx(2 / 3)
    assert q["sparse_recall"] == pytest.approx(2 / 3)


def test_quality_matches_oracle_single_token():
    pl = synth.planted_layer(512, 1376, 0.9, config=6, layer=0, p_active=0.47, p_inactive=0.53)
    wg, x = u16(pl.w_gate), u16(pl.x)
    packed = oracle.pack_signs(wg)
    truth = oracle.gate_truly_positive(wg, x)
    for alpha in (0.95, 1.0, 1.05):
        mask, active, _ = oracle.predict_rows(packed, x, alpha)
        q = schedule.quality(torch.from_numpy(mask.astype(bool)), torch.from_numpy(truth))
        r = oracle.prediction_quality(active, truth)
        assert q["missed"] == r["missed"]
        assert q["active_recall"] == pytest.approx(r["active_recall"])
        assert q["sparse_precision"] == pytest.approx(r["precision"])
        assert q["sparse_recall"] == pytest.approx(r["recall"])


def test_calibrate_smallest_alpha_on_grid():
    grid = (0.9, 1.0, 1.02, 1.05, 1.1)
    recall = {0.9: 0.90, 1.0: 0.97, 1.02: 0.99, 1.05: 0.995, 1.1: 1.0}
    calls = []

    def recall_at(a):
        calls.append(a)
        return recall[a]

    assert schedule.calibrate(recall_at, 0.99, grid) == 1.02
    assert calls == [0.9, 1.0, 1.02]  # walks upwards and stops at the first hit
    assert schedule.calibrate(lambda a: recall[a], 0.5, grid) == 0.9
    assert schedule.calibrate(lambda a: recall[a], 1.0, grid) == 1.1
    assert math.isinf(schedule.calibrate(lambda a: 0.5, 0.9, grid))
    with pytest.raises(ValueError):
        schedule.calibrate(lambda a: 1.0, 1.5, grid)


def test_calibration_with_the_oracle_predictor():
    """With the oracle as the predictor and the exact truth, recall does not
    decrease along the grid, and the calibrated alpha is the first grid
    value that reaches the target."""
    pl = synth.planted_layer(512, 1376, 0.9, config=6, layer=1, p_active=0.47, p_inactive=0.53)
    wg, x = u16(pl.w_gate), u16(pl.x)
    packed = oracle.pack_signs(wg)
    truth = torch.from_numpy(oracle.gate_truly_positive(wg, x))

    def recall_at(a):
        mask, _, _ = oracle.predict_rows(packed, x, a)
        return schedule.quality(torch.from_numpy(mask.astype(bool)), truth)["active_recall"]

    grid = schedule.DEFAULT_ALPHAS
    curve = [recall_at(a) for a in grid]
    assert all(b >= a for a, b in zip(curve, curve[1:]))
    assert curve[0] < 1.0  # the workload leaves something to calibrate
    target = 0.99
    a_star = schedule.calibrate(recall_at, target, grid)
    i = list(grid).index(a_star)
    assert curve[i] >= target and all(c < target for c in curve[:i])
