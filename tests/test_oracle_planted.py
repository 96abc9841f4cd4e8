"""Oracle pins on the planted synthetic layers (CPU only).

The planted construction fixes which rows are meant to be inactive, so it
gives the oracle an answer it did not compute itself.
"""

import math

import numpy as np
import pytest
import torch

import oracle
from paper_2411_12692_amd import synth


def _np(t):
    return t.contiguous().view(torch.int16).numpy().view(np.uint16)


@pytest.fixture(scope="module")
def layer_7b():
    return synth.planted_layer(4096, 11008, 0.9, config=2, layer=0)


@pytest.fixture(scope="module")
def layer_tiny():
    return synth.planted_layer(512, 1376, 0.9, config=1, layer=0)


def test_planted_counts(layer_tiny, layer_7b):
    assert int(layer_tiny.inactive.sum()) == 1238
    assert int(layer_7b.inactive.sum()) == 9907


def test_alpha1_recovers_the_planted_rows_at_7b(layer_7b):
    # Active rows disagree on ~40% of 4096 coordinates, inactive ones on ~60%;
    # at alpha = 1 the threshold sits 13 standard deviations from either mean,
    # so the predicted-active set is exactly the planted active set.
    packed = oracle.pack_signs(_np(layer_7b.w_gate))
    mask, _, n_neg = oracle.predict_rows(packed, _np(layer_7b.x), 1.0)
    planted_active = (~layer_7b.inactive).numpy().astype(np.uint8)
    assert np.array_equal(mask, planted_active)
    frac = n_neg[0] / 4096.0
    assert abs(frac[planted_active == 1].mean() - 0.4) < 0.002
    assert abs(frac[planted_active == 0].mean() - 0.6) < 0.002


def test_superset_of_truth_reproduces_dense(layer_tiny):
    wg, wu, wd, x = (_np(layer_tiny.w_gate), _np(layer_tiny.w_up),
                     _np(layer_tiny.w_down), _np(layer_tiny.x))
    truth = oracle.gate_truly_positive(wg, x)[0]
    rng = np.random.default_rng(0)
    mask = (truth | (rng.random(truth.size) < 0.05)).astype(np.uint8)
    dense = oracle.dense_mlp(wg, wu, wd, x)
    part = oracle.sparse_mlp(wg, wu, wd, x, mask)
    scale = np.abs(dense["y"]).max()
    assert np.max(np.abs(part["y"] - dense["y"])) <= 1e-12 * scale
    # dropping one truly positive row does change the output
    drop = mask.copy()
    drop[np.flatnonzero(truth)[0]] = 0
    assert np.max(np.abs(oracle.sparse_mlp(wg, wu, wd, x, drop)["y"] - dense["y"])) > 1e-6 * scale


def test_recall_counts_on_tiny_layer(layer_tiny):
    wg, x = _np(layer_tiny.w_gate), _np(layer_tiny.x)
    packed = oracle.pack_signs(wg)
    truth = oracle.gate_truly_positive(wg, x)
    _, act1, _ = oracle.predict_rows(packed, x, 1.0)
    _, act07, _ = oracle.predict_rows(packed, x, 0.7)
    q1 = oracle.prediction_quality(act1, truth)
    q07 = oracle.prediction_quality(act07, truth)
    missed1 = int((truth & ~act1).sum())
    assert q1["missed"] == missed1
    assert q1["active_recall"] == pytest.approx((truth.sum() - missed1) / truth.sum())
    # a more aggressive alpha can only miss more truly positive rows
    assert q07["missed"] >= q1["missed"]
    assert q07["pred_sparse"] >= q1["pred_sparse"]
    # planted data: the gate pre-activation of inactive rows is centred well below 0
    assert q1["precision"] > 0.99


def test_alpha_inf_equals_dense(layer_tiny):
    wg, wu, wd, x = (_np(layer_tiny.w_gate), _np(layer_tiny.w_up),
                     _np(layer_tiny.w_down), _np(layer_tiny.x))
    mask, _, _ = oracle.predict_rows(oracle.pack_signs(wg), x, math.inf)
    assert mask.all()
    a = oracle.sparse_mlp(wg, wu, wd, x, mask)["y"]
    b = oracle.dense_mlp(wg, wu, wd, x)["y"]
    assert np.array_equal(a, b)


def test_union_mask_density():
    layer = synth.planted_layer(256, 4000, 0.9, config=5, layer=0)
    for b in [1, 2, 4, 8]:
        m = synth.batch_union_mask(layer, b, config=5).numpy()
        expect = 1 - 0.9 ** b
        assert abs(m.mean() - expect) < 0.03
