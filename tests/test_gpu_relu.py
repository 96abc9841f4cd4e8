"""Parity of the non-gated ReLU MLP path (no W_up: ``si_sparse_relu_mlp``,
``si_predict_sparse_relu_mlp``) with the CPU oracle's ``relu_mlp``.

Same bars as the gated path: masks, kept lists and counts bit-exact; y within
1e-2 relative L2 and 1e-4 of the largest |y| element-wise; n_gate exact,
n_up zero, n_down within a few rows of the oracle's.
"""

import math

import numpy as np
import pytest
import torch

import oracle
import paper_2411_12692_amd as si
from h3check import check_h3, fp16_rows, workspace_ok
from paper_2411_12692_amd import synth

pytestmark = pytest.mark.gpu

DEV = "cuda"


def u16(t: torch.Tensor) -> np.ndarray:
    return t.detach().cpu().contiguous().view(torch.int16).numpy().view(np.uint16)


def to_dev(a: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(a.view(np.int16).copy()).to(DEV)


def rand_bits(rng, shape):
    return rng.standard_normal(shape).astype(np.float16).view(np.uint16)


class ReluCase:
    """Host arrays (fp16 bits) of one non-gated layer plus its device state."""

    def __init__(self, w1, wd, x, max_batch=1):
        self.w1, self.wd, self.x = w1, wd, x
        self.k, self.d = w1.shape
        self.layer = si.MLPLayer(to_dev(w1), None, to_dev(wd), max_batch=max_batch)
        self.packed = oracle.pack_signs(w1)

    @classmethod
    def planted(cls, d, k, s, config, b=1):
        """The planted construction with W_gate as W_fc1 (W_up unused)."""
        L = synth.planted_layer(d, k, s, config=config)
        x = synth.batch_tokens(L, b, config=config)
        return cls(u16(L.w_gate), u16(L.w_down), u16(x), max_batch=b)


def check(c: ReluCase, mask_ref, y, cnt=None, flags=0):
    """y, the counters and the per-row h = ReLU(g) of the call just made
    (the last one on the layer's workspace) against the oracle."""
    assert workspace_ok(c.layer.workspace)
    out = oracle.relu_mlp(c.w1, c.wd, c.x, mask_ref)
    X = oracle.fp16_to_f64(np.atleast_2d(c.x))
    check_h3(c.layer.workspace, c.k, c.d, X.shape[0], mask_ref, out["h"], X, fp16_rows(c.w1), None, out["g"])
    yr = out["y"]
    yg = y.cpu().numpy().astype(np.float64)
    nb = np.linalg.norm(yr)
    err = float(np.linalg.norm(yg - yr) / nb) if nb > 0 else float(np.linalg.norm(yg))
    assert err <= 1e-2, err
    scale = max(np.abs(yr).max(), 1e-30)
    assert np.abs(yg - yr).max() <= 1e-4 * scale + 1e-30
    if cnt is not None:
        n_gate, n_up, n_down = cnt.cpu().numpy().tolist()
        assert n_gate == out["n_gate"] and n_up == 0
        if flags & si.SI_NO_AS:
            assert n_down == out["n_gate"]
        elif flags & si.SI_NO_SPECULATION:
            assert abs(n_down - out["n_down"]) <= 3, (n_down, out["n_down"])
        else:  # speculative requests may read more rows, never fewer
            assert out["n_down"] - 3 <= n_down <= out["n_gate"], (n_down, out["n_down"])
    return out


def fused(c: ReluCase, alpha, flags=0):
    y, (mask, idx, n, cnt) = c.layer(to_dev(c.x), alpha, flags=flags, outputs=True)
    torch.cuda.synchronize()
    m_ref = oracle.predict_rows(c.packed, c.x, alpha)[0]
    assert np.array_equal(mask.cpu().numpy(), m_ref)
    nref = int(m_ref.sum())
    assert int(n.item()) == nref
    assert np.array_equal(idx.cpu().numpy()[:nref], oracle.active_rows(m_ref))
    check(c, m_ref, y, cnt, flags)
    return m_ref, mask, idx, n


@pytest.fixture(scope="module")
def tiny():
    return ReluCase.planted(512, 1376, 0.9, config=1)


@pytest.mark.parametrize("alpha", [0.0, 0.7, 1.0, 1.45, 1.5, math.inf])
def test_relu_fused_tiny(tiny, alpha):
    fused(tiny, alpha)


def test_relu_separate_calls(tiny):
    """Mask-driven and list-driven calls on the predicted rows equal the fused
    call's rows."""
    m_ref, mask, idx, n = fused(tiny, 1.0)
    x = to_dev(tiny.x)
    y1, c1 = tiny.layer.sparse_mlp(x, mask=mask, counters=True)
    torch.cuda.synchronize()
    check(tiny, m_ref, y1, c1)
    y2, c2 = tiny.layer.sparse_mlp(x, mask, idx, n, counters=True)
    torch.cuda.synchronize()
    check(tiny, m_ref, y2, c2)


@pytest.mark.parametrize("flags", [si.SI_NO_AS, si.SI_NO_SPECULATION, si.SI_NO_AS | si.SI_NO_SPECULATION])
def test_relu_flags(tiny, flags):
    m_ref, mask, idx, n = fused(tiny, 1.0, flags=flags)
    y, cnt = tiny.layer.sparse_mlp(to_dev(tiny.x), mask, idx, n, flags=flags, counters=True)
    torch.cuda.synchronize()
    check(tiny, m_ref, y, cnt, flags)


def test_relu_opt_shape():
    """OPT-6.7B-shaped MLP (d = 4096, k = 16384), planted sparsity 0.9."""
    c = ReluCase.planted(4096, 16384, 0.9, config=7)
    assert si._lib.load().si_single_launch(c.k, c.d, 1) == 1
    m_ref, mask, idx, n = fused(c, 1.0)
    y, cnt = c.layer.sparse_mlp(to_dev(c.x), mask, idx, n, counters=True)
    torch.cuda.synchronize()
    check(c, m_ref, y, cnt)


@pytest.mark.parametrize("b", [2, 5, 8])
def test_relu_batches(b):
    rng = np.random.default_rng(40 + b)
    k, d = 1500, 1024
    c = ReluCase(rand_bits(rng, (k, d)), rand_bits(rng, (d, k)), rand_bits(rng, (b, d)), max_batch=b)
    for alpha in [1.0, math.inf]:
        m_ref, mask, idx, n = fused(c, alpha)
        y, cnt = c.layer.sparse_mlp(to_dev(c.x), mask, idx, n, counters=True)
        torch.cuda.synchronize()
        check(c, m_ref, y, cnt)
        y2, cnt2 = c.layer.sparse_mlp(to_dev(c.x), mask=mask, counters=True)
        torch.cuda.synchronize()
        check(c, m_ref, y2, cnt2)


def test_relu_one_token_large_groups():
    """One token in groups of more than 512 rows (k = 20000 at d = 4096:
    groups of 8 blocks x 80 rows) takes the kernel instance with the wider
    down-projection batches: the planted construction at alpha = 1 and
    +inf, and without speculation."""
    c = ReluCase.planted(4096, 20000, 0.9, config=6)
    for alpha, flags in [(1.0, 0), (math.inf, 0), (1.0, si.SI_NO_SPECULATION)]:
        fused(c, alpha, flags)


@pytest.mark.parametrize("k,d,b,one", [(1, 128, 1, 1), (65, 384, 2, 1), (129, 8192, 3, 1), (20000, 384, 1, 1),
                                       (65537, 128, 1, 0)])
def test_relu_edge_shapes(k, d, b, one):
    """Ragged rows and tiles, several groups per block, and the multi-launch
    path (more than 256 rows per compute unit)."""
    assert si._lib.load().si_single_launch(k, d, b) == one
    rng = np.random.default_rng(k * 13 + d)
    c = ReluCase(rand_bits(rng, (k, d)), rand_bits(rng, (d, k)), rand_bits(rng, (b, d)), max_batch=b)
    for alpha in [1.0, math.inf]:
        if not one:  # the multi-launch path keeps h3 as plain floats: no stale value may pass for this call's
            c.layer.workspace.zero_()
        m_ref, mask, idx, n = fused(c, alpha)
        if m_ref.any():
            if not one:
                c.layer.workspace.zero_()
            y, cnt = c.layer.sparse_mlp(to_dev(c.x), mask, idx, n, counters=True)
            torch.cuda.synchronize()
            check(c, m_ref, y, cnt)
            if not one:
                c.layer.workspace.zero_()
            y2 = c.layer.sparse_mlp(to_dev(c.x), mask=mask)
            torch.cuda.synchronize()
            check(c, m_ref, y2)


def test_relu_rejects_bad_arguments(tiny):
    lib = si._lib.load()
    ws = tiny.layer.workspace
    x = to_dev(tiny.x)
    y = torch.empty(1, tiny.d, dtype=torch.float32, device=DEV)
    st = lib.si_sparse_relu_mlp(None, si._vp(tiny.layer.w_down_t), tiny.k, tiny.d, si._vp(x), 1, None, None, None,
                                si._vp(y), si._vp(ws), ws.numel(), 0, None, None)
    assert st == 1  # SI_ERR_NULL: w_fc1
    st = lib.si_predict_sparse_relu_mlp(si._vp(tiny.layer.signs), si._vp(tiny.layer.w_gate),
                                        si._vp(tiny.layer.w_down_t), tiny.k, tiny.d, si._vp(x), 1, -1.0, None,
                                        None, None, si._vp(y), si._vp(ws), ws.numel(), 0, None, None)
    assert st == 4  # SI_ERR_ALPHA
