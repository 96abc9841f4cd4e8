"""Parity over the sparsity/batch sweep at the 7B shape: planted sparsity s in
{0.5, 0.7, 0.8, 0.9, 0.95, 0.97} and decode batches of 1, 2, 4 and 8 tokens.

The batch's kept set is the union of independently drawn per-token active
sets (``synth.batch_union_mask``), handed to ``si_sparse_mlp`` through its
mask argument; y must match the oracle within 1e-2 relative L2 and the work
counters must match the mask.  The fused call with the predictor on the same
tokens is checked too (mask bit-exact, y in tolerance).
"""

import numpy as np
import pytest
import torch

import oracle
import paper_2411_12692_amd as si
from paper_2411_12692_amd import synth

pytestmark = pytest.mark.gpu
DEV = "cuda"
D, K, CONFIG = 4096, 11008, 5
SPARSITY = [0.5, 0.7, 0.8, 0.9, 0.95, 0.97]
BATCH = [1, 2, 4, 8]


def u16(t: torch.Tensor) -> np.ndarray:
    return t.detach().cpu().contiguous().view(torch.int16).numpy().view(np.uint16)


def rel_l2(a, b):
    return float(np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300))


def check_y(y, ref):
    y = y.cpu().numpy().astype(np.float64)
    assert rel_l2(y, ref) <= 1e-2
    assert np.abs(y - ref).max() <= 1e-4 * np.abs(ref).max()


@pytest.mark.parametrize("s", SPARSITY)
def test_sweep(s):
    li = SPARSITY.index(s)
    L = synth.planted_layer(D, K, s, config=CONFIG, layer=li, device=DEV)
    layer = si.MLPLayer(L.w_gate, L.w_up, L.w_down, max_batch=max(BATCH))
    wg, wu, wd = u16(L.w_gate), u16(L.w_up), u16(L.w_down)
    packed = oracle.pack_signs(wg)
    for b in BATCH:
        x = synth.batch_tokens(L, b, config=CONFIG, layer_id=li)
        mask = synth.batch_union_mask(L, b, config=CONFIG, layer_id=li)
        y, cnt = layer.sparse_mlp(x, mask=mask, counters=True)
        torch.cuda.synchronize()
        m = mask.cpu().numpy()
        xh = u16(x)
        out = oracle.sparse_mlp(wg, wu, wd, xh, m)
        check_y(y, out["y"])
        c = cnt.cpu().tolist()
        assert c[0] == int(m.sum()) and out["n_up"] - 3 <= c[1] <= c[0] and out["n_down"] - 3 <= c[2] <= c[0]
        # the fused path with the predictor on the same tokens
        yf, (mf, idx, n, _) = layer(x, 1.0, outputs=True)
        torch.cuda.synchronize()
        m_ref, _, _ = oracle.predict_rows(packed, xh, 1.0)
        assert np.array_equal(mf.cpu().numpy(), m_ref)
        nref = int(m_ref.sum())
        assert int(n.item()) == nref
        assert np.array_equal(idx.cpu().numpy()[:nref], oracle.active_rows(m_ref))
        check_y(yf, oracle.sparse_mlp(wg, wu, wd, xh, m_ref)["y"])
    assert si.workspace_check(layer.workspace) == 0
    del layer, L
    torch.cuda.empty_cache()
