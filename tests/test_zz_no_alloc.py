"""The entry point for callers that cannot allocate
(``si_predict_sparse_mlp_noalloc``: the whole path with the library's own
per-device scratch array in place of a caller's workspace) against the
workspace form ``si_predict_sparse_mlp`` and the oracle.

Four calls in a row on the one scratch array, each smaller or different in
shape from the one before (a 13B-shaped layer with 1 token, whose groups of
more than 512 rows take the instance with the wider down batches, a
7B-shaped layer with 2 tokens, the small planted block with 1 token, then a
ragged random shape with 3 tokens), so that whatever a call leaves in the
array cannot pass for the next call's data.  Masks, kept lists, counts and work counters bit-exact against the
workspace form (and the masks, lists and counts against the oracle); y within
1e-2 relative L2 and 1e-4 of its largest element of the oracle's, and within
fp32 summation order (1e-5 of its largest element) of the workspace form's.
"""

import math

import numpy as np
import pytest
import torch

import oracle
import paper_2411_12692_amd as si
from paper_2411_12692_amd import synth

pytestmark = pytest.mark.gpu

DEV = "cuda"


def u16(t: torch.Tensor) -> np.ndarray:
    return t.detach().cpu().contiguous().view(torch.int16).numpy().view(np.uint16)


def to_dev(a: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(a.view(np.int16).copy()).to(DEV)


def noalloc(layer, x, alpha, flags=0):
    """One call of the no-allocation entry point through the C ABI."""
    k, d = layer.k, layer.d
    b = x.shape[0]
    y = torch.empty(b, d, dtype=torch.float32, device=DEV)
    mask = torch.empty(k, dtype=torch.uint8, device=DEV)
    idx = torch.empty(k, dtype=torch.int32, device=DEV)
    n = torch.empty(1, dtype=torch.int32, device=DEV)
    cnt = torch.zeros(3, dtype=torch.int32, device=DEV)
    vp = si._vp
    st = si._lib.status("si_predict_sparse_mlp_noalloc", vp(layer.signs), vp(layer.w_gate), vp(layer.w_up),
                        vp(layer.w_down_t), k, d, vp(x), b, float(alpha), vp(mask), vp(idx), vp(n), vp(y), flags,
                        vp(cnt), si._stream())
    assert st == 0, (st, si._lib.last_error())
    return y, mask, idx, n, cnt


def compare(wg, wu, wd, xb, alpha):
    k, d = wg.shape
    b = xb.shape[0]
    print(f"no-alloc call k={k} d={d} b={b} alpha={alpha}", flush=True)
    layer = si.MLPLayer(to_dev(wg), to_dev(wu), to_dev(wd), max_batch=b)
    x = to_dev(xb)
    y0, (m0, i0, n0, c0) = layer(x, alpha, outputs=True)
    y1, m1, i1, n1, c1 = noalloc(layer, x, alpha)
    torch.cuda.synchronize()
    m_ref = oracle.predict_rows(oracle.pack_signs(wg), xb, alpha)[0]
    nref = int(m_ref.sum())
    for m, i, n in ((m0, i0, n0), (m1, i1, n1)):
        assert np.array_equal(m.cpu().numpy(), m_ref)
        assert int(n.item()) == nref
        assert np.array_equal(i.cpu().numpy()[:nref], oracle.active_rows(m_ref))
    assert torch.equal(c0, c1), (c0.tolist(), c1.tolist())
    yr = oracle.sparse_mlp(wg, wu, wd, xb, m_ref)["y"]
    yg = y1.cpu().numpy().astype(np.float64)
    scale = max(np.abs(yr).max(), 1e-30)
    assert np.linalg.norm(yg - yr) <= 1e-2 * np.linalg.norm(yr) + 1e-30
    assert np.abs(yg - yr).max() <= 1e-4 * scale + 1e-30
    assert (y1 - y0).abs().max().item() <= 1e-5 * scale + 1e-30
    assert si.workspace_check(layer.workspace) == 0


def test_noalloc_matches_workspace_form_calls_in_a_row():
    # 13B shape, one token (groups of more than 512 rows), then smaller calls on the same scratch
    B = synth.planted_layer(5120, 13824, 0.88, config=4, layer=3)
    compare(u16(B.w_gate), u16(B.w_up), u16(B.w_down), u16(B.x), 1.0)
    del B
    L = synth.planted_layer(4096, 11008, 0.9, config=2, layer=5)
    x = synth.batch_tokens(L, 2, config=2)
    compare(u16(L.w_gate), u16(L.w_up), u16(L.w_down), u16(x), 1.0)
    s = synth.planted_layer(512, 1376, 0.9, config=1, layer=2)
    compare(u16(s.w_gate), u16(s.w_up), u16(s.w_down), u16(s.x), 1.45)
    rng = np.random.default_rng(77)
    k, d, b = 3001, 1152, 3
    bits = lambda shape: rng.standard_normal(shape).astype(np.float16).view(np.uint16)
    compare(bits((k, d)), bits((k, d)), bits((d, k)), bits((b, d)), math.inf)


def test_noalloc_rejects_a_shape_beyond_its_scratch():
    lib = si._lib.load()
    k, d, b = 1 << 20, 4096, 8
    assert lib.si_workspace_bytes(k, d, b) > 8 << 20
    p = si._vp(torch.empty(16, dtype=torch.uint8, device=DEV))
    st = lib.si_predict_sparse_mlp_noalloc(p, p, p, p, k, d, p, b, 1.0, None, None, None, p, 0, None, None)
    assert st == 5, si._lib.last_error()  # SI_ERR_WORKSPACE
    assert "scratch" in si._lib.last_error()
