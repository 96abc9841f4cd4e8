"""Guard bands around every output of the C ABI: each output buffer is a
window in the middle of a larger device buffer filled with a sentinel
pattern, and after the call every byte outside the window must still hold
the sentinel (no kernel writes past its outputs).  Covers the fused,
mask-driven, list-driven and predictor-only calls, fp16 gated, non-gated and
INT8 forms, at a small ragged shape and a batch of 3 tokens.  The masks of
repeated calls (fresh and reused workspaces) must be bit-identical.
"""

import ctypes
import math

import numpy as np
import pytest
import torch

import oracle
import paper_2411_12692_amd as si

pytestmark = pytest.mark.gpu

DEV = "cuda"
GUARD = 256  # bytes on each side (keeps 16-byte alignment)
PATTERN = 0xA5


class Guarded:
    """A device window of ``nbytes`` inside a sentinel-filled buffer."""

    def __init__(self, nbytes):
        self.nbytes = nbytes
        self.buf = torch.full((nbytes + 2 * GUARD,), PATTERN, dtype=torch.uint8, device=DEV)

    @property
    def ptr(self):
        return ctypes.c_void_p(self.buf.data_ptr() + GUARD)

    def view(self, dtype, shape):
        return self.buf[GUARD:GUARD + self.nbytes].view(dtype).view(*shape)

    def check(self, name):
        host = self.buf.cpu().numpy()
        assert np.all(host[:GUARD] == PATTERN), f"{name}: bytes written before the output"
        assert np.all(host[GUARD + self.nbytes:] == PATTERN), f"{name}: bytes written past the output"


def to_dev(a):
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to(DEV)


def outputs(k, d, b):
    return {"mask": Guarded(k), "idx": Guarded(4 * k), "n": Guarded(4), "y": Guarded(4 * b * d),
            "cnt": Guarded(12)}


def check_all(out):
    for name, g in out.items():
        g.check(name)


@pytest.fixture(scope="module", params=[(777, 640, 3), (1376, 512, 1)], ids=["k777-d640-b3", "k1376-d512-b1"])
def case(request):
    k, d, b = request.param
    rng = np.random.default_rng(k + d + b)
    wg = rng.standard_normal((k, d)).astype(np.float16)
    wu = rng.standard_normal((k, d)).astype(np.float16)
    wd = rng.standard_normal((d, k)).astype(np.float16)
    x = rng.standard_normal((b, d)).astype(np.float16)
    return k, d, b, wg, wu, wd, x


@pytest.mark.parametrize("gated", [True, False])
def test_guards_fp16_calls(case, gated):
    k, d, b, wg, wu, wd, x = case
    lib = si._lib.load()
    vp = si._vp
    layer = si.MLPLayer(to_dev(wg), to_dev(wu) if gated else None, to_dev(wd), max_batch=b)
    xd = to_dev(x)
    ws = layer.workspace
    mask_ref = oracle.predict_rows(oracle.pack_signs(wg.view(np.uint16)), x.view(np.uint16), 1.0)[0]

    out = outputs(k, d, b)
    args = (k, d, vp(xd), b, 1.0, out["mask"].ptr, out["idx"].ptr, out["n"].ptr, out["y"].ptr, vp(ws), ws.numel(),
            0, out["cnt"].ptr, None)
    if gated:
        st = lib.si_predict_sparse_mlp(vp(layer.signs), vp(layer.w_gate), vp(layer.w_up), vp(layer.w_down_t), *args)
    else:
        st = lib.si_predict_sparse_relu_mlp(vp(layer.signs), vp(layer.w_gate), vp(layer.w_down_t), *args)
    assert st == 0, si._lib.last_error()
    torch.cuda.synchronize()
    check_all(out)
    assert np.array_equal(out["mask"].view(torch.uint8, (k,)).cpu().numpy(), mask_ref)

    # mask-driven and list-driven calls on the predicted rows
    for use_list in (False, True):
        o2 = {"y": Guarded(4 * b * d), "cnt": Guarded(12)}
        mask_in = out["mask"].view(torch.uint8, (k,))
        idx_in = out["idx"].view(torch.int32, (k,)) if use_list else None
        n_in = out["n"].view(torch.int32, (1,)) if use_list else None
        tail = (k, d, vp(xd), b, vp(mask_in), vp(idx_in), vp(n_in), o2["y"].ptr, vp(ws), ws.numel(), 0,
                o2["cnt"].ptr, None)
        if gated:
            st = lib.si_sparse_mlp(vp(layer.w_gate), vp(layer.w_up), vp(layer.w_down_t), *tail)
        else:
            st = lib.si_sparse_relu_mlp(vp(layer.w_gate), vp(layer.w_down_t), *tail)
        assert st == 0, si._lib.last_error()
        torch.cuda.synchronize()
        check_all(o2)

    # the predictor alone
    o3 = {"mask": Guarded(k), "idx": Guarded(4 * k), "n": Guarded(4)}
    st = lib.si_predict(vp(layer.signs), k, d, vp(xd), b, 1.0, o3["mask"].ptr, o3["idx"].ptr, o3["n"].ptr, vp(ws),
                        ws.numel(), None)
    assert st == 0, si._lib.last_error()
    torch.cuda.synchronize()
    check_all(o3)
    assert np.array_equal(o3["mask"].view(torch.uint8, (k,)).cpu().numpy(), mask_ref)


def test_guards_int8_calls(case):
    k, d, b, wg, wu, wd, x = case
    lib = si._lib.load()
    vp = si._vp
    layer = si.Int8MLPLayer(to_dev(wg), to_dev(wu), to_dev(wd), max_batch=b)
    xd = to_dev(x)
    ws = layer.workspace
    out = outputs(k, d, b)
    st = lib.si_predict_sparse_mlp_i8(vp(layer.signs), vp(layer.q_gate), vp(layer.s_gate), vp(layer.q_up),
                                      vp(layer.s_up), vp(layer.q_down_t), vp(layer.s_down), k, d, vp(xd), b, 1.0,
                                      out["mask"].ptr, out["idx"].ptr, out["n"].ptr, out["y"].ptr, vp(ws),
                                      ws.numel(), 0, out["cnt"].ptr, None)
    assert st == 0, si._lib.last_error()
    torch.cuda.synchronize()
    check_all(out)
    o2 = {"y": Guarded(4 * b * d), "cnt": Guarded(12)}
    st = lib.si_sparse_mlp_i8(vp(layer.q_gate), vp(layer.s_gate), vp(layer.q_up), vp(layer.s_up),
                              vp(layer.q_down_t), vp(layer.s_down), k, d, vp(xd), b,
                              vp(out["mask"].view(torch.uint8, (k,))), o2["y"].ptr, vp(ws), ws.numel(), 0,
                              o2["cnt"].ptr, None)
    assert st == 0, si._lib.last_error()
    torch.cuda.synchronize()
    check_all(o2)
    # load-time outputs: quantization, sign packing and the transpose
    g = {"q": Guarded(k * d), "s": Guarded(4 * k), "signs": Guarded(si.signs_bytes(k, d)), "t": Guarded(k * d)}
    assert lib.si_quantize_rows_i8(vp(to_dev(wg)), k, d, g["q"].ptr, g["s"].ptr, None) == 0
    assert lib.si_pack_signs_i8(vp(layer.q_gate), k, d, g["signs"].ptr, None) == 0
    qd, _ = si.quantize_rows_i8(to_dev(wd))
    assert lib.si_transpose_down_i8(vp(qd), d, k, g["t"].ptr, None) == 0
    torch.cuda.synchronize()
    check_all(g)
    assert torch.equal(g["q"].view(torch.int8, (k, d)), layer.q_gate)
    assert torch.equal(g["t"].view(torch.int8, (k, d)), layer.q_down_t)


def test_masks_are_identical_across_calls_and_workspaces(case):
    k, d, b, wg, wu, wd, x = case
    layer = si.MLPLayer(to_dev(wg), to_dev(wu), to_dev(wd), max_batch=b)
    xd = to_dev(x)
    masks = []
    for rep in range(4):
        if rep == 2:  # a fresh workspace half way
            layer.workspace = si.new_workspace(k, d, b)
        for alpha in (1.0, 1.5, math.inf):
            _, (mask, idx, n, _) = layer(xd, alpha, outputs=True)
            masks.append((alpha, mask.cpu().numpy().copy(), int(n.item())))
    by_alpha = {}
    for alpha, m, n in masks:
        by_alpha.setdefault(alpha, []).append((m, n))
    for alpha, ms in by_alpha.items():
        for m, n in ms[1:]:
            assert np.array_equal(m, ms[0][0]) and n == ms[0][1], alpha
