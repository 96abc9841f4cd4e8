"""Parity of the INT8-weight path (``si_quantize_rows_i8``,
``si_pack_signs_i8``, ``si_transpose_down_i8``, ``si_sparse_mlp_i8``,
``si_predict_sparse_mlp_i8``) with the CPU oracle's ``quantize_rows_int8``,
``pack_signs_int8`` and ``int8_mlp``.

Each side quantizes the same fp16 weights on its own (the device at load,
the oracle on the host); INT8 values, scales, packed signs, the transpose,
masks, kept lists and counts are compared bit-exact; y within 1e-2 relative
L2 and 1e-4 of the largest |y| element-wise (fp32 accumulation of exact
INT8 x fp16 products); n_gate exact and n_up / n_down within a few rows.
"""

import math

import numpy as np
import pytest
import torch

import oracle
import paper_2411_12692_amd as si
from h3check import check_h3, int8_rows, workspace_ok
from paper_2411_12692_amd import synth

pytestmark = pytest.mark.gpu

DEV = "cuda"


def u16(t: torch.Tensor) -> np.ndarray:
    return t.detach().cpu().contiguous().view(torch.int16).numpy().view(np.uint16)


def to_dev(a: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(a.view(np.int16).copy()).to(DEV)


def rand_bits(rng, shape):
    return rng.standard_normal(shape).astype(np.float16).view(np.uint16)


class I8Case:
    """fp16 weights (bits), their INT8 form on both sides, and the device
    layer."""

    def __init__(self, wg, wu, wd, x, max_batch=1):
        self.x = x
        self.k, self.d = wg.shape
        self.gated = wu is not None
        self.layer = si.Int8MLPLayer(to_dev(wg), to_dev(wu) if self.gated else None, to_dev(wd),
                                     max_batch=max_batch)
        self.qg, self.sg = oracle.quantize_rows_int8(wg)
        self.qu, self.su = oracle.quantize_rows_int8(wu) if self.gated else (None, None)
        self.qd, self.sd = oracle.quantize_rows_int8(wd)
        self.packed = oracle.pack_signs_int8(self.qg)

    @classmethod
    def planted(cls, d, k, s, config, b=1, gated=True):
        L = synth.planted_layer(d, k, s, config=config)
        x = synth.batch_tokens(L, b, config=config)
        return cls(u16(L.w_gate), u16(L.w_up) if gated else None, u16(L.w_down), u16(x), max_batch=b)

    def oracle_mlp(self, mask):
        return oracle.int8_mlp(self.qg, self.sg, self.qu, self.su, self.qd, self.sd, self.x, mask)


def check_weights(c: I8Case):
    L = c.layer
    assert np.array_equal(L.q_gate.cpu().numpy(), c.qg)
    assert np.array_equal(L.s_gate.cpu().numpy().view(np.uint32), c.sg.view(np.uint32))
    if c.gated:
        assert np.array_equal(L.q_up.cpu().numpy(), c.qu)
        assert np.array_equal(L.s_up.cpu().numpy().view(np.uint32), c.su.view(np.uint32))
    assert np.array_equal(L.q_down_t.cpu().numpy(), c.qd.T)
    assert np.array_equal(L.s_down.cpu().numpy().view(np.uint32), c.sd.view(np.uint32))
    canon = si.signs_to_canonical(L.signs, c.k, c.d).cpu().numpy().view(np.uint32)
    assert np.array_equal(canon, c.packed)


def check(c: I8Case, mask_ref, y, cnt=None, flags=0):
    """y, the counters and the per-row h3 of the call just made (the last one
    on the layer's workspace) against the oracle."""
    assert workspace_ok(c.layer.workspace)
    out = c.oracle_mlp(mask_ref)
    X = oracle.fp16_to_f64(np.atleast_2d(c.x))
    check_h3(c.layer.workspace, c.k, c.d, X.shape[0], mask_ref, out["h3"], X, int8_rows(c.qg, c.sg),
             int8_rows(c.qu, c.su) if c.gated else None, out["g"])
    yr = out["y"]
    yg = y.cpu().numpy().astype(np.float64)
    nb = np.linalg.norm(yr)
    err = float(np.linalg.norm(yg - yr) / nb) if nb > 0 else float(np.linalg.norm(yg))
    assert err <= 1e-2, err
    scale = max(np.abs(yr).max(), 1e-30)
    assert np.abs(yg - yr).max() <= 1e-4 * scale + 1e-30
    if cnt is not None:
        n_gate, n_up, n_down = cnt.cpu().numpy().tolist()
        assert n_gate == out["n_gate"]
        if not c.gated:
            assert n_up == 0
        elif flags & si.SI_NO_AS:
            assert n_up == out["n_gate"]
        else:  # speculative requests may read more rows, never fewer
            assert out["n_up"] - 3 <= n_up <= out["n_gate"], (n_up, out["n_up"])
        if flags & si.SI_NO_AS:
            assert n_down == out["n_gate"]
        else:
            assert out["n_down"] - 3 <= n_down <= out["n_gate"], (n_down, out["n_down"])
    return out


def fused(c: I8Case, alpha, flags=0):
    y, (mask, idx, n, cnt) = c.layer(to_dev(c.x), alpha, flags=flags, outputs=True)
    torch.cuda.synchronize()
    m_ref = oracle.predict_rows(c.packed, c.x, alpha)[0]
    assert np.array_equal(mask.cpu().numpy(), m_ref)
    nref = int(m_ref.sum())
    assert int(n.item()) == nref
    assert np.array_equal(idx.cpu().numpy()[:nref], oracle.active_rows(m_ref))
    check(c, m_ref, y, cnt, flags)
    return m_ref, mask


@pytest.fixture(scope="module")
def tiny():
    c = I8Case.planted(512, 1376, 0.9, config=1)
    check_weights(c)
    return c


def test_int8_quantize_special_rows():
    """Rows of zeros (+0 and -0), a single nonzero, ties at half steps,
    the largest finite fp16 values and subnormals, at a row length that is a
    multiple of nothing."""
    n = 1001
    rows = [np.zeros(n), -np.zeros(n), np.eye(1, n, 17)[0] * -3.0,
            np.arange(n) % 7 - 3.0, np.full(n, 65504.0) * np.where(np.arange(n) % 2, 1, -1),
            np.arange(n) * 2.0 ** -24, (np.arange(n) - 500) * 0.5]
    w = np.stack(rows).astype(np.float16).view(np.uint16)
    q, s = si.quantize_rows_i8(to_dev(w))
    qo, so = oracle.quantize_rows_int8(w)
    assert np.array_equal(q.cpu().numpy(), qo)
    assert np.array_equal(s.cpu().numpy().view(np.uint32), so.view(np.uint32))


@pytest.mark.parametrize("alpha", [0.0, 0.7, 1.0, 1.45, 1.5, math.inf])
def test_int8_fused_tiny(tiny, alpha):
    fused(tiny, alpha)


def test_int8_mask_call(tiny):
    m_ref, mask = fused(tiny, 1.0)
    y, cnt = tiny.layer.sparse_mlp(to_dev(tiny.x), mask, counters=True)
    torch.cuda.synchronize()
    check(tiny, m_ref, y, cnt)
    dense = torch.ones(tiny.k, dtype=torch.uint8, device=DEV)
    y, cnt = tiny.layer.sparse_mlp(to_dev(tiny.x), dense, counters=True)
    torch.cuda.synchronize()
    check(tiny, np.ones(tiny.k, np.uint8), y, cnt)


@pytest.mark.parametrize("flags", [si.SI_NO_AS, si.SI_NO_SPECULATION, si.SI_NO_AS | si.SI_NO_SPECULATION])
def test_int8_flags(tiny, flags):
    m_ref, mask = fused(tiny, 1.0, flags=flags)
    y, cnt = tiny.layer.sparse_mlp(to_dev(tiny.x), mask, flags=flags, counters=True)
    torch.cuda.synchronize()
    check(tiny, m_ref, y, cnt, flags)


def test_int8_relu_tiny():
    c = I8Case.planted(512, 1376, 0.9, config=1, gated=False)
    check_weights(c)
    for alpha in [0.7, 1.0, math.inf]:
        m_ref, mask = fused(c, alpha)
    for flags in [si.SI_NO_AS, si.SI_NO_SPECULATION]:
        y, cnt = c.layer.sparse_mlp(to_dev(c.x), mask, flags=flags, counters=True)
        torch.cuda.synchronize()
        check(c, m_ref, y, cnt, flags)


@pytest.mark.parametrize("d,k,s,config", [(4096, 11008, 0.9, 2), (5120, 13824, 0.88, 4)])
def test_int8_full_layers(d, k, s, config):
    """7B- and 13B-shaped planted layers at alpha = 1, quantized on the
    device, in the launch configuration of the benchmark."""
    c = I8Case.planted(d, k, s, config=config)
    check_weights(c)
    assert si._lib.load().si_single_launch(c.k, c.d, 1) == 1
    m_ref, mask = fused(c, 1.0)
    # the predictor on the INT8 signs keeps nearly the planted active rows
    planted_active = k - synth.n_inactive(k, s)
    assert abs(int(m_ref.sum()) - planted_active) <= 0.02 * planted_active


@pytest.mark.parametrize("b", [2, 5, 8])
def test_int8_batches(b):
    rng = np.random.default_rng(60 + b)
    k, d = 1500, 1024
    c = I8Case(rand_bits(rng, (k, d)), rand_bits(rng, (k, d)), rand_bits(rng, (d, k)), rand_bits(rng, (b, d)),
               max_batch=b)
    check_weights(c)
    for alpha in [1.0, math.inf]:
        m_ref, mask = fused(c, alpha)
        y, cnt = c.layer.sparse_mlp(to_dev(c.x), mask, counters=True)
        torch.cuda.synchronize()
        check(c, m_ref, y, cnt)


@pytest.mark.parametrize("k,d,b", [(1, 128, 1), (65, 384, 2), (129, 8192, 3), (20000, 384, 1), (777, 640, 8)])
def test_int8_edge_shapes(k, d, b):
    """Ragged rows and tiles, a ragged last INT8 unit per lane (d = 640: 40
    units of 16 values), several groups per block, d = 8192."""
    rng = np.random.default_rng(k * 17 + d)
    c = I8Case(rand_bits(rng, (k, d)), rand_bits(rng, (k, d)), rand_bits(rng, (d, k)), rand_bits(rng, (b, d)),
               max_batch=b)
    check_weights(c)
    for alpha in [1.0, math.inf]:
        m_ref, mask = fused(c, alpha)
        if m_ref.any():
            y, cnt = c.layer.sparse_mlp(to_dev(c.x), mask, counters=True)
            torch.cuda.synchronize()
            check(c, m_ref, y, cnt)


@pytest.mark.parametrize("k,d,gated", [(9000, 8192, True), (40000, 2048, True), (20000, 4096, False)])
def test_int8_one_token_large_groups(k, d, gated):
    """One token with groups of more than 512 rows (T = ceil(d / 512) blocks
    of R rows, R the rows over the grid's whole groups rounded up to a
    multiple of 8) takes the INT8 instance with the wider down batches:
    alpha = 1 and +inf (every row kept: the most batches), without
    speculation, and a random mask.  9000 x 8192 leaves a last group of 40
    rows, 40000 x 2048 half a group; 20000 x 4096 is the non-gated form."""
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    T = (d + 511) // 512
    working = cus // T * T
    assert T * (((k + working - 1) // working + 7) // 8 * 8) > 512
    rng = np.random.default_rng(k + 5 * d)
    c = I8Case(rand_bits(rng, (k, d)), rand_bits(rng, (k, d)) if gated else None, rand_bits(rng, (d, k)),
               rand_bits(rng, (1, d)))
    check_weights(c)
    assert si._lib.load().si_single_launch(c.k, c.d, 1) == 1
    for alpha, flags in [(1.0, 0), (math.inf, 0), (1.0, si.SI_NO_SPECULATION)]:
        print(f"k={k} d={d} gated={gated} alpha={alpha} flags={flags}", flush=True)
        fused(c, alpha, flags)
    m = rng.random(k) < 0.3
    y, cnt = c.layer.sparse_mlp(to_dev(c.x), torch.from_numpy(m.astype(np.uint8)).to(DEV), counters=True)
    torch.cuda.synchronize()
    check(c, m, y, cnt)


@pytest.mark.parametrize("seed", range(8))
def test_int8_random_shapes(seed):
    """Seeded random shapes (d a multiple of 128 up to 8192, k up to 12000,
    1 to 8 tokens, gated or not, alpha from 0.7 to +inf): the device's INT8
    weights and the fused call against the oracle, then a random mask of
    random density through the mask form."""
    rng = np.random.default_rng(5200 + seed)
    d = 128 * int(rng.integers(1, 65))
    k = int(rng.integers(1, min(12000, 4_000_000 // d) + 1))
    b = int(rng.integers(1, 9))
    gated = seed % 3 != 2
    alpha = float(rng.choice([0.7, 1.0, 1.03, 1.45, math.inf]))
    print(f"seed={seed} k={k} d={d} b={b} gated={gated} alpha={alpha}", flush=True)
    c = I8Case(rand_bits(rng, (k, d)), rand_bits(rng, (k, d)) if gated else None, rand_bits(rng, (d, k)),
               rand_bits(rng, (b, d)), max_batch=b)
    check_weights(c)
    fused(c, alpha)
    m = rng.random(k) < rng.uniform(0.02, 1.0)
    m[int(rng.integers(0, k))] = True
    y, cnt = c.layer.sparse_mlp(to_dev(c.x), torch.from_numpy(m.astype(np.uint8)).to(DEV), counters=True)
    torch.cuda.synchronize()
    check(c, m, y, cnt)


def test_int8_rejects_bad_arguments(tiny):
    lib = si._lib.load()
    L = tiny.layer
    ws = L.workspace
    x = to_dev(tiny.x)
    y = torch.empty(1, tiny.d, dtype=torch.float32, device=DEV)
    vp = si._vp
    st = lib.si_predict_sparse_mlp_i8(vp(L.signs), vp(L.q_gate), None, vp(L.q_up), vp(L.s_up), vp(L.q_down_t),
                                      vp(L.s_down), tiny.k, tiny.d, vp(x), 1, 1.0, None, None, None, vp(y), vp(ws),
                                      ws.numel(), 0, None, None)
    assert st == 1  # SI_ERR_NULL: s_gate
    st = lib.si_sparse_mlp_i8(vp(L.q_gate), vp(L.s_gate), vp(L.q_up), vp(L.s_up), vp(L.q_down_t), vp(L.s_down),
                              tiny.k, tiny.d, vp(x), 1, None, vp(y), vp(ws), ws.numel(), 0, None, None)
    assert st == 1  # SI_ERR_NULL: mask
    st = lib.si_predict_sparse_mlp_i8(vp(L.signs), vp(L.q_gate), vp(L.s_gate), vp(L.q_up), vp(L.s_up),
                                      vp(L.q_down_t), vp(L.s_down), tiny.k, tiny.d, vp(x), 1, float("nan"), None,
                                      None, None, vp(y), vp(ws), ws.numel(), 0, None, None)
    assert st == 4  # SI_ERR_ALPHA
    # more than 256 rows per compute unit: the single-launch path does not apply
    k = 65537
    assert lib.si_single_launch(k, 128, 1) == 0
    big = si.new_workspace(k, 128, 1)
    st = lib.si_predict_sparse_mlp_i8(vp(L.signs), vp(L.q_gate), vp(L.s_gate), vp(L.q_up), vp(L.s_up),
                                      vp(L.q_down_t), vp(L.s_down), k, 128, vp(x), 1, 1.0, None, None, None, vp(y),
                                      vp(big), big.numel(), 0, None, None)
    assert st == 2  # SI_ERR_SHAPE
