"""Parity of the HIP path (through the C ABI) with the CPU oracle.

Bars: packed signs, masks, kept lists and counts bit-exact; y within 1e-2
relative L2 (fp16 weights, fp32 accumulation; the observed error is ~1e-6,
which the tighter secondary bound below keeps honest); work counters exact
for n_gate and within a few rows for n_up / n_down (rows whose gate value is
within fp32 rounding of zero may fall either way).
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

ALPHAS = [0.0, 0.7, 1.0, 1.03, 1.45, 1.5, math.inf]
DEV = "cuda"


def u16(t: torch.Tensor) -> np.ndarray:
    return t.detach().cpu().contiguous().view(torch.int16).numpy().view(np.uint16)


def rand_bits(rng, shape, special=True):
    vals = rng.standard_normal(shape).astype(np.float16).view(np.uint16)
    if special:
        pool = np.array([0x0000, 0x8000, 0x0001, 0x8001, 0x03FF, 0x7BFF, 0xFBFF], dtype=np.uint16)
        pick = rng.random(shape) < 0.1
        vals = np.where(pick, pool[rng.integers(0, pool.size, size=shape)], vals)
    return vals.astype(np.uint16)


def to_dev(a: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(a.view(np.int16).copy()).to(DEV)


class Case:
    """Host arrays (fp16 bits) of one layer plus its device state."""

    def __init__(self, wg, wu, wd, x, max_batch=1):
        self.wg, self.wu, self.wd, self.x = wg, wu, wd, x
        self.k, self.d = wg.shape
        self.layer = si.MLPLayer(to_dev(wg), to_dev(wu), to_dev(wd), max_batch=max_batch)
        self.packed = oracle.pack_signs(wg)

    @classmethod
    def planted(cls, d, k, s, config, layer=0, b=1):
        L = synth.planted_layer(d, k, s, config=config, layer=layer)
        x = synth.batch_tokens(L, b, config=config)
        return cls(u16(L.w_gate), u16(L.w_up), u16(L.w_down), u16(x), max_batch=b)


def rel_l2(a, b):
    nb = np.linalg.norm(b)
    return float(np.linalg.norm(a - b) / nb) if nb > 0 else float(np.linalg.norm(a))


def check_predict(c: Case, x, alpha):
    xd = to_dev(x)
    mask, idx, n = c.layer.predict(xd, alpha)
    sentinel = -7
    idx.fill_(sentinel)
    mask, idx2, n = si.predict(c.layer.signs, xd, alpha, c.k, c.layer.workspace)
    # run again into a pre-filled list to check nothing past n is written
    idx3 = torch.full((c.k,), sentinel, dtype=torch.int32, device=DEV)
    nn3 = torch.zeros(1, dtype=torch.int32, device=DEV)
    si._lib.call("si_predict", si._vp(c.layer.signs), c.k, c.d, si._vp(xd), x.shape[0], float(alpha),
                 si._vp(mask), si._vp(idx3), si._vp(nn3), si._vp(c.layer.workspace), c.layer.workspace.numel(),
                 si._stream())
    torch.cuda.synchronize()
    m_ref, act_ref, _ = oracle.predict_rows(c.packed, x, alpha)
    m = mask.cpu().numpy()
    assert np.array_equal(m, m_ref), f"alpha={alpha}: {int((m != m_ref).sum())} rows differ"
    nref = int(m_ref.sum())
    assert int(n.item()) == nref and int(nn3.item()) == nref
    ref_idx = oracle.active_rows(m_ref)
    assert np.array_equal(idx2.cpu().numpy()[:nref], ref_idx)
    i3 = idx3.cpu().numpy()
    assert np.array_equal(i3[:nref], ref_idx)
    assert np.all(i3[nref:] == sentinel)
    return m_ref


def device_errors(ws: torch.Tensor) -> int:
    """Status of the sticky device-side error word the kernels keep in the
    workspace header (a wait that hit its spin limit, an out-of-range row),
    through ``si_workspace_check``: 0 = SI_OK."""
    return si.workspace_check(ws)


def check_list(idx, n, mask_ref):
    """The fused call's ascending kept list and count, bit-exact."""
    nref = int(mask_ref.sum())
    assert int(n.item()) == nref
    assert np.array_equal(idx.cpu().numpy()[:nref], oracle.active_rows(mask_ref))


def check_mlp(c: Case, x, mask_ref, y, counters=None, flags=0, h3=True):
    """y, the work counters and (``h3``: the MLP call with this mask was the
    last call on the layer's workspace) the per-row h3 against the oracle."""
    assert device_errors(c.layer.workspace) == 0
    out = oracle.sparse_mlp(c.wg, c.wu, c.wd, x, mask_ref)
    if h3:
        X = oracle.fp16_to_f64(np.atleast_2d(x))
        check_h3(c.layer.workspace, c.k, c.d, X.shape[0], mask_ref, out["h3"], X, fp16_rows(c.wg), fp16_rows(c.wu),
                 out["g"])
    yr = out["y"]
    yg = y.cpu().numpy().astype(np.float64)
    err = rel_l2(yg, yr)
    assert err <= 1e-2, err
    scale = max(np.abs(yr).max(), 1e-30)
    assert np.abs(yg - yr).max() <= 1e-4 * scale + 1e-30, np.abs(yg - yr).max() / scale
    if counters is not None:
        cnt = counters.cpu().numpy().tolist()
        ng = out["n_gate"]
        assert cnt[0] == ng
        if flags & si.SI_NO_AS:
            assert cnt[1] == cnt[2] == ng
        elif flags & si.SI_NO_SPECULATION:
            # rows read exactly where the values say so, up to rows whose gate
            # value is within fp32 rounding of zero
            assert abs(cnt[1] - out["n_up"]) <= 3, (cnt, out["n_up"])
            assert abs(cnt[2] - out["n_down"]) <= 3, (cnt, out["n_down"])
        else:
            # speculative requests may read more rows, never fewer
            assert out["n_up"] - 3 <= cnt[1] <= ng, (cnt, out["n_up"])
            assert out["n_down"] - 3 <= cnt[2] <= ng, (cnt, out["n_down"])
    return out


# ---------------------------------------------------------------------------
# load-time steps
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("k,d", [(1, 128), (63, 128), (65, 256), (1376, 512), (200, 640), (300, 5120),
                                 (70, 8192), (11008, 4096)])
def test_pack_signs_bit_exact(k, d):
    rng = np.random.default_rng(k + d)
    w = rand_bits(rng, (k, d))
    signs = si.pack_signs(to_dev(w))
    can = si.signs_to_canonical(signs, k, d).cpu().numpy().view(np.uint32)
    assert np.array_equal(can, oracle.pack_signs(w))


@pytest.mark.parametrize("d,k", [(128, 1), (256, 65), (512, 1376), (640, 200), (4096, 300)])
def test_transpose_exact(d, k):
    rng = np.random.default_rng(d * 7 + k)
    w = rand_bits(rng, (d, k))
    out = si.transpose_down(to_dev(w))
    assert np.array_equal(u16(out), w.T)


# ---------------------------------------------------------------------------
# predictor
# ---------------------------------------------------------------------------

@pytest.fixture(scope="module")
def tiny():
    return Case.planted(512, 1376, 0.9, config=1)


@pytest.mark.parametrize("alpha", ALPHAS)
def test_predict_tiny_all_alphas(tiny, alpha):
    check_predict(tiny, tiny.x, alpha)


def test_predict_random_with_special_values():
    rng = np.random.default_rng(5)
    wg = rand_bits(rng, (1000, 640))
    c = Case(wg, rand_bits(rng, (1000, 640)), rand_bits(rng, (640, 1000)), rand_bits(rng, (3, 640)), max_batch=3)
    for alpha in [0.0, 0.9, 1.0, 1.1, math.inf]:
        check_predict(c, c.x, alpha)
        check_predict(c, c.x[:1], alpha)


def test_predict_repeated_calls_share_workspace(tiny):
    for alpha in [1.0, 0.7, 1.5, 1.0, math.inf, 1.03]:
        check_predict(tiny, tiny.x, alpha)


@pytest.mark.parametrize("k,d", [(1, 128), (63, 128), (64, 128), (65, 384), (129, 8192), (4097, 1024)])
def test_predict_edge_shapes(k, d):
    rng = np.random.default_rng(k * 31 + d)
    c = Case(rand_bits(rng, (k, d)), rand_bits(rng, (k, d)), rand_bits(rng, (d, k)), rand_bits(rng, (2, d)),
             max_batch=2)
    for alpha in [0.0, 1.0, 1.2]:
        check_predict(c, c.x, alpha)


# ---------------------------------------------------------------------------
# sparse MLP
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("alpha", ALPHAS)
def test_sparse_mlp_tiny_all_alphas(tiny, alpha):
    x = to_dev(tiny.x)
    y, (mask, idx, n, cnt) = tiny.layer(x, alpha, outputs=True)
    torch.cuda.synchronize()
    m_ref, _, _ = oracle.predict_rows(tiny.packed, tiny.x, alpha)
    assert np.array_equal(mask.cpu().numpy(), m_ref)
    check_list(idx, n, m_ref)
    check_mlp(tiny, tiny.x, m_ref, y, cnt)


def test_separate_calls_match_fused(tiny):
    x = to_dev(tiny.x)
    mask, idx, n = tiny.layer.predict(x, 1.0)
    y1, c1 = tiny.layer.sparse_mlp(x, mask, idx, n, counters=True)
    y2 = tiny.layer.sparse_mlp(x, mask=mask)  # list built from the mask
    y3 = tiny.layer(x, 1.0)
    torch.cuda.synchronize()
    m_ref = oracle.predict_rows(tiny.packed, tiny.x, 1.0)[0]
    for y in (y1, y2, y3):
        check_mlp(tiny, tiny.x, m_ref, y)  # h3: of the fused call, the last one (same rows as the others)
    assert torch.allclose(y1, y3, rtol=1e-5, atol=1e-6)


def test_empty_and_full_masks(tiny):
    x = to_dev(tiny.x)
    zero = torch.zeros(tiny.k, dtype=torch.uint8, device=DEV)
    y, cnt = tiny.layer.sparse_mlp(x, mask=zero, counters=True)
    torch.cuda.synchronize()
    assert torch.count_nonzero(y).item() == 0
    assert cnt.tolist() == [0, 0, 0]
    ones = torch.ones(tiny.k, dtype=torch.uint8, device=DEV)
    y, cnt = tiny.layer.sparse_mlp(x, mask=ones, counters=True)
    torch.cuda.synchronize()
    check_mlp(tiny, tiny.x, np.ones(tiny.k, np.uint8), y, cnt)


@pytest.mark.parametrize("flags", [si.SI_NO_AS, si.SI_NO_SPECULATION, si.SI_NO_AS | si.SI_NO_SPECULATION])
def test_work_flags(tiny, flags):
    x = to_dev(tiny.x)
    for alpha in [1.0, 1.5, math.inf]:
        y, (mask, _, _, cnt) = tiny.layer(x, alpha, flags=flags, outputs=True)
        torch.cuda.synchronize()
        m_ref = oracle.predict_rows(tiny.packed, tiny.x, alpha)[0]
        check_mlp(tiny, tiny.x, m_ref, y, cnt, flags=flags)


def test_work_flags_7b(l7b):
    x = to_dev(l7b.x)
    for flags in [si.SI_NO_SPECULATION, si.SI_NO_AS]:
        y, (mask, _, _, cnt) = l7b.layer(x, 1.45, flags=flags, outputs=True)
        torch.cuda.synchronize()
        m_ref = oracle.predict_rows(l7b.packed, l7b.x, 1.45)[0]
        check_mlp(l7b, l7b.x, m_ref, y, cnt, flags=flags)


def test_repeated_layer_calls_are_reproducible(l7b):
    """Masks and kept lists are identical call after call; y agrees to fp32
    summation order (the down-projection adds tiles with atomics)."""
    x = to_dev(l7b.x)
    first = None
    for _ in range(5):
        y, (mask, idx, n, cnt) = l7b.layer(x, 1.0, outputs=True)
        torch.cuda.synchronize()
        cur = (mask.clone(), idx[: int(n.item())].clone(), y.clone(), cnt.clone())
        if first is None:
            first = cur
            continue
        assert torch.equal(cur[0], first[0]) and torch.equal(cur[1], first[1]) and torch.equal(cur[3], first[3])
        scale = first[2].abs().max().item()
        assert (cur[2] - first[2]).abs().max().item() <= 1e-5 * scale
    assert device_errors(l7b.layer.workspace) == 0


@pytest.mark.parametrize("b", [2, 3, 8])
def test_batch_union(b):
    c = Case.planted(512, 1376, 0.9, config=1, b=b)
    x = to_dev(c.x)
    for alpha in [1.0, 1.45]:
        m_ref = check_predict(c, c.x, alpha)
        y, (mask, idx, n, cnt) = c.layer(x, alpha, outputs=True)
        torch.cuda.synchronize()
        assert np.array_equal(mask.cpu().numpy(), m_ref)
        check_list(idx, n, m_ref)
        check_mlp(c, c.x, m_ref, y, cnt)


@pytest.mark.parametrize("k,d,b", [(1000, 640, 3), (1000, 640, 4), (2500, 1152, 3), (700, 8192, 4)])
def test_batch_token_staging_ragged(k, d, b):
    """3-4 tokens, whose token block is copied from memory straight into LDS:
    units past d (d = 640: 80 units of 128 per token; d = 1152: 144 of 192)
    and the missing fourth token must read as zero in every form."""
    rng = np.random.default_rng(k + d + 31 * b)
    c = Case(rand_bits(rng, (k, d), False), rand_bits(rng, (k, d), False), rand_bits(rng, (d, k), False),
             rand_bits(rng, (b, d), False), max_batch=b)
    x = to_dev(c.x)
    for alpha in [1.0, math.inf]:
        m_ref = check_predict(c, c.x, alpha)
        y, (mask, idx, n, cnt) = c.layer(x, alpha, outputs=True)
        torch.cuda.synchronize()
        assert np.array_equal(mask.cpu().numpy(), m_ref)
        check_list(idx, n, m_ref)
        check_mlp(c, c.x, m_ref, y, cnt)
    m = rng.random(k) < 0.4
    y1, c1 = c.layer.sparse_mlp(x, mask=torch.from_numpy(m.astype(np.uint8)).to(DEV), counters=True)
    torch.cuda.synchronize()
    check_mlp(c, c.x, m, y1, c1)


@pytest.mark.parametrize("b", [4, 5, 8])
def test_batch_7b_fused(b):
    """The fused call at the 7B shape with 4 to 8 tokens.  With 5 or more,
    every kept row's W_up and W_down^T rows are requested before its gate
    result: rows whose ReLU output turns out zero must add nothing to y, and
    the read counters may exceed the oracle's n_up and n_down but never
    n_gate."""
    c = Case.planted(4096, 11008, 0.9, config=2, b=b)
    m_ref = check_predict(c, c.x, 1.0)
    y, (mask, idx, n, cnt) = c.layer(to_dev(c.x), 1.0, outputs=True)
    torch.cuda.synchronize()
    assert np.array_equal(mask.cpu().numpy(), m_ref)
    check_list(idx, n, m_ref)
    check_mlp(c, c.x, m_ref, y, cnt)


@pytest.mark.parametrize("b", [5, 8])
def test_list_form_batch_7b(b):
    """The list form with 5 to 8 tokens at the 7B shape (there the list is
    turned into a mask in the workspace for the row-owning kernel): a call
    with every row listed, then one with the predicted rows and garbage past
    n, must each give the oracle's result on its own rows."""
    c = Case.planted(4096, 11008, 0.9, config=2, b=b)
    x = to_dev(c.x)
    m_ref = oracle.predict_rows(c.packed, c.x, 1.0)[0]
    all_idx = torch.arange(c.k, dtype=torch.int32, device=DEV)
    all_n = torch.tensor([c.k], dtype=torch.int32, device=DEV)
    y0, c0 = c.layer.sparse_mlp(x, None, all_idx, all_n, counters=True)
    torch.cuda.synchronize()
    check_mlp(c, c.x, np.ones(c.k, dtype=bool), y0, c0)
    rows = np.flatnonzero(m_ref)
    idx = np.full(c.k, c.k + 5, dtype=np.int32)
    idx[rows.size:] = np.where(np.arange(c.k - rows.size) % 2 == 0, -7, c.k + 5)
    idx[: rows.size] = rows
    y1, c1 = c.layer.sparse_mlp(x, None, torch.from_numpy(idx).to(DEV),
                                torch.tensor([rows.size], dtype=torch.int32, device=DEV), counters=True)
    torch.cuda.synchronize()
    check_mlp(c, c.x, m_ref, y1, c1)


@pytest.mark.parametrize("k,d,b", [(700, 8192, 5), (700, 8192, 8), (1500, 5120, 8), (1300, 4096, 7)])
def test_batch_wide_rows(k, d, b):
    """Batches of 5 to 8 tokens with the widest rows: the token block fills
    most of the LDS and the per-token accumulators most of the registers."""
    rng = np.random.default_rng(k * 13 + d + b)
    c = Case(rand_bits(rng, (k, d), False), rand_bits(rng, (k, d), False), rand_bits(rng, (d, k), False),
             rand_bits(rng, (b, d), False), max_batch=b)
    for alpha in [1.0, math.inf]:
        m_ref = check_predict(c, c.x, alpha)
        y, (mask, idx, n, cnt) = c.layer(to_dev(c.x), alpha, outputs=True)
        torch.cuda.synchronize()
        assert np.array_equal(mask.cpu().numpy(), m_ref)
        check_list(idx, n, m_ref)
        check_mlp(c, c.x, m_ref, y, cnt)
        # the list-driven and the mask-driven sparse MLP on the same rows
        y1, c1 = c.layer.sparse_mlp(to_dev(c.x), mask, idx, n, counters=True)
        torch.cuda.synchronize()
        check_mlp(c, c.x, m_ref, y1, c1)
        y2, c2 = c.layer.sparse_mlp(to_dev(c.x), mask=mask, counters=True)
        torch.cuda.synchronize()
        check_mlp(c, c.x, m_ref, y2, c2)


@pytest.mark.parametrize("seed", range(12))
def test_random_shapes_every_form(seed):
    """Seeded random shapes (d a multiple of 128 up to 8192, k up to 20000,
    1 to 8 tokens, alpha from 0.7 to +inf): the fused call against the
    oracle's prediction and MLP, then a random mask of random density through
    the mask form and the same rows through the list form."""
    rng = np.random.default_rng(4100 + seed)
    d = 128 * int(rng.integers(1, 65))
    k = int(rng.integers(1, min(20000, 6_000_000 // d) + 1))
    b = int(rng.integers(1, 9))
    alpha = float(rng.choice([0.7, 1.0, 1.03, 1.45, math.inf]))
    print(f"seed={seed} k={k} d={d} b={b} alpha={alpha}", flush=True)
    c = Case(rand_bits(rng, (k, d), False), rand_bits(rng, (k, d), False), rand_bits(rng, (d, k), False),
             rand_bits(rng, (b, d), seed % 2 == 0), max_batch=b)
    x = to_dev(c.x)
    y, (mask, idx, n, cnt) = c.layer(x, alpha, outputs=True)
    torch.cuda.synchronize()
    m_ref = oracle.predict_rows(c.packed, c.x, alpha)[0]
    assert np.array_equal(mask.cpu().numpy(), m_ref)
    check_list(idx, n, m_ref)
    if m_ref.any():
        check_mlp(c, c.x, m_ref, y, cnt)
    m = rng.random(k) < rng.uniform(0.02, 1.0)
    m[int(rng.integers(0, k))] = True
    rows = np.flatnonzero(m).astype(np.int32)
    y1, c1 = c.layer.sparse_mlp(x, mask=torch.from_numpy(m.astype(np.uint8)).to(DEV), counters=True)
    torch.cuda.synchronize()
    check_mlp(c, c.x, m, y1, c1)
    lst = np.full(k, -1, dtype=np.int32)
    lst[: rows.size] = rows
    y2, c2 = c.layer.sparse_mlp(x, None, torch.from_numpy(lst).to(DEV),
                                torch.tensor([rows.size], dtype=torch.int32, device=DEV), counters=True)
    torch.cuda.synchronize()
    check_mlp(c, c.x, m, y2, c2)


@pytest.mark.parametrize("k,d", [(1, 128), (63, 128), (65, 384), (129, 8192), (1000, 640), (1, 8192),
                                 (20000, 384), (65536, 128)])
def test_sparse_mlp_edge_shapes(k, d):
    """Ragged tails of rows, pieces and tiles; k = 20000 and 65536 give more
    64-row groups than there are blocks (several groups per block)."""
    rng = np.random.default_rng(k * 17 + d)
    c = Case(rand_bits(rng, (k, d), False), rand_bits(rng, (k, d), False), rand_bits(rng, (d, k), False),
             rand_bits(rng, (1, d), False))
    for alpha in [1.0, math.inf]:
        y, (mask, idx, n, cnt) = c.layer(to_dev(c.x), alpha, outputs=True)
        torch.cuda.synchronize()
        m_ref = oracle.predict_rows(c.packed, c.x, alpha)[0]
        assert np.array_equal(mask.cpu().numpy(), m_ref)
        check_list(idx, n, m_ref)
        if m_ref.any():
            check_mlp(c, c.x, m_ref, y, cnt)


# ---------------------------------------------------------------------------
# full-size layers (7B and 13B shapes)
# ---------------------------------------------------------------------------

@pytest.fixture(scope="module")
def l7b():
    return Case.planted(4096, 11008, 0.9, config=2)


@pytest.mark.parametrize("alpha", [0.7, 1.0, 1.03, 1.45, 1.5])
def test_7b_layer(l7b, alpha):
    x = to_dev(l7b.x)
    m_ref = check_predict(l7b, l7b.x, alpha)
    y, (mask, idx, n, cnt) = l7b.layer(x, alpha, outputs=True)
    torch.cuda.synchronize()
    assert np.array_equal(mask.cpu().numpy(), m_ref)
    check_list(idx, n, m_ref)
    check_mlp(l7b, l7b.x, m_ref, y, cnt)


def test_13b_layer():
    c = Case.planted(5120, 13824, 0.88, config=4)
    x = to_dev(c.x)
    m_ref = check_predict(c, c.x, 1.0)
    y, (mask, idx, n, cnt) = c.layer(x, 1.0, outputs=True)
    torch.cuda.synchronize()
    assert np.array_equal(mask.cpu().numpy(), m_ref)
    check_list(idx, n, m_ref)
    check_mlp(c, c.x, m_ref, y, cnt)


def group_rows(k, d):
    """Rows of one group of the one-launch kernel: groups of T = ceil(d / 512)
    blocks over the device's compute units, R rows per block (the rows spread
    over the grid's whole groups, rounded up to a multiple of 8)."""
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    T = (d + 511) // 512
    working = cus // T * T
    return T * (((k + working - 1) // working + 7) // 8 * 8)


@pytest.mark.parametrize("k,d", [(9000, 8192), (40000, 2048)])
def test_one_token_large_groups(k, d):
    """One token with groups of more than 512 rows takes the kernel instance
    with the wider down batches (12 pieces instead of 10): every form at
    alpha = 1 and +inf (all rows kept: the most rounds), a random mask and
    list, and without speculation.  9000 x 8192 leaves a last group of 40
    rows; 40000 x 2048 half a group."""
    assert group_rows(k, d) > 512
    rng = np.random.default_rng(k + 3 * d)
    c = Case(rand_bits(rng, (k, d), False), rand_bits(rng, (k, d), False), rand_bits(rng, (d, k), False),
             rand_bits(rng, (1, d), False))
    x = to_dev(c.x)
    for alpha, flags in [(1.0, 0), (math.inf, 0), (1.0, si.SI_NO_SPECULATION), (math.inf, si.SI_NO_SPECULATION)]:
        print(f"k={k} d={d} alpha={alpha} flags={flags}", flush=True)
        y, (mask, idx, n, cnt) = c.layer(x, alpha, flags=flags, outputs=True)
        torch.cuda.synchronize()
        m_ref = oracle.predict_rows(c.packed, c.x, alpha)[0]
        assert np.array_equal(mask.cpu().numpy(), m_ref)
        check_list(idx, n, m_ref)
        check_mlp(c, c.x, m_ref, y, cnt, flags=flags)
    m = rng.random(k) < 0.3
    rows = np.flatnonzero(m).astype(np.int32)
    y1, c1 = c.layer.sparse_mlp(x, mask=torch.from_numpy(m.astype(np.uint8)).to(DEV), counters=True)
    torch.cuda.synchronize()
    check_mlp(c, c.x, m, y1, c1)
    lst = np.full(k, -1, dtype=np.int32)
    lst[: rows.size] = rows
    y2, c2 = c.layer.sparse_mlp(x, None, torch.from_numpy(lst).to(DEV),
                                torch.tensor([rows.size], dtype=torch.int32, device=DEV), counters=True)
    torch.cuda.synchronize()
    check_mlp(c, c.x, m, y2, c2)


@pytest.mark.parametrize("k,d,b,one", [(11008, 4096, 1, 1), (13824, 5120, 1, 1), (1376, 512, 1, 1),
                                       (11008, 4096, 2, 1), (1, 128, 1, 1), (65536, 128, 1, 1),
                                       (11008, 4096, 3, 1), (11008, 4096, 8, 1), (13824, 5120, 8, 1),
                                       (129, 8192, 4, 1), (129, 8192, 5, 1), (700, 8192, 8, 1),
                                       (65537, 128, 1, 0), (11008, 4096, 9, 0)])
def test_single_launch_path(k, d, b, one):
    """The shapes the parity tests use run the one-launch kernel (so its
    results are the ones checked); k above 65536 (256 rows per compute unit)
    takes the two-launch path, and batches above 8 are rejected."""
    assert si._lib.load().si_single_launch(k, d, b) == one


@pytest.mark.parametrize("flags", [0, si.SI_NO_SPECULATION])
def test_first_call_on_a_fresh_workspace(flags):
    """The exchange words between blocks are tagged with a per-call counter
    that starts at zero; the first call on a zero-filled workspace must not
    take zero-filled words for published ones."""
    c = Case.planted(4096, 11008, 0.9, config=2, layer=3)
    y, (mask, idx, n, cnt) = c.layer(to_dev(c.x), 1.0, flags=flags, outputs=True)
    torch.cuda.synchronize()
    m_ref = oracle.predict_rows(c.packed, c.x, 1.0)[0]
    assert np.array_equal(mask.cpu().numpy(), m_ref)
    check_mlp(c, c.x, m_ref, y, cnt, flags=flags)


@pytest.mark.parametrize("b", [1, 3])
def test_multi_launch_gated_every_form(b):
    """Above 256 rows per compute unit (k = 65600 at d = 128) every gated call
    takes the multi-launch path: the predictor alone, the fused predict +
    gate/up followed by the down-projection, and the mask and list forms of
    the sparse MLP.  Masks, lists and counts bit-exact, y and the h3 of every
    kept row against the oracle at alpha = 1 and +inf.  This path keeps h3 as
    plain floats in the workspace, so the workspace is zero-filled before
    each MLP call: no value of an earlier call can pass for this one's."""
    k, d = 65600, 128
    assert si._lib.load().si_single_launch(k, d, b) == 0
    rng = np.random.default_rng(65600 + b)
    c = Case(rand_bits(rng, (k, d), False), rand_bits(rng, (k, d), False), rand_bits(rng, (d, k), False),
             rand_bits(rng, (b, d), False), max_batch=b)
    x = to_dev(c.x)
    for alpha in [1.0, math.inf]:
        print(f"multi-launch k={k} d={d} b={b} alpha={alpha}", flush=True)
        m_ref = check_predict(c, c.x, alpha)
        c.layer.workspace.zero_()
        y, (mask, idx, n, cnt) = c.layer(x, alpha, outputs=True)
        torch.cuda.synchronize()
        assert np.array_equal(mask.cpu().numpy(), m_ref)
        check_list(idx, n, m_ref)
        check_mlp(c, c.x, m_ref, y, cnt)
        c.layer.workspace.zero_()
        y1, c1 = c.layer.sparse_mlp(x, mask=mask, counters=True)
        torch.cuda.synchronize()
        check_mlp(c, c.x, m_ref, y1, c1)
        c.layer.workspace.zero_()
        y2, c2 = c.layer.sparse_mlp(x, mask, idx, n, counters=True)
        torch.cuda.synchronize()
        check_mlp(c, c.x, m_ref, y2, c2)
