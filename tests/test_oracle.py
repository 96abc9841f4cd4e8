"""Pins of the CPU oracle against what the paper and the mathematics fix.

Each test checks the oracle against something other than itself: a
hand-worked example (``tests/golden``), the numbers the paper prints, exact
rational brute force (``tests/brute.py``), closed forms, special cases and
invariants of Eq. (1)/(2).
"""

import math
import os

import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

import brute
import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _golden_lines(name):
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                yield line.split()


def _bits(values):
    return np.array([brute.fp16_bits(float(v)) for v in values], dtype=np.uint16)


def _random_bits(rng, shape, special=True):
    """Random finite fp16 bit patterns; with ``special`` also +-0, subnormals
    and the largest finite values."""
    vals = rng.standard_normal(shape).astype(np.float16).view(np.uint16)
    if special:
        pool = np.array([0x0000, 0x8000, 0x0001, 0x8001, 0x03FF, 0x83FF,
                         0x7BFF, 0xFBFF, 0x3C00, 0xBC00], dtype=np.uint16)
        pick = rng.random(shape) < 0.15
        vals = np.where(pick, pool[rng.integers(0, pool.size, size=shape)], vals)
    return vals.astype(np.uint16)


# ---------------------------------------------------------------------------
# Element decoding and packing
# ---------------------------------------------------------------------------

def test_fp16_decode_every_pattern():
    bits = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    got = oracle.fp16_to_f64(bits)
    for b in range(1 << 16):
        want = brute.decode_fp16_by_fields(b)
        if want is None:
            continue
        assert got[b] == want and math.copysign(1, got[b]) == math.copysign(1, want), hex(b)


def test_sign_bits_are_msb():
    bits = np.array([0x0000, 0x8000, 0x3C00, 0xBC00, 0x0001, 0x8001], dtype=np.uint16)
    assert oracle.sign_bits(bits).tolist() == [0, 1, 0, 1, 0, 1]


def test_pack_golden_example():
    rows = {r[0]: r[1:] for r in _golden_lines("pack_example.txt")}
    d = int(rows["d"][0])
    neg = {int(v) for v in rows["negative"]}
    vals = _bits([-1.0 if j in neg else 1.0 for j in range(d)])
    words = [int(w, 16) for w in rows["words"]]
    assert oracle.pack_signs(vals).tolist() == words


@pytest.mark.parametrize("d", [1, 5, 31, 32, 33, 64, 100, 128])
def test_pack_bit_by_bit(d):
    rng = np.random.default_rng(d)
    a = _random_bits(rng, (7, d))
    p = oracle.pack_signs(a)
    assert p.shape == (7, (d + 31) // 32) and p.dtype == np.uint32
    for i in range(7):
        for j in range((d + 31) // 32 * 32):
            bit = (int(p[i, j // 32]) >> (j % 32)) & 1
            want = (int(a[i, j]) >> 15) if j < d else 0
            assert bit == want


# ---------------------------------------------------------------------------
# Counting and Eq. (2)
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("d", [1, 5, 31, 32, 33, 64, 128])
def test_count_matches_elementwise_product_signs(d):
    rng = np.random.default_rng(100 + d)
    k, b = 40, 3
    w = _random_bits(rng, (k, d))
    x = _random_bits(rng, (b, d))
    n_neg, n_pos = oracle.count_sign_products(oracle.pack_signs(w), oracle.pack_signs(x), d)
    for t in range(b):
        for i in range(k):
            want = brute.n_neg(w[i].tolist(), x[t].tolist())
            assert n_neg[t, i] == want
            assert n_pos[t, i] == d - want


def test_eq2_golden_example():
    lines = list(_golden_lines("eq2_worked_example.txt"))
    x = _bits([float(v) for v in lines[0][1:]])
    rows = [l for l in lines if l[0] == "row"]
    w = np.stack([_bits([float(v) for v in r[2:10]]) for r in rows])
    n_neg_want = [int(r[10]) for r in rows]
    g_want = [float(r[11]) for r in rows]
    packed = oracle.pack_signs(w)
    for l in lines:
        if l[0] != "alpha":
            continue
        alpha = float(l[1])
        mask, active, n_neg = oracle.predict_rows(packed, x, alpha)
        assert n_neg[0].tolist() == n_neg_want
        assert mask.tolist() == [int(v) for v in l[2:7]], alpha
    truth = oracle.gate_truly_positive(w, x)[0]
    assert truth.tolist() == [g > 0 for g in g_want]
    for l in lines:
        if l[0] != "quality":
            continue
        alpha = float(l[1])
        _, active, _ = oracle.predict_rows(packed, x, alpha)
        q = oracle.prediction_quality(active[0], truth)
        want = dict(zip(l[2::2], map(float, l[3::2])))
        for key, val in want.items():
            assert q[key] == pytest.approx(val, abs=1e-12), (alpha, key)


ALPHAS = [0.0, 0.5, 0.7, 1.0, 1.01, 1.03, 1.45, 1.5, 2.75, math.inf]


@pytest.mark.parametrize("d", [1, 5, 32, 33, 64, 128])
def test_predict_matches_exact_rational_rule(d):
    rng = np.random.default_rng(200 + d)
    k, b = 48, 2
    w = _random_bits(rng, (k, d))
    x = _random_bits(rng, (b, d))
    packed = oracle.pack_signs(w)
    for alpha in ALPHAS:
        mask, active, _ = oracle.predict_rows(packed, x, alpha)
        bmask, bact = brute.predict(w.tolist(), x.tolist(), alpha)
        assert mask.tolist() == bmask, alpha
        assert active.tolist() == bact, alpha


def test_exact_ties_are_kept():
    # alpha = 1 and N_neg == N_pos: not sparse; one more negative: sparse.
    d = 64
    x = _bits([1.0] * d)
    tie = _bits([-1.0] * 32 + [1.0] * 32)
    over = _bits([-1.0] * 33 + [1.0] * 31)
    w = np.stack([tie, over])
    mask, _, n_neg = oracle.predict_rows(oracle.pack_signs(w), x, 1.0)
    assert n_neg[0].tolist() == [32, 33]
    assert mask.tolist() == [1, 0]
    # alpha = 0.5 (exact in binary): tie at N_neg = d/3 is impossible for d=64,
    # so use d = 48: N_pos = 32, N_neg = 16 -> 0.5*32 == 16 -> kept.
    d = 48
    x = _bits([1.0] * d)
    w = np.stack([_bits([-1.0] * 16 + [1.0] * 32), _bits([-1.0] * 17 + [1.0] * 31)])
    mask, _, _ = oracle.predict_rows(oracle.pack_signs(w), x, 0.5)
    assert mask.tolist() == [1, 0]


def test_alpha_special_cases():
    rng = np.random.default_rng(7)
    d, k = 96, 64
    x = _random_bits(rng, (1, d), special=False)
    w = _random_bits(rng, (k, d), special=False)
    # row 0 agrees with x everywhere, row 1 disagrees everywhere
    w[0] = (w[0] & 0x7FFF) | (x[0] & 0x8000)
    w[1] = (w[1] & 0x7FFF) | (~x[0] & 0x8000)
    packed = oracle.pack_signs(w)
    m_inf, _, _ = oracle.predict_rows(packed, x, math.inf)
    assert m_inf.all()
    m0, _, n_neg = oracle.predict_rows(packed, x, 0.0)
    assert m0.tolist() == (n_neg[0] == 0).astype(np.uint8).tolist()
    for alpha in [0.0, 0.3, 1.0, 7.0, 1e30]:
        m, _, _ = oracle.predict_rows(packed, x, alpha)
        assert m[0] == 1 and m[1] == 0
    with pytest.raises(ValueError):
        oracle.predict_rows(packed, x, -0.5)
    with pytest.raises(ValueError):
        oracle.predict_rows(packed, x, math.nan)


@settings(max_examples=40, deadline=None)
@given(seed=st.integers(0, 2**31 - 1), d=st.sampled_from([3, 32, 47, 64, 130]),
       a1=st.floats(0, 4), a2=st.floats(0, 4))
def test_active_set_grows_with_alpha(seed, d, a1, a2):
    lo, hi = min(a1, a2), max(a1, a2)
    rng = np.random.default_rng(seed)
    w = _random_bits(rng, (32, d))
    x = _random_bits(rng, (2, d))
    packed = oracle.pack_signs(w)
    m_lo, act_lo, _ = oracle.predict_rows(packed, x, lo)
    m_hi, act_hi, _ = oracle.predict_rows(packed, x, hi)
    assert np.all(m_hi >= m_lo)
    assert np.all(act_hi >= act_lo)


def test_batch_mask_is_union_of_tokens():
    rng = np.random.default_rng(11)
    d, k, b = 64, 50, 5
    w = _random_bits(rng, (k, d))
    x = _random_bits(rng, (b, d))
    packed = oracle.pack_signs(w)
    mask, active, _ = oracle.predict_rows(packed, x, 1.0)
    for t in range(b):
        m_t, _, _ = oracle.predict_rows(packed, x[t:t + 1], 1.0)
        assert m_t.tolist() == active[t].astype(np.uint8).tolist()
    assert mask.tolist() == active.any(axis=0).astype(np.uint8).tolist()


def test_one_sign_flip_moves_count_by_one():
    rng = np.random.default_rng(12)
    d, k = 128, 16
    w = _random_bits(rng, (k, d), special=False)
    x = _random_bits(rng, (1, d), special=False)
    _, _, n0 = oracle.predict_rows(oracle.pack_signs(w), x, 1.0)
    for j in [0, 31, 32, 77, 127]:
        w2 = w.copy()
        w2[3, j] ^= 0x8000
        _, _, n1 = oracle.predict_rows(oracle.pack_signs(w2), x, 1.0)
        agreed = ((w[3, j] ^ x[0, j]) & 0x8000) == 0
        assert n1[0, 3] - n0[0, 3] == (1 if agreed else -1)
        assert np.array_equal(np.delete(n1[0], 3), np.delete(n0[0], 3))


@pytest.mark.parametrize("d", [512, 4096, 5120])
def test_integer_percent_form_matches_eq2(d):
    """The printed listing takes alpha as an integer percentage; with the skip
    flag assigned as Eq. (2) and the prose say (sparse iff
    100 * N_neg > alpha_pct * N_pos), it must agree with the float32 route for
    the paper's alphas 1.00 .. 1.03 at every possible N_neg."""
    n_neg = np.arange(d + 1)
    x = np.full((1, d), brute.fp16_bits(1.0), dtype=np.uint16)
    # row r has its first r signs negative -> N_neg = r
    w = np.where(np.arange(d)[None, :] < n_neg[:, None], brute.fp16_bits(-1.0),
                 brute.fp16_bits(1.0)).astype(np.uint16)
    packed = oracle.pack_signs(w)
    for pct in [100, 101, 102, 103]:
        mask, _, got_neg = oracle.predict_rows(packed, x, pct / 100)
        assert got_neg[0].tolist() == n_neg.tolist()
        sparse = 100 * n_neg > pct * (d - n_neg)
        assert mask.tolist() == (~sparse).astype(np.uint8).tolist(), pct


# ---------------------------------------------------------------------------
# Eq. (1) with row skipping
# ---------------------------------------------------------------------------

def test_eq1_golden_example():
    lines = list(_golden_lines("eq1_worked_example.txt"))
    def mat(tokens):
        return [list(map(float, part.split())) for part in " ".join(tokens).split("|")]
    rec = {l[0]: l[1:] for l in lines if l[0] != "case"}
    x = _bits(map(float, rec["x"]))[None, :]
    wg = np.stack([_bits(r) for r in mat(rec["gate"])])
    wu = np.stack([_bits(r) for r in mat(rec["up"])])
    wd = np.stack([_bits(r) for r in mat(rec["down"])])
    assert wg.shape == (3, 2) and wd.shape == (2, 3)
    h3_all = list(map(float, rec["h3"]))
    for l in lines:
        if l[0] != "case":
            continue
        arrow = l.index("->")
        mask = np.array(list(map(int, l[1:arrow])), dtype=np.uint8)
        y0, y1, ng, nu, nd = map(float, l[arrow + 1:])
        out = oracle.sparse_mlp(wg, wu, wd, x, mask)
        assert out["y"][0].tolist() == [y0, y1]
        assert (out["n_gate"], out["n_up"], out["n_down"]) == (ng, nu, nd)
        assert out["h3"][0].tolist() == [h if m else 0.0 for h, m in zip(h3_all, mask)]


@pytest.mark.parametrize("k,d,b", [(5, 3, 1), (17, 8, 2), (33, 16, 1), (24, 40, 3)])
def test_sparse_mlp_matches_exact_rationals(k, d, b):
    rng = np.random.default_rng(k * 100 + d)
    wg = _random_bits(rng, (k, d), special=False)
    wu = _random_bits(rng, (k, d), special=False)
    wd = _random_bits(rng, (d, k), special=False)
    x = _random_bits(rng, (b, d), special=False)
    for mask in [np.ones(k, np.uint8), np.zeros(k, np.uint8),
                 (rng.random(k) < 0.4).astype(np.uint8)]:
        out = oracle.sparse_mlp(wg, wu, wd, x, mask)
        y, g, h3 = brute.mlp(wg.tolist(), wu.tolist(), wd.tolist(), x.tolist(), mask.tolist())
        for t in range(b):
            scale = max(1e-300, max(abs(float(v)) for v in y[t]))
            for c in range(d):
                assert abs(out["y"][t, c] - float(y[t][c])) <= 1e-12 * scale
            for i in range(k):
                assert abs(out["h3"][t, i] - float(h3[t][i])) <= 1e-12 * max(1.0, abs(float(h3[t][i])))
        nz_up = [i for i in range(k) if mask[i] and any(g[t][i] > 0 for t in range(b))]
        nz_dn = [i for i in range(k) if mask[i] and any(h3[t][i] != 0 for t in range(b))]
        assert out["n_gate"] == int(mask.sum())
        assert out["n_up"] == len(nz_up)
        assert out["n_down"] == len(nz_dn)


def test_empty_mask_gives_zero_output():
    rng = np.random.default_rng(3)
    k, d = 20, 16
    out = oracle.sparse_mlp(_random_bits(rng, (k, d)), _random_bits(rng, (k, d)),
                            _random_bits(rng, (d, k)), _random_bits(rng, (2, d)),
                            np.zeros(k, np.uint8))
    assert np.all(out["y"] == 0) and out["y"].shape == (2, d)


def test_linear_in_w_down():
    rng = np.random.default_rng(4)
    k, d = 30, 24
    wg = _random_bits(rng, (k, d), special=False)
    wu = _random_bits(rng, (k, d), special=False)
    wd = _random_bits(rng, (d, k), special=False)
    x = _random_bits(rng, (1, d), special=False)
    mask = (rng.random(k) < 0.5).astype(np.uint8)
    y1 = oracle.sparse_mlp(wg, wu, wd, x, mask)["y"]
    wd2 = (oracle.fp16_to_f64(wd) * 2).astype(np.float16).view(np.uint16)  # exact doubling
    y2 = oracle.sparse_mlp(wg, wu, wd2, x, mask)["y"]
    assert np.allclose(y2, 2 * y1, rtol=1e-13, atol=0)


def test_truth_exact_on_cancellations():
    # g is exactly zero, or positive by one subnormal, or negative by one subnormal
    x = _bits([1.0, 1.0, 1.0])
    w = np.stack([_bits([0.5, -0.5, 0.0]),
                  np.array([brute.fp16_bits(0.5), brute.fp16_bits(-0.5), 0x0001], np.uint16),
                  np.array([brute.fp16_bits(0.5), brute.fp16_bits(-0.5), 0x8001], np.uint16),
                  _bits([60000.0, -60000.0, 0.0])])
    truth = oracle.gate_truly_positive(w, x[None, :])
    assert truth[0].tolist() == [False, True, False, False]
    rng = np.random.default_rng(5)
    wg = _random_bits(rng, (40, 24), special=True)
    xx = _random_bits(rng, (2, 24), special=True)
    assert oracle.gate_truly_positive(wg, xx).tolist() == brute.gate_positive(wg.tolist(), xx.tolist())


# ---------------------------------------------------------------------------
# Numbers printed in Section V-A
# ---------------------------------------------------------------------------

def test_section5_counts():
    g = {r[0]: r[1] for r in _golden_lines("section5_counts.txt")}
    d, k, blocks = int(g["d"]), int(g["k"]), int(g["blocks"])
    assert (d + 31) // 32 == int(g["words_per_row"])
    # the table prints four significant digits (2,211,840 appears as 2.211e6,
    # i.e. truncated): the count must lie within one unit of the last digit
    for count, printed in [(oracle.sign_words(k, d), g["table1_prediction_xor"]),
                           (oracle.dense_mlp_macs(k, d), g["table1_dense_mlp_ops"])]:
        p = float(printed)
        ulp = 10.0 ** (math.floor(math.log10(p)) - 3)
        assert abs(count - p) < ulp, (count, printed)
    assert oracle.signs_bytes(k, d) * blocks / 2**20 == float(g["signs_total_mib"])


def test_alpha_is_the_float32_value():
    # float32(0.7) = 0.699999988... < 0.7: with N_pos = 10 and N_neg = 7 the
    # float32 rule declares the row sparse (6.99999988 < 7), while the decimal
    # 0.7 would give a tie (kept).  The library receives alpha as float32, so
    # the oracle must decide with that value.
    d = 17
    x = _bits([1.0] * d)
    w = _bits([-1.0] * 7 + [1.0] * 10)[None, :]
    mask, _, n_neg = oracle.predict_rows(oracle.pack_signs(w), x, 0.7)
    assert n_neg[0, 0] == 7 and mask[0] == 0
    bmask, _ = brute.predict(w.tolist(), [x.tolist()], 0.7)
    assert bmask == [0]
    # an alpha exactly representable in binary keeps the tie: 0.5 * 14 == 7
    w = _bits([-1.0] * 7 + [1.0] * 14)[None, :]
    mask, _, _ = oracle.predict_rows(oracle.pack_signs(w), _bits([1.0] * 21), 0.5)
    assert mask[0] == 1


def test_exactly_zero_gate_is_not_counted_as_up_work():
    # row 0: g = 0.5 - 0.5 = 0 exactly -> h1 = 0 -> W_up is skipped (actual sparsity)
    # row 1: g = 1 > 0; row 2: g = -1 < 0
    x = _bits([1.0, 1.0])[None, :]
    wg = np.stack([_bits([0.5, -0.5]), _bits([0.5, 0.5]), _bits([-0.5, -0.5])])
    wu = np.stack([_bits([1.0, 2.0]), _bits([0.0, -0.0]), _bits([1.0, 1.0])])
    wd = np.stack([_bits([1.0, 1.0, 1.0]), _bits([2.0, 2.0, 2.0])])
    out = oracle.sparse_mlp(wg, wu, wd, x, np.ones(3, np.uint8))
    assert out["g"][0].tolist() == [0.0, 1.0, -1.0]
    # row 1: h1 = 1 but u = 0 -> h3 = 0 -> W_down^T row skipped
    assert (out["n_gate"], out["n_up"], out["n_down"]) == (3, 1, 0)
    assert np.all(out["y"] == 0)


# ---------------------------------------------------------------------------
# The non-gated ReLU MLP (Section III: blocks without step 2)
# ---------------------------------------------------------------------------

def test_relu_mlp_golden_example():
    lines = list(_golden_lines("relu_mlp_worked_example.txt"))
    def mat(tokens):
        return [list(map(float, part.split())) for part in " ".join(tokens).split("|")]
    rec = {l[0]: l[1:] for l in lines if l[0] != "case"}
    x = _bits(map(float, rec["x"]))[None, :]
    w1 = np.stack([_bits(r) for r in mat(rec["fc1"])])
    wd = np.stack([_bits(r) for r in mat(rec["down"])])
    h_all = list(map(float, rec["h"]))
    for l in lines:
        if l[0] != "case":
            continue
        arrow = l.index("->")
        mask = np.array(list(map(int, l[1:arrow])), dtype=np.uint8)
        y0, y1, ng, nd = map(float, l[arrow + 1:])
        out = oracle.relu_mlp(w1, wd, x, mask)
        assert out["y"][0].tolist() == [y0, y1]
        assert (out["n_gate"], out["n_up"], out["n_down"]) == (ng, 0, nd)
        assert out["h"][0].tolist() == [h if m else 0.0 for h, m in zip(h_all, mask)]


@pytest.mark.parametrize("k,d,b", [(5, 3, 1), (17, 8, 2), (33, 16, 1), (24, 40, 3)])
def test_relu_mlp_matches_exact_rationals(k, d, b):
    rng = np.random.default_rng(k * 100 + d + 7)
    w1 = _random_bits(rng, (k, d), special=False)
    wd = _random_bits(rng, (d, k), special=False)
    x = _random_bits(rng, (b, d), special=False)
    for mask in [np.ones(k, np.uint8), np.zeros(k, np.uint8), (rng.random(k) < 0.4).astype(np.uint8)]:
        out = oracle.relu_mlp(w1, wd, x, mask)
        y, h = brute.relu_mlp(w1.tolist(), wd.tolist(), x.tolist(), mask.tolist())
        for t in range(b):
            scale = max(1e-300, max(abs(float(v)) for v in y[t]))
            for c in range(d):
                assert abs(out["y"][t, c] - float(y[t][c])) <= 1e-12 * scale
            for i in range(k):
                assert abs(out["h"][t, i] - float(h[t][i])) <= 1e-12 * max(1.0, abs(float(h[t][i])))
        assert out["n_gate"] == int(mask.sum())
        assert out["n_down"] == sum(1 for i in range(k) if mask[i] and any(h[t][i] != 0 for t in range(b)))


def test_relu_mlp_is_the_gated_mlp_with_unit_up():
    """With x_0 = 1 in every token and every W_up row the unit vector e_0,
    u = 1 exactly, so the gated MLP of Eq. (1) reduces to the non-gated one
    (h3 = ReLU(g) * 1)."""
    rng = np.random.default_rng(11)
    k, d, b = 40, 24, 3
    w1 = _random_bits(rng, (k, d), special=False)
    wd = _random_bits(rng, (d, k), special=False)
    x = _random_bits(rng, (b, d), special=False)
    x[:, 0] = brute.fp16_bits(1.0)
    wu = np.zeros((k, d), dtype=np.uint16)
    wu[:, 0] = brute.fp16_bits(1.0)
    for mask in [np.ones(k, np.uint8), (rng.random(k) < 0.5).astype(np.uint8)]:
        gated = oracle.sparse_mlp(w1, wu, wd, x, mask)
        plain = oracle.relu_mlp(w1, wd, x, mask)
        assert np.array_equal(gated["u"][:, mask.astype(bool)], np.ones((b, int(mask.sum()))))
        assert np.array_equal(gated["y"], plain["y"])
        assert np.array_equal(gated["h3"], plain["h"])
        assert gated["n_down"] == plain["n_down"]


def test_relu_mlp_superset_of_positive_rows_equals_dense():
    """Dropping only rows whose ReLU output is zero for every token leaves y
    unchanged (the exact truth decides which rows those are)."""
    rng = np.random.default_rng(12)
    k, d, b = 64, 32, 2
    w1 = _random_bits(rng, (k, d), special=False)
    wd = _random_bits(rng, (d, k), special=False)
    x = _random_bits(rng, (b, d), special=False)
    pos = oracle.gate_truly_positive(w1, x).any(axis=0)
    dense = oracle.relu_mlp(w1, wd, x, np.ones(k, np.uint8))
    extra = (rng.random(k) < 0.3)
    part = oracle.relu_mlp(w1, wd, x, (pos | extra).astype(np.uint8))
    assert np.allclose(part["y"], dense["y"], rtol=1e-12, atol=0)
    none = oracle.relu_mlp(w1, wd, x, np.zeros(k, np.uint8))
    assert np.all(none["y"] == 0)


# ---------------------------------------------------------------------------
# The neighbours: RMSNorm producing X, and the residual around the MLP
# ---------------------------------------------------------------------------

def test_rmsnorm_golden_example():
    rec = {l[0]: l[1:] for l in _golden_lines("rmsnorm_worked_example.txt")}
    h = np.array([float(v) for v in rec["h"]], dtype=np.float32)
    w = np.array([float(v) for v in rec["w"]], dtype=np.float32)
    x0 = oracle.rmsnorm_fp16(h, w, 0.0)[0]
    assert [int(v) for v in x0] == [int(v, 16) for v in rec["eps0"]]
    x1 = oracle.rmsnorm_fp16(h, w, 3.75)[0]
    assert int(x1[0]) == int(rec["eps3.75"][0], 16)


def test_rmsnorm_scale_invariance_and_unit_rms():
    rng = np.random.default_rng(21)
    h = rng.standard_normal((3, 256)).astype(np.float32)
    w = rng.standard_normal(256).astype(np.float32)
    x = oracle.rmsnorm_fp16(h, w, 0.0)
    for e in (-6, 3, 20):  # power-of-two scaling is exact, so x is unchanged
        assert np.array_equal(oracle.rmsnorm_fp16(h * np.float32(2.0 ** e), w, 0.0), x)
    signs = np.where(rng.random((2, 64)) < 0.5, -1.0, 1.0).astype(np.float32)  # mean square exactly 1
    wv = rng.standard_normal(64).astype(np.float32)
    assert np.array_equal(oracle.rmsnorm_fp16(signs, wv, 0.0), (signs * wv).astype(np.float16).view(np.uint16))


def test_rmsnorm_sign_is_the_xor_of_the_operand_signs():
    """The predictor reads only the sign of x, which is the XOR of the signs
    of h and w (zeros included), whatever the rounding."""
    rng = np.random.default_rng(22)
    h = rng.standard_normal((4, 512)).astype(np.float32)
    w = rng.standard_normal(512).astype(np.float32)
    h[:, :8] = 0.0
    h[:, 8:16] = -0.0
    h[:, 16:24] *= np.float32(1e-30)  # underflows to a signed zero in fp16
    x = oracle.rmsnorm_fp16(h, w, 1e-6)
    want = np.signbit(h) ^ np.signbit(w)[None, :]
    assert np.array_equal(oracle.sign_bits(x).astype(bool), want)


def test_mlp_block_adds_the_residual():
    rng = np.random.default_rng(23)
    k, d = 48, 64
    wg = _random_bits(rng, (k, d), special=False)
    wu = _random_bits(rng, (k, d), special=False)
    wd = _random_bits(rng, (d, k), special=False)
    h = rng.standard_normal((2, d)).astype(np.float32)
    wn = rng.standard_normal(d).astype(np.float32)
    packed = oracle.pack_signs(wg)
    out = oracle.mlp_block(h, wn, 1e-5, packed, wg, wu, wd, 1.0)
    x = oracle.rmsnorm_fp16(h, wn, 1e-5)
    mask = oracle.predict_rows(packed, x, 1.0)[0]
    assert np.array_equal(out["mask"], mask) and np.array_equal(out["x"], x)
    m = oracle.sparse_mlp(wg, wu, wd, x, mask)["y"]
    assert np.array_equal(out["mlp_y"], m) and np.array_equal(out["y"], h.astype(np.float64) + m)
    zero_down = np.zeros((d, k), np.uint16)
    assert np.array_equal(oracle.mlp_block(h, wn, 1e-5, packed, wg, wu, zero_down, 1.0)["y"], h.astype(np.float64))
    relu = oracle.mlp_block(h, wn, 1e-5, packed, wg, None, wd, 1.0)
    assert np.array_equal(relu["mlp_y"], oracle.relu_mlp(wg, wd, x, mask)["y"])


# ---------------------------------------------------------------------------
# INT8 weights (Section IV-A: only the sign bit is needed, so the predictor
# applies to INT8 weights unchanged)
# ---------------------------------------------------------------------------

def _int8_golden():
    rows = []
    rec = {}
    cases = []
    for l in _golden_lines("int8_worked_example.txt"):
        if l[0] == "qrow":
            arrow, colon = l.index("->"), l.index(":")
            rows.append((list(map(float, l[2:arrow])), float(l[arrow + 1]), list(map(int, l[colon + 1:]))))
        elif l[0] in ("gated", "relu"):
            arrow = l.index("->")
            cases.append((l[0], list(map(int, l[1:arrow])), list(map(float, l[arrow + 1:]))))
        else:
            rec[l[0]] = l[1:]
    return rows, rec, cases


def test_int8_quantization_golden_example():
    rows, _, _ = _int8_golden()
    w = np.stack([_bits(r) for r, _, _ in rows])
    q, s = oracle.quantize_rows_int8(w)
    assert q.dtype == np.int8 and s.dtype == np.float32
    for i, (_, scale, want) in enumerate(rows):
        assert float(s[i]) == scale
        assert q[i].tolist() == want
    # the MSB of an INT8 zero is 0, whatever the sign of the weight it came from
    assert oracle.sign_bits_int8(q)[0].tolist() == [0, 1, 0, 0, 0, 0]


def test_int8_mlp_golden_example():
    _, rec, cases = _int8_golden()
    def mat(tokens):
        return np.array([list(map(int, part.split())) for part in " ".join(tokens).split("|")], dtype=np.int8)
    x = _bits(map(float, rec["x"]))[None, :]
    qg, qu, qd = mat(rec["gate"]), mat(rec["up"]), mat(rec["down"])
    sg, su, sd = (np.array(list(map(float, rec[n])), dtype=np.float32) for n in ("sgate", "sup", "sdown"))
    for kind, mask, (y0, y1, ng, nu, nd) in cases:
        m = np.array(mask, dtype=np.uint8)
        out = oracle.int8_mlp(qg, sg, qu if kind == "gated" else None, su, qd, sd, x, m)
        assert out["y"][0].tolist() == [y0, y1]
        assert (out["n_gate"], out["n_up"], out["n_down"]) == (ng, nu, nd)


@pytest.mark.parametrize("d", [1, 5, 31, 32, 33, 64, 100])
def test_int8_sign_packing_bit_by_bit_and_as_fp16(d):
    rng = np.random.default_rng(300 + d)
    q = rng.integers(-128, 128, size=(6, d)).astype(np.int8)
    q[:, ::3] = 0
    packed = oracle.pack_signs_int8(q)
    for i in range(6):
        for j in range(d):
            assert (int(packed[i, j // 32]) >> (j % 32)) & 1 == (1 if int(q[i, j]) < 0 else 0)
        for j in range(d, 32 * packed.shape[1]):
            assert (int(packed[i, j // 32]) >> (j % 32)) & 1 == 0
    # every INT8 value is an fp16 value with the same sign bit (0 -> +0)
    assert np.array_equal(packed, oracle.pack_signs(q.astype(np.float16)))


def test_int8_quantization_invariants():
    rng = np.random.default_rng(31)
    w = _random_bits(rng, (40, 96), special=True)
    w[3] = 0
    w[4] = 0x8000  # a row of -0
    q, s = oracle.quantize_rows_int8(w)
    W = oracle.fp16_to_f64(w)
    assert np.all(np.abs(q.astype(int)) <= 127)
    nz = np.max(np.abs(W), axis=1) > 0
    assert np.array_equal(nz, s > 0)
    assert np.all(np.max(np.abs(q[nz].astype(int)), axis=1) == 127)
    assert np.all(q[~nz] == 0)
    # rounding to nearest: |w - s q| <= s / 2, up to the float32 quotient's rounding
    err = np.abs(W - oracle.dequantize_int8(q, s))
    assert np.all(err <= s.astype(np.float64)[:, None] * (0.5 + 64 * 2.0 ** -24))
    # the sign survives wherever q is not 0
    qs = q.astype(int)
    assert np.all((qs[qs != 0] < 0) == (W[qs != 0] < 0))


def test_int8_quantization_is_lossless_on_scaled_integers():
    """A row of fp16 values q0 * 2^e with max |q0| = 127 has scale 2^e exactly
    and quantizes back to q0."""
    rng = np.random.default_rng(32)
    q0 = rng.integers(-127, 128, size=(12, 50)).astype(np.int8)
    q0[:, 7] = np.where(rng.random(12) < 0.5, 127, -127)
    e = rng.integers(-12, 3, size=12)
    w = (q0.astype(np.float64) * (2.0 ** e)[:, None]).astype(np.float16)
    assert np.array_equal(w.astype(np.float64), q0.astype(np.float64) * (2.0 ** e)[:, None])
    q, s = oracle.quantize_rows_int8(w)
    assert np.array_equal(q, q0) and np.array_equal(s, (2.0 ** e).astype(np.float32))


@pytest.mark.parametrize("k,d,b", [(24, 24, 1), (40, 16, 3), (17, 64, 2)])
def test_int8_mlp_is_the_fp16_mlp_of_its_dequantized_weights(k, d, b):
    """With power-of-two scales every dequantized weight is an fp16 value, so
    the INT8 MLP must equal the fp16 MLP of those values exactly (per-row
    scales that differ from row to row, and d == k, expose a scale taken along
    the wrong axis)."""
    rng = np.random.default_rng(k * 7 + d)
    qg, qu = (rng.integers(-127, 128, size=(k, d)).astype(np.int8) for _ in range(2))
    qd = rng.integers(-127, 128, size=(d, k)).astype(np.int8)
    sg, su = ((2.0 ** rng.integers(-9, 1, size=k)).astype(np.float32) for _ in range(2))
    sd = (2.0 ** rng.integers(-9, 1, size=d)).astype(np.float32)
    fp = [(oracle.dequantize_int8(q, s)).astype(np.float16) for q, s in ((qg, sg), (qu, su), (qd, sd))]
    x = _random_bits(rng, (b, d), special=False)
    for mask in [np.ones(k, np.uint8), (rng.random(k) < 0.4).astype(np.uint8), np.zeros(k, np.uint8)]:
        a = oracle.int8_mlp(qg, sg, qu, su, qd, sd, x, mask)
        r = oracle.sparse_mlp(fp[0], fp[1], fp[2], x, mask)
        assert np.array_equal(a["y"], r["y"]) and np.array_equal(a["h3"], r["h3"])
        assert (a["n_gate"], a["n_up"], a["n_down"]) == (r["n_gate"], r["n_up"], r["n_down"])
        a = oracle.int8_mlp(qg, sg, None, None, qd, sd, x, mask)
        r = oracle.relu_mlp(fp[0], fp[2], x, mask)
        assert np.array_equal(a["y"], r["y"]) and np.array_equal(a["h3"], r["h"])
        assert (a["n_gate"], a["n_up"], a["n_down"]) == (r["n_gate"], 0, r["n_down"])
