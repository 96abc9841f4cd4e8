"""The bound of ``tests/test_gpu_down_wide.py`` catches the plausible mistakes
of a down-projection that carries h3 as scaled fp16 parts.

The arithmetic of the kernel is simulated on the CPU in numpy (float32 and
float16 casts, float64 sums): each token's h3 over chunks of 32 kept rows,
multiplied by the power of two that puts the chunk's largest |h3| in
[2^14, 2^15), split into hi = fp16(v) and lo = fp16(v - hi).  That passes the
bound; keeping only hi (2^-12 per term), or rounding h3 to fp16 without the
scale (overflow to inf, underflow to 0), must not.
"""

import numpy as np

import oracle
from test_gpu_down_wide import group_depth, one_hot_tokens, scaled_rows, y_bound


def represented(h3, mode):
    """h3 ``[b][n]`` float64 as the down-projection would carry it."""
    out = np.empty_like(h3)
    for t in range(h3.shape[0]):
        for c0 in range(0, h3.shape[1], 32):
            v = h3[t, c0:c0 + 32]
            if mode == "fp16":
                out[t, c0:c0 + 32] = v.astype(np.float32).astype(np.float16).astype(np.float64)
                continue
            m = np.abs(v).max()
            if m == 0:
                out[t, c0:c0 + 32] = 0.0
                continue
            e = int(np.floor(np.log2(m)))
            s = 2.0 ** (14 - e)
            vs = (v * s).astype(np.float32)
            hi = vs.astype(np.float16).astype(np.float32)
            lo = (vs - hi).astype(np.float16).astype(np.float32)
            kept = hi + lo if mode == "hi+lo" else hi
            out[t, c0:c0 + 32] = kept.astype(np.float64) / s
    return out


def case(seed, d=640, k=3000, b=8):
    rng = np.random.default_rng(seed)
    wg = scaled_rows(rng, k, d, -10, 10)
    wu = scaled_rows(rng, k, d, -10, 10)
    wd = rng.standard_normal((d, k)).astype(np.float16).view(np.uint16)
    x = one_hot_tokens(rng, b, d)
    mask = (rng.random(k) < 0.7).astype(np.uint8)
    out = oracle.sparse_mlp(wg, wu, wd, x, mask)
    keep = oracle.active_rows(mask)
    h3 = np.asarray(out["h3"])[:, keep].astype(np.float32).astype(np.float64)  # h3's own rounding
    WdT = oracle.fp16_to_f64(wd[:, keep]).T
    return out["y"], h3, WdT, y_bound(out["h3"][:, keep], WdT, group_depth(k, d, 256))


def test_hi_lo_within_bound():
    for seed in range(3):
        y, h3, WdT, bound = case(seed)
        err = np.abs(represented(h3, "hi+lo") @ WdT - y)
        assert np.all(err <= bound), float((err / bound).max())


def test_hi_only_exceeds_bound():
    y, h3, WdT, bound = case(11)
    err = np.abs(represented(h3, "hi") @ WdT - y)
    assert (err > bound).mean() > 0.1, float((err / bound).max())


def test_unscaled_fp16_exceeds_bound():
    y, h3, WdT, bound = case(12)
    with np.errstate(over="ignore", invalid="ignore"):
        err = np.abs(represented(h3, "fp16") @ WdT - y)
    assert np.any(~(err <= bound))
