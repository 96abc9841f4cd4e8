"""The down-projection (Eq. (1) step 4) with h3 far outside fp16's range.

With 4-8 tokens the row-owning kernel runs the down-projection on fp16
matrix-core instructions, each h3 carried as two fp16 parts (hi, lo) after a
power-of-two scale chosen per token and chunk of 32 rows; with 1-2 tokens,
or without speculation, on fp32 FMAs.  Here every token is one-hot (one
element +-2^a, a in [-6, 6]) and the W_gate and W_up rows are scaled by 2^e
(e in [-10, 10]), so g and u are single exact products and h3 = ReLU(g) u
carries one rounding, while spanning about 2^-40 .. 2^36 within a token,
beyond fp16's range at both ends.  y must match the oracle element by
element within a bound derived from the arithmetic, not a tolerance:

    |y_gpu - y_ref| <= (2^-22 + 2^-23) Y + 2^-39 M_t sum_r |W_down^T[r, c]| + D 2^-24 Y

with Y = sum_r |h3[t, r] W_down^T[r, c]|; 2^-22 the hi + lo representation
of a scaled h3 (11 + 11 bits), 2^-23 h3's own rounding, 2^-39 M_t the
representation floor of values more than 2^17 below the token's largest
|h3| M_t (fp16's subnormal step under the scale), and D the depth of the
kernel's summation tree: 64 (the hi and lo products of a chunk of 32 rows)
+ the chunks of a group + the groups summed into y + 2.  The shapes give
groups of up to 6 chunks (more than the 3 in flight), a ragged last chunk and
a ragged last tile of y (d = 640).  Dropping the lo part (2^-12 per term)
exceeds this bound (checked on the CPU in ``tests/test_down_bound.py``).
With one token h3 stays fp32 and a wave takes down batches as they come, so
a lane may sum every row of its group: D is then the group's rows + the 8
waves' partial tiles + the groups + 2 (the representation terms only widen
the bound).  The one-token cases include groups of 640 rows (d = 2048, k =
40000), which take the instance with the wider down batches.
"""

import numpy as np
import pytest
import torch

import oracle
import paper_2411_12692_amd as si
from h3check import U24, check_h3, fp16_rows, workspace_ok

pytestmark = pytest.mark.gpu
DEV = "cuda"


def to_dev(a: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(a.view(np.int16).copy()).to(DEV)


def scaled_rows(rng, k, d, lo, hi):
    """fp16 rows of N(0,1) values times 2^e_r, e_r uniform in [lo, hi]."""
    e = rng.integers(lo, hi + 1, size=k)
    w = np.clip(rng.standard_normal((k, d)) * np.exp2(e)[:, None], -60000.0, 60000.0)
    return w.astype(np.float16).view(np.uint16)


def one_hot_tokens(rng, b, d):
    """b fp16 tokens with one non-zero element each, +-2^a at distinct positions."""
    x = np.zeros((b, d), dtype=np.float16)
    pos = rng.choice(d, size=b, replace=False)
    for t in range(b):
        x[t, pos[t]] = rng.choice([-1.0, 1.0]) * 2.0 ** int(rng.integers(-6, 7))
    return x.view(np.uint16)


def group_depth(k, d, cus, b=8):
    """Depth of the summation tree of one y element in the row-owning kernel:
    the blocks form groups of T = ceil(d / 512) and own R rows each (the rows
    spread over the grid's whole groups, rounded up to a multiple of 8), a
    group's T R rows are summed in chunks of 32 (b > 1; with one token a lane
    may sum all of them, then the 8 waves' partial tiles), the groups' tiles
    into y."""
    T = (d + 511) // 512
    working = cus // T * T
    R = ((k + working - 1) // working + 7) // 8 * 8
    rows = R * T
    groups = (k + rows - 1) // rows
    if b == 1:
        return rows + 8 + groups + 2
    return 64 + (rows + 31) // 32 + groups + 2


def y_bound(h3, WdT, depth):
    """The bound of the module docstring; ``h3`` ``[b][n]`` (the kept rows),
    ``WdT`` ``[n][d]`` float64."""
    AW = np.abs(WdT)
    Y = np.abs(h3) @ AW
    M = np.abs(h3).max(axis=1) if h3.shape[1] else np.zeros(h3.shape[0])
    return (2.0 ** -22 + 2.0 ** -23 + depth * U24) * Y + 2.0 ** -39 * M[:, None] * AW.sum(axis=0)[None, :]


CASES = [
    # (d, k, tokens, form, flags): 640 columns = a full and a 128-column tile; k = 21000 gives groups of 176
    # rows (6 chunks, the last half full); k = 3001 at d = 4096 groups of 128 rows (about 90 kept) and a
    # ragged last group
    (640, 21000, 8, "mask", 0),
    (640, 21000, 5, "fused", 0),
    (4096, 3001, 4, "mask", 0),
    (640, 21000, 8, "mask", si.SI_NO_SPECULATION),  # the fp32 rounds, same bound
    (640, 21000, 2, "mask", 0),
    (640, 21000, 1, "mask", 0),  # one token: fp32 h3 and down
    (2048, 40000, 1, "fused", 0),  # one token, groups of 640 rows
]


@pytest.mark.parametrize("d,k,b,form,flags", CASES)
def test_down_wide_h3_range(d, k, b, form, flags):
    print(f"d={d} k={k} b={b} form={form} flags={flags}", flush=True)
    rng = np.random.default_rng(7100 + d + k + b + flags)
    wg = scaled_rows(rng, k, d, -10, 10)
    wu = scaled_rows(rng, k, d, -10, 10)
    wd = rng.standard_normal((d, k)).astype(np.float16).view(np.uint16)
    x = one_hot_tokens(rng, b, d)
    layer = si.MLPLayer(to_dev(wg), to_dev(wu), to_dev(wd), max_batch=b)
    xd = to_dev(x)
    if form == "fused":  # alpha = +inf keeps every row
        mask = np.ones(k, dtype=np.uint8)
        y = layer(xd, float("inf"), flags=flags)
    else:  # a mask that keeps 70% of the rows
        mask = (rng.random(k) < 0.7).astype(np.uint8)
        y = layer.sparse_mlp(xd, mask=torch.from_numpy(mask).to(DEV), flags=flags)
    torch.cuda.synchronize()
    assert workspace_ok(layer.workspace)
    out = oracle.sparse_mlp(wg, wu, wd, x, mask)
    X = oracle.fp16_to_f64(x)
    h3 = out["h3"][:, mask.astype(bool)]
    assert np.abs(h3).max() > 1e6 and np.abs(h3[h3 != 0]).min() < 1e-3, "h3 does not span fp16's range"
    check_h3(layer.workspace, k, d, b, mask, out["h3"], X, fp16_rows(wg), fp16_rows(wu), out["g"])
    yg = y.cpu().numpy().astype(np.float64)
    err = np.abs(yg - out["y"])
    keep = oracle.active_rows(mask)
    depth = group_depth(k, d, torch.cuda.get_device_properties(0).multi_processor_count, b)
    bound = y_bound(out["h3"][:, keep], oracle.fp16_to_f64(wd[:, keep]).T, depth)
    bad = err > bound
    if bad.any():
        t, c = np.argwhere(bad)[0]
        raise AssertionError(f"{int(bad.sum())} elements of y out of bounds; first: token {t} column {c}: "
                             f"gpu {yg[t, c]!r} oracle {out['y'][t, c]!r} bound {bound[t, c]!r}")
