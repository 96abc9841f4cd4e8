"""Per-row h3 parity (Eq. (1) step 3) and the workspace's error word, shared
by the GPU parity tests.

y alone can hide a kept row whose h3 was dropped or miscomputed when that
row's contribution is small, so every parity check also reads back the h3
values the kernel published for the kept rows (``si_read_h3``) and compares
them, row by row and token by token, with the oracle's.

The bar: ``|h3_gpu - h3_ref| <= 1e-3 |h3_ref| + bound``.  ``bound`` is the
rounding error of the kernel's arithmetic: the gate and up dot products
accumulate d products in fp32 (each fp16 x fp16 product, and each INT8 x
fp16 product, is exact in fp32), so each sum is within ``gamma * S`` of its
exact value, with ``S`` the sum of the absolute products and ``gamma =
(d + 66) 2^-24`` (at most d - 1 additions in any order, the 64-lane
reduction and, for INT8, the row scale); ReLU does not increase an error, and
``h3 = h1 u`` adds one more rounding.  Rows where g or u nearly cancel have a
large relative error but a tiny absolute one; the bound covers exactly those.
A kept row for which the call left no value reads NaN and fails.
"""

import numpy as np
import torch

import oracle
import paper_2411_12692_amd as si

U24 = 2.0 ** -24


def workspace_ok(ws: torch.Tensor) -> bool:
    """``si_workspace_check`` returns SI_OK: no wait inside a kernel gave up
    and no list row was out of range since the workspace was last checked."""
    return si.workspace_check(ws) == 0


def h3_bound(X, Wg, Wu, g_ref, x_ulp=False):
    """Bound on |h3_gpu - h3_ref| per (token, row), ``[b][n]`` for the rows of
    ``Wg`` (float64 values, ``[n][d]``); ``Wu`` None for the non-gated MLP.
    ``x_ulp``: the two sides rounded x to fp16 separately (the decoder-block
    call), so an element of x may differ by one fp16 unit: at most 2^-10 of
    its value, or 2^-24 below the normal range."""
    d = X.shape[1]
    gamma = (d + 66) * U24 * 1.01
    AX = np.abs(X)

    def err(W):
        S = AX @ np.abs(W).T
        e = gamma * S
        if x_ulp:
            e = e + 2.0 ** -10 * S + U24 * np.abs(W).sum(axis=1)[None, :]
        return e

    h1 = np.maximum(g_ref, 0.0)
    eg = err(Wg)
    if Wu is None:
        return eg + U24 * np.abs(h1)
    u = X @ Wu.T
    eu = err(Wu)
    return eg * np.abs(u) + np.abs(h1) * eu + eg * eu + 2 * U24 * np.abs(h1 * u)


def check_h3(ws, k, d, b, mask, h3_ref, X, gate_rows, up_rows, g_ref, x_ulp=False):
    """The h3 of the last MLP call made with ``ws`` against the oracle's.

    ``mask``: ``[k]`` kept rows of that call; ``h3_ref``, ``g_ref``: the
    oracle's ``[b][k]``; ``X`` ``[b][d]`` float64; ``gate_rows(rows)`` and
    ``up_rows(rows)`` give those rows of W_gate / W_up as float64 values
    (dequantized for INT8); ``up_rows`` None for the non-gated MLP."""
    mask = np.asarray(mask).astype(bool)
    m_dev = torch.from_numpy(mask.astype(np.uint8)).to("cuda")
    got = si.read_h3(ws, k, d, b, m_dev).cpu().numpy().astype(np.float64)  # [k][b]
    kept = np.flatnonzero(mask)
    assert np.all(got[~mask] == 0.0), "h3 read back outside the kept rows"
    if kept.size == 0:
        return
    gk = got[kept].T  # [b][n]
    assert not np.isnan(gk).any(), f"kept rows without an h3 of this call: {kept[np.isnan(gk).any(axis=0)][:8]}"
    ref = np.asarray(h3_ref)[:, kept]
    bound = h3_bound(X, gate_rows(kept), None if up_rows is None else up_rows(kept), np.asarray(g_ref)[:, kept],
                     x_ulp)
    err = np.abs(gk - ref)
    lim = 1e-3 * np.abs(ref) + bound
    bad = err > lim
    if bad.any():
        t, j = np.argwhere(bad)[0]
        raise AssertionError(f"{int(bad.sum())} h3 values out of bounds; first: token {t} row {kept[j]}: "
                             f"gpu {gk[t, j]!r} oracle {ref[t, j]!r} bound {lim[t, j]!r}")


def fp16_rows(bits):
    """``rows -> float64 values`` of those rows of an fp16 ``[k][d]`` array."""
    return lambda rows: oracle.fp16_to_f64(np.asarray(bits)[rows])


def int8_rows(q, scale):
    """``rows -> float64 values`` of those rows of an INT8 ``[k][d]`` array
    with per-row scales."""
    return lambda rows: oracle.dequantize_int8(np.asarray(q)[rows], np.asarray(scale)[rows])
