"""CPU oracle for SparseInfer's decode-time MLP path (arXiv 2411.12692).

TEST INFRASTRUCTURE ONLY.  Nothing in the product path imports this module:
only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may call it.  It shares no code with the HIP library (no common
headers, tables, helpers or pre/post-processing).  It is written from the
paper's definitions, in plain NumPy with float64 arithmetic, for a reader to
check by eye against the paper:

* Section III, Eq. (1): the gated MLP
  ``MLP(X) = (ReLU(X W_gate) * (X W_up)) W_down^T`` with weights of size
  ``d x k``.  Storage follows the kernels' orientation: ``w_gate`` and ``w_up``
  hold one row of length ``d`` per hidden unit (``[k][d]``); ``w_down`` is
  given as ``[d][k]`` (the paper's ``W_down``), so column ``i`` of ``w_down``
  is the row of ``W_down^T`` that hidden unit ``i`` scales.
* Section IV-A: the sign of each element-wise product ``x_j * w_ij`` is
  predicted by the XOR of the two sign bits (MSBs); counting the predicted
  negatives and positives gives ``N_neg`` and ``N_pos = d - N_neg``; Eq. (2)
  declares row ``i`` sparse when ``alpha * N_pos < N_neg``.
* Section IV-B 1): signs are packed 32 consecutive elements per 32-bit word,
  for the weights once at load time and for the input once per token.
* Section III also names MLP blocks without step 2 (OPT, Falcon after
  ReLUfication): ``relu_mlp`` is that non-gated form,
  ``MLP(X) = ReLU(X W_fc1) W_down^T``, with the predictor on ``W_fc1``.
* Section IV-A (robustness to quantization): the predictor needs only the
  sign bit, so it applies to INT8 weights as they are; ``int8_mlp`` is
  Eq. (1) with each weight taken as ``scale * q`` (symmetric per-row INT8,
  ``quantize_rows_int8``) and ``pack_signs_int8`` packs the MSBs of ``q``.
* Section IV-B 3)/4): the sparse GEMVs skip predicted-sparse rows of
  ``W_gate``, ``W_up`` and ``W_down^T``; "actual sparsity" additionally skips
  rows whose gate output is exactly zero.  Skipping a row whose value is zero
  cannot change the result, so the oracle has no separate branch for it and
  reports the work it saves as counters.

Readings of points the paper leaves open (each one is listed in the design
notes of the repository):

* The literal MSB is the sign: -0.0 counts as negative, +0.0 as positive.
* Bit ``j`` of packed word ``w`` holds element ``32*w + j`` (LSB first); pad
  bits past ``d`` are 0 in both operands, so they never count.
* ``N_pos`` uses the true ``d``, not the padded ``32 * ceil(d/32)``.
* Eq. (2) is evaluated exactly: ``alpha`` is taken as the float32 value the
  library receives, and ``alpha * N_pos`` is exact in float64.  A tie
  ``alpha * N_pos == N_neg`` is *not* sparse.  ``alpha = +inf`` means no row
  is sparse.  The printed CUDA listing assigns the skip flag the other way
  round from Eq. (2) and the prose; the oracle follows Eq. (2) and the prose.
* A batch of ``b`` tokens keeps a row when any token keeps it (union).
* Accumulation precision is not stated in the paper; the oracle uses float64.
"""

from __future__ import annotations

import math

import numpy as np

__all__ = [
    "fp16_to_f64",
    "sign_bits",
    "pack_signs",
    "count_sign_products",
    "predict_rows",
    "active_rows",
    "sparse_mlp",
    "relu_mlp",
    "rmsnorm_fp16",
    "mlp_block",
    "quantize_rows_int8",
    "sign_bits_int8",
    "pack_signs_int8",
    "dequantize_int8",
    "int8_mlp",
    "dense_mlp",
    "gate_truly_positive",
    "prediction_quality",
    "sign_words",
    "signs_bytes",
    "dense_mlp_macs",
]


# ---------------------------------------------------------------------------
# Element decoding
# ---------------------------------------------------------------------------

def _as_u16(a) -> np.ndarray:
    a = np.asarray(a)
    if a.dtype == np.float16:
        return a.view(np.uint16)
    if a.dtype in (np.uint16, np.int16):
        return a.view(np.uint16)
    raise TypeError(f"expected fp16 bit patterns (uint16/int16/float16), got {a.dtype}")


def fp16_to_f64(a) -> np.ndarray:
    """Decode IEEE binary16 bit patterns to float64 (exact: every fp16 value is a
    float64 value)."""
    return _as_u16(a).view(np.float16).astype(np.float64)


def sign_bits(a) -> np.ndarray:
    """Section IV-A: the sign of an element is its most significant bit."""
    return (_as_u16(a) >> np.uint16(15)).astype(np.uint32)


# ---------------------------------------------------------------------------
# Section IV-B 1): sign packing
# ---------------------------------------------------------------------------

def pack_signs(a) -> np.ndarray:
    """Pack the sign bits of the last axis, 32 consecutive elements per uint32.

    ``a``: fp16 bit patterns of shape ``[..., d]``.  Returns ``[..., ceil(d/32)]``
    uint32 where bit ``j`` of word ``w`` is the sign of element ``32*w + j``.
    Pad bits past ``d`` are 0.
    """
    bits = sign_bits(a)
    d = bits.shape[-1]
    nwords = (d + 31) // 32
    pad = nwords * 32 - d
    if pad:
        bits = np.concatenate(
            [bits, np.zeros(bits.shape[:-1] + (pad,), dtype=np.uint32)], axis=-1)
    bits = bits.reshape(bits.shape[:-1] + (nwords, 32))
    place = np.left_shift(np.uint64(1), np.arange(32, dtype=np.uint64))
    return (bits.astype(np.uint64) * place).sum(axis=-1).astype(np.uint32)


# ---------------------------------------------------------------------------
# Section IV-A: counting predicted-negative products
# ---------------------------------------------------------------------------

def count_sign_products(packed_w: np.ndarray, packed_x: np.ndarray, d: int):
    """XOR the packed signs of every row against the packed input signs and
    count the ones (predicted-negative products).

    ``packed_w``: ``[k][nwords]`` uint32; ``packed_x``: ``[b][nwords]`` uint32.
    Returns ``(n_neg, n_pos)``, both ``[b][k]`` int64, with ``n_pos = d - n_neg``.
    """
    packed_w = np.asarray(packed_w, dtype=np.uint32)
    packed_x = np.atleast_2d(np.asarray(packed_x, dtype=np.uint32))
    if packed_w.shape[-1] != packed_x.shape[-1] or packed_w.shape[-1] != (d + 31) // 32:
        raise ValueError("packed word counts do not match d")
    n_neg = np.empty((packed_x.shape[0], packed_w.shape[0]), dtype=np.int64)
    for t in range(packed_x.shape[0]):
        xored = np.bitwise_xor(packed_w, packed_x[t][None, :])
        n_neg[t] = np.bitwise_count(xored).sum(axis=-1, dtype=np.int64)
    return n_neg, d - n_neg


def _check_alpha(alpha) -> float:
    a = float(np.float32(alpha))
    if math.isnan(a) or a < 0.0:
        raise ValueError(f"alpha must be a non-negative number or +inf, got {alpha!r}")
    return a


def predict_rows(packed_w: np.ndarray, x, alpha: float):
    """Eq. (2) on every row, for every token of ``x``.

    ``packed_w``: ``[k][ceil(d/32)]`` uint32 from :func:`pack_signs` of ``W_gate``.
    ``x``: fp16 bit patterns ``[b][d]`` (or ``[d]``).
    Returns ``(mask, active_per_token, n_neg)``: ``mask`` is ``[k]`` uint8 with
    1 = predicted active (not predicted sparse by any token), ``active_per_token``
    is ``[b][k]`` bool, ``n_neg`` is ``[b][k]`` int64.
    """
    x = np.atleast_2d(_as_u16(x))
    d = x.shape[-1]
    a = _check_alpha(alpha)
    n_neg, n_pos = count_sign_products(packed_w, pack_signs(x), d)
    if math.isinf(a):
        sparse = np.zeros(n_neg.shape, dtype=bool)
    else:
        sparse = (a * n_pos.astype(np.float64)) < n_neg.astype(np.float64)
    active = ~sparse
    mask = active.any(axis=0).astype(np.uint8)
    return mask, active, n_neg


def active_rows(mask) -> np.ndarray:
    """Ascending indices of the rows kept by ``mask`` (int32)."""
    return np.flatnonzero(np.asarray(mask) != 0).astype(np.int32)


# ---------------------------------------------------------------------------
# Eq. (1) restricted to the kept rows
# ---------------------------------------------------------------------------

def sparse_mlp(w_gate, w_up, w_down, x, mask):
    """Gated MLP of Eq. (1) computed over the rows kept by ``mask`` only.

    ``w_gate``, ``w_up``: ``[k][d]`` fp16 bits; ``w_down``: ``[d][k]`` fp16 bits
    (the paper's ``W_down``); ``x``: ``[b][d]`` fp16 bits; ``mask``: ``[k]``.
    Returns a dict with ``y`` (``[b][d]`` float64), ``g`` (gate pre-activation),
    ``u`` (``X W_up``), ``h1``, ``h3`` (all ``[b][k]`` float64, 0 on dropped
    rows) and the work counters ``n_gate`` (rows whose gate GEMV runs),
    ``n_up`` (rows with some token's ``h1 > 0``, the rows ``W_up`` is read for
    under actual sparsity) and ``n_down`` (rows with some ``h3 != 0``).
    """
    w_gate = _as_u16(w_gate)
    w_up = _as_u16(w_up)
    w_down = _as_u16(w_down)
    xs = np.atleast_2d(_as_u16(x))
    k, d = w_gate.shape
    if w_up.shape != (k, d) or w_down.shape != (d, k) or xs.shape[-1] != d:
        raise ValueError("shape mismatch")
    keep = active_rows(mask)
    b = xs.shape[0]
    X = fp16_to_f64(xs)                        # [b][d]
    Wg = fp16_to_f64(w_gate[keep])             # [n][d]
    Wu = fp16_to_f64(w_up[keep])               # [n][d]
    WdT = fp16_to_f64(w_down[:, keep]).T       # [n][d]: rows of W_down^T
    g_kept = X @ Wg.T                          # step 1, before sigma
    u_kept = X @ Wu.T                          # step 2
    h1_kept = np.maximum(g_kept, 0.0)          # sigma = ReLU
    h3_kept = h1_kept * u_kept                 # step 3
    y = h3_kept @ WdT                          # step 4
    g = np.zeros((b, k)); u = np.zeros((b, k))
    h1 = np.zeros((b, k)); h3 = np.zeros((b, k))
    g[:, keep] = g_kept; u[:, keep] = u_kept
    h1[:, keep] = h1_kept; h3[:, keep] = h3_kept
    return {
        "y": y,
        "g": g,
        "u": u,
        "h1": h1,
        "h3": h3,
        "n_gate": int(keep.size),
        "n_up": int((h1_kept > 0).any(axis=0).sum()),
        "n_down": int((h3_kept != 0).any(axis=0).sum()),
    }


def relu_mlp(w_fc1, w_down, x, mask):
    """Non-gated ReLU MLP over the rows kept by ``mask``: the MLP block of
    models without step 2 of Section III (no ``W_up``; e.g. OPT and Falcon
    after ReLUfication), ``MLP(X) = ReLU(X W_fc1) W_down^T``.  The predictor
    runs on the signs of ``W_fc1`` exactly as on ``W_gate`` (its ReLU output
    is the one that is sparse), and rows whose ReLU output is zero skip
    ``W_down^T`` (actual sparsity, Section IV-B).

    ``w_fc1``: ``[k][d]`` fp16 bits; ``w_down``: ``[d][k]``; ``x``: ``[b][d]``.
    Returns ``y`` (``[b][d]`` float64), ``g`` and ``h`` (``[b][k]``, 0 on
    dropped rows), ``n_gate`` (rows whose ``W_fc1`` row is read), ``n_up``
    (always 0: there is no ``W_up``) and ``n_down`` (rows with some
    ``h != 0``).
    """
    w_fc1 = _as_u16(w_fc1)
    w_down = _as_u16(w_down)
    xs = np.atleast_2d(_as_u16(x))
    k, d = w_fc1.shape
    if w_down.shape != (d, k) or xs.shape[-1] != d:
        raise ValueError("shape mismatch")
    keep = active_rows(mask)
    b = xs.shape[0]
    X = fp16_to_f64(xs)                        # [b][d]
    W1 = fp16_to_f64(w_fc1[keep])              # [n][d]
    WdT = fp16_to_f64(w_down[:, keep]).T       # [n][d]: rows of W_down^T
    g_kept = X @ W1.T
    h_kept = np.maximum(g_kept, 0.0)           # sigma = ReLU
    y = h_kept @ WdT
    g = np.zeros((b, k)); h = np.zeros((b, k))
    g[:, keep] = g_kept; h[:, keep] = h_kept
    return {
        "y": y,
        "g": g,
        "h": h,
        "n_gate": int(keep.size),
        "n_up": 0,
        "n_down": int((h_kept != 0).any(axis=0).sum()),
    }


def rmsnorm_fp16(h, w_norm, eps: float) -> np.ndarray:
    """The input of the MLP in a decoder layer: ``x = RMSNorm(h) * w_norm``,
    ``x_j = h_j / sqrt(mean_j(h_j^2) + eps) * w_j`` per token, computed in
    float64 and rounded to fp16 (round to nearest even), returned as fp16
    bits ``[b][d]``.  ``h`` (the residual stream) and ``w_norm`` are float32
    values.  This is the neighbour of the path that produces ``X``; the
    paper packs the signs of ``X`` during decode (Section IV-B 1), so a
    kernel that forms ``X`` can form its sign words too."""
    H = np.atleast_2d(np.asarray(h, dtype=np.float32)).astype(np.float64)
    Wn = np.asarray(w_norm, dtype=np.float32).astype(np.float64)
    if H.shape[-1] != Wn.shape[0]:
        raise ValueError("shape mismatch")
    ms = np.mean(H * H, axis=1, keepdims=True)
    X = H / np.sqrt(ms + float(np.float32(eps))) * Wn[None, :]
    return X.astype(np.float16).view(np.uint16)


def mlp_block(h, w_norm, eps: float, packed_w, w_gate, w_up, w_down, alpha: float):
    """The MLP half of a decoder layer around the path: ``x = RMSNorm(h) *
    w_norm`` (fp16), the prediction on ``x``, the MLP over the kept rows
    (gated, or non-gated when ``w_up`` is None), and the residual:
    ``y = h + MLP(x)``.  Returns a dict with ``x`` (fp16 bits), ``mask``,
    ``y`` (float64) and the MLP's outputs."""
    x = rmsnorm_fp16(h, w_norm, eps)
    mask, act, counts = predict_rows(packed_w, x, alpha)
    out = relu_mlp(w_gate, w_down, x, mask) if w_up is None else sparse_mlp(w_gate, w_up, w_down, x, mask)
    out = dict(out)
    out["mlp_y"] = out["y"]
    out["y"] = np.atleast_2d(np.asarray(h, dtype=np.float32)).astype(np.float64) + out["mlp_y"]
    out["x"] = x
    out["mask"] = mask
    return out


# ---------------------------------------------------------------------------
# INT8 weights (Section IV-A: the predictor needs only the sign bit, so it
# applies unchanged to INT8 weights)
# ---------------------------------------------------------------------------

def quantize_rows_int8(w):
    """Symmetric per-row INT8 quantization of fp16 weights ``[rows][d]``
    (bit patterns): ``scale_i = max_j |w_ij| / 127`` and
    ``q_ij = rint(w_ij / scale_i)`` (ties to even), both in float32
    arithmetic, ``q`` clamped to ``[-127, 127]``; a row of zeros has scale 0
    and ``q = 0``.  Returns ``(q int8 [rows][d], scale float32 [rows])``.

    The paper names INT8 without a scheme; one scale per row of the stored
    matrix is a scale per output channel for ``W_gate`` and ``W_up``
    (``[k][d]``) and for ``W_down`` (``[d][k]``)."""
    W = fp16_to_f64(_as_u16(w)).astype(np.float32)
    amax = np.max(np.abs(W), axis=1)
    scale = (amax / np.float32(127.0)).astype(np.float32)
    safe = np.where(scale > 0, scale, np.float32(1.0)).astype(np.float32)
    q = np.rint((W / safe[:, None]).astype(np.float32))
    q = np.clip(q, -127, 127).astype(np.int8)
    q[scale == 0] = 0
    return q, scale


def sign_bits_int8(q) -> np.ndarray:
    """The MSB of each INT8 weight (two's complement): 1 for negative values,
    0 for zero and positive ones."""
    return (np.asarray(q, dtype=np.int8).view(np.uint8) >> 7).astype(np.uint32)


def pack_signs_int8(q) -> np.ndarray:
    """Packed sign words of INT8 weights ``[rows][d]``, in the layout of
    :func:`pack_signs`: bit ``j`` of word ``w`` is the MSB of element
    ``32*w + j``; pad bits are 0."""
    bits = sign_bits_int8(q)
    rows, d = bits.shape
    nw = (d + 31) // 32
    padded = np.zeros((rows, nw * 32), dtype=np.uint64)
    padded[:, :d] = bits
    place = np.left_shift(np.uint64(1), np.arange(32, dtype=np.uint64))
    return (padded.reshape(rows, nw, 32) * place).sum(axis=2).astype(np.uint32)


def dequantize_int8(q, scale) -> np.ndarray:
    """``scale_i * q_ij`` in float64 (exact: a float32 times an integer of
    at most 8 bits)."""
    return np.asarray(scale, dtype=np.float64)[:, None] * np.asarray(q, dtype=np.float64)


def int8_mlp(q_gate, s_gate, q_up, s_up, q_down, s_down, x, mask):
    """Eq. (1) over the kept rows with INT8 weights, every weight taken as
    its dequantized value ``scale * q``.

    ``q_gate``, ``q_up``: ``[k][d]`` int8 with per-row scales ``[k]``;
    ``q_down``: ``[d][k]`` int8 (the paper's ``W_down``) with per-row scales
    ``[d]``; ``q_up = None`` gives the non-gated ReLU MLP.  ``x``: ``[b][d]``
    fp16 bits.  Returns ``y``, ``g``, ``h3`` and the work counters of
    :func:`sparse_mlp` (``n_up = 0`` without ``W_up``)."""
    q_gate = np.asarray(q_gate, dtype=np.int8)
    q_down = np.asarray(q_down, dtype=np.int8)
    xs = np.atleast_2d(_as_u16(x))
    k, d = q_gate.shape
    if q_down.shape != (d, k) or xs.shape[-1] != d:
        raise ValueError("shape mismatch")
    if q_up is not None and np.asarray(q_up).shape != (k, d):
        raise ValueError("shape mismatch")
    keep = active_rows(mask)
    b = xs.shape[0]
    X = fp16_to_f64(xs)                                    # [b][d]
    s_gate = np.asarray(s_gate)
    Wg = dequantize_int8(q_gate[keep], s_gate[keep])       # [n][d]
    WdT = dequantize_int8(q_down[:, keep], s_down).T       # [n][d]: rows of W_down^T
    g_kept = X @ Wg.T                                      # step 1, before sigma
    h1_kept = np.maximum(g_kept, 0.0)                      # sigma = ReLU
    if q_up is None:
        h3_kept = h1_kept
        n_up = 0
    else:
        q_up = np.asarray(q_up, dtype=np.int8)
        u_kept = X @ dequantize_int8(q_up[keep], np.asarray(s_up)[keep]).T   # step 2
        h3_kept = h1_kept * u_kept                         # step 3
        n_up = int((h1_kept > 0).any(axis=0).sum())
    y = h3_kept @ WdT                                      # step 4
    g = np.zeros((b, k)); h3 = np.zeros((b, k))
    g[:, keep] = g_kept; h3[:, keep] = h3_kept
    return {
        "y": y,
        "g": g,
        "h3": h3,
        "n_gate": int(keep.size),
        "n_up": n_up,
        "n_down": int((h3_kept != 0).any(axis=0).sum()),
    }


def dense_mlp(w_gate, w_up, w_down, x):
    """Eq. (1) with every row kept (the dense reference)."""
    k = _as_u16(w_gate).shape[0]
    return sparse_mlp(w_gate, w_up, w_down, x, np.ones(k, dtype=np.uint8))


# ---------------------------------------------------------------------------
# Diagnostics: ground truth and the prediction-quality measures
# ---------------------------------------------------------------------------

def gate_truly_positive(w_gate, x) -> np.ndarray:
    """Exact sign of the gate pre-activation ``X . W_gate,i`` for every token
    and row: returns ``[b][k]`` bool, True where the exact sum is > 0.

    Every fp16 x fp16 product is exact in float64.  The float64 dot product
    differs from the exact sum by at most ``d * 2**-52 * sum|w_j x_j|``; rows
    whose float64 value is further than that from 0 have a certain sign, the
    rest are summed exactly with ``math.fsum`` (correctly rounded, so its sign
    is the sign of the exact sum).
    """
    Wg = fp16_to_f64(w_gate)
    X = fp16_to_f64(np.atleast_2d(_as_u16(x)))
    d = Wg.shape[1]
    approx = X @ Wg.T
    bound = (2.0 * d * 2.0 ** -52) * (np.abs(X) @ np.abs(Wg).T)
    out = approx > 0
    unsure = np.argwhere(np.abs(approx) <= bound)
    for t, i in unsure:
        out[t, i] = math.fsum((X[t] * Wg[i]).tolist()) > 0
    return out


def prediction_quality(active_pred, truly_positive):
    """Counts and ratios for a prediction against the exact truth.

    ``active_pred`` / ``truly_positive``: bool arrays of one shape (per token
    and row).  The sparse class is ``h1 == 0`` (gate pre-activation <= 0).

    * ``precision`` (Section IV-A, Fig. 3 text): of the rows predicted
      sparse, the fraction that are truly sparse.
    * ``recall`` (same passage): of the truly sparse rows, the fraction
      predicted sparse.
    * ``active_recall``: of the truly positive rows, the fraction predicted
      active; ``missed`` counts truly positive rows predicted sparse.
    """
    pa = np.asarray(active_pred, dtype=bool)
    tp = np.asarray(truly_positive, dtype=bool)
    pred_sparse = ~pa
    true_sparse = ~tp
    both_sparse = int((pred_sparse & true_sparse).sum())
    n_pred_sparse = int(pred_sparse.sum())
    n_true_sparse = int(true_sparse.sum())
    n_true_pos = int(tp.sum())
    missed = int((tp & pred_sparse).sum())
    return {
        "pred_sparse": n_pred_sparse,
        "true_sparse": n_true_sparse,
        "true_positive": n_true_pos,
        "missed": missed,
        "precision": both_sparse / n_pred_sparse if n_pred_sparse else 1.0,
        "recall": both_sparse / n_true_sparse if n_true_sparse else 1.0,
        "active_recall": (n_true_pos - missed) / n_true_pos if n_true_pos else 1.0,
    }


# ---------------------------------------------------------------------------
# Operation and memory counts stated in Section V-A
# ---------------------------------------------------------------------------

def sign_words(k: int, d: int) -> int:
    """Packed 32-bit sign words of one ``W_gate`` (one XOR each per token)."""
    return k * ((d + 31) // 32)


def signs_bytes(k: int, d: int) -> int:
    """Bytes of the packed signs of one ``W_gate`` in the canonical layout."""
    return 4 * sign_words(k, d)


def dense_mlp_macs(k: int, d: int) -> int:
    """Multiply-accumulates of one dense gated MLP block for one token."""
    return 3 * k * d
