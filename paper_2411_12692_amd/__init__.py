"""MI355X-native SparseInfer decode path (arXiv 2411.12692).

Thin PyTorch-facing binding of ``libsparseinfer.so`` (see
``include/sparseinfer.h``).  PyTorch only provides device memory and the
current stream; every step of the path runs in the library's HIP kernels.
The functions take contiguous CUDA tensors: fp16 weights/inputs (``float16``
or ``int16`` bit patterns), and return new tensors.
"""

from __future__ import annotations

import ctypes

import torch

from . import _lib
from ._lib import SI_NO_AS, SI_NO_SPECULATION, SparseInferError

__all__ = [
    "SI_NO_AS", "SI_NO_SPECULATION", "SparseInferError", "signs_bytes", "alpha_threshold", "workspace_bytes",
    "new_workspace", "workspace_check", "read_h3", "pack_signs", "signs_to_canonical", "transpose_down", "predict",
    "sparse_mlp", "predict_sparse_mlp", "mlp_block", "MLPLayer",
    "quantize_rows_i8", "pack_signs_i8", "transpose_down_i8", "sparse_mlp_i8", "predict_sparse_mlp_i8",
    "Int8MLPLayer",
]


def _vp(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream():
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _dev(t: torch.Tensor, name: str, dtypes, ndim=None):
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a tensor")
    if t.device.type != "cuda":
        raise ValueError(f"{name} must be a CUDA tensor (got {t.device})")
    if t.dtype not in dtypes:
        raise TypeError(f"{name} has dtype {t.dtype}, expected one of {dtypes}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if ndim is not None and t.dim() != ndim:
        raise ValueError(f"{name} must have {ndim} dims, got {tuple(t.shape)}")
    return t


_F16 = (torch.float16, torch.int16)


def signs_bytes(k: int, d: int) -> int:
    return int(_lib.load().si_signs_bytes(k, d))


def alpha_threshold(alpha: float, d: int) -> int:
    """Integer form of Eq. (2): rows are kept iff N_neg < T (host only)."""
    return int(_lib.load().si_alpha_threshold(alpha, d))


def workspace_bytes(k: int, d: int, b: int = 1) -> int:
    return int(_lib.load().si_workspace_bytes(k, d, b))


def new_workspace(k: int, d: int, b: int = 1, device=None) -> torch.Tensor:
    """Zero-filled workspace for calls with up to ``b`` tokens."""
    n = workspace_bytes(k, d, b)
    if n == 0:
        raise ValueError(f"unsupported shape k={k} d={d} b={b}")
    return torch.zeros(n, dtype=torch.uint8, device=device or "cuda")


def workspace_check(workspace: torch.Tensor, stream=None) -> int:
    """``si_workspace_check``: waits for the stream, returns the status of the
    workspace's sticky device error word (``SI_OK``, ``SI_ERR_TIMEOUT`` or
    ``SI_ERR_LIST``) and resets the workspace when it is not ``SI_OK``."""
    st = stream if stream is not None else _stream()
    return int(_lib.status("si_workspace_check", _vp(workspace), workspace.numel(), st))


def read_h3(workspace: torch.Tensor, k: int, d: int, b: int, mask: torch.Tensor) -> torch.Tensor:
    """``si_read_h3``: the per-row h3 (Eq. (1) step 3) of the last MLP call
    made with ``workspace``, ``[k][b]`` float32 (0 off ``mask``, NaN for a
    kept row the call left no value for)."""
    _dev(mask, "mask", (torch.uint8,), 1)
    out = torch.empty(k, b, dtype=torch.float32, device=mask.device)
    _lib.call("si_read_h3", _vp(workspace), workspace.numel(), k, d, b, _vp(mask), _vp(out), _stream())
    return out


def pack_signs(w_gate: torch.Tensor) -> torch.Tensor:
    """Packed sign bits of ``W_gate [k][d]`` (private layout, int32 words)."""
    _dev(w_gate, "w_gate", _F16, 2)
    k, d = w_gate.shape
    nbytes = signs_bytes(k, d)
    if nbytes == 0:
        raise ValueError(f"unsupported shape k={k} d={d}")
    out = torch.empty(nbytes // 4, dtype=torch.int32, device=w_gate.device)
    _lib.call("si_pack_signs", _vp(w_gate), k, d, _vp(out), _stream())
    return out


def signs_to_canonical(signs: torch.Tensor, k: int, d: int) -> torch.Tensor:
    """``[k][d/32]`` int32 words, bit j of word w = sign of element 32w+j."""
    _dev(signs, "signs", (torch.int32,))
    out = torch.empty(k, d // 32, dtype=torch.int32, device=signs.device)
    _lib.call("si_signs_to_canonical", _vp(signs), k, d, _vp(out), _stream())
    return out


def transpose_down(w_down: torch.Tensor) -> torch.Tensor:
    """``W_down [d][k]`` -> ``W_down^T [k][d]`` (fp16)."""
    _dev(w_down, "w_down", _F16, 2)
    d, k = w_down.shape
    out = torch.empty(k, d, dtype=w_down.dtype, device=w_down.device)
    _lib.call("si_transpose_down", _vp(w_down), d, k, _vp(out), _stream())
    return out


def _x2(x: torch.Tensor, d: int):
    _dev(x, "x", _F16)
    if x.dim() == 1:
        x = x.view(1, -1)
    if x.dim() != 2 or x.shape[1] != d:
        raise ValueError(f"x must be [b][{d}], got {tuple(x.shape)}")
    return x


def predict(signs: torch.Tensor, x: torch.Tensor, alpha: float, k: int, workspace: torch.Tensor):
    """Eq. (2) for every row: returns ``(mask [k] uint8, active_idx [k] int32,
    n_active [1] int32)``; entries ``n..k-1`` of ``active_idx`` are undefined."""
    _dev(signs, "signs", (torch.int32,))
    d = x.shape[-1]
    x = _x2(x, d)
    b = x.shape[0]
    mask = torch.empty(k, dtype=torch.uint8, device=x.device)
    idx = torch.empty(k, dtype=torch.int32, device=x.device)
    n = torch.empty(1, dtype=torch.int32, device=x.device)
    _lib.call("si_predict", _vp(signs), k, d, _vp(x), b, float(alpha), _vp(mask), _vp(idx), _vp(n),
              _vp(workspace), workspace.numel(), _stream())
    return mask, idx, n


def sparse_mlp(w_gate, w_up, w_down_t, x, workspace, mask=None, active_idx=None, n_active=None,
               flags: int = 0, counters: bool = False):
    """Eq. (1) over the kept rows; returns ``y [b][d]`` float32 (and the
    ``[3]`` work counters when ``counters``).  ``w_up=None`` runs the
    non-gated ReLU MLP ``ReLU(x W_fc1) W_down^T`` with ``w_gate`` as
    ``W_fc1`` (``si_sparse_relu_mlp``)."""
    for t, nm in ((w_gate, "w_gate"), (w_up, "w_up"), (w_down_t, "w_down_t")):
        if t is not None or nm != "w_up":
            _dev(t, nm, _F16, 2)
    k, d = w_gate.shape
    x = _x2(x, d)
    b = x.shape[0]
    y = torch.empty(b, d, dtype=torch.float32, device=x.device)
    cnt = torch.zeros(3, dtype=torch.int32, device=x.device) if counters else None
    tail = (k, d, _vp(x), b, _vp(mask), _vp(active_idx), _vp(n_active), _vp(y), _vp(workspace),
            workspace.numel(), flags, _vp(cnt), _stream())
    if w_up is None:
        _lib.call("si_sparse_relu_mlp", _vp(w_gate), _vp(w_down_t), *tail)
    else:
        _lib.call("si_sparse_mlp", _vp(w_gate), _vp(w_up), _vp(w_down_t), *tail)
    return (y, cnt) if counters else y


def predict_sparse_mlp(signs, w_gate, w_up, w_down_t, x, alpha, workspace, flags: int = 0,
                       outputs: bool = False, y: torch.Tensor = None):
    """The whole per-token path.  Returns ``y`` (written into ``y`` when
    given); with ``outputs`` also ``(mask, active_idx, n_active, counters)``.
    ``w_up=None``: the non-gated ReLU MLP (``si_predict_sparse_relu_mlp``)."""
    k, d = w_gate.shape
    x = _x2(x, d)
    b = x.shape[0]
    if y is None:
        y = torch.empty(b, d, dtype=torch.float32, device=x.device)
    else:
        _dev(y, "y", (torch.float32,))
        if y.numel() != b * d:
            raise ValueError(f"y must hold [{b}][{d}] floats")
    if outputs:
        mask = torch.empty(k, dtype=torch.uint8, device=x.device)
        idx = torch.empty(k, dtype=torch.int32, device=x.device)
        n = torch.empty(1, dtype=torch.int32, device=x.device)
        cnt = torch.zeros(3, dtype=torch.int32, device=x.device)
    else:
        mask = idx = n = cnt = None
    tail = (k, d, _vp(x), b, float(alpha), _vp(mask), _vp(idx), _vp(n), _vp(y), _vp(workspace),
            workspace.numel(), flags, _vp(cnt), _stream())
    if w_up is None:  # the non-gated ReLU MLP, w_gate as W_fc1
        _lib.call("si_predict_sparse_relu_mlp", _vp(signs), _vp(w_gate), _vp(w_down_t), *tail)
    else:
        _lib.call("si_predict_sparse_mlp", _vp(signs), _vp(w_gate), _vp(w_up), _vp(w_down_t), *tail)
    return (y, (mask, idx, n, cnt)) if outputs else y


def mlp_block(h, norm_w, eps, signs, w_gate, w_up, w_down_t, alpha, workspace, flags: int = 0,
              outputs: bool = False, y: torch.Tensor = None):
    """The MLP half of a decoder layer with its neighbours fused
    (``si_rmsnorm_predict_sparse_mlp``): ``y = h + MLP(fp16(RMSNorm(h) *
    norm_w))``; ``h`` ``[b][d]`` and ``norm_w`` ``[d]`` float32.  Returns
    ``y`` (and ``(mask, active_idx, n_active, counters)`` with ``outputs``);
    ``w_up=None``: the non-gated ReLU MLP."""
    _dev(h, "h", (torch.float32,))
    _dev(norm_w, "norm_w", (torch.float32,), 1)
    k, d = w_gate.shape
    h2 = h.view(-1, d)
    b = h2.shape[0]
    if y is None:
        y = torch.empty(b, d, dtype=torch.float32, device=h.device)
    else:
        _dev(y, "y", (torch.float32,))
        if y.numel() != b * d:
            raise ValueError(f"y must hold [{b}][{d}] floats")
    if outputs:
        mask = torch.empty(k, dtype=torch.uint8, device=h.device)
        idx = torch.empty(k, dtype=torch.int32, device=h.device)
        n = torch.empty(1, dtype=torch.int32, device=h.device)
        cnt = torch.zeros(3, dtype=torch.int32, device=h.device)
    else:
        mask = idx = n = cnt = None
    _lib.call("si_rmsnorm_predict_sparse_mlp", _vp(h2), _vp(norm_w), float(eps), _vp(signs), _vp(w_gate),
              _vp(w_up), _vp(w_down_t), k, d, b, float(alpha), _vp(mask), _vp(idx), _vp(n), _vp(y),
              _vp(workspace), workspace.numel(), flags, _vp(cnt), _stream())
    return (y, (mask, idx, n, cnt)) if outputs else y


class MLPLayer:
    """One layer's device-resident state: weights, packed signs and
    ``W_down^T`` (both made once at load), plus a workspace.  With
    ``w_up=None`` the layer is a non-gated ReLU MLP and ``w_gate`` is its
    ``W_fc1``."""

    def __init__(self, w_gate: torch.Tensor, w_up: torch.Tensor, w_down: torch.Tensor, max_batch: int = 1,
                 keep_w_down: bool = False):
        self.k, self.d = w_gate.shape
        self.w_gate = w_gate
        self.w_up = w_up
        self.signs = pack_signs(w_gate)
        self.w_down_t = transpose_down(w_down)
        self.w_down = w_down if keep_w_down else None
        self.workspace = new_workspace(self.k, self.d, max_batch, w_gate.device)

    def __call__(self, x, alpha: float, flags: int = 0, outputs: bool = False, y: torch.Tensor = None):
        return predict_sparse_mlp(self.signs, self.w_gate, self.w_up, self.w_down_t, x, alpha, self.workspace,
                                  flags=flags, outputs=outputs, y=y)

    def block(self, h, norm_w, eps: float, alpha: float, flags: int = 0, outputs: bool = False,
              y: torch.Tensor = None):
        """``h + MLP(RMSNorm(h) * norm_w)`` in one launch (see ``mlp_block``)."""
        return mlp_block(h, norm_w, eps, self.signs, self.w_gate, self.w_up, self.w_down_t, alpha, self.workspace,
                         flags=flags, outputs=outputs, y=y)

    def predict(self, x, alpha: float):
        return predict(self.signs, x, alpha, self.k, self.workspace)

    def sparse_mlp(self, x, mask=None, active_idx=None, n_active=None, flags: int = 0, counters: bool = False):
        return sparse_mlp(self.w_gate, self.w_up, self.w_down_t, x, self.workspace, mask, active_idx, n_active,
                          flags, counters)


# ---- INT8 weights ---------------------------------------------------------

def quantize_rows_i8(w: torch.Tensor):
    """Symmetric per-row INT8 quantization of fp16 ``w [rows][n]``: returns
    ``(q int8 [rows][n], scale float32 [rows])`` (``si_quantize_rows_i8``)."""
    _dev(w, "w", _F16, 2)
    rows, n = w.shape
    q = torch.empty(rows, n, dtype=torch.int8, device=w.device)
    scale = torch.empty(rows, dtype=torch.float32, device=w.device)
    _lib.call("si_quantize_rows_i8", _vp(w), rows, n, _vp(q), _vp(scale), _stream())
    return q, scale


def pack_signs_i8(q_gate: torch.Tensor) -> torch.Tensor:
    """Packed MSBs of INT8 ``W_gate [k][d]`` (the layout of ``pack_signs``)."""
    _dev(q_gate, "q_gate", (torch.int8,), 2)
    k, d = q_gate.shape
    nbytes = signs_bytes(k, d)
    if nbytes == 0:
        raise ValueError(f"unsupported shape k={k} d={d}")
    out = torch.empty(nbytes // 4, dtype=torch.int32, device=q_gate.device)
    _lib.call("si_pack_signs_i8", _vp(q_gate), k, d, _vp(out), _stream())
    return out


def transpose_down_i8(q_down: torch.Tensor) -> torch.Tensor:
    """INT8 ``W_down [d][k]`` -> ``W_down^T [k][d]``."""
    _dev(q_down, "q_down", (torch.int8,), 2)
    d, k = q_down.shape
    out = torch.empty(k, d, dtype=torch.int8, device=q_down.device)
    _lib.call("si_transpose_down_i8", _vp(q_down), d, k, _vp(out), _stream())
    return out


def _i8_weights(q_gate, s_gate, q_up, s_up, q_down_t, s_down):
    _dev(q_gate, "q_gate", (torch.int8,), 2)
    _dev(q_down_t, "q_down_t", (torch.int8,), 2)
    k, d = q_gate.shape
    _dev(s_gate, "s_gate", (torch.float32,), 1)
    _dev(s_down, "s_down", (torch.float32,), 1)
    if q_up is not None:
        _dev(q_up, "q_up", (torch.int8,), 2)
        _dev(s_up, "s_up", (torch.float32,), 1)
        if tuple(q_up.shape) != (k, d) or s_up.numel() != k:
            raise ValueError("q_up / s_up do not match q_gate")
    if tuple(q_down_t.shape) != (k, d) or s_gate.numel() != k or s_down.numel() != d:
        raise ValueError("q_down_t [k][d], s_gate [k] and s_down [d] expected")
    return k, d


def sparse_mlp_i8(q_gate, s_gate, q_up, s_up, q_down_t, s_down, x, workspace, mask, flags: int = 0,
                  counters: bool = False):
    """Eq. (1) over the rows kept by ``mask`` with INT8 weights
    (``si_sparse_mlp_i8``); ``q_up=None``: the non-gated ReLU MLP.  Returns
    ``y [b][d]`` float32 (and the ``[3]`` work counters with ``counters``)."""
    k, d = _i8_weights(q_gate, s_gate, q_up, s_up, q_down_t, s_down)
    x = _x2(x, d)
    b = x.shape[0]
    y = torch.empty(b, d, dtype=torch.float32, device=x.device)
    cnt = torch.zeros(3, dtype=torch.int32, device=x.device) if counters else None
    _lib.call("si_sparse_mlp_i8", _vp(q_gate), _vp(s_gate), _vp(q_up), _vp(s_up if q_up is not None else None),
              _vp(q_down_t), _vp(s_down), k, d, _vp(x), b, _vp(mask), _vp(y), _vp(workspace), workspace.numel(),
              flags, _vp(cnt), _stream())
    return (y, cnt) if counters else y


def predict_sparse_mlp_i8(signs, q_gate, s_gate, q_up, s_up, q_down_t, s_down, x, alpha, workspace,
                          flags: int = 0, outputs: bool = False, y: torch.Tensor = None):
    """The whole per-token path with INT8 weights
    (``si_predict_sparse_mlp_i8``); ``signs`` from ``pack_signs_i8``.
    Returns ``y`` (and ``(mask, active_idx, n_active, counters)`` with
    ``outputs``)."""
    k, d = _i8_weights(q_gate, s_gate, q_up, s_up, q_down_t, s_down)
    _dev(signs, "signs", (torch.int32,))
    x = _x2(x, d)
    b = x.shape[0]
    if y is None:
        y = torch.empty(b, d, dtype=torch.float32, device=x.device)
    else:
        _dev(y, "y", (torch.float32,))
        if y.numel() != b * d:
            raise ValueError(f"y must hold [{b}][{d}] floats")
    if outputs:
        mask = torch.empty(k, dtype=torch.uint8, device=x.device)
        idx = torch.empty(k, dtype=torch.int32, device=x.device)
        n = torch.empty(1, dtype=torch.int32, device=x.device)
        cnt = torch.zeros(3, dtype=torch.int32, device=x.device)
    else:
        mask = idx = n = cnt = None
    _lib.call("si_predict_sparse_mlp_i8", _vp(signs), _vp(q_gate), _vp(s_gate), _vp(q_up),
              _vp(s_up if q_up is not None else None), _vp(q_down_t), _vp(s_down), k, d, _vp(x), b, float(alpha),
              _vp(mask), _vp(idx), _vp(n), _vp(y), _vp(workspace), workspace.numel(), flags, _vp(cnt), _stream())
    return (y, (mask, idx, n, cnt)) if outputs else y


class Int8MLPLayer:
    """One layer with INT8 weights, made on the device at load from fp16
    weights: per-row quantization of ``W_gate``, ``W_up`` (``[k][d]``) and
    ``W_down`` (``[d][k]``), the packed MSBs of the INT8 ``W_gate`` and the
    INT8 ``W_down^T``.  ``w_up=None``: a non-gated ReLU MLP."""

    def __init__(self, w_gate: torch.Tensor, w_up: torch.Tensor, w_down: torch.Tensor, max_batch: int = 1):
        self.k, self.d = w_gate.shape
        self.q_gate, self.s_gate = quantize_rows_i8(w_gate)
        self.q_up, self.s_up = quantize_rows_i8(w_up) if w_up is not None else (None, None)
        q_down, self.s_down = quantize_rows_i8(w_down)
        self.q_down_t = transpose_down_i8(q_down)
        self.signs = pack_signs_i8(self.q_gate)
        self.workspace = new_workspace(self.k, self.d, max_batch, w_gate.device)

    def __call__(self, x, alpha: float, flags: int = 0, outputs: bool = False, y: torch.Tensor = None):
        return predict_sparse_mlp_i8(self.signs, self.q_gate, self.s_gate, self.q_up, self.s_up, self.q_down_t,
                                     self.s_down, x, alpha, self.workspace, flags=flags, outputs=outputs, y=y)

    def sparse_mlp(self, x, mask, flags: int = 0, counters: bool = False):
        return sparse_mlp_i8(self.q_gate, self.s_gate, self.q_up, self.s_up, self.q_down_t, self.s_down, x,
                             self.workspace, mask, flags, counters)
