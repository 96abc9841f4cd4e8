"""Host-side checks of the C ABI (no GPU needed, no kernel is launched).

The library must load, export every entry point its header declares, compute
the Eq. (2) threshold exactly as the oracle's direct comparison decides, and
reject bad arguments before enqueueing anything.
"""

import ctypes
import math
import os
import re

import numpy as np
import pytest

import oracle
from paper_2411_12692_amd import _lib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "sparseinfer.h")


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(_lib.LIB_PATH):
        from paper_2411_12692_amd import build
        build.build()
    return _lib.load()


def _declared_symbols():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(si_[a-z_0-9]+)\s*\(", text)))


def test_every_declared_symbol_is_exported(lib):
    names = _declared_symbols()
    assert len(names) >= 11
    for name in names:
        assert hasattr(lib, name), name
    assert set(names) == set(_lib.SIGNATURES)


def test_version(lib):
    assert lib.si_version().decode().startswith("sparseinfer")


SWEEP = [0.0, 0.5, 0.7, 1.0, 1.01, 1.02, 1.03, 1.45, 1.5, 2.0, 1e30]


@pytest.mark.parametrize("d", [1, 7, 128, 512, 4096, 5120])
def test_threshold_matches_direct_comparison(lib, d):
    """T(alpha, d) is the first N_neg the oracle's Eq. (2) calls sparse."""
    n_neg = np.arange(d + 1)
    x = np.full((1, d), 0x3C00, dtype=np.uint16)  # +1.0
    w = np.where(np.arange(d)[None, :] < n_neg[:, None], 0xBC00, 0x3C00).astype(np.uint16)
    packed = oracle.pack_signs(w)
    for alpha in SWEEP + [math.inf]:
        T = lib.si_alpha_threshold(alpha, d)
        mask, _, got = oracle.predict_rows(packed, x, alpha)
        assert got[0].tolist() == n_neg.tolist()
        assert mask.tolist() == (n_neg < T).astype(np.uint8).tolist(), (alpha, T)


def test_threshold_values(lib):
    # alpha = +inf keeps everything; alpha = 0 keeps only N_neg = 0; alpha = 1
    # keeps ties (N_neg = d/2).
    assert lib.si_alpha_threshold(math.inf, 4096) == 4097
    assert lib.si_alpha_threshold(0.0, 4096) == 1
    assert lib.si_alpha_threshold(1.0, 4096) == 2049
    for bad in [math.nan, -1.0, -1e-30]:
        assert lib.si_alpha_threshold(bad, 4096) == -1
    assert lib.si_alpha_threshold(1.0, 0) == -1
    prev = 0
    for a in np.linspace(0, 5, 200):
        t = lib.si_alpha_threshold(float(a), 4096)
        assert t >= prev
        prev = t


def test_sizes(lib):
    assert lib.si_signs_bytes(11008, 4096) == 11008 * 4096 // 8
    # 13B: packed signs of 40 blocks = 337.5 MiB (Section V-A 2))
    assert lib.si_signs_bytes(13824, 5120) * 40 / 2**20 == 337.5
    assert lib.si_signs_bytes(1376, 512) == 1408 * 512 // 8  # rows padded to 64
    assert lib.si_signs_bytes(1376, 500) == 0
    assert lib.si_signs_bytes(0, 512) == 0
    assert lib.si_signs_bytes(10, 8320) == 0
    w1 = lib.si_workspace_bytes(11008, 4096, 1)
    w8 = lib.si_workspace_bytes(11008, 4096, 8)
    assert w8 > w1 > 11008 * 9
    assert lib.si_workspace_bytes(11008, 4096, 9) == 0


def _p(v):
    return ctypes.c_void_p(v)


A = 1 << 20  # a 16-byte-aligned fake address: never dereferenced, validation fails first


def test_validation_errors(lib):
    ws = lib.si_workspace_bytes(128, 256, 1)
    cases = [
        # (entry, args, expected status)
        ("si_pack_signs", (None, 128, 256, _p(A), None), _lib.SI_ERR_NULL),
        ("si_pack_signs", (_p(A), 128, 200, _p(A), None), _lib.SI_ERR_SHAPE),
        ("si_pack_signs", (_p(A), 0, 256, _p(A), None), _lib.SI_ERR_SHAPE),
        ("si_pack_signs", (_p(A + 8), 128, 256, _p(A), None), _lib.SI_ERR_ALIGN),
        ("si_transpose_down", (_p(A), 256, 128, _p(A), None), _lib.SI_ERR_SHAPE),  # overlap
        ("si_predict", (_p(A), 128, 256, _p(A), 1, math.nan, _p(A), None, None, _p(A), ws, None),
         _lib.SI_ERR_ALPHA),
        ("si_predict", (_p(A), 128, 256, _p(A), 1, -1.0, _p(A), None, None, _p(A), ws, None), _lib.SI_ERR_ALPHA),
        ("si_predict", (_p(A), 128, 256, _p(A), 9, 1.0, _p(A), None, None, _p(A), ws, None), _lib.SI_ERR_SHAPE),
        ("si_predict", (_p(A), 128, 256, _p(A), 0, 1.0, _p(A), None, None, _p(A), ws, None), _lib.SI_ERR_SHAPE),
        ("si_predict", (_p(A), 128, 256, _p(A), 1, 1.0, None, None, None, _p(A), ws, None), _lib.SI_ERR_NULL),
        ("si_predict", (_p(A), 128, 256, _p(A), 1, 1.0, _p(A), None, None, _p(A), ws - 1, None),
         _lib.SI_ERR_WORKSPACE),
        ("si_predict", (_p(A), 128, 256, _p(A), 1, 1.0, _p(A), None, None, None, ws, None), _lib.SI_ERR_NULL),
        ("si_sparse_mlp", (_p(A), _p(A), _p(A), 128, 256, _p(A), 1, _p(A), _p(A), None, _p(A), _p(A), ws, 0,
                           None, None), _lib.SI_ERR_NULL),
        ("si_sparse_mlp", (_p(A), _p(A), _p(A), 128, 256, _p(A), 1, _p(A), None, None, _p(A), _p(A), ws, 4,
                           None, None), _lib.SI_ERR_FLAGS),
        ("si_sparse_mlp", (_p(A), _p(A), _p(A), 128, 256, _p(A), 1, None, None, None, _p(A), _p(A), ws, 0,
                           None, None), _lib.SI_ERR_NULL),
        ("si_sparse_mlp", (_p(A), _p(A), _p(A), 128, 256, _p(A), 1, _p(A), None, None, None, _p(A), ws, 0,
                           None, None), _lib.SI_ERR_NULL),
        ("si_predict_sparse_mlp", (_p(A), _p(A), _p(A), _p(A), 128, 256, _p(A), 1, 1.0, None, None, None, _p(A),
                                   _p(A), ws - 16, 0, None, None), _lib.SI_ERR_WORKSPACE),
        ("si_predict_sparse_mlp", (_p(A), _p(A), _p(A), _p(A), 128, 256, _p(A), 1, 1.0, None, None, None,
                                   _p(A + 4), _p(A), ws, 0, None, None), _lib.SI_ERR_ALIGN),
    ]
    for name, args, want in cases:
        st = _lib.status(name, *args)
        assert st == want, (name, args, st, _lib.last_error())
        assert _lib.last_error() != ""


def test_device_error_status_mapping(lib):
    """The sticky error word of a workspace -> the status si_workspace_check
    returns: 0 -> OK, bit 0 (a wait gave up) -> TIMEOUT (over any other bit),
    bit 2 (a list row outside [0, k)) -> LIST, unknown bits -> ARG."""
    assert lib.si_device_error_status(0) == _lib.SI_OK
    assert lib.si_device_error_status(1) == _lib.SI_ERR_TIMEOUT
    assert lib.si_device_error_status(4) == _lib.SI_ERR_LIST
    assert lib.si_device_error_status(5) == _lib.SI_ERR_TIMEOUT
    for bad in (2, 8, 0x80000000, 0xFFFFFFFF):
        assert lib.si_device_error_status(bad) == _lib.SI_ERR_ARG, bad
    assert "resident" in (lib.si_device_error_status(1) and _lib.last_error())


def test_workspace_check_and_read_h3_validation(lib):
    ws = lib.si_workspace_bytes(128, 256, 1)
    cases = [
        ("si_workspace_check", (None, ws, None), _lib.SI_ERR_NULL),
        ("si_workspace_check", (_p(A + 8), ws, None), _lib.SI_ERR_ALIGN),
        ("si_workspace_check", (_p(A), 255, None), _lib.SI_ERR_WORKSPACE),
        ("si_read_h3", (_p(A), ws, 128, 256, 1, None, _p(A), None), _lib.SI_ERR_NULL),
        ("si_read_h3", (_p(A), ws, 128, 256, 1, _p(A), None, None), _lib.SI_ERR_NULL),
        ("si_read_h3", (_p(A), ws, 128, 256, 9, _p(A), _p(A), None), _lib.SI_ERR_SHAPE),
        ("si_read_h3", (_p(A), ws - 1, 128, 256, 1, _p(A), _p(A), None), _lib.SI_ERR_WORKSPACE),
        ("si_read_h3", (None, ws, 128, 256, 1, _p(A), _p(A), None), _lib.SI_ERR_NULL),
        ("si_read_bandwidth_probe", (None, 1024, _p(A), None), _lib.SI_ERR_NULL),
        ("si_read_bandwidth_probe", (_p(A), 1024, None, None), _lib.SI_ERR_NULL),
        ("si_read_bandwidth_probe", (_p(A + 4), 1024, _p(A), None), _lib.SI_ERR_ALIGN),
        ("si_read_bandwidth_probe", (_p(A), 1000, _p(A), None), _lib.SI_ERR_SHAPE),
        ("si_read_bandwidth_probe", (_p(A), 0, _p(A), None), _lib.SI_ERR_SHAPE),
    ]
    for name, args, want in cases:
        st = _lib.status(name, *args)
        assert st == want, (name, args, st, _lib.last_error())


def test_noalloc_validation(lib):
    """The no-allocation entry point rejects shapes beyond its 8 MiB scratch
    and missing pointers before touching the device."""
    k, d, b = 1 << 20, 4096, 8
    assert lib.si_workspace_bytes(k, d, b) > 8 << 20
    args = (_p(A), _p(A), _p(A), _p(A), k, d, _p(A), b, 1.0, None, None, None, _p(A), 0, None, None)
    assert _lib.status("si_predict_sparse_mlp_noalloc", *args) == _lib.SI_ERR_WORKSPACE
    assert "scratch" in _lib.last_error()
    args = (_p(A), _p(A), None, _p(A), 11008, 4096, _p(A), 1, 1.0, None, None, None, _p(A), 0, None, None)
    assert _lib.status("si_predict_sparse_mlp_noalloc", *args) == _lib.SI_ERR_NULL
    args = (_p(A), _p(A), _p(A), _p(A), 11008, 4096, _p(A), 9, 1.0, None, None, None, _p(A), 0, None, None)
    assert _lib.status("si_predict_sparse_mlp_noalloc", *args) == _lib.SI_ERR_SHAPE
