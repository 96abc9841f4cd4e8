"""Seeded synthetic inputs shaped like the workloads of SparseInfer's evaluation.

This module only draws random numbers and lays them out; it contains none of
the method's arithmetic (no sign packing, counting, thresholding or GEMV).  It
serves both the HIP path's tests/benchmarks and the CPU oracle, which is the
only thing the two sides share.

The paper evaluates ReLU-fied Llama-2 models (ProSparse-Llama2-7B/13B) whose
inputs and gate rows it observes to be zero-mean and close to Gaussian
(Section IV-A, Fig. 2), with roughly 90% activation sparsity (Section IV).
Real weights are not available here; the *planted* construction below stands
in for them:

* ``x ~ N(0, 1)`` in fp16.
* ``round(s * k)`` gate rows are chosen inactive by a seeded permutation.
* For every gate element an independent coin decides whether its sign
  disagrees with ``sign(x_j)``: probability 0.6 on inactive rows, 0.4 on
  active rows.  Magnitudes are ``|N(0, 0.02)|``; the sign bit is set on the
  fp16 bit pattern so that a magnitude that rounds to zero keeps its sign.
* ``W_up`` and ``W_down`` are ``N(0, 0.02)`` in fp16; ``W_down`` is stored
  ``[d][k]``.

Every tensor is drawn from its own ``torch.Generator`` seeded from
``SeedSequence([12692, config, layer, tensor_id])``.  The draws depend on the
device (CPU and GPU generators differ), so a test that compares two sides
generates once and hands the same arrays to both.
"""

from __future__ import annotations

import math
from dataclasses import dataclass

import numpy as np
import torch

_TENSOR_IDS = {
    "x": 0, "perm": 1, "disagree": 2, "gate_mag": 3, "up": 4, "down": 5,
    "noise": 6, "ref_sign": 7, "tokens": 8, "token_sets": 9, "sparsity": 10, "calib": 11,
}


def generator(config: int, layer: int, tensor: str, device="cpu") -> torch.Generator:
    """Independent, reproducible generator for one tensor of one layer."""
    ss = np.random.SeedSequence([12692, int(config), int(layer), _TENSOR_IDS[tensor]])
    seed = int(ss.generate_state(1, dtype=np.uint64)[0]) & ((1 << 63) - 1)
    g = torch.Generator(device=torch.device(device))
    g.manual_seed(seed)
    return g


def n_inactive(k: int, s: float) -> int:
    """Number of planted-inactive rows: ``floor(s * k + 0.5)``."""
    return int(math.floor(s * k + 0.5))


def fp16_with_sign(magnitude: torch.Tensor, negative: torch.Tensor) -> torch.Tensor:
    """fp16 tensor with ``|magnitude|`` rounded to fp16 and the sign bit taken
    from ``negative`` (set on the bit pattern, so -0.0 is produced where the
    magnitude rounds to zero)."""
    m = magnitude.abs().to(torch.float16).view(torch.int16)
    m = m & 0x7FFF  # Python scalars keep int16 and need no host-to-device copy (graph capture)
    return torch.where(negative, m | -32768, m).view(torch.float16)  # -32768: the 0x8000 sign bit


@dataclass
class PlantedLayer:
    """One gated-MLP layer with planted gate-row sparsity.

    ``w_gate``, ``w_up``: ``[k][d]`` fp16; ``w_down``: ``[d][k]`` fp16;
    ``x``: ``[b][d]`` fp16; ``inactive``: ``[k]`` bool (the planted choice).
    """
    d: int
    k: int
    s: float
    x: torch.Tensor
    w_gate: torch.Tensor
    w_up: torch.Tensor
    w_down: torch.Tensor
    inactive: torch.Tensor


def planted_gate(d: int, k: int, s: float, ref_negative: torch.Tensor,
                 config: int, layer: int, device="cpu", p_active: float = 0.4, p_inactive: float = 0.6):
    """``W_gate [k][d]`` fp16 planted against the sign pattern ``ref_negative``
    (``[d]`` bool, True = negative), plus the ``[k]`` bool inactive set.
    Elements disagree in sign with the pattern with probability ``p_active``
    on active rows and ``p_inactive`` on inactive rows (0.4 / 0.6 by default;
    values closer to 0.5 make the sign-bit prediction less certain)."""
    perm = torch.randperm(k, generator=generator(config, layer, "perm", device), device=device)
    inactive = torch.zeros(k, dtype=torch.bool, device=device)
    inactive[perm[: n_inactive(k, s)]] = True
    p_disagree = torch.where(inactive, p_inactive, p_active).to(device)
    coins = torch.rand(k, d, generator=generator(config, layer, "disagree", device), device=device)
    disagree = coins < p_disagree[:, None]
    del coins
    mag = torch.randn(k, d, generator=generator(config, layer, "gate_mag", device), device=device)
    mag.mul_(0.02)
    w_gate = fp16_with_sign(mag, ref_negative[None, :] ^ disagree)
    return w_gate, inactive


def normal_fp16(shape, std: float, config: int, layer: int, tensor: str, device="cpu"):
    t = torch.randn(*shape, generator=generator(config, layer, tensor, device), device=device)
    return t.mul_(std).to(torch.float16)


def planted_layer(d: int, k: int, s: float, config: int = 1, layer: int = 0,
                  device="cpu", p_active: float = 0.4, p_inactive: float = 0.6) -> PlantedLayer:
    """Single-token layer of the planted construction (see module docstring)."""
    x = normal_fp16((1, d), 1.0, config, layer, "x", device)
    x_negative = x[0].view(torch.int16) < 0
    w_gate, inactive = planted_gate(d, k, s, x_negative, config, layer, device, p_active, p_inactive)
    w_up = normal_fp16((k, d), 0.02, config, layer, "up", device)
    w_down = normal_fp16((d, k), 0.02, config, layer, "down", device)
    return PlantedLayer(d, k, s, x, w_gate, w_up, w_down, inactive)


def batch_tokens(layer: PlantedLayer, b: int, config: int, layer_id: int = 0) -> torch.Tensor:
    """``[b][d]`` fp16 decode batch whose token 0 is the layer's planted token
    and tokens 1..b-1 are fresh iid ``N(0, 1)``."""
    dev = layer.x.device
    if b == 1:
        return layer.x.clone()
    extra = normal_fp16((b - 1, layer.d), 1.0, config, layer_id, "tokens", dev)
    return torch.cat([layer.x, extra], dim=0)


def batch_union_mask(layer: PlantedLayer, b: int, config: int, layer_id: int = 0) -> torch.Tensor:
    """Union over ``b`` tokens of per-token active sets, as ``[k]`` uint8.

    For a fixed row and isotropic Gaussian tokens a row is positive for half
    of the tokens, so iid tokens cannot all be sparse; the sparsity/batch
    sweep therefore draws the per-token active sets directly: token 0 keeps
    the planted active set, tokens 1..b-1 draw independent sets of the same
    size.
    """
    k, dev = layer.k, layer.inactive.device
    mask = ~layer.inactive
    n_act = k - n_inactive(k, layer.s)
    g = generator(config, layer_id, "token_sets", dev)
    for _ in range(1, b):
        perm = torch.randperm(k, generator=g, device=dev)
        extra = torch.zeros(k, dtype=torch.bool, device=dev)
        extra[perm[:n_act]] = True
        mask = mask | extra
    return mask.to(torch.uint8)


def reference_signs(d: int, config: int, layer: int, device="cpu") -> torch.Tensor:
    """Seeded reference sign pattern (``[d]`` bool, True = negative) that a
    stacked layer's gate rows are planted against."""
    g = generator(config, layer, "ref_sign", device)
    return torch.rand(d, generator=g, device=device) < 0.5


def stack_layer(d: int, k: int, s: float, config: int, layer: int, device="cpu",
                p_active: float = 0.4, p_inactive: float = 0.6):
    """Layer ``layer`` of a planted stack: gate rows planted against
    :func:`reference_signs` of that layer.  Returns ``(w_gate, w_up, w_down,
    inactive, ref_negative)``."""
    ref = reference_signs(d, config, layer, device)
    w_gate, inactive = planted_gate(d, k, s, ref, config, layer, device, p_active, p_inactive)
    w_up = normal_fp16((k, d), 0.02, config, layer, "up", device)
    w_down = normal_fp16((d, k), 0.02, config, layer, "down", device)
    return w_gate, w_up, w_down, inactive, ref


def stack_sparsities(n_layers: int, lo: float, hi: float, config: int) -> list:
    """Per-layer planted sparsity drawn from ``U(lo, hi)`` (seeded)."""
    g = generator(config, 0, "sparsity", "cpu")
    u = torch.rand(n_layers, generator=g, dtype=torch.float64)
    return [float(lo + (hi - lo) * v) for v in u]


def stack_noise(d: int, b: int, config: int, layer: int, token: int, device="cpu") -> torch.Tensor:
    """Fresh ``N(0, 1)`` noise ``[b][d]`` float32 for one (layer, token)."""
    g = generator(config, layer * 1_000_003 + token, "noise", device)
    return torch.randn(b, d, generator=g, device=device)


def stack_input(y_prev, d: int, b: int, config: int, layer: int, token: int, device="cpu") -> torch.Tensor:
    """Input ``[b][d]`` fp16 of layer ``layer`` of a planted stack at decode
    step ``token``.

    The magnitudes come from the previous layer's output, normalised to unit
    RMS, plus fresh ``N(0, 1)`` noise (``|noise|`` alone for layer 0); the
    signs are the layer's reference pattern, which its gate rows are planted
    against, so each layer keeps its planted active set for every token.
    This is harness glue between stacked MLP blocks, not part of the method.
    """
    eps = stack_noise(d, b, config, layer, token, device)
    return stack_glue(y_prev, eps, reference_signs(d, config, layer, device))


def stack_glue(y_prev, eps: torch.Tensor, negative: torch.Tensor) -> torch.Tensor:
    """The chaining of :func:`stack_input` from its random draws: ``eps``
    ``[b][d]`` float32 noise and the layer's reference signs ``negative``
    (``[d]`` bool).  Only elementwise torch operations, so a benchmark can
    replay it from a graph with the noise of each token gathered from a
    precomputed buffer."""
    b, d = eps.shape
    if y_prev is None:
        mag = eps.abs()
    else:
        y = y_prev.float().reshape(b, d)
        rms = y.pow(2).mean(dim=-1, keepdim=True).sqrt().clamp_min(1e-30)
        mag = (y / rms + eps).abs()
    return fp16_with_sign(mag, negative[None, :].expand(b, d))


def calibration_tokens(d: int, n: int, config: int, layer: int, flip: float = 0.0, device="cpu") -> torch.Tensor:
    """``[n][d]`` fp16 tokens for calibrating a stacked layer: magnitudes
    ``|N(0, 1)|``, signs the layer's reference pattern with each sign flipped
    independently with probability ``flip`` (0 keeps the planted relation)."""
    g = generator(config, layer, "calib", device)
    mag = torch.randn(n, d, generator=g, device=device).abs()
    flips = torch.rand(n, d, generator=g, device=device) < flip
    neg = reference_signs(d, config, layer, device)[None, :] ^ flips
    return fp16_with_sign(mag, neg)
