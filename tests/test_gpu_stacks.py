"""Parity on the decode stacks: 32 layers of the 7B-shaped MLP block with
per-layer planted sparsity drawn from U(0.85, 0.95), and 40 layers of the
13B-shaped block at 0.88.  Each layer's input is built from the previous
layer's output (``synth.stack_input``), as in sequential decode.

At full size the oracle cannot follow every layer, so: every layer's kept
set must equal its planted active set (the inputs carry the layer's
reference signs; the oracle tests pin this property on planted layers), and
sampled (layer, token) pairs are recomputed by the oracle from the very
input the GPU path received: mask and kept list bit-exact, y within 1e-2
relative L2.
"""

import numpy as np
import pytest
import torch

import oracle
import paper_2411_12692_amd as si
from paper_2411_12692_amd import synth

pytestmark = pytest.mark.gpu
DEV = "cuda"


def u16(t: torch.Tensor) -> np.ndarray:
    return t.detach().cpu().contiguous().view(torch.int16).numpy().view(np.uint16)


def rel_l2(a, b):
    return float(np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300))


STACKS = [
    pytest.param(dict(d=4096, k=11008, layers=32, s=(0.85, 0.95), config=3), id="7b-32-layers"),
    pytest.param(dict(d=5120, k=13824, layers=40, s=(0.88, 0.88), config=4), id="13b-40-layers"),
]


@pytest.mark.parametrize("cfg", STACKS)
def test_stack_decode(cfg):
    d, k, nl, config = cfg["d"], cfg["k"], cfg["layers"], cfg["config"]
    lo, hi = cfg["s"]
    sp = synth.stack_sparsities(nl, lo, hi, config) if hi > lo else [lo] * nl
    sample = {0, nl // 2, nl - 1}
    tokens = 2
    layers, planted, host = [], [], {}
    for l in range(nl):
        wg, wu, wd, inactive, _ = synth.stack_layer(d, k, sp[l], config, l, device=DEV)
        layers.append(si.MLPLayer(wg, wu, wd))
        planted.append((~inactive).to(torch.uint8))
        if l in sample:
            host[l] = (u16(wg), u16(wu), u16(wd))
        del wd, inactive
    torch.cuda.synchronize()
    records = []
    for t in range(tokens):
        y = None
        for l in range(nl):
            x = synth.stack_input(y, d, 1, config, l, t, device=DEV)
            y, (mask, idx, n, _) = layers[l](x, 1.0, outputs=True)
            assert torch.equal(mask, planted[l]), f"layer {l} token {t}: kept set differs from the planted one"
            if l in sample:
                records.append((l, t, u16(x), mask.cpu().numpy(), idx.cpu().numpy(), int(n.item()),
                                y.cpu().numpy().astype(np.float64)))
    torch.cuda.synchronize()
    for lay in layers:
        assert si.workspace_check(lay.workspace) == 0
    for l, t, x, mask, idx, n, y in records:
        wg, wu, wd = host[l]
        packed = oracle.pack_signs(wg)
        m_ref, _, _ = oracle.predict_rows(packed, x, 1.0)
        assert np.array_equal(mask, m_ref), (l, t)
        ref_idx = oracle.active_rows(m_ref)
        assert n == ref_idx.size and np.array_equal(idx[:n], ref_idx), (l, t)
        out = oracle.sparse_mlp(wg, wu, wd, x, m_ref)
        err = rel_l2(y, out["y"])
        assert err <= 1e-2, (l, t, err)
        scale = np.abs(out["y"]).max()
        assert np.abs(y - out["y"]).max() <= 1e-4 * scale, (l, t)
    del layers
    torch.cuda.empty_cache()
