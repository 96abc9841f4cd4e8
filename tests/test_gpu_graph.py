"""Calls replayed from a HIP graph give the eager results on every replay.

The benchmark times the path from graph replays, and the kernels keep a call
counter in the workspace on the device (the tags of the exchange words), so
replays of one captured call must behave like fresh calls.  A graph of calls
over several layers (fp16 gated, non-gated, INT8 and decoder-block forms, at
one and three tokens; and one token at the 13B shape, whose groups of more
than 512 rows take the instance with the wider down batches) is replayed
several times, with eager calls on the same workspaces in between; masks,
kept lists and counts must equal the eager call's bit for bit and y must
match it to fp32 summation order.
"""

import numpy as np
import pytest
import torch

import paper_2411_12692_amd as si
from paper_2411_12692_amd import synth

pytestmark = pytest.mark.gpu

DEV = "cuda"


def make_layers(form, b, n_layers=3, d=1024, k=2752):
    out = []
    for l in range(n_layers):
        pl = synth.planted_layer(d, k, 0.9, config=9, layer=l, device=DEV)
        x = synth.batch_tokens(pl, b, config=9, layer_id=l)
        if form == "int8":
            layer = si.Int8MLPLayer(pl.w_gate, pl.w_up, pl.w_down, max_batch=b)
        else:
            layer = si.MLPLayer(pl.w_gate, None if form == "relu" else pl.w_up, pl.w_down, max_batch=b)
        g = torch.Generator(device="cpu").manual_seed(77 + l)
        h = (x.float() * 3.0).contiguous()
        nw = (0.5 + torch.rand(d, generator=g)).to(DEV)
        out.append((layer, x, h, nw))
    return out


def call(form, layer, x, h, nw, y):
    if form == "block":
        return layer.block(h, nw, 1e-5, 1.0, outputs=True, y=y)
    return layer(x, 1.0, outputs=True, y=y)


def snapshot(res):
    y, (mask, idx, n, cnt) = res
    nn = int(n.item())
    return (y.cpu().numpy().copy(), mask.cpu().numpy().copy(), idx.cpu().numpy()[:nn].copy(), nn,
            cnt.cpu().numpy().copy())


@pytest.mark.parametrize("form", ["gated", "relu", "int8", "block"])
@pytest.mark.parametrize("b", [1, 3])
def test_graph_replays_match_eager(form, b):
    replay_and_compare(form, b, make_layers(form, b))


@pytest.mark.parametrize("form", ["gated", "int8", "block"])
def test_graph_replays_large_groups(form):
    # 13B shape: on 256 compute units, groups of 10 blocks x 56 rows = 560 rows
    replay_and_compare(form, 1, make_layers(form, 1, d=5120, k=13824))


def replay_and_compare(form, b, layers):
    print(f"form={form} b={b} d={layers[0][1].shape[1]}", flush=True)
    ys = [torch.empty(b, layers[0][1].shape[1], dtype=torch.float32, device=DEV) for _ in layers]
    eager = []
    for (layer, x, h, nw), y in zip(layers, ys):
        eager.append(snapshot(call(form, layer, x, h, nw, y)))
    torch.cuda.synchronize()

    stream = torch.cuda.Stream()
    with torch.cuda.stream(stream):
        for (layer, x, h, nw), y in zip(layers, ys):
            call(form, layer, x, h, nw, y)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=stream):
        outs = [call(form, layer, x, h, nw, y) for (layer, x, h, nw), y in zip(layers, ys)]
    torch.cuda.synchronize()

    for rep in range(4):
        graph.replay()
        torch.cuda.synchronize()
        for l, (res, ref) in enumerate(zip(outs, eager)):
            got = snapshot(res)
            assert np.array_equal(got[1], ref[1]), (rep, l, "mask")
            assert got[3] == ref[3] and np.array_equal(got[2], ref[2]), (rep, l, "kept list")
            assert np.array_equal(got[4], ref[4]), (rep, l, "counters")
            scale = max(float(np.abs(ref[0]).max()), 1e-30)
            assert np.abs(got[0] - ref[0]).max() <= 1e-5 * scale, (rep, l, "y")
        # eager calls on the same workspaces between the replays
        layer, x, h, nw = layers[rep % len(layers)]
        call(form, layer, x, h, nw, torch.empty_like(ys[0]))
        torch.cuda.synchronize()
    for layer, *_ in layers:
        assert si.workspace_check(layer.workspace) == 0  # no wait ran out
