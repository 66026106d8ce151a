"""One layer step captured as a HIP graph (LayerGraph): every replay gives the bits
of the eager step on the same inputs -- replays interleaved with eager steps on the
same layer buffers, and replays after new inputs are copied into the captured
tensors (the graph reads them by address).  bf16 with and without the gather, with
a shared expert, and the MXFP8 layer."""
import pytest
import torch

import moegen
import paper_2606_21712_amd as moe
from gpu_util import log, to_dev

pytestmark = pytest.mark.gpu

# a small DeepSeek-style layer: shared expert, ragged groups, several m- and n-tiles
CFG = moegen.CONFIGS["deepseek"].scaled(name="graph_small", T=1500, H=256, E=12, k=3, F=384, Fs=256, seed=31)


def _same(a, b):
    return torch.equal(a.view(torch.int16), b.view(torch.int16))


def _weights(I, mx):
    w = [to_dev(a) for a in (I.w_gate, I.w_up, I.w_down, I.ws_gate, I.ws_up, I.ws_down)]
    return [moe.quantize_weights_mxfp8(t) for t in w] if mx else w


@pytest.mark.parametrize("mode", ["bf16_gather", "bf16_xperm", "mxfp8"])
def test_layer_graph_replays_match_eager(mode):
    c = CFG
    Ia, Ib = moegen.make_inputs(c), moegen.make_inputs(c, seed=c.seed + 1)
    mx = mode == "mxfp8"
    W = _weights(Ia, mx)                                   # one set of weights for both inputs

    def make_layer():
        if mx:
            return moe.MoELayerMXFP8(c.T, c.H, c.E, c.k, c.F, c.Fs)
        return moe.MoELayer(c.T, c.H, c.E, c.k, c.F, c.Fs, gather=(mode == "bf16_gather"))

    xa, la, xb, lb = to_dev(Ia.x), to_dev(Ia.logits), to_dev(Ib.x), to_dev(Ib.logits)
    log(f"[gpu] graph {mode}: eager reference steps")
    ref = make_layer()
    ya = ref.run(xa, la, *W).clone()
    yb = ref.run(xb, lb, *W).clone()
    torch.cuda.synchronize()
    assert not _same(ya, yb)

    layer = make_layer()
    x, lg = xa.clone(), la.clone()                         # the captured input tensors
    log(f"[gpu] graph {mode}: capture")
    g = moe.LayerGraph(layer, x, lg, *W)
    torch.cuda.synchronize()
    for rep in range(3):
        log(f"[gpu] graph {mode}: replay {rep} on inputs a")
        x.copy_(xa)
        lg.copy_(la)
        y = g.replay()
        torch.cuda.synchronize()
        assert _same(y, ya), (mode, rep, "a")
        log(f"[gpu] graph {mode}: eager step on inputs b, same layer buffers")
        layer.run(xb, lb, *W)
        torch.cuda.synchronize()
        assert _same(layer.y, yb), (mode, rep, "eager b")
        log(f"[gpu] graph {mode}: replay {rep} on inputs b")
        x.copy_(xb)
        lg.copy_(lb)
        g.replay()
        torch.cuda.synchronize()
        assert _same(layer.y, yb), (mode, rep, "b")
