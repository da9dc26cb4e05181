"""The layer step captured as a HIP graph (the launch mode ``bench.py`` times
by default): every replay reproduces the eager step, with eager steps and
synchronisations between replays."""
import pytest
import torch

from paper_2501_08582_amd import synth
from paper_2501_08582_amd.step import LayerStep

pytestmark = pytest.mark.gpu


def _rel(a, b):
    return float((a.double() - b.double()).norm()) / max(float(b.double().norm()), 1e-30)


_RAGGED = dict(R=520, C=776, L=300, r=24)


@pytest.mark.parametrize("name,ragged,ste", [("fp32_256x256_r8", False, False),
                                             ("llama2_7b_q_proj", True, False),
                                             ("llama2_7b_q_proj", True, True),
                                             ("llama2_7b_q_proj", False, False),
                                             ("llama2_7b_q_proj", False, True)],
                         ids=["fp32", "bf16-ragged", "bf16-ragged-ste", "bf16-4096", "bf16-4096-ste"])
def test_graph_replays_match_eager(name, ragged, ste):
    wl = synth.workload(name)
    if ragged:
        wl = wl.with_(name=wl.name + "_ragged", **_RAGGED)
    layer = LayerStep(synth.make(wl), ste=ste)
    layer.run()
    torch.cuda.synchronize()
    outs = (layer.Y, layer.dX, layer.dB, layer.dA)
    ref = [t.clone() for t in outs]
    graph = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        layer.run()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    with torch.cuda.graph(graph):
        layer.run()
    torch.cuda.synchronize()
    for rep in range(4):
        for t in outs:
            t.zero_()
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(layer.Y, ref[0]), f"replay {rep}: Y"
        assert torch.equal(layer.dX, ref[1]), f"replay {rep}: dX"
        assert _rel(layer.dB, ref[2]) <= 1e-5 and _rel(layer.dA, ref[3]) <= 1e-5, f"replay {rep}: dB/dA"
        layer.run()  # eager work between replays
        torch.cuda.synchronize()
        assert torch.equal(layer.Y, ref[0]) and torch.equal(layer.dX, ref[1])
