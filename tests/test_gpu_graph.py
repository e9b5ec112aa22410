"""The layer forward captured into a HIP graph (torch.cuda.CUDAGraph around
the C-ABI calls on the capture stream): moe_layer_forward with a caller
workspace, and the allocation-free moe_layer_forward_noalloc, whose callers
include code under graph capture. Each graph is replayed three times, with
eager calls of the same layer and synchronisations between the replays, and
every replay's output must equal the eager output bit for bit. The layer
enqueues kernels only (no memset nodes: its counters are zeroed by kernels)."""

import pytest
import torch

from gpu_util import DeviceLayer
from paper_2608_17402_amd import binding
from workloads import get_config, make_inputs

pytestmark = pytest.mark.gpu


def _bits(t):
    return t.view(torch.int16) if t.dtype == torch.bfloat16 else t.view(torch.int32)


@pytest.mark.parametrize("entry", ["workspace", "noalloc"])
@pytest.mark.parametrize("name,T", [("c5", None), ("c2", 700), ("c1", None)])
def test_layer_graph_replays_match_eager(name, T, entry):
    cfg = get_config(name)
    if T is not None:
        cfg = cfg.with_tokens(T)
    lay = DeviceLayer(make_inputs(cfg))
    d = lay.desc
    y = lay.empty(d.T, d.d)
    idx = lay.empty(d.T, d.K, dtype=torch.int32)
    gate = lay.empty(d.T, d.K, dtype=torch.float32)
    s = torch.cuda.Stream()

    def run():
        st = torch.cuda.current_stream()
        if entry == "noalloc":
            binding.moe_layer_forward_noalloc(d, lay.x, lay.w_router, lay.bias, lay.w1, lay.w2, lay.w1s, lay.w2s,
                                              y, idx, gate, stream=st)
        else:
            binding.moe_layer_forward(d, lay.x, lay.w_router, lay.bias, lay.w1, lay.w2, lay.w1s, lay.w2s, y, idx,
                                      gate, lay.ws, stream=st)

    # Eager reference (also the first call on this device, outside capture).
    with torch.cuda.stream(s):
        run()
    torch.cuda.synchronize()
    ref = (_bits(y).clone(), idx.clone(), _bits(gate).clone())

    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        run()
    torch.cuda.synchronize()
    for rep in range(3):
        y.zero_()
        idx.zero_()
        gate.zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(_bits(y), ref[0]), f"{name} {entry}: replay {rep} y differs"
        assert torch.equal(idx, ref[1]) and torch.equal(_bits(gate), ref[2]), f"{name} {entry}: replay {rep} routing"
        with torch.cuda.stream(s):  # eager work between replays
            run()
        torch.cuda.synchronize()
        assert torch.equal(_bits(y), ref[0])
    del g
