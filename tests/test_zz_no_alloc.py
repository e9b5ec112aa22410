"""The allocation-free layer forward (moe_layer_forward_noalloc) against
moe_layer_forward with a caller workspace, through the C ABI: two calls in a
row on the library's per-GPU scratch, the second with fewer tokens (so it
runs on what the first call left in the scratch), each bit-identical to the
workspace entry point (routing, gates and y), and the second also within the
layer tolerances of the oracle. A descriptor whose workspace exceeds the
scratch is refused before anything is enqueued."""

import numpy as np
import pytest
import torch

import oracle
from gpu_util import DeviceLayer, check_close, host
from paper_2608_17402_amd import binding
from workloads import get_config, make_inputs

pytestmark = pytest.mark.gpu


def _bits(t):
    return t.view(torch.int16) if t.dtype == torch.bfloat16 else t.view(torch.int32)


def _noalloc(lay):
    d = lay.desc
    y = lay.empty(d.T, d.d)
    idx = lay.empty(d.T, d.K, dtype=torch.int32)
    gate = lay.empty(d.T, d.K, dtype=torch.float32)
    binding.moe_layer_forward_noalloc(d, lay.x, lay.w_router, lay.bias, lay.w1, lay.w2, lay.w1s, lay.w2s, y, idx,
                                      gate)
    return y, idx, gate


@pytest.mark.parametrize("name,T1,T2", [("c5", None, 300), ("c1", None, 77), ("c2", 2000, 513)])
def test_noalloc_matches_workspace_entry_point(name, T1, T2):
    cfg = get_config(name)
    results = []
    for T in (T1, T2):
        c = cfg if T is None else cfg.with_tokens(T)
        inp = make_inputs(c)
        lay = DeviceLayer(inp)
        assert binding.workspace_size(lay.desc) <= binding.NOALLOC_SCRATCH_BYTES
        y_n, i_n, g_n = _noalloc(lay)
        y_w, i_w, g_w = lay.forward()
        torch.cuda.synchronize()
        assert torch.equal(i_n, i_w) and torch.equal(_bits(g_n), _bits(g_w)), f"{name} T={c.T}: routing differs"
        assert torch.equal(_bits(y_n), _bits(y_w)), f"{name} T={c.T}: y differs from moe_layer_forward"
        results.append((c, inp, y_n, i_n))
    # The second (smaller) call also against the oracle.
    c, inp, y_n, i_n = results[1]
    bf16 = c.dtype == "bf16"
    o_idx, _, y_ref = oracle.layer(inp.f32("x"), inp.f32("w_router"), inp.bias, inp.f32("w1"), inp.f32("w2"),
                                   inp.f32("w1s"), inp.f32("w2s"), c.K, c.lam, bf16)
    assert np.array_equal(host(i_n), o_idx)
    check_close(host(y_n), y_ref, bf16, f"{name} noalloc y")


def test_noalloc_refuses_oversize_layer():
    cfg = get_config("c4")
    desc = binding.make_desc(cfg.T, cfg.d, cfg.E, cfg.K, cfg.h, cfg.h_shared, cfg.lam, cfg.dtype)
    assert binding.workspace_size(desc) > binding.NOALLOC_SCRATCH_BYTES
    z = torch.zeros(16, dtype=torch.bfloat16, device="cuda")
    with pytest.raises(binding.MoeError) as e:
        binding.moe_layer_forward_noalloc(desc, z, z, None, z, z, z, z, z)
    assert e.value.status == 3 and "scratch" in str(e.value)
