"""Seeded random layer shapes against the oracle, forward and backward.

The fixed cases elsewhere pick shapes by hand; here a seeded generator draws
them from the whole legal space of the descriptor: model widths d (multiples
of 64), expert widths h (multiples of 64 for GELU, any width for SwiGLU),
1 to 1024 experts (most up to 300; a third of the cases at most 12, which
reach the 256-row tiles), K up to min(E, 16), 1 to 6000 tokens, with or without a
shared expert, bf16 or fp32 layers, uniform or zero selection bias. Routing is
compared bit for bit and y (or dx, dW1, dW2) within the tolerances of the
other parity tests, over every token. Shapes are kept small enough for the
oracle to run over every token in about a second.
"""

import numpy as np
import pytest
import torch

import oracle
from gpu_util import DeviceLayer, check_close, dev, host
from paper_2608_17402_amd import binding
from workloads import bf16_bits_to_f32, f32_to_bf16_bits, make_inputs, pad_last_dim
from workloads.configs import LayerConfig

pytestmark = pytest.mark.gpu

D_CHOICES = [64, 128, 192, 256, 320, 448, 512]
FLOP_CAP = 4.0e9  # multiply-adds of the oracle per case


def _draw(rng, i, backward=False):
    swiglu = rng.random() < 0.35
    dtype = "bf16" if (swiglu or backward or rng.random() < 0.8) else "f32"
    d = int(rng.choice(D_CHOICES))
    u = rng.random()  # few experts reach the 256-row tiles; many, the 1024-expert router paths
    E = int(rng.integers(1, 13)) if u < 0.3 else (int(rng.integers(300, 1025)) if u < 0.4 else int(rng.integers(1, 301)))
    K = int(rng.integers(1, min(E, 16) + 1))
    h = int(rng.integers(1, 701)) if swiglu else 64 * int(rng.integers(1, 11))
    hs = 0
    if not backward and rng.random() < 0.6:
        hs = int(rng.integers(1, 701)) if swiglu else 64 * int(rng.integers(1, 11))
    T = int(np.exp(rng.uniform(0.0, np.log(6000.0))))
    n_mats = 3 if swiglu else 2
    per_token = K * d * h * n_mats + d * hs * n_mats + d * E
    T = max(1, min(T, int(FLOP_CAP / per_token)))
    bias = "zero" if rng.random() < 0.2 else "uniform"
    return LayerConfig(name=f"rand{i}", T=T, d=d, E=E, K=K, h=h, h_shared=hs, dtype=dtype, bias=bias,
                       seed=1000 + i, act="swiglu" if swiglu else "gelu")


FWD = [_draw(np.random.default_rng(77 + i), i) for i in range(40)]
BWD = [_draw(np.random.default_rng(991 + i), i, backward=True) for i in range(16)]


def _cid(c):
    return f"{c.name}-T{c.T}-d{c.d}-E{c.E}-K{c.K}-h{c.h}-hs{c.h_shared}-{c.dtype}-{c.act}"


@pytest.mark.parametrize("cfg", FWD, ids=_cid)
def test_random_shape_layer_forward(cfg):
    inp = make_inputs(cfg)
    lay = DeviceLayer(inp)
    y, idx, gate = lay.forward()
    torch.cuda.synchronize()
    bf16 = cfg.dtype == "bf16"
    o_idx, o_gate, y_ref = oracle.layer(inp.f32("x"), inp.f32("w_router"), inp.bias, inp.f32("w1"), inp.f32("w2"),
                                        inp.f32("w1s"), inp.f32("w2s"), cfg.K, cfg.lam, bf16, act=cfg.act)
    assert np.array_equal(host(idx), o_idx), "routing differs"
    assert np.array_equal(host(gate), o_gate), "gates differ"
    check_close(host(y), y_ref, bf16, _cid(cfg))


def _check_grad(got, ref, what):
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    assert got.shape == ref.shape and np.all(np.isfinite(got)), what
    err = got - ref
    scale = max(1.0, float(np.max(np.abs(ref))) if ref.size else 1.0)
    max_abs = float(np.max(np.abs(err))) if err.size else 0.0
    den = float(np.linalg.norm(ref))
    rel = float(np.linalg.norm(err)) / den if den > 0 else float(np.linalg.norm(err))
    assert max_abs <= 2e-2 * scale and rel <= 5e-3, f"{what}: max_abs={max_abs:.3e} (scale {scale:.2f}), rel={rel:.3e}"


@pytest.mark.parametrize("cfg", BWD, ids=_cid)
def test_random_shape_backward(cfg):
    T, d, E, K, h = cfg.T, cfg.d, cfg.E, cfg.K, cfg.h
    sw = cfg.act == "swiglu"
    rng = np.random.default_rng(cfg.seed)
    x = f32_to_bf16_bits(rng.standard_normal((T, d)).astype(np.float32))
    w1 = f32_to_bf16_bits((rng.standard_normal((E, 2 * h if sw else h, d)) * 0.05).astype(np.float32))
    w2 = f32_to_bf16_bits((rng.standard_normal((E, d, h)) * 0.05).astype(np.float32))
    g = f32_to_bf16_bits((rng.standard_normal((T * K, d)) * 0.5).astype(np.float32))
    idx = np.stack([rng.choice(E, K, replace=False) for _ in range(T)]).astype(np.int32)
    w2p = pad_last_dim(w2, 64) if sw else w2
    desc = binding.make_desc(T, d, E, K, h, 0, 1.0, "bf16", flags=binding.MOE_FLAG_SWIGLU if sw else 0)
    ws = binding.alloc_workspace(desc)
    counts = torch.empty(E, dtype=torch.int32, device="cuda")
    offsets = torch.empty(E + 1, dtype=torch.int32, device="cuda")
    slots = torch.empty(T * K, dtype=torch.int32, device="cuda")
    binding.moe_permute(desc, dev(idx), counts, offsets, slots, ws)
    bws = binding.alloc_backward_workspace(desc)
    dx = torch.empty(T, d, dtype=torch.bfloat16, device="cuda")
    dw1 = torch.empty(E, w1.shape[1], d, dtype=torch.float32, device="cuda")
    dw2 = torch.empty(E, d, w2p.shape[2], dtype=torch.float32, device="cuda")
    binding.moe_grouped_mlp_backward(desc, dev(x), slots, offsets, dev(w1), dev(w2p), dev(g), dx, dw1, dw2, bws)
    torch.cuda.synchronize()
    rdx, rdw1, rdw2 = oracle.grouped_backward(bf16_bits_to_f32(x), idx, bf16_bits_to_f32(w1), bf16_bits_to_f32(w2),
                                              bf16_bits_to_f32(g), True, act=cfg.act)
    _check_grad(host(dx), rdx, f"{_cid(cfg)} dx")
    _check_grad(host(dw1), rdw1, f"{_cid(cfg)} dw1")
    got_w2 = host(dw2)
    if sw:  # padding columns of dW2 are zero
        assert np.all(got_w2[:, :, h:] == 0)
        got_w2 = got_w2[:, :, :h]
    _check_grad(got_w2, rdw2, f"{_cid(cfg)} dw2")
