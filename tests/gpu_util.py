"""Helpers shared by the GPU parity tests: moving seeded inputs to the device,
running the C ABI through the binding, and the tolerance checks."""

from __future__ import annotations

import numpy as np
import torch

from paper_2608_17402_amd import binding
from workloads import bf16_bits_to_f32, pad_last_dim

BF16_MAX_ABS = 2e-2
BF16_REL_L2 = 5e-3
F32_MAX_ABS = 1e-5
F32_REL_L2 = 1e-5


def dev(a: np.ndarray | None) -> torch.Tensor | None:
    """numpy (bf16 bit patterns as uint16, or float32/int32) -> device tensor."""
    if a is None:
        return None
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        return torch.from_numpy(a.view(np.int16)).cuda().view(torch.bfloat16)
    return torch.from_numpy(a).cuda()


def host(t: torch.Tensor) -> np.ndarray:
    """Device tensor -> numpy; bf16 widened exactly to float32."""
    if t.dtype == torch.bfloat16:
        return bf16_bits_to_f32(t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16))
    return t.cpu().numpy()


def desc_for(cfg, T=None, **over):
    flags = binding.MOE_FLAG_SWIGLU if getattr(cfg, "act", "gelu") == "swiglu" else 0
    kw = dict(T=cfg.T if T is None else T, d=cfg.d, E=cfg.E, K=cfg.K, h=cfg.h, h_shared=cfg.h_shared,
              lam=cfg.lam, dtype=cfg.dtype, flags=flags)
    kw.update(over)
    return binding.make_desc(**kw)


def pad_cols(a: np.ndarray | None, mult: int = 64) -> np.ndarray | None:
    """Zero-pad the last axis to a multiple of `mult` (the second-layer weight
    layout of SwiGLU experts: rows of ldh = h rounded up to 64)."""
    return pad_last_dim(a, mult)


def check_close(got: np.ndarray, ref: np.ndarray, bf16: bool, what: str = ""):
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    assert got.shape == ref.shape, (got.shape, ref.shape)
    assert np.all(np.isfinite(got)), f"{what}: non-finite output"
    err = got - ref
    max_abs = float(np.max(np.abs(err))) if err.size else 0.0
    den = float(np.linalg.norm(ref))
    rel = float(np.linalg.norm(err)) / den if den > 0 else float(np.linalg.norm(err))
    lim_abs, lim_rel = (BF16_MAX_ABS, BF16_REL_L2) if bf16 else (F32_MAX_ABS, F32_REL_L2)
    assert max_abs <= lim_abs and rel <= lim_rel, \
        f"{what}: max_abs={max_abs:.3e} (<= {lim_abs}), rel_l2={rel:.3e} (<= {lim_rel})"
    return max_abs, rel


class DeviceLayer:
    """Device copies of one layer's inputs plus a workspace."""

    def __init__(self, inp, T=None):
        # The kernels read T rows of x through a raw pointer: T past the rows
        # that exist would read outside the allocation.
        if T is not None and not 0 <= T <= inp.x.shape[0]:
            raise ValueError(f"T = {T} but the inputs hold {inp.x.shape[0]} token rows")
        self.inp = inp
        self.cfg = inp.cfg
        self.desc = desc_for(self.cfg, T)
        self.x = dev(inp.x)
        self.w_router = dev(inp.w_router)
        self.bias = dev(inp.bias)
        self.w1 = dev(inp.w1)
        swiglu = getattr(self.cfg, "act", "gelu") == "swiglu"
        self.w2 = dev(pad_cols(inp.w2) if swiglu else inp.w2)
        self.w1s = dev(inp.w1s)
        self.w2s = dev(pad_cols(inp.w2s) if swiglu else inp.w2s)
        self.ws = binding.alloc_workspace(self.desc)
        self.dt = binding.torch_dtype(self.desc)

    def empty(self, *shape, dtype=None):
        return torch.empty(*shape, dtype=dtype or self.dt, device="cuda")

    def route(self, bias="default"):
        d = self.desc
        idx = self.empty(d.T, d.K, dtype=torch.int32)
        gate = self.empty(d.T, d.K, dtype=torch.float32)
        b = self.bias if bias == "default" else bias
        binding.moe_route(d, self.x, self.w_router, b, idx, gate, self.ws)
        return idx, gate

    def permute(self, idx):
        d = self.desc
        counts = self.empty(d.E, dtype=torch.int32)
        offsets = self.empty(d.E + 1, dtype=torch.int32)
        slots = self.empty(d.T * d.K, dtype=torch.int32)
        binding.moe_permute(d, idx, counts, offsets, slots, self.ws)
        return counts, offsets, slots

    def grouped_mlp(self, slots, offsets):
        d = self.desc
        eo = self.empty(d.T * d.K, d.d)
        binding.moe_grouped_mlp(d, self.x, slots, offsets, self.w1, self.w2, eo, self.ws)
        return eo

    def forward(self, with_routing=True):
        d = self.desc
        y = self.empty(d.T, d.d)
        idx = self.empty(d.T, d.K, dtype=torch.int32) if with_routing else None
        gate = self.empty(d.T, d.K, dtype=torch.float32) if with_routing else None
        binding.moe_layer_forward(d, self.x, self.w_router, self.bias, self.w1, self.w2, self.w1s, self.w2s, y,
                                  idx, gate, self.ws)
        return y, idx, gate
