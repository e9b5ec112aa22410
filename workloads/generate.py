"""Seeded synthetic inputs for one MoE layer.

Recipe (one fixed order, each tensor from its own child of
``numpy.random.SeedSequence(cfg.seed).spawn(7)`` so that generating one tensor
never shifts another):

  0  x    [T, d]        N(0, 1)
  1  W_r  [E, d]        N(0, weight_std)     router, nn.Linear layout [out, in]
  2  b    [E]           per ``cfg.bias``: U(-0.1, 0.1), zeros, or the stored
                        Zipf-load bias vector (fp32)
  3  W1   [E, h, d]     N(0, weight_std)     fc1 of every routed expert
  4  W2   [E, d, h]     N(0, weight_std)     fc2 of every routed expert
  5  W1s  [h_s, d]      N(0, weight_std)     shared expert fc1 (if h_s > 0)
  6  W2s  [d, h_s]      N(0, weight_std)     shared expert fc2

SwiGLU experts draw W1 as [E, 2h, d] and W1s as [2 h_s, d] (gate rows, then
up rows) from the same streams.

Normal draws are float32; a bf16 layer stores the round-to-nearest-even bf16 of
each draw (kept as raw uint16 bit patterns here). x rows are drawn row-major in
one call, so the first T' rows of a config are the whole x of the same config
with T' tokens.
"""

from __future__ import annotations

import os
from dataclasses import dataclass
from typing import Iterable, Optional

import numpy as np

from .configs import LayerConfig

_N_STREAMS = 7
_ORDER = ("x", "w_router", "bias", "w1", "w2", "w1s", "w2s")

_HERE = os.path.dirname(os.path.abspath(__file__))
_REPO = os.path.dirname(_HERE)
ZIPF_BIAS_FILE = os.path.join(_REPO, "tests", "golden", "vitg_skew_bias_seed0.txt")


def f32_to_bf16_bits(a: np.ndarray, chunk: int = 1 << 24) -> np.ndarray:
    """Round float32 values to bf16 (nearest, ties to even); return uint16 bit
    patterns. Inputs are finite."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    flat = a.reshape(-1)
    out = np.empty(flat.shape, dtype=np.uint16)
    for s in range(0, flat.size, chunk):
        u = flat[s:s + chunk].view(np.uint32)
        lsb = (u >> np.uint32(16)) & np.uint32(1)
        out[s:s + chunk] = ((u + np.uint32(0x7FFF) + lsb) >> np.uint32(16)).astype(np.uint16)
    return out.reshape(a.shape)


def pad_last_dim(a: Optional[np.ndarray], mult: int = 64, fill: int = 0) -> Optional[np.ndarray]:
    """Copy of `a` with its last axis padded to a multiple of `mult` with
    `fill` (raw element value). Second-layer weights of SwiGLU experts are
    passed to the GPU library in this layout: rows of h rounded up to 64."""
    if a is None:
        return None
    n = a.shape[-1]
    ld = -(-n // mult) * mult
    if ld == n:
        return a
    out = np.full(a.shape[:-1] + (ld,), fill, dtype=a.dtype)
    out[..., :n] = a
    return out


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bit patterns to float32."""
    return (bits.astype(np.uint32) << np.uint32(16)).view(np.float32)


@dataclass
class LayerInputs:
    cfg: LayerConfig
    x: Optional[np.ndarray] = None
    w_router: Optional[np.ndarray] = None
    bias: Optional[np.ndarray] = None
    w1: Optional[np.ndarray] = None
    w2: Optional[np.ndarray] = None
    w1s: Optional[np.ndarray] = None
    w2s: Optional[np.ndarray] = None

    @property
    def is_bf16(self) -> bool:
        return self.cfg.dtype == "bf16"

    def f32(self, name: str) -> Optional[np.ndarray]:
        """The tensor as float32 values (exact for bf16 storage)."""
        a = getattr(self, name)
        if a is None:
            return None
        if a.dtype == np.uint16:
            return bf16_bits_to_f32(a)
        return a


def _normal(ss: np.random.SeedSequence, shape, std: float) -> np.ndarray:
    rng = np.random.Generator(np.random.PCG64(ss))
    a = rng.standard_normal(size=shape, dtype=np.float32)
    if std != 1.0:
        a *= np.float32(std)
    return a


def load_zipf_bias(E: int) -> np.ndarray:
    if not os.path.exists(ZIPF_BIAS_FILE):
        raise FileNotFoundError(
            f"{ZIPF_BIAS_FILE} is missing; it is written by tests/golden/make_vitg_skew_bias.py")
    b = np.loadtxt(ZIPF_BIAS_FILE, dtype=np.float64).astype(np.float32)
    if b.shape != (E,):
        raise ValueError(f"stored skew bias has shape {b.shape}, expected ({E},)")
    return b


def make_inputs(cfg: LayerConfig, parts: Optional[Iterable[str]] = None,
                bias_override: Optional[str] = None) -> LayerInputs:
    """Generate the layer's inputs. ``parts`` limits which tensors are drawn
    (the others stay None); ``bias_override`` replaces ``cfg.bias``."""
    want = set(_ORDER if parts is None else parts)
    unknown = want - set(_ORDER)
    if unknown:
        raise ValueError(f"unknown parts {sorted(unknown)}")
    children = np.random.SeedSequence(cfg.seed).spawn(_N_STREAMS)
    bf16 = cfg.dtype == "bf16"
    if cfg.dtype not in ("bf16", "f32"):
        raise ValueError(f"dtype {cfg.dtype!r}")

    def store(a: np.ndarray) -> np.ndarray:
        return f32_to_bf16_bits(a) if bf16 else a

    out = LayerInputs(cfg=cfg)
    std = cfg.weight_std
    if "x" in want:
        out.x = store(_normal(children[0], (cfg.T, cfg.d), 1.0))
    if "w_router" in want:
        out.w_router = store(_normal(children[1], (cfg.E, cfg.d), std))
    if "bias" in want:
        kind = bias_override or cfg.bias
        if kind == "uniform":
            rng = np.random.Generator(np.random.PCG64(children[2]))
            out.bias = rng.uniform(-0.1, 0.1, size=cfg.E).astype(np.float32)
        elif kind == "zero":
            out.bias = np.zeros(cfg.E, dtype=np.float32)
        elif kind == "zipf":
            out.bias = load_zipf_bias(cfg.E)
        else:
            raise ValueError(f"bias kind {kind!r}")
    rows = 2 if cfg.act == "swiglu" else 1
    if cfg.act not in ("gelu", "swiglu"):
        raise ValueError(f"act {cfg.act!r}")
    if "w1" in want:
        out.w1 = store(_normal(children[3], (cfg.E, rows * cfg.h, cfg.d), std))
    if "w2" in want:
        out.w2 = store(_normal(children[4], (cfg.E, cfg.d, cfg.h), std))
    if cfg.h_shared > 0:
        if "w1s" in want:
            out.w1s = store(_normal(children[5], (rows * cfg.h_shared, cfg.d), std))
        if "w2s" in want:
            out.w2s = store(_normal(children[6], (cfg.d, cfg.h_shared), std))
    return out
