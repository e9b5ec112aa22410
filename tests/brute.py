"""Brute-force float64 reference for tiny layers, written independently of the
oracle: routing in float64 from numpy matmuls, every expert evaluated densely
for every token, then selected and mixed (MoE output, Eq. (3)/(6); sigmoid
gating Eqs. (4)-(5); selection bias Eq. (7)). Used only to validate the oracle.
"""

from __future__ import annotations

import numpy as np
from scipy.special import erf


def gelu64(v: np.ndarray) -> np.ndarray:
    return 0.5 * v * (1.0 + erf(v / np.sqrt(2.0)))


def bf16_round64(v: np.ndarray) -> np.ndarray:
    """Nearest bf16 of float64 values, ties to even (normal range)."""
    v = np.asarray(v, dtype=np.float64)
    out = np.zeros_like(v)
    nz = v != 0
    m, e = np.frexp(v[nz])
    out[nz] = np.ldexp(np.rint(m * 256.0), e - 8)
    return out


def route64(x, wr, bias, K):
    """(idx [T, K], gates [T, K], sorted keys [T, E]) with float64 arithmetic;
    ties in the key go to the lower expert index."""
    x = np.asarray(x, np.float64)
    wr = np.asarray(wr, np.float64)
    s = x @ wr.T
    sig = 1.0 / (1.0 + np.exp(-s))
    key = sig + (0.0 if bias is None else np.asarray(bias, np.float64)[None, :])
    T, E = key.shape
    experts = np.broadcast_to(np.arange(E), (T, E))
    order = np.lexsort((experts, -key), axis=-1)
    idx = order[:, :K]
    chosen = np.take_along_axis(sig, idx, axis=1)
    gates = chosen / chosen.sum(axis=1, keepdims=True)
    return idx, gates, np.take_along_axis(key, order, axis=1)


def expert64(xr, w1, w2, act_bf16):
    a = gelu64(np.asarray(xr, np.float64) @ np.asarray(w1, np.float64).T)
    if act_bf16:
        a = bf16_round64(a)
    return a @ np.asarray(w2, np.float64).T


def layer64(x, wr, bias, w1, w2, w1s, w2s, K, lam, act_bf16):
    idx, gates, keys = route64(x, wr, bias, K)
    T = x.shape[0]
    E = w1.shape[0]
    dense = np.stack([expert64(x, w1[e], w2[e], act_bf16) for e in range(E)])  # [E, T, d]
    y = np.zeros((T, x.shape[1]))
    for j in range(K):
        y += gates[:, j:j + 1] * dense[idx[:, j], np.arange(T)]
    if w1s is not None:
        y += lam * expert64(x, w1s, w2s, act_bf16)
    return idx, gates, keys, y
