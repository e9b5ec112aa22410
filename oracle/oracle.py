"""ctypes binding of the plain C oracle (``moe_oracle.c``).

TEST INFRASTRUCTURE ONLY: the tests, the smoke check and the benchmark's
CPU-baseline leg use it to produce expected values. All arrays are numpy;
float inputs are float32 values (a bf16 tensor is passed as its exact float32
widening), integer arrays are int32, the MLP and combine results are float64.
"""

from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "moe_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
# A test may point the binding at a deliberately broken build of the oracle.
_LIB_OVERRIDE = os.environ.get("MOE_ORACLE_LIB")

CFLAGS = ["-O2", "-mfma", "-ffp-contract=off", "-fno-fast-math", "-fopenmp", "-fPIC", "-shared",
          "-std=c11", "-Wall", "-Wextra"]


def build_oracle(force: bool = True) -> str:
    """Compile liboracle.so with gcc (plain IEEE arithmetic: no fast-math, no
    contraction of multiply-add pairs). Returns the library path."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + f".tmp{os.getpid()}"
        cmd = ["gcc", *CFLAGS, _SRC, "-o", tmp, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB)
    return _LIB


_lib = None


def _load():
    global _lib
    if _lib is None:
        if _LIB_OVERRIDE:
            lib = ctypes.CDLL(_LIB_OVERRIDE)
        else:
            if not os.path.exists(_LIB):
                build_oracle(force=False)
            lib = ctypes.CDLL(_LIB)
        P = ctypes.c_void_p
        I = ctypes.c_int
        F = ctypes.c_float
        D = ctypes.c_double
        sigs = {
            "oracle_version": ([], I),
            "oracle_num_threads": ([], I),
            "oracle_sigmoid": ([F], F),
            "oracle_gelu": ([D], D),
            "oracle_round_bf16": ([D], D),
            "oracle_logits": ([I, I, I, P, P, P], None),
            "oracle_scores": ([I, I, I, P, P, P], None),
            "oracle_route": ([I, I, I, I, P, P, P, P, P], None),
            "oracle_topk_from_scores": ([I, I, I, P, P, P, P], None),
            "oracle_permute": ([I, I, I, P, P, P, P], None),
            "oracle_expert_rows": ([I, I, I, P, P, P, I, P], None),
            "oracle_combine": ([I, I, I, P, P, P, D, P], None),
            "oracle_layer": ([I, P, I, I, I, I, I, I, F, I, P, P, P, P, P, P, P, P, P, P], None),
            "oracle_bias_update": ([I, P, P, F, I], None),
            "oracle_silu": ([D], D),
            "oracle_expert_rows_swiglu": ([I, I, I, P, P, P, I, P], None),
            "oracle_layer_swiglu": ([I, P, I, I, I, I, I, I, F, I, P, P, P, P, P, P, P, P, P, P], None),
            "oracle_gelu_grad": ([D], D),
            "oracle_silu_grad": ([D], D),
            "oracle_expert_backward": ([I, I, I, P, P, P, P, I, P, P, P], None),
            "oracle_expert_backward_swiglu": ([I, I, I, P, P, P, P, I, P, P, P], None),
        }
        for name, (args, res) in sigs.items():
            fn = getattr(lib, name)
            fn.argtypes = args
            fn.restype = res
        _lib = lib
    return _lib


def _ptr(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _f32(a):
    return None if a is None else np.ascontiguousarray(a, dtype=np.float32)


def num_threads() -> int:
    return _load().oracle_num_threads()


def sigmoid(s) -> np.ndarray:
    """Recipe-S sigmoid, elementwise, float32 in and out."""
    lib = _load()
    s = np.asarray(s, dtype=np.float32)
    out = np.array([lib.oracle_sigmoid(float(v)) for v in s.reshape(-1)], dtype=np.float32)
    return out.reshape(s.shape)


def gelu(v) -> np.ndarray:
    lib = _load()
    v = np.asarray(v, dtype=np.float64)
    return np.array([lib.oracle_gelu(float(a)) for a in v.reshape(-1)]).reshape(v.shape)


def round_bf16(v) -> np.ndarray:
    lib = _load()
    v = np.asarray(v, dtype=np.float64)
    return np.array([lib.oracle_round_bf16(float(a)) for a in v.reshape(-1)]).reshape(v.shape)


def logits(x, wr) -> np.ndarray:
    """Recipe-R router logits [T, E] (float32)."""
    x, wr = _f32(x), _f32(wr)
    T, d = x.shape
    E = wr.shape[0]
    out = np.empty((T, E), dtype=np.float32)
    _load().oracle_logits(T, d, E, _ptr(x), _ptr(wr), _ptr(out))
    return out


def scores(x, wr) -> np.ndarray:
    """Sigmoid scores [T, E] (recipes R and S, float32)."""
    x, wr = _f32(x), _f32(wr)
    T, d = x.shape
    E = wr.shape[0]
    out = np.empty((T, E), dtype=np.float32)
    _load().oracle_scores(T, d, E, _ptr(x), _ptr(wr), _ptr(out))
    return out


def route(x, wr, bias, K: int):
    """(topk_idx [T, K] int32, topk_gate [T, K] float32)."""
    x, wr, bias = _f32(x), _f32(wr), _f32(bias)
    T, d = x.shape
    E = wr.shape[0]
    idx = np.empty((T, K), dtype=np.int32)
    gate = np.empty((T, K), dtype=np.float32)
    _load().oracle_route(T, d, E, K, _ptr(x), _ptr(wr), _ptr(bias), _ptr(idx), _ptr(gate))
    return idx, gate


def topk_from_scores(sc, bias, K: int):
    sc, bias = _f32(sc), _f32(bias)
    T, E = sc.shape
    idx = np.empty((T, K), dtype=np.int32)
    gate = np.empty((T, K), dtype=np.float32)
    _load().oracle_topk_from_scores(T, E, K, _ptr(sc), _ptr(bias), _ptr(idx), _ptr(gate))
    return idx, gate


def permute(topk_idx, E: int):
    """(counts [E], offsets [E+1], sorted_slots [T*K]) as int32."""
    idx = np.ascontiguousarray(topk_idx, dtype=np.int32)
    T, K = idx.shape
    counts = np.empty(E, dtype=np.int32)
    offsets = np.empty(E + 1, dtype=np.int32)
    slots = np.empty(T * K, dtype=np.int32)
    _load().oracle_permute(T, E, K, _ptr(idx), _ptr(counts), _ptr(offsets), _ptr(slots))
    return counts, offsets, slots


def silu(v) -> np.ndarray:
    """SiLU v / (1 + exp(-v)) in double precision (elementwise)."""
    f = _load().oracle_silu
    return np.vectorize(lambda z: f(float(z)), otypes=[np.float64])(np.asarray(v, dtype=np.float64))


def expert_rows(rows, w1, w2, act_bf16: bool, act: str = "gelu") -> np.ndarray:
    """W2 act(W1 r) for each row r of rows [n, d]; w2 [d, h]. float64 [n, d].
    act "gelu": w1 [h, d]; act "swiglu": w1 [2h, d] holds the gate rows then the
    up rows and act(.) = SiLU(gate) * up."""
    rows, w1, w2 = _f32(rows), _f32(w1), _f32(w2)
    n, d = rows.shape
    h = w2.shape[1]
    assert w1.shape == ((2 * h if act == "swiglu" else h), d) and w2.shape == (d, h)
    out = np.empty((n, d), dtype=np.float64)
    fn = _load().oracle_expert_rows_swiglu if act == "swiglu" else _load().oracle_expert_rows
    assert act in ("gelu", "swiglu")
    fn(n, d, h, _ptr(rows), _ptr(w1), _ptr(w2), int(bool(act_bf16)), _ptr(out))
    return out


def gelu_grad(v) -> np.ndarray:
    """d/dv GELU(v) in double precision (elementwise)."""
    f = _load().oracle_gelu_grad
    return np.vectorize(lambda z: f(float(z)), otypes=[np.float64])(np.asarray(v, dtype=np.float64))


def silu_grad(v) -> np.ndarray:
    """d/dv SiLU(v) in double precision (elementwise)."""
    f = _load().oracle_silu_grad
    return np.vectorize(lambda z: f(float(z)), otypes=[np.float64])(np.asarray(v, dtype=np.float64))


def expert_backward(rows, w1, w2, grad_out, act_bf16: bool, act: str = "gelu"):
    """Backward of one expert MLP over the rows [n, d] given grad_out [n, d]
    (the gradient of W2 act(W1 r) for each row). Returns float64 (dx [n, d],
    dw1 [h, d] or [2h, d] for SwiGLU, dw2 [d, h]); the weight gradients are
    sums over the rows."""
    assert act in ("gelu", "swiglu")
    rows, w1, w2, grad_out = _f32(rows), _f32(w1), _f32(w2), _f32(grad_out)
    n, d = rows.shape
    h = w2.shape[1]
    hr = 2 * h if act == "swiglu" else h
    assert w1.shape == (hr, d) and w2.shape == (d, h) and grad_out.shape == (n, d)
    dx = np.empty((n, d), dtype=np.float64)
    dw1 = np.empty((hr, d), dtype=np.float64)
    dw2 = np.empty((d, h), dtype=np.float64)
    fn = _load().oracle_expert_backward_swiglu if act == "swiglu" else _load().oracle_expert_backward
    fn(n, d, h, _ptr(rows), _ptr(w1), _ptr(w2), _ptr(grad_out), int(bool(act_bf16)), _ptr(dx), _ptr(dw1),
       _ptr(dw2))
    return dx, dw1, dw2


def grouped_backward(x, topk_idx, w1, w2, grad_expert_out, act_bf16: bool, act: str = "gelu"):
    """Backward of the routed experts of a layer: x [T, d], topk_idx [T, K],
    w1 [E, h or 2h, d], w2 [E, d, h], grad_expert_out [T*K, d] in slot order.
    Returns float64 (dx [T, d] summed over each token's K slots in slot
    order, dw1 like w1, dw2 like w2)."""
    x = _f32(x)
    g = _f32(grad_expert_out)
    T, K = np.asarray(topk_idx).shape
    E = w1.shape[0]
    _, offsets, slots = permute(topk_idx, E)
    dxs = np.zeros((T * K, x.shape[1]), dtype=np.float64)
    dw1 = np.zeros(w1.shape, dtype=np.float64)
    dw2 = np.zeros(w2.shape, dtype=np.float64)
    for e in range(E):
        seg = slots[offsets[e]:offsets[e + 1]]
        if seg.size == 0:
            continue
        dxr, dw1[e], dw2[e] = expert_backward(x[seg // K], w1[e], w2[e], g[seg], act_bf16, act)
        dxs[seg] = dxr
    dx = dxs.reshape(T, K, -1)[:, 0, :].copy()
    for j in range(1, K):
        dx += dxs.reshape(T, K, -1)[:, j, :]
    return dx, dw1, dw2


def combine(expert_out, gate, shared, lam: float) -> np.ndarray:
    """y [T, d] float64 from expert_out [T*K, d], gate [T, K] and shared [T, d] (or None)."""
    gate = _f32(gate)
    T, K = gate.shape
    eo = np.ascontiguousarray(expert_out, dtype=np.float64)
    d = eo.shape[1]
    assert eo.shape == (T * K, d)
    sh = None if shared is None else np.ascontiguousarray(shared, dtype=np.float64)
    y = np.empty((T, d), dtype=np.float64)
    _load().oracle_combine(T, d, K, _ptr(eo), _ptr(gate), _ptr(sh), float(lam), _ptr(y))
    return y


def layer(x, wr, bias, w1, w2, w1s, w2s, K: int, lam: float, act_bf16: bool, tokens=None, act: str = "gelu"):
    """The whole layer for the listed tokens (all tokens when None).
    act "swiglu": w1 [E, 2h, d] and w1s [2h_s, d] hold the gate rows then the up
    rows of each expert. Returns (topk_idx [n, K], topk_gate [n, K], y [n, d] float64)."""
    assert act in ("gelu", "swiglu")
    x, wr, bias, w1, w2 = _f32(x), _f32(wr), _f32(bias), _f32(w1), _f32(w2)
    w1s, w2s = _f32(w1s), _f32(w2s)
    T, d = x.shape
    E, h = w2.shape[0], w2.shape[2]
    hs = 0 if w2s is None else w2s.shape[1]
    tok = None if tokens is None else np.ascontiguousarray(tokens, dtype=np.int32)
    n = T if tok is None else tok.size
    idx = np.empty((n, K), dtype=np.int32)
    gate = np.empty((n, K), dtype=np.float32)
    y = np.empty((n, d), dtype=np.float64)
    fn = _load().oracle_layer_swiglu if act == "swiglu" else _load().oracle_layer
    fn(n, _ptr(tok), T, d, E, K, h, hs, float(lam), int(bool(act_bf16)),
       _ptr(x), _ptr(wr), _ptr(bias), _ptr(w1), _ptr(w2), _ptr(w1s), _ptr(w2s),
       _ptr(idx), _ptr(gate), _ptr(y))
    return idx, gate, y


BIAS_SIGN = 0
BIAS_ZSCORE = 1


def bias_update(counts, bias, alpha: float, rule: int) -> np.ndarray:
    """Loss-free balancing update of the selection bias (Sec. 3.2 "Load
    Balancing", Eq. (8) for rule BIAS_SIGN, Eq. (9) for BIAS_ZSCORE) from the
    per-expert token counts of one iteration. Returns the new fp32 bias."""
    c = np.ascontiguousarray(counts, dtype=np.int32)
    b = np.array(bias, dtype=np.float32, copy=True)
    assert c.shape == b.shape and c.ndim == 1
    _load().oracle_bias_update(int(c.size), _ptr(c), _ptr(b), float(alpha), int(rule))
    return b
