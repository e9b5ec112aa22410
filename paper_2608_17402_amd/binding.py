"""Thin ctypes binding of libmoevie.so (include/moe_vie.h).

Argument marshalling only: every function here checks the tensors it is
given, passes their device pointers and the current HIP stream to the C
entry point of the same name, and raises MoeError on a non-OK status. All
computation happens in the HIP kernels behind the C ABI. There is no
fallback: if the library is missing, loading it raises.
"""

from __future__ import annotations

import ctypes
import os
from typing import Optional

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libmoevie.so")

MOE_F32 = 0
MOE_BF16 = 1
MOE_FLAG_EXACT_ROUTER = 1
MOE_FLAG_SWIGLU = 2
STATUS = {0: "MOE_OK", 1: "MOE_ERR_INVALID_ARG", 2: "MOE_ERR_UNSUPPORTED", 3: "MOE_ERR_WORKSPACE",
          4: "MOE_ERR_HIP"}

# Public entry points declared in include/moe_vie.h.
EXPORTS = ("moe_status_string", "moe_last_error", "moe_workspace_size", "moe_route", "moe_permute",
           "moe_grouped_mlp", "moe_combine", "moe_layer_forward", "moe_bias_update", "moe_backward_workspace_size",
           "moe_grouped_mlp_backward", "moe_layer_forward_noalloc")
MOE_BIAS_SIGN = 0
MOE_BIAS_ZSCORE = 1


class MoeDesc(ctypes.Structure):
    _fields_ = [
        ("T", ctypes.c_int32),
        ("d", ctypes.c_int32),
        ("E", ctypes.c_int32),
        ("K", ctypes.c_int32),
        ("h", ctypes.c_int32),
        ("h_shared", ctypes.c_int32),
        ("lam", ctypes.c_float),
        ("dtype", ctypes.c_int32),
        ("flags", ctypes.c_int32),
    ]


class MoeError(RuntimeError):
    def __init__(self, status: int, where: str, detail: str):
        self.status = status
        super().__init__(f"{where}: {STATUS.get(status, status)}: {detail}")


_lib = None


def load(path: Optional[str] = None):
    """Load the HIP library (raises if it has not been built)."""
    global _lib
    if _lib is not None and path is None:
        return _lib
    p = path or LIB_PATH
    if not os.path.exists(p):
        raise RuntimeError(f"{p} is missing: build it with `python -m paper_2608_17402_amd.build` "
                           "(there is no CPU fallback)")
    lib = ctypes.CDLL(p)
    P = ctypes.c_void_p
    S = ctypes.c_size_t
    D = ctypes.POINTER(MoeDesc)
    st = ctypes.c_int
    lib.moe_status_string.argtypes = [st]
    lib.moe_status_string.restype = ctypes.c_char_p
    lib.moe_last_error.argtypes = []
    lib.moe_last_error.restype = ctypes.c_char_p
    lib.moe_workspace_size.argtypes = [D, ctypes.POINTER(ctypes.c_size_t)]
    lib.moe_workspace_size.restype = st
    lib.moe_route.argtypes = [D, P, P, P, P, P, P, S, P]
    lib.moe_route.restype = st
    lib.moe_permute.argtypes = [D, P, P, P, P, P, S, P]
    lib.moe_permute.restype = st
    lib.moe_grouped_mlp.argtypes = [D, P, P, P, P, P, P, P, S, P]
    lib.moe_grouped_mlp.restype = st
    lib.moe_combine.argtypes = [D, P, P, P, P, P]
    lib.moe_combine.restype = st
    lib.moe_layer_forward.argtypes = [D, P, P, P, P, P, P, P, P, P, P, P, S, P, P]
    lib.moe_layer_forward.restype = st
    lib.moe_layer_forward_noalloc.argtypes = [D, P, P, P, P, P, P, P, P, P, P, P]
    lib.moe_layer_forward_noalloc.restype = st
    lib.moe_bias_update.argtypes = [D, P, P, ctypes.c_float, ctypes.c_int32, P]
    lib.moe_bias_update.restype = st
    lib.moe_backward_workspace_size.argtypes = [D, ctypes.POINTER(ctypes.c_size_t)]
    lib.moe_backward_workspace_size.restype = st
    lib.moe_grouped_mlp_backward.argtypes = [D, P, P, P, P, P, P, P, P, P, P, S, P]
    lib.moe_grouped_mlp_backward.restype = st
    if path is None:
        _lib = lib
    return lib


def make_desc(T: int, d: int, E: int, K: int, h: int, h_shared: int = 0, lam: float = 1.0,
              dtype: str = "bf16", flags: int = 0) -> MoeDesc:
    code = {"bf16": MOE_BF16, "f32": MOE_F32}[dtype] if isinstance(dtype, str) else int(dtype)
    return MoeDesc(T, d, E, K, h, h_shared, lam, code, flags)


def torch_dtype(desc: MoeDesc) -> torch.dtype:
    return torch.bfloat16 if desc.dtype == MOE_BF16 else torch.float32


def _check(status: int, where: str):
    if status != 0:
        raise MoeError(status, where, load().moe_last_error().decode())


def _ptr(t: Optional[torch.Tensor], name: str, dtype: Optional[torch.dtype] = None):
    if t is None:
        return None
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.device.type != "cuda":
        raise ValueError(f"{name} must be a device tensor (got {t.device})")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise TypeError(f"{name} has dtype {t.dtype}, expected {dtype}")
    return ctypes.c_void_p(t.data_ptr())


def _stream(stream) -> ctypes.c_void_p:
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def workspace_size(desc: MoeDesc) -> int:
    n = ctypes.c_size_t(0)
    _check(load().moe_workspace_size(ctypes.byref(desc), ctypes.byref(n)), "moe_workspace_size")
    return n.value


def alloc_workspace(desc: MoeDesc, device="cuda") -> torch.Tensor:
    return torch.empty(max(workspace_size(desc), 256), dtype=torch.uint8, device=device)


def moe_route(desc, x, w_router, bias, topk_idx, topk_gate, workspace, stream=None):
    dt = torch_dtype(desc)
    _check(load().moe_route(ctypes.byref(desc), _ptr(x, "x", dt), _ptr(w_router, "w_router", dt),
                            _ptr(bias, "bias", torch.float32), _ptr(topk_idx, "topk_idx", torch.int32),
                            _ptr(topk_gate, "topk_gate", torch.float32), _ptr(workspace, "workspace"),
                            workspace.numel(), _stream(stream)), "moe_route")


def moe_permute(desc, topk_idx, counts, offsets, sorted_slots, workspace, stream=None):
    i32 = torch.int32
    _check(load().moe_permute(ctypes.byref(desc), _ptr(topk_idx, "topk_idx", i32), _ptr(counts, "counts", i32),
                              _ptr(offsets, "offsets", i32), _ptr(sorted_slots, "sorted_slots", i32),
                              _ptr(workspace, "workspace"), workspace.numel(), _stream(stream)), "moe_permute")


def moe_grouped_mlp(desc, x, sorted_slots, offsets, w1, w2, expert_out, workspace, stream=None):
    dt = torch_dtype(desc)
    i32 = torch.int32
    _check(load().moe_grouped_mlp(ctypes.byref(desc), _ptr(x, "x", dt), _ptr(sorted_slots, "sorted_slots", i32),
                                  _ptr(offsets, "offsets", i32), _ptr(w1, "w1", dt), _ptr(w2, "w2", dt),
                                  _ptr(expert_out, "expert_out", dt), _ptr(workspace, "workspace"),
                                  workspace.numel(), _stream(stream)), "moe_grouped_mlp")


def moe_combine(desc, expert_out, topk_gate, shared_out, y, stream=None):
    dt = torch_dtype(desc)
    _check(load().moe_combine(ctypes.byref(desc), _ptr(expert_out, "expert_out", dt),
                              _ptr(topk_gate, "topk_gate", torch.float32), _ptr(shared_out, "shared_out", dt),
                              _ptr(y, "y", dt), _stream(stream)), "moe_combine")


def moe_layer_forward(desc, x, w_router, bias, w1, w2, w1s, w2s, y, topk_idx_out=None, topk_gate_out=None,
                      workspace=None, stream=None, events=None):
    """events: None or three raw hipEvent_t handles (ints) recorded before the
    routed fc1, between fc1 and fc2, and after fc2; the middle one may be
    None (not recorded)."""
    dt = torch_dtype(desc)
    ev = None
    if events is not None:
        if len(events) != 3:
            raise ValueError("events must hold three hipEvent_t handles (the middle one may be None)")
        ev = (ctypes.c_void_p * 3)(*events)
    _check(load().moe_layer_forward(ctypes.byref(desc), _ptr(x, "x", dt), _ptr(w_router, "w_router", dt),
                                    _ptr(bias, "bias", torch.float32), _ptr(w1, "w1", dt), _ptr(w2, "w2", dt),
                                    _ptr(w1s, "w1s", dt), _ptr(w2s, "w2s", dt), _ptr(y, "y", dt),
                                    _ptr(topk_idx_out, "topk_idx_out", torch.int32),
                                    _ptr(topk_gate_out, "topk_gate_out", torch.float32),
                                    _ptr(workspace, "workspace"), workspace.numel(), ev, _stream(stream)),
           "moe_layer_forward")


def moe_layer_forward_noalloc(desc, x, w_router, bias, w1, w2, w1s, w2s, y, topk_idx_out=None,
                              topk_gate_out=None, stream=None):
    """moe_layer_forward on the library's own per-GPU scratch (no workspace)."""
    dt = torch_dtype(desc)
    _check(load().moe_layer_forward_noalloc(
        ctypes.byref(desc), _ptr(x, "x", dt), _ptr(w_router, "w_router", dt), _ptr(bias, "bias", torch.float32),
        _ptr(w1, "w1", dt), _ptr(w2, "w2", dt), _ptr(w1s, "w1s", dt), _ptr(w2s, "w2s", dt), _ptr(y, "y", dt),
        _ptr(topk_idx_out, "topk_idx_out", torch.int32), _ptr(topk_gate_out, "topk_gate_out", torch.float32),
        _stream(stream)), "moe_layer_forward_noalloc")


NOALLOC_SCRATCH_BYTES = 64 << 20


def backward_workspace_size(desc: MoeDesc) -> int:
    n = ctypes.c_size_t(0)
    _check(load().moe_backward_workspace_size(ctypes.byref(desc), ctypes.byref(n)), "moe_backward_workspace_size")
    return n.value


def alloc_backward_workspace(desc: MoeDesc, device="cuda") -> torch.Tensor:
    return torch.empty(max(backward_workspace_size(desc), 256), dtype=torch.uint8, device=device)


def moe_grouped_mlp_backward(desc, x, sorted_slots, offsets, w1, w2, grad_expert_out, dx, dw1, dw2, workspace,
                             stream=None):
    """dx [T, d], dw1 [E, h, d] and dw2 [E, d, h] (fp32) of the routed experts
    from the gradient of their slot-order outputs."""
    dt = torch_dtype(desc)
    _check(load().moe_grouped_mlp_backward(
        ctypes.byref(desc), _ptr(x, "x", dt), _ptr(sorted_slots, "sorted_slots", torch.int32),
        _ptr(offsets, "offsets", torch.int32), _ptr(w1, "w1", dt), _ptr(w2, "w2", dt),
        _ptr(grad_expert_out, "grad_expert_out", dt), _ptr(dx, "dx", dt), _ptr(dw1, "dw1", torch.float32),
        _ptr(dw2, "dw2", torch.float32), _ptr(workspace, "workspace"), workspace.numel() * workspace.element_size(),
        _stream(stream)), "moe_grouped_mlp_backward")


def moe_bias_update(desc, counts, bias, alpha: float, rule: int, stream=None):
    """Loss-free balancing update of `bias` in place from per-expert `counts`."""
    _check(load().moe_bias_update(ctypes.byref(desc), _ptr(counts, "counts", torch.int32),
                                  _ptr(bias, "bias", torch.float32), float(alpha), int(rule), _stream(stream)),
           "moe_bias_update")


class HipEvents:
    """Raw HIP events through the HIP runtime (timing only)."""

    def __init__(self, n: int):
        self._hip = ctypes.CDLL("libamdhip64.so")
        self._hip.hipEventCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
        self._hip.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p, ctypes.c_void_p]
        self._hip.hipEventDestroy.argtypes = [ctypes.c_void_p]
        self.handles = []
        for _ in range(n):
            h = ctypes.c_void_p()
            if self._hip.hipEventCreate(ctypes.byref(h)) != 0:
                raise RuntimeError("hipEventCreate failed")
            self.handles.append(h.value)

    def elapsed_ms(self, a: int, b: int) -> float:
        ms = ctypes.c_float()
        if self._hip.hipEventElapsedTime(ctypes.byref(ms), self.handles[a], self.handles[b]) != 0:
            raise RuntimeError("hipEventElapsedTime failed")
        return ms.value

    def close(self):
        for h in self.handles:
            self._hip.hipEventDestroy(h)
        self.handles = []
