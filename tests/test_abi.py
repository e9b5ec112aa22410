"""The C ABI library on the CPU: it loads, exports every entry point that
include/moe_vie.h declares, and rejects bad arguments on the host (before any
HIP call, so these run without a GPU)."""

import ctypes
import os
import re

import pytest

from paper_2608_17402_amd import binding

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "moe_vie.h")


def declared_functions():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^\s*(?:const\s+char\s*\*|moe_status_t|size_t)\s*(moe_\w+)\s*\(", text, re.M)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(binding.LIB_PATH):
        pytest.fail("libmoevie.so is not built (run __graft_entry__.build())")
    return binding.load()


def test_header_declares_the_boundary():
    names = declared_functions()
    for n in ("moe_route", "moe_permute", "moe_grouped_mlp", "moe_combine", "moe_layer_forward",
              "moe_bias_update", "moe_workspace_size", "moe_status_string", "moe_last_error"):
        assert n in names
    assert set(names) == set(binding.EXPORTS)


def test_library_exports_every_declared_symbol(lib):
    for name in declared_functions():
        assert hasattr(lib, name), f"{name} is declared but not exported"


def test_status_strings(lib):
    assert lib.moe_status_string(0) == b"MOE_OK"
    assert lib.moe_status_string(3) == b"MOE_ERR_WORKSPACE"
    assert lib.moe_status_string(99) == b"MOE_ERR_UNKNOWN"


def _ws(desc):
    n = ctypes.c_size_t(0)
    st = binding.load().moe_workspace_size(ctypes.byref(desc), ctypes.byref(n))
    return st, n.value


def test_workspace_size_and_desc_validation(lib):
    st, n = _ws(binding.make_desc(196, 256, 8, 2, 256, 0, 1.0, "f32"))
    assert st == 0 and n > 196 * 2 * 256 * 4 * 2
    st4, n4 = _ws(binding.make_desc(65536, 1536, 256, 8, 768, 1536, 1.0, "bf16"))
    assert st4 == 0
    # routed activation + expert outputs + shared activation (bf16) at least
    assert n4 >= 65536 * 8 * (768 + 1536) * 2 + 65536 * 1536 * 2
    st1, n1 = _ws(binding.make_desc(196, 256, 8, 2, 256, 128, 1.0, "f32"))
    # the fp32 layer also keeps the shared expert's fp32 output for the combine
    assert st1 == 0 and n1 >= 196 * 2 * (256 + 256) * 4 + 196 * 128 * 4 + 196 * 256 * 4
    bad = {
        "K=0": (binding.make_desc(10, 64, 8, 0, 64), 1),
        "K>16": (binding.make_desc(10, 64, 32, 17, 64), 1),
        "E<K": (binding.make_desc(10, 64, 2, 4, 64), 1),
        "E>1024": (binding.make_desc(10, 64, 1025, 4, 64), 1),
        "T=0": (binding.make_desc(0, 64, 8, 2, 64), 1),
        "d%64": (binding.make_desc(10, 96, 8, 2, 64), 2),
        "h%64": (binding.make_desc(10, 64, 8, 2, 100), 2),
        "hs%64": (binding.make_desc(10, 64, 8, 2, 64, 65), 2),
        "d>8192": (binding.make_desc(10, 8256, 8, 2, 64), 1),
        "dtype": (binding.make_desc(10, 64, 8, 2, 64, 0, 1.0, 7), 2),
        "flags": (binding.make_desc(10, 64, 8, 2, 64, 0, 1.0, "bf16", flags=4), 1),
        "swiglu f32": (binding.make_desc(10, 64, 8, 2, 64, 0, 1.0, "f32", flags=binding.MOE_FLAG_SWIGLU), 2),
        "swiglu h=0": (binding.make_desc(10, 64, 8, 2, 0, 0, 1.0, "bf16", flags=binding.MOE_FLAG_SWIGLU), 1),
        "swiglu h>8192": (binding.make_desc(10, 64, 8, 2, 8193, 0, 1.0, "bf16",
                                            flags=binding.MOE_FLAG_SWIGLU), 1),
        "4GiB": (binding.make_desc(2 ** 21, 1024, 8, 2, 64, 0, 1.0, "bf16"), 2),
        "lambda": (binding.make_desc(10, 64, 8, 2, 64, 0, float("nan")), 1),
        "T*K": (binding.make_desc(2 ** 28, 64, 16, 8, 64), 1),
    }
    for name, (desc, want) in bad.items():
        st, _ = _ws(desc)
        assert st == want, name
        assert lib.moe_last_error() != b""


def test_swiglu_desc_and_workspace(lib):
    """SwiGLU experts take any hidden width; the activations are stored with
    rows padded to a multiple of 64 columns."""
    sw = binding.MOE_FLAG_SWIGLU
    st, n = _ws(binding.make_desc(65536, 1280, 31, 7, 854, 854, 1.0, "bf16", flags=sw))
    assert st == 0
    # routed activations [T*K, 896] + expert outputs [T*K, d] + shared activations [T, 896]
    assert n >= 65536 * 7 * (896 + 1280) * 2 + 65536 * 896 * 2
    st_g, n_g = _ws(binding.make_desc(65536, 1280, 31, 7, 896, 896, 1.0, "bf16"))
    assert st_g == 0 and n == n_g  # padded SwiGLU activations take what GELU ones of width 896 take
    for h in (1, 40, 100, 8192):
        assert _ws(binding.make_desc(100, 64, 8, 2, h, h, 1.0, "bf16", flags=sw))[0] == 0, h
    assert _ws(binding.make_desc(100, 64, 8, 2, 100, 0, 1.0, "bf16", flags=sw | binding.MOE_FLAG_EXACT_ROUTER))[0] == 0


def test_entry_points_reject_bad_pointers_before_any_launch(lib):
    desc = binding.make_desc(100, 64, 8, 2, 64, 64, 1.0, "bf16")
    _, need = _ws(desc)
    P = ctypes.c_void_p
    fake = P(1 << 20)  # 16-byte aligned, never dereferenced: validation fails first
    mis = P((1 << 20) + 4)
    S = ctypes.c_size_t
    d = ctypes.byref(desc)
    assert lib.moe_route(d, None, fake, None, fake, fake, fake, S(need), None) == 1
    assert b"x is NULL" in lib.moe_last_error()
    assert lib.moe_route(d, mis, fake, None, fake, fake, fake, S(need), None) == 1
    assert b"aligned" in lib.moe_last_error()
    assert lib.moe_route(d, fake, fake, None, fake, fake, fake, S(need - 1), None) == 3
    assert lib.moe_permute(d, fake, fake, fake, fake, None, S(0), None) == 3
    assert lib.moe_grouped_mlp(d, fake, fake, fake, fake, None, fake, fake, S(need), None) == 1
    assert lib.moe_combine(d, fake, None, None, fake, None) == 1
    assert lib.moe_layer_forward(d, fake, fake, None, fake, fake, None, fake, fake, None, None, fake,
                                 S(need), None, None) == 1  # shared weights required when h_shared > 0
    bad = binding.make_desc(100, 64, 8, 0, 64)
    assert lib.moe_layer_forward(ctypes.byref(bad), fake, fake, None, fake, fake, None, None, fake, None,
                                 None, fake, S(need), None, None) == 1
    half = (ctypes.c_void_p * 3)(1 << 20, 1 << 21, None)
    desc0 = binding.make_desc(100, 64, 8, 2, 64, 0, 1.0, "bf16")
    assert lib.moe_layer_forward(ctypes.byref(desc0), fake, fake, None, fake, fake, None, None, fake, None,
                                 None, fake, S(need), half, None) == 1
    assert b"events" in lib.moe_last_error()
    first_null = (ctypes.c_void_p * 3)(None, 1 << 21, 1 << 22)
    assert lib.moe_layer_forward(ctypes.byref(desc0), fake, fake, None, fake, fake, None, None, fake, None,
                                 None, fake, S(need), first_null, None) == 1
    assert b"events" in lib.moe_last_error()


def test_bias_update_rejects_bad_arguments(lib):
    desc = binding.make_desc(100, 64, 8, 2, 64)
    P = ctypes.c_void_p
    fake = P(1 << 20)
    d = ctypes.byref(desc)
    assert lib.moe_bias_update(d, None, fake, ctypes.c_float(0.1), 1, None) == 1
    assert b"counts" in lib.moe_last_error()
    assert lib.moe_bias_update(d, fake, None, ctypes.c_float(0.1), 1, None) == 1
    assert lib.moe_bias_update(d, fake, fake, ctypes.c_float(float("nan")), 1, None) == 1
    assert b"alpha" in lib.moe_last_error()
    assert lib.moe_bias_update(d, fake, fake, ctypes.c_float(-1.0), 0, None) == 1
    assert lib.moe_bias_update(d, fake, fake, ctypes.c_float(float("inf")), 0, None) == 1
    assert lib.moe_bias_update(d, fake, fake, ctypes.c_float(0.1), 2, None) == 1
    assert b"rule" in lib.moe_last_error()
    bad = binding.make_desc(100, 64, 8, 0, 64)
    assert lib.moe_bias_update(ctypes.byref(bad), fake, fake, ctypes.c_float(0.1), 0, None) == 1


def test_backward_validation(lib):
    n = ctypes.c_size_t(0)
    ok = binding.make_desc(1000, 256, 8, 2, 192, 0, 1.0, "bf16")
    assert lib.moe_backward_workspace_size(ctypes.byref(ok), ctypes.byref(n)) == 0
    # at least the transposed operands: (2 d + 2 h) x (T*K + 64 E) bf16
    assert n.value >= (2 * 256 + 2 * 192) * (2000 + 64 * 8) * 2
    f32 = binding.make_desc(1000, 256, 8, 2, 192, 0, 1.0, "f32")
    assert lib.moe_backward_workspace_size(ctypes.byref(f32), ctypes.byref(n)) == 2
    assert lib.moe_last_error() != b""
    sw = binding.make_desc(1000, 256, 8, 2, 300, 0, 1.0, "bf16", flags=binding.MOE_FLAG_SWIGLU)
    assert lib.moe_backward_workspace_size(ctypes.byref(sw), ctypes.byref(n)) == 0
    # SwiGLU: the stacked pre-activation gradients are 2 * 320 wide
    assert n.value >= (2 * 256 + 320 + 2 * 320) * (2000 + 128 * 8) * 2
    P, S = ctypes.c_void_p, ctypes.c_size_t
    fake = P(1 << 20)
    d = ctypes.byref(ok)
    assert lib.moe_grouped_mlp_backward(d, fake, fake, fake, fake, fake, None, fake, fake, fake, fake, S(1 << 40),
                                        None) == 1
    assert b"grad_expert_out is NULL" in lib.moe_last_error()
    assert lib.moe_grouped_mlp_backward(d, fake, fake, fake, fake, fake, fake, fake, fake, fake, fake, S(256),
                                        None) == 3
    assert lib.moe_grouped_mlp_backward(d, fake, fake, fake, fake, fake, fake, fake, fake, P((1 << 20) + 8),
                                        fake, S(1 << 40), None) == 1


def test_noalloc_rejects_before_any_hip_call(lib):
    """The allocation-free layer forward validates the descriptor and its
    scratch need on the host first: a layer whose workspace exceeds the
    library's scratch, or a bad descriptor, is refused without a HIP call."""
    P = ctypes.c_void_p
    fake = P(1 << 20)
    big = binding.make_desc(65536, 1536, 256, 8, 768, 1536, 1.0, "bf16")
    _, need = _ws(big)
    assert need > binding.NOALLOC_SCRATCH_BYTES
    assert lib.moe_layer_forward_noalloc(ctypes.byref(big), fake, fake, None, fake, fake, fake, fake, fake, None,
                                         None, None) == 3
    assert b"scratch" in lib.moe_last_error()
    bad = binding.make_desc(100, 64, 8, 0, 64)
    assert lib.moe_layer_forward_noalloc(ctypes.byref(bad), fake, fake, None, fake, fake, None, None, fake, None,
                                         None, None) == 1
    # The single-image ViT-G layer fits.
    one = binding.make_desc(1025, 1536, 256, 8, 768, 1536, 1.0, "bf16")
    assert _ws(one)[1] <= binding.NOALLOC_SCRATCH_BYTES
    text = open(HEADER).read()
    assert "#define MOE_NOALLOC_SCRATCH_BYTES (64u << 20)" in text and binding.NOALLOC_SCRATCH_BYTES == 64 << 20
