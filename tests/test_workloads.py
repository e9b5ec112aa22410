"""The seeded input generator: determinism, shapes, bf16 storage, prefix property."""

import numpy as np
import pytest

from workloads import CONFIGS, bf16_bits_to_f32, f32_to_bf16_bits, get_config, make_inputs


def test_bf16_rounding_ties_to_even():
    v = np.array([1.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, 1.0 + 2 ** -8 + 2 ** -20, -2.5, 0.0],
                 dtype=np.float32)
    got = bf16_bits_to_f32(f32_to_bf16_bits(v))
    assert got.tolist() == [1.0, 1.0, 1.0 + 2 ** -6, 1.0 + 2 ** -7, -2.5, 0.0]


def test_config_table():
    assert [c.name for c in CONFIGS.values()] == [
        "tiny_f32", "vitb_bf16", "vitl_bf16", "vitg_skew_bf16", "single_image_bf16",
        "single_image_swiglu_bf16", "vith_swiglu_bf16"]
    assert get_config("c3").T == 65536 and get_config("c5").T == 1025
    for c in CONFIGS.values():
        assert c.d % 64 == 0 and 1 <= c.K <= c.E
        assert c.act == "swiglu" or (c.h % 64 == 0 and c.h_shared % 64 == 0)
    # SwiGLU: three matrices per expert; the single-image layer holds 1.81 GB of routed weights
    c6 = get_config("c6")
    assert c6.act == "swiglu" and c6.routed_weight_bytes() == 3 * 256 * 768 * 1536 * 2
    assert c6.gemm_flops() == 6.0 * 1025 * 1536 * (8 * 768 + 1536)
    # the paper's H layer: 32 experts of width 854, one shared, 8 active
    c7 = get_config("vith_swiglu_bf16")
    assert (c7.d, c7.E + 1, c7.K + 1, c7.h, c7.h_shared) == (1280, 32, 8, 854, 854)
    # useful GEMM flops of the ViT-G layer: 4*T*d*(K*h + h_s)
    assert get_config("c4").gemm_flops() == 4.0 * 65536 * 1536 * (8 * 768 + 1536)
    assert get_config("c5").routed_weight_bytes() == 2 * 256 * 768 * 1536 * 2


def test_deterministic_and_independent_streams():
    cfg = get_config("c1")
    a = make_inputs(cfg)
    b = make_inputs(cfg)
    for name in ("x", "w_router", "bias", "w1", "w2"):
        assert np.array_equal(getattr(a, name), getattr(b, name))
    only_w2 = make_inputs(cfg, parts=["w2"])
    assert only_w2.x is None and np.array_equal(only_w2.w2, a.w2)
    assert a.x.dtype == np.float32 and a.w1.shape == (8, 256, 256) and a.w2.shape == (8, 256, 256)
    assert a.w1s is None and a.w2s is None
    assert np.all(np.abs(a.bias) <= 0.1)


def test_swiglu_weight_shapes():
    cfg = get_config("vith_swiglu_bf16").with_tokens(8)
    a = make_inputs(cfg, parts=["w1", "w2", "w1s", "w2s"])
    assert a.w1.shape == (31, 2 * 854, 1280) and a.w2.shape == (31, 1280, 854)
    assert a.w1s.shape == (2 * 854, 1280) and a.w2s.shape == (1280, 854)
    assert a.w1.dtype == np.uint16


def test_bf16_config_storage_and_prefix():
    cfg = get_config("c2").with_tokens(300)
    a = make_inputs(cfg, parts=["x", "w_router", "w1s"])
    assert a.x.dtype == np.uint16 and a.x.shape == (300, 768)
    assert a.w1s.shape == (768, 768)
    big = make_inputs(get_config("c2").with_tokens(1000), parts=["x"])
    assert np.array_equal(big.x[:300], a.x)
    xf = a.f32("x")
    assert abs(float(xf.std()) - 1.0) < 0.02
    assert abs(float(a.f32("w_router").std()) - 0.02) < 0.001


@pytest.mark.parametrize("name", ["c3", "c5"])
def test_zero_bias_configs(name):
    a = make_inputs(get_config(name).with_tokens(4), parts=["bias"])
    assert np.all(a.bias == 0)
