"""Parity of the expert-MLP backward (moe_grouped_mlp_backward) with the CPU
oracle's chain rule.

dx (bf16) and the fp32 weight gradients are compared with max-abs <=
2e-2 * max(1, max |ref|) and rel-L2 <= 5e-3: the forward's bound, scaled to
the gradient's magnitude (dx is rounded to bf16 once, half an ulp is 2^-9 of
its value). Both sides round the activation and the pre-activation gradient to
bf16 at the same points, so what remains is fp32 accumulation order and
isolated one-ulp rounding flips.
"""

import numpy as np
import pytest
import torch

import oracle
from gpu_util import dev, host
from paper_2608_17402_amd import binding
from workloads import bf16_bits_to_f32, f32_to_bf16_bits, get_config, make_inputs

pytestmark = pytest.mark.gpu


def check_grad(got, ref, what):
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    assert got.shape == ref.shape and np.all(np.isfinite(got)), what
    err = got - ref
    scale = max(1.0, float(np.max(np.abs(ref))) if ref.size else 1.0)
    max_abs = float(np.max(np.abs(err))) if err.size else 0.0
    den = float(np.linalg.norm(ref))
    rel = float(np.linalg.norm(err)) / den if den > 0 else float(np.linalg.norm(err))
    assert max_abs <= 2e-2 * scale and rel <= 5e-3, f"{what}: max_abs={max_abs:.3e} (scale {scale:.2f}), rel={rel:.3e}"


def _bf16(rng, shape, std):
    return f32_to_bf16_bits((rng.standard_normal(shape) * std).astype(np.float32))


def run_backward(T, d, E, K, h, idx, x, w1, w2, g, swiglu=False):
    """Permute idx on the GPU, then the backward; returns host arrays. SwiGLU:
    w1 [E, 2h, d], w2 [E, d, ldh] (padded), dw1 [E, 2h, d], dw2 [E, d, ldh]."""
    flags = binding.MOE_FLAG_SWIGLU if swiglu else 0
    desc = binding.make_desc(T, d, E, K, h, 0, 1.0, "bf16", flags=flags)
    ws = binding.alloc_workspace(desc)
    counts = torch.empty(E, dtype=torch.int32, device="cuda")
    offsets = torch.empty(E + 1, dtype=torch.int32, device="cuda")
    slots = torch.empty(T * K, dtype=torch.int32, device="cuda")
    binding.moe_permute(desc, dev(idx), counts, offsets, slots, ws)
    bws = binding.alloc_backward_workspace(desc)
    dx = torch.empty(T, d, dtype=torch.bfloat16, device="cuda")
    dw1 = torch.empty(E, w1.shape[1], d, dtype=torch.float32, device="cuda")
    dw2 = torch.empty(E, d, w2.shape[2], dtype=torch.float32, device="cuda")
    xd, w1d, w2d, gd = dev(x), dev(w1), dev(w2), dev(g)
    binding.moe_grouped_mlp_backward(desc, xd, slots, offsets, w1d, w2d, gd, dx, dw1, dw2, bws)
    torch.cuda.synchronize()
    out = (host(dx), host(dw1), host(dw2))
    # A second call on the same buffers is bit-identical (no atomics).
    binding.moe_grouped_mlp_backward(desc, xd, slots, offsets, w1d, w2d, gd, dx, dw1, dw2, bws)
    torch.cuda.synchronize()
    for a, b in zip(out, (host(dx), host(dw1), host(dw2))):
        assert np.array_equal(a.view(np.uint32), b.view(np.uint32)), "repeat differs"
    return out


def _idx(rng, T, E, K, probs=None):
    return np.stack([rng.choice(E, K, replace=False, p=probs) for _ in range(T)]).astype(np.int32)


CASES = {
    # ~75 rows per expert: 64-row tiles; the ViT-B layer's widths
    "vitb_T600": dict(T=600, d=768, E=64, K=8, h=384),
    # ViT-G widths, 64-row tiles, ragged windows
    "vitg_T400": dict(T=400, d=1536, E=256, K=8, h=768),
    # ~750 rows per expert: 256-row tiles; dW2 on 256-row tiles (d = 256),
    # dW1 on 64-row tiles (h = 192), 64-column tiles where N = 192
    "tiles256": dict(T=3000, d=256, E=8, K=2, h=192),
    # K = 1, a single expert
    "one_expert": dict(T=333, d=128, E=1, K=1, h=128),
    # the largest model width, d = 8192 (128 K slabs in dA and its windows)
    "max_width": dict(T=64, d=8192, E=2, K=1, h=2048),
}


@pytest.mark.parametrize("name", sorted(CASES))
def test_backward_matches_oracle(name):
    c = CASES[name]
    T, d, E, K, h = c["T"], c["d"], c["E"], c["K"], c["h"]
    rng = np.random.default_rng(len(name))
    x = _bf16(rng, (T, d), 1.0)
    w1 = _bf16(rng, (E, h, d), 0.05)
    w2 = _bf16(rng, (E, d, h), 0.05)
    g = _bf16(rng, (T * K, d), 0.5)
    idx = _idx(rng, T, E, K)
    dx, dw1, dw2 = run_backward(T, d, E, K, h, idx, x, w1, w2, g)
    rdx, rdw1, rdw2 = oracle.grouped_backward(bf16_bits_to_f32(x), idx, bf16_bits_to_f32(w1), bf16_bits_to_f32(w2),
                                              bf16_bits_to_f32(g), True)
    check_grad(dx, rdx, f"{name} dx")
    check_grad(dw1, rdw1, f"{name} dw1")
    check_grad(dw2, rdw2, f"{name} dw2")


def test_backward_empty_and_dominant_experts():
    # Experts 0..2 take most slots, 10..15 none (their gradients are zero).
    T, d, E, K, h = 900, 128, 16, 2, 64
    rng = np.random.default_rng(5)
    probs = np.r_[np.full(3, 0.25), np.full(7, 0.25 / 7), np.zeros(6)]
    idx = _idx(rng, T, E, K, probs)
    x = _bf16(rng, (T, d), 1.0)
    w1 = _bf16(rng, (E, h, d), 0.1)
    w2 = _bf16(rng, (E, d, h), 0.1)
    g = _bf16(rng, (T * K, d), 0.5)
    dx, dw1, dw2 = run_backward(T, d, E, K, h, idx, x, w1, w2, g)
    assert np.all(dw1[10:] == 0) and np.all(dw2[10:] == 0)
    rdx, rdw1, rdw2 = oracle.grouped_backward(bf16_bits_to_f32(x), idx, bf16_bits_to_f32(w1), bf16_bits_to_f32(w2),
                                              bf16_bits_to_f32(g), True)
    check_grad(dx, rdx, "skewed dx")
    check_grad(dw1, rdw1, "skewed dw1")
    check_grad(dw2, rdw2, "skewed dw2")


def test_backward_split_windows():
    # One expert with ~18 000 rows: its K window (work items take at most 128
    # slabs of 64 rows) is cut into three work items whose partial sums are
    # added afterwards; one small expert, one empty.
    T, d, E, K, h = 20000, 128, 3, 1, 64
    rng = np.random.default_rng(6)
    idx = _idx(rng, T, E, K, np.array([0.9, 0.1, 0.0]))
    x = _bf16(rng, (T, d), 1.0)
    w1 = _bf16(rng, (E, h, d), 0.1)
    w2 = _bf16(rng, (E, d, h), 0.1)
    g = _bf16(rng, (T * K, d), 0.5)
    dx, dw1, dw2 = run_backward(T, d, E, K, h, idx, x, w1, w2, g)
    assert np.sum(idx == 0) > 2 * 128 * 64  # more rows than two work items take
    assert np.all(dw1[2] == 0) and np.all(dw2[2] == 0)
    rdx, rdw1, rdw2 = oracle.grouped_backward(bf16_bits_to_f32(x), idx, bf16_bits_to_f32(w1), bf16_bits_to_f32(w2),
                                              bf16_bits_to_f32(g), True)
    check_grad(dx, rdx, "split dx")
    check_grad(dw1, rdw1, "split dw1")
    check_grad(dw2, rdw2, "split dw2")


def test_backward_transposed_outputs_small_experts():
    """h a multiple of 256 on 256-row tiles: the recompute and dA products write
    the activation's and dH's transposes into the weight-gradient windows
    themselves. Expert 4 holds one row, expert 5 none, expert 3 a ragged tail
    (rows past it must be written as zeros in its window)."""
    T, d, E, K, h = 3000, 128, 6, 2, 256
    rng = np.random.default_rng(11)
    idx = _idx(rng, T, E, K, np.array([0.3, 0.3, 0.3, 0.1, 0.0, 0.0]))
    idx[0] = [0, 4]
    x = _bf16(rng, (T, d), 1.0)
    w1 = _bf16(rng, (E, h, d), 0.1)
    w2 = _bf16(rng, (E, d, h), 0.1)
    g = _bf16(rng, (T * K, d), 0.5)
    counts = np.bincount(idx.ravel(), minlength=E)
    assert counts[4] == 1 and counts[5] == 0 and counts[3] % 64 != 0 and counts.sum() // E >= 512
    dx, dw1, dw2 = run_backward(T, d, E, K, h, idx, x, w1, w2, g)
    assert np.all(dw1[5] == 0) and np.all(dw2[5] == 0)
    rdx, rdw1, rdw2 = oracle.grouped_backward(bf16_bits_to_f32(x), idx, bf16_bits_to_f32(w1), bf16_bits_to_f32(w2),
                                              bf16_bits_to_f32(g), True)
    check_grad(dw1[4], rdw1[4], "one-row dw1")
    check_grad(dw2[4], rdw2[4], "one-row dw2")
    check_grad(dx, rdx, "transposed dx")
    check_grad(dw1, rdw1, "transposed dw1")
    check_grad(dw2, rdw2, "transposed dw2")


@pytest.mark.slow
def test_backward_full_vitg_sampled():
    """ViT-G skewed layer at 65 536 tokens with its own routing: the weight
    gradients of the rarest experts and of one mid-size expert, and dx of
    sampled tokens (each from the backward of its own K slots)."""
    cfg = get_config("vitg_skew_bf16")
    inp = make_inputs(cfg, parts=["x", "w_router", "bias", "w1", "w2"])
    T, d, E, K, h = cfg.T, cfg.d, cfg.E, cfg.K, cfg.h
    desc = binding.make_desc(T, d, E, K, h, 0, 1.0, "bf16")
    ws = binding.alloc_workspace(desc)
    xd = dev(inp.x)
    idx_d = torch.empty(T, K, dtype=torch.int32, device="cuda")
    gate_d = torch.empty(T, K, dtype=torch.float32, device="cuda")
    binding.moe_route(desc, xd, dev(inp.w_router), dev(inp.bias), idx_d, gate_d, ws)
    torch.cuda.synchronize()
    idx = host(idx_d)
    rng = np.random.default_rng(9)
    g = _bf16(rng, (T * K, d), 0.5)
    dx, dw1, dw2 = run_backward(T, d, E, K, h, idx, inp.x, inp.w1, inp.w2, g)
    counts, offsets, slots = oracle.permute(idx, E)
    x32, w1f, w2f, g32 = inp.f32("x"), inp.f32("w1"), inp.f32("w2"), bf16_bits_to_f32(g)
    nz = np.nonzero(counts)[0]
    picks = list(nz[np.argsort(counts[nz])[:3]]) + [int(nz[np.argsort(np.abs(counts[nz] - 600))[0]])]
    for e in picks:
        seg = slots[offsets[e]:offsets[e + 1]]
        _, rw1, rw2 = oracle.expert_backward(x32[seg // K], w1f[e], w2f[e], g32[seg], True)
        check_grad(dw1[e], rw1, f"dw1[{e}] ({counts[e]} rows)")
        check_grad(dw2[e], rw2, f"dw2[{e}] ({counts[e]} rows)")
    assert np.all(dw1[counts == 0] == 0) and np.all(dw2[counts == 0] == 0)
    tok = np.unique(np.r_[0, T - 1, rng.choice(T, 14, replace=False)])
    ref = np.zeros((tok.size, d))
    for n_t, t in enumerate(tok):
        for j in range(K):
            e = idx[t, j]
            rdx, _, _ = oracle.expert_backward(x32[t:t + 1], w1f[e], w2f[e], g32[t * K + j:t * K + j + 1], True)
            ref[n_t] += rdx[0]
    check_grad(dx[tok], ref, "sampled dx")


SW_CASES = {
    # h = 300 (ldh 320): padded halves, compaction of dW13; 256-row tiles
    "sw_h300": dict(T=3000, d=256, E=4, K=2, h=300),
    # the paper's H layer widths (h = 854, ldh = 896) at 2400 tokens
    "sw_vith_T2400": dict(T=2400, d=1280, E=31, K=7, h=854),
    # d = 64: 64-row tiles; h = 40
    "sw_h40_d64": dict(T=700, d=64, E=6, K=3, h=40),
    # h a multiple of 64: no padding, dW13 written in place
    "sw_h128": dict(T=900, d=128, E=5, K=2, h=128),
}


@pytest.mark.parametrize("name", sorted(SW_CASES))
def test_swiglu_backward_matches_oracle(name):
    from workloads import pad_last_dim

    c = SW_CASES[name]
    T, d, E, K, h = c["T"], c["d"], c["E"], c["K"], c["h"]
    rng = np.random.default_rng(100 + len(name))
    x = _bf16(rng, (T, d), 1.0)
    w13 = _bf16(rng, (E, 2 * h, d), 0.05)
    w2 = _bf16(rng, (E, d, h), 0.05)
    g = _bf16(rng, (T * K, d), 0.5)
    idx = _idx(rng, T, E, K)
    w2p = pad_last_dim(w2, 64, fill=0x3F80)  # padding columns 1.0: they must not leak into anything
    dx, dw13, dw2 = run_backward(T, d, E, K, h, idx, x, w13, w2p, g, swiglu=True)
    ldh = w2p.shape[2]
    assert dw13.shape == (E, 2 * h, d) and dw2.shape == (E, d, ldh)
    assert np.all(dw2[:, :, h:] == 0)
    rdx, rdw13, rdw2 = oracle.grouped_backward(bf16_bits_to_f32(x), idx, bf16_bits_to_f32(w13),
                                               bf16_bits_to_f32(w2), bf16_bits_to_f32(g), True, act="swiglu")
    check_grad(dx, rdx, f"{name} dx")
    check_grad(dw13, rdw13, f"{name} dw13")
    check_grad(dw2[:, :, :h], rdw2, f"{name} dw2")


@pytest.mark.slow
def test_swiglu_backward_full_vith_sampled():
    """The H layer (SwiGLU, 65 536 tokens, K = 7 of 31 experts) at full size on
    256-row persistent tiles: routing drawn without replacement with experts 0-2
    rare (a few dozen rows each), so that the oracle checks their whole dW13 and
    dW2; dx on sampled tokens, each from the backward of its own K slots."""
    from workloads import pad_last_dim

    cfg = get_config("vith_swiglu_bf16")
    inp = make_inputs(cfg, parts=["x", "w1", "w2"])
    T, d, E, K, h = cfg.T, cfg.d, cfg.E, cfg.K, cfg.h
    rng = np.random.default_rng(12)
    p = np.full(E, 1.0)
    p[:3] = 1e-4
    keys = np.log(p)[None, :] - np.log(-np.log(rng.random((T, E))))  # Gumbel top-K: K distinct experts per token
    idx = np.argsort(-keys, axis=1)[:, :K].astype(np.int32)
    g = _bf16(rng, (T * K, d), 0.5)
    w2p = pad_last_dim(inp.w2, 64)
    dx, dw13, dw2 = run_backward(T, d, E, K, h, idx, inp.x, inp.w1, w2p, g, swiglu=True)
    counts, offsets, slots = oracle.permute(idx, E)
    assert 0 < counts[:3].max() < 200 and counts[3:].min() > 10000
    x32, w1f, w2f, g32 = inp.f32("x"), inp.f32("w1"), inp.f32("w2"), bf16_bits_to_f32(g)
    assert np.all(dw2[:, :, h:] == 0)
    for e in range(3):
        seg = slots[offsets[e]:offsets[e + 1]]
        _, rw1, rw2 = oracle.expert_backward(x32[seg // K], w1f[e], w2f[e], g32[seg], True, act="swiglu")
        check_grad(dw13[e], rw1, f"dw13[{e}] ({counts[e]} rows)")
        check_grad(dw2[e][:, :h], rw2, f"dw2[{e}] ({counts[e]} rows)")
    tok = np.unique(np.r_[0, T - 1, rng.choice(T, 14, replace=False)])
    ref = np.zeros((tok.size, d))
    for n_t, t in enumerate(tok):
        for j in range(K):
            e = idx[t, j]
            rdx, _, _ = oracle.expert_backward(x32[t:t + 1], w1f[e], w2f[e], g32[t * K + j:t * K + j + 1], True,
                                               act="swiglu")
            ref[n_t] += rdx[0]
    check_grad(dx[tok], ref, "sampled dx")
