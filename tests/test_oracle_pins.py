"""Pins of the CPU oracle against facts that do not come from the oracle itself:
closed forms, textbook values, library routines, invariants and a brute-force
float64 reference written independently (tests/brute.py)."""

import math

import numpy as np
import pytest

import oracle
from brute import bf16_round64, expert64, gelu64, layer64, route64
from workloads import bf16_bits_to_f32, f32_to_bf16_bits

F32_EPS = 2.0 ** -23


def bf16_values(rng, shape, std):
    return bf16_bits_to_f32(f32_to_bf16_bits(rng.standard_normal(shape).astype(np.float32) * std))


# ---------------------------------------------------------------- recipe S


def test_sigmoid_exact_points():
    assert oracle.sigmoid([0.0])[0] == np.float32(0.5)
    # Saturation: exp(-s) is clamped at exp(-87), so 1 + e rounds to 1.
    assert oracle.sigmoid([87.0, 200.0, 1e30])[0] == np.float32(1.0)
    lo = oracle.sigmoid([-87.0, -200.0, -1e30])
    assert lo[0] == lo[1] == lo[2]
    assert lo[0] >= np.finfo(np.float32).tiny  # stays a normal number
    assert abs(float(lo[0]) - 1.0 / (1.0 + math.exp(87.0))) < 1e-3 * float(lo[0])


def test_sigmoid_within_3_ulp_of_float64():
    s = np.concatenate([np.linspace(-30, 30, 60001, dtype=np.float32),
                        np.random.default_rng(1).normal(0, 3, 20000).astype(np.float32)])
    got = oracle.sigmoid(s).astype(np.float64)
    ref = 1.0 / (1.0 + np.exp(-s.astype(np.float64)))
    ulp = np.spacing(ref.astype(np.float32)).astype(np.float64)
    assert np.max(np.abs(got - ref) / ulp) <= 3.0


def test_sigmoid_symmetry():
    s = np.linspace(-10, 10, 2001, dtype=np.float32)
    a = oracle.sigmoid(s).astype(np.float64)
    b = oracle.sigmoid(-s).astype(np.float64)
    assert np.max(np.abs(a + b - 1.0)) <= 4 * F32_EPS
    assert np.all(a[s > 0] > 0.5) and np.all(a[s < 0] < 0.5)


def test_sigmoid_constants_derivation():
    # The recipe's reduction constants are defined from ln 2; check the
    # definitions hold for the literals the recipe uses.
    hi = float.fromhex("0x1.62e4p-1")
    lo = float(np.float32(float.fromhex("0x1.7f7d1cp-20")))
    assert hi == 22713 * 2.0 ** -15 == round(math.log(2) * 2 ** 15) / 2 ** 15
    assert all(float(np.float32(n * hi)) == n * hi for n in range(-126, 127))
    assert lo == float(np.float32(math.log(2) - hi))
    assert float(np.float32(float.fromhex("0x1.715476p+0"))) == float(np.float32(1 / math.log(2)))


# ---------------------------------------------------------------- recipe R


def test_logit_exact_on_integers():
    rng = np.random.default_rng(2)
    x = rng.integers(-8, 9, size=(5, 96)).astype(np.float32)
    w = rng.integers(-8, 9, size=(7, 96)).astype(np.float32) * np.float32(0.25)
    got = oracle.logits(x, w)
    assert np.array_equal(got.astype(np.float64), x.astype(np.float64) @ w.T.astype(np.float64))


def test_logit_chain_is_ascending_and_fused():
    # Ascending order: 1 + 2^-24 rounds back to 1 (tie to even) at each step,
    # so the chain gives exactly 1; any other summation order gives 1 + 2^-23.
    x = np.array([[1.0, 1.0, 1.0]], np.float32)
    w = np.array([[1.0, 2.0 ** -24, 2.0 ** -24]], np.float32)
    assert oracle.logits(x, w)[0, 0] == np.float32(1.0)
    w_rev = np.array([[2.0 ** -24, 2.0 ** -24, 1.0]], np.float32)
    assert oracle.logits(x, w_rev)[0, 0] == np.float32(1.0 + 2.0 ** -23)
    # Fused multiply-add: (1 + 2^-12)^2 - 1 = 2^-11 + 2^-24 exactly when the
    # product is not rounded first (a separate multiply gives 2^-11).
    a = 1.0 + 2.0 ** -12
    x = np.array([[1.0, a]], np.float32)
    w = np.array([[-1.0, a]], np.float32)
    assert oracle.logits(x, w)[0, 0] == np.float32(2.0 ** -11 + 2.0 ** -24)


def test_logit_error_bound_bf16():
    rng = np.random.default_rng(3)
    d = 1536
    x = bf16_values(rng, (64, d), 1.0)
    w = bf16_values(rng, (32, d), 0.02)
    got = oracle.logits(x, w).astype(np.float64)
    exact = x.astype(np.float64) @ w.T.astype(np.float64)  # bf16 products are exact in fp64
    absdot = np.abs(x.astype(np.float64)) @ np.abs(w.T.astype(np.float64))
    u = 2.0 ** -24
    gamma = d * u / (1 - d * u)
    assert np.all(np.abs(got - exact) <= gamma * absdot)
    assert np.max(np.abs(got - exact)) > 0  # genuinely fp32, not a float64 dot


# ------------------------------------------------------------------ route


def _tiny_router(seed, T, d, E, std=0.5):
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((T, d)).astype(np.float32)
    wr = (rng.standard_normal((E, d)) * std / math.sqrt(d)).astype(np.float32)
    b = rng.uniform(-0.1, 0.1, E).astype(np.float32)
    return x, wr, b


@pytest.mark.parametrize("E,K", [(8, 2), (16, 4), (64, 8)])
def test_route_matches_float64_brute_force(E, K):
    x, wr, b = _tiny_router(10 + E, 200, 64, E, std=4.0)
    idx, gate = oracle.route(x, wr, b, K)
    bidx, bgate, keys = route64(x, wr, b, K)
    gap = keys[:, K - 1] - keys[:, K]
    ok = gap > 1e-4  # far from a tie: any correct arithmetic agrees
    assert ok.mean() > 0.9
    assert np.array_equal(idx[ok], bidx[ok])
    assert np.max(np.abs(gate[ok] - bgate[ok])) < 1e-6


def test_route_gates_sum_to_one():
    x, wr, b = _tiny_router(5, 500, 64, 32, std=4.0)
    _, gate = oracle.route(x, wr, b, 8)
    assert np.max(np.abs(gate.astype(np.float64).sum(1) - 1.0)) <= 8 * F32_EPS


def test_route_bias_forces_selection_but_not_gates():
    # sigma is in (0, 1), so a bias of +2 puts these experts above all others.
    x, wr, _ = _tiny_router(6, 100, 32, 16, std=4.0)
    forced = [3, 7, 11, 12]
    b = np.zeros(16, np.float32)
    b[forced] = 2.0
    idx, gate = oracle.route(x, wr, b, 4)
    assert all(sorted(r) == forced for r in idx.tolist())
    sig = 1.0 / (1.0 + np.exp(-(x.astype(np.float64) @ wr.T.astype(np.float64))))
    chosen = np.take_along_axis(sig, idx, axis=1)
    # slots ordered by descending key = descending sigma within the forced set
    assert np.all(np.diff(chosen, axis=1) <= 1e-6)
    assert np.max(np.abs(gate - chosen / chosen.sum(1, keepdims=True))) < 1e-6


def test_route_k_equals_e():
    x, wr, b = _tiny_router(7, 50, 16, 8, std=4.0)
    idx, gate = oracle.route(x, wr, b, 8)
    assert all(sorted(r) == list(range(8)) for r in idx.tolist())
    sig = 1.0 / (1.0 + np.exp(-(x.astype(np.float64) @ wr.T.astype(np.float64))))
    g = np.take_along_axis(sig, idx, axis=1)
    assert np.max(np.abs(gate - g / sig.sum(1, keepdims=True))) < 1e-6


def test_route_exact_ties_go_to_lower_index():
    x, wr, _ = _tiny_router(8, 64, 32, 8, std=4.0)
    wr[5] = wr[2]  # experts 2 and 5 tie exactly for every token
    wr[6] = wr[1]  # and so do 1 and 6
    b = np.zeros(8, np.float32)
    b[[1, 2, 5, 6]] = 2.0  # all four are forced above the rest
    idx, _ = oracle.route(x, wr, b, 3)
    s = x.astype(np.float64) @ wr.T.astype(np.float64)
    n_checked = 0
    for t, r in enumerate(idx.tolist()):
        a, c = s[t, 1], s[t, 2]
        if abs(a - c) < 1e-3:
            continue
        # key order is (pair with the larger score: lower index first), then the other pair
        want = [1, 6, 2] if a > c else [2, 5, 1]
        assert r == want
        n_checked += 1
    assert n_checked > 50


def test_route_single_expert():
    x, wr, b = _tiny_router(9, 20, 16, 1)
    idx, gate = oracle.route(x, wr, b, 1)
    assert np.all(idx == 0) and np.all(gate == np.float32(1.0))


def test_route_no_bias_equals_zero_bias():
    x, wr, _ = _tiny_router(11, 100, 32, 16, std=4.0)
    a = oracle.route(x, wr, None, 4)
    b = oracle.route(x, wr, np.zeros(16, np.float32), 4)
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])


def test_topk_from_scores_agrees_with_route():
    x, wr, b = _tiny_router(12, 100, 32, 16, std=4.0)
    sc = oracle.scores(x, wr)
    assert np.array_equal(sc, oracle.sigmoid(oracle.logits(x, wr)))
    i1, g1 = oracle.route(x, wr, b, 4)
    i2, g2 = oracle.topk_from_scores(sc, b, 4)
    assert np.array_equal(i1, i2) and np.array_equal(g1, g2)


# ---------------------------------------------------------------- permute


@pytest.mark.parametrize("T,E,K", [(1, 4, 2), (37, 8, 2), (300, 64, 8), (257, 16, 16)])
def test_permute_is_stable_argsort(T, E, K):
    rng = np.random.default_rng(T)
    # distinct experts per token, some experts left empty on purpose
    idx = np.stack([rng.permutation(E)[:K] for _ in range(T)]).astype(np.int32)
    idx[idx == E - 1] = 0 if K == 1 else idx[idx == E - 1]
    counts, offsets, slots = oracle.permute(idx, E)
    flat = idx.reshape(-1)
    assert np.array_equal(slots, np.argsort(flat, kind="stable"))
    assert np.array_equal(counts, np.bincount(flat, minlength=E))
    assert np.array_equal(offsets, np.concatenate([[0], np.cumsum(counts)]))
    assert np.array_equal(np.sort(slots), np.arange(T * K))
    for e in range(E):
        seg = slots[offsets[e]:offsets[e + 1]]
        assert np.all(flat[seg] == e) and np.all(np.diff(seg) > 0)


def test_permute_empty_experts():
    idx = np.array([[0, 3], [3, 0], [0, 3]], np.int32)
    counts, offsets, slots = oracle.permute(idx, 6)
    assert counts.tolist() == [3, 0, 0, 3, 0, 0]
    assert offsets.tolist() == [0, 3, 3, 3, 6, 6, 6]
    assert slots.tolist() == [0, 3, 4, 1, 2, 5]


# ------------------------------------------------------------- expert MLP


def test_gelu_textbook_values():
    # GELU(v) = v * Phi(v); Phi(1) = 0.8413447460685429 (standard normal CDF).
    g = oracle.gelu([0.0, 1.0, -1.0, 10.0, -10.0])
    assert g[0] == 0.0
    assert abs(g[1] - 0.8413447460685429) < 1e-15
    assert abs(g[2] + 0.15865525393145707) < 1e-15
    assert abs(g[3] - 10.0) < 1e-12 and abs(g[4]) < 1e-12
    v = np.linspace(-6, 6, 1001)
    gv = oracle.gelu(v)
    assert np.max(np.abs(gv - oracle.gelu(-v) - v)) < 1e-14  # v*Phi(v) - (-v)Phi(-v) = v
    assert np.max(np.abs(gv - gelu64(v))) < 1e-15


def test_round_bf16_ties_and_exact_values():
    r = oracle.round_bf16
    assert r([1.0 + 2 ** -8])[0] == 1.0                      # tie -> even (1.0)
    assert r([1.0 + 3 * 2 ** -8])[0] == 1.0 + 2 ** -6        # tie -> even
    assert r([1.0 + 2 ** -8 + 2 ** -30])[0] == 1.0 + 2 ** -7  # above the tie
    assert r([-3.0 - 2 ** -7])[0] == -3.0                    # tie at exponent 1
    rng = np.random.default_rng(4)
    v = rng.standard_normal(20000).astype(np.float32)
    ref = bf16_bits_to_f32(f32_to_bf16_bits(v)).astype(np.float64)
    assert np.array_equal(r(v.astype(np.float64)), ref)


@pytest.mark.parametrize("act_bf16", [False, True])
def test_expert_identity_closed_form(act_bf16):
    rng = np.random.default_rng(5)
    d = 48
    x = rng.standard_normal((9, d)).astype(np.float32)
    c = 0.375
    out = oracle.expert_rows(x, np.eye(d, dtype=np.float32), (c * np.eye(d)).astype(np.float32), act_bf16)
    a = gelu64(x.astype(np.float64))
    if act_bf16:
        a = oracle.round_bf16(a)
    assert np.max(np.abs(out - c * a)) < 1e-15


@pytest.mark.parametrize("act_bf16", [False, True])
def test_expert_matches_float64_matmul(act_bf16):
    rng = np.random.default_rng(6)
    d, h = 40, 24  # non-square: a transposed operand cannot pass
    x = rng.standard_normal((17, d)).astype(np.float32)
    w1 = (rng.standard_normal((h, d)) * 0.3).astype(np.float32)
    w2 = (rng.standard_normal((d, h)) * 0.3).astype(np.float32)
    out = oracle.expert_rows(x, w1, w2, act_bf16)
    ref = expert64(x, w1, w2, act_bf16)
    tol = 1e-12 if not act_bf16 else 1e-2  # bf16 rounding may flip at half-way points
    assert np.max(np.abs(out - ref)) < tol
    if act_bf16:
        assert np.mean(np.abs(out - ref) < 1e-12) > 0.95


# ---------------------------------------------------------------- combine


def test_combine_matches_einsum_and_special_cases():
    rng = np.random.default_rng(7)
    T, K, d = 11, 3, 16
    eo = rng.standard_normal((T * K, d))
    g = rng.random((T, K)).astype(np.float32)
    sh = rng.standard_normal((T, d))
    y = oracle.combine(eo, g, sh, 1.0)
    ref = np.einsum("tk,tkd->td", g.astype(np.float64), eo.reshape(T, K, d)) + sh
    assert np.max(np.abs(y - ref)) < 1e-13
    assert np.array_equal(oracle.combine(eo, g, None, 1.0), oracle.combine(eo, g, sh, 0.0))
    onehot = np.zeros((T, K), np.float32)
    onehot[:, 1] = 1.0
    assert np.array_equal(oracle.combine(eo, onehot, None, 0.0), eo.reshape(T, K, d)[:, 1])


# ------------------------------------------------------------------ layer


def _tiny_layer(seed, T=40, d=32, E=8, K=2, h=16, hs=24, act_bf16=False):
    rng = np.random.default_rng(seed)
    cast = (lambda a: bf16_bits_to_f32(f32_to_bf16_bits(a.astype(np.float32)))) if act_bf16 else \
        (lambda a: a.astype(np.float32))
    x = cast(rng.standard_normal((T, d)))
    wr = cast(rng.standard_normal((E, d)) * 0.5)
    b = rng.uniform(-0.1, 0.1, E).astype(np.float32)
    w1 = cast(rng.standard_normal((E, h, d)) * 0.2)
    w2 = cast(rng.standard_normal((E, d, h)) * 0.2)
    w1s = cast(rng.standard_normal((hs, d)) * 0.2) if hs else None
    w2s = cast(rng.standard_normal((d, hs)) * 0.2) if hs else None
    return x, wr, b, w1, w2, w1s, w2s


@pytest.mark.parametrize("act_bf16,hs,K", [(False, 24, 2), (False, 0, 3), (True, 24, 4)])
def test_layer_matches_brute_force(act_bf16, hs, K):
    x, wr, b, w1, w2, w1s, w2s = _tiny_layer(20 + K, K=K, hs=hs, act_bf16=act_bf16)
    idx, gate, y = oracle.layer(x, wr, b, w1, w2, w1s, w2s, K, 1.0, act_bf16)
    bidx, bgate, keys, by = layer64(x, wr, b, w1, w2, w1s, w2s, K, 1.0, act_bf16)
    ok = keys[:, K - 1] - keys[:, K] > 1e-4
    assert ok.mean() > 0.8
    assert np.array_equal(idx[ok], bidx[ok])
    tol = 1e-6 if not act_bf16 else 2e-2
    assert np.max(np.abs(y[ok] - by[ok])) < tol
    if act_bf16:
        rel = np.linalg.norm(y[ok] - by[ok]) / np.linalg.norm(by[ok])
        assert rel < 1e-4


def test_layer_identical_experts_ignore_routing():
    x, wr, b, w1, w2, w1s, w2s = _tiny_layer(30, K=3)
    w1[:] = w1[0]
    w2[:] = w2[0]
    _, _, y = oracle.layer(x, wr, b, w1, w2, w1s, w2s, 3, 0.5, False)
    ref = expert64(x, w1[0], w2[0], False) + 0.5 * expert64(x, w1s, w2s, False)
    assert np.max(np.abs(y - ref)) < 1e-6  # gates sum to 1 up to fp32 rounding


def test_layer_zero_routed_output_is_shared_mlp():
    x, wr, b, w1, w2, w1s, w2s = _tiny_layer(31)
    w2[:] = 0
    _, _, y = oracle.layer(x, wr, b, w1, w2, w1s, w2s, 2, 1.0, False)
    assert np.max(np.abs(y - expert64(x, w1s, w2s, False))) < 1e-12


def test_layer_scaled_identity_experts_closed_form():
    # d = h, W1[e] = I, W2[e] = c_e I: y_t = (sum_j g_j c_{e_j}) GELU(x_t)
    x, wr, b, _, _, _, _ = _tiny_layer(32, d=16, h=16, hs=0, K=2)
    E = wr.shape[0]
    c = np.arange(1, E + 1, dtype=np.float32) / 4
    w1 = np.broadcast_to(np.eye(16, dtype=np.float32), (E, 16, 16)).copy()
    w2 = (c[:, None, None] * np.eye(16, dtype=np.float32)).astype(np.float32)
    idx, gate, y = oracle.layer(x, wr, b, w1, w2, None, None, 2, 1.0, False)
    coef = (gate.astype(np.float64) * c[idx]).sum(1, keepdims=True)
    assert np.max(np.abs(y - coef * gelu64(x.astype(np.float64)))) < 1e-12


def test_layer_token_permutation_equivariance_and_subsets():
    x, wr, b, w1, w2, w1s, w2s = _tiny_layer(33, T=30)
    idx, gate, y = oracle.layer(x, wr, b, w1, w2, w1s, w2s, 2, 1.0, False)
    perm = np.random.default_rng(0).permutation(30)
    idx_p, gate_p, y_p = oracle.layer(x[perm], wr, b, w1, w2, w1s, w2s, 2, 1.0, False)
    assert np.array_equal(idx_p, idx[perm]) and np.array_equal(gate_p, gate[perm])
    assert np.array_equal(y_p, y[perm])
    sub = np.array([29, 0, 7, 7], np.int32)
    i_s, g_s, y_s = oracle.layer(x, wr, b, w1, w2, w1s, w2s, 2, 1.0, False, tokens=sub)
    assert np.array_equal(i_s, idx[sub]) and np.array_equal(y_s, y[sub])


def test_layer_route_agrees_with_route_stage():
    x, wr, b, w1, w2, w1s, w2s = _tiny_layer(34, K=3)
    idx, gate, _ = oracle.layer(x, wr, b, w1, w2, w1s, w2s, 3, 1.0, False)
    i2, g2 = oracle.route(x, wr, b, 3)
    assert np.array_equal(idx, i2) and np.array_equal(gate, g2)


def test_layer_stages_compose_to_layer():
    # route -> permute -> per-expert MLP over grouped rows -> combine equals the
    # per-token layer definition (grouping only reorders the work).
    x, wr, b, w1, w2, w1s, w2s = _tiny_layer(35, T=50, K=3)
    K = 3
    idx, gate = oracle.route(x, wr, b, K)
    counts, offsets, slots = oracle.permute(idx, w1.shape[0])
    eo = np.zeros((x.shape[0] * K, x.shape[1]))
    for e in range(w1.shape[0]):
        seg = slots[offsets[e]:offsets[e + 1]]
        if seg.size:
            eo[seg] = oracle.expert_rows(x[seg // K], w1[e], w2[e], False)
    sh = oracle.expert_rows(x, w1s, w2s, False)
    y = oracle.combine(eo, gate, sh, 1.0)
    _, _, y_ref = oracle.layer(x, wr, b, w1, w2, w1s, w2s, K, 1.0, False)
    assert np.max(np.abs(y - y_ref)) < 1e-12


def test_bf16_round64_helper_agrees():
    v = np.random.default_rng(9).standard_normal(1000)
    assert np.array_equal(bf16_round64(v), oracle.round_bf16(v))


# ---- Loss-free balancing bias update (Sec. 3.2 "Load Balancing", Eqs. (8)-(9))


def test_bias_update_zscore_closed_form():
    # counts {1, 2, 3}: mean 2, population deviation sqrt(2/3), so the z-scores
    # are -sqrt(3/2), 0, +sqrt(3/2); the overloaded expert's bias goes down.
    out = oracle.bias_update([1, 2, 3], [0.0, 0.0, 0.0], 1.0, oracle.BIAS_ZSCORE)
    z = math.sqrt(1.5)
    assert out.tolist() == [np.float32(z), np.float32(0.0), np.float32(-z)]
    out = oracle.bias_update([1, 2, 3], [0.5, -0.25, 0.125], 0.125, oracle.BIAS_ZSCORE)
    want = np.array([0.5 + 0.125 * z, -0.25, 0.125 - 0.125 * z]).astype(np.float32)
    assert np.array_equal(out, want)


def test_bias_update_zscore_uses_population_deviation():
    rng = np.random.default_rng(7)
    for E in (8, 64, 256):
        counts = rng.integers(0, 5000, size=E).astype(np.int32)
        out = -oracle.bias_update(counts, np.zeros(E, np.float32), 1.0, oracle.BIAS_ZSCORE).astype(np.float64)
        # z-scores over the whole population: mean 0 and mean square 1
        assert abs(out.sum()) < 1e-4 and abs((out ** 2).mean() - 1.0) < 1e-6
        c = counts.astype(np.float64)
        ref = (c - c.mean()) / c.std(ddof=0)
        assert np.max(np.abs(out - ref)) <= 1e-6 * max(1.0, np.max(np.abs(ref)))
        b = rng.normal(0, 0.05, E).astype(np.float32)
        got = oracle.bias_update(counts, b, 0.01, oracle.BIAS_ZSCORE)
        want = (b.astype(np.float64) - 0.01 * np.float64(np.float32(1)) * ref).astype(np.float32)
        assert np.max(np.abs(got.astype(np.float64) - want)) <= np.spacing(np.abs(want)).max()


def test_bias_update_sign_rule():
    b = np.array([0.5, 0.5, 0.5, 0.5], np.float32)
    out = oracle.bias_update([5, 1, 3, 3], b, 0.25, oracle.BIAS_SIGN)
    assert out.tolist() == [0.25, 0.75, 0.5, 0.5]
    # a fractional mean (1.5): both experts move, in opposite directions
    out = oracle.bias_update([1, 2], [0.0, 0.0], 0.125, oracle.BIAS_SIGN)
    assert out.tolist() == [0.125, -0.125]
    # the update is one fp32 add of -alpha or +alpha
    b = np.array([0.1, 0.1], np.float32)
    out = oracle.bias_update([3, 0], b, np.float32(0.3), oracle.BIAS_SIGN)
    assert out.tolist() == [np.float32(np.float32(0.1) - np.float32(0.3)), np.float32(np.float32(0.1) + np.float32(0.3))]


def test_bias_update_balanced_load_changes_nothing():
    b = np.array([0.3, -0.2, 0.0, 1e-3], np.float32)
    for rule in (oracle.BIAS_SIGN, oracle.BIAS_ZSCORE):
        assert np.array_equal(oracle.bias_update([7, 7, 7, 7], b, 0.5, rule), b)
        assert np.array_equal(oracle.bias_update([0, 0, 0, 0], b, 0.5, rule), b)
    assert np.array_equal(oracle.bias_update([9], [0.25], 1.0, oracle.BIAS_ZSCORE), np.float32([0.25]))


# ---- SwiGLU experts (App. "MoE Kernel", Algorithm 1 Phase 2: SiLU(gate) * up)


def test_silu_known_values_and_identities():
    from scipy.special import expit

    assert oracle.silu([0.0])[0] == 0.0
    assert abs(oracle.silu([1.0])[0] - 0.7310585786300049) < 1e-15  # logistic(1) = e / (1 + e)
    v = np.linspace(-30, 30, 601)
    s = oracle.silu(v)
    assert np.max(np.abs(s - v * expit(v))) < 1e-13 * np.maximum(1, np.abs(v)).max()
    assert np.max(np.abs(oracle.silu(-v) - (s - v))) < 1e-12  # silu(-v) = silu(v) - v
    eps = 1e-6
    assert abs((oracle.silu([eps])[0] - oracle.silu([-eps])[0]) / (2 * eps) - 0.5) < 1e-9  # slope 1/2 at 0


@pytest.mark.parametrize("act_bf16", [False, True])
def test_swiglu_expert_closed_form(act_bf16):
    from scipy.special import expit

    rng = np.random.default_rng(15)
    d = 32
    x = rng.standard_normal((7, d)).astype(np.float32)
    c = 0.625
    w13 = np.concatenate([np.eye(d), c * np.eye(d)]).astype(np.float32)  # gate = I, up = c I
    out = oracle.expert_rows(x, w13, np.eye(d, dtype=np.float32), act_bf16, act="swiglu")
    xd = x.astype(np.float64)
    a = xd * expit(xd) * (c * xd)
    if act_bf16:
        a = oracle.round_bf16(a)
    assert np.max(np.abs(out - a)) < 1e-15


@pytest.mark.parametrize("act_bf16", [False, True])
def test_swiglu_expert_matches_float64_matmul(act_bf16):
    from scipy.special import expit

    rng = np.random.default_rng(16)
    d, h = 40, 24  # non-square: a transposed operand cannot pass
    x = rng.standard_normal((13, d)).astype(np.float32)
    w13 = (rng.standard_normal((2 * h, d)) * 0.3).astype(np.float32)
    w2 = (rng.standard_normal((d, h)) * 0.3).astype(np.float32)
    out = oracle.expert_rows(x, w13, w2, act_bf16, act="swiglu")
    xd = x.astype(np.float64)
    g = xd @ w13[:h].astype(np.float64).T
    u = xd @ w13[h:].astype(np.float64).T
    hid = g * expit(g) * u
    if act_bf16:
        hid = bf16_round64(hid)
    ref = hid @ w2.astype(np.float64).T
    tol = 1e-12 if not act_bf16 else 1e-2
    assert np.max(np.abs(out - ref)) < tol
    if act_bf16:
        assert np.mean(np.abs(out - ref) < 1e-12) > 0.95


def test_swiglu_layer_identical_experts_and_shared():
    rng = np.random.default_rng(17)
    x, wr, b, w1, w2, w1s, w2s = _tiny_layer(32, K=3)
    E, h, d = w1.shape
    hs = w1s.shape[0]
    w13 = (rng.standard_normal((E, 2 * h, d)) * 0.2).astype(np.float32)
    w13[:] = w13[0]
    w2[:] = w2[0]
    w13s = (rng.standard_normal((2 * hs, d)) * 0.2).astype(np.float32)
    idx, _, y = oracle.layer(x, wr, b, w13, w2, w13s, w2s, 3, 0.5, False, act="swiglu")
    ref = oracle.expert_rows(x, w13[0], w2[0], False, act="swiglu") + \
        0.5 * oracle.expert_rows(x, w13s, w2s, False, act="swiglu")
    assert np.max(np.abs(y - ref)) < 1e-6  # gates sum to 1 up to fp32 rounding
    gi, _, _ = oracle.layer(x, wr, b, w1, w2, w1s, w2s, 3, 0.5, False)
    assert np.array_equal(idx, gi)  # routing does not depend on the expert type
    w2[:] = 0
    _, _, y0 = oracle.layer(x, wr, b, w13, w2, w13s, w2s, 3, 1.0, False, act="swiglu")
    assert np.max(np.abs(y0 - oracle.expert_rows(x, w13s, w2s, False, act="swiglu"))) < 1e-12


# ---------------------------------------------------------- expert backward


def test_activation_gradients_against_scipy_and_differences():
    from scipy.special import expit
    from scipy.stats import norm

    assert oracle.gelu_grad([0.0])[0] == 0.5
    assert abs(oracle.gelu_grad([1.0])[0] - (norm.cdf(1.0) + norm.pdf(1.0))) < 1e-15
    assert oracle.silu_grad([0.0])[0] == 0.5
    v = np.linspace(-8, 8, 161)
    eps = 1e-5
    gelu = lambda z: z * norm.cdf(z)  # noqa: E731
    silu = lambda z: z * expit(z)  # noqa: E731
    assert np.max(np.abs(oracle.gelu_grad(v) - (gelu(v + eps) - gelu(v - eps)) / (2 * eps))) < 1e-8
    assert np.max(np.abs(oracle.silu_grad(v) - (silu(v + eps) - silu(v - eps)) / (2 * eps))) < 1e-8


def _dyadic(rng, shape, scale):
    """float32 values on a 2^-8 grid: x +- 2^-14 stays exact in float32."""
    return (np.round(rng.uniform(-scale, scale, shape) * 256) / 256).astype(np.float32)


@pytest.mark.parametrize("act", ["gelu", "swiglu"])
def test_expert_backward_matches_central_differences(act):
    # L = sum_r <G_r, W2 act(W1 x_r)>; the oracle's forward (float64 from
    # float32 inputs) is differentiated numerically in every input and weight.
    rng = np.random.default_rng(31)
    n, d, h = 3, 6, 5  # d != h: a transposed operand cannot pass
    hr = 2 * h if act == "swiglu" else h
    x = _dyadic(rng, (n, d), 1.5)
    w1 = _dyadic(rng, (hr, d), 0.7)
    w2 = _dyadic(rng, (d, h), 0.7)
    g = rng.standard_normal((n, d)).astype(np.float32)
    dx, dw1, dw2 = oracle.expert_backward(x, w1, w2, g, False, act=act)
    step = 2.0 ** -14

    def loss(xx, a1, a2):
        return float(np.sum(oracle.expert_rows(xx, a1, a2, False, act=act) * g.astype(np.float64)))

    def fd(which, arr, idx):
        p, m = arr.copy(), arr.copy()
        p[idx] += np.float32(step)
        m[idx] -= np.float32(step)
        args_p = [x, w1, w2]
        args_m = [x, w1, w2]
        args_p[which], args_m[which] = p, m
        return (loss(*args_p) - loss(*args_m)) / (2 * step)

    for which, arr, grad in ((0, x, dx), (1, w1, dw1), (2, w2, dw2)):
        for idx in np.ndindex(arr.shape):
            want = fd(which, arr, idx)
            assert abs(grad[idx] - want) <= 1e-7 * (1 + abs(want)), (act, which, idx, grad[idx], want)


def test_expert_backward_identity_closed_form():
    from scipy.stats import norm

    rng = np.random.default_rng(32)
    d, c = 16, 0.375
    x = rng.standard_normal((9, d)).astype(np.float32)
    g = rng.standard_normal((9, d)).astype(np.float32)
    eye = np.eye(d, dtype=np.float32)
    dx, dw1, dw2 = oracle.expert_backward(x, eye, c * eye, g, False)
    xd, gd = x.astype(np.float64), g.astype(np.float64)
    gp = norm.cdf(xd) + xd * norm.pdf(xd)  # GELU'
    assert np.max(np.abs(dx - c * gd * gp)) < 1e-13
    assert np.max(np.abs(dw2 - gd.T @ (xd * norm.cdf(xd)))) < 1e-12
    assert np.max(np.abs(dw1 - (c * gd * gp).T @ xd)) < 1e-12


@pytest.mark.parametrize("act", ["gelu", "swiglu"])
def test_expert_backward_bf16_rounding_points(act):
    # bf16 layers: dW2 uses the rounded activation (the forward's), and the
    # pre-activation gradient is rounded before it meets x and W1.
    from scipy.special import expit
    from scipy.stats import norm

    rng = np.random.default_rng(33)
    n, d, h = 11, 24, 10
    hr = 2 * h if act == "swiglu" else h
    x = bf16_values(rng, (n, d), 1.0)
    w1 = bf16_values(rng, (hr, d), 0.3)
    w2 = bf16_values(rng, (d, h), 0.3)
    g = bf16_values(rng, (n, d), 1.0)
    dx, dw1, dw2 = oracle.expert_backward(x, w1, w2, g, True, act=act)
    xd, gd = x.astype(np.float64), g.astype(np.float64)
    p = xd @ w1[:h].astype(np.float64).T
    da = gd @ w2.astype(np.float64)
    if act == "gelu":
        a = p * norm.cdf(p)
        dpre = bf16_round64(da * (norm.cdf(p) + p * norm.pdf(p)))
    else:
        q = xd @ w1[h:].astype(np.float64).T
        s = expit(p)
        a = p * s * q
        dpre = np.concatenate([bf16_round64(da * q * s * (1 + p * (1 - s))), bf16_round64(da * p * s)], axis=1)
    a = bf16_round64(a)
    assert np.max(np.abs(dw2 - gd.T @ a)) < 1e-9
    assert np.max(np.abs(dw1 - dpre.T @ xd)) < 1e-9
    assert np.max(np.abs(dx - dpre @ w1.astype(np.float64))) < 1e-9


def test_grouped_backward_sums_slots_and_experts():
    # Identical experts: each token's dx is the sum over its K slots of one
    # expert's backward, and the weight gradients summed over experts equal
    # one expert's over all slots; linear in the output gradient.
    rng = np.random.default_rng(34)
    T, d, E, K, h = 30, 12, 5, 3, 7
    x = rng.standard_normal((T, d)).astype(np.float32)
    w1 = np.repeat(rng.standard_normal((1, h, d)).astype(np.float32) * 0.4, E, axis=0)
    w2 = np.repeat(rng.standard_normal((1, d, h)).astype(np.float32) * 0.4, E, axis=0)
    idx = np.stack([rng.choice(E, K, replace=False) for _ in range(T)]).astype(np.int32)
    g1 = rng.standard_normal((T * K, d)).astype(np.float32)
    g2 = rng.standard_normal((T * K, d)).astype(np.float32)
    dx, dw1, dw2 = oracle.grouped_backward(x, idx, w1, w2, g1, False)
    rows = np.repeat(x, K, axis=0)
    dxr, dw1r, dw2r = oracle.expert_backward(rows, w1[0], w2[0], g1, False)
    assert np.max(np.abs(dx - dxr.reshape(T, K, d).sum(1))) < 1e-12
    assert np.max(np.abs(dw1.sum(0) - dw1r)) < 1e-11 and np.max(np.abs(dw2.sum(0) - dw2r)) < 1e-11
    used = np.zeros(E, bool)
    used[np.unique(idx)] = True
    assert np.all(dw1[~used] == 0) and np.all(dw2[~used] == 0)
    a = oracle.grouped_backward(x, idx, w1, w2, g1 + g2, False)
    b = oracle.grouped_backward(x, idx, w1, w2, g2, False)
    for u, v, w in zip(a, (dx, dw1, dw2), b):
        assert np.max(np.abs(u - (v + w))) < 1e-5
