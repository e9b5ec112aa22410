"""The skewed ViT-G workload (65 536 tokens, 256 experts, top-8) keeps the load
profile it is defined by: routed by the oracle (fp32 recipes R and S, the
stored selection bias), the experts whose Zipf(1.2) target is capped at T
receive every token, the eight lowest-ranked experts receive exactly 15, 12,
10, 8, 6, 4, 2 and 1 tokens (the experts under 16 tokens), and every other
expert gets between 16 and T tokens. If the stored bias or the input
generator drifted, the tiny-group paths would silently stop being exercised
at full size; this pins them. CPU only (the oracle's routing, about a minute
with the input generation)."""

import os
import sys

import numpy as np
import pytest

import oracle
from workloads import get_config, make_inputs

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.join(HERE, "golden"))

import make_vitg_skew_bias as skew  # noqa: E402


@pytest.fixture(scope="module")
def c4_counts():
    cfg = get_config("c4")
    inp = make_inputs(cfg, parts=["x", "w_router", "bias"])
    idx, gate = oracle.route(inp.f32("x"), inp.f32("w_router"), inp.bias, cfg.K)
    counts = np.bincount(idx.reshape(-1), minlength=cfg.E)
    return cfg, counts, gate


def test_skewed_workload_tail_and_capped_experts(c4_counts):
    cfg, counts, _ = c4_counts
    L, tail, capped = skew.targets(cfg.E, cfg.T, cfg.K)
    assert counts.sum() == cfg.T * cfg.K
    # The tail, expert by expert, in the order of the construction.
    assert counts[tail].tolist() == skew.TAIL == [15, 12, 10, 8, 6, 4, 2, 1]
    assert int((counts < 16).sum()) == len(skew.TAIL)
    # Capped experts take every token (a token picks an expert at most once).
    assert len(capped) >= 2 and np.all(counts[capped] == cfg.T)
    # The bulk: at least 16 and at most T tokens, following the Zipf profile
    # (realised within 5 % of the target for the median expert).
    bulk = np.setdiff1d(np.arange(cfg.E), np.r_[tail, capped])
    assert counts[bulk].min() >= 16 and counts[bulk].max() <= cfg.T
    assert float(np.median(np.abs(counts[bulk] / L[bulk] - 1))) < 0.05
    # Larger targets get larger loads (rank correlation of the bulk).
    rt = np.argsort(np.argsort(L[bulk]))
    rc = np.argsort(np.argsort(counts[bulk]))
    assert np.corrcoef(rt, rc)[0, 1] > 0.99


def test_skewed_workload_gates_sum_to_one(c4_counts):
    cfg, _, gate = c4_counts
    assert np.max(np.abs(gate.astype(np.float64).sum(1) - 1.0)) <= cfg.K * 2.0 ** -23
