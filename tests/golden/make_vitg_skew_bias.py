"""Write the selection-bias vector of the skewed ViT-G layer (65536 tokens,
d = 1536, 256 experts, top-8) so that the expert loads follow a Zipf(1.2)
profile, with a tail of experts that receive fewer than 16 tokens.

The bias enters only the selection key sigmoid(s) + b (paper Sec. 3.2,
Eq. (7)); it is an *input* of the layer. Zipf(1.2) over 256 ranks asks more
than T tokens of the top expert, which top-K routing cannot give (one token
picks an expert at most once), so the target is capped at T and the excess
spread over the other experts in proportion (water filling). The eight
lowest-ranked experts are then set to 15, 12, 10, 8, 6, 4, 2 and 1 tokens and
the mass they give up is spread the same way.

Construction, on the actual seed-0 batch:
  1. sigmoid scores of every (token, expert) from the oracle (recipes R, S);
  2. experts whose target is all T tokens get b = 3 (sigma + 3 beats any
     other key, since every other bias stays <= 1.5);
  3. the rest: b += eta * (ln(L + 0.5) - ln(count + 0.5)), re-centred, 300
     steps with eta = 0.2 * 0.985^step;
  4. each tail expert e: b_e is placed between the L_e-th and (L_e + 1)-th
     smallest thresholds kth_t(other keys) - sigma_{t,e}, so exactly L_e tokens
     select it given the others.
The realised loads (from the oracle's fp32 routing) are printed; they follow
the target shape, not every count exactly.

Run from the repository root:  python tests/golden/make_vitg_skew_bias.py
"""

import os
import sys

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)

import oracle  # noqa: E402
from workloads import get_config, make_inputs  # noqa: E402
from workloads.generate import ZIPF_BIAS_FILE  # noqa: E402

ZIPF_S = 1.2
TAIL = [15, 12, 10, 8, 6, 4, 2, 1]
PERM_SEED = 1200


def water_fill(L, cap, fixed):
    L = L.astype(np.float64).copy()
    for _ in range(100):
        over = (L > cap) & ~fixed
        if not over.any():
            break
        excess = float((L[over] - cap).sum())
        L[over] = cap
        fixed = fixed | over
        free = ~fixed
        L[free] += excess * L[free] / L[free].sum()
    return L


def targets(E, T, K):
    ranks = np.arange(1, E + 1, dtype=np.float64)
    p = ranks ** -ZIPF_S
    L = p / p.sum() * T * K
    L = water_fill(L, T, np.zeros(E, bool))
    tail_ranks = np.arange(E - len(TAIL), E)
    fixed = L >= T
    removed = L[tail_ranks].sum() - sum(TAIL)
    L[tail_ranks] = TAIL
    fixed[tail_ranks] = True
    free = ~fixed
    L[free] += removed * L[free] / L[free].sum()
    L = water_fill(L, T, fixed)
    perm = np.random.default_rng(PERM_SEED).permutation(E)  # expert perm[r] has rank r+1
    by_expert = np.empty(E)
    by_expert[perm] = L
    tail = perm[tail_ranks]
    capped = perm[L >= T - 0.5]
    return by_expert, tail, capped


def counts_of(keys, K):
    top = np.argpartition(-keys, K - 1, axis=1)[:, :K]
    return np.bincount(top.reshape(-1), minlength=keys.shape[1])


def main():
    cfg = get_config("vitg_skew_bf16")
    T, E, K = cfg.T, cfg.E, cfg.K
    inp = make_inputs(cfg, parts=["x", "w_router"])
    sig = oracle.scores(inp.f32("x"), inp.f32("w_router"))
    L, tail, capped = targets(E, T, K)
    b = np.zeros(E)
    b[capped] = 3.0
    bulk = np.ones(E, bool)
    bulk[tail] = False
    bulk[capped] = False
    b[tail] = -1.0
    eta = 0.2
    for step in range(300):
        c = counts_of(sig + b[None, :].astype(np.float32), K)
        b[bulk] += eta * (np.log(L[bulk] + 0.5) - np.log(c[bulk] + 0.5))
        b[bulk] -= b[bulk].mean()
        b[bulk] = np.clip(b[bulk], -3.0, 1.5)
        eta *= 0.985
    for e in tail[np.argsort(L[tail])[::-1]]:
        keys = sig + b[None, :].astype(np.float32)
        keys[:, e] = -np.inf
        kth = -np.partition(-keys, K - 1, axis=1)[:, K - 1]
        tau = np.sort(kth.astype(np.float64) - sig[:, e])
        n = int(L[e])
        b[e] = 0.5 * (tau[n - 1] + tau[n])
    b32 = b.astype(np.float32)
    idx, _ = oracle.topk_from_scores(sig, b32, K)
    real = np.bincount(idx.reshape(-1), minlength=E)
    order = np.argsort(-L)
    print("target (top 8) ", np.round(L[order[:8]]).astype(int).tolist())
    print("realised       ", real[order[:8]].tolist())
    print("target (tail)  ", np.round(L[order[-10:]]).astype(int).tolist())
    print("realised       ", real[order[-10:]].tolist())
    mid = order[8:-8]
    print("median |realised/target - 1| over the bulk:",
          float(np.median(np.abs(real[mid] / L[mid] - 1))))
    print("experts under 16 tokens:", int((real < 16).sum()), " max load:", int(real.max()))
    with open(ZIPF_BIAS_FILE, "w") as f:
        f.write("# Selection bias of the skewed ViT-G layer (seed 0), one fp32 value per expert.\n")
        f.write("# Written by tests/golden/make_vitg_skew_bias.py (calls only the oracle and numpy).\n")
        for v in b32:
            f.write(f"{float(v)!r}\n")
    print("wrote", ZIPF_BIAS_FILE)


if __name__ == "__main__":
    main()
