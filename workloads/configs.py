"""The five layer shapes the MoE-layer forward pass is built and measured on.

Each shape is a ViT encoder's patch-token batch fed to one fine-grained MoE MLP
layer (fine-grained experts and one always-on shared expert, Sec. 3.2
"Architecture Design"; sigmoid gating with a selection-only balancing bias,
Sec. 3.2 "Load Balancing", Eq. (7)). Token counts follow the paper's image
resolutions: 224 px / patch 16 -> 196, 336 px / patch 14 -> 576 (the token count
of the latency table, Sec. 4.6), 448 px / patch 14 -> 1024.

Experts are fc1 -> GELU -> fc2 by default. SwiGLU experts (act="swiglu":
SiLU(W1 x) * (W3 x), then W2; the form of the paper's models, appendix
"Implementation Details", and of its inference kernel, appendix "MoE Kernel",
Algorithm 1) store the gate and up projections stacked, W1 [E, 2h, d] with the
gate rows first.
"""

from __future__ import annotations

from dataclasses import dataclass, replace


@dataclass(frozen=True)
class LayerConfig:
    name: str
    T: int            # tokens in the batch
    d: int            # model width
    E: int            # routed experts
    K: int            # experts chosen per token
    h: int            # hidden width of one routed expert (fc1 d->h, fc2 h->d)
    h_shared: int     # hidden width of the shared expert, 0 = no shared expert
    dtype: str        # "f32" or "bf16": x, all weights, expert outputs and y
    bias: str         # "uniform" (U(-0.1, 0.1)), "zero" or "zipf" (skewed load)
    lam: float = 1.0  # shared-expert weight lambda (the paper fixes lambda = 1)
    weight_std: float = 0.02
    seed: int = 0
    images: int = 1
    tokens_per_image: int = 0
    note: str = ""
    act: str = "gelu"  # expert activation: "gelu" (two matrices) or "swiglu" (three)

    @property
    def slots(self) -> int:
        """Number of (token, chosen expert) assignments, T*K."""
        return self.T * self.K

    def with_tokens(self, T: int) -> "LayerConfig":
        """Same layer, a different token count (for tests that must run the
        oracle over every token)."""
        return replace(self, T=T, name=f"{self.name}@T{T}")

    @property
    def n_mats(self) -> int:
        """Weight matrices of one expert: 2 (W1, W2) or 3 for SwiGLU (W1, W3, W2)."""
        return 3 if self.act == "swiglu" else 2

    def gemm_flops(self) -> float:
        """Useful grouped-GEMM flops of one forward pass: the expert matrices of
        the K chosen experts per token plus the shared expert (padding
        excluded)."""
        return 2.0 * self.n_mats * self.T * self.d * (self.K * self.h + self.h_shared)

    def router_flops(self) -> float:
        return 2.0 * self.T * self.d * self.E

    def routed_weight_bytes(self) -> int:
        es = 2 if self.dtype == "bf16" else 4
        return self.n_mats * self.E * self.h * self.d * es

    def shared_weight_bytes(self) -> int:
        es = 2 if self.dtype == "bf16" else 4
        return self.n_mats * self.h_shared * self.d * es


CONFIGS = {
    "tiny_f32": LayerConfig(
        name="tiny_f32", T=196, d=256, E=8, K=2, h=256, h_shared=0, dtype="f32",
        bias="uniform", images=1, tokens_per_image=196,
        note="1 image at 224px/patch16; top-2 of 8; no shared expert; fp32"),
    "vitb_bf16": LayerConfig(
        name="vitb_bf16", T=18432, d=768, E=64, K=8, h=384, h_shared=768, dtype="bf16",
        bias="uniform", images=32, tokens_per_image=576,
        note="32 images x 576 tokens (336px/patch14); top-8 of 64"),
    "vitl_bf16": LayerConfig(
        name="vitl_bf16", T=65536, d=1024, E=128, K=8, h=512, h_shared=1024, dtype="bf16",
        bias="zero", images=64, tokens_per_image=1024,
        note="64 images x 1024 tokens (448px/patch14); top-8 of 128; balanced (b=0)"),
    "vitg_skew_bf16": LayerConfig(
        name="vitg_skew_bf16", T=65536, d=1536, E=256, K=8, h=768, h_shared=1536, dtype="bf16",
        bias="zipf", images=64, tokens_per_image=1024,
        note="64 images x 1024 tokens; top-8 of 256; bias gives a Zipf(1.2) expert load"),
    "single_image_bf16": LayerConfig(
        name="single_image_bf16", T=1025, d=1536, E=256, K=8, h=768, h_shared=1536, dtype="bf16",
        bias="zero", images=1, tokens_per_image=1025,
        note="1 image x (1024 patches + 1 extra token); ~32 rows per expert; weight-read bound"),
    "single_image_swiglu_bf16": LayerConfig(
        name="single_image_swiglu_bf16", T=1025, d=1536, E=256, K=8, h=768, h_shared=1536, dtype="bf16",
        bias="zero", images=1, tokens_per_image=1025, act="swiglu",
        note="single_image_bf16 with SwiGLU experts: 1.81 GB of routed weights; weight-read bound"),
    "vith_swiglu_bf16": LayerConfig(
        name="vith_swiglu_bf16", T=65536, d=1280, E=31, K=7, h=854, h_shared=854, dtype="bf16",
        bias="uniform", images=64, tokens_per_image=1024, act="swiglu",
        note="the paper's H vision layer: 32 SwiGLU experts of width 854 (1 shared + 31 routed), "
             "8 active (the shared one + top-7); 64 images x 1024 tokens"),
}

# Short aliases c1..c7 in the order the configs are listed above.
ALIASES = {f"c{i + 1}": k for i, k in enumerate(CONFIGS)}


def get_config(name: str) -> LayerConfig:
    name = ALIASES.get(name, name)
    if name not in CONFIGS:
        raise KeyError(f"unknown layer config {name!r}; known: {sorted(CONFIGS)} or c1..c{len(CONFIGS)}")
    return CONFIGS[name]
