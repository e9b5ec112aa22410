"""MI355X-native forward pass of one fine-grained MoE MLP layer (MoE-ViE).

The compute lives in libmoevie.so (HIP kernels for gfx950 behind the C ABI
in include/moe_vie.h); ``binding`` marshals torch device tensors into it.
"""

__all__ = ["binding", "build"]
