"""MI355X-native sparse Mixture-of-Experts FFN layer (Mixtral-8x7B shape).

The layer is the engine hot spot of the serving system in "ScaleLLM: A
Resource-Frugal LLM Serving Framework by Optimizing End-to-End Efficiency"
(Sec. 4.1 targets MoE models; Sec. 5 serves Mixtral-8x7B): router GEMM,
softmax top-k gating, token-to-expert permutation, per-expert SwiGLU GEMMs
and the gate-weighted combine, all as hand-written gfx950 HIP kernels behind
the C ABI in ``include/moe.h`` (``libmoe.so``).

``binding`` wraps that ABI for torch tensors (device memory and streams only);
``inputs`` draws the seeded synthetic workloads; ``stack`` chains layers with
RMSNorm and a residual stream.  Importing the package does not load the GPU
library; the first binding call does, and fails loudly if it is not built.
"""

from . import inputs  # noqa: F401  (pure tensor generation, no GPU)

__all__ = ["inputs", "binding", "stack"]


def __getattr__(name):
    if name in ("binding", "stack"):
        import importlib

        return importlib.import_module(f".{name}", __name__)
    raise AttributeError(name)
