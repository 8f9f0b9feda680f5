"""Seeded synthetic inputs for the Mixtral-shaped MoE FFN layer.

This module only draws random tensors.  It holds none of the layer's
arithmetic (no routing, no GEMM, no activation), so both the GPU path and the
fp64 oracle can be fed from it without sharing any computation.

Each tensor is drawn as float32 standard normals times a per-tensor standard
deviation, from its own ``torch.Generator`` seeded with
``seed * 65536 + layer * 16 + tensor_id`` and rounded to bfloat16 with
round-to-nearest-even (the cast ``Tensor.to(torch.bfloat16)`` performs).

Tensor ids: x=0, router_w=1, w1=2, w3=3, w2=4, gamma=5.

Layouts follow ``nn.Linear`` (out x in, reduction dimension contiguous), the
convention of Mixtral checkpoints:

* ``x``        [T, d]
* ``router_w`` [E, d]
* ``w1, w3``   [E, ffn, d]
* ``w2``       [E, d, ffn]
* ``router_bias`` float32 [E] or None

8-bit variants (:func:`make_layer_fp8`) quantize the same float draws per
weight row to OCP E4M3 bytes with a float32 scale per row; that rounding is
input preparation, like the rounding to bfloat16 above.

The workloads mirror the serving setting of the paper's experiments section
(a Mixtral-8x7B endpoint at 64 concurrent requests): a 64-token decode step, a
skewed-routing decode step, a 4096-token prefill chunk (8 requests x 512 prompt
tokens), and a 32-layer decode stack.  The paper's own prompt dataset is not
used; seeded normals of the same shapes stand in for it.
"""

from __future__ import annotations

import dataclasses
import math
from typing import Optional

import torch

TID_X, TID_ROUTER, TID_W1, TID_W3, TID_W2, TID_GAMMA = 0, 1, 2, 3, 4, 5


@dataclasses.dataclass(frozen=True)
class Workload:
    """Shape and distribution of one synthetic MoE workload."""

    name: str
    T: int
    d: int
    ffn: int
    E: int
    k: int
    std_x: float
    std_router: float
    std_w1: float
    std_w3: float
    std_w2: float
    bias0: float = 0.0  # added to expert 0's router logit (skew stress); 0 = no bias
    layers: int = 1  # >1: a stack of MoE layers, each preceded by RMSNorm + residual
    eps: float = 1e-5  # RMSNorm epsilon for stacks
    seed: int = 0
    fp8: bool = False  # expert weights as E4M3 bytes with per-row scales

    def replace(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)

    @property
    def has_bias(self) -> bool:
        return self.bias0 != 0.0


MIXTRAL_D, MIXTRAL_FFN, MIXTRAL_E, MIXTRAL_K = 4096, 14336, 8, 2

WORKLOADS = {
    # tiny layer: fan-in scaled weights (variance 1/d and 1/ffn)
    "tiny_t16": Workload("tiny_t16", 16, 128, 256, 8, 2,
                         1.0, 1 / math.sqrt(128), 1 / math.sqrt(128), 1 / math.sqrt(128),
                         1 / math.sqrt(256)),
    # Mixtral-8x7B layer, one decode step of 64 concurrent requests
    "decode_t64": Workload("decode_t64", 64, MIXTRAL_D, MIXTRAL_FFN, MIXTRAL_E, MIXTRAL_K,
                           1.0, 0.02, 0.02, 0.02, 0.02),
    # decode step of 256 requests with expert 0 favoured by +2.0 on its logit
    "decode_t256_skew": Workload("decode_t256_skew", 256, MIXTRAL_D, MIXTRAL_FFN, MIXTRAL_E,
                                 MIXTRAL_K, 1.0, 0.02, 0.02, 0.02, 0.02, bias0=2.0),
    # prefill chunk of 8 x 512 prompt tokens; router logits ~ N(0,1)
    "prefill_t4096": Workload("prefill_t4096", 4096, MIXTRAL_D, MIXTRAL_FFN, MIXTRAL_E, MIXTRAL_K,
                              1.0, 1 / 64.0, 0.02, 0.02, 0.02),
    # the decode step with 8-bit (E4M3, per-row scale) expert weights
    "decode_t64_fp8": Workload("decode_t64_fp8", 64, MIXTRAL_D, MIXTRAL_FFN, MIXTRAL_E, MIXTRAL_K,
                               1.0, 0.02, 0.02, 0.02, 0.02, fp8=True),
    "decode_t256_skew_fp8": Workload("decode_t256_skew_fp8", 256, MIXTRAL_D, MIXTRAL_FFN,
                                     MIXTRAL_E, MIXTRAL_K, 1.0, 0.02, 0.02, 0.02, 0.02,
                                     bias0=2.0, fp8=True),
    # one GPU's share of the decode step under 8-way tensor parallelism: every
    # expert with ffn / 8 hidden units (the partial outputs are then summed
    # across GPUs)
    "decode_t64_tp8": Workload("decode_t64_tp8", 64, MIXTRAL_D, MIXTRAL_FFN // 8, MIXTRAL_E,
                               MIXTRAL_K, 1.0, 0.02, 0.02, 0.02, 0.02),
    # a continuous-batching step mixing 64 decode tokens with a 512-token
    # prefill chunk in one call
    "mixed_t576": Workload("mixed_t576", 576, MIXTRAL_D, MIXTRAL_FFN, MIXTRAL_E, MIXTRAL_K,
                           1.0, 0.02, 0.02, 0.02, 0.02),
    # 32 stacked layers, RMSNorm + residual around each, one decode step of 64
    "stack32_t64": Workload("stack32_t64", 64, MIXTRAL_D, MIXTRAL_FFN, MIXTRAL_E, MIXTRAL_K,
                            1.0, 0.02, 0.02, 0.02, 0.02, layers=32),
}


def _gen(seed: int, layer: int, tid: int, device) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(seed * 65536 + layer * 16 + tid)
    return g


def randn_bf16(shape, std: float, seed: int, layer: int, tid: int,
               device="cpu") -> torch.Tensor:
    """float32 N(0, std^2) draws rounded (RNE) to bfloat16."""
    g = _gen(seed, layer, tid, device)
    t = torch.randn(*shape, generator=g, device=device, dtype=torch.float32)
    t.mul_(std)
    return t.to(torch.bfloat16)


def make_x(w: Workload, device="cpu", T: Optional[int] = None) -> torch.Tensor:
    return randn_bf16((w.T if T is None else T, w.d), w.std_x, w.seed, 0, TID_X, device)


def make_layer(w: Workload, layer: int = 0, device="cpu") -> dict:
    """Weights of one MoE layer: router_w, w1, w3, w2 (bf16) and router_bias."""
    E, d, f = w.E, w.d, w.ffn
    out = {
        "router_w": randn_bf16((E, d), w.std_router, w.seed, layer, TID_ROUTER, device),
        "w1": randn_bf16((E, f, d), w.std_w1, w.seed, layer, TID_W1, device),
        "w3": randn_bf16((E, f, d), w.std_w3, w.seed, layer, TID_W3, device),
        "w2": randn_bf16((E, d, f), w.std_w2, w.seed, layer, TID_W2, device),
        "router_bias": None,
    }
    if w.has_bias:
        b = torch.zeros(E, dtype=torch.float32, device=device)
        b[0] = w.bias0
        out["router_bias"] = b
    return out


FP8_MAX = 448.0  # largest finite OCP E4M3 value


def quantize_rows_fp8(w: torch.Tensor):
    """8-bit expert weights from float ones, one scale per row (output channel):
    s = max|row| / 448, q = E4M3(row / s) rounded to nearest even (torch's
    float8_e4m3fn cast).  Returns (q as uint8 bytes, s as float32 [..., rows]).
    An all-zero row gets scale 1."""
    w = w.float()
    amax = w.abs().amax(dim=-1)
    s = torch.where(amax > 0, amax / FP8_MAX, torch.ones_like(amax))
    q = (w / s.unsqueeze(-1)).clamp(-FP8_MAX, FP8_MAX).to(torch.float8_e4m3fn)
    return q.view(torch.uint8), s.contiguous()


def randn_f32(shape, std: float, seed: int, layer: int, tid: int, device="cpu") -> torch.Tensor:
    """float32 N(0, std^2) draws (the source the bf16 weights are rounded from)."""
    g = _gen(seed, layer, tid, device)
    t = torch.randn(*shape, generator=g, device=device, dtype=torch.float32)
    return t.mul_(std)


def make_layer_fp8(w: Workload, layer: int = 0, device="cpu") -> dict:
    """One MoE layer with 8-bit expert weights: router_w (bf16) and router_bias
    as in :func:`make_layer`; w1q, w3q [E, ffn, d] and w2q [E, d, ffn] as
    E4M3 bytes (uint8) with per-row float32 scales w1s, w3s [E, ffn] and
    w2s [E, d].  The float weights are the same draws the bf16 layer rounds."""
    E, d, f = w.E, w.d, w.ffn
    out = {
        "router_w": randn_bf16((E, d), w.std_router, w.seed, layer, TID_ROUTER, device),
        "router_bias": None,
    }
    for name, shape, std, tid in (("w1", (E, f, d), w.std_w1, TID_W1), ("w3", (E, f, d), w.std_w3, TID_W3),
                                  ("w2", (E, d, f), w.std_w2, TID_W2)):
        q, sc = quantize_rows_fp8(randn_f32(shape, std, w.seed, layer, tid, device))
        out[name + "q"], out[name + "s"] = q, sc
    if w.has_bias:
        b = torch.zeros(E, dtype=torch.float32, device=device)
        b[0] = w.bias0
        out["router_bias"] = b
    return out


def make_gamma(w: Workload, layer: int = 0, device="cpu", random: bool = False) -> torch.Tensor:
    """RMSNorm scale: ones for the stack workload; U(0.5, 1.5) when ``random``."""
    if not random:
        return torch.ones(w.d, dtype=torch.bfloat16, device=device)
    g = _gen(w.seed, layer, TID_GAMMA, device)
    t = torch.rand(w.d, generator=g, device=device, dtype=torch.float32) + 0.5
    return t.to(torch.bfloat16)


def bf16_bits(t: torch.Tensor):
    """Raw bfloat16 bit patterns of a tensor as a host numpy uint16 array."""
    import numpy as np

    assert t.dtype == torch.bfloat16
    return t.detach().contiguous().cpu().view(torch.int16).numpy().view(np.uint16)


def from_bits(a, device="cpu") -> torch.Tensor:
    """Inverse of :func:`bf16_bits`."""
    import numpy as np

    a = np.ascontiguousarray(a, dtype=np.uint16)
    return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).to(device)
