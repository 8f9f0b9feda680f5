"""Seeded synthetic inputs for the Mixtral-shaped MoE FFN layer.

This module only draws random tensors.  It holds none of the layer's
arithmetic (no routing, no GEMM, no activation), so both the GPU path and the
fp64 oracle can be fed from it without sharing any computation.

Each tensor is drawn as float32 standard normals times a per-tensor standard
deviation, from its own ``torch.Generator`` seeded with
``seed * 65536 + layer * 16 + tensor_id`` and rounded to bfloat16 with
round-to-nearest-even (the cast ``Tensor.to(torch.bfloat16)`` performs).

Tensor ids: x=0, router_w=1, w1=2, w3=3, w2=4, gamma=5; for the decoder layer
around the MoE block: wq=6, wk=7, wv=8, wo=9, gamma_attn=10, k_cache=11,
v_cache=12, page assignment=13, cached lengths=14, residual stream h=15.

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
TID_WQ, TID_WK, TID_WV, TID_WO, TID_GAMMA_ATTN = 6, 7, 8, 9, 10
TID_KC, TID_VC, TID_PAGES, TID_LENS, TID_H = 11, 12, 13, 14, 15


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
    # decoder layer around the MoE block (hq = 0: the MoE layer alone)
    hq: int = 0          # query heads
    hkv: int = 0         # key/value heads
    hd: int = 128        # head dimension
    page: int = 16       # KV-cache positions per page
    ctx: int = 0         # positions already cached per request (the largest, if ragged)
    ctx_ragged: bool = False  # cached lengths uniform in [0, ctx] instead of all ctx
    theta: float = 1e6   # RoPE base
    std_attn: float = 0.02  # std of the attention projections

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
    # the prefill chunk and the mixed step with 8-bit expert weights
    "prefill_t4096_fp8": Workload("prefill_t4096_fp8", 4096, MIXTRAL_D, MIXTRAL_FFN, MIXTRAL_E,
                                  MIXTRAL_K, 1.0, 1 / 64.0, 0.02, 0.02, 0.02, fp8=True),
    "mixed_t576_fp8": Workload("mixed_t576_fp8", 576, MIXTRAL_D, MIXTRAL_FFN, MIXTRAL_E,
                               MIXTRAL_K, 1.0, 0.02, 0.02, 0.02, 0.02, fp8=True),
    # one GPU's share of the decode step under 8-way tensor parallelism: every
    # expert with ffn / 8 hidden units (the partial outputs are then summed
    # across GPUs)
    "decode_t64_tp8": Workload("decode_t64_tp8", 64, MIXTRAL_D, MIXTRAL_FFN // 8, MIXTRAL_E,
                               MIXTRAL_K, 1.0, 0.02, 0.02, 0.02, 0.02),
    # a continuous-batching step mixing 64 decode tokens with a 512-token
    # prefill chunk in one call
    "mixed_t576": Workload("mixed_t576", 576, MIXTRAL_D, MIXTRAL_FFN, MIXTRAL_E, MIXTRAL_K,
                           1.0, 0.02, 0.02, 0.02, 0.02),
    # one decoder layer of Mixtral-8x7B (32 query heads, 8 KV heads of 128),
    # decode step of 64 requests with 1024 positions cached each
    "decoder_t64_ctx1024": Workload("decoder_t64_ctx1024", 64, MIXTRAL_D, MIXTRAL_FFN, MIXTRAL_E,
                                    MIXTRAL_K, 1.0, 0.02, 0.02, 0.02, 0.02, hq=32, hkv=8,
                                    ctx=1024),
    # few requests with long contexts: 8 requests x 8192 cached positions (the
    # same cache bytes per layer as 64 x 1024)
    "decoder_t8_ctx8192": Workload("decoder_t8_ctx8192", 8, MIXTRAL_D, MIXTRAL_FFN, MIXTRAL_E,
                                   MIXTRAL_K, 1.0, 0.02, 0.02, 0.02, 0.02, hq=32, hkv=8,
                                   ctx=8192),
    # the whole model: 32 decoder layers, one decode step of 64 requests with
    # 1024 positions cached each (every layer has its own cache)
    "decoder32_t64_ctx1024": Workload("decoder32_t64_ctx1024", 64, MIXTRAL_D, MIXTRAL_FFN,
                                      MIXTRAL_E, MIXTRAL_K, 1.0, 0.02, 0.02, 0.02, 0.02,
                                      layers=32, hq=32, hkv=8, ctx=1024),
    # the same with 8-bit (E4M3, per-row scale) expert weights, the paper's
    # 8-bit Mixtral
    "decoder32_t64_ctx1024_fp8": Workload("decoder32_t64_ctx1024_fp8", 64, MIXTRAL_D, MIXTRAL_FFN,
                                          MIXTRAL_E, MIXTRAL_K, 1.0, 0.02, 0.02, 0.02, 0.02,
                                          layers=32, hq=32, hkv=8, ctx=1024, fp8=True),
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


# ---- the decoder layer around the MoE block -----------------------------------

def make_attention(w: Workload, layer: int = 0, device="cpu") -> dict:
    """Attention projections (nn.Linear layout) and the two RMSNorm scales:
    wq [hq*hd, d], wk, wv [hkv*hd, d], wo [d, hq*hd] bf16 with std w.std_attn;
    gamma_attn, gamma_moe U(0.5, 1.5) bf16."""
    d, qd, kd = w.d, w.hq * w.hd, w.hkv * w.hd
    g = _gen(w.seed, layer, TID_GAMMA_ATTN, device)
    ga = (torch.rand(d, generator=g, device=device) + 0.5).to(torch.bfloat16)
    return {"wq": randn_bf16((qd, d), w.std_attn, w.seed, layer, TID_WQ, device),
            "wk": randn_bf16((kd, d), w.std_attn, w.seed, layer, TID_WK, device),
            "wv": randn_bf16((kd, d), w.std_attn, w.seed, layer, TID_WV, device),
            "wo": randn_bf16((d, qd), w.std_attn, w.seed, layer, TID_WO, device),
            "gamma_attn": ga, "gamma_moe": make_gamma(w, layer, device, random=True)}


def make_kv_cache(w: Workload, layer: int = 0, device="cpu") -> dict:
    """A paged KV cache holding the requests' earlier positions.  Request t
    has pos[t] positions cached (w.ctx, or uniform in [0, w.ctx]) and owns
    maxp = ceil((w.ctx + 1) / page) pages, taken from a seeded permutation of
    all T * maxp pages; its new token goes to position pos[t].  Cached keys
    and values are N(0, 1) bf16 (every slot is filled; slots at or past a
    request's position are never read before they are written).  Returns
    k_cache, v_cache [T*maxp, hkv, page, hd] bf16, page_table [T, maxp] int32,
    pos [T] and ctx = pos + 1 [T] int32."""
    maxp = (w.ctx + 1 + w.page - 1) // w.page
    npages = w.T * maxp
    shape = (npages, w.hkv, w.page, w.hd)
    kc = randn_bf16(shape, 1.0, w.seed, layer, TID_KC, device)
    vc = randn_bf16(shape, 1.0, w.seed, layer, TID_VC, device)
    gp = _gen(w.seed, layer, TID_PAGES, "cpu")
    table = torch.randperm(npages, generator=gp).reshape(w.T, maxp).to(torch.int32)
    if w.ctx_ragged:
        gl = _gen(w.seed, layer, TID_LENS, "cpu")
        pos = torch.randint(0, w.ctx + 1, (w.T,), generator=gl, dtype=torch.int32)
    else:
        pos = torch.full((w.T,), w.ctx, dtype=torch.int32)
    return {"k_cache": kc, "v_cache": vc, "page_table": table.to(device), "pos": pos.to(device),
            "ctx": (pos + 1).to(device)}


def make_h(w: Workload, device="cpu") -> torch.Tensor:
    """The residual stream entering the layer, float32 N(0, 1)."""
    g = _gen(w.seed, 0, TID_H, device)
    return torch.randn(w.T, w.d, generator=g, device=device, dtype=torch.float32)

