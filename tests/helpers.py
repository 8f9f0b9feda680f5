"""Host-side helpers shared by the tests (no layer arithmetic beyond widening)."""

from __future__ import annotations

import numpy as np
import torch

from paper_2408_00008_amd import inputs


def widen(bits) -> np.ndarray:
    """bf16 bit patterns (uint16) -> float64, exactly."""
    b = np.ascontiguousarray(bits, dtype=np.uint16)
    return (b.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def bits_of(a64) -> np.ndarray:
    """float64 values that are exactly bf16-representable -> bf16 bit patterns."""
    f = np.ascontiguousarray(a64, dtype=np.float32)
    u = f.view(np.uint32)
    assert np.all((u & 0xFFFF) == 0), "value is not exactly representable in bf16"
    return (u >> 16).astype(np.uint16)


def tiny_case(T, d, ffn, E, k, seed=0, std=0.5, bias=None):
    """Seeded bf16 tensors for a small MoE layer, as host bit arrays."""
    w = inputs.Workload("tiny", T, d, ffn, E, k, 1.0, std, std, std, std, seed=seed)
    lay = inputs.make_layer(w)
    case = {
        "x": inputs.bf16_bits(inputs.make_x(w)),
        "wr": inputs.bf16_bits(lay["router_w"]),
        "w1": inputs.bf16_bits(lay["w1"]),
        "w3": inputs.bf16_bits(lay["w3"]),
        "w2": inputs.bf16_bits(lay["w2"]),
        "bias": None if bias is None else np.asarray(bias, np.float32),
        "T": T, "d": d, "ffn": ffn, "E": E, "k": k,
    }
    return case


def workload_case(name, seed=0, device="cpu", T=None):
    """bf16 host bit arrays of a named workload's layer 0."""
    w = inputs.WORKLOADS[name].replace(seed=seed)
    if T is not None:
        w = w.replace(T=T)
    lay = inputs.make_layer(w, 0, device)
    x = inputs.make_x(w, device)
    return w, {
        "x": inputs.bf16_bits(x),
        "wr": inputs.bf16_bits(lay["router_w"]),
        "w1": inputs.bf16_bits(lay["w1"]),
        "w3": inputs.bf16_bits(lay["w3"]),
        "w2": inputs.bf16_bits(lay["w2"]),
        "bias": None if lay["router_bias"] is None else lay["router_bias"].cpu().numpy(),
        "T": w.T, "d": w.d, "ffn": w.ffn, "E": w.E, "k": w.k,
    }


def rowwise_rel(got, ref) -> float:
    """max over rows of max|got-ref| / max|ref| (rows with an all-zero
    reference use an absolute error)."""
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    if ref.size == 0:
        return 0.0
    num = np.abs(got - ref).max(axis=-1)
    den = np.abs(ref).max(axis=-1)
    den = np.where(den == 0, 1.0, den)
    return float((num / den).max())


def tiny_case_fp8(T, d, ffn, E, k, seed=0, std=0.5, bias=None):
    """tiny_case with E4M3 expert weights (per-row scales), quantized from
    float normals by the input generator's row quantizer."""
    from paper_2408_00008_amd import inputs

    c = tiny_case(T, d, ffn, E, k, seed=seed, std=std, bias=bias)
    g = torch.Generator().manual_seed(seed * 7919 + 17)
    for name, shape in (("w1", (E, ffn, d)), ("w3", (E, ffn, d)), ("w2", (E, d, ffn))):
        w = torch.randn(*shape, generator=g, dtype=torch.float32) * std
        q, s = inputs.quantize_rows_fp8(w)
        c[name + "q"], c[name + "s"] = q.numpy(), s.numpy()
    return c
