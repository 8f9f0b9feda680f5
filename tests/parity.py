"""Host-side comparison rules between the GPU library and the fp64 oracle.

Routing.  The GPU scores tokens in f32, the oracle in f64, so a token whose
top-k decision hinges on a logit gap below the rounding of an f32 dot product
can legitimately come out differently.  On the oracle's sorted logits
l(1) >= ... >= l(E) of a token:

  m_set = l(k) - l(k+1)                 (gap that decides the chosen SET)
  m_ord = min_{j<k} l(j) - l(j+1)       (gaps that decide the slot ORDER)

If m_set > tol the GPU's set must equal the oracle's, and if m_ord > tol too
the ordered ids must match exactly.  Otherwise the token is ambiguous: the
GPU's ids must still be k distinct experts, each within tol of the k-th
largest logit, and the oracle recomputes that token's output with the GPU's
ids so the output check still covers it.  tol = 1e-4.

Outputs.  Row-wise relative max-norm error
  max_t max_i |got - ref| / max_i |ref|  <= 1e-2
(bf16 operands and bf16 rounding of the SwiGLU intermediate and the output,
f32 accumulation, against exact f64).
"""

from __future__ import annotations

import numpy as np

ROUTE_TOL = 1e-4
OUT_TOL = 1e-2


def sorted_logits(logits_row):
    E = len(logits_row)
    order = sorted(range(E), key=lambda e: (-logits_row[e], e))
    return order, [logits_row[e] for e in order]


def check_routing(gpu_ids, ref_logits, k, tol=ROUTE_TOL):
    """Applies the margin rule.  Returns the boolean mask of ambiguous tokens;
    raises AssertionError on a violation."""
    gpu_ids = np.asarray(gpu_ids)
    ref_logits = np.asarray(ref_logits, np.float64)
    T, E = ref_logits.shape
    amb = np.zeros(T, bool)
    for t in range(T):
        order, l = sorted_logits(ref_logits[t])
        g = [int(v) for v in gpu_ids[t]]
        assert len(set(g)) == k and all(0 <= v < E for v in g), f"token {t}: invalid ids {g}"
        m_set = l[k - 1] - l[k] if k < E else np.inf
        m_ord = min((l[j] - l[j + 1] for j in range(k - 1)), default=np.inf)
        if m_set > tol:
            assert set(g) == set(order[:k]), f"token {t}: set {g} != {order[:k]} (margin {m_set:.2e})"
            if m_ord > tol:
                assert g == order[:k], f"token {t}: order {g} != {order[:k]} (margin {m_ord:.2e})"
            else:
                amb[t] = True
        else:
            amb[t] = True
        if amb[t]:
            kth = l[k - 1]
            assert all(ref_logits[t, v] >= kth - tol for v in g), f"token {t}: {g} not a top-{k}"
            # slots must still be in non-increasing logit order within tol
            for j in range(k - 1):
                assert ref_logits[t, g[j]] >= ref_logits[t, g[j + 1]] - tol, f"token {t}: order"
    return amb


def rowwise_rel(got, ref) -> float:
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    if ref.size == 0:
        return 0.0
    num = np.abs(got - ref).max(axis=-1)
    den = np.abs(ref).max(axis=-1)
    den = np.where(den == 0, 1.0, den)
    return float((num / den).max())


def norm_rel(got, ref) -> float:
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    if ref.size == 0:
        return 0.0
    den = np.abs(ref).max()
    return float(np.abs(got - ref).max() / (den if den > 0 else 1.0))


def bf16_ulp_diff(a_bits, b_bits):
    """|ulp distance| between two arrays of bf16 bit patterns (finite values)."""
    def key(u):
        u = np.asarray(u, np.uint16).astype(np.int32)
        return np.where(u & 0x8000, -(u & 0x7FFF), u & 0x7FFF)
    return np.abs(key(a_bits) - key(b_bits))


def round_bf16_bits(a64):
    """float64 -> bf16 bits, rounding the f64 value to nearest-even bf16 in one step."""
    a64 = np.asarray(a64, np.float64)
    # round to the nearest bf16 directly from f64: decompose via f32 is double rounding;
    # instead use exact integer arithmetic on the f64 value.
    m, e = np.frexp(a64)  # a = m * 2^e, 0.5 <= |m| < 1
    scaled = np.ldexp(m, 8)  # 8 significant bits for bf16
    r = np.round(scaled)  # numpy rounds half to even
    vals = np.ldexp(r, e - 8).astype(np.float32)  # exact: r has <= 8 significant bits
    u = vals.view(np.uint32)
    return (u >> 16).astype(np.uint16)
