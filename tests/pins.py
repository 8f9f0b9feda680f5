"""Pins of the fp64 oracle against facts outside itself.

Each pin takes an ``Oracle`` (the real one, or a deliberately broken build in
the mutation test) and raises AssertionError if the oracle disagrees with:

* a pure-Python brute force on tiny inputs (subset enumeration for top-k,
  dense all-expert evaluation) -- a different algorithm;
* textbook reductions computed by a library routine (torch fp64 on the CPU):
  E=1,k=1 is a dense SwiGLU FFN; k=E is the softmax-weighted mixture of all
  experts; RMSNorm against ``torch.nn.functional.rms_norm``;
* closed forms: one-hot inputs, constant rows, a hand-worked example whose
  numbers are stored in ``tests/golden/hand_example.json``;
* invariants of the layer: gate weights sum to one, token-permutation
  equivariance, a zeroed expert contributes nothing, relabelling experts
  changes nothing, scaling W2 by a power of two scales the output exactly;
* for 8-bit (OCP E4M3) expert weights: every byte against torch's
  float8_e4m3fn conversion, the values the OCP specification tabulates, and
  the brute force fed with weights dequantized by torch;
* for the decoder layer around the MoE block: bf16 rounding against torch's
  float32 -> bfloat16 conversion and exact ties, RoPE on unit vectors in
  closed form, paged attention against torch's fp64
  scaled_dot_product_attention, GQA against repeated KV heads, page
  relocation, one-position and equal-key closed forms, and the layer's
  composition (Wo = 0 leaves the MoE block; position 0 returns the new
  value rows).
"""

from __future__ import annotations

import json
import math
import os

import numpy as np
import torch

import bruteforce as bf
from helpers import bits_of, tiny_case, tiny_case_fp8, widen

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")

TINY_SHAPES = [  # (T, d, ffn, E, k)
    (1, 4, 6, 1, 1),
    (5, 8, 12, 2, 1),
    (6, 8, 16, 4, 2),
    (7, 16, 8, 8, 2),
    (4, 12, 10, 8, 1),
    (3, 8, 8, 5, 3),
    (2, 6, 4, 4, 4),
]


def _nested(a):
    return widen(a).tolist()


def _bf_case(c):
    x = _nested(c["x"])
    wr = _nested(c["wr"])
    w1 = _nested(c["w1"])
    w3 = _nested(c["w3"])
    w2 = _nested(c["w2"])
    bias = None if c["bias"] is None else [float(b) for b in c["bias"]]
    return bf.moe_layer(x, wr, w1, w3, w2, c["k"], bias)


def _run(o, c):
    return o.moe_layer(c["x"], c["wr"], c["w1"], c["w3"], c["w2"], c["k"], c["bias"])


def _close(a, b, rtol=1e-12, atol=1e-13):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    assert a.shape == b.shape, (a.shape, b.shape)
    err = np.abs(a - b)
    tol = atol + rtol * np.abs(b)
    assert np.all(err <= tol), f"max err {err.max():.3e} (rtol {rtol}, atol {atol})"


# --------------------------------------------------------------------------
def pin_bruteforce_random(o):
    """Oracle == brute force on random tiny layers (with and without bias)."""
    for i, (T, d, ffn, E, k) in enumerate(TINY_SHAPES):
        for bias in (None, [0.75 * (e % 3) - 0.5 for e in range(E)]):
            c = tiny_case(T, d, ffn, E, k, seed=100 + i, bias=bias)
            r = _run(o, c)
            out, ids, gates, logits = _bf_case(c)
            _close(r["logits"], logits)
            assert r["ids"].tolist() == ids, (r["ids"].tolist(), ids)
            _close(r["gates"], gates)
            _close(r["out"], out, rtol=1e-11, atol=1e-12)


def pin_bruteforce_ties(o):
    """Exactly tied logits rank the lower expert index first."""
    T, d, ffn, E, k = 4, 8, 8, 6, 2
    c = tiny_case(T, d, ffn, E, k, seed=7)
    wr = c["wr"].copy()
    wr[4] = wr[1]  # experts 1 and 4 always tie
    wr[5] = wr[2]  # experts 2 and 5 always tie
    c["wr"] = wr
    x = c["x"].copy()
    x[0] = 0  # token 0: every logit is exactly 0 -> experts 0 and 1, gates 1/2
    c["x"] = x
    r = _run(o, c)
    out, ids, gates, _ = _bf_case(c)
    assert r["ids"].tolist() == ids
    assert r["ids"][0].tolist() == [0, 1]
    assert r["gates"][0].tolist() == [0.5, 0.5]
    for t in range(T):
        row = r["ids"][t].tolist()
        for lo, hi in ((1, 4), (2, 5)):  # tie partners: the lower index is taken first
            if hi in row:
                assert lo in row and row.index(lo) < row.index(hi), (t, row)
    _close(r["gates"], gates)
    _close(r["out"], out, rtol=1e-11, atol=1e-12)
    # a bias that makes the tie partner strictly larger flips the choice
    c2 = dict(c)
    b = np.zeros(E, np.float32)
    b[4] = 1e-3
    c2["bias"] = b
    r2 = _run(o, c2)
    _, ids2, _, _ = _bf_case(c2)
    assert r2["ids"].tolist() == ids2


def pin_gates_sum_to_one_and_shift(o):
    """sum_j g_j = 1; adding one constant to every logit changes nothing."""
    c = tiny_case(32, 16, 8, 8, 2, seed=3)
    r = _run(o, c)
    assert np.all(np.abs(r["gates"].sum(1) - 1.0) <= 4e-16)
    assert np.all(r["gates"][:, 0] >= r["gates"][:, 1])
    c2 = dict(c)
    c2["bias"] = np.full(8, 0.375, np.float32)
    r2 = _run(o, c2)
    assert r2["ids"].tolist() == r["ids"].tolist()
    _close(r2["gates"], r["gates"], rtol=1e-12, atol=1e-14)


def pin_dense_e1k1(o):
    """E=1, k=1 is the dense SwiGLU FFN (torch fp64 on the CPU)."""
    T, d, ffn = 9, 24, 40
    c = tiny_case(T, d, ffn, 1, 1, seed=11)
    r = _run(o, c)
    x = torch.from_numpy(widen(c["x"]))
    w1 = torch.from_numpy(widen(c["w1"])[0])
    w3 = torch.from_numpy(widen(c["w3"])[0])
    w2 = torch.from_numpy(widen(c["w2"])[0])
    ref = (torch.nn.functional.silu(x @ w1.T) * (x @ w3.T)) @ w2.T
    assert np.all(r["ids"] == 0) and np.all(r["gates"] == 1.0)
    _close(r["out"], ref.numpy(), rtol=1e-12, atol=1e-13)


def pin_k_equals_e_mixture(o):
    """k = E: the softmax-weighted mixture over all experts (torch fp64)."""
    T, d, ffn, E = 6, 16, 12, 4
    c = tiny_case(T, d, ffn, E, E, seed=13, bias=[0.1, -0.2, 0.3, 0.0])
    r = _run(o, c)
    x = torch.from_numpy(widen(c["x"]))
    wr = torch.from_numpy(widen(c["wr"]))
    logits = x @ wr.T + torch.tensor(c["bias"], dtype=torch.float64)
    p = torch.softmax(logits, dim=-1)
    w1, w3, w2 = (torch.from_numpy(widen(c[n])) for n in ("w1", "w3", "w2"))
    ref = torch.zeros(T, d, dtype=torch.float64)
    for e in range(E):
        ye = (torch.nn.functional.silu(x @ w1[e].T) * (x @ w3[e].T)) @ w2[e].T
        ref += p[:, e:e + 1] * ye
    _close(r["out"], ref.numpy(), rtol=1e-11, atol=1e-13)


def pin_token_permutation(o):
    """out(P x) == P out(x), bit for bit."""
    c = tiny_case(24, 16, 12, 8, 2, seed=17)
    r = _run(o, c)
    P = np.random.default_rng(5).permutation(24)
    c2 = dict(c)
    c2["x"] = c["x"][P]
    r2 = _run(o, c2)
    assert np.array_equal(r2["out"], r["out"][P])
    assert np.array_equal(r2["ids"], r["ids"][P])
    assert np.array_equal(r2["gates"], r["gates"][P])


def pin_zeroed_expert(o):
    """Zeroing W1[e], W3[e] or W2[e] leaves routing unchanged and that slot adds exactly 0."""
    T, d, ffn, E, k = 20, 16, 12, 4, 2
    c = tiny_case(T, d, ffn, E, k, seed=19)
    r = _run(o, c)
    ids, gates = r["ids"], r["gates"]
    _, _, y = o.moe_apply(c["x"], c["w1"], c["w3"], c["w2"], ids, gates, want_slots=True)
    y = y.reshape(T, k, d)
    e0 = 2
    assert (ids == e0).any()
    for name in ("w1", "w3", "w2"):
        c2 = dict(c)
        w = c[name].copy()
        w[e0] = 0
        c2[name] = w
        r2 = _run(o, c2)
        assert np.array_equal(r2["ids"], ids) and np.array_equal(r2["gates"], gates)
        for t in range(T):
            exp_row = np.zeros(d)
            for j in range(k):
                if ids[t, j] != e0:
                    exp_row = exp_row + gates[t, j] * y[t, j]
            assert np.array_equal(r2["out"][t], exp_row), (name, t)


def pin_relabel_experts(o):
    """Permuting the experts (router rows with their weight stacks) changes nothing."""
    c = tiny_case(16, 16, 8, 6, 2, seed=23)
    r = _run(o, c)
    sigma = np.array([3, 0, 5, 1, 4, 2])
    c2 = dict(c)
    for n in ("wr", "w1", "w3", "w2"):
        c2[n] = c[n][sigma]
    r2 = _run(o, c2)
    inv = np.argsort(sigma)
    assert np.array_equal(sigma[r2["ids"]], r["ids"])
    assert np.array_equal(r2["out"], r["out"])
    del inv


def pin_scale_w2(o):
    """W2 -> 2 W2 doubles the output exactly; W2 -> -W2 negates it."""
    c = tiny_case(10, 16, 12, 4, 2, seed=29)
    r = _run(o, c)
    for s in (2.0, -1.0):
        c2 = dict(c)
        c2["w2"] = bits_of(widen(c["w2"]) * s)
        r2 = _run(o, c2)
        assert np.array_equal(r2["out"], s * r["out"])


def pin_one_hot_closed_form(o):
    """x = c e_i: u = c W1[:, i], v = c W3[:, i], logits = c Wr[:, i]."""
    T, d, ffn, E, k = 3, 8, 6, 4, 2
    c = tiny_case(T, d, ffn, E, k, seed=31)
    xs = np.zeros((T, d))
    cols = [1, 6, 3]
    scale = [2.0, -0.5, 1.0]
    for t in range(T):
        xs[t, cols[t]] = scale[t]
    c["x"] = bits_of(xs)
    r = _run(o, c)
    wr, w1, w3, w2 = (widen(c[n]) for n in ("wr", "w1", "w3", "w2"))
    for t in range(T):
        i, s = cols[t], scale[t]
        lg = s * wr[:, i]
        _close(r["logits"][t], lg, rtol=0, atol=0)
        order = sorted(range(E), key=lambda e: (-lg[e], e))[:k]
        assert r["ids"][t].tolist() == order
        ex = np.exp(lg[order] - lg[order[0]])
        g = ex / ex.sum()
        ref = np.zeros(d)
        for gj, e in zip(g, order):
            u = s * w1[e][:, i]
            v = s * w3[e][:, i]
            h = u / (1 + np.exp(-u)) * v
            ref += gj * (w2[e] @ h)
        _close(r["out"][t], ref, rtol=1e-12, atol=1e-15)


def pin_hand_example(o):
    """A hand-worked layer whose values are textbook constants (golden file)."""
    with open(os.path.join(GOLDEN, "hand_example.json")) as f:
        g = json.load(f)
    E, k = g["E"], g["k"]
    r = o.moe_layer(bits_of(np.array(g["x"])), bits_of(np.array(g["router_w"])),
                    bits_of(np.array(g["w1"])), bits_of(np.array(g["w3"])),
                    bits_of(np.array(g["w2"])), k,
                    None if g.get("router_bias") is None else np.array(g["router_bias"], np.float32))
    assert r["ids"].tolist() == g["expect_ids"]
    _close(r["logits"], g["expect_logits"], rtol=0, atol=0)
    _close(r["gates"], g["expect_gates"], rtol=1e-15, atol=1e-16)
    _close(r["out"], g["expect_out"], rtol=1e-14, atol=1e-16)
    del E


def pin_dispatch(o):
    """counts/offsets/perm equal a brute-force recount; perm is a permutation."""
    rng = np.random.default_rng(37)
    for T, E, k in [(0, 4, 2), (1, 1, 1), (9, 4, 2), (33, 8, 2), (17, 8, 3), (12, 5, 5)]:
        ids = np.stack([rng.permutation(E)[:k] for _ in range(T)]).astype(np.int32) \
            if T else np.zeros((0, k), np.int32)
        counts, offsets, perm = o.dispatch(ids, E)
        bc, bo, bp = bf.dispatch(ids.tolist(), E)
        assert counts.tolist() == bc and offsets.tolist() == bo and perm.tolist() == bp
        assert offsets[-1] == T * k
        assert sorted(perm.tolist()) == list(range(T * k))


def pin_rmsnorm(o):
    """RMSNorm: constant rows in closed form; random rows vs torch fp64."""
    d = 64
    for cval in (1e-3, 0.5, -3.0):
        h = np.full((1, d), cval, np.float32)
        gamma = bits_of(np.full(d, 1.5))
        eps = 1e-5
        a = o.rmsnorm(h, gamma, eps)
        c64 = float(np.float32(cval))
        ref = c64 / math.sqrt(c64 * c64 + eps) * 1.5
        _close(a, np.full((1, d), ref), rtol=1e-14, atol=0)
    rng = np.random.default_rng(41)
    h = rng.standard_normal((5, d)).astype(np.float32) * 3
    gamma = bits_of(np.round(rng.uniform(0.5, 1.5, d) * 64) / 64)  # k/64: exact in bf16
    a = o.rmsnorm(h, gamma, 1e-5)
    ref = torch.nn.functional.rms_norm(torch.from_numpy(h.astype(np.float64)), (d,),
                                       torch.from_numpy(widen(gamma)), eps=1e-5)
    _close(a, ref.numpy(), rtol=1e-13, atol=1e-15)


def pin_gates_for_ids(o):
    """Gates of a given expert choice: equal to the routed gates for the
    oracle's own choice, and to brute-force softmax values for another one."""
    c = tiny_case(12, 16, 8, 6, 3, seed=47)
    r = _run(o, c)
    g = o.gates_for_ids(r["logits"], r["ids"])
    assert np.array_equal(g, r["gates"])
    other = np.array([[5, 0, 2]] * 12, np.int32)
    g2 = o.gates_for_ids(r["logits"], other)
    for t in range(12):
        lg = r["logits"][t]
        ex = [math.exp(lg[e] - lg[5]) for e in (5, 0, 2)]
        ref = [v / sum(ex) for v in ex]
        _close(g2[t], ref, rtol=1e-14, atol=1e-16)


def pin_empty(o):
    """T = 0 is a valid, empty layer."""
    c = tiny_case(1, 8, 8, 4, 2, seed=43)
    c["x"] = c["x"][:0]
    r = _run(o, c)
    assert r["out"].shape == (0, 8) and r["ids"].shape == (0, 2)


def _fp8_torch(q):
    return torch.from_numpy(np.ascontiguousarray(q, np.uint8)).view(torch.float8_e4m3fn).to(torch.float64).numpy()


def pin_fp8_decode_table(o):
    """All 256 E4M3 bytes decode like torch's float8_e4m3fn (a library
    implementation of the OCP format), signs of zeros included."""
    codes = np.arange(256, dtype=np.uint8)
    got = o.fp8_e4m3(codes)
    ref = _fp8_torch(codes)
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(got), nan)
    assert np.array_equal(got[~nan], ref[~nan])
    assert np.array_equal(np.signbit(got[~nan]), np.signbit(ref[~nan]))


def pin_fp8_spec_values(o):
    """Values the OCP 8-bit floating point specification gives for E4M3: the
    smallest subnormal and normal, one, the largest finite value, NaN."""
    table = {0x00: 0.0, 0x01: 2.0 ** -9, 0x07: 7 * 2.0 ** -9, 0x08: 2.0 ** -6, 0x38: 1.0,
             0x39: 1.125, 0x7E: 448.0, 0xFE: -448.0, 0xB8: -1.0}
    codes = np.array(sorted(table), dtype=np.uint8)
    got = o.fp8_e4m3(codes)
    assert got.tolist() == [table[c] for c in sorted(table)]
    nz = o.fp8_e4m3(np.array([0x80, 0x7F, 0xFF], dtype=np.uint8))
    assert nz[0] == 0.0 and np.signbit(nz[0]) and np.isnan(nz[1]) and np.isnan(nz[2])


def _run_fp8(o, c):
    return o.moe_layer_fp8(c["x"], c["wr"], c["w1q"], c["w1s"], c["w3q"], c["w3s"], c["w2q"], c["w2s"],
                           c["k"], c["bias"])


def pin_fp8_layer_bruteforce(o):
    """The 8-bit layer == the brute force on weights dequantized by torch
    (decoded byte times the row's scale)."""
    for i, (T, d, ffn, E, k) in enumerate(TINY_SHAPES[:5]):
        c = tiny_case_fp8(T, d, ffn, E, k, seed=300 + i)
        deq = {n: (_fp8_torch(c[n + "q"]) * c[n + "s"].astype(np.float64)[..., None]).tolist()
               for n in ("w1", "w3", "w2")}
        out, ids, gates, logits = bf.moe_layer(_nested(c["x"]), _nested(c["wr"]), deq["w1"], deq["w3"],
                                               deq["w2"], k, None)
        r = _run_fp8(o, c)
        assert r["ids"].tolist() == ids
        _close(r["gates"], gates)
        _close(r["out"], out, rtol=1e-11, atol=1e-12)


def pin_fp8_row_scale(o):
    """Doubling the scale of W2 row i doubles output column i exactly and
    leaves the other columns unchanged."""
    c = tiny_case_fp8(6, 8, 12, 4, 2, seed=331)
    r = _run_fp8(o, c)
    c2 = dict(c)
    s2 = c["w2s"].copy()
    s2[:, 3] *= 2.0
    c2["w2s"] = s2
    r2 = _run_fp8(o, c2)
    assert np.array_equal(r2["out"][:, 3], 2.0 * r["out"][:, 3])
    keep = [i for i in range(8) if i != 3]
    assert np.array_equal(r2["out"][:, keep], r["out"][:, keep])


# ---- the decoder layer around the MoE block (one decode step) ---------------


def pin_round_bf16(o):
    """fp64 -> bf16 rounds to nearest, ties to even, in one step: float32
    values round like torch's float32 -> bfloat16 conversion (a library
    implementation), exact ties go to the even neighbour, and a value just
    above a tie rounds up (rounding through float32 first would land on the
    tie and round down)."""
    g = np.random.default_rng(501)
    f32 = np.concatenate([g.standard_normal(4000) * 10.0 ** g.integers(-40, 38, 4000),
                          g.standard_normal(500) * 1e-39]).astype(np.float32)
    f32 = f32[np.isfinite(f32) & (np.abs(f32) < 3e38)]
    ref = torch.from_numpy(f32).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(o.round_bf16(f32.astype(np.float64)), ref)
    one_ulp = 2.0 ** -7
    cases = [(1.0 + one_ulp / 2, 0x3F80), (1.0 + 1.5 * one_ulp, 0x3F82), (-(1.0 + one_ulp / 2), 0xBF80),
             (1.0 + one_ulp / 2 + 2.0 ** -40, 0x3F81), (3.0, 0x4040), (0.0, 0x0000), (-0.0, 0x8000),
             (2.0 ** -134, 0x0000), (1.5 * 2.0 ** -134, 0x0001), (3 * 2.0 ** -134, 0x0002)]
    got = o.round_bf16(np.array([x for x, _ in cases], dtype=np.float64))
    assert got.tolist() == [b for _, b in cases]


def pin_rope_closed_form(o):
    """RoPE of a unit vector e_i at position p is cos(p w_i) at i and
    sin(p w_i) at i + hd/2 with w_i = base^(-2i/hd) (the rotate-half pairing);
    position 0 is the identity; scores depend only on the position
    difference."""
    hd, base = 16, 10000.0
    for i in (0, 3, 7):
        for p in (1, 5, 1000):
            x = np.zeros((1, 1, hd))
            x[0, 0, i] = 1.0
            y = o.rope(x, [p], base)[0, 0]
            w = base ** (-2.0 * i / hd)
            want = np.zeros(hd)
            want[i], want[i + hd // 2] = math.cos(p * w), math.sin(p * w)
            _close(y, want, rtol=1e-14, atol=1e-15)
    g = np.random.default_rng(502)
    x = g.standard_normal((3, 2, hd))
    assert np.array_equal(o.rope(x, [0, 0, 0], base), x)
    q, k = g.standard_normal((1, 1, hd)), g.standard_normal((1, 1, hd))
    d1 = float(np.sum(o.rope(q, [9], base) * o.rope(k, [4], base)))
    d2 = float(np.sum(o.rope(q, [1009], base) * o.rope(k, [1004], base)))
    assert abs(d1 - d2) < 1e-12 * (1 + abs(d1))


def _randn_bits(g, shape, scale=1.0):
    """bf16 bit patterns of scaled normal draws (rounded by torch)."""
    x = torch.from_numpy((g.standard_normal(shape) * scale).astype(np.float32))
    return x.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


def _attn_case(g, T, Hq, Hkv, hd, page, npages, maxp, ctx):
    kc = _randn_bits(g, (npages, Hkv, page, hd))
    vc = _randn_bits(g, (npages, Hkv, page, hd))
    pt = np.stack([g.permutation(npages)[:maxp] for _ in range(T)]).astype(np.int32)
    q = g.standard_normal((T, Hq, hd))
    return q, kc, vc, pt, np.asarray(ctx, np.int32)


def _gather(cache, pt_row, L):
    page = cache.shape[2]
    return np.stack([widen(cache[pt_row[s // page], :, s % page, :]) for s in range(L)])  # [L, Hkv, hd]


def pin_attention_sdpa(o):
    """Paged decode attention with one query head per KV head equals torch's
    fp64 scaled_dot_product_attention on the gathered contiguous cache."""
    g = np.random.default_rng(503)
    T, H, hd, page = 3, 2, 8, 4
    q, kc, vc, pt, ctx = _attn_case(g, T, H, H, hd, page, 9, 4, [1, 7, 16])
    got = o.attention_decode(q, kc, vc, pt, ctx, 1 / math.sqrt(hd))
    for t in range(T):
        K = torch.from_numpy(_gather(kc, pt[t], ctx[t])).permute(1, 0, 2)  # [H, L, hd]
        V = torch.from_numpy(_gather(vc, pt[t], ctx[t])).permute(1, 0, 2)
        Q = torch.from_numpy(q[t][:, None, :])  # [H, 1, hd]
        ref = torch.nn.functional.scaled_dot_product_attention(Q, K, V)[:, 0, :].numpy()
        _close(got[t], ref, rtol=1e-12, atol=1e-13)


def pin_attention_gqa_and_pages(o):
    """Grouped heads: query head h reads KV head h // (Hq/Hkv), so GQA equals
    attention over a cache whose KV heads are repeated per query head.
    Relocating the pages (with the page table updated) changes nothing, one
    cached position returns its value row, and identical keys average the
    values."""
    g = np.random.default_rng(504)
    T, Hq, Hkv, hd, page, npages, maxp = 2, 8, 2, 8, 4, 10, 4
    q, kc, vc, pt, ctx = _attn_case(g, T, Hq, Hkv, hd, page, npages, maxp, [5, 13])
    sc = 1 / math.sqrt(hd)
    got = o.attention_decode(q, kc, vc, pt, ctx, sc)
    rep = np.repeat(np.arange(Hkv), Hq // Hkv)
    assert np.array_equal(got, o.attention_decode(q, kc[:, rep], vc[:, rep], pt, ctx, sc))
    perm = g.permutation(npages)
    inv = np.argsort(perm)
    kc2, vc2 = np.empty_like(kc), np.empty_like(vc)
    kc2[perm], vc2[perm] = kc, vc
    assert np.array_equal(got, o.attention_decode(q, kc2, vc2, perm[pt].astype(np.int32), ctx, sc))
    del inv
    one = o.attention_decode(q, kc, vc, pt, np.ones(T, np.int32), sc)
    for t in range(T):
        for h in range(Hq):
            assert np.array_equal(one[t, h], widen(vc[pt[t, 0], h // (Hq // Hkv), 0]))
    kc3 = kc.copy()
    kc3[...] = kc[0, 0, 0]
    avg = o.attention_decode(q, kc3, vc, pt, ctx, sc)
    for t in range(T):
        V = _gather(vc, pt[t], ctx[t])
        for h in range(Hq):
            _close(avg[t, h], V[:, h // (Hq // Hkv)].mean(axis=0), rtol=1e-13, atol=1e-14)


def _decoder_case(g, T=3, d=16, hq=4, hkv=2, hd=4, ffn=8, E=4, k=2, page=4, npages=10, maxp=3):
    def w(*shape):
        return _randn_bits(g, shape, 1 / math.sqrt(shape[-1]))

    def gamma():
        return torch.from_numpy(g.uniform(0.5, 1.5, d).astype(np.float32)).to(
            torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    c = {"h": g.standard_normal((T, d)).astype(np.float32),
         "gamma_attn": gamma(), "gamma_moe": gamma(),
         "wq": w(hq * hd, d), "wk": w(hkv * hd, d), "wv": w(hkv * hd, d), "wo": w(d, hq * hd),
         "k_cache": _randn_bits(g, (npages, hkv, page, hd)),
         "v_cache": _randn_bits(g, (npages, hkv, page, hd)),
         # every request owns its pages (the new entries are written)
         "page_table": g.permutation(npages)[:T * maxp].reshape(T, maxp).astype(np.int32),
         "pos": g.integers(0, maxp * page, T).astype(np.int32),
         "wr": w(E, d), "w1": w(E, ffn, d), "w3": w(E, ffn, d), "w2": w(E, d, ffn),
         "k": k, "hq": hq, "hkv": hkv, "theta": 1e6, "eps": 1e-5}
    return c


def _decoder(o, c):
    return o.decoder_layer(c["h"], c["gamma_attn"], c["wq"], c["wk"], c["wv"], c["wo"], c["k_cache"],
                           c["v_cache"], c["page_table"], c["pos"], c["gamma_moe"], c["wr"], c["w1"],
                           c["w3"], c["w2"], c["k"], c["hq"], c["hkv"], c["theta"], c["eps"])


def pin_decoder_layer_composition(o):
    """With Wo = 0 the attention block adds exactly nothing and the layer is
    the MoE residual block of the stack; at position 0 (nothing cached yet)
    the attention output of every query head is its KV head's new value row
    as stored (bf16), so the block adds Wo applied to those rows; the new
    key/value rows land in the cache at their request's position."""
    g = np.random.default_rng(505)
    c = _decoder_case(g)
    c0 = dict(c, wo=np.zeros(c["wo"].shape, np.uint16))
    r0 = _decoder(o, c0)
    assert np.array_equal(r0["h1"], c["h"].astype(np.float64))
    a2 = o.round_bf16(o.rmsnorm(c["h"], c["gamma_moe"], c["eps"]))
    moe = o.moe_layer(a2, c["wr"], c["w1"], c["w3"], c["w2"], c["k"])
    assert np.array_equal(r0["h2"], c["h"].astype(np.float64) + moe["out"])
    cp = dict(c, pos=np.zeros(3, np.int32))
    r = _decoder(o, cp)
    vrow = widen(o.round_bf16(r["v_new"]))  # [T, hkv, hd]
    grp = c["hq"] // c["hkv"]
    o_ref = np.stack([np.concatenate([vrow[t, h // grp] for h in range(c["hq"])]) for t in range(3)])
    assert np.array_equal(r["attn"].reshape(3, -1), o_ref)
    _close(r["h1"], c["h"].astype(np.float64) + o_ref @ widen(c["wo"]).T, rtol=1e-13, atol=1e-13)
    r = _decoder(o, c)
    page = c["k_cache"].shape[2]
    for t in range(3):
        pg, sl = c["page_table"][t, c["pos"][t] // page], c["pos"][t] % page
        assert np.array_equal(r["k_cache"][pg, :, sl], o.round_bf16(r["k_new"][t]))
        assert np.array_equal(r["v_cache"][pg, :, sl], o.round_bf16(r["v_new"][t]))


ALL_PINS = [
    pin_bruteforce_random,
    pin_bruteforce_ties,
    pin_gates_sum_to_one_and_shift,
    pin_dense_e1k1,
    pin_k_equals_e_mixture,
    pin_token_permutation,
    pin_zeroed_expert,
    pin_relabel_experts,
    pin_scale_w2,
    pin_one_hot_closed_form,
    pin_hand_example,
    pin_dispatch,
    pin_rmsnorm,
    pin_gates_for_ids,
    pin_empty,
    pin_fp8_decode_table,
    pin_fp8_spec_values,
    pin_fp8_layer_bruteforce,
    pin_fp8_row_scale,
    pin_round_bf16,
    pin_rope_closed_form,
    pin_attention_sdpa,
    pin_attention_gqa_and_pages,
    pin_decoder_layer_composition,
]
