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
  the brute force fed with weights dequantized by torch.
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
]
