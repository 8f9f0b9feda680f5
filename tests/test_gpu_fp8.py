"""GPU parity of the 8-bit expert weight path (E4M3 bytes, one f32 scale per
weight row; Sec. 4.1 "Model Quantization", Sec. 5's 8-bit Mixtral) against
the fp64 oracle on the same bytes and scales.

The kernels convert each E4M3 byte exactly to a bf16 operand and scale each
row's f32 sum, so the error budget is that of the bf16 path: the same
row-wise relative tolerance and routing rule apply."""

import numpy as np
import pytest
import torch

from gpu_common import (DEV, bf16_to_f64, fp8_small_case, fp8_workload_case, full_logits,
                        full_reference, gpu_forward_fp8, gpu_route, orc, oracle_out_fp8,
                        random_large_shapes, random_shapes, say, tile_cover_rows)
from parity import OUT_TOL, check_routing, rowwise_rel
from paper_2408_00008_amd import binding as B

pytestmark = pytest.mark.gpu


def _forward_check(c, rows=None):
    out = gpu_forward_fp8(c)
    ids, *_ = gpu_route(c)
    g_ids = ids.cpu().numpy()
    if rows is None:
        rows = np.arange(c.T)
        logits = full_logits(c, fp8=True)
        check_routing(g_ids, logits, c.k)
        ref, _ = full_reference(c, g_ids, fp8=True)
    else:
        rows = np.asarray(rows)
        ref, logits, *_ = oracle_out_fp8(c, rows, g_ids[rows])
        check_routing(g_ids[rows], logits, c.k)
    err = rowwise_rel(bf16_to_f64(out)[rows], ref)
    say(f"  {c.name} T={c.T}: rowwise rel {err:.3e} over {len(rows)} tokens")
    assert err < OUT_TOL
    return out


@pytest.mark.parametrize("shape", [(16, 256, 512, 8, 2), "decode_t64_fp8",
                                   (600, 256, 512, 8, 2)])
def test_fp8_stages_teacher_forced(shape):
    """up/down fed the oracle's routing; h and y compared slot by slot, with
    and without the fused gather and the fused gate-weighted scatter."""
    c = fp8_workload_case(shape) if isinstance(shape, str) else fp8_small_case(*shape, seed=3)
    say(f"[fp8 stages] {c.name}")
    o = orc()
    x = c.host("x")
    logits = o.router_logits(x, c.host("router_w"), c.bias_np)
    ids, gates = o.topk_gate(logits, c.k)
    _, offs, perm = o.dispatch(ids, c.E)
    _, h_ref, y_ref = o.moe_apply_fp8(x, *c.weights(), ids, gates, want_slots=True)
    A = c.T * c.k
    d_offs = torch.from_numpy(offs).to(DEV)
    d_perm = torch.from_numpy(perm).to(DEV)
    d_gw = torch.from_numpy(gates.astype(np.float32).reshape(-1)).to(DEV)
    h = torch.empty(A, c.ffn, dtype=torch.bfloat16, device=DEV)
    B.moe_swiglu_up_fp8(c.x, d_offs, c.w1q, c.w1s, c.w3q, c.w3s, c.T, c.k, h, perm=d_perm)
    xp = torch.empty(A, c.d, dtype=torch.bfloat16, device=DEV)
    B.moe_permute(c.x, d_perm, c.k, xp)
    h_np = torch.empty_like(h)
    B.moe_swiglu_up_fp8(xp, d_offs, c.w1q, c.w1s, c.w3q, c.w3s, c.T, c.k, h_np)
    y = torch.empty(A, c.d, dtype=torch.float32, device=DEV)
    B.moe_swiglu_down_fp8(h, d_offs, c.w2q, c.w2s, c.T, c.k, y, topk_w=d_gw, perm=d_perm)
    y_plain = torch.empty_like(y)
    B.moe_swiglu_down_fp8(h, d_offs, c.w2q, c.w2s, c.T, c.k, y_plain)
    torch.cuda.synchronize()
    # the gathered and the pre-permuted token rows are the same bits
    assert torch.equal(h, h_np)
    e_h = rowwise_rel(bf16_to_f64(h), h_ref[perm])
    e_y = rowwise_rel(y.cpu().numpy(), y_ref * gates.reshape(-1, 1))
    e_yp = rowwise_rel(y_plain.cpu().numpy(), y_ref[perm])
    say(f"  rowwise rel: h {e_h:.2e} y {e_y:.2e} y_plain {e_yp:.2e}")
    assert e_h < OUT_TOL and e_y < OUT_TOL and e_yp < OUT_TOL


@pytest.mark.parametrize("name", ["decode_t64_fp8", "decode_t256_skew_fp8", "prefill_t4096_fp8",
                                  "mixed_t576_fp8"])
def test_fp8_forward_full(name):
    """Every token of each 8-bit workload the benchmark runs."""
    say(f"[fp8 forward] {name} (every token)")
    c = fp8_workload_case(name)
    _forward_check(c)
    del c
    torch.cuda.empty_cache()


@pytest.mark.parametrize("shape", [
    (1, 64, 64, 1, 1),        # single token, single expert
    (37, 192, 320, 8, 2),     # ragged T, d/ffn not multiples of 128
    (5, 128, 128, 4, 4),      # k = E
    (300, 128, 192, 64, 8),   # E = 64, k = 8 limits
    (513, 256, 512, 8, 2),    # rows per expert > 64
    (200, 256, 256, 8, 2),    # 33..64 rows per expert
    (96, 1024, 512, 8, 2),    # several 256-element chunks per row (rotated starts)
])
def test_fp8_forward_shapes(shape):
    say(f"[fp8 forward] shape {shape}")
    _forward_check(fp8_small_case(*shape, seed=13))


@pytest.mark.parametrize("shape", [
    (600, 512, 1024, 8, 2),   # tiled: 2 weight blocks, down cut in 2 parts
    (1000, 512, 384, 8, 2),   # tiled: odd count of 128-column output blocks
    (288, 256, 2048, 8, 2),   # tiled: one token tile per expert, down cut in 4 parts
    (700, 256, 256, 4, 2),    # tiled: several ragged 256-row token tiles per expert
])
def test_fp8_forward_tiled_shapes(shape):
    """Above 64 rows per expert the 8-bit weights take the tiled kernels (E4M3
    bytes staged in LDS, widened to bf16 at the fragment reads, row scales in
    the epilogue)."""
    say(f"[fp8 forward] tiled shape {shape}")
    c = fp8_small_case(*shape, seed=14)
    assert B.moe_gemm_variant_for(c.T, c.d, c.ffn, c.E, c.k) == 2
    _forward_check(c)


@pytest.mark.parametrize("shape", random_shapes(10, seed=2409), ids=lambda s: "x".join(map(str, s)))
def test_fp8_forward_random_shapes(shape):
    """The automatic kernel choice with 8-bit weights on seeded random shapes,
    every token against the oracle."""
    say(f"[fp8 forward] random shape {shape} (auto: {B.moe_gemm_variant_for(*shape)})")
    _forward_check(fp8_small_case(*shape, seed=32))


@pytest.mark.parametrize("shape", random_large_shapes(8, seed=2410), ids=lambda s: "x".join(map(str, s)))
def test_fp8_forward_random_large_shapes(shape):
    """8-bit weights on seeded larger layers (skewed routing on every other
    draw): every kernel family on tokens that cover every (expert, 256-row
    tile) work item, then moe_forward_fp8_ex with the caller's workspace,
    twice for the same bits."""
    T, d, ffn, E, k, hot = shape
    bias = None
    if hot >= 0:
        bias = [0.0] * E
        bias[hot] = 2.0
    say(f"[fp8 forward] large random shape {shape}")
    c = fp8_small_case(T, d, ffn, E, k, seed=38, bias=bias)
    ids, *_ = gpu_route(c)
    g_ids = ids.cpu().numpy()
    rows = tile_cover_rows(g_ids, k, E, seed=7)
    if len(rows) > 96:
        pick = np.random.default_rng(8).choice(rows, 96, replace=False)
        rows = np.array(sorted(set(pick.tolist()) | {0, T - 1}))
    ref, logits, *_ = oracle_out_fp8(c, rows, g_ids[rows])
    check_routing(g_ids[rows], logits, k)
    for variant in (0, 1, 2):
        prev = B.moe_set_gemm_variant(variant)
        try:
            out = gpu_forward_fp8(c)
        finally:
            B.moe_set_gemm_variant(prev)
        err = rowwise_rel(bf16_to_f64(out)[rows], ref)
        say(f"  variant {variant}: rowwise rel {err:.3e} over {len(rows)} tokens")
        assert err < OUT_TOL
    ws = torch.empty(B.moe_workspace_size(T, d, ffn, E, k), dtype=torch.uint8, device=DEV)
    outs = []
    for _ in range(2):
        of = torch.empty(T, d, dtype=torch.float32, device=DEV)
        B.moe_forward_fp8_ex(c.x, c.router_w, c.w1q, c.w1s, c.w3q, c.w3s, c.w2q, c.w2s, k,
                             out_f32=of, router_bias=c.router_bias, workspace=ws)
        outs.append(of)
    torch.cuda.synchronize()
    err = rowwise_rel(outs[0].double().cpu().numpy()[rows], ref)
    say(f"  forward_fp8_ex with workspace: rowwise rel {err:.3e}")
    assert err < OUT_TOL
    assert torch.equal(outs[0], outs[1])


@pytest.mark.parametrize("shape,bias", [
    ((288, 256, 2048, 8, 2), None),                 # tiled, down cut into 4 parts
    ((256, 256, 2048, 8, 2), [2.0] + [0.0] * 7),    # split: heavy expert tiled beside the rest
])
def test_fp8_forward_graph_replays(shape, bias):
    """8-bit weights: graph replays of the step (with the workspace cleared in
    between) give the bits of the eager runs, which match the oracle."""
    say(f"[fp8 forward] graph capture {shape}")
    c = fp8_small_case(*shape, seed=39, bias=bias)
    _forward_check(c)
    T, d, k = c.T, c.d, c.k
    ws = torch.empty(B.moe_workspace_size(T, d, c.ffn, c.E, k), dtype=torch.uint8, device=DEV)
    outs = [torch.empty(T, d, dtype=torch.float32, device=DEV) for _ in range(3)]

    def step(o, s):
        B.moe_forward_fp8_ex(c.x, c.router_w, c.w1q, c.w1s, c.w3q, c.w3s, c.w2q, c.w2s, k,
                             out_f32=o, router_bias=c.router_bias, workspace=ws, stream=s)

    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        step(outs[0], s)
        step(outs[1], s)
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    assert torch.equal(outs[0], outs[1])
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        step(outs[2], s)
    for rep in range(3):
        outs[2].fill_(7.0)
        ws.zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(outs[2], outs[0]), rep


@pytest.mark.parametrize("shape,bias0", [
    ((288, 256, 2048, 8, 2), None),   # tiled: down cut in 4 parts, summed by the combine
    ((256, 256, 2048, 8, 2), 2.0),    # split step: heavy expert cut in 2 parts, folded
])
def test_fp8_down_parts_pair_equals_forward(shape, bias0):
    """moe_swiglu_down_parts_fp8 + moe_combine_parts, fed the forward's own
    routing and h, reproduce moe_forward_fp8_ex bitwise."""
    say(f"[fp8] parts pair {shape}")
    bias = None if bias0 is None else [bias0] + [0.0] * (shape[3] - 1)
    c = fp8_small_case(*shape, seed=15, bias=bias)
    T, d, k = c.T, c.d, c.k
    _, of = gpu_forward_fp8(c, out_f32=True)
    ids, gw, offs, perm, _ = gpu_route(c)
    h = torch.empty(T * k, c.ffn, dtype=torch.bfloat16, device=DEV)
    B.moe_swiglu_up_fp8(c.x, offs, c.w1q, c.w1s, c.w3q, c.w3s, T, k, h, perm=perm)
    slices = 4 if bias0 is None else 2  # the forward's caps in the two regimes
    y = torch.empty(slices, T * k, d, dtype=torch.float32, device=DEV)
    parts = torch.zeros(1, dtype=torch.int32, device=DEV)
    B.moe_swiglu_down_parts_fp8(h, offs, c.w2q, c.w2s, T, k, y, parts, topk_w=gw, perm=perm)
    st = torch.empty(T, d, dtype=torch.float32, device=DEV)
    B.moe_combine_parts(y, parts, T, d, k, out_f32=st)
    torch.cuda.synchronize()
    assert int(parts.item()) == (4 if bias0 is None else 1)
    assert torch.equal(st, of)


def test_fp8_forward_heavy_expert():
    """Every token on expert 0: more passes than a slab has pass slots."""
    say("[fp8 forward] heavy expert")
    c = fp8_small_case(700, 256, 256, 4, 2, seed=21, bias=[60.0, 0.0, 0.0, 0.0])
    _, _, offs, _, _ = gpu_route(c)
    o = offs.cpu().numpy()
    assert o[1] - o[0] == c.T
    _forward_check(c)


def test_fp8_deterministic():
    c = fp8_small_case(64, 512, 512, 8, 2, seed=5)
    a = gpu_forward_fp8(c)
    b = gpu_forward_fp8(c)
    assert torch.equal(a, b)


def test_fp8_nan_byte_reaches_only_its_expert():
    """An E4M3 NaN byte in one w1 row of expert e turns exactly the tokens
    routed to e into NaN; every other token still matches the oracle."""
    say("[fp8] NaN byte")
    c = fp8_small_case(48, 128, 256, 8, 2, seed=9)
    ids, *_ = gpu_route(c)
    g_ids = ids.cpu().numpy()
    e = int(np.bincount(g_ids.reshape(-1), minlength=c.E).argmax())
    c.w1q[e, 7, 33] = 0x7F
    c._host.pop("w1q", None)
    out = gpu_forward_fp8(c).float().cpu().numpy()
    hit = (g_ids == e).any(axis=1)
    assert hit.any() and (~hit).any()
    assert np.isnan(out[hit]).all()
    rows = np.nonzero(~hit)[0]
    assert np.isfinite(out[rows]).all()
    ref, *_ = oracle_out_fp8(c, rows, g_ids[rows])
    assert rowwise_rel(out[rows].astype(np.float64), ref) < OUT_TOL


def test_fp8_t0():
    c = fp8_small_case(3, 64, 64, 4, 2)
    out = torch.zeros(0, 64, dtype=torch.bfloat16, device=DEV)
    B.moe_forward_fp8_ex(c.x[:0], c.router_w, c.w1q, c.w1s, c.w3q, c.w3s, c.w2q, c.w2s, 2, out=out)
    torch.cuda.synchronize()
