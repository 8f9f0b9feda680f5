"""GPU path (through the C ABI) against the fp64 oracle on the same bits."""

import numpy as np
import pytest
import torch

from gpu_common import (DEV, bf16_to_f64, full_logits, full_reference, gpu_forward, gpu_route,
                        oracle_logits, oracle_out, orc, random_large_shapes, random_shapes, say,
                        small_case,
                        tile_cover_rows, workload_case)
from parity import OUT_TOL, check_routing, rowwise_rel
from paper_2408_00008_amd import binding as B
from paper_2408_00008_amd import inputs

pytestmark = pytest.mark.gpu

_cases = {}


def wl(name):
    if name not in _cases:
        say(f"[gen] {name}")
        _cases[name] = workload_case(name)
    return _cases[name]


def _route_checks(c, sample=None):
    ids, gw, offs, perm, logits = gpu_route(c)
    rows = np.arange(c.T) if sample is None else sample
    ref_logits = oracle_logits(c, rows)
    g_ids = ids.cpu().numpy()
    amb = check_routing(g_ids[rows], ref_logits, c.k)
    # f32 logits against f64: relative to the row's logit scale
    gl = logits.cpu().numpy().astype(np.float64)[rows]
    scale = np.abs(ref_logits).max(axis=1, keepdims=True) + 1e-30
    assert np.max(np.abs(gl - ref_logits) / scale) < 1e-5
    # gates: the softmax over the GPU's own f32 logits of its selected
    # experts, evaluated in f64, must match to a few f32 rounding units.  The
    # GPU subtracts the largest selected logit in f32 (rounding relative to
    # the gap), takes exp and sums k terms in f32 and divides: the bound is
    # (6 + k + 2 * gap) units of 2^-24 relative to the gate, gap the largest
    # logit difference inside the token's selection.
    sel = np.take_along_axis(gl, g_ids[rows].astype(np.int64), axis=1)
    shift = sel - sel[:, :1]
    ex = np.exp(shift)
    ref_g = ex / ex.sum(axis=1, keepdims=True)
    gap = np.abs(shift).max(axis=1, keepdims=True)
    got_g = gw.cpu().numpy().astype(np.float64)[rows]
    units = np.abs(got_g - ref_g) / (ref_g * 2.0 ** -24)
    say(f"  gates: max error {units.max():.2f} units of 2^-24 (bound {6 + c.k} + 2 * gap)")
    assert np.all(units <= 6 + c.k + 2 * gap)
    # and against the oracle's own f64 logits (the f32 logit error enters here)
    ref_o = orc().gates_for_ids(ref_logits, g_ids[rows])
    assert np.max(np.abs(got_g - ref_o)) < 2e-5
    assert np.all(np.abs(gw.cpu().numpy().sum(1) - 1.0) < 4e-7)
    # dispatch: exact integers, recomputed by the oracle from the GPU's ids
    _, r_off, r_perm = orc().dispatch(g_ids, c.E)
    assert np.array_equal(offs.cpu().numpy(), r_off)
    assert np.array_equal(perm.cpu().numpy(), r_perm)
    return amb, g_ids


@pytest.mark.parametrize("name", ["tiny_t16", "decode_t64", "decode_t256_skew", "prefill_t4096",
                                  "mixed_t576", "decode_t64_tp8"])
def test_route(name):
    say(f"[route] {name}")
    c = wl(name)
    amb, _ = _route_checks(c)
    say(f"  ambiguous tokens: {int(amb.sum())} of {c.T}")
    assert amb.sum() <= max(2, c.T // 500)


@pytest.mark.parametrize("shape", [(1, 64, 64, 1, 1), (37, 192, 320, 8, 2), (5, 128, 128, 4, 4),
                                   (300, 64, 128, 64, 8), (129, 256, 64, 3, 2),
                                   # several tokens per router workgroup (T >= 256 * 64 / E),
                                   # with a partial last pass
                                   (2053, 256, 64, 8, 2), (1029, 512, 64, 16, 4),
                                   (515, 4096, 64, 32, 8), (2051, 128, 64, 5, 3)])
def test_route_shapes(shape):
    say(f"[route] shape {shape}")
    c = small_case(*shape, seed=5)
    _route_checks(c)


def test_route_tokens_per_workgroup_bitwise():
    """Long inputs put several tokens in one router workgroup; the logits,
    ids and gates of a token do not depend on that: routing the first 300
    tokens alone (one per workgroup) gives the same bits."""
    say("[route] tokens per workgroup")
    c = small_case(2053, 512, 64, 8, 2, seed=6)
    ids, gw, _, _, logits = gpu_route(c)
    c2 = c.with_x(c.x[:300].contiguous())
    ids2, gw2, _, _, logits2 = gpu_route(c2)
    assert torch.equal(logits[:300], logits2) and torch.equal(ids[:300], ids2)
    assert torch.equal(gw[:300], gw2)


def test_route_ties_lower_index():
    """Experts with identical router rows tie exactly: the lower index wins."""
    say("[route] ties")
    c = small_case(64, 128, 128, 8, 2, seed=9)
    rw = c.router_w.clone()
    rw[5] = rw[1]
    rw[7] = rw[0]
    c.router_w = rw
    c._bits.pop("router_w", None)
    ids, _, _, _, logits = gpu_route(c)
    ids = ids.cpu().numpy()
    ref_ids, _ = orc().topk_gate(oracle_logits(c), 2)
    for t in range(c.T):
        row = ids[t].tolist()
        for lo, hi in ((1, 5), (0, 7)):
            if hi in row:
                assert lo in row and row.index(lo) < row.index(hi)
    check_routing(ids, oracle_logits(c), 2)
    del ref_ids


def test_permute_bitwise():
    say("[permute]")
    c = small_case(37, 192, 64, 8, 2, seed=3)
    ids, gw, offs, perm, _ = gpu_route(c)
    xp = torch.empty(c.T * c.k, c.d, dtype=torch.bfloat16, device=DEV)
    B.moe_permute(c.x, perm, c.k, xp)
    torch.cuda.synchronize()
    ref = c.bits("x")[perm.cpu().numpy() // c.k]
    assert np.array_equal(inputs.bf16_bits(xp), ref)


@pytest.mark.parametrize("name", ["tiny_t16", "decode_t64"])
@pytest.mark.parametrize("variant", [1, 2])
def test_stages_teacher_forced(name, variant):
    """up/down/combine fed the oracle's routing, compared stage by stage."""
    say(f"[stages] {name} variant {variant}")
    c = wl(name)
    o = orc()
    x = c.bits("x")
    logits = o.router_logits(x, c.bits("router_w"), c.bias_np)
    ids, gates = o.topk_gate(logits, c.k)
    _, offs, perm = o.dispatch(ids, c.E)
    out_ref, h_ref, y_ref = o.moe_apply(x, c.bits("w1"), c.bits("w3"), c.bits("w2"), ids, gates,
                                        want_slots=True)
    A = c.T * c.k
    d_offs = torch.from_numpy(offs).to(DEV)
    d_perm = torch.from_numpy(perm).to(DEV)
    d_gw = torch.from_numpy(gates.astype(np.float32).reshape(-1)).to(DEV)
    xp = torch.empty(A, c.d, dtype=torch.bfloat16, device=DEV)
    B.moe_permute(c.x, d_perm, c.k, xp)
    h = torch.empty(A, c.ffn, dtype=torch.bfloat16, device=DEV)
    y = torch.empty(A, c.d, dtype=torch.float32, device=DEV)
    prev = B.moe_set_gemm_variant(variant)
    try:
        B.moe_swiglu_up(xp, d_offs, c.w1, c.w3, c.T, c.k, h)
        B.moe_swiglu_down(h, d_offs, c.w2, c.T, c.k, y, topk_w=d_gw, perm=d_perm)
        y_plain = torch.empty_like(y)
        B.moe_swiglu_down(h, d_offs, c.w2, c.T, c.k, y_plain)
    finally:
        B.moe_set_gemm_variant(prev)
    out = torch.empty(c.T, c.d, dtype=torch.bfloat16, device=DEV)
    B.moe_combine(y, c.T, c.d, c.k, out=out)
    torch.cuda.synchronize()
    # h rows are in permuted order r; the oracle's are in assignment order a = perm[r]
    e_h = rowwise_rel(bf16_to_f64(h), h_ref[perm])
    e_y = rowwise_rel(y.cpu().numpy(), y_ref * gates.reshape(-1, 1))
    e_yp = rowwise_rel(y_plain.cpu().numpy(), y_ref[perm])
    e_o = rowwise_rel(bf16_to_f64(out), out_ref)
    say(f"  rowwise rel: h {e_h:.2e} y {e_y:.2e} y_plain {e_yp:.2e} out {e_o:.2e}")
    assert e_h < OUT_TOL and e_y < OUT_TOL and e_yp < OUT_TOL and e_o < OUT_TOL


def _forward_check(c, rows=None, variant=None):
    out = gpu_forward(c, variant)
    ids, *_ = gpu_route(c)
    g_ids = ids.cpu().numpy()
    if rows is None:
        # every token, against the oracle output cached for this case
        ref_logits = full_logits(c)
        check_routing(g_ids, ref_logits, c.k)
        ref, _ = full_reference(c, g_ids)
        rows = np.arange(c.T)
    else:
        rows = np.asarray(rows)
        ref_logits = oracle_logits(c, rows)
        check_routing(g_ids[rows], ref_logits, c.k)
        ref, *_ = oracle_out(c, rows, g_ids[rows])
    err = rowwise_rel(bf16_to_f64(out)[rows], ref)
    say(f"  {c.name} T={c.T} variant={variant}: rowwise rel {err:.3e} over {len(rows)} tokens")
    assert err < OUT_TOL
    return out


# Every token of every workload the benchmark runs, under the automatic
# kernel choice (0) and with every expert GEMM on the weight-streaming kernel
# (1); the oracle output of a workload is computed once for both.
@pytest.mark.parametrize("name", ["tiny_t16", "decode_t64", "decode_t256_skew", "prefill_t4096",
                                  "mixed_t576", "decode_t64_tp8"])
@pytest.mark.parametrize("variant", [0, 1])
def test_forward_full(name, variant):
    say(f"[forward] {name} variant {variant} (every token)")
    _forward_check(wl(name), variant=variant)


@pytest.mark.parametrize("shape", [
    (1, 64, 64, 1, 1),        # single token, single expert
    (37, 192, 320, 8, 2),     # ragged T, d/ffn not multiples of 128
    (5, 128, 128, 4, 4),      # k = E: every expert on every token
    (200, 64, 128, 16, 2),    # many experts, several tiles of rows
    (300, 128, 192, 64, 8),   # E = 64, k = 8 limits
    (513, 256, 512, 8, 2),    # rows per expert > 64
    (700, 256, 256, 4, 2),    # several ragged 256-row token tiles per expert
    (1000, 512, 384, 8, 2),   # odd count of 128-column output blocks
    (96, 256, 128, 64, 8),    # E = 64 with 1..20 rows per expert
    (200, 256, 256, 8, 2),    # 33..64 rows per expert (partial tiles of every width)
])
@pytest.mark.parametrize("variant", [1, 2])
def test_forward_shapes(shape, variant):
    say(f"[forward] shape {shape} variant {variant}")
    _forward_check(small_case(*shape, seed=13), variant=variant)


@pytest.mark.parametrize("shape", random_shapes(), ids=lambda s: "x".join(map(str, s)))
def test_forward_random_shapes(shape):
    """The automatic kernel choice (streaming, split by rows, tiled with a
    cut reduction) on seeded random shapes, every token against the oracle."""
    say(f"[forward] random shape {shape} (auto: {B.moe_gemm_variant_for(*shape)})")
    _forward_check(small_case(*shape, seed=31), variant=0)


@pytest.mark.parametrize("shape", random_large_shapes(), ids=lambda s: "x".join(map(str, s)))
def test_forward_random_large_shapes(shape):
    """Seeded larger layers (up to 6000 tokens, skewed routing on every other
    draw), every kernel family, on tokens that cover every (expert, 256-row
    tile) work item; then moe_forward_ex with the caller's workspace (where
    the down GEMM may cut its reduction or split its last tiles) against the
    same oracle rows, and twice for the same bits."""
    T, d, ffn, E, k, hot = shape
    bias = None
    if hot >= 0:
        bias = [0.0] * E
        bias[hot] = 2.0
    say(f"[forward] large random shape {shape} (auto: {B.moe_gemm_variant_for(T, d, ffn, E, k)})")
    c = small_case(T, d, ffn, E, k, seed=37, bias=bias)
    ids, *_ = gpu_route(c)
    g_ids = ids.cpu().numpy()
    rows = tile_cover_rows(g_ids, k, E, seed=5)
    if len(rows) > 96:
        pick = np.random.default_rng(6).choice(rows, 96, replace=False)
        rows = np.array(sorted(set(pick.tolist()) | {0, T - 1}))
    check_routing(g_ids[rows], oracle_logits(c, rows), k)
    ref, *_ = oracle_out(c, rows, g_ids[rows])
    for variant in (0, 1, 2):
        err = rowwise_rel(bf16_to_f64(gpu_forward(c, variant))[rows], ref)
        say(f"  variant {variant}: rowwise rel {err:.3e} over {len(rows)} tokens")
        assert err < OUT_TOL
    ws = torch.empty(B.moe_workspace_size(T, d, ffn, E, k), dtype=torch.uint8, device=DEV)
    outs = []
    for _ in range(2):
        of = torch.empty(T, d, dtype=torch.float32, device=DEV)
        B.moe_forward_ex(c.x, c.router_w, c.w1, c.w3, c.w2, k, out_f32=of,
                         router_bias=c.router_bias, workspace=ws)
        outs.append(of)
    torch.cuda.synchronize()
    err = rowwise_rel(outs[0].double().cpu().numpy()[rows], ref)
    say(f"  forward_ex with workspace: rowwise rel {err:.3e}")
    assert err < OUT_TOL
    assert torch.equal(outs[0], outs[1])


def test_forward_empty_experts():
    """A bias that sends every token to experts 2 and 5 leaves the rest idle."""
    say("[forward] empty experts")
    bias = [0.0] * 8
    bias[2], bias[5] = 50.0, 40.0
    c = small_case(48, 128, 256, 8, 2, seed=17, bias=bias)
    ids, _, offs, _, _ = gpu_route(c)
    o = offs.cpu().numpy()
    assert (np.diff(o) > 0).sum() == 2
    _forward_check(c)


@pytest.mark.parametrize("variant", [1, 2])
def test_forward_heavy_expert(variant):
    """A bias that sends every token to expert 0 (and one other): expert 0
    takes all T rows, more passes than a slab has pass slots, so slots loop."""
    say(f"[forward] heavy expert variant {variant}")
    bias = [60.0, 0.0, 0.0, 0.0]
    c = small_case(700, 256, 256, 4, 2, seed=21, bias=bias)
    ids, _, offs, _, _ = gpu_route(c)
    o = offs.cpu().numpy()
    assert o[1] - o[0] == c.T
    _forward_check(c, variant=variant)


@pytest.mark.parametrize("shape", [
    (256, 256, 512, 8, 2),    # heavy experts take the tiled up kernel
    (256, 192, 320, 8, 2),    # no tiled shape: heavy experts stream in 128-row passes
    (130, 128, 256, 4, 1),    # k = 1, T just above 64
])
def test_forward_split_by_rows(shape):
    """Automatic choice in the streaming regime with T > 64: a +2 logit bias
    gives expert 0 more than 64 rows and the rest fewer, so each expert GEMM
    runs as two launches split on the device by rows per expert."""
    say(f"[forward] split by rows {shape}")
    bias = [2.0] + [0.0] * (shape[3] - 1)
    c = small_case(*shape, seed=23, bias=bias)
    assert B.moe_gemm_variant_for(c.T, c.d, c.ffn, c.E, c.k) == 3
    _, _, offs, _, _ = gpu_route(c)
    rows = np.diff(offs.cpu().numpy())
    assert rows.max() > 64 and (rows[rows > 0] <= 64).any(), rows
    _forward_check(c, variant=0)


@pytest.mark.parametrize("shape,parts", [
    ((288, 256, 2048, 8, 2), 4),   # one token tile per expert, 4 parts of 8 steps
    ((600, 512, 1024, 8, 2), 2),   # 2 weight blocks per expert, 2 parts of 8 steps
    ((600, 256, 2048, 64, 8), None),  # E = 64, k = 8: 64 ragged tiles (count not pinned)
    # slices large enough for the tail split: tiles uncut (count 1); the
    # tiles past the grid's whole rounds are cut into pieces over all the
    # workgroups and folded back into slice 0.  96 tiles, no whole round:
    # every tile in 2 pieces
    ((3000, 1024, 2048, 8, 2), 1),
    # 320 tiles: one whole round, the 64 left in 4 pieces each
    ((4800, 2048, 2048, 8, 2), 1),
    # 192 tiles, no whole round and more than half the grid: uncut, no pieces
    ((6000, 1024, 2048, 8, 2), 1),
    # E = 64, k = 8, ~256 rows per expert: many experts' short last tiles
    # ordered after the full ones, two whole rounds, the rest split
    ((2048, 1024, 1024, 64, 8), 1),
])
def test_forward_down_split(shape, parts):
    """Prefill-regime sizes with few token tiles: the tiled down GEMM cuts its
    reduction into parts written as separate f32 slices that the combine
    sums.  Parity with the oracle; the part count the kernel chose (the int
    in the last 256 bytes of the forward's workspace); and agreement with the
    staged calls, which run the same GEMM uncut."""
    say(f"[forward] down reduction split {shape}")
    c = small_case(*shape, seed=29)
    assert B.moe_gemm_variant_for(c.T, c.d, c.ffn, c.E, c.k) == 2
    _forward_check(c, variant=0)
    T, d, k = c.T, c.d, c.k
    ws = torch.empty(B.moe_workspace_size(T, d, c.ffn, c.E, k), dtype=torch.uint8, device=DEV)
    of = torch.empty(T, d, dtype=torch.float32, device=DEV)
    B.moe_forward_ex(c.x, c.router_w, c.w1, c.w3, c.w2, k, out_f32=of, workspace=ws)
    torch.cuda.synchronize()
    used = int(ws[-256:].view(torch.int32)[0])
    assert used in (1, 2, 4) if parts is None else used == parts
    ids, gw, offs, perm, _ = gpu_route(c)
    xp = torch.empty(T * k, d, dtype=torch.bfloat16, device=DEV)
    B.moe_permute(c.x, perm, k, xp)
    h = torch.empty(T * k, c.ffn, dtype=torch.bfloat16, device=DEV)
    y = torch.empty(T * k, d, dtype=torch.float32, device=DEV)
    B.moe_grouped_swiglu(xp, offs, c.w1, c.w3, c.w2, T, k, h, y, topk_w=gw, perm=perm)
    staged = torch.empty(T, d, dtype=torch.float32, device=DEV)
    B.moe_combine(y, T, d, k, out_f32=staged)
    torch.cuda.synchronize()
    err = rowwise_rel(of.double().cpu().numpy(), staged.double().cpu().numpy())
    say(f"  forward (cut) vs staged (uncut): rowwise rel {err:.3e}")
    assert err < 1e-5
    # the staged pair that the forward runs gives the same bits
    yp = torch.empty(4, T * k, d, dtype=torch.float32, device=DEV)
    np_dev = torch.zeros(1, dtype=torch.int32, device=DEV)
    B.moe_swiglu_down_parts(h, offs, c.w2, T, k, yp, np_dev, topk_w=gw, perm=perm)
    st2 = torch.empty(T, d, dtype=torch.float32, device=DEV)
    B.moe_combine_parts(yp, np_dev, T, d, k, out_f32=st2)
    torch.cuda.synchronize()
    assert int(np_dev.item()) == used
    assert torch.equal(st2, of)
    # the same inputs give the same bits
    of2 = torch.empty_like(of)
    B.moe_forward_ex(c.x, c.router_w, c.w1, c.w3, c.w2, k, out_f32=of2, workspace=ws)
    torch.cuda.synchronize()
    assert torch.equal(of, of2)


@pytest.mark.parametrize("shape", [
    (256, 256, 2048, 8, 2),   # heavy expert: 2 parts of 16 steps
    (256, 256, 8192, 8, 2),   # heavy expert: 2 parts of 64 steps
])
def test_forward_split_heavy_cut(shape):
    """Streaming regime with a heavy expert: its down GEMM takes the tiled
    kernel with the reduction cut (slices folded into slice 0 before the
    combine).  Parity with the oracle; the forward equals the staged pair
    moe_swiglu_down_parts + moe_combine_parts bitwise, whose count reads 1
    after the fold; and the uncut staged calls agree to f32 rounding."""
    say(f"[forward] heavy expert, cut down GEMM {shape}")
    bias = [2.0] + [0.0] * (shape[3] - 1)
    c = small_case(*shape, seed=31, bias=bias)
    assert B.moe_gemm_variant_for(c.T, c.d, c.ffn, c.E, c.k) == 3
    T, d, k = c.T, c.d, c.k
    ids, gw, offs, perm, _ = gpu_route(c)
    rows = np.diff(offs.cpu().numpy())
    assert rows.max() > 64, rows
    _forward_check(c, variant=0)
    of = gpu_forward(c, out_f32=True)[1]
    h = torch.empty(T * k, c.ffn, dtype=torch.bfloat16, device=DEV)
    B.moe_swiglu_up(c.x, offs, c.w1, c.w3, T, k, h, perm=perm)
    # 2 slices: the forward's cap in this regime
    yp = torch.empty(2, T * k, d, dtype=torch.float32, device=DEV)
    np_dev = torch.zeros(1, dtype=torch.int32, device=DEV)
    B.moe_swiglu_down_parts(h, offs, c.w2, T, k, yp, np_dev, topk_w=gw, perm=perm)
    st = torch.empty(T, d, dtype=torch.float32, device=DEV)
    B.moe_combine_parts(yp, np_dev, T, d, k, out_f32=st)
    y = torch.empty(T * k, d, dtype=torch.float32, device=DEV)
    B.moe_swiglu_down(h, offs, c.w2, T, k, y, topk_w=gw, perm=perm)
    unc = torch.empty(T, d, dtype=torch.float32, device=DEV)
    B.moe_combine(y, T, d, k, out_f32=unc)
    torch.cuda.synchronize()
    assert int(np_dev.item()) == 1
    assert torch.equal(st, of)
    err = rowwise_rel(st.double().cpu().numpy(), unc.double().cpu().numpy())
    say(f"  cut vs uncut: rowwise rel {err:.3e}")
    assert err < 1e-5
    # plain mode (no gate weights, rows in permuted order): the fold works on
    # row r itself; slice 0 then matches the uncut plain down GEMM
    yp.fill_(0.0)
    np_dev.fill_(0)
    B.moe_swiglu_down_parts(h, offs, c.w2, T, k, yp, np_dev)
    yplain = torch.empty(T * k, d, dtype=torch.float32, device=DEV)
    B.moe_swiglu_down(h, offs, c.w2, T, k, yplain)
    torch.cuda.synchronize()
    assert int(np_dev.item()) == 1
    err = rowwise_rel(yp[0].double().cpu().numpy(), yplain.double().cpu().numpy())
    say(f"  plain rows, cut vs uncut: rowwise rel {err:.3e}")
    assert err < 1e-5


def test_forward_split_side_by_side_and_graph():
    """A split step runs the heavy expert's tiled launches on the library's
    side stream next to the light experts' streaming launches; captured into
    a graph the same calls run in sequence on the capturing stream.  Eager
    runs and graph replays (with eager work in between) give the same bits,
    and the eager result matches the oracle."""
    say("[forward] split step: side stream and graph capture")
    c = small_case(256, 256, 2048, 8, 2, seed=37, bias=[2.0] + [0.0] * 7)
    assert B.moe_gemm_variant_for(c.T, c.d, c.ffn, c.E, c.k) == 3
    _forward_check(c, variant=0)
    _graph_replays_match_eager(c)


def test_forward_tiled_parts_graph():
    """A prefill-regime step whose down GEMM is cut into 4 parts (the count
    chosen and stored on the device, read by the combine): graph replays give
    the bits of the eager runs, which match the oracle."""
    say("[forward] tiled step with reduction parts: graph capture")
    c = small_case(288, 256, 2048, 8, 2, seed=38)
    assert B.moe_gemm_variant_for(c.T, c.d, c.ffn, c.E, c.k) == 2
    _forward_check(c, variant=0)
    _graph_replays_match_eager(c)


def test_forward_tiled_tail_graph():
    """A prefill-regime step whose down GEMM splits its last round's tiles
    across workgroups (pieces folded back by a second kernel): graph replays
    give the bits of the eager runs, which match the oracle."""
    say("[forward] tiled step with a split last round: graph capture")
    c = small_case(3000, 1024, 2048, 8, 2, seed=39)
    assert B.moe_gemm_variant_for(c.T, c.d, c.ffn, c.E, c.k) == 2
    _forward_check(c, variant=0)
    _graph_replays_match_eager(c)


def _staged_out(c):
    """route -> up -> down -> combine through the stage entry points (the
    dispatch kernel's offsets and row order), as bf16 output bits"""
    T, d, ffn, k = c.T, c.d, c.ffn, c.k
    ids, gw, offs, perm, _ = gpu_route(c)
    h = torch.empty(T * k, ffn, dtype=torch.bfloat16, device=DEV)
    y = torch.empty(T * k, d, dtype=torch.float32, device=DEV)
    out = torch.empty(T, d, dtype=torch.bfloat16, device=DEV)
    B.moe_swiglu_up(c.x, offs, c.w1, c.w3, T, k, h, perm=perm)
    B.moe_swiglu_down(h, offs, c.w2, T, k, y, topk_w=gw, perm=perm)
    B.moe_combine(y, T, d, k, out=out)
    torch.cuda.synchronize()
    return out


@pytest.mark.parametrize("shape,bias", [
    ((64, 4096, 1792, 8, 2), None),            # one GPU's TP8 share of a decode step
    ((1, 128, 256, 8, 2), None),               # a single token
    ((64, 256, 512, 64, 8), None),             # E = 64, k = 8: 512 assignments
    ((48, 128, 256, 8, 2), [0, 0, 50, 0, 0, 40, 0, 0]),  # six experts idle
    ((64, 256, 256, 4, 1), [60, 0, 0, 0]),     # one expert takes every token
    ((512, 256, 256, 16, 2), None),            # 1024 assignments: the LDS table limit
    ((333, 128, 384, 8, 3), [30, 0, 0, 0, 0, 0, 0, 0]),  # 999 assignments, 333 rows on expert 0
])
def test_forward_routes_from_ids_bitwise(shape, bias):
    """With both GEMMs on the streaming kernels and at most 1024 assignments,
    the forward skips the dispatch kernel and every workgroup builds the
    expert offsets and row order from the top-k ids in LDS.  Its output must
    be bitwise the output of the stage entry points fed by the dispatch
    kernel (same kernels, same row order), and match the oracle."""
    say(f"[forward] routing from ids: {shape} bias {bias}")
    c = small_case(*shape, seed=41, bias=bias)
    prev = B.moe_set_gemm_variant(1)
    try:
        got = gpu_forward(c)
        ref = _staged_out(c)
    finally:
        B.moe_set_gemm_variant(prev)
    assert torch.equal(got.view(torch.int16), ref.view(torch.int16))
    _forward_check(c, variant=1)


def test_forward_routes_from_ids_graph():
    """The decode step that routes from ids, captured into a graph: replays
    (with the workspace cleared in between) give the eager bits."""
    say("[forward] routing from ids: graph capture")
    c = small_case(64, 512, 1024, 8, 2, seed=42)
    assert B.moe_gemm_variant_for(c.T, c.d, c.ffn, c.E, c.k) == 1
    _graph_replays_match_eager(c)


def _graph_replays_match_eager(c):
    T, d, k = c.T, c.d, c.k
    ws = torch.empty(B.moe_workspace_size(T, d, c.ffn, c.E, k), dtype=torch.uint8, device=DEV)
    outs = [torch.empty(T, d, dtype=torch.float32, device=DEV) for _ in range(3)]
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        for o in outs[:2]:
            B.moe_forward_ex(c.x, c.router_w, c.w1, c.w3, c.w2, k, out_f32=o,
                             router_bias=c.router_bias, workspace=ws, stream=s)
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    assert torch.equal(outs[0], outs[1])
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        B.moe_forward_ex(c.x, c.router_w, c.w1, c.w3, c.w2, k, out_f32=outs[2],
                         router_bias=c.router_bias, workspace=ws, stream=s)
    for rep in range(3):
        outs[2].fill_(7.0)
        ws.zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(outs[2], outs[0]), rep


@pytest.mark.parametrize("variant", [0, 1])
def test_forward_long_prefill_chunk(variant):
    """32768 tokens at the Mixtral shapes (65536 assignments, ~8192 rows per
    expert, 32 token tiles each): row and item indices well past the bench
    sizes; against the oracle, one token of every (expert, token tile) work
    item plus the first and last token."""
    say(f"[forward] 32768-token prefill chunk, variant {variant}")
    c = workload_case("prefill_t4096", T=32768)
    ids, *_ = gpu_route(c)
    # one token in every (expert, 256-row tile) of the tiled kernel's items
    rows = tile_cover_rows(ids.cpu().numpy(), c.k, c.E, seed=19)
    say(f"  {len(rows)} tokens cover every (expert, 256-row tile)")
    _forward_check(c, rows, variant)
    del c
    torch.cuda.empty_cache()


def test_forward_t0():
    c = small_case(3, 64, 64, 4, 2)
    out = torch.zeros(0, 64, dtype=torch.bfloat16, device=DEV)
    B.moe_forward(c.x[:0], c.router_w, c.w1, c.w3, c.w2, 2, out)
    torch.cuda.synchronize()


def test_rmsnorm_within_one_ulp():
    say("[rmsnorm]")
    from parity import bf16_ulp_diff, round_bf16_bits
    T, d = 64, 4096
    g = torch.Generator(device=DEV).manual_seed(5)
    h = torch.randn(T, d, device=DEV, generator=g) * 3
    w = inputs.Workload("g", T, d, 64, 1, 1, 1, 1, 1, 1, 1)
    gamma = inputs.make_gamma(w, 0, DEV, random=True)
    a = torch.empty(T, d, dtype=torch.bfloat16, device=DEV)
    B.moe_rmsnorm(h, gamma, 1e-5, a)
    torch.cuda.synchronize()
    ref = orc().rmsnorm(h.cpu().numpy(), inputs.bf16_bits(gamma), 1e-5)
    ulps = bf16_ulp_diff(inputs.bf16_bits(a), round_bf16_bits(ref))
    assert ulps.max() <= 1


def test_combine_residual_inplace():
    say("[combine]")
    T, d, k = 33, 192, 3
    g = torch.Generator(device=DEV).manual_seed(8)
    y = torch.randn(T * k, d, device=DEV, generator=g)
    res = torch.randn(T, d, device=DEV, generator=g)
    res0 = res.clone()
    out = torch.empty(T, d, dtype=torch.bfloat16, device=DEV)
    B.moe_combine(y, T, d, k, out=out, out_f32=res, residual=res)
    torch.cuda.synchronize()
    yy = y.cpu().numpy().reshape(T, k, d)
    ref = res0.cpu().numpy().copy()
    for j in range(k):  # same f32 order: residual, then slots ascending
        ref = (ref + yy[:, j]).astype(np.float32)
    assert np.array_equal(res.cpu().numpy(), ref)
    assert np.array_equal(out.float().cpu().numpy(), torch.from_numpy(ref).bfloat16().float().numpy())
