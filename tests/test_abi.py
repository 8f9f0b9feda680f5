"""The C ABI library loads, exports every declared symbol, and rejects bad
arguments before touching the GPU (CPU only: every call here fails validation
or has T = 0, so no HIP call is made)."""

import ctypes
import os
import re

import pytest

from paper_2408_00008_amd import binding as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "moe.h")


def declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(moe_[a-z0-9_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(B.LIB_PATH):
        from paper_2408_00008_amd import build
        build.build()
    return B.lib()


def test_exports_every_declared_symbol(L):
    names = declared()
    assert len(names) >= 14
    for n in names:
        assert hasattr(L, n), f"{n} declared in moe.h but not exported"
    assert set(names) == set(B.EXPORTS)


def test_status_strings(L):
    assert L.moe_status_string(0) == b"MOE_OK"
    assert L.moe_status_string(1) == b"MOE_ERR_INVALID_ARG"
    assert L.moe_status_string(2) == b"MOE_ERR_UNSUPPORTED"
    assert L.moe_status_string(3) == b"MOE_ERR_NO_MEMORY"
    assert L.moe_status_string(4) == b"MOE_ERR_HIP"
    assert L.moe_status_string(99) == b"MOE_ERR_UNKNOWN"
    assert L.moe_version() >= 100


# fake device addresses: never dereferenced because every call below is
# rejected by validation (or is empty)
X, RW, W1, W3, W2, OUT = (0x10000 * (i + 1) for i in range(6))
BIG = 1 << 40  # far apart so no two fake ranges overlap


def fwd(L, x=X, rw=RW, w1=W1 * BIG // 0x10000, w3=W3 * BIG // 0x10000, w2=W2 * BIG // 0x10000,
        T=4, d=128, ffn=256, E=8, k=2, out=OUT * BIG // 0x10000):
    return L.moe_forward(x, rw, w1, w3, w2, T, d, ffn, E, k, out, None)


@pytest.mark.parametrize("kw,status,msg", [
    (dict(E=65), B.MOE_ERR_UNSUPPORTED, "E=65"),
    (dict(E=0), B.MOE_ERR_INVALID_ARG, "E=0"),
    (dict(k=0), B.MOE_ERR_INVALID_ARG, "k=0"),
    (dict(k=9, E=16), B.MOE_ERR_UNSUPPORTED, "k=9"),
    (dict(k=3, E=2), B.MOE_ERR_INVALID_ARG, "exceeds E"),
    (dict(d=100), B.MOE_ERR_UNSUPPORTED, "multiple of 64"),
    (dict(ffn=96), B.MOE_ERR_UNSUPPORTED, "multiple of 64"),
    (dict(d=0), B.MOE_ERR_INVALID_ARG, "d=0"),
    (dict(d=65536 + 64), B.MOE_ERR_UNSUPPORTED, "exceeds"),
    (dict(T=-1), B.MOE_ERR_INVALID_ARG, "T=-1"),
    (dict(T=1 << 30, k=2), B.MOE_ERR_UNSUPPORTED, "2^31"),
    (dict(x=0), B.MOE_ERR_INVALID_ARG, "x is NULL"),
    (dict(x=X + 2), B.MOE_ERR_INVALID_ARG, "aligned"),
    (dict(out=0), B.MOE_ERR_INVALID_ARG, "out is NULL"),
    (dict(out=X), B.MOE_ERR_INVALID_ARG, "overlaps x"),
])
def test_forward_rejects(L, kw, status, msg):
    st = fwd(L, **kw)
    assert st == status, (st, L.moe_last_error())
    assert msg in L.moe_last_error().decode()


def test_forward_empty_is_ok(L):
    assert fwd(L, T=0) == B.MOE_OK
    assert L.moe_last_error() == b""


def test_route_and_stage_rejects(L):
    p = ctypes.c_void_p
    # k > E
    st = L.moe_route(X, RW, None, 4, 128, 2, 3, 0x100000, 0x200000, 0x300000, 0x400000, None, None)
    assert st == B.MOE_ERR_INVALID_ARG
    # overlapping outputs
    st = L.moe_route(X, RW, None, 4, 128, 8, 2, 0x100000, 0x100000, 0x300000, 0x400000, None, None)
    assert st == B.MOE_ERR_INVALID_ARG and b"overlaps" in L.moe_last_error()
    # misaligned bias
    st = L.moe_route(X, RW, 0x500004, 4, 128, 8, 2, 0x100000, 0x200000, 0x300000, 0x400000,
                     None, None)
    assert st == B.MOE_ERR_INVALID_ARG and b"router_bias" in L.moe_last_error()
    assert L.moe_route(X, RW, None, 0, 128, 8, 2, 0x100000, 0x200000, 0x300000, 0x400000,
                       None, None) == B.MOE_OK
    # combine needs an output
    assert L.moe_combine(X, None, 4, 128, 2, None, None, None) == B.MOE_ERR_INVALID_ARG
    # rmsnorm eps
    assert L.moe_rmsnorm(X, RW, 4, 128, ctypes.c_float(-1.0), OUT, None) == B.MOE_ERR_INVALID_ARG
    # swiglu: h overlapping a weight
    w = 1 << 36
    st = L.moe_swiglu_up(X, None, 0x700000, w, 2 * w, 4, 128, 256, 8, 2, w + 64, None)
    assert st == B.MOE_ERR_INVALID_ARG and b"overlaps w1" in L.moe_last_error()
    # permute into its own input
    assert L.moe_permute(X, 0x700000, 4, 128, 2, X, None) == B.MOE_ERR_INVALID_ARG
    del p


def test_parts_entry_points_reject(L):
    """The cut down GEMM and its combine: the part count pointer and bound are
    checked, and y's full extent (max_parts slices) may overlap nothing."""
    T, d, ffn, E, k = 4, 128, 256, 8, 2
    yb = T * k * d * 4  # one slice
    w2 = 1 << 36
    y, parts = 1 << 38, 1 << 39

    def down(**kw):
        a = dict(mp=4, y=y, parts=parts, w2=w2)
        a.update(kw)
        return L.moe_swiglu_down_parts(X, 0x700000, a["w2"], None, None, T, d, ffn, E, k,
                                       a["mp"], a["y"], a["parts"], None)

    assert down(mp=0) == B.MOE_ERR_INVALID_ARG and b"max_parts" in L.moe_last_error()
    assert down(parts=None) == B.MOE_ERR_INVALID_ARG and b"parts is NULL" in L.moe_last_error()
    assert down(parts=parts + 2) == B.MOE_ERR_INVALID_ARG and b"4-byte" in L.moe_last_error()
    # the count inside the last slice; the last slice over w2
    assert down(parts=y + 3 * yb + 64) == B.MOE_ERR_INVALID_ARG
    assert b"parts overlaps y" in L.moe_last_error()
    assert down(y=w2 - 3 * yb - 256) == B.MOE_ERR_INVALID_ARG
    assert b"y overlaps w2" in L.moe_last_error()

    def comb(**kw):
        a = dict(mp=4, parts=parts, out=OUT)
        a.update(kw)
        return L.moe_combine_parts(y, a["parts"], a["mp"], None, T, d, k, a["out"], None, None)

    # the 8-bit weight form: same checks, and the scales are required
    q2, s2 = 1 << 36, 1 << 37
    st = L.moe_swiglu_down_parts_fp8(X, 0x700000, q2, s2, None, None, T, d, ffn, E, k, 0, y,
                                      parts, None)
    assert st == B.MOE_ERR_INVALID_ARG and b"max_parts" in L.moe_last_error()
    st = L.moe_swiglu_down_parts_fp8(X, 0x700000, q2, None, None, None, T, d, ffn, E, k, 4, y,
                                      parts, None)
    assert st == B.MOE_ERR_INVALID_ARG and b"w2s is NULL" in L.moe_last_error()
    st = L.moe_swiglu_down_parts_fp8(X, 0x700000, q2, s2, None, None, T, d, ffn, E, k, 4, y,
                                      y + 3 * yb + 64, None)
    assert st == B.MOE_ERR_INVALID_ARG and b"parts overlaps y" in L.moe_last_error()

    assert comb(mp=0) == B.MOE_ERR_INVALID_ARG and b"max_parts" in L.moe_last_error()
    assert comb(parts=None) == B.MOE_ERR_INVALID_ARG and b"parts is NULL" in L.moe_last_error()
    assert comb(out=y + 3 * yb) == B.MOE_ERR_INVALID_ARG and b"overlaps y" in L.moe_last_error()
    assert comb(out=parts - 64) == B.MOE_ERR_INVALID_ARG and b"overlaps parts" in L.moe_last_error()


def test_forward_ex_workspace_checks(L):
    big = 1 << 40
    args = [X, RW, None, big, 2 * big, 3 * big, 4, 128, 256, 8, 2, None, 4 * big, None]
    need = L.moe_workspace_size(4, 128, 256, 8, 2)
    assert need > 0
    st = L.moe_forward_ex(*args, 5 * big + 16, need, None)
    assert st == B.MOE_ERR_INVALID_ARG and b"256-byte" in L.moe_last_error()
    st = L.moe_forward_ex(*args, 5 * big, need - 1, None)
    assert st == B.MOE_ERR_NO_MEMORY
    st = L.moe_forward_ex(X, RW, None, big, 2 * big, 3 * big, 4, 128, 256, 8, 2, None, None,
                          None, None, 0, None)
    assert st == B.MOE_ERR_INVALID_ARG and b"both NULL" in L.moe_last_error()


def test_workspace_size(L):
    assert L.moe_workspace_size(0, 128, 256, 8, 2) > 0  # offsets still have E+1 entries
    assert L.moe_workspace_size(4, 128, 256, 8, 9) == 0
    T, d, f, E, k = 64, 4096, 14336, 8, 2
    ws = L.moe_workspace_size(T, d, f, E, k)
    A = T * k
    assert ws >= A * f * 2 + A * d * 4 + 3 * A * 4


def _ws_bytes(T, d, ffn, E, k, slices):
    """moe_forward's scratch for these sizes: routing arrays, h, y with
    `slices` f32 partial-sum slices, the part count; each 256-byte aligned."""
    a = lambda v: (v + 255) // 256 * 256
    A = T * k
    return (a(A * 4) * 3 + a((E + 1) * 4) + a(A * ffn * 2) + a(A * d * 4 * slices) + 256)


@pytest.mark.parametrize("T,d,ffn,E,k,slices", [
    (4096, 4096, 14336, 8, 2, 4),   # prefill: tiled, down cut in up to 4 parts
    (256, 4096, 14336, 8, 2, 2),    # streaming with T > 64: heavy experts cut in up to 2
    (64, 4096, 14336, 8, 2, 1),     # decode: no heavy expert possible, one slice
    (1000, 512, 384, 8, 2, 1),      # tiled, but 6 reduction steps: too short to cut
    (1000, 512, 1024, 8, 2, 2),     # 16 steps: 2 parts of 8
    (600, 192, 320, 8, 2, 1),       # no tiled shape
    (40000, 4096, 14336, 8, 2, 1),  # 80000 rows: the grid is full anyway
])
def test_workspace_holds_part_slices(L, T, d, ffn, E, k, slices):
    assert L.moe_workspace_size(T, d, ffn, E, k) == _ws_bytes(T, d, ffn, E, k, slices)


def test_variant_switch(L):
    assert L.moe_gemm_variant_for(64, 4096, 14336, 8, 2) == 1
    assert L.moe_gemm_variant_for(64, 4096, 14336, 8, 9) == 0
    # streaming regime with T > 64: split by rows per expert; mean above 64: tiled
    assert L.moe_gemm_variant_for(256, 4096, 14336, 8, 2) == 3
    assert L.moe_gemm_variant_for(4096, 4096, 14336, 8, 2) == 2
    assert L.moe_gemm_variant_for(257, 4096, 14336, 8, 2) == 2
    prev = L.moe_set_gemm_variant(1)
    assert L.moe_gemm_variant_for(256, 4096, 14336, 8, 2) == 1
    L.moe_set_gemm_variant(prev)
    prev = L.moe_set_gemm_variant(1)
    assert L.moe_set_gemm_variant(2) == 1
    assert L.moe_set_gemm_variant(7) == -1
    assert L.moe_set_gemm_variant(prev) == 2


def test_fp8_entry_points_reject(L):
    """8-bit weight calls: byte arrays and scales are required and 16-byte
    aligned, outputs may not overlap them, T = 0 is a no-op."""
    big = 1 << 40
    q1, s1, q3, s3, q2, s2 = (big * (i + 1) for i in range(6))
    out = 7 * big

    def fwd8(**kw):
        a = dict(x=X, rw=RW, q1=q1, s1=s1, q3=q3, s3=s3, q2=q2, s2=s2, T=4, out=out)
        a.update(kw)
        return L.moe_forward_fp8_ex(a["x"], a["rw"], None, a["q1"], a["s1"], a["q3"], a["s3"],
                                    a["q2"], a["s2"], a["T"], 128, 256, 8, 2, None, a["out"],
                                    None, None, 0, None)

    assert fwd8(s1=0) == B.MOE_ERR_INVALID_ARG and b"w1s is NULL" in L.moe_last_error()
    assert fwd8(q2=0) == B.MOE_ERR_INVALID_ARG and b"w2q is NULL" in L.moe_last_error()
    assert fwd8(q3=q3 + 8) == B.MOE_ERR_INVALID_ARG and b"w3q" in L.moe_last_error()
    assert fwd8(s2=s2 + 4) == B.MOE_ERR_INVALID_ARG and b"w2s" in L.moe_last_error()
    assert fwd8(out=s3 + 64) == B.MOE_ERR_INVALID_ARG and b"overlaps w3s" in L.moe_last_error()
    assert fwd8(T=0) == B.MOE_OK
    # up: h overlapping a scale array; down: y overlapping the byte array
    st = L.moe_swiglu_up_fp8(X, None, 0x700000, q1, s1, q3, s3, 4, 128, 256, 8, 2, s1 + 16, None)
    assert st == B.MOE_ERR_INVALID_ARG and b"overlaps w1s" in L.moe_last_error()
    st = L.moe_swiglu_down_fp8(X, 0x700000, q2, s2, None, None, 4, 128, 256, 8, 2, q2 + 256, None)
    assert st == B.MOE_ERR_INVALID_ARG and b"overlaps w2q" in L.moe_last_error()
    st = L.moe_swiglu_down_fp8(X, 0x700000, None, s2, None, None, 4, 128, 256, 8, 2, out, None)
    assert st == B.MOE_ERR_INVALID_ARG and b"w2q is NULL" in L.moe_last_error()
    assert L.moe_swiglu_up_fp8(None, None, 0x700000, q1, s1, q3, s3, 0, 128, 256, 8, 2, None,
                               None) == B.MOE_OK


def test_decoder_entry_points_reject(L):
    """moe_linear, moe_rope_kv_append and moe_attention_decode validate
    shapes, head layouts, cache geometry, scale/theta and aliasing before
    touching the GPU; T = 0 is a no-op."""
    big = 1 << 40
    x, w, y, q, kc, vc, pt, ctx, out = (big * (i + 1) for i in range(9))
    c_double, c_float = ctypes.c_double, ctypes.c_float
    # linear
    assert L.moe_linear(x, w, 4, 100, 128, y, None) == B.MOE_ERR_UNSUPPORTED
    assert L.moe_linear(x, w, 4, 128, 128, w + 64, None) == B.MOE_ERR_INVALID_ARG
    assert b"overlaps w" in L.moe_last_error()
    assert L.moe_linear(None, w, 0, 128, 128, None, None) == B.MOE_OK

    def rope(**kw):
        a = dict(T=4, Hq=32, Hkv=8, hd=128, page=16, maxp=4, npages=64, theta=1e6, q_out=q, kc=kc)
        a.update(kw)
        return L.moe_rope_kv_append(x, ctx, pt, a["T"], a["Hq"], a["Hkv"], a["hd"], a["page"], a["maxp"],
                                    a["npages"], c_double(a["theta"]), a["q_out"], a["kc"], vc, None)
    assert rope(Hq=30) == B.MOE_ERR_INVALID_ARG and b"multiple of Hkv" in L.moe_last_error()
    assert rope(hd=127) == B.MOE_ERR_INVALID_ARG
    assert rope(theta=0.0) == B.MOE_ERR_INVALID_ARG
    assert rope(page=0) == B.MOE_ERR_INVALID_ARG
    assert rope(q_out=kc + 32) == B.MOE_ERR_INVALID_ARG and b"overlaps" in L.moe_last_error()
    assert rope(kc=vc) == B.MOE_ERR_INVALID_ARG
    assert rope(T=0) == B.MOE_OK

    def attn(**kw):
        a = dict(T=4, Hq=32, Hkv=8, hd=128, page=16, maxp=4, npages=64, scale=0.088, out=out)
        a.update(kw)
        return L.moe_attention_decode(q, kc, vc, pt, ctx, a["T"], a["Hq"], a["Hkv"], a["hd"], a["page"],
                                      a["maxp"], a["npages"], c_float(a["scale"]), a["out"], None)
    assert attn(hd=64) == B.MOE_ERR_UNSUPPORTED
    assert attn(page=12) == B.MOE_ERR_UNSUPPORTED
    assert attn(Hq=48, Hkv=3) == B.MOE_ERR_UNSUPPORTED  # group of 16
    assert attn(maxp=5000) == B.MOE_ERR_UNSUPPORTED
    assert attn(scale=0.0) == B.MOE_ERR_INVALID_ARG
    assert attn(out=q + 16) == B.MOE_ERR_INVALID_ARG and b"overlaps q" in L.moe_last_error()
    assert attn(T=0) == B.MOE_OK


@pytest.fixture
def ws_limit():
    """Sets MOE_WORKSPACE_LIMIT_BYTES for one test (the library reads it on
    every call) and removes it afterwards."""
    old = os.environ.get("MOE_WORKSPACE_LIMIT_BYTES")

    def set_(v):
        os.environ["MOE_WORKSPACE_LIMIT_BYTES"] = v

    yield set_
    if old is None:
        os.environ.pop("MOE_WORKSPACE_LIMIT_BYTES", None)
    else:
        os.environ["MOE_WORKSPACE_LIMIT_BYTES"] = old


def test_workspace_limit_forces_no_memory(L, ws_limit):
    """A cap below what moe_forward needs returns MOE_ERR_NO_MEMORY after
    validation and before any HIP call (so it runs here without a GPU); an
    unparsable cap is an argument error."""
    need = L.moe_workspace_size(4, 128, 256, 8, 2)
    ws_limit(str(need - 1))
    assert fwd(L) == B.MOE_ERR_NO_MEMORY
    msg = L.moe_last_error().decode()
    assert "MOE_WORKSPACE_LIMIT_BYTES" in msg and str(need) in msg
    # the 8-bit forward shares the scratch and the cap
    big = 1 << 40
    st = L.moe_forward_fp8_ex(X, RW, None, big, 2 * big, 3 * big, 4 * big, 5 * big, 6 * big,
                              4, 128, 256, 8, 2, None, 7 * big, None, None, 0, None)
    assert st == B.MOE_ERR_NO_MEMORY
    # a caller workspace is not capped (rejected here only for its size)
    st = L.moe_forward_ex(X, RW, None, big, 2 * big, 3 * big, 4, 128, 256, 8, 2, None, 4 * big,
                          None, 5 * big, need - 1, None)
    assert st == B.MOE_ERR_NO_MEMORY and b"smaller than" in L.moe_last_error()
    for bad in ("abc", "-5", "12kb", "99999999999999999999999"):
        ws_limit(bad)
        assert fwd(L) == B.MOE_ERR_INVALID_ARG, bad
        assert b"not a byte count" in L.moe_last_error()
    # validation still comes first
    ws_limit("0")
    assert fwd(L, E=65) == B.MOE_ERR_UNSUPPORTED
    assert fwd(L, T=0) == B.MOE_OK


def test_noalloc_validates_then_refuses_large_sizes(L):
    """moe_forward_noalloc validates like moe_forward_ex, then refuses sizes
    beyond its fixed 64 MiB scratch array before any HIP call."""
    big = 1 << 40
    args = (X, RW, None, big, 2 * big, 3 * big)
    st = L.moe_forward_noalloc(*args, 4, 128, 256, 65, 2, None, 4 * big, None, None)
    assert st == B.MOE_ERR_UNSUPPORTED
    st = L.moe_forward_noalloc(*args, 4, 128, 256, 8, 2, None, None, None, None)
    assert st == B.MOE_ERR_INVALID_ARG and b"both NULL" in L.moe_last_error()
    assert L.moe_forward_noalloc(*args, 0, 128, 256, 8, 2, None, 4 * big, None, None) == B.MOE_OK
    T, d, ffn = 1024, 4096, 14336
    need = L.moe_workspace_size(T, d, ffn, 8, 2)
    assert need > 64 << 20
    st = L.moe_forward_noalloc(X, RW, None, big, 2 * big, 3 * big, T, d, ffn, 8, 2, None, 4 * big,
                               None, None)
    assert st == B.MOE_ERR_NO_MEMORY
    msg = L.moe_last_error().decode()
    assert "fixed" in msg and str(need) in msg
