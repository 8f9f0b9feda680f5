"""ctypes binding of libmoe.so.

Argument marshalling only: each function takes torch tensors that already live
on the GPU, checks dtype/shape/contiguity, passes raw device pointers and the
current HIP stream to the C ABI of the same name, and raises ``MoeError`` on a
non-zero status.  Every step of the layer runs in the library's HIP kernels;
there is no fallback path.  PyTorch provides device memory and streams only.
"""

from __future__ import annotations

import ctypes
import os
from typing import Optional

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.environ.get("MOE_LIB", os.path.join(_PKG, "libmoe.so"))

MOE_OK, MOE_ERR_INVALID_ARG, MOE_ERR_UNSUPPORTED, MOE_ERR_NO_MEMORY, MOE_ERR_HIP = range(5)
VARIANT_AUTO, VARIANT_STREAM, VARIANT_TILED = 0, 1, 2

EXPORTS = (
    "moe_route", "moe_permute", "moe_swiglu_up", "moe_swiglu_down", "moe_swiglu_down_parts",
    "moe_grouped_swiglu", "moe_combine", "moe_combine_parts", "moe_forward", "moe_forward_ex", "moe_rmsnorm", "moe_workspace_size",
    "moe_swiglu_up_fp8", "moe_swiglu_down_fp8", "moe_swiglu_down_parts_fp8", "moe_forward_fp8_ex",
    "moe_linear", "moe_rope_kv_append", "moe_attention_decode",
    "moe_set_gemm_variant", "moe_gemm_variant_for", "moe_status_string", "moe_last_error", "moe_version",
    "moe_release_workspace", "moe_forward_noalloc",
)


class MoeError(RuntimeError):
    def __init__(self, status: int, fn: str, msg: str):
        self.status = status
        super().__init__(f"{fn}: {_status_name(status)}: {msg}")


_lib = None


def _status_name(s: int) -> str:
    return lib().moe_status_string(s).decode()


def lib() -> ctypes.CDLL:
    """Load libmoe.so (built by ``python -m paper_2408_00008_amd.build``)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: build it with "
                          "`python -m paper_2408_00008_amd.build` (hipcc, gfx950)")
    L = ctypes.CDLL(LIB_PATH)
    p, i64, i32, f32, sz = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_float, ctypes.c_size_t
    sig = {
        "moe_route": [p, p, p, i64, i32, i32, i32, p, p, p, p, p, p],
        "moe_permute": [p, p, i64, i32, i32, p, p],
        "moe_swiglu_up": [p, p, p, p, p, i64, i32, i32, i32, i32, p, p],
        "moe_swiglu_down": [p, p, p, p, p, i64, i32, i32, i32, i32, p, p],
        "moe_grouped_swiglu": [p, p, p, p, p, p, p, i64, i32, i32, i32, i32, p, p, p],
        "moe_swiglu_down_parts": [p, p, p, p, p, i64, i32, i32, i32, i32, i32, p, p, p],
        "moe_combine": [p, p, i64, i32, i32, p, p, p],
        "moe_combine_parts": [p, p, i32, p, i64, i32, i32, p, p, p],
        "moe_forward": [p, p, p, p, p, i64, i32, i32, i32, i32, p, p],
        "moe_forward_ex": [p, p, p, p, p, p, i64, i32, i32, i32, i32, p, p, p, p, sz, p],
        "moe_forward_noalloc": [p, p, p, p, p, p, i64, i32, i32, i32, i32, p, p, p, p],
        "moe_rmsnorm": [p, p, i64, i32, f32, p, p],
        "moe_swiglu_up_fp8": [p, p, p, p, p, p, p, i64, i32, i32, i32, i32, p, p],
        "moe_swiglu_down_fp8": [p, p, p, p, p, p, i64, i32, i32, i32, i32, p, p],
        "moe_swiglu_down_parts_fp8": [p, p, p, p, p, p, i64, i32, i32, i32, i32, i32, p, p, p],
        "moe_forward_fp8_ex": [p, p, p, p, p, p, p, p, p, i64, i32, i32, i32, i32, p, p, p, p,
                               sz, p],
        "moe_linear": [p, p, i64, i32, i32, p, p],
        "moe_rope_kv_append": [p, p, p, i64, i32, i32, i32, i32, i32, i64, ctypes.c_double, p, p,
                               p, p],
        "moe_attention_decode": [p, p, p, p, p, i64, i32, i32, i32, i32, i32, i64, f32, p, p],
    }
    for name, args in sig.items():
        fn = getattr(L, name)
        fn.argtypes = args
        fn.restype = ctypes.c_int
    L.moe_workspace_size.argtypes = [i64, i32, i32, i32, i32]
    L.moe_workspace_size.restype = sz
    L.moe_gemm_variant_for.argtypes = [i64, i32, i32, i32, i32]
    L.moe_gemm_variant_for.restype = ctypes.c_int
    L.moe_set_gemm_variant.argtypes = [ctypes.c_int]
    L.moe_set_gemm_variant.restype = ctypes.c_int
    L.moe_status_string.argtypes = [ctypes.c_int]
    L.moe_status_string.restype = ctypes.c_char_p
    L.moe_last_error.argtypes = []
    L.moe_last_error.restype = ctypes.c_char_p
    L.moe_version.argtypes = []
    L.moe_version.restype = ctypes.c_int
    L.moe_release_workspace.argtypes = []
    L.moe_release_workspace.restype = ctypes.c_int
    _lib = L
    return L


def _check(status: int, fn: str):
    if status != MOE_OK:
        raise MoeError(status, fn, lib().moe_last_error().decode())


def _ptr(t: Optional[torch.Tensor], dtype=None, name="tensor"):
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError(f"{name} must be a GPU tensor")
    if dtype is not None and t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return t.data_ptr()


def _stream(stream) -> Optional[int]:
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, torch.cuda.Stream):
        return stream.cuda_stream
    return int(stream)


bf16, f32, i32, u8 = torch.bfloat16, torch.float32, torch.int32, torch.uint8


def moe_route(x, router_w, k, topk_ids, topk_w, expert_offsets, perm, router_bias=None,
              logits=None, stream=None):
    T, d = x.shape
    E = router_w.shape[0]
    _check(lib().moe_route(_ptr(x, bf16, "x"), _ptr(router_w, bf16, "router_w"),
                           _ptr(router_bias, f32, "router_bias"), T, d, E, k,
                           _ptr(topk_ids, i32, "topk_ids"), _ptr(topk_w, f32, "topk_w"),
                           _ptr(expert_offsets, i32, "expert_offsets"), _ptr(perm, i32, "perm"),
                           _ptr(logits, f32, "logits"), _stream(stream)), "moe_route")


def moe_permute(x, perm, k, x_perm, stream=None):
    T, d = x.shape
    _check(lib().moe_permute(_ptr(x, bf16, "x"), _ptr(perm, i32, "perm"), T, d, k,
                             _ptr(x_perm, bf16, "x_perm"), _stream(stream)), "moe_permute")


def moe_swiglu_up(x, expert_offsets, w1, w3, T, k, h, perm=None, stream=None):
    """x: permuted rows [T*k,d] (perm None) or token rows [T,d] gathered via perm."""
    E, ffn, d = w1.shape
    _check(lib().moe_swiglu_up(_ptr(x, bf16, "x"), _ptr(perm, i32, "perm"),
                               _ptr(expert_offsets, i32, "offsets"), _ptr(w1, bf16, "w1"),
                               _ptr(w3, bf16, "w3"), T, d, ffn, E, k, _ptr(h, bf16, "h"),
                               _stream(stream)), "moe_swiglu_up")


def moe_swiglu_down(h, expert_offsets, w2, T, k, y, topk_w=None, perm=None, stream=None):
    E, d, ffn = w2.shape
    _check(lib().moe_swiglu_down(_ptr(h, bf16, "h"), _ptr(expert_offsets, i32, "offsets"),
                                 _ptr(w2, bf16, "w2"), _ptr(topk_w, f32, "topk_w"),
                                 _ptr(perm, i32, "perm"), T, d, ffn, E, k, _ptr(y, f32, "y"),
                                 _stream(stream)), "moe_swiglu_down")


def moe_swiglu_down_parts(h, expert_offsets, w2, T, k, y, parts, topk_w=None, perm=None,
                          stream=None):
    """y: [max_parts, T*k, d] f32 slices; parts: one device int32 receiving the count used."""
    E, d, ffn = w2.shape
    max_parts = y.shape[0]
    _check(lib().moe_swiglu_down_parts(
        _ptr(h, bf16, "h"), _ptr(expert_offsets, i32, "offsets"), _ptr(w2, bf16, "w2"),
        _ptr(topk_w, f32, "topk_w"), _ptr(perm, i32, "perm"), T, d, ffn, E, k, max_parts,
        _ptr(y, f32, "y"), _ptr(parts, i32, "parts"), _stream(stream)), "moe_swiglu_down_parts")


def moe_swiglu_down_parts_fp8(h, expert_offsets, w2q, w2s, T, k, y, parts, topk_w=None,
                              perm=None, stream=None):
    """8-bit weights: y [max_parts, T*k, d] f32 slices; parts one device int32."""
    E, d, ffn = w2q.shape
    _check(lib().moe_swiglu_down_parts_fp8(
        _ptr(h, bf16, "h"), _ptr(expert_offsets, i32, "offsets"), _ptr(w2q, u8, "w2q"),
        _ptr(w2s, f32, "w2s"), _ptr(topk_w, f32, "topk_w"), _ptr(perm, i32, "perm"), T, d, ffn,
        E, k, y.shape[0], _ptr(y, f32, "y"), _ptr(parts, i32, "parts"), _stream(stream)),
        "moe_swiglu_down_parts_fp8")


def moe_grouped_swiglu(x_perm, expert_offsets, w1, w3, w2, T, k, h_ws, y, topk_w=None,
                       perm=None, stream=None):
    E, ffn, d = w1.shape
    _check(lib().moe_grouped_swiglu(
        _ptr(x_perm, bf16, "x_perm"), _ptr(expert_offsets, i32, "offsets"), _ptr(w1, bf16, "w1"),
        _ptr(w3, bf16, "w3"), _ptr(w2, bf16, "w2"), _ptr(topk_w, f32, "topk_w"),
        _ptr(perm, i32, "perm"), T, d, ffn, E, k, _ptr(h_ws, bf16, "h_ws"), _ptr(y, f32, "y"),
        _stream(stream)), "moe_grouped_swiglu")


def moe_combine(y, T, d, k, out=None, out_f32=None, residual=None, stream=None):
    _check(lib().moe_combine(_ptr(y, f32, "y"), _ptr(residual, f32, "residual"), T, d, k,
                             _ptr(out, bf16, "out"), _ptr(out_f32, f32, "out_f32"),
                             _stream(stream)), "moe_combine")


def moe_combine_parts(y, parts, T, d, k, out=None, out_f32=None, residual=None, stream=None):
    """y: [max_parts, T*k, d] f32 slices of moe_swiglu_down_parts, parts its device count."""
    _check(lib().moe_combine_parts(_ptr(y, f32, "y"), _ptr(parts, i32, "parts"), y.shape[0],
                                   _ptr(residual, f32, "residual"), T, d, k,
                                   _ptr(out, bf16, "out"), _ptr(out_f32, f32, "out_f32"),
                                   _stream(stream)), "moe_combine_parts")


def moe_forward(x, router_w, w1, w3, w2, k, out, stream=None):
    T, d = x.shape
    E, ffn, _ = w1.shape
    _check(lib().moe_forward(_ptr(x, bf16, "x"), _ptr(router_w, bf16, "router_w"),
                             _ptr(w1, bf16, "w1"), _ptr(w3, bf16, "w3"), _ptr(w2, bf16, "w2"),
                             T, d, ffn, E, k, _ptr(out, bf16, "out"), _stream(stream)),
           "moe_forward")


def moe_forward_ex(x, router_w, w1, w3, w2, k, out=None, out_f32=None, router_bias=None,
                   residual=None, workspace=None, stream=None):
    T, d = x.shape
    E, ffn, _ = w1.shape
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(lib().moe_forward_ex(
        _ptr(x, bf16, "x"), _ptr(router_w, bf16, "router_w"), _ptr(router_bias, f32, "router_bias"),
        _ptr(w1, bf16, "w1"), _ptr(w3, bf16, "w3"), _ptr(w2, bf16, "w2"), T, d, ffn, E, k,
        _ptr(residual, f32, "residual"), _ptr(out, bf16, "out"), _ptr(out_f32, f32, "out_f32"),
        _ptr(workspace, None, "workspace"), ws_bytes, _stream(stream)), "moe_forward_ex")


def moe_forward_noalloc(x, router_w, w1, w3, w2, k, out=None, out_f32=None, router_bias=None,
                        residual=None, stream=None):
    """moe_forward_ex without a workspace: the library's fixed device scratch array."""
    T, d = x.shape
    E, ffn, _ = w1.shape
    _check(lib().moe_forward_noalloc(
        _ptr(x, bf16, "x"), _ptr(router_w, bf16, "router_w"), _ptr(router_bias, f32, "router_bias"),
        _ptr(w1, bf16, "w1"), _ptr(w3, bf16, "w3"), _ptr(w2, bf16, "w2"), T, d, ffn, E, k,
        _ptr(residual, f32, "residual"), _ptr(out, bf16, "out"), _ptr(out_f32, f32, "out_f32"),
        _stream(stream)), "moe_forward_noalloc")


def moe_swiglu_up_fp8(x, expert_offsets, w1q, w1s, w3q, w3s, T, k, h, perm=None, stream=None):
    """8-bit weights: w1q/w3q [E,ffn,d] E4M3 bytes (uint8), w1s/w3s [E,ffn] f32 row scales."""
    E, ffn, d = w1q.shape
    _check(lib().moe_swiglu_up_fp8(
        _ptr(x, bf16, "x"), _ptr(perm, i32, "perm"), _ptr(expert_offsets, i32, "offsets"),
        _ptr(w1q, u8, "w1q"), _ptr(w1s, f32, "w1s"), _ptr(w3q, u8, "w3q"), _ptr(w3s, f32, "w3s"),
        T, d, ffn, E, k, _ptr(h, bf16, "h"), _stream(stream)), "moe_swiglu_up_fp8")


def moe_swiglu_down_fp8(h, expert_offsets, w2q, w2s, T, k, y, topk_w=None, perm=None,
                        stream=None):
    """8-bit weights: w2q [E,d,ffn] E4M3 bytes (uint8), w2s [E,d] f32 row scales."""
    E, d, ffn = w2q.shape
    _check(lib().moe_swiglu_down_fp8(
        _ptr(h, bf16, "h"), _ptr(expert_offsets, i32, "offsets"), _ptr(w2q, u8, "w2q"),
        _ptr(w2s, f32, "w2s"), _ptr(topk_w, f32, "topk_w"), _ptr(perm, i32, "perm"), T, d, ffn,
        E, k, _ptr(y, f32, "y"), _stream(stream)), "moe_swiglu_down_fp8")


def moe_forward_fp8_ex(x, router_w, w1q, w1s, w3q, w3s, w2q, w2s, k, out=None, out_f32=None,
                       router_bias=None, residual=None, workspace=None, stream=None):
    T, d = x.shape
    E, ffn, _ = w1q.shape
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(lib().moe_forward_fp8_ex(
        _ptr(x, bf16, "x"), _ptr(router_w, bf16, "router_w"), _ptr(router_bias, f32, "router_bias"),
        _ptr(w1q, u8, "w1q"), _ptr(w1s, f32, "w1s"), _ptr(w3q, u8, "w3q"), _ptr(w3s, f32, "w3s"),
        _ptr(w2q, u8, "w2q"), _ptr(w2s, f32, "w2s"), T, d, ffn, E, k,
        _ptr(residual, f32, "residual"), _ptr(out, bf16, "out"), _ptr(out_f32, f32, "out_f32"),
        _ptr(workspace, None, "workspace"), ws_bytes, _stream(stream)), "moe_forward_fp8_ex")


def moe_linear(x, w, y, stream=None):
    """y [T, N] f32 = x [T, K] bf16 . w [N, K]^T bf16."""
    T, K = x.shape
    N = w.shape[0]
    _check(lib().moe_linear(_ptr(x, bf16, "x"), _ptr(w, bf16, "w"), T, K, N, _ptr(y, f32, "y"),
                            _stream(stream)), "moe_linear")


def moe_rope_kv_append(qkv, pos, page_table, Hq, Hkv, theta, q_out, k_cache, v_cache, stream=None):
    """qkv [T, (Hq+2Hkv) hd] f32; caches [npages, Hkv, page, hd] bf16."""
    T = qkv.shape[0]
    npages, _, page, hd = k_cache.shape
    _check(lib().moe_rope_kv_append(
        _ptr(qkv, f32, "qkv"), _ptr(pos, i32, "pos"), _ptr(page_table, i32, "page_table"), T, Hq,
        Hkv, hd, page, page_table.shape[1], npages, float(theta), _ptr(q_out, bf16, "q_out"),
        _ptr(k_cache, bf16, "k_cache"), _ptr(v_cache, bf16, "v_cache"), _stream(stream)),
        "moe_rope_kv_append")


def moe_attention_decode(q, k_cache, v_cache, page_table, ctx, scale, out, stream=None):
    """q [T, Hq, hd] bf16; out [T, Hq*hd] bf16."""
    T, Hq, hd = q.shape
    npages, Hkv, page, _ = k_cache.shape
    _check(lib().moe_attention_decode(
        _ptr(q, bf16, "q"), _ptr(k_cache, bf16, "k_cache"), _ptr(v_cache, bf16, "v_cache"),
        _ptr(page_table, i32, "page_table"), _ptr(ctx, i32, "ctx"), T, Hq, Hkv, hd, page,
        page_table.shape[1], npages, float(scale), _ptr(out, bf16, "out"), _stream(stream)),
        "moe_attention_decode")


def moe_rmsnorm(h, gamma, eps, a, stream=None):
    T, d = h.shape
    _check(lib().moe_rmsnorm(_ptr(h, f32, "h"), _ptr(gamma, bf16, "gamma"), T, d, float(eps),
                             _ptr(a, bf16, "a"), _stream(stream)), "moe_rmsnorm")


def moe_workspace_size(T, d, ffn, E, k) -> int:
    return int(lib().moe_workspace_size(T, d, ffn, E, k))


def moe_gemm_variant_for(T, d, ffn, E, k) -> int:
    return int(lib().moe_gemm_variant_for(T, d, ffn, E, k))


def moe_set_gemm_variant(v: int) -> int:
    return int(lib().moe_set_gemm_variant(v))


def moe_release_workspace():
    """Frees the library-owned scratch of the current device (after a device sync)."""
    _check(lib().moe_release_workspace(), "moe_release_workspace")
