"""ctypes front end of the fp64 CPU oracle (``moe_oracle.c``).

TEST INFRASTRUCTURE ONLY: the test suite, the smoke check and the benchmark's
CPU-baseline leg are its only callers.  It takes host numpy arrays (bf16 as
raw ``uint16`` bit patterns), never imports the GPU package and never touches
a device.

Definitions follow the Mixtral MoE layer that the paper's engine serves
(Sec. 4.1 and Sec. 5 of the paper); the C file's header states them.
"""

from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "moe_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

_i64, _i32, _f64 = ctypes.c_int64, ctypes.c_int32, ctypes.c_double
_p = ctypes.c_void_p


class OracleError(RuntimeError):
    pass


def build(src: str = _SRC, out: str = _LIB, extra=()) -> str:
    """Compile the oracle with gcc (OpenMP, no fast-math: sums keep their order)."""
    cmd = ["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c11", "-Wall", "-Werror",
           *extra, src, "-o", out + ".tmp", "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(out + ".tmp", out)
    return out


class Oracle:
    """One loaded copy of the oracle library (a mutant build may be loaded too)."""

    def __init__(self, lib_path: str = _LIB):
        if lib_path == _LIB and not os.path.exists(_LIB):
            build()
        self.lib = ctypes.CDLL(lib_path)
        L = self.lib
        L.oracle_threads.argtypes = [ctypes.c_int]
        L.oracle_threads.restype = ctypes.c_int
        L.oracle_router_logits.argtypes = [_p, _p, _p, _i64, _i64, _i64, _p]
        L.oracle_topk_gate.argtypes = [_p, _i64, ctypes.c_int, ctypes.c_int, _p, _p]
        L.oracle_gates_for_ids.argtypes = [_p, _p, _i64, ctypes.c_int, ctypes.c_int, _p]
        L.oracle_dispatch.argtypes = [_p, _i64, ctypes.c_int, ctypes.c_int, _p, _p, _p]
        L.oracle_moe_apply.argtypes = [_p, _p, _p, _p, _p, _p, _i64, _i64, _i64,
                                       ctypes.c_int, ctypes.c_int, _p, _p, _p]
        L.oracle_moe_layer.argtypes = [_p, _p, _p, _p, _p, _p, _i64, _i64, _i64,
                                       ctypes.c_int, ctypes.c_int, _p, _p, _p, _p]
        L.oracle_rmsnorm.argtypes = [_p, _p, _i64, _i64, _f64, _p]
        L.oracle_fp8_e4m3.argtypes = [_p, _i64, _p]
        L.oracle_moe_apply_fp8.argtypes = [_p, _p, _p, _p, _p, _p, _p, _p, _p, _i64, _i64, _i64,
                                           ctypes.c_int, ctypes.c_int, _p, _p, _p]
        L.oracle_moe_layer_fp8.argtypes = [_p, _p, _p, _p, _p, _p, _p, _p, _p, _i64, _i64, _i64,
                                           ctypes.c_int, ctypes.c_int, _p, _p, _p, _p]
        L.oracle_round_bf16.argtypes = [_p, _i64, _p]
        L.oracle_rope.argtypes = [_p, _i64, ctypes.c_int, ctypes.c_int, _p, _f64]
        L.oracle_attention_decode.argtypes = [_p, _p, _p, _p, _i64, _i64, _p, _i64, ctypes.c_int,
                                              ctypes.c_int, ctypes.c_int, ctypes.c_int, _f64, _p]
        for f in ("oracle_router_logits", "oracle_topk_gate", "oracle_gates_for_ids", "oracle_dispatch",
                  "oracle_moe_apply", "oracle_moe_layer", "oracle_rmsnorm", "oracle_fp8_e4m3",
                  "oracle_moe_apply_fp8", "oracle_moe_layer_fp8", "oracle_round_bf16", "oracle_rope",
                  "oracle_attention_decode"):
            getattr(L, f).restype = ctypes.c_int

    # -- helpers -----------------------------------------------------------
    @staticmethod
    def _bits(a, shape=None):
        a = np.ascontiguousarray(a)
        if a.dtype != np.uint16:
            raise TypeError("bf16 operands are passed as uint16 bit patterns")
        if shape is not None and a.shape != tuple(shape):
            raise ValueError(f"shape {a.shape} != {tuple(shape)}")
        return a

    @staticmethod
    def _ptr(a):
        return None if a is None else a.ctypes.data

    @staticmethod
    def _check(rc, what):
        if rc != 0:
            raise OracleError(f"{what} failed with code {rc}")

    def threads(self, n: int = 0) -> int:
        """Set (n>0) and return the OpenMP thread count."""
        return self.lib.oracle_threads(n)

    # -- API -----------------------------------------------------------------
    def router_logits(self, x, wr, bias=None):
        T, d = x.shape
        E = wr.shape[0]
        x, wr = self._bits(x), self._bits(wr, (E, d))
        b = None if bias is None else np.ascontiguousarray(bias, dtype=np.float32)
        out = np.empty((T, E), np.float64)
        self._check(self.lib.oracle_router_logits(self._ptr(x), self._ptr(wr), self._ptr(b),
                                                  T, d, E, self._ptr(out)), "router_logits")
        return out

    def topk_gate(self, logits, k):
        logits = np.ascontiguousarray(logits, dtype=np.float64)
        T, E = logits.shape
        ids = np.empty((T, k), np.int32)
        gates = np.empty((T, k), np.float64)
        self._check(self.lib.oracle_topk_gate(self._ptr(logits), T, E, k, self._ptr(ids),
                                              self._ptr(gates)), "topk_gate")
        return ids, gates

    def gates_for_ids(self, logits, ids):
        logits = np.ascontiguousarray(logits, dtype=np.float64)
        ids = np.ascontiguousarray(ids, dtype=np.int32)
        T, E = logits.shape
        k = ids.shape[1]
        gates = np.empty((T, k), np.float64)
        self._check(self.lib.oracle_gates_for_ids(self._ptr(logits), self._ptr(ids), T, E, k,
                                                  self._ptr(gates)), "gates_for_ids")
        return gates

    def dispatch(self, ids, E):
        ids = np.ascontiguousarray(ids, dtype=np.int32)
        T, k = ids.shape
        counts = np.empty(E, np.int32)
        offsets = np.empty(E + 1, np.int32)
        perm = np.empty(T * k, np.int32)
        self._check(self.lib.oracle_dispatch(self._ptr(ids), T, E, k, self._ptr(counts),
                                             self._ptr(offsets), self._ptr(perm)), "dispatch")
        return counts, offsets, perm

    def moe_apply(self, x, w1, w3, w2, ids, gates, want_slots=False):
        T, d = x.shape
        E, ffn, _ = w1.shape
        ids = np.ascontiguousarray(ids, dtype=np.int32)
        gates = np.ascontiguousarray(gates, dtype=np.float64)
        k = ids.shape[1]
        x = self._bits(x)
        w1, w3 = self._bits(w1, (E, ffn, d)), self._bits(w3, (E, ffn, d))
        w2 = self._bits(w2, (E, d, ffn))
        out = np.empty((T, d), np.float64)
        h = np.empty((T * k, ffn), np.float64) if want_slots else None
        y = np.empty((T * k, d), np.float64) if want_slots else None
        self._check(self.lib.oracle_moe_apply(
            self._ptr(x), self._ptr(w1), self._ptr(w3), self._ptr(w2), self._ptr(ids),
            self._ptr(gates), T, d, ffn, E, k, self._ptr(out), self._ptr(h), self._ptr(y)),
            "moe_apply")
        return (out, h, y) if want_slots else out

    def moe_layer(self, x, wr, w1, w3, w2, k, bias=None):
        """Returns dict(out, logits, ids, gates) for the whole layer."""
        T, d = x.shape
        E, ffn, _ = w1.shape
        x, wr = self._bits(x), self._bits(wr, (E, d))
        w1, w3 = self._bits(w1, (E, ffn, d)), self._bits(w3, (E, ffn, d))
        w2 = self._bits(w2, (E, d, ffn))
        b = None if bias is None else np.ascontiguousarray(bias, dtype=np.float32)
        out = np.empty((T, d), np.float64)
        logits = np.empty((T, E), np.float64)
        ids = np.empty((T, k), np.int32)
        gates = np.empty((T, k), np.float64)
        self._check(self.lib.oracle_moe_layer(
            self._ptr(x), self._ptr(wr), self._ptr(b), self._ptr(w1), self._ptr(w3),
            self._ptr(w2), T, d, ffn, E, k, self._ptr(out), self._ptr(logits), self._ptr(ids),
            self._ptr(gates)), "moe_layer")
        return {"out": out, "logits": logits, "ids": ids, "gates": gates}

    @staticmethod
    def _u8(a, shape=None):
        a = a.cpu().numpy() if hasattr(a, "cpu") else a
        a = np.ascontiguousarray(a, dtype=np.uint8)
        if shape is not None:
            assert a.shape == tuple(shape), (a.shape, shape)
        return a

    @staticmethod
    def _f32(a, shape=None):
        a = a.cpu().numpy() if hasattr(a, "cpu") else a
        a = np.ascontiguousarray(a, dtype=np.float32)
        if shape is not None:
            assert a.shape == tuple(shape), (a.shape, shape)
        return a

    def fp8_e4m3(self, q):
        q = self._u8(q)
        out = np.empty(q.shape, np.float64)
        self._check(self.lib.oracle_fp8_e4m3(self._ptr(q), q.size, self._ptr(out)), "fp8_e4m3")
        return out

    def _fp8_weights(self, w1q, w1s, w3q, w3s, w2q, w2s, d):
        E, ffn = w1s.shape
        return (self._u8(w1q, (E, ffn, d)), self._f32(w1s, (E, ffn)), self._u8(w3q, (E, ffn, d)),
                self._f32(w3s, (E, ffn)), self._u8(w2q, (E, d, ffn)), self._f32(w2s, (E, d)))

    def moe_apply_fp8(self, x, w1q, w1s, w3q, w3s, w2q, w2s, ids, gates, want_slots=False):
        T, d = x.shape
        ws = self._fp8_weights(w1q, w1s, w3q, w3s, w2q, w2s, d)
        E, ffn = ws[1].shape
        ids = np.ascontiguousarray(ids, dtype=np.int32)
        gates = np.ascontiguousarray(gates, dtype=np.float64)
        k = ids.shape[1]
        x = self._bits(x)
        out = np.empty((T, d), np.float64)
        h = np.empty((T * k, ffn), np.float64) if want_slots else None
        y = np.empty((T * k, d), np.float64) if want_slots else None
        self._check(self.lib.oracle_moe_apply_fp8(
            self._ptr(x), *[self._ptr(a) for a in ws], self._ptr(ids), self._ptr(gates),
            T, d, ffn, E, k, self._ptr(out), self._ptr(h), self._ptr(y)), "moe_apply_fp8")
        return (out, h, y) if want_slots else out

    def moe_layer_fp8(self, x, wr, w1q, w1s, w3q, w3s, w2q, w2s, k, bias=None):
        """The layer with E4M3 expert weights; returns dict(out, logits, ids, gates)."""
        T, d = x.shape
        ws = self._fp8_weights(w1q, w1s, w3q, w3s, w2q, w2s, d)
        E, ffn = ws[1].shape
        x, wr = self._bits(x), self._bits(wr, (E, d))
        b = None if bias is None else np.ascontiguousarray(bias, dtype=np.float32)
        out = np.empty((T, d), np.float64)
        logits = np.empty((T, E), np.float64)
        ids = np.empty((T, k), np.int32)
        gates = np.empty((T, k), np.float64)
        self._check(self.lib.oracle_moe_layer_fp8(
            self._ptr(x), self._ptr(wr), self._ptr(b), *[self._ptr(a) for a in ws],
            T, d, ffn, E, k, self._ptr(out), self._ptr(logits), self._ptr(ids), self._ptr(gates)),
            "moe_layer_fp8")
        return {"out": out, "logits": logits, "ids": ids, "gates": gates}

    def rmsnorm(self, h, gamma, eps):
        h = np.ascontiguousarray(h, dtype=np.float32)
        T, d = h.shape
        gamma = self._bits(gamma, (d,))
        a = np.empty((T, d), np.float64)
        self._check(self.lib.oracle_rmsnorm(self._ptr(h), self._ptr(gamma), T, d, float(eps),
                                            self._ptr(a)), "rmsnorm")
        return a

    # -- the decoder layer around the MoE block (one decode step) --------------

    def round_bf16(self, x):
        """float64 -> bf16 bit patterns, round to nearest, ties to even."""
        x = np.ascontiguousarray(x, dtype=np.float64)
        out = np.empty(x.shape, np.uint16)
        self._check(self.lib.oracle_round_bf16(self._ptr(x), x.size, self._ptr(out)), "round_bf16")
        return out

    def rope(self, x, pos, base):
        """RoPE of x [T, H, hd] (float64) at positions pos [T]; returns a copy."""
        x = np.array(x, dtype=np.float64, order="C", copy=True)
        T, H, hd = x.shape
        pos = np.ascontiguousarray(pos, dtype=np.int32)
        self._check(self.lib.oracle_rope(self._ptr(x), T, H, hd, self._ptr(pos), float(base)), "rope")
        return x

    def attention_decode(self, q, k_cache, v_cache, page_table, ctx, scale):
        """q [T, Hq, hd] float64; caches [pages, Hkv, page, hd] bf16 bits;
        page_table [T, maxp] int32; ctx [T] positions attended per token."""
        q = np.ascontiguousarray(q, dtype=np.float64)
        T, Hq, hd = q.shape
        P, Hkv, page, hd2 = k_cache.shape
        assert hd2 == hd and v_cache.shape == k_cache.shape
        kc, vc = self._bits(k_cache), self._bits(v_cache)
        pt = np.ascontiguousarray(page_table, dtype=np.int32)
        ctx = np.ascontiguousarray(ctx, dtype=np.int32)
        out = np.empty((T, Hq, hd), np.float64)
        self._check(self.lib.oracle_attention_decode(
            self._ptr(q), self._ptr(kc), self._ptr(vc), self._ptr(pt), pt.shape[1], P, self._ptr(ctx),
            T, Hq, Hkv, hd, page, float(scale), self._ptr(out)), "attention_decode")
        return out

    def decoder_layer(self, h, gamma_attn, wq, wk, wv, wo, k_cache, v_cache, page_table, pos,
                      gamma_moe, wr, w1, w3, w2, k, hq, hkv, theta, eps, fp8_experts=None):
        """One decode step of a decoder layer for T tokens (one per request):
        h [T, d] float32 residual stream; projections bf16 bits (nn.Linear
        layout: wq [hq*hd, d], wk, wv [hkv*hd, d], wo [d, hq*hd]); the new
        token of request t sits at position pos[t] (pos[t] earlier positions
        are in the cache).  Returns the intermediates and the layer output
        h2 (float64); the caches passed in are not modified (copies with the
        new entries are returned).  fp8_experts: (w1q, w1s, w3q, w3s, w2q, w2s)
        to run the MoE block on 8-bit expert weights (then w1, w3, w2 are
        unused)."""
        h = np.ascontiguousarray(h, dtype=np.float32)
        T, d = h.shape
        hd = wq.shape[0] // hq
        a = self.round_bf16(self.rmsnorm(h, gamma_attn, eps))
        af = a.astype(np.uint32) << 16
        A = af.view(np.float32).astype(np.float64)

        def lin(w):
            wf = (self._bits(w).astype(np.uint32) << 16).view(np.float32).astype(np.float64)
            return A @ wf.T

        q = self.rope(lin(wq).reshape(T, hq, hd), pos, theta)
        kn = self.rope(lin(wk).reshape(T, hkv, hd), pos, theta)
        vn = lin(wv).reshape(T, hkv, hd)
        kc, vc = np.array(k_cache, copy=True), np.array(v_cache, copy=True)
        page = kc.shape[2]
        pos = np.asarray(pos, dtype=np.int64)
        for t in range(T):
            pg = page_table[t, pos[t] // page]
            kc[pg, :, pos[t] % page, :] = self.round_bf16(kn[t])
            vc[pg, :, pos[t] % page, :] = self.round_bf16(vn[t])
        o = self.attention_decode(q, kc, vc, page_table, pos + 1, 1.0 / np.sqrt(hd))
        wof = (self._bits(wo).astype(np.uint32) << 16).view(np.float32).astype(np.float64)
        h1 = h.astype(np.float64) + o.reshape(T, hq * hd) @ wof.T
        # the residual stream is kept in float32 between the two blocks
        h1f = h1.astype(np.float32)
        a2 = self.round_bf16(self.rmsnorm(h1f, gamma_moe, eps))
        if fp8_experts is not None:
            moe = self.moe_layer_fp8(a2, wr, *fp8_experts, k)
        else:
            moe = self.moe_layer(a2, wr, w1, w3, w2, k)
        h2 = h1f.astype(np.float64) + moe["out"]
        return {"a": a, "q": q, "k_new": kn, "v_new": vn, "k_cache": kc, "v_cache": vc,
                "attn": o, "h1": h1, "a2": a2, "moe": moe, "h2": h2}


_default = None


def get() -> Oracle:
    global _default
    if _default is None:
        _default = Oracle()
    return _default
