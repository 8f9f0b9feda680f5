"""One decoder layer of the served model (Mixtral-8x7B) for a decode step,
sequenced on the device through the C ABI of libmoe.

Per token t (one per request; the new token sits at position pos[t]):

    a   = bf16(RMSNorm(h) * gamma_attn)              moe_rmsnorm
    qkv = a [Wq; Wk; Wv]^T                            moe_linear (one fused matrix)
    RoPE(q, k); k, v -> paged cache                   moe_rope_kv_append
    o   = attention over the request's positions      moe_attention_decode
    h  += o Wo^T                                      moe_linear + moe_combine (k = 1)
    h  += MoE(bf16(RMSNorm(h) * gamma_moe))           moe_rmsnorm + moe_forward_ex

h is the float32 residual stream and is updated in place.  Every step runs in
the library's HIP kernels; torch only provides the buffers and the stream.
The sequence issues no host synchronisation, so a step can be captured into a
HIP graph.
"""

from __future__ import annotations

import math

import torch

from . import binding as B


class DecoderLayer:
    """Weights of one layer, kept resident: the query/key/value projections
    are stored as one [(hq + 2 hkv) hd, d] matrix (a layout choice made once,
    at load time), so one streaming GEMM reads them all."""

    def __init__(self, attn: dict, moe: dict, hq: int, hkv: int, k: int, theta: float,
                 eps: float = 1e-5):
        self.wqkv = torch.cat([attn["wq"], attn["wk"], attn["wv"]], dim=0).contiguous()
        self.wo = attn["wo"].contiguous()
        self.gamma_attn, self.gamma_moe = attn["gamma_attn"], attn["gamma_moe"]
        self.router_w, self.router_bias = moe["router_w"], moe.get("router_bias")
        # expert weights: bf16 (w1, w3, w2) or E4M3 bytes with row scales
        self.fp8 = "w1q" in moe
        if self.fp8:
            self.q = [moe[n] for n in ("w1q", "w1s", "w3q", "w3s", "w2q", "w2s")]
        else:
            self.w1, self.w3, self.w2 = moe["w1"], moe["w3"], moe["w2"]
        self.hq, self.hkv, self.k, self.theta, self.eps = hq, hkv, k, theta, eps
        self.d = self.wo.shape[0]
        self.hd = self.wo.shape[1] // hq
        self._bufs = {}

    def buffers(self, T: int, device):
        """Per-step scratch for T tokens (allocated once per T)."""
        if T not in self._bufs:
            d, nqkv, nq = self.d, self.wqkv.shape[0], self.hq * self.hd
            self._bufs[T] = {
                "a": torch.empty(T, d, dtype=torch.bfloat16, device=device),
                "qkv": torch.empty(T, nqkv, dtype=torch.float32, device=device),
                "q": torch.empty(T, self.hq, self.hd, dtype=torch.bfloat16, device=device),
                "attn": torch.empty(T, nq, dtype=torch.bfloat16, device=device),
                "o": torch.empty(T, d, dtype=torch.float32, device=device),
                "a2": torch.empty(T, d, dtype=torch.bfloat16, device=device),
            }
        return self._bufs[T]

    def step(self, h, k_cache, v_cache, page_table, pos, ctx, stream=None):
        """One decode step for the T tokens of h [T, d] (float32, updated in
        place).  pos [T]: the new token's position; ctx [T] = pos + 1, the
        positions attended (engine metadata, like the page table)."""
        T = h.shape[0]
        b = self.buffers(T, h.device)
        B.moe_rmsnorm(h, self.gamma_attn, self.eps, b["a"], stream=stream)
        B.moe_linear(b["a"], self.wqkv, b["qkv"], stream=stream)
        B.moe_rope_kv_append(b["qkv"], pos, page_table, self.hq, self.hkv, self.theta, b["q"],
                             k_cache, v_cache, stream=stream)
        B.moe_attention_decode(b["q"], k_cache, v_cache, page_table, ctx,
                               1.0 / math.sqrt(self.hd), b["attn"], stream=stream)
        B.moe_linear(b["attn"], self.wo, b["o"], stream=stream)
        B.moe_combine(b["o"], T, self.d, 1, out_f32=h, residual=h, stream=stream)
        B.moe_rmsnorm(h, self.gamma_moe, self.eps, b["a2"], stream=stream)
        self.moe_block(b["a2"], h, stream)
        return h

    def moe_block(self, a2, h, stream=None):
        """h += MoE(a2), the f32 residual updated in place."""
        if self.fp8:
            B.moe_forward_fp8_ex(a2, self.router_w, *self.q, self.k, out_f32=h,
                                 router_bias=self.router_bias, residual=h, stream=stream)
        else:
            B.moe_forward_ex(a2, self.router_w, self.w1, self.w3, self.w2, self.k, out_f32=h,
                             router_bias=self.router_bias, residual=h, stream=stream)


class DecoderStack:
    """w.layers decoder layers with their own weights and KV caches (all
    resident), sharing the requests' page table and positions.  A step runs
    every layer in order; it can be captured once into a HIP graph."""

    def __init__(self, w, device="cuda:0"):
        from . import inputs

        self.w = w
        self.layers, self.caches = [], []
        for l in range(w.layers):
            attn = inputs.make_attention(w, l, device)
            moe = inputs.make_layer_fp8(w, l, device) if w.fp8 else inputs.make_layer(w, l, device)
            kv = inputs.make_kv_cache(w, l, device)
            self.layers.append(DecoderLayer(attn, moe, w.hq, w.hkv, w.k, w.theta, w.eps))
            self.caches.append((kv["k_cache"], kv["v_cache"]))
            self.page_table, self.pos, self.ctx = kv["page_table"], kv["pos"], kv["ctx"]
        self.graph = None

    def step(self, h, stream=None):
        for layer, (kc, vc) in zip(self.layers, self.caches):
            layer.step(h, kc, vc, self.page_table, self.pos, self.ctx, stream=stream)
        return h

    def capture(self, h):
        """Capture one step on h's buffer (run it once eagerly first, so that
        every scratch buffer exists)."""
        self.step(h)
        torch.cuda.synchronize()
        s = torch.cuda.Stream()
        self.graph = torch.cuda.CUDAGraph()
        with torch.cuda.stream(s):
            with torch.cuda.graph(self.graph, stream=s):
                self.step(h, stream=s)
        torch.cuda.synchronize()

    def replay(self):
        self.graph.replay()


def bench_decoder_stack(args, w):
    """bench.py for a stack of decoder layers: one decode step of the whole
    model (graph replays).  Returns the JSON record (its CPU baseline left
    for bench.py) and what that baseline needs: the first layer, its cache,
    the page table, positions and the residual stream."""
    import time

    import numpy as np

    from . import inputs

    HBM_PEAK_GBS = 8000.0
    st = DecoderStack(w)
    h = inputs.make_h(w, "cuda:0")
    st.capture(h)
    stream = torch.cuda.current_stream()
    for _ in range(args.warmup):
        st.replay()
    torch.cuda.synchronize()
    bounds = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    t0 = time.perf_counter()
    bounds[0].record(stream)
    for i in range(args.steps):
        st.replay()
        bounds[i + 1].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms = bounds[0].elapsed_time(bounds[-1]) / args.steps
    step_ms = np.array([bounds[i].elapsed_time(bounds[i + 1]) for i in range(args.steps)])
    T, d = w.T, w.d
    ctx = st.ctx.cpu().numpy().astype(np.int64)
    kv_bytes = int(ctx.sum()) * w.hkv * w.hd * 2 * 2
    proj_bytes = (st.layers[0].wqkv.numel() + st.layers[0].wo.numel()) * 2
    expert_bytes = w.E * 3 * w.ffn * d * (1 if w.fp8 else 2) + w.E * (2 * w.ffn + d) * 4 * w.fp8
    layer_bytes = proj_bytes + expert_bytes + w.E * d * 2 + kv_bytes + T * d * 4 * 2
    step_bytes = w.layers * layer_bytes
    gbs = step_bytes / (ms * 1e-3) / 1e9
    rec = {
        "metric": "model decode tokens/s",
        "value": round(T / (ms * 1e-3), 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "step_ms_p10_p50_p90": [round(float(np.percentile(step_ms, q)), 4) for q in (10, 50, 90)],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded normals: %d random-init Mixtral-8x7B decoder layers%s, random KV caches)"
                % (w.layers, ", E4M3 expert weights" if w.fp8 else ""),
        "config": {"workload": args.workload, "T": T, "d": d, "ffn": w.ffn, "E": w.E, "k": w.k,
                   "layers": w.layers, "hq": w.hq, "hkv": w.hkv, "hd": w.hd, "page": w.page,
                   "cached_positions_per_layer": int(ctx.sum() - T), "graph": True},
        "roofline": {"bound": "hbm", "achieved": round(gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(gbs / HBM_PEAK_GBS, 4), "traffic": None,
                     "kernel": "whole step (%d x attention block + MoE block)" % w.layers,
                     "algorithmic_bytes_per_launch": step_bytes},
        "cpu_baseline": None,
        "wall_s_timed": round(wall, 3),
    }
    return rec, (st.layers[0], st.caches[0], st.page_table, st.pos, h)


def bench_decoder(args, w):
    """bench.py for a decoder-layer workload: one decode step of the layer
    for w.T requests.  Each step rewrites the same cache slot and advances
    h, so every step does the same work.  Returns the JSON record (its CPU
    baseline left for bench.py) and the layer, cache, page table, positions
    and residual stream that baseline needs."""
    if w.layers > 1:
        return bench_decoder_stack(args, w)
    import time

    import numpy as np

    from . import inputs

    HBM_PEAK_GBS = 8000.0
    dev = "cuda:0"
    attn = inputs.make_attention(w, 0, dev)
    moe = inputs.make_layer_fp8(w, 0, dev) if w.fp8 else inputs.make_layer(w, 0, dev)
    kv = inputs.make_kv_cache(w, 0, dev)
    layer = DecoderLayer(attn, moe, w.hq, w.hkv, w.k, w.theta, w.eps)
    h = inputs.make_h(w, dev)
    stream = torch.cuda.current_stream()
    T, d = w.T, w.d
    b = layer.buffers(T, h.device)

    def step(ev=None):
        B.moe_rmsnorm(h, layer.gamma_attn, layer.eps, b["a"], stream=stream)
        B.moe_linear(b["a"], layer.wqkv, b["qkv"], stream=stream)
        B.moe_rope_kv_append(b["qkv"], kv["pos"], kv["page_table"], w.hq, w.hkv, w.theta, b["q"],
                             kv["k_cache"], kv["v_cache"], stream=stream)
        if ev is not None:
            ev[0].record(stream)
        B.moe_attention_decode(b["q"], kv["k_cache"], kv["v_cache"], kv["page_table"], kv["ctx"],
                               1.0 / math.sqrt(layer.hd), b["attn"], stream=stream)
        if ev is not None:
            ev[1].record(stream)
        B.moe_linear(b["attn"], layer.wo, b["o"], stream=stream)
        B.moe_combine(b["o"], T, d, 1, out_f32=h, residual=h, stream=stream)
        B.moe_rmsnorm(h, layer.gamma_moe, layer.eps, b["a2"], stream=stream)
        layer.moe_block(b["a2"], h, stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(args.steps)]
    bounds = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    t0 = time.perf_counter()
    bounds[0].record(stream)
    for i in range(args.steps):
        step(evs[i])
        bounds[i + 1].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms = bounds[0].elapsed_time(bounds[-1]) / args.steps
    step_ms = np.array([bounds[i].elapsed_time(bounds[i + 1]) for i in range(args.steps)])
    attn_us = float(np.mean([a.elapsed_time(z) for a, z in evs])) * 1e3

    # algorithmic bytes: every weight once (attention projections, router,
    # the routed experts), the cached keys/values each request attends to,
    # the new key/value rows and the residual stream in and out
    ctx = kv["ctx"].cpu().numpy().astype(np.int64)
    kv_bytes = int(ctx.sum()) * w.hkv * w.hd * 2 * 2
    proj_bytes = (layer.wqkv.numel() + layer.wo.numel()) * 2
    ids = torch.empty(T, w.k, dtype=torch.int32, device=dev)
    gw = torch.empty(T, w.k, dtype=torch.float32, device=dev)
    offs = torch.empty(w.E + 1, dtype=torch.int32, device=dev)
    perm = torch.empty(T * w.k, dtype=torch.int32, device=dev)
    B.moe_route(b["a2"], layer.router_w, w.k, ids, gw, offs, perm)
    active = int((torch.diff(offs) > 0).sum())
    moe_bytes = (active * 3 * w.ffn * d * (1 if w.fp8 else 2) + active * (2 * w.ffn + d) * 4 * w.fp8
                 + w.E * d * 2)
    step_bytes = proj_bytes + moe_bytes + kv_bytes + T * d * 4 * 2
    gbs = step_bytes / (ms * 1e-3) / 1e9
    attn_gbs = kv_bytes / (attn_us * 1e-6) / 1e9
    rec = {
        "metric": "decoder-layer tokens/s",
        "value": round(T / (ms * 1e-3), 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "step_ms_p10_p50_p90": [round(float(np.percentile(step_ms, q)), 4) for q in (10, 50, 90)],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded normals: one random-init Mixtral-8x7B decoder layer, random KV cache)",
        "config": {"workload": args.workload, "T": T, "d": d, "ffn": w.ffn, "E": w.E, "k": w.k,
                   "hq": w.hq, "hkv": w.hkv, "hd": w.hd, "page": w.page,
                   "cached_positions": int(ctx.sum() - T), "active_experts": active},
        "roofline": {"bound": "hbm", "achieved": round(gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(gbs / HBM_PEAK_GBS, 4), "traffic": None,
                     "kernel": "whole step (attention block + MoE block)",
                     "algorithmic_bytes_per_launch": step_bytes},
        "attention": {"avg_launch_us": round(attn_us, 2), "kv_bytes": kv_bytes,
                      "achieved_gbs": round(attn_gbs, 1), "frac": round(attn_gbs / HBM_PEAK_GBS, 4)},
        "cpu_baseline": None,
        "wall_s_timed": round(wall, 3),
    }
    return rec, (layer, (kv["k_cache"], kv["v_cache"]), kv["page_table"], kv["pos"], h)
