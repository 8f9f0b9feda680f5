"""A stack of MoE layers with pre-norm residual blocks, one decode step.

Each block l computes, with the residual stream h kept in f32,

    a_l     = bf16( RMSNorm(h_l) * gamma_l )          moe_rmsnorm
    h_{l+1} = h_l + MoE_l(a_l)                          moe_forward_ex(residual=h, out_f32=h)

which is the layer structure of Mixtral's decoder with the attention block
left out (the paper's engine serves Mixtral-8x7B, Sec. 4.1 and Sec. 5).  All
arithmetic runs in the library's kernels; this module only owns buffers and
sequences the C ABI calls, optionally captured once into a HIP graph (through
torch.cuda.CUDAGraph) so a 32-layer step is a single launch.
"""

from __future__ import annotations

import time
from typing import List, Optional

import torch

from . import binding as B
from . import inputs


class MoeStack:
    def __init__(self, w: inputs.Workload, device="cuda:0", layers: Optional[int] = None,
                 gamma_random: bool = False):
        self.w = w
        self.device = device
        self.L = w.layers if layers is None else layers
        self.layers: List[dict] = []
        for l in range(self.L):
            lay = inputs.make_layer(w, l, device)
            lay["gamma"] = inputs.make_gamma(w, l, device, random=gamma_random)
            self.layers.append(lay)
        T, d = w.T, w.d
        self.h = torch.empty(T, d, dtype=torch.float32, device=device)
        self.a = torch.empty(T, d, dtype=torch.bfloat16, device=device)
        ws = B.moe_workspace_size(T, d, w.ffn, w.E, w.k)
        self.ws = torch.empty(ws, dtype=torch.uint8, device=device)
        self.graph = None

    def load_input(self, x: torch.Tensor):
        self.h.copy_(x.float())

    def layer(self, l: int, stream=None):
        lay = self.layers[l]
        B.moe_rmsnorm(self.h, lay["gamma"], self.w.eps, self.a, stream=stream)
        B.moe_forward_ex(self.a, lay["router_w"], lay["w1"], lay["w3"], lay["w2"], self.w.k,
                         out_f32=self.h, residual=self.h, router_bias=lay["router_bias"],
                         workspace=self.ws, stream=stream)

    def step(self, stream=None):
        for l in range(self.L):
            self.layer(l, stream)

    def capture(self, x: torch.Tensor):
        """Records one whole step -- x copied into the residual stream, then
        every layer -- into a HIP graph.  x must stay allocated; replays read
        its current contents."""
        self.x_graph = x
        s = torch.cuda.Stream(device=self.device)
        s.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(s):
            self.load_input(x)
            self.step(stream=s)  # warm-up outside capture
        torch.cuda.current_stream().wait_stream(s)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=s):
            self.load_input(x)
            self.step(stream=s)
        self.graph = g
        return g

    def replay(self):
        self.graph.replay()

    def trace(self, x: torch.Tensor, layers=None):
        """Runs the step layer by layer, returning (h_l, a_l, h_{l+1}) copies
        for the requested layers (for per-layer parity checks)."""
        self.load_input(x)
        want = set(range(self.L) if layers is None else layers)
        out = {}
        for l in range(self.L):
            h_in = self.h.clone() if l in want else None
            self.layer(l)
            if l in want:
                out[l] = (h_in, self.a.clone(), self.h.clone())
        torch.cuda.synchronize()
        return out


def bench_stack(args, w: inputs.Workload):
    """bench.py entry for the stack workload: graph-captured steps.  Returns
    the JSON record (its CPU baseline left for bench.py to fill in), the
    stack and its input."""
    HBM_PEAK_GBS = 8000.0
    dev = "cuda:0"
    st = MoeStack(w, dev)
    x = inputs.make_x(w, dev)
    st.capture(x)
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
    step_ms = sorted(bounds[i].elapsed_time(bounds[i + 1]) for i in range(args.steps))
    pct = [step_ms[min(len(step_ms) - 1, int(q * len(step_ms)))] for q in (0.1, 0.5, 0.9)]
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    # the same step without the graph, for the launch-overhead comparison
    st.load_input(x)
    torch.cuda.synchronize()
    e0.record(stream)
    st.step()
    e1.record(stream)
    torch.cuda.synchronize()
    ms_eager = e0.elapsed_time(e1)
    T, d, ffn, E, k = w.T, w.d, w.ffn, w.E, w.k
    layer_bytes = E * 3 * ffn * d * 2 + E * d * 2 + T * d * 2 * 2
    step_bytes = st.L * layer_bytes
    gbs = step_bytes / (ms * 1e-3) / 1e9
    rec = {
        "metric": "MoE-layer tokens/s",
        "value": round(T / (ms * 1e-3), 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "step_ms_p10_p50_p90": [round(v, 4) for v in pct],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded normals, 32 random-init Mixtral-8x7B MoE layers)",
        "config": {"workload": args.workload, "T": T, "d": d, "ffn": ffn, "E": E, "k": k,
                   "layers": st.L, "eps": w.eps, "graph": True, "ms_per_step_eager": round(ms_eager, 4)},
        "roofline": {"bound": "hbm", "achieved": round(gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(gbs / HBM_PEAK_GBS, 4), "traffic": None,
                     "kernel": "whole step (32 x rmsnorm + MoE layer)",
                     "algorithmic_bytes_per_launch": step_bytes},
        "cpu_baseline": None,
        "wall_s_timed": round(wall, 3),
    }
    return rec, st, x
