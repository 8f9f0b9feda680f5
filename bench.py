"""Benchmark of the MoE FFN layer on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload decode_t64]

A step is one pass of the whole layer over one batch of T tokens already
resident in HBM: router GEMM + top-k + dispatch, the SwiGLU up GEMM (with the
row gather fused in), the down GEMM with the gate-weighted scatter, and the
combine.  The step time is K `moe_forward_ex` calls back to back; the
roofline of the dominant kernel comes from a second timed pass of the same
kernels issued stage by stage through the C ABI, so that HIP events can
bracket every launch of it on the stream it runs on.

Prints one JSON line: tokens/s of the layer, the roofline of the dominant
kernel (algorithmic bytes or FLOPs per launch over its event-timed duration),
and the fp64 CPU oracle timed on a bounded sample of the same workload.
"""

from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0  # MI355X HBM3E, published
BF16_PEAK_TFLOPS = 2500.0  # MI355X dense bf16 MFMA, published

KERNEL_SOURCES = {"stream": "paper_2408_00008_amd/csrc/expert_stream.hip",
                  "tiled": "paper_2408_00008_amd/csrc/expert_tiled.hip",
                  "split": "paper_2408_00008_amd/csrc/expert_stream.hip"}


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="decode_t64")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="target wall time of the oracle baseline sample")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-prefill", action="store_true",
                    help="decode_t64 only: skip the prefill_t4096 sub-record")
    ap.add_argument("--no-library-reference", action="store_true",
                    help="skip the hipBLASLt comparison on the tiled workloads' GEMMs")
    ap.add_argument("--prefill-steps", type=int, default=20,
                    help="timed steps of the prefill_t4096 sub-record")
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="only run a plain device copy of this many MiB (3 times), for "
                         "scaling rocprofv3 FETCH_SIZE/WRITE_SIZE counters")
    return ap.parse_args()


def copy_calibration(mib: int):
    import torch

    n = mib * 1024 * 1024
    src = torch.empty(n, dtype=torch.uint8, device="cuda:0").fill_(1)
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_calibration_bytes": n, "launches": 3}), flush=True)


def source_digest(path: str) -> str:
    with open(os.path.join(ROOT, path), "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


def load_traffic(workload: str, kernel: str, family: str):
    """HBM bytes per launch from committed rocprofv3 counter runs, if they were
    taken on the kernel source as it is now."""
    path = os.path.join(ROOT, "profiles", f"traffic_{kernel}_{workload}.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f)
    if rec.get("source_sha256_16") != source_digest(KERNEL_SOURCES[family]):
        return None
    return rec.get("hbm_bytes_per_launch")


def main():
    args = parse()
    if args.copy_calibration_mib:
        return copy_calibration(args.copy_calibration_mib)
    if args.gpus != 1:
        print(f"bench.py: the MoE layer is measured on exactly one GPU (asked for --gpus "
              f"{args.gpus}); runs over several GPUs are not supported", file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_2408_00008_amd import inputs

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    w = inputs.WORKLOADS[args.workload].replace(seed=args.seed)
    if w.hq:
        from paper_2408_00008_amd import decoder
        rec, state = decoder.bench_decoder(args, w)
        rec["cpu_baseline"] = None if args.no_cpu_baseline else cpu_baseline_decoder(args, w, *state)
        print(json.dumps(rec), flush=True)
        return
    if w.layers != 1:
        from paper_2408_00008_amd import stack
        rec, st, x = stack.bench_stack(args, w)
        rec["cpu_baseline"] = None if args.no_cpu_baseline else cpu_baseline_stack(args, w, st, x)
        print(json.dumps(rec), flush=True)
        return
    rec, state = measure_layer(args, w, args.steps, args.warmup)
    rec["cpu_baseline"] = None if args.no_cpu_baseline else cpu_baseline(args, w, *state)
    del state
    if args.workload == "decode_t64" and not args.no_prefill:
        # the metric's second half: the 4096-token prefill chunk against the
        # bf16 MFMA peak, measured in the same run
        pw = inputs.WORKLOADS["prefill_t4096"].replace(seed=args.seed)
        sub, pstate = measure_layer(args, pw, args.prefill_steps, args.warmup)
        sub["cpu_baseline"] = None if args.no_cpu_baseline else cpu_baseline(args, pw, *pstate)
        del pstate
        for key in ("metric", "n_gpus", "higher_is_better", "scaling", "vs_baseline", "dtype",
                    "data"):
            sub.pop(key, None)
        rec["prefill_t4096"] = sub
    print(json.dumps(rec), flush=True)


def measure_layer(args, w, steps, warmup):
    """Times `steps` whole-layer steps of workload w (after `warmup`) and
    returns the bench record (without the CPU baseline) and the inputs the
    baseline reuses."""
    import numpy as np
    import torch

    from paper_2408_00008_amd import binding as B
    from paper_2408_00008_amd import inputs

    dev = "cuda:0"
    T, d, ffn, E, k = w.T, w.d, w.ffn, w.E, w.k
    A = T * k
    x = inputs.make_x(w, dev)
    if w.fp8:
        # E4M3 expert weights with per-row f32 scales
        lay = inputs.make_layer_fp8(w, 0, dev)
        q = [lay[n] for n in ("w1q", "w1s", "w3q", "w3s", "w2q", "w2s")]
        wbytes_per_elem = 1
    else:
        lay = inputs.make_layer(w, 0, dev)
        w1, w3, w2 = lay["w1"], lay["w3"], lay["w2"]
        wbytes_per_elem = 2
    rw, bias = lay["router_w"], lay["router_bias"]

    ids = torch.empty(T, k, dtype=torch.int32, device=dev)
    gw = torch.empty(T, k, dtype=torch.float32, device=dev)
    offs = torch.empty(E + 1, dtype=torch.int32, device=dev)
    perm = torch.empty(A, dtype=torch.int32, device=dev)
    h = torch.empty(A, ffn, dtype=torch.bfloat16, device=dev)
    # as in moe_forward, the down GEMM may cut its reduction into parts written
    # as separate slices: up to 4 where the tiled kernels run, up to 2 for
    # the heavy experts of a split streaming step
    variant = {1: "stream", 2: "tiled", 3: "split"}[B.moe_gemm_variant_for(T, d, ffn, E, k)]
    cut = variant in ("tiled", "split")
    y = torch.empty({"tiled": 4, "split": 2}[variant] if cut else 1, A, d, dtype=torch.float32,
                    device=dev)
    parts = torch.ones(1, dtype=torch.int32, device=dev)
    out = torch.empty(T, d, dtype=torch.bfloat16, device=dev)
    stream = torch.cuda.current_stream()

    def step(ev0=None, ev1=None):
        """One layer step issued stage by stage through the C ABI (the calls
        moe_forward makes internally), with events around the up kernel."""
        B.moe_route(x, rw, k, ids, gw, offs, perm, router_bias=bias, stream=stream)
        if ev0 is not None:
            ev0.record(stream)
        if w.fp8:
            B.moe_swiglu_up_fp8(x, offs, q[0], q[1], q[2], q[3], T, k, h, perm=perm, stream=stream)
        else:
            B.moe_swiglu_up(x, offs, w1, w3, T, k, h, perm=perm, stream=stream)
        if ev1 is not None:
            ev1.record(stream)
        if w.fp8 and cut:
            B.moe_swiglu_down_parts_fp8(h, offs, q[4], q[5], T, k, y, parts, topk_w=gw, perm=perm,
                                        stream=stream)
        elif w.fp8:
            B.moe_swiglu_down_fp8(h, offs, q[4], q[5], T, k, y[0], topk_w=gw, perm=perm,
                                  stream=stream)
        elif cut:
            B.moe_swiglu_down_parts(h, offs, w2, T, k, y, parts, topk_w=gw, perm=perm,
                                    stream=stream)
        else:
            B.moe_swiglu_down(h, offs, w2, T, k, y[0], topk_w=gw, perm=perm, stream=stream)
        if cut:
            B.moe_combine_parts(y, parts, T, d, k, out=out, stream=stream)
        else:
            B.moe_combine(y[0], T, d, k, out=out, stream=stream)

    # the production entry point: one moe_forward_ex call per step
    ws = torch.empty(B.moe_workspace_size(T, d, ffn, E, k), dtype=torch.uint8, device=dev)
    fout = torch.empty(T, d, dtype=torch.bfloat16, device=dev)

    def forward():
        if w.fp8:
            B.moe_forward_fp8_ex(x, rw, *q, k, out=fout, router_bias=bias, workspace=ws,
                                 stream=stream)
        else:
            B.moe_forward_ex(x, rw, w1, w3, w2, k, out=fout, router_bias=bias, workspace=ws,
                             stream=stream)

    for _ in range(warmup):
        forward()
        step()
    torch.cuda.synchronize()

    # timed region 1 (value, ms_per_step): K whole-layer steps, nothing between them
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    t0.record(stream)
    for _ in range(steps):
        forward()
    t1.record(stream)
    torch.cuda.synchronize()
    wall1 = time.perf_counter()
    ms_total = t0.elapsed_time(t1)
    ms_per_step = ms_total / steps

    # timed region 2 (roofline): K steps of the same kernels issued stage by
    # stage, HIP events around every launch of the dominant (up) kernel, plus
    # one event per step boundary for the spread of step times
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(steps)]
    bounds = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
    torch.cuda.synchronize()
    bounds[0].record(stream)
    for i in range(steps):
        step(*evs[i])
        bounds[i + 1].record(stream)
    torch.cuda.synchronize()
    step_ms = np.array([bounds[i].elapsed_time(bounds[i + 1]) for i in range(steps)])
    staged_ms = bounds[0].elapsed_time(bounds[-1]) / steps
    up_ms = sorted(e0.elapsed_time(e1) for e0, e1 in evs)
    up_avg_ms = sum(up_ms) / len(up_ms)
    # the staged step gives the production call's bits
    assert torch.equal(fout, out), "moe_forward_ex and the staged calls disagree"

    counts = np.diff(offs.cpu().numpy())
    active = int((counts > 0).sum())
    # algorithmic work of the up kernel: each active expert's w1 and w3 once
    # (bf16, or E4M3 bytes plus one f32 scale per row) and the routed token
    # rows read once; 4*d*ffn FLOP per row.  h is an intermediate and not
    # counted.
    scale_bytes = 4 if w.fp8 else 0
    up_bytes = active * 2 * ffn * (d * wbytes_per_elem + scale_bytes) + A * d * 2
    up_flops = 4.0 * A * d * ffn
    kernel = "expert_up_" + variant
    layer_flops = 2.0 * T * d * E + 6.0 * A * d * ffn
    layer_bytes = (active * (3 * ffn * d * wbytes_per_elem + (2 * ffn + d) * scale_bytes)
                   + E * d * 2 + T * d * 2 * 2)
    layer_s = ms_per_step * 1e-3
    if variant in ("stream", "split"):
        # HBM-bound (split: experts of up to 64 rows stream, heavier ones take
        # a second launch; both sit between the same two events)
        achieved = up_bytes / (up_avg_ms * 1e-3) / 1e9
        roof = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS,
                "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4)}
        lach = layer_bytes / layer_s / 1e9
        layer_roof = {"bound": "hbm", "achieved": round(lach, 1), "peak": HBM_PEAK_GBS,
                      "unit": "GB/s", "frac": round(lach / HBM_PEAK_GBS, 4)}
    else:
        achieved = up_flops / (up_avg_ms * 1e-3) / 1e12
        roof = {"bound": "mfma", "achieved": round(achieved, 1), "peak": BF16_PEAK_TFLOPS,
                "unit": "TFLOP/s", "frac": round(achieved / BF16_PEAK_TFLOPS, 4)}
        lach = layer_flops / layer_s / 1e12
        layer_roof = {"bound": "mfma", "achieved": round(lach, 1), "peak": BF16_PEAK_TFLOPS,
                      "unit": "TFLOP/s", "frac": round(lach / BF16_PEAK_TFLOPS, 4)}
    roof["traffic"] = load_traffic(w.name, kernel, variant)
    roof["kernel"] = kernel
    roof["avg_launch_us"] = round(up_avg_ms * 1e3, 2)
    roof["algorithmic_bytes_per_launch"] = up_bytes
    roof["algorithmic_flop_per_launch"] = up_flops
    layer_roof["scope"] = "whole layer step (route, up, down, combine)"
    tok_s = T * steps / (ms_total * 1e-3)

    rec = {
        "metric": "MoE-layer tokens/s",
        "value": round(tok_s, 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": steps,
        "warmup": warmup,
        "ms_per_step": round(ms_per_step, 4),
        "timing": "value/ms_per_step: K moe_forward_ex calls back to back; roofline: K staged "
                  "steps of the same kernels with events around each up launch",
        "staged_ms_per_step": round(staged_ms, 4),
        "step_ms_p10_p50_p90": [round(float(np.percentile(step_ms, q)), 4) for q in (10, 50, 90)],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",  # MFMA operands; E4M3 weights are widened exactly to bf16
        "data": "synthetic (seeded normals of the Mixtral-8x7B layer shapes; no dataset, random weights)",
        "config": {"workload": w.name, "T": T, "d": d, "ffn": ffn, "E": E, "k": k,
                   "expert_weights": "e4m3 + f32 row scale" if w.fp8 else "bf16",
                   "router_bias0": w.bias0, "seed": args.seed, "active_experts": active,
                   "rows_per_expert": counts.tolist(),
                   "down_reduction_parts": int(parts.item()) if cut else 1},
        "layer": {"tflops": round(layer_flops / layer_s / 1e12, 2),
                  "gbs": round(layer_bytes / layer_s / 1e9, 1),
                  "hbm_frac": round(layer_bytes / layer_s / 1e9 / HBM_PEAK_GBS, 4),
                  "mfma_frac": round(layer_flops / layer_s / 1e12 / BF16_PEAK_TFLOPS, 4),
                  "algorithmic_bytes": layer_bytes, "algorithmic_flop": layer_flops},
        "roofline": roof,
        "layer_roofline": layer_roof,
        "cpu_baseline": None,
        "wall_s_timed": round(wall1 - wall0, 3),
    }
    if variant == "tiled" and not w.fp8 and not args.no_library_reference:
        rec["library_reference"] = library_reference(x, perm, offs, h, lay, k, up_avg_ms)
    return rec, (x, lay, T)


def library_reference(x, perm, offs, h, lay, k, up_avg_ms, reps=10):
    """hipBLASLt (torch.matmul, bf16) on the same expert GEMMs, on the same
    GPU in the same run, for comparison with the tiled kernels: per expert e
    with M_e routed rows, up = [M_e, d] x [d, 2 ffn] (w1 and w3 as one matrix,
    the token rows already gathered, no SiLU) and down = [M_e, ffn] x [ffn, d]
    (no gate weight, no scatter) -- less work than the fused kernels do."""
    import numpy as np
    import torch

    counts = np.diff(offs.cpu().numpy())
    starts = offs.cpu().numpy()[:-1]
    src = (perm.long() // k)
    E = len(counts)
    xs, w13, hs, w2 = [], [], [], []
    for e in range(E):
        s, m = int(starts[e]), int(counts[e])
        xs.append(x[src[s:s + m]].contiguous())
        w13.append(torch.cat([lay["w1"][e], lay["w3"][e]], 0).t())
        hs.append(h[s:s + m])
        w2.append(lay["w2"][e].t())
    u = [torch.empty(xs[e].shape[0], w13[e].shape[1], dtype=torch.bfloat16, device=x.device)
         for e in range(E)]
    yv = [torch.empty(hs[e].shape[0], w2[e].shape[1], dtype=torch.bfloat16, device=x.device)
          for e in range(E)]

    def up():
        for e in range(E):
            torch.matmul(xs[e], w13[e], out=u[e])

    def down():
        for e in range(E):
            torch.matmul(hs[e], w2[e], out=yv[e])

    d, ffn = x.shape[1], h.shape[1]
    rows = int(counts.sum())
    res = {}
    for name, fn, flop in (("up", up, 4.0 * rows * d * ffn), ("down", down, 2.0 * rows * d * ffn)):
        for _ in range(3):
            fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        us = e0.elapsed_time(e1) * 1e3 / reps
        res[name] = {"us": round(us, 1), "tflops": round(flop / us / 1e6, 1)}
    res["tiled_up_us"] = round(up_avg_ms * 1e3, 1)
    res["tiled_up_vs_library"] = round(res["up"]["us"] / (up_avg_ms * 1e3), 3)
    res["kind"] = ("torch.matmul (hipBLASLt) per expert, bf16, same rows per expert, dense "
                   "pre-gathered operands, no epilogue")
    del xs, w13, hs, w2, u, yv
    return res


def _oracle():
    """The fp64 oracle with one OpenMP thread per host core this process may use."""
    from oracle import oracle as oracle_mod

    o = oracle_mod.get()
    cores = len(os.sched_getaffinity(0))
    cores = min(cores, int(os.environ.get("OMP_NUM_THREADS", cores)))
    o.threads(cores)
    return o


def _cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for ln in f:
                if ln.startswith("model name"):
                    return ln.split(":", 1)[1].strip()
    except OSError:
        pass
    return ""


def _sample_rate(fn, T, seconds):
    """Runs fn(n) on the first n tokens, n = T when a whole pass fits the
    time budget, else the count a probe on 8 tokens says fits; repeats until
    about `seconds` of wall time.  Returns (tokens, seconds, passes, n)."""
    S = T
    t0 = time.perf_counter()
    fn(min(T, 8))
    probe = time.perf_counter() - t0
    if T > 8 and probe * T / 8 > 3 * seconds:
        S = max(8, int(8 * seconds / probe))
    tokens, el, reps = 0, 0.0, 0
    while el < seconds and reps < 1000:
        t0 = time.perf_counter()
        fn(S)
        el += time.perf_counter() - t0
        tokens += S
        reps += 1
    return tokens, el, reps, S


def cpu_baseline(args, w, x, lay, T):
    """The fp64 oracle, as it is, on this host: whole layers of the same
    workload (all T tokens when that fits the time budget, else the first
    tokens), repeated until about --cpu-seconds of wall time."""
    from paper_2408_00008_amd import inputs

    o = _oracle()
    xb = inputs.bf16_bits(x)
    rwb = inputs.bf16_bits(lay["router_w"])
    bias = None if lay["router_bias"] is None else lay["router_bias"].cpu().numpy()
    if w.fp8:
        ws = [lay[n].cpu().numpy() for n in ("w1q", "w1s", "w3q", "w3s", "w2q", "w2s")]

        def layer(n):
            o.moe_layer_fp8(xb[:n], rwb, *ws, w.k, bias)
    else:
        ws = [inputs.bf16_bits(lay[n]) for n in ("w1", "w3", "w2")]

        def layer(n):
            o.moe_layer(xb[:n], rwb, *ws, w.k, bias)
    tokens, el, reps, S = _sample_rate(layer, T, args.cpu_seconds)
    return {"value": round(tokens / el, 3), "unit": "tokens/s", "cores": o.threads(),
            "kind": "oracle",
            "sample": f"{reps} x full fp64 layer over the first {S} of {T} tokens of "
                      f"{w.name} ({el:.1f} s wall)",
            "cpu_model": _cpu_model()}


def cpu_baseline_stack(args, w, st, x):
    """The oracle on the stack workload: layer 0 of the stack (RMSNorm of the
    residual stream, rounding to bf16, the fp64 MoE layer) on this host;
    every layer does the same work, so the 32-layer step's rate is the
    layer's divided by the layer count."""
    from paper_2408_00008_amd import inputs

    o = _oracle()
    lay = st.layers[0]
    h = x.float().cpu().numpy()
    gamma = inputs.bf16_bits(lay["gamma"])
    wb = [inputs.bf16_bits(lay[n]) for n in ("router_w", "w1", "w3", "w2")]

    def layer(n):
        a = o.round_bf16(o.rmsnorm(h[:n], gamma, w.eps))
        o.moe_layer(a, *wb, w.k)

    tokens, el, reps, S = _sample_rate(layer, w.T, args.cpu_seconds)
    return {"value": round(tokens / el / st.L, 4), "unit": "tokens/s", "cores": o.threads(),
            "kind": "oracle",
            "sample": f"{reps} x layer 0 of {st.L} (RMSNorm + fp64 MoE layer) over the first {S} "
                      f"of {w.T} tokens of {w.name} ({el:.1f} s wall); rate divided by {st.L} "
                      f"layers",
            "cpu_model": _cpu_model()}


def cpu_baseline_decoder(args, w, layer, cache, page_table, pos, h):
    """The oracle on a decoder workload: one decoder layer (RMSNorm, the
    projections, RoPE, paged attention over the request's cached positions,
    the output projection, RMSNorm and the fp64 MoE layer) on this host; for
    a stack of layers the rate is divided by the layer count."""
    from paper_2408_00008_amd import inputs

    o = _oracle()
    hq, hkv, hd = w.hq, w.hkv, w.hd
    wqkv = inputs.bf16_bits(layer.wqkv)
    wq, wk, wv = wqkv[:hq * hd], wqkv[hq * hd:(hq + hkv) * hd], wqkv[(hq + hkv) * hd:]
    wo = inputs.bf16_bits(layer.wo)
    ga, gm = inputs.bf16_bits(layer.gamma_attn), inputs.bf16_bits(layer.gamma_moe)
    rw = inputs.bf16_bits(layer.router_w)
    kc, vc = inputs.bf16_bits(cache[0]), inputs.bf16_bits(cache[1])
    pt, ps = page_table.cpu().numpy(), pos.cpu().numpy()
    hn = h.cpu().numpy()
    if layer.fp8:
        ex = {"fp8_experts": [t.cpu().numpy() for t in layer.q]}
        w1 = w3 = w2 = None
    else:
        ex = {}
        w1, w3, w2 = (inputs.bf16_bits(t) for t in (layer.w1, layer.w3, layer.w2))

    def one(n):
        o.decoder_layer(hn[:n], ga, wq, wk, wv, wo, kc, vc, pt[:n], ps[:n], gm, rw, w1, w3, w2,
                        w.k, hq, hkv, w.theta, w.eps, **ex)

    tokens, el, reps, S = _sample_rate(one, w.T, args.cpu_seconds)
    L = max(1, w.layers)
    return {"value": round(tokens / el / L, 4), "unit": "tokens/s", "cores": o.threads(),
            "kind": "oracle",
            "sample": f"{reps} x one fp64 decoder layer over the first {S} of {w.T} requests of "
                      f"{w.name} ({el:.1f} s wall)"
                      + (f"; rate divided by {L} layers" if L > 1 else ""),
            "cpu_model": _cpu_model()}


if __name__ == "__main__":
    main()
