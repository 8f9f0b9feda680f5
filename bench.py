"""Benchmark of the MoE FFN layer on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload decode_t64]

A step is one pass of the whole layer over one batch of T tokens already
resident in HBM: router GEMM + top-k + dispatch, the SwiGLU up GEMM (with the
row gather fused in), the down GEMM with the gate-weighted scatter, and the
combine -- the same kernels `moe_forward` enqueues, called stage by stage so
that HIP events can bracket the dominant kernel on the stream it runs on.

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
    ap.add_argument("--cpu-seconds", type=float, default=12.0,
                    help="target wall time of the oracle baseline sample")
    ap.add_argument("--no-cpu-baseline", action="store_true")
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

    import numpy as np
    import torch

    from paper_2408_00008_amd import binding as B
    from paper_2408_00008_amd import inputs

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = "cuda:0"
    w = inputs.WORKLOADS[args.workload].replace(seed=args.seed)
    if w.hq:
        from paper_2408_00008_amd import decoder
        return decoder.bench_decoder(args, w)
    if w.layers != 1:
        from paper_2408_00008_amd import stack
        return stack.bench_stack(args, w)
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

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(args.steps)]
    # one event at every step boundary: the first and last bracket the timed
    # region, the ones between give the per-step spread
    bounds = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    bounds[0].record(stream)
    for i in range(args.steps):
        step(*evs[i])
        bounds[i + 1].record(stream)
    torch.cuda.synchronize()
    wall1 = time.perf_counter()
    ms_total = bounds[0].elapsed_time(bounds[-1])
    step_ms = np.array([bounds[i].elapsed_time(bounds[i + 1]) for i in range(args.steps)])
    ms_per_step = ms_total / args.steps
    up_ms = sorted(e0.elapsed_time(e1) for e0, e1 in evs)
    up_avg_ms = sum(up_ms) / len(up_ms)

    counts = np.diff(offs.cpu().numpy())
    active = int((counts > 0).sum())
    # algorithmic work of the up kernel: each active expert's w1 and w3 once
    # (bf16, or E4M3 bytes plus one f32 scale per row), the routed token rows
    # read once, h written once; 4*d*ffn FLOP per row
    scale_bytes = 4 if w.fp8 else 0
    up_bytes = (active * 2 * ffn * (d * wbytes_per_elem + scale_bytes) + A * d * 2
                + A * ffn * 2)
    up_flops = 4.0 * A * d * ffn
    kernel = "expert_up_" + variant
    if variant in ("stream", "split"):
        # split: experts of up to 64 rows stream, heavier ones take a second
        # launch; both sit between the same two events
        achieved = up_bytes / (up_avg_ms * 1e-3) / 1e9
        roof = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS,
                "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4)}
    else:
        achieved = up_flops / (up_avg_ms * 1e-3) / 1e12
        roof = {"bound": "mfma", "achieved": round(achieved, 1), "peak": BF16_PEAK_TFLOPS,
                "unit": "TFLOP/s", "frac": round(achieved / BF16_PEAK_TFLOPS, 4)}
    roof["traffic"] = load_traffic(args.workload, kernel, variant)
    roof["kernel"] = kernel
    roof["avg_launch_us"] = round(up_avg_ms * 1e3, 2)
    roof["algorithmic_bytes_per_launch"] = up_bytes
    roof["algorithmic_flop_per_launch"] = up_flops

    layer_flops = 2.0 * T * d * E + 6.0 * A * d * ffn
    layer_bytes = (active * (3 * ffn * d * wbytes_per_elem + (2 * ffn + d) * scale_bytes)
                   + E * d * 2 + T * d * 2 * 2)
    tok_s = T * args.steps / (ms_total * 1e-3)

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(args, w, x, lay, T)

    rec = {
        "metric": "MoE-layer tokens/s",
        "value": round(tok_s, 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "step_ms_p10_p50_p90": [round(float(np.percentile(step_ms, q)), 4) for q in (10, 50, 90)],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",  # MFMA operands; E4M3 weights are widened exactly to bf16
        "data": "synthetic (seeded normals of the Mixtral-8x7B layer shapes; no dataset, random weights)",
        "config": {"workload": args.workload, "T": T, "d": d, "ffn": ffn, "E": E, "k": k,
                   "expert_weights": "e4m3 + f32 row scale" if w.fp8 else "bf16",
                   "router_bias0": w.bias0, "seed": args.seed, "active_experts": active,
                   "rows_per_expert": counts.tolist(),
                   "down_reduction_parts": int(parts.item()) if cut else 1},
        "layer": {"tflops": round(layer_flops / (ms_per_step * 1e-3) / 1e12, 2),
                  "gbs": round(layer_bytes / (ms_per_step * 1e-3) / 1e9, 1),
                  "hbm_frac": round(layer_bytes / (ms_per_step * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
                  "mfma_frac": round(layer_flops / (ms_per_step * 1e-3) / 1e12 / BF16_PEAK_TFLOPS, 4),
                  "algorithmic_bytes": layer_bytes, "algorithmic_flop": layer_flops},
        "roofline": roof,
        "cpu_baseline": cpu,
        "wall_s_timed": round(wall1 - wall0, 3),
    }
    print(json.dumps(rec), flush=True)


def cpu_baseline(args, w, x, lay, T):
    """The fp64 oracle, as it is, on this host: whole layers of the same
    workload (all T tokens when that fits the time budget, else the first
    tokens), repeated until about --cpu-seconds of wall time."""
    import numpy as np

    from oracle import oracle as oracle_mod
    from paper_2408_00008_amd import inputs

    o = oracle_mod.get()
    cores = len(os.sched_getaffinity(0))
    cores = min(cores, int(os.environ.get("OMP_NUM_THREADS", cores)))
    o.threads(cores)
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
    S = T
    # probe with a small slice, then size the sample
    t0 = time.perf_counter()
    layer(min(T, 8))
    probe = time.perf_counter() - t0
    if T > 8 and probe * T / 8 > 3 * args.cpu_seconds:
        S = max(8, int(8 * args.cpu_seconds / probe))
    tokens, el, reps = 0, 0.0, 0
    while el < args.cpu_seconds and reps < 1000:
        t0 = time.perf_counter()
        layer(S)
        el += time.perf_counter() - t0
        tokens += S
        reps += 1
    model = ""
    try:
        with open("/proc/cpuinfo") as f:
            for ln in f:
                if ln.startswith("model name"):
                    model = ln.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    del np
    return {"value": round(tokens / el, 3), "unit": "tokens/s", "cores": o.threads(),
            "kind": "oracle",
            "sample": f"{reps} x full fp64 layer over the first {S} of {T} tokens of "
                      f"{args.workload} ({el:.1f} s wall)",
            "cpu_model": model}


if __name__ == "__main__":
    main()
