"""The residual MoE stack: graph replay equals eager execution, and every
layer matches the oracle when fed the GPU's own layer input (teacher forcing:
a free-running bf16 stack and an f64 stack drift apart through discrete
routing flips, so the check is per layer)."""

import numpy as np
import pytest
import torch

from gpu_common import DEV, orc, say
from paper_2408_00008_amd import inputs
from paper_2408_00008_amd.stack import MoeStack
from parity import OUT_TOL, bf16_ulp_diff, check_routing, round_bf16_bits, rowwise_rel

pytestmark = pytest.mark.gpu


def _small_stack(layers=4, T=64, d=256, ffn=512, E=8, k=2):
    w = inputs.Workload("small_stack", T, d, ffn, E, k, 1.0, 1 / np.sqrt(d), 1 / np.sqrt(d),
                        1 / np.sqrt(d), 1 / np.sqrt(ffn), layers=layers, seed=3)
    return w, MoeStack(w, DEV, gamma_random=True)


def _teacher_forced(w, st, x, layers):
    o = orc()
    tr = st.trace(x, layers)
    worst = 0.0
    for l in layers:
        h_in, a, h_out = tr[l]
        lay = st.layers[l]
        h_np = h_in.cpu().numpy()
        # (i) the GPU's normalised input is the correctly rounded RMSNorm of its h
        ref_a = o.rmsnorm(h_np, inputs.bf16_bits(lay["gamma"]), w.eps)
        assert bf16_ulp_diff(inputs.bf16_bits(a), round_bf16_bits(ref_a)).max() <= 1, l
        # (ii) the oracle layer on the GPU's exact a_l bits
        a_bits = inputs.bf16_bits(a)
        bits = {n: inputs.bf16_bits(lay[n]) for n in ("router_w", "w1", "w3", "w2")}
        logits = o.router_logits(a_bits, bits["router_w"], None)
        # the GPU routing of this layer's input, through the library
        ids = torch.empty(w.T, w.k, dtype=torch.int32, device=DEV)
        gw = torch.empty(w.T, w.k, dtype=torch.float32, device=DEV)
        offs = torch.empty(w.E + 1, dtype=torch.int32, device=DEV)
        perm = torch.empty(w.T * w.k, dtype=torch.int32, device=DEV)
        from paper_2408_00008_amd import binding as B
        B.moe_route(a, lay["router_w"], w.k, ids, gw, offs, perm)
        torch.cuda.synchronize()
        g_ids = ids.cpu().numpy()
        check_routing(g_ids, logits, w.k)
        gates = o.gates_for_ids(logits, g_ids)
        ref = o.moe_apply(a_bits, bits["w1"], bits["w3"], bits["w2"], g_ids, gates)
        # (iii) the layer's contribution to the residual stream
        delta = h_out.cpu().numpy().astype(np.float64) - h_np.astype(np.float64)
        err = rowwise_rel(delta, ref)
        worst = max(worst, err)
        say(f"  layer {l}: delta rowwise rel {err:.3e}")
        assert err < OUT_TOL, (l, err)
    return worst


def test_stack_teacher_forced_small():
    say("[stack] small shape, every layer teacher-forced")
    w, st = _small_stack()
    x = inputs.make_x(w, DEV)
    _teacher_forced(w, st, x, range(w.layers))


def test_stack_graph_replay_matches_eager():
    say("[stack] graph replay vs eager")
    w, st = _small_stack(layers=3)
    x = inputs.make_x(w, DEV)
    st.load_input(x)
    st.step()
    torch.cuda.synchronize()
    eager = st.h.clone()
    st.capture(x)
    for rep in range(3):
        st.h.fill_(7.0)  # eager work between replays
        torch.cuda.synchronize()
        st.replay()
        torch.cuda.synchronize()
        assert torch.equal(st.h, eager), rep


def test_stack_mixtral_shape_all_layers():
    """The benchmarked 32-layer Mixtral-shape stack (90 GB of weights): the
    captured graph's replays give the eager step's bits, and every one of the
    32 layers matches the oracle on its own GPU input (teacher forcing)."""
    say("[stack] Mixtral shape, 32 layers: graph replay vs eager, then teacher-forced")
    w = inputs.WORKLOADS["stack32_t64"]
    st = MoeStack(w, DEV)
    assert st.L == 32
    x = inputs.make_x(w, DEV)
    st.load_input(x)
    st.step()
    torch.cuda.synchronize()
    eager = st.h.clone()
    st.capture(x)
    for rep in range(3):
        st.h.fill_(7.0)  # eager work between replays
        torch.cuda.synchronize()
        st.replay()
        torch.cuda.synchronize()
        assert torch.equal(st.h, eager), rep
    say("  32-layer graph replays equal the eager step bitwise")
    worst = _teacher_forced(w, st, x, range(st.L))
    say(f"  worst layer delta rowwise rel {worst:.3e}")
    del st
    torch.cuda.empty_cache()
