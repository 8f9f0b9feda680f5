"""One GPU's share of a sharded layer (tensor- and expert-parallel MoE, the
configurations of the paper's Exp4: TP8, EP4-TP2, EP2-TP4): every shard runs
through the same C ABI at its real shape, and the sum of the shards' partial
outputs -- the all-reduce, done here on one GPU -- must equal the unsharded
layer.

A shard owns experts [e0, e0 + El) and hidden units [f0, f0 + F) of each of
them: those rows of W1 and W3 and those columns of W2, copied contiguous as a
GPU would hold them.  Routing is replicated (every shard computes the same
ids), the shard computes only the rows routed to its experts, scatters them
gate-weighted into their (token, slot) positions (other slots stay zero) and
combines: out_s = sum over its slots of g_j W2_s h_s."""

import numpy as np
import pytest
import torch

from gpu_common import DEV, gpu_route, oracle_out, say, small_case, workload_case
from parity import OUT_TOL, check_routing, rowwise_rel
from paper_2408_00008_amd import binding as B

pytestmark = pytest.mark.gpu


def shard_partial(c, route, e0, el, f0, f):
    _, gw, offs, perm, _ = route
    A = c.T * c.k
    e, u = slice(e0, e0 + el), slice(f0, f0 + f)
    w1 = c.w1[e, u, :].contiguous()
    w3 = c.w3[e, u, :].contiguous()
    w2 = c.w2[e, :, u].contiguous()
    # this shard's experts' offsets (absolute row numbers), in a buffer of its own
    offs_s = offs[e0:e0 + el + 1].clone()
    h = torch.empty(A, f, dtype=torch.bfloat16, device=DEV)
    y = torch.zeros(A, c.d, dtype=torch.float32, device=DEV)
    B.moe_swiglu_up(c.x, offs_s, w1, w3, c.T, c.k, h, perm=perm)
    B.moe_swiglu_down(h, offs_s, w2, c.T, c.k, y, topk_w=gw.reshape(-1), perm=perm)
    out = torch.empty(c.T, c.d, dtype=torch.float32, device=DEV)
    B.moe_combine(y, c.T, c.d, c.k, out_f32=out)
    return out


def sharded_sum(c, n_ep, n_tp):
    route = gpu_route(c)
    el, f = c.E // n_ep, c.ffn // n_tp
    total = torch.zeros(c.T, c.d, dtype=torch.float32, device=DEV)
    for s_ep in range(n_ep):
        for s_tp in range(n_tp):
            total += shard_partial(c, route, s_ep * el, el, s_tp * f, f)
    torch.cuda.synchronize()
    return total, route


def check_sum(c, total, route, rows=None):
    rows = np.arange(c.T) if rows is None else np.asarray(rows)
    g_ids = route[0].cpu().numpy()[rows]
    ref, logits, *_ = oracle_out(c, rows, g_ids)
    check_routing(g_ids, logits, c.k)
    err = rowwise_rel(total.cpu().numpy().astype(np.float64)[rows], ref)
    say(f"  {c.name}: rowwise rel of the shard sum {err:.3e}")
    assert err < OUT_TOL


@pytest.mark.parametrize("n_ep,n_tp", [(1, 2), (1, 8), (2, 1), (8, 1), (4, 2), (2, 4)])
def test_shards_sum_to_layer(n_ep, n_tp):
    say(f"[shards] EP{n_ep}-TP{n_tp}")
    c = small_case(96, 256, 1024, 8, 2, seed=31)
    total, route = sharded_sum(c, n_ep, n_tp)
    check_sum(c, total, route)


def test_tp_forward_share_equals_partial():
    """TP shards through moe_forward_ex (routing inside the call, f32 out)."""
    say("[shards] TP4 via moe_forward_ex")
    c = small_case(64, 256, 1024, 8, 2, seed=33)
    f = c.ffn // 4
    total = torch.zeros(c.T, c.d, dtype=torch.float32, device=DEV)
    for s in range(4):
        u = slice(s * f, (s + 1) * f)
        part = torch.empty(c.T, c.d, dtype=torch.float32, device=DEV)
        B.moe_forward_ex(c.x, c.router_w, c.w1[:, u, :].contiguous(), c.w3[:, u, :].contiguous(),
                         c.w2[:, :, u].contiguous(), c.k, out_f32=part)
        total += part
    torch.cuda.synchronize()
    check_sum(c, total, gpu_route(c))


def test_ep2_tp4_mixtral_decode():
    """EP2-TP4, the paper's best hybrid, on the Mixtral decode step: 8 shards
    of 4 experts x 3584 hidden units at their real shape; every token."""
    say("[shards] EP2-TP4 decode_t64")
    c = workload_case("decode_t64")
    total, route = sharded_sum(c, 2, 4)
    check_sum(c, total, route)
