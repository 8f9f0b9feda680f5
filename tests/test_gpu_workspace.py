"""The library-owned scratch of moe_forward and moe_attention_decode on the
GPU: a growth while the stream is being captured is refused with
MOE_ERR_NO_MEMORY and enqueues nothing; a growth after a capture keeps the
buffer the graph holds alive, so the graph still replays correctly; the
MOE_WORKSPACE_LIMIT_BYTES cap forces MOE_ERR_NO_MEMORY on a real device."""

import math
import os

import pytest
import torch

from gpu_common import DEV, say, small_case
from paper_2408_00008_amd import binding as B
from paper_2408_00008_amd import inputs

pytestmark = pytest.mark.gpu


def _forward(c, out, stream=None):
    B.moe_forward(c.x, c.router_w, c.w1, c.w3, c.w2, c.k, out, stream=stream)


def test_forward_scratch_growth_refused_under_capture():
    say("[workspace] growth under capture (moe_forward)")
    c = small_case(64, 256, 512, 8, 2, seed=41)
    out = torch.empty(c.T, c.d, dtype=torch.bfloat16, device=DEV)
    B.moe_release_workspace()
    s = torch.cuda.Stream()
    g = torch.cuda.CUDAGraph()
    with pytest.raises(B.MoeError) as ei:
        with torch.cuda.graph(g, stream=s):
            _forward(c, out, stream=s)
    assert ei.value.status == B.MOE_ERR_NO_MEMORY
    assert "captured" in str(ei.value)
    # one call outside capture sizes the scratch; the capture then works
    _forward(c, out)
    torch.cuda.synchronize()
    ref = out.clone()
    out.zero_()
    g2 = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g2, stream=s):
        _forward(c, out, stream=s)
    g2.replay()
    torch.cuda.synchronize()
    assert torch.equal(out, ref)


def test_captured_graph_survives_scratch_growth():
    """A graph captured with the library scratch still replays correctly
    after a larger call has grown (replaced) that scratch."""
    say("[workspace] graph replay after a growth")
    c = small_case(64, 256, 512, 8, 2, seed=42)
    out = torch.empty(c.T, c.d, dtype=torch.bfloat16, device=DEV)
    B.moe_release_workspace()
    _forward(c, out)
    torch.cuda.synchronize()
    ref = out.clone()
    s = torch.cuda.Stream()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        _forward(c, out, stream=s)
    # a bigger step grows the scratch (the captured buffer is retired, not freed)
    big = small_case(3000, 256, 512, 8, 2, seed=43)
    big_out = torch.empty(big.T, big.d, dtype=torch.bfloat16, device=DEV)
    _forward(big, big_out)
    torch.cuda.synchronize()
    for rep in range(3):
        out.fill_(0)
        _forward(big, big_out)  # eager work on the new scratch between replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(out, ref), rep
    del g
    B.moe_release_workspace()


def test_attention_scratch_growth_refused_under_capture():
    say("[workspace] growth under capture (attention split scratch)")
    w = inputs.Workload("dec", 2, 256, 256, 8, 2, 1.0, 1 / 16, 1 / 16, 1 / 16, 1 / 16, seed=19,
                        hq=32, hkv=8, hd=128, page=16, ctx=3000, ctx_ragged=False, std_attn=1 / 16)
    kv = inputs.make_kv_cache(w, 0, DEV)
    g = torch.Generator(device=DEV).manual_seed(21)
    q = (torch.randn(2, 32, 128, generator=g, device=DEV) * 1.5).to(torch.bfloat16)
    out = torch.empty(2, 32 * 128, dtype=torch.bfloat16, device=DEV)
    scale = 1 / math.sqrt(128)
    args = (q, kv["k_cache"], kv["v_cache"], kv["page_table"], kv["ctx"], scale, out)
    B.moe_release_workspace()
    s = torch.cuda.Stream()
    graph = torch.cuda.CUDAGraph()
    with pytest.raises(B.MoeError) as ei:
        with torch.cuda.graph(graph, stream=s):
            B.moe_attention_decode(*args, stream=s)
    assert ei.value.status == B.MOE_ERR_NO_MEMORY
    B.moe_attention_decode(*args)
    torch.cuda.synchronize()
    ref = out.clone()
    out.zero_()
    graph2 = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph2, stream=s):
        B.moe_attention_decode(*args, stream=s)
    graph2.replay()
    torch.cuda.synchronize()
    assert torch.equal(out, ref)


def test_workspace_limit_on_device():
    say("[workspace] MOE_WORKSPACE_LIMIT_BYTES on the device")
    c = small_case(64, 256, 512, 8, 2, seed=44)
    out = torch.empty(c.T, c.d, dtype=torch.bfloat16, device=DEV)
    need = B.moe_workspace_size(c.T, c.d, c.ffn, c.E, c.k)
    old = os.environ.get("MOE_WORKSPACE_LIMIT_BYTES")
    try:
        os.environ["MOE_WORKSPACE_LIMIT_BYTES"] = str(need - 256)
        out.fill_(3.0)
        with pytest.raises(B.MoeError) as ei:
            _forward(c, out)
        assert ei.value.status == B.MOE_ERR_NO_MEMORY
        torch.cuda.synchronize()
        assert bool((out == 3.0).all())  # nothing was enqueued
        os.environ["MOE_WORKSPACE_LIMIT_BYTES"] = str(need)
        _forward(c, out)  # exactly enough (the growth slack is capped)
        torch.cuda.synchronize()
        assert not bool((out == 3.0).all())
    finally:
        if old is None:
            os.environ.pop("MOE_WORKSPACE_LIMIT_BYTES", None)
        else:
            os.environ["MOE_WORKSPACE_LIMIT_BYTES"] = old
        B.moe_release_workspace()
