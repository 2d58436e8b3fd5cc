"""The forward path captured in a HIP graph (torch.cuda.CUDAGraph) and
replayed: every replay must equal the eager result bit for bit.  The input
buffer is refilled between replays with two different token sets, so the
replays also show that routing, permutation and tile lists are recomputed on
the device from the current input (nothing host-side is frozen at capture).
Eager work and synchronisations run between the replays.  Covers the decode
GEMVs (T = 4), the grouped GEMM (T = 300), the chained stack, and two
decoder layers (attention block with its norms, then the MoE layer) at
decode and through the prefill path."""
import numpy as np
import pytest

import moe_inputs as mi
from harness import load_workload_host, make_layer

pytestmark = pytest.mark.gpu

TINY = mi.WORKLOADS["tiny"]
REPLAYS = 6


@pytest.fixture(scope="module")
def torch_mod():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch


def _inputs(torch, wl, T):
    a = mi.gen_bf16(wl.seed, mi.stream_id(mi.KIND_X), (T, wl.d), 1.0)
    b = mi.gen_bf16(wl.seed + 1, mi.stream_id(mi.KIND_X), (T, wl.d), 1.0)
    return [torch.from_numpy(v.view(np.int16)).cuda() for v in (a, b)]


def _noise(torch):
    # unrelated eager work between replays
    m = torch.randn(512, 512, device="cuda")
    (m @ m).sum().item()


@pytest.mark.parametrize("T", [4, 300])
def test_forward_graph_replays_match_eager(torch_mod, T):
    torch = torch_mod
    wl = TINY.with_(T=T)
    layer = make_layer(wl, max_tokens=T)
    load_workload_host(layer, wl)
    try:
        xs = _inputs(torch, wl, T)
        refs = []
        for x in xs:
            y = torch.empty((T, wl.d), dtype=torch.int16, device="cuda")
            layer.forward(0, x, y)
            torch.cuda.synchronize()
            refs.append(y.clone())
        assert not torch.equal(refs[0], refs[1])
        x_in = xs[0].clone()
        y_out = torch.zeros((T, wl.d), dtype=torch.int16, device="cuda")
        layer.forward(0, x_in, y_out)          # warm up on the capture buffers
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            layer.forward(0, x_in, y_out)
        for i in range(REPLAYS):
            x_in.copy_(xs[i % 2])
            y_out.fill_(0x3F80)
            g.replay()
            torch.cuda.synchronize()
            assert torch.equal(y_out, refs[i % 2]), f"replay {i}"
            _noise(torch)
        del g
    finally:
        layer.close()


def test_stack_graph_replays_match_eager(torch_mod):
    torch = torch_mod
    wl = TINY.with_(T=4, n_layers=3)
    layer = make_layer(wl, max_tokens=4)
    for li in range(3):
        load_workload_host(layer, wl, layer_idx=li)
    try:
        xs = _inputs(torch, wl, 4)
        refs = []
        for x in xs:
            v = x.clone()
            layer.forward_stack(v)
            torch.cuda.synchronize()
            refs.append(v)
        x0 = xs[0].clone()
        cur = x0.clone()

        def step():
            cur.copy_(x0)
            layer.forward_stack(cur)

        step()
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            step()
        for i in range(REPLAYS):
            x0.copy_(xs[i % 2])
            g.replay()
            torch.cuda.synchronize()
            assert torch.equal(cur, refs[i % 2]), f"replay {i}"
            _noise(torch)
        del g
    finally:
        layer.close()


ATTN = mi.ATTN_WORKLOADS["attn_tiny"]


@pytest.mark.parametrize("T,pos0", [(1, 29), (40, 0)])
def test_decoder_layers_graph_replays_match_eager(torch_mod, T, pos0):
    """Two DBRX decoder layers (attn_forward_norm, then moe_forward_residual
    on the normalised input) captured once and replayed, at decode (T = 1:
    the norm inside the projection, attention over position chunks) and
    through the prefill path (T = 40: projection GEMMs, causal attention):
    every replay equals the eager chain, for two alternating inputs.  The
    key/value cache positions a call appends are rewritten by every replay."""
    import paper_2506_23635_amd as moe
    torch = torch_mod
    aw = ATTN.with_(T=T, pos0=pos0)
    wl = TINY.with_(T=T, n_layers=2)
    acfg = moe.make_attn_config(aw.d, aw.n_heads, aw.n_kv, aw.hd, n_layers=2, max_seq=128,
                                max_tokens=64, rope_theta=aw.theta, norm_eps=aw.eps)
    att = moe.AttnLayer(acfg)
    ffn = make_layer(wl, max_tokens=64, n_layers=2)
    try:
        for li in range(2):
            att.load_layer(li, torch.from_numpy(aw.gamma(li)), torch.from_numpy(aw.wqkv(li).view(np.int16)),
                           torch.from_numpy(aw.wo(li).view(np.int16)))
            att.load_post_norm(li, torch.from_numpy(aw.gamma2(li)))
            K, V = att.cache_views(li)
            K.zero_()
            V.zero_()
            if pos0:
                k0, v0 = aw.cache_prefix(li)
                K[:, :pos0] = torch.from_numpy(np.ascontiguousarray(k0.transpose(1, 0, 2)).view(np.int16)).cuda()
                V[:, :pos0] = torch.from_numpy(np.ascontiguousarray(v0.transpose(1, 0, 2)).view(np.int16)).cuda()
            load_workload_host(ffn, wl, layer_idx=li)
        xs = _inputs(torch, wl, T)
        x0 = xs[0].clone()
        x = x0.clone()
        z = torch.empty_like(x)

        def step():
            x.copy_(x0)
            for li in range(2):
                att.forward_norm(li, x, x, z, pos0)
                ffn.forward_residual(li, z, x)

        refs = []
        for v in xs:
            x0.copy_(v)
            step()
            torch.cuda.synchronize()
            refs.append(x.clone())
        assert not torch.equal(refs[0], refs[1])
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            step()
        for i in range(REPLAYS):
            x0.copy_(xs[i % 2])
            x.fill_(0x3F80)
            g.replay()
            torch.cuda.synchronize()
            assert torch.equal(x, refs[i % 2]), f"replay {i}"
            _noise(torch)
        del g
    finally:
        att.close()
        ffn.close()
