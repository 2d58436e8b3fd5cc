"""Guard zones around every buffer the caller hands the library: the
weight arena, the workspace and the output (and the in-place stack input)
sit inside larger allocations whose margins hold a byte pattern; after
loads, routing and forwards on the decode GEMVs, the grouped GEMM, an
expert-parallel share and the stack, every margin must be intact (no kernel
writes outside the buffers it was given).  Inside the workspace, every
sub-buffer (moe_workspace_map) is guarded too: after a forward, the bytes of
each region past what the call may write there, and the padding between
regions, still hold the pattern.  The attention block's arena, cache,
workspace, input and outputs are guarded the same way."""
import numpy as np
import pytest

import moe_inputs as mi
from harness import load_workload_host, x_device

pytestmark = pytest.mark.gpu

TINY = mi.WORKLOADS["tiny"]
GUARD = 64 << 10      # bytes on each side
PATTERN = 0xA5


@pytest.fixture(scope="module")
def torch_mod():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch


class Guarded:
    """A device buffer of n bytes with GUARD patterned bytes on each side."""

    def __init__(self, torch, n):
        self.n = n
        self.full = torch.full((n + 2 * GUARD,), PATTERN, dtype=torch.uint8, device="cuda")
        self.inner = self.full[GUARD:GUARD + n]

    def intact(self):
        h = self.full.cpu().numpy()
        return bool(np.all(h[:GUARD] == PATTERN) and np.all(h[GUARD + self.n:] == PATTERN))


def _layer(torch, wl, max_tokens, **kw):
    import paper_2506_23635_amd as moe
    cfg = moe.make_config(wl.d, wl.f, wl.E, wl.k, max_tokens=max_tokens,
                          n_layers=kw.get("n_layers", 1),
                          expert_begin=kw.get("e_begin", 0), n_local_experts=kw.get("n_local", 0))
    arena = Guarded(torch, moe.moe_weight_bytes(cfg))
    ws = Guarded(torch, moe.moe_workspace_bytes(cfg))
    return moe.MoeLayer(cfg, arena=arena.inner, workspace=ws.inner), arena, ws


@pytest.mark.parametrize("T,e_begin,n_local", [(4, 0, 0), (300, 0, 0), (16, 2, 2), (300, 6, 2)])
def test_forward_stays_inside_its_buffers(torch_mod, T, e_begin, n_local):
    torch = torch_mod
    wl = TINY.with_(T=T)
    layer, arena, ws = _layer(torch, wl, T, e_begin=e_begin, n_local=n_local)
    try:
        load_workload_host(layer, wl)
        x_t, _ = x_device(wl)
        y = Guarded(torch, T * wl.d * 2)
        y16 = y.inner.view(torch.int16).view(T, wl.d)
        for _ in range(2):
            layer.route(0, x_t)
            layer.forward(0, x_t, y16)
        torch.cuda.synchronize()
        assert arena.intact() and ws.intact() and y.intact()
    finally:
        layer.close()


def test_stack_stays_inside_its_buffers(torch_mod):
    torch = torch_mod
    wl = TINY.with_(T=4, n_layers=3)
    layer, arena, ws = _layer(torch, wl, 4, n_layers=3)
    try:
        for li in range(3):
            load_workload_host(layer, wl, layer_idx=li)
        x_t, _ = x_device(wl)
        x = Guarded(torch, 4 * wl.d * 2)
        x16 = x.inner.view(torch.int16).view(4, wl.d)
        x16.copy_(x_t)
        layer.forward_stack(x16)
        torch.cuda.synchronize()
        assert arena.intact() and ws.intact() and x.intact()
    finally:
        layer.close()


def test_dbrx_shapes_stay_inside_their_buffers(torch_mod):
    """The full DBRX layer (16 experts, d 6144, f 10752): prefill at 2048
    tokens through the grouped GEMM, then one decode token."""
    from harness import load_workload_device
    torch = torch_mod
    wl = mi.WORKLOADS["prefill"]
    layer, arena, ws = _layer(torch, wl, wl.T)
    try:
        load_workload_device(layer, wl)
        for T in (wl.T, 1):
            w = wl.with_(T=T)
            x = torch.empty(T * w.d, dtype=torch.int16, device="cuda")
            mi.gen_bf16_device(w.seed, mi.stream_id(mi.KIND_X), T * w.d, w.sigma_x, x.data_ptr(),
                               layer.stream)
            y = Guarded(torch, T * w.d * 2)
            layer.forward(0, x.view(T, w.d), y.inner.view(torch.int16).view(T, w.d))
            torch.cuda.synchronize()
            assert y.intact(), T
        assert arena.intact() and ws.intact()
    finally:
        layer.close()


def _may_write(name, T, k, E, d, f, rt, decode_route, n_wg=None):
    """Byte ranges (relative to the region) that a forward of T tokens may
    write in workspace region `name`, given its routing."""
    rows = int(rt["offsets"][-1])
    n_active = int((rt["counts"] > 0).sum())
    if name == "route_partials":
        # the small-T router writes T of 16 token slots of each workgroup's
        # 16 x 16 fp64 block (32 KiB at most)
        return [(b * 16 * 16 * 8, (b * 16 + T) * 16 * 8) for b in range(n_wg)] if decode_route else []
    sizes = {"logits": T * E * 4, "topk_idx": T * k * 4, "topk_w": T * k * 4, "counts": E * 4,
             "offsets": (E + 1) * 4, "pair_row": T * k * 4, "row_token": rows * 4,
             "active": (1 + n_active) * 4, "n_tiles": 4, "h": rows * f * 2, "o": rows * d * 4}
    if name == "tiles":
        return None      # checked through n_tiles below
    return [(0, sizes[name])]


@pytest.mark.parametrize("T,e_begin,n_local", [(3, 0, 0), (16, 2, 4), (40, 0, 0), (300, 6, 2)])
def test_workspace_regions_stay_inside_themselves(torch_mod, T, e_begin, n_local):
    """max_tokens is twice T, so every region has room past what the call
    uses: an overrun (H into its tail, O past its rows, a routing array past
    T entries) shows as a changed byte."""
    import paper_2506_23635_amd as moe
    torch = torch_mod
    wl = TINY.with_(T=T)
    layer, arena, ws = _layer(torch, wl, 2 * T, e_begin=e_begin, n_local=n_local)
    try:
        load_workload_host(layer, wl)
        x_t, _ = x_device(wl)
        y = torch.empty((T, wl.d), dtype=torch.int16, device="cuda")
        ws.inner.fill_(PATTERN)
        torch.cuda.synchronize()
        layer.forward(0, x_t, y)
        torch.cuda.synchronize()
        after = ws.inner.cpu().numpy()
        rt = layer.routing_tensors(layer.route(0, x_t))   # same routing; re-written in place
        torch.cuda.synchronize()
        m = moe.moe_workspace_map(layer.cfg)
        E, k, d, f = wl.E, wl.k, wl.d, wl.f
        decode_route = T <= 16 and E <= 16 and T * k <= 64
        n_wg = (d // 8 + 63) // 64
        allowed = np.zeros(after.size, dtype=bool)
        n_tiles = int(np.frombuffer(after[m["n_tiles"][0]:m["n_tiles"][0] + 4].tobytes(), np.int32)[0])
        for name, (off, nb) in m.items():
            if name == "tiles":
                spans = [(0, n_tiles * 8)]
            else:
                spans = _may_write(name, T, k, E, d, f, rt, decode_route, n_wg)
            for a, b in spans:
                assert b <= nb, (name, b, nb)
                allowed[off + a: off + b] = True
        bad = np.nonzero((after != PATTERN) & ~allowed)[0]
        where = [n for n, (o, nb) in m.items() if bad.size and o <= bad[0] < o + nb]
        assert bad.size == 0, (int(bad[0]), where)
        assert ws.intact() and arena.intact()
    finally:
        layer.close()


ATTN = mi.ATTN_WORKLOADS["attn_tiny"]


@pytest.mark.parametrize("T,pos0", [(1, 29), (4, 29), (16, 100), (40, 0), (130, 37)])
def test_attention_stays_inside_its_buffers(torch_mod, T, pos0):
    """The attention block (decode and prefill paths, with the post-attention
    norm) on layer 1 of 2: the margins of its arena, cache, workspace, input
    and outputs hold, layer 0's cache is untouched, and in layer 1's cache
    only the new positions change."""
    import paper_2506_23635_amd as moe
    torch = torch_mod
    aw = ATTN.with_(T=T, pos0=pos0)
    max_seq = 256
    cfg = moe.make_attn_config(aw.d, aw.n_heads, aw.n_kv, aw.hd, n_layers=2, max_seq=max_seq,
                               max_tokens=256, rope_theta=aw.theta, norm_eps=aw.eps)
    arena = Guarded(torch, moe.attn_weight_bytes(cfg))
    cache = Guarded(torch, moe.attn_cache_bytes(cfg))
    ws = Guarded(torch, moe.attn_workspace_bytes(cfg))
    cache.inner.fill_(0x5A)
    layer = moe.AttnLayer(cfg, arena=arena.inner, cache=cache.inner, workspace=ws.inner)
    try:
        for li in range(2):
            layer.load_layer(li, torch.from_numpy(aw.gamma(li)), torch.from_numpy(aw.wqkv(li).view(np.int16)),
                             torch.from_numpy(aw.wo(li).view(np.int16)))
            layer.load_post_norm(li, torch.from_numpy(aw.gamma2(li)))
        n = T * aw.d * 2
        x, y, z = Guarded(torch, n), Guarded(torch, n), Guarded(torch, n)
        x.inner.copy_(torch.from_numpy(aw.x().view(np.uint8).reshape(-1)).cuda())
        as_bf = lambda g: g.inner.view(torch.int16).view(T, aw.d)
        layer.forward_norm(1, as_bf(x), as_bf(y), as_bf(z), pos0)
        torch.cuda.synchronize()
        for g in (arena, cache, ws, x, y, z):
            assert g.intact()
        c = cache.inner.cpu().numpy()
        per_layer = c.size // 2
        assert np.all(c[:per_layer] == 0x5A)
        kv = c[per_layer:].reshape(2, aw.n_kv, max_seq, aw.hd * 2)
        assert np.all(kv[:, :, :pos0] == 0x5A) and np.all(kv[:, :, pos0 + T:] == 0x5A)
        assert not np.all(kv[:, :, pos0:pos0 + T] == 0x5A)
    finally:
        layer.close()
