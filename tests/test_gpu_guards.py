"""Guard zones around every buffer the caller hands the library: the
weight arena, the workspace and the output (and the in-place stack input)
sit inside larger allocations whose margins hold a byte pattern; after
loads, routing and forwards on the decode GEMVs, the grouped GEMM, an
expert-parallel share and the stack, every margin must be intact (no kernel
writes outside the buffers it was given)."""
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
