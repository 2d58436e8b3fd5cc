"""moe_forward_static: the layer on the library's static device scratch
(for callers that cannot allocate), through the C-ABI, against moe_forward
on the same context.  The two run the same kernels in the same order, so the
outputs must be equal bit for bit; each case makes two calls in a row, the
second with fewer tokens, so the second runs on scratch the first left
behind.  The context's workspace is not touched, a routing from moe_route
stays valid across the call, and a T beyond the scratch is refused before
anything is enqueued."""
import numpy as np
import pytest

import moe_inputs as mi
import paper_2506_23635_amd as moe
from harness import load_workload_device, load_workload_host, make_layer, to_np_u16

pytestmark = pytest.mark.gpu

TINY = mi.WORKLOADS["tiny"]
DECODE = mi.WORKLOADS["decode"]


@pytest.fixture(scope="module")
def torch_mod():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch


def _x(torch, wl, T, stream_layer=0):
    x = mi.gen_bf16(wl.seed, mi.stream_id(mi.KIND_X, stream_layer), (T, wl.d), wl.sigma_x)
    return torch.from_numpy(x.view(np.int16)).cuda()


def _pair(torch, layer, x_t, f32=False):
    """(moe_forward output, moe_forward_static output) for x_t."""
    T, d = x_t.shape[0], layer.cfg.d_model
    dt = torch.float32 if f32 else torch.int16
    fill = 1.5 if f32 else 0x3F80
    a = torch.full((T, d), fill, dtype=dt, device="cuda")
    b = torch.full((T, d), fill, dtype=dt, device="cuda")
    layer.forward(0, x_t, a)
    layer.forward_static(0, x_t, b)
    torch.cuda.synchronize()
    return a.cpu().numpy(), b.cpu().numpy()


@pytest.mark.parametrize("Ts,share,f32", [((300, 5), None, False), ((16, 1), (2, 2), False),
                                          ((40, 3), (6, 2), True)])
def test_static_equals_forward_small_layer(torch_mod, Ts, share, f32):
    torch = torch_mod
    eb, nl = share or (0, 0)
    wl = TINY.with_(T=max(Ts))
    layer = make_layer(wl, max_tokens=max(Ts), e_begin=eb, n_local=nl or wl.E,
                       flags=moe.MOE_PARTIAL_F32 if f32 else 0)
    try:
        load_workload_host(layer, wl)
        for i, T in enumerate(Ts):                      # second call: fewer tokens
            x_t = _x(torch, wl, T, i)
            a, b = _pair(torch, layer, x_t, f32)
            assert np.array_equal(a.view(np.uint32) if f32 else a, b.view(np.uint32) if f32 else b)
            assert not np.all(a == (1.5 if f32 else 0x3F80))
    finally:
        layer.close()


def test_static_leaves_workspace_and_routing_alone(torch_mod):
    torch = torch_mod
    wl = TINY.with_(T=16)
    layer = make_layer(wl, max_tokens=64)
    try:
        load_workload_host(layer, wl)
        x_t = _x(torch, wl, 16)
        r = layer.route(0, x_t)
        torch.cuda.synchronize()
        before = layer.workspace.clone()
        y = torch.empty((16, wl.d), dtype=torch.int16, device="cuda")
        for T in (16, 7):
            layer.forward_static(0, x_t[:T], y[:T])
        torch.cuda.synchronize()
        assert torch.equal(layer.workspace, before)
        layer.forward(0, x_t, y, routing=r)     # still the current routing
        torch.cuda.synchronize()
    finally:
        layer.close()


def test_static_dbrx_decode_and_capacity(torch_mod):
    """The DBRX decode layer (16 experts, d 6144, f 10752): T = 16 then T = 1
    equal moe_forward bit for bit; T = 48 needs more than the 8 MiB scratch
    and is refused with MOE_E_CAPACITY, nothing written."""
    torch = torch_mod
    layer = make_layer(DECODE, max_tokens=64)
    try:
        load_workload_device(layer, DECODE)
        for i, T in enumerate((16, 1)):
            a, b = _pair(torch, layer, _x(torch, DECODE, T, i))
            assert np.array_equal(a, b)
        x_t = _x(torch, DECODE, 48)
        y = torch.full((48, DECODE.d), 7, dtype=torch.int16, device="cuda")
        with pytest.raises(moe.MoeError) as ei:
            layer.forward_static(0, x_t, y)
        assert ei.value.status == -4 and "scratch" in str(ei.value)
        torch.cuda.synchronize()
        assert bool((y == 7).all())
    finally:
        layer.close()
