"""GPU parity on the small workload (16 tokens, d 256, 8 experts of ffn 512,
top-2) and its variants, through the C-ABI, against the fp64 oracle."""
import numpy as np
import pytest

import moe_inputs as mi
import oracle
import paper_2506_23635_amd as moe
from harness import (bf16_f64, check_chain, check_layer_output, host_experts, load_workload_host,
                     make_layer, read_intermediates, rel_l2, to_np_u16, x_device)

pytestmark = pytest.mark.gpu

TINY = mi.WORKLOADS["tiny"]


@pytest.fixture(scope="module")
def torch_mod():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch


def _oracle_full(wl, x, layer_idx=0, e_begin=0, n_local=0):
    G, U, D = host_experts(wl, range(wl.E), layer_idx)
    return oracle.layer(x, wl.router(layer_idx), wl.bias(layer_idx), G, U, D, wl.k,
                        e_begin=e_begin, n_local=n_local)


def test_device_generator_matches_host(torch_mod):
    torch = torch_mod
    for kind, n, sigma in ((mi.KIND_GATE, 100_003, 0.02), (mi.KIND_X, 4096, 1.0)):
        st = mi.stream_id(kind, 3, 5)
        t = torch.empty(n, dtype=torch.int16, device="cuda")
        mi.gen_bf16_device(7, st, n, sigma, t.data_ptr(), torch.cuda.current_stream().cuda_stream)
        torch.cuda.synchronize()
        assert np.array_equal(to_np_u16(t), mi.gen_bf16(7, st, (n,), sigma))
    f = torch.empty(5000, dtype=torch.float32, device="cuda")
    mi.gen_f32_device(1, mi.stream_id(mi.KIND_ROUTER), 5000, 0.02, f.data_ptr(),
                      torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    assert np.array_equal(f.cpu().numpy(), mi.gen_f32(1, mi.stream_id(mi.KIND_ROUTER), (5000,), 0.02))


@pytest.fixture(scope="module")
def tiny_layer(torch_mod):
    layer = make_layer(TINY, max_tokens=512)
    load_workload_host(layer, TINY)
    yield layer
    layer.close()


def _check_routing(got, idx, w, E, e_begin=0, n_local=0):
    assert np.array_equal(got["idx"], idx)
    assert np.abs(got["w"].astype(np.float64) - w).max() <= 2e-6
    counts, offsets, pair_row, row_token = oracle.permutation(idx, E, e_begin, n_local)
    assert np.array_equal(got["counts"], counts)
    assert np.array_equal(got["offsets"], offsets)
    assert np.array_equal(got["pair_row"], pair_row)
    assert np.array_equal(got["row_token"], row_token)


def test_route_given_logits_bit_exact(torch_mod, tiny_layer):
    torch = torch_mod
    x_t, x = x_device(TINY)
    lg = oracle.router_logits(x, TINY.router())
    r = tiny_layer.route(0, x_t, logits_in=torch.from_numpy(lg).cuda())
    got = tiny_layer.routing_tensors(r)
    idx, w = oracle.route_from_logits(lg, TINY.k)
    assert np.array_equal(got["logits"], lg)
    _check_routing(got, idx, w, TINY.E)


@pytest.mark.parametrize("case", ["ties", "signed_zero", "equal_rows", "one_token", "max_tokens"])
def test_route_adversarial_logits(torch_mod, tiny_layer, case):
    torch = torch_mod
    E, k = TINY.E, TINY.k
    rng = np.random.default_rng(len(case))
    if case == "ties":
        lg = rng.integers(-1, 2, size=(64, E)).astype(np.float32)
    elif case == "signed_zero":
        lg = np.where(rng.random((32, E)) < 0.5, -0.0, 0.0).astype(np.float32)
        lg[:, E - 1] = -1.0
    elif case == "equal_rows":
        lg = np.tile(rng.standard_normal((1, E)).astype(np.float32), (40, 1))
    elif case == "one_token":
        lg = rng.standard_normal((1, E)).astype(np.float32)
    else:
        lg = rng.standard_normal((512, E)).astype(np.float32) * 3
    T = lg.shape[0]
    x_t = torch.zeros((T, TINY.d), dtype=torch.int16, device="cuda")
    r = tiny_layer.route(0, x_t, logits_in=torch.from_numpy(lg).cuda())
    got = tiny_layer.routing_tensors(r)
    idx, w = oracle.route_from_logits(lg, k)
    _check_routing(got, idx, w, E)


def test_route_from_x_matches_oracle(torch_mod, tiny_layer):
    x_t, x = x_device(TINY)
    r = tiny_layer.route(0, x_t)
    got = tiny_layer.routing_tensors(r)
    lg = oracle.router_logits(x, TINY.router())
    assert np.all(np.abs(got["logits"] - lg) <= 1e-5 * np.abs(lg).max())
    assert np.mean(got["logits"] == lg) >= 0.99
    idx, w = oracle.route_from_logits(lg, TINY.k)
    _check_routing(got, idx, w, TINY.E)


@pytest.mark.parametrize("T", [17, 300, 512])
def test_route_from_x_many_tokens(torch_mod, tiny_layer, T):
    """The multi-workgroup router + selection and the one-workgroup
    permutation (every T above the decode routing's 16 tokens)."""
    wl = TINY.with_(T=T)
    x_t, x = x_device(wl)
    got = tiny_layer.routing_tensors(tiny_layer.route(0, x_t))
    lg = oracle.router_logits(x, wl.router())
    assert np.all(np.abs(got["logits"] - lg) <= 1e-5 * np.abs(lg).max())
    assert np.mean(got["logits"] == lg) >= 0.99
    idx, w = oracle.route_from_logits(lg, wl.k)
    _check_routing(got, idx, w, wl.E)


@pytest.mark.parametrize("T", [1, 4, 5, 16])
def test_decode_routing_ties(torch_mod, tiny_layer, T):
    """A zero router weight makes every logit equal to its expert's bias, so
    the decode routing must break ties by the lower expert id (and order the
    slots by logit, then id) exactly like the oracle's scan."""
    torch = torch_mod
    layer = make_layer(TINY, max_tokens=16)
    bias = np.array([0.5, 1.0, 1.0, -0.0, 0.0, 1.0, 0.5, -2.0], dtype=np.float32)
    layer.load_router(0, torch.zeros(TINY.d * TINY.E, dtype=torch.float32, device="cuda"),
                      torch.from_numpy(bias).cuda())
    x_t, x = x_device(TINY.with_(T=T))
    got = layer.routing_tensors(layer.route(0, x_t))
    lg = oracle.router_logits(x, np.zeros((TINY.d, TINY.E), np.float32), bias)
    assert np.array_equal(lg, np.tile(bias, (T, 1)))      # values (0 + -0 is +0)
    assert np.array_equal(got["logits"].view(np.uint32), lg.view(np.uint32))
    idx, w = oracle.route_from_logits(lg, TINY.k)
    _check_routing(got, idx, w, TINY.E)
    assert idx[0].tolist() == [1, 2]
    layer.close()


@pytest.mark.parametrize("T", [4, 8])
def test_decode_routing_nan_token(torch_mod, tiny_layer, T):
    """A token whose activations hold a NaN has NaN logits (the oracle rejects
    such rows, so no reference exists for them): it still gets k distinct
    valid experts, and the other tokens route exactly as the oracle says."""
    torch = torch_mod
    wl = TINY.with_(T=T)
    x = wl.x().copy()
    x[2, 5] = 0x7FC0                       # bf16 quiet NaN
    x_t = torch.from_numpy(x.view(np.int16)).cuda()
    got = tiny_layer.routing_tensors(tiny_layer.route(0, x_t))
    assert np.isnan(got["logits"][2]).all()
    ids = got["idx"][2]
    assert len(set(ids.tolist())) == wl.k and ids.min() >= 0 and ids.max() < wl.E
    ok = np.array([t for t in range(T) if t != 2])
    lg = oracle.router_logits(x[ok], wl.router())
    idx, w = oracle.route_from_logits(lg, wl.k)
    assert np.array_equal(got["idx"][ok], idx)
    assert np.abs(got["w"][ok] - w).max() <= 2e-6


# 24 experts, top-6: above the decode routing's limits (16 experts, 64 pairs),
# so even one token goes through the general router and permutation
WIDE = TINY.with_(E=24, k=6, T=40)


@pytest.mark.parametrize("T", [1, 16, 40])
def test_wide_routing_layer(torch_mod, T):
    torch = torch_mod
    wl = WIDE.with_(T=T)
    layer = make_layer(wl, max_tokens=40)
    load_workload_host(layer, wl)
    x_t, x = x_device(wl)
    got = layer.routing_tensors(layer.route(0, x_t))
    ref = _oracle_full(wl, x)
    lg = oracle.router_logits(x, wl.router())
    assert np.all(np.abs(got["logits"] - lg) <= 1e-5 * np.abs(lg).max())
    _check_routing(got, ref["idx"], ref["w"], wl.E)
    y = _forward(torch, layer, x_t)
    check_layer_output(y, ref["y64"])
    layer.close()


def _forward(torch, layer, x_t, T=None):
    T = x_t.shape[0] if T is None else T
    # a non-zero fill, so that an output element the layer never writes shows
    y = torch.full((T, layer.cfg.d_model), 0x3F80, dtype=torch.int16, device="cuda")
    layer.forward(0, x_t, y, T=T)
    torch.cuda.synchronize()
    return to_np_u16(y)


def test_binding_rejects_bad_tensors_before_launch(torch_mod, tiny_layer):
    """A short output, a host tensor, a strided view or a wrong dtype never
    reaches the library: the call raises and the output stays untouched."""
    torch = torch_mod
    wl = TINY.with_(T=8)
    x_t, _ = x_device(wl)
    d = wl.d
    y = torch.full((8, d), 0x3F80, dtype=torch.int16, device="cuda")
    wide = torch.zeros((8, 2 * d), dtype=torch.int16, device="cuda")
    cases = [
        (x_t, y[:7], "elements"),                       # 7 rows for 8 tokens
        (x_t.cpu(), y, "expected cuda"),
        (wide[:, ::2], y, "contiguous"),
        (x_t.view(torch.float16), y, "dtype"),
        (x_t, y.float(), "dtype"),
    ]
    for xa, ya, what in cases:
        with pytest.raises(moe.MoeError, match=what):
            tiny_layer.forward(0, xa, ya)
    with pytest.raises(moe.MoeError, match="elements"):
        tiny_layer.forward(0, x_t[:4], y, T=8)
    with pytest.raises(moe.MoeError, match="elements"):
        tiny_layer.route(0, None, T=8, logits_in=torch.zeros((7, wl.E), device="cuda"))
    torch.cuda.synchronize()
    assert bool((y == 0x3F80).all())
    # bfloat16 tensors are accepted as well as their int16 bits
    yb = torch.empty((8, d), dtype=torch.bfloat16, device="cuda")
    tiny_layer.forward(0, x_t.view(torch.bfloat16), yb)
    torch.cuda.synchronize()
    assert np.array_equal(to_np_u16(yb.view(torch.int16)), _forward(torch, tiny_layer, x_t))


def test_binding_rejects_bad_weights_before_load(torch_mod, tiny_layer):
    """Weight loads are checked like activations: a short matrix, weights
    split between host and device, a wrong router dtype or a short bias
    raise before anything is copied, and the loaded layer is unchanged."""
    torch = torch_mod
    wl = TINY
    d, f, E = wl.d, wl.f, wl.E
    x_t, _ = x_device(wl)
    before = _forward(torch, tiny_layer, x_t)
    g = torch.zeros(d * f, dtype=torch.int16, device="cuda")
    cases = [
        (lambda: tiny_layer.load_expert(0, 0, g[:-1], g, g), "elements"),
        (lambda: tiny_layer.load_expert(0, 0, g, g.cpu(), g), "all on the GPU or all on the host"),
        (lambda: tiny_layer.load_expert(0, 0, g.view(torch.float16), g, g), "dtype"),
        (lambda: tiny_layer.load_router(0, torch.zeros(d * E, dtype=torch.float64, device="cuda")),
         "dtype"),
        (lambda: tiny_layer.load_router(0, torch.zeros(d * E, device="cuda"),
                                        torch.zeros(E - 1, device="cuda")), "elements"),
    ]
    for call, what in cases:
        with pytest.raises(moe.MoeError, match=what):
            call()
    assert np.array_equal(_forward(torch, tiny_layer, x_t), before)


def _chain(torch, layer, wl, x, x_t, y, e_begin=0, n_local=0, y_f32=False):
    """check_chain on every token of the layer's last forward (routing
    re-read from an identical moe_route, which leaves H and O in place)."""
    rt = layer.routing_tensors(layer.route(0, x_t))
    lg = oracle.router_logits(x, wl.router(), wl.bias())
    idx, w = oracle.route_from_logits(lg, wl.k)
    assert np.array_equal(rt["idx"], idx)
    G, U, D = host_experts(wl, range(wl.E))
    y64, y16, hb = oracle.layer_with_routing_ex(x, idx, w, G, U, D, e_begin=e_begin,
                                                n_local=n_local, want_hb=True)
    H, O = read_intermediates(torch, layer, int(rt["offsets"][-1]))
    return check_chain(x, rt, H, O, y, {"y64": y64, "y16": y16, "hb": hb, "w": w},
                       lambda e: (G[e], U[e], D[e]), y_f32=y_f32)


@pytest.mark.parametrize("T", [1, 2, 5, 16])
def test_forward_decode_path(torch_mod, tiny_layer, T):
    torch = torch_mod
    wl = TINY.with_(T=T)
    x_t, x = x_device(wl)
    y = _forward(torch, tiny_layer, x_t)
    ref = _oracle_full(wl, x)
    check_layer_output(y, ref["y64"])
    st = _chain(torch, tiny_layer, wl, x, x_t, y)
    assert st["rows"] == T * wl.k


@pytest.mark.parametrize("T", [1, 2, 3])
def test_forward_leaves_the_routing_of_moe_route(torch_mod, tiny_layer, T):
    """A forward without a routing argument routes itself: the views it
    leaves equal moe_route's bit for bit.  Route x, forward another x (the
    views change), forward x again and read the same views."""
    torch = torch_mod
    wl = TINY.with_(T=T)
    x_t, x = x_device(wl)
    x2_t, _ = x_device(wl, layer_idx=1)
    r = tiny_layer.route(0, x_t)
    want = tiny_layer.routing_tensors(r)
    y = torch.empty((T, wl.d), dtype=torch.int16, device="cuda")
    tiny_layer.forward(0, x2_t, y)
    other = tiny_layer.routing_tensors(r)
    assert not np.array_equal(other["logits"].view(np.uint32), want["logits"].view(np.uint32))
    tiny_layer.forward(0, x_t, y)
    got = tiny_layer.routing_tensors(r)
    for key in want:
        assert np.array_equal(np.asarray(got[key]).view(np.uint8),
                              np.asarray(want[key]).view(np.uint8)), key


@pytest.mark.parametrize("T", [17, 100, 300, 512])
def test_forward_gemm_path(torch_mod, tiny_layer, T):
    torch = torch_mod
    wl = TINY.with_(T=T)
    x_t, x = x_device(wl)
    y = _forward(torch, tiny_layer, x_t)
    ref = _oracle_full(wl, x)
    check_layer_output(y, ref["y64"])
    st = _chain(torch, tiny_layer, wl, x, x_t, y)
    assert st["rows"] == T * wl.k


@pytest.mark.parametrize("T", [1, 16, 300])
def test_partial_f32_shares(torch_mod, T):
    """MOE_PARTIAL_F32: a share writes its unrounded fp32 partial (Sec. 4.3:
    what the all-reduce adds).  Its bf16 rounding is the bf16 partial of the
    same share bit for bit (same kernels, same order), it passes the
    per-element chain with the fp32 bound, and the four fp32 partials sum to
    the full layer within the sum of their bounds."""
    torch = torch_mod
    wl = TINY.with_(T=T)
    x_t, x = x_device(wl)
    full = _oracle_full(wl, x)
    total = np.zeros_like(full["y64"])
    bound = np.zeros_like(full["y64"])
    for s in range(4):
        ys = {}
        for flags in (0, moe.MOE_PARTIAL_F32):
            layer = make_layer(wl, max_tokens=max(T, 16), e_begin=2 * s, n_local=2, flags=flags)
            load_workload_host(layer, wl)
            if flags:
                y = torch.full((T, wl.d), 1.5, dtype=torch.float32, device="cuda")
                layer.forward(0, x_t, y)
                torch.cuda.synchronize()
                ys[flags] = y.cpu().numpy()
                st = _chain(torch, layer, wl, x, x_t, ys[flags], e_begin=2 * s, n_local=2,
                            y_f32=True)
                total += ys[flags]
                bound += st["y_bound"]
            else:
                ys[flags] = _forward(torch, layer, x_t)
            layer.close()
        assert np.array_equal(oracle.bf16_round(ys[moe.MOE_PARTIAL_F32].astype(np.float64)), ys[0])
    assert np.all(np.abs(total - full["y64"]) <= bound + 1e-12 * np.abs(full["y64"]))


def test_gemm_timeline_records_and_changes_nothing(torch_mod, tiny_layer):
    """moe_profile_gemm_timeline (measurement): outputs are bit-identical with
    it on, every workgroup with a tile records increasing counters and its
    tile, the rows of each token tile add up to the routing's rows once per
    feature tile, and turning it off stops the recording."""
    torch = torch_mod
    wl = TINY.with_(T=300)
    x_t, _ = x_device(wl)
    before = _forward(torch, tiny_layer, x_t)
    n = 512
    bufs = [torch.zeros(n * 8, dtype=torch.int64, device="cuda") for _ in range(2)]
    moe.moe_profile_gemm_timeline(tiny_layer.ctx, bufs[0].data_ptr(), bufs[1].data_ptr(), n)
    y = _forward(torch, tiny_layer, x_t)
    moe.moe_profile_gemm_timeline(tiny_layer.ctx, None, None, 0)
    assert np.array_equal(y, before)
    rt = tiny_layer.routing_tensors(tiny_layer.route(0, x_t))
    rows = int(rt["offsets"][-1])
    for buf, n_ft in ((bufs[0], 2 * wl.f // 256), (bufs[1], wl.d // 256)):
        t = buf.cpu().numpy().view(np.uint64).reshape(n, 8)
        live = t[t[:, 1] > 0]
        assert len(live) > 0
        assert np.all(live[:, 1] >= live[:, 0]) and np.all(live[:, 3] > live[:, 2])
        r = ((live[:, 5] >> 32) & 0xFFFF).astype(np.int64)
        ft = (live[:, 5] & 0xFFFF).astype(np.int64)
        assert np.all((r > 0) & (r <= 256)) and np.all(ft < n_ft)
        assert int(r.sum()) == rows * n_ft
    for b in bufs:
        b.zero_()
    _forward(torch, tiny_layer, x_t)
    assert not bool(bufs[0].any()) and not bool(bufs[1].any())


def test_routing_validity_rules(torch_mod):
    """moe_forward accepts a routing only while it is the current result of
    the last moe_route for that layer, T and x: an internal re-route, a stack
    forward, another x or a reload of that layer's router make it stale
    (MOE_E_STATE, nothing launched); routing from given logits accepts any x."""
    torch = torch_mod
    wl = TINY.with_(T=8, n_layers=2)
    layer = make_layer(wl, max_tokens=16, n_layers=2)
    try:
        for li in range(2):
            load_workload_host(layer, wl, layer_idx=li)
        x_t, x = x_device(wl)
        x2_t = x_t.flip(0).contiguous()
        y = torch.zeros((8, wl.d), dtype=torch.int16, device="cuda")

        def stale(r, xx=x_t, layer_idx=0):
            y.fill_(7)
            with pytest.raises(moe.MoeError) as ei:
                layer.forward(layer_idx, xx, y, routing=r)
            assert ei.value.status == -5
            torch.cuda.synchronize()
            assert bool((y == 7).all())

        r = layer.route(0, x_t)
        layer.forward(0, x_t, y, routing=r)          # current: accepted
        stale(r, xx=x2_t)                             # computed from another x
        stale(r, layer_idx=1)                         # another layer
        layer.forward(0, x_t, y)                      # internal re-route
        stale(r)
        r = layer.route(0, x_t)
        layer.forward_stack(x2_t.clone())             # the stack re-routes every layer
        stale(r)
        r = layer.route(0, x_t)
        wr = torch.from_numpy(wl.router(0)).cuda()
        layer.load_router(0, wr)                      # same values, still a reload
        stale(r)
        r = layer.route(1, x_t)
        layer.load_router(0, wr)                      # another layer's reload: still valid
        layer.forward(1, x_t, y, routing=r)
        lg = oracle.router_logits(x, wl.router(0))
        r = layer.route(0, None, T=8, logits_in=torch.from_numpy(lg).cuda())
        layer.forward(0, x2_t, y, routing=r)          # given logits: any x
        torch.cuda.synchronize()
    finally:
        layer.close()


@pytest.mark.parametrize("T", [3, 200])
def test_intermediate_h_within_fp32_error_bound(torch_mod, tiny_layer, T):
    """H (the SiLU-gated activations) per grouped row vs the oracle's hb.

    The GPU sums g = x.w1 and u = x.v1 in fp32, so beyond the final bf16
    rounding its H may differ where a sum cancels.  Bound per element: one bf16
    step of the reference plus the fp32 dot-product error bound
    gamma_d * sum|x_i w_i| (gamma_d = d u / (1 - d u), u = 2^-24), carried
    through h = silu(g) u to first order, plus a few fp32 ulps for the
    logistic."""
    torch = torch_mod
    wl = TINY.with_(T=T)
    x_t, x = x_device(wl)
    _forward(torch, tiny_layer, x_t)
    r = tiny_layer.route(0, x_t)   # same routing; H of the last forward stays
    rt = tiny_layer.routing_tensors(r)
    hptr, _ = moe.moe_intermediates(tiny_layer.ctx)
    rows = int(rt["offsets"][-1])
    H = torch.empty((rows, wl.f), dtype=torch.int16, device="cuda")
    moe._copy_dev(H.data_ptr(), hptr, H.numel() * 2)
    H = to_np_u16(H)
    G, U, D = host_experts(wl, range(wl.E))
    u32 = 2.0 ** -24
    gamma = wl.d * u32 / (1 - wl.d * u32)
    exact = []
    for e in range(wl.E):
        r0, r1 = rt["offsets"][e], rt["offsets"][e + 1]
        if r1 == r0:
            continue
        xr = x[rt["row_token"][r0:r1]]
        hb, _ = oracle.expert_glu(xr, G[e], U[e], D[e])
        xf, w1, v1 = bf16_f64(xr), bf16_f64(G[e]), bf16_f64(U[e])
        g, u = xf @ w1, xf @ v1
        s1, s2 = np.abs(xf) @ np.abs(w1), np.abs(xf) @ np.abs(v1)
        sig = 1.0 / (1.0 + np.exp(-g))
        silu = g * sig
        dsilu = sig * (1.0 + g * (1.0 - sig))
        ref = bf16_f64(hb)
        step = np.spacing(np.abs(ref).astype(np.float32)).astype(np.float64) * 65536.0
        bound = step + gamma * (np.abs(dsilu * u) * s1 + np.abs(silu) * s2) + 8 * u32 * np.abs(silu * u)
        err = np.abs(bf16_f64(H[r0:r1]) - ref)
        assert np.all(err <= bound), float((err / bound).max())
        exact.append(np.mean(_ordered(H[r0:r1]) == _ordered(hb)))
    assert np.mean(exact) > 0.95


def _ordered(bits):
    """bf16 bit patterns as integers ordered like their values (+0 == -0)."""
    b = np.asarray(bits, np.uint16).astype(np.int32)
    mag = b & 0x7FFF
    return np.where(b & 0x8000, -mag, mag)


@pytest.mark.parametrize("T", [1, 2, 16])
def test_expert_parallel_shares(torch_mod, T):
    """Shares of 2 of the 8 experts: partial outputs (zero for tokens with no
    local expert, and for a whole share that no token selects) summing to the
    layer."""
    torch = torch_mod
    wl = TINY.with_(T=T)
    x_t, x = x_device(wl)
    full = _oracle_full(wl, x)
    total = np.zeros_like(full["y64"])
    idle = 0
    for s in range(4):
        layer = make_layer(wl, max_tokens=wl.T, e_begin=2 * s, n_local=2)
        load_workload_host(layer, wl)
        y = _forward(torch, layer, x_t)
        ref = _oracle_full(wl, x, e_begin=2 * s, n_local=2)
        has = np.any((full["idx"] >= 2 * s) & (full["idx"] < 2 * s + 2), axis=1)
        assert np.all(y[~has] & 0x7FFF == 0)
        if has.any():
            check_layer_output(y[has], ref["y64"][has])
        total += bf16_f64(y)
        idle += not has.any()
        layer.close()
    assert rel_l2(total, full["y64"]) <= 2e-3
    if T == 1:
        assert idle >= 2      # top-2 of one token leaves at least two shares idle


@pytest.mark.parametrize("T", [40, 300])
def test_expert_parallel_shares_many_tokens(torch_mod, T):
    """Shares through the many-token routing (router + permutation kernels)
    and the grouped GEMM: local counts and rows, partial outputs, and the
    four partials summing to the layer."""
    torch = torch_mod
    wl = TINY.with_(T=T)
    x_t, x = x_device(wl)
    full = _oracle_full(wl, x)
    total = np.zeros_like(full["y64"])
    for s in range(4):
        layer = make_layer(wl, max_tokens=T, e_begin=2 * s, n_local=2)
        load_workload_host(layer, wl)
        got = layer.routing_tensors(layer.route(0, x_t))
        _check_routing(got, full["idx"], full["w"], wl.E, e_begin=2 * s, n_local=2)
        y = _forward(torch, layer, x_t)
        ref = _oracle_full(wl, x, e_begin=2 * s, n_local=2)
        has = np.any((full["idx"] >= 2 * s) & (full["idx"] < 2 * s + 2), axis=1)
        assert np.all(y[~has] & 0x7FFF == 0)
        check_layer_output(y[has], ref["y64"][has])
        total += bf16_f64(y)
        layer.close()
    assert rel_l2(total, full["y64"]) <= 2e-3


def test_deterministic_bitwise(torch_mod, tiny_layer):
    # repeated forwards are bit-identical; d = 256 and f = 512 give the
    # GEMMs one and two K stages after their three-stage main loop, whose
    # barrier waits must still cover the previous stage's B loads
    torch = torch_mod
    for T in (16, 100, 300):
        x_t, _ = x_device(TINY.with_(T=T))
        a = _forward(torch, tiny_layer, x_t)
        for _ in range(30):
            assert np.array_equal(_forward(torch, tiny_layer, x_t), a)


def test_zero_tokens_and_capacity(torch_mod, tiny_layer):
    torch = torch_mod
    x_t = torch.zeros((1, TINY.d), dtype=torch.int16, device="cuda")
    y = torch.full((1, TINY.d), 7, dtype=torch.int16, device="cuda")
    tiny_layer.forward(0, x_t, y, T=0)
    torch.cuda.synchronize()
    assert int(y[0, 0]) == 7           # T == 0 enqueues nothing
    # buffers that hold 513 tokens pass the binding's checks; the library
    # rejects T above max_tokens (512) before launching
    xb = torch.zeros((513, TINY.d), dtype=torch.int16, device="cuda")
    yb = torch.full((513, TINY.d), 7, dtype=torch.int16, device="cuda")
    with pytest.raises(moe.MoeError) as ei:
        tiny_layer.forward(0, xb, yb)
    assert ei.value.status == -4
    torch.cuda.synchronize()
    assert bool((yb == 7).all())


def test_stack_three_layers(torch_mod):
    torch = torch_mod
    wl = TINY.with_(T=4, n_layers=3)
    layer = make_layer(wl, max_tokens=4)
    for li in range(3):
        load_workload_host(layer, wl, layer_idx=li)
    x_t, x = x_device(wl)
    layer.forward_stack(x_t)
    torch.cuda.synchronize()
    got = to_np_u16(x_t)
    # oracle chain, teacher-forced per layer on the GPU's own layer input is
    # not observable here, so compare the end-to-end chain
    cur = x
    for li in range(3):
        ref = _oracle_full(wl, cur, layer_idx=li)
        cur = oracle.residual_add(cur, ref["y"])
    assert rel_l2(bf16_f64(got), bf16_f64(cur)) <= 2e-3
    layer.close()


def test_forward_layers_is_the_stack_in_pieces(torch_mod):
    """moe_forward_layers over ranges that cover the stack equals
    moe_forward_stack bit for bit; one layer of it is moe_forward followed by
    the bf16 residual; an empty range leaves x alone."""
    torch = torch_mod
    wl = TINY.with_(T=4, n_layers=3)
    layer = make_layer(wl, max_tokens=4)
    for li in range(3):
        load_workload_host(layer, wl, layer_idx=li)
    x_t, x = x_device(wl)
    a = x_t.clone()
    layer.forward_stack(a)
    b = x_t.clone()
    layer.forward_layers(0, 1, b)
    layer.forward_layers(1, 2, b)
    c = x_t.clone()
    layer.forward_layers(0, 3, c)
    d = x_t.clone()
    layer.forward_layers(1, 1, d)
    y = torch.empty_like(x_t)
    layer.forward(1, x_t, y)
    e = x_t.clone()
    layer.forward_layers(2, 0, e)
    torch.cuda.synchronize()
    assert np.array_equal(to_np_u16(a), to_np_u16(b)) and np.array_equal(to_np_u16(a), to_np_u16(c))
    assert np.array_equal(to_np_u16(d), oracle.residual_add(x, to_np_u16(y)))
    assert np.array_equal(to_np_u16(e), x)
    layer.close()


def test_forward_residual(torch_mod):
    """moe_forward_residual adds layer(x) into another stream r bit for bit
    as moe_forward plus the bf16 residual, and with r = x it is one layer of
    moe_forward_layers."""
    torch = torch_mod
    wl = TINY.with_(T=4, n_layers=2)
    layer = make_layer(wl, max_tokens=300)
    for li in range(2):
        load_workload_host(layer, wl, layer_idx=li)
    for T in (4, 300):                          # decode GEMVs, then the grouped GEMM
        x_t, x = x_device(wl, T=T)
        r_t, r = x_device(wl, layer_idx=1, T=T)
        y = torch.empty_like(x_t)
        layer.forward(1, x_t, y)
        got = r_t.clone()
        layer.forward_residual(1, x_t, got)
        same = x_t.clone()
        layer.forward_residual(1, same, same)
        ref = x_t.clone()
        layer.forward_layers(1, 1, ref)
        torch.cuda.synchronize()
        assert np.array_equal(to_np_u16(got), oracle.residual_add(r, to_np_u16(y)))
        assert np.array_equal(to_np_u16(same), to_np_u16(ref))
    layer.close()


@pytest.mark.parametrize("nbytes", [16, (1 << 20) + 48, (200 << 20) + 16])
def test_diag_stream_read_reads_every_word_once(torch_mod, nbytes):
    """The bench's streaming-read ceiling: the XOR of the per-workgroup XORs
    equals the XOR of the buffer's 16-byte words (each read once), for sizes
    from one workgroup to a partial last chunk and the unrolled loop's
    remainder."""
    torch = torch_mod
    g = torch.Generator(device="cuda").manual_seed(5)
    buf = torch.randint(-2**31, 2**31 - 1, (nbytes // 4,), dtype=torch.int32, device="cuda", generator=g)
    out = torch.zeros(4 * moe.DIAG_MAX_WG, dtype=torch.int32, device="cuda")
    moe.moe_diag_stream_read(buf.data_ptr(), nbytes, out.data_ptr(),
                             torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    words = buf.cpu().numpy().view(np.uint32).reshape(-1, 4)
    expect = np.bitwise_xor.reduce(words, axis=0)
    got = np.bitwise_xor.reduce(out.cpu().numpy().view(np.uint32).reshape(-1, 4), axis=0)
    assert np.array_equal(got, expect)


def test_diag_bf16_is_round_to_nearest_even_on_every_fp32_pattern(torch_mod):
    """The hardware fp32 -> bf16 conversion that the grouped GEMM's gate/up
    epilogue applies to H, over all 2^32 fp32 bit patterns (16 chunks of
    2^28): equal, bit for bit, to the integer round-to-nearest-even
    (u + 0x7FFF + ((u >> 16) & 1)) >> 16 on every non-NaN input, and a NaN
    for every NaN input."""
    torch = torch_mod
    n = 1 << 28
    s = torch.cuda.current_stream().cuda_stream
    out = torch.empty(n, dtype=torch.int16, device="cuda")
    for c in range(16):
        lo = -(1 << 31) + c * n
        bits = torch.arange(lo, lo + n, dtype=torch.int32, device="cuda")
        moe.moe_diag_bf16(bits.data_ptr(), out.data_ptr(), n, s)
        u = bits.to(torch.int64) & 0xFFFFFFFF
        want = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16) & 0xFFFF
        got = out.to(torch.int64) & 0xFFFF
        nan_in = ((u & 0x7F800000) == 0x7F800000) & ((u & 0x7FFFFF) != 0)
        nan_out = ((got & 0x7F80) == 0x7F80) & ((got & 0x7F) != 0)
        assert torch.equal(nan_in, nan_in & nan_out), f"chunk {c}: a NaN input gave a non-NaN"
        bad = (~nan_in) & (got != want)
        assert int(bad.sum()) == 0, f"chunk {c}: {int(bad.sum())} mismatches"
        del bits, u, want, got, nan_in, nan_out, bad
    torch.cuda.synchronize()
