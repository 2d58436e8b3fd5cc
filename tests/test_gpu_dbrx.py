"""GPU parity at DBRX shape (d_model 6144, ffn 10752, 16 experts, top-4)
through the C-ABI, in the launch configuration the benchmark times.

Weights are generated straight into HBM by the device generator (bit-equal to
the host generator, checked in test_gpu_tiny) and prestacked by
moe_load_expert; the oracle regenerates the experts it needs on the host.
Full-size routing is checked for every token; layer outputs on all tokens for
decode, on sampled tokens for prefill (the oracle computes a token alone)."""
import functools

import numpy as np
import pytest

import moe_inputs as mi
import oracle
from harness import (bf16_f64, check_layer_output, load_workload_device, make_layer, rel_l2,
                     to_np_u16)

pytestmark = pytest.mark.gpu

DECODE = mi.WORKLOADS["decode"]
SHARE = mi.WORKLOADS["ep_share"]
PREFILL = mi.WORKLOADS["prefill"]


@pytest.fixture(scope="module")
def torch_mod():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch


@functools.lru_cache(maxsize=32)
def host_weights(wl, e, layer=0):
    return wl.gate(e, layer), wl.up(e, layer), wl.down(e, layer)


def weights_for(wl, experts, layer=0):
    G, U, D = [None] * wl.E, [None] * wl.E, [None] * wl.E
    for e in experts:
        G[e], U[e], D[e] = host_weights(wl, e, layer)
    return G, U, D


def x_dev(torch, wl):
    x = wl.x()
    return torch.from_numpy(x.view(np.int16)).cuda(), x


def run_forward(torch, layer, x_t):
    # a non-zero fill, so that an output element the layer never writes shows
    y = torch.full((x_t.shape[0], layer.cfg.d_model), 0x3F80, dtype=torch.int16, device="cuda")
    layer.forward(0, x_t, y)
    torch.cuda.synchronize()
    return to_np_u16(y)


@pytest.fixture(scope="module")
def decode_layer(torch_mod):
    layer = make_layer(DECODE, max_tokens=16)
    load_workload_device(layer, DECODE)
    yield layer
    layer.close()


@pytest.mark.parametrize("T", [1, 4, 8, 16])
def test_decode_full_layer(torch_mod, decode_layer, T):
    torch = torch_mod
    wl = DECODE.with_(T=T)
    x_t, x = x_dev(torch, wl)
    r = decode_layer.route(0, x_t)
    rt = decode_layer.routing_tensors(r)
    lg = oracle.router_logits(x, wl.router())
    assert np.all(np.abs(rt["logits"] - lg) <= 1e-5 * np.abs(lg).max())
    idx, w = oracle.route_from_logits(lg, wl.k)
    assert np.array_equal(rt["idx"], idx)
    assert np.abs(rt["w"] - w).max() <= 2e-6
    y = run_forward(torch, decode_layer, x_t)
    G, U, D = weights_for(wl, sorted(set(idx.reshape(-1).tolist())))
    y64, _ = oracle.layer_with_routing(x, idx, w, G, U, D)
    check_layer_output(y, y64)
    # the K-split GEMVs' H and O, every row
    checked, exact, _ = check_intermediates(torch, decode_layer, wl, x, rt,
                                            lambda r0, r1: list(range(r0, r1)))
    assert checked == T * wl.k and exact > 0.9


@pytest.mark.parametrize("T", [1, 4, 8])
def test_expert_parallel_share(torch_mod, T):
    """One node's 4-of-16 share (experts 4s..4s+3) for each s; routing from the
    full 16-way logits; partial outputs; the four partials sum to the layer."""
    torch = torch_mod
    wl = SHARE.with_(T=T)
    x_t, x = x_dev(torch, wl)
    lg = oracle.router_logits(x, wl.router())
    idx, w = oracle.route_from_logits(lg, wl.k)
    G, U, D = weights_for(wl, sorted(set(idx.reshape(-1).tolist())))
    full64, _ = oracle.layer_with_routing(x, idx, w, G, U, D)
    total = np.zeros_like(full64)
    staging = None
    for s in range(4):
        share = wl.with_(e_begin=4 * s, n_local=4)
        layer = make_layer(share, max_tokens=8)
        staging = load_workload_device(layer, share, staging=staging)
        y = run_forward(torch, layer, x_t)
        rt = layer.routing_tensors(layer.route(0, x_t))
        assert np.array_equal(rt["idx"], idx)
        local = (idx >= 4 * s) & (idx < 4 * s + 4)
        assert np.array_equal(rt["counts"][4 * s:4 * s + 4],
                              np.bincount(idx[local].reshape(-1) - 4 * s, minlength=4))
        ref64, _ = oracle.layer_with_routing(x, idx, w, G, U, D, e_begin=4 * s, n_local=4)
        has = local.any(axis=1)
        assert np.all((y[~has] & 0x7FFF) == 0)
        if has.any():
            check_layer_output(y[has], ref64[has])
        total += bf16_f64(y)
        layer.close()
    assert rel_l2(total, full64) <= 2e-3


@pytest.fixture(scope="module")
def prefill_layer(torch_mod):
    layer = make_layer(PREFILL, max_tokens=PREFILL.T)
    load_workload_device(layer, PREFILL)
    yield layer
    layer.close()


@pytest.fixture(scope="module")
def prefill_ref():
    x = PREFILL.x()
    lg = oracle.router_logits(x, PREFILL.router(), PREFILL.bias())
    idx, w = oracle.route_from_logits(lg, PREFILL.k)
    return x, lg, idx, w


def test_prefill_routing_all_tokens(torch_mod, prefill_layer, prefill_ref):
    torch = torch_mod
    x, lg, idx, w = prefill_ref
    x_t = torch.from_numpy(x.view(np.int16)).cuda()
    # from identical fp32 logits: bit-exact ids and permutation
    rt = prefill_layer.routing_tensors(prefill_layer.route(0, x_t, logits_in=torch.from_numpy(lg).cuda()))
    assert np.array_equal(rt["idx"], idx)
    assert np.abs(rt["w"] - w).max() <= 2e-6
    counts, offsets, pair_row, row_token = oracle.permutation(idx, PREFILL.E)
    assert np.array_equal(rt["counts"], counts)
    assert np.array_equal(rt["pair_row"], pair_row)
    assert np.array_equal(rt["row_token"], row_token)
    # the skew bias makes the expert loads uneven
    assert counts.max() > 2 * counts.mean()
    # from x: the router's fp64 accumulation reproduces the oracle's logits
    rt2 = prefill_layer.routing_tensors(prefill_layer.route(0, x_t))
    assert np.mean(rt2["logits"] == lg) > 0.999
    assert np.all(np.abs(rt2["logits"] - lg) <= 1e-5 * np.abs(lg).max())
    assert np.array_equal(rt2["idx"], idx)


def test_prefill_layer_sampled_tokens(torch_mod, prefill_layer, prefill_ref):
    torch = torch_mod
    x, lg, idx, w = prefill_ref
    x_t = torch.from_numpy(x.view(np.int16)).cuda()
    y = run_forward(torch, prefill_layer, x_t)
    T = PREFILL.T
    rng = np.random.default_rng(0)
    counts = np.bincount(idx.reshape(-1), minlength=PREFILL.E)
    rare = int(np.argmin(np.where(counts > 0, counts, 10 ** 9)))
    picks = {0, 1, T - 1, T // 2} | set(rng.choice(T, 8, replace=False).tolist())
    picks |= set(np.nonzero((idx == rare).any(axis=1))[0][:2].tolist())
    picks = sorted(picks)
    G, U, D = weights_for(PREFILL, range(PREFILL.E))
    y64, _ = oracle.layer_with_routing(x[picks], idx[picks], w[picks], G, U, D)
    check_layer_output(y[picks], y64)
    assert np.all(np.isfinite(bf16_f64(y)))


def _edge_rows(r0, r1, tile=256):
    """Grouped rows of one expert at MFMA-block (32), pair (64) and tile
    (256) edges, and its last row (the partial tile's end)."""
    out = set()
    for base in range(r0, r1, tile):
        for off in (0, 31, 32, 63, 64, 127, 128, 191, 192, tile - 1):
            if base + off < r1:
                out.add(base + off)
    out.add(r1 - 1)
    return sorted(out)


def check_intermediates(torch, layer, wl, x, rt, pick_rows):
    """H and O of the layer's last forward, for the grouped rows
    pick_rows(r0, r1) of every expert: H against the oracle within the
    fp32-accumulation bound (gamma_d sum |x||w| carried through silu(g) u,
    one bf16 step, a few fp32 ulps for the logistic); O against an fp64 down
    projection of the GPU's own H within gamma_f sum |h||w2| (bf16 x bf16
    products are exact in fp32, so only the accumulation rounds).  Returns
    (rows checked, fraction of H bit-exact, tokens of the checked rows)."""
    import paper_2506_23635_amd as moe
    hptr, optr = moe.moe_intermediates(layer.ctx)
    rows, d, f = int(rt["offsets"][-1]), wl.d, wl.f
    H = torch.empty((rows, f), dtype=torch.int16, device="cuda")
    O = torch.empty((rows, d), dtype=torch.float32, device="cuda")
    moe._copy_dev(H.data_ptr(), hptr, H.numel() * 2)
    moe._copy_dev(O.data_ptr(), optr, O.numel() * 4)
    torch.cuda.synchronize()
    H = H.cpu().numpy().view(np.uint16)
    O = O.cpu().numpy().astype(np.float64)
    u32 = 2.0 ** -24
    gd, gf = d * u32 / (1 - d * u32), f * u32 / (1 - f * u32)
    tokens, exact, checked = set(), [], 0
    for e in range(wl.E):
        r0, r1 = int(rt["offsets"][e]), int(rt["offsets"][e + 1])
        if r1 == r0:
            continue
        er = pick_rows(r0, r1)
        toks = rt["row_token"][er]
        tokens.update(toks.tolist())
        g_w, u_w, d_w = host_weights(wl, e)
        hb, _ = oracle.expert_glu(x[toks], g_w, u_w, d_w)
        xf, w1, v1 = bf16_f64(x[toks]), bf16_f64(g_w), bf16_f64(u_w)
        g, u = xf @ w1, xf @ v1
        s1, s2 = np.abs(xf) @ np.abs(w1), np.abs(xf) @ np.abs(v1)
        sig = 1.0 / (1.0 + np.exp(-g))
        silu, dsilu = g * sig, sig * (1.0 + g * (1.0 - sig))
        ref = bf16_f64(hb)
        step = np.spacing(np.abs(ref).astype(np.float32)).astype(np.float64) * 65536.0
        bound = step + gd * (np.abs(dsilu * u) * s1 + np.abs(silu) * s2) + 8 * u32 * np.abs(silu * u)
        hg = bf16_f64(H[er])
        assert np.all(np.abs(hg - ref) <= bound), (e, float((np.abs(hg - ref) / bound).max()))
        exact.append(np.mean(hg == ref))
        w2 = bf16_f64(d_w)
        o_ref = hg @ w2
        o_bound = gf * (np.abs(hg) @ np.abs(w2)) + 1e-30
        assert np.all(np.abs(O[er] - o_ref) <= o_bound), (e, float((np.abs(O[er] - o_ref) / o_bound).max()))
        checked += len(er)
    return checked, float(np.mean(exact)), sorted(tokens)


def test_prefill_tile_edges(torch_mod, prefill_layer, prefill_ref):
    """Full DBRX shape, 2048 skewed tokens: for every expert, the grouped rows
    at block, pair and tile edges and the last row of its partial tile; H and
    O (check_intermediates), and y of those rows' tokens against the
    oracle."""
    torch = torch_mod
    x, lg, idx, w = prefill_ref
    x_t = torch.from_numpy(x.view(np.int16)).cuda()
    y = run_forward(torch, prefill_layer, x_t)
    rt = prefill_layer.routing_tensors(prefill_layer.route(0, x_t))   # same routing
    checked, exact, picks = check_intermediates(torch, prefill_layer, PREFILL, x, rt, _edge_rows)
    assert checked > 100 and exact > 0.9
    G, U, D = weights_for(PREFILL, range(PREFILL.E))
    y64, _ = oracle.layer_with_routing(x[picks], idx[picks], w[picks], G, U, D)
    check_layer_output(y[picks], y64)


def test_prefill_deterministic(torch_mod, prefill_layer, prefill_ref):
    torch = torch_mod
    x = prefill_ref[0]
    x_t = torch.from_numpy(x.view(np.int16)).cuda()
    a = run_forward(torch, prefill_layer, x_t)
    b = run_forward(torch, prefill_layer, x_t)
    assert np.array_equal(a, b)
