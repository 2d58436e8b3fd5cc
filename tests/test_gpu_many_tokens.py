"""Token counts whose expert-grouped permutation takes several rounds of the
permutation kernel (it places pairs 8192 at a time, carrying per-expert
cursors between rounds): 5000 tokens at top-4 (20000 pairs, three rounds)
and 20000 tokens at top-2 (40000 pairs, five rounds), with the prefill
workload's skew bias so that expert loads are uneven, on a small layer
(d 256, ffn 128, 16 experts) the oracle evaluates in seconds.  Routing from
identical logits and from x is bit-exact against the oracle; the layer and a
4-of-16 share are checked per element on every token."""
import numpy as np
import pytest

import moe_inputs as mi
import oracle
from harness import (check_chain, check_layer_output, load_workload_host, make_layer,
                     read_intermediates, to_np_u16)

pytestmark = pytest.mark.gpu

BASE = mi.Workload("many_tokens", T=5000, d=256, f=128, E=16, k=4, sigma_w=0.05, sigma_b=1.0,
                   seed=3)
CASES = [(5000, 4), (20000, 2)]


@pytest.fixture(scope="module")
def torch_mod():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch


def _weights(wl):
    cache = {}

    def get(e):
        if e not in cache:
            cache[e] = (wl.gate(e), wl.up(e), wl.down(e))
        return cache[e]
    return get


def _ref(wl, x, idx, w, get, e_begin=0, n_local=0):
    G, U, D = [None] * wl.E, [None] * wl.E, [None] * wl.E
    for e in range(wl.E):
        G[e], U[e], D[e] = get(e)
    y64, y16, hb = oracle.layer_with_routing_ex(x, idx, w, G, U, D, e_begin=e_begin,
                                                n_local=n_local, want_hb=True)
    return {"y64": y64, "y16": y16, "hb": hb, "w": w}


@pytest.mark.parametrize("T,k", CASES)
def test_multi_round_permutation_and_layer(torch_mod, T, k):
    torch = torch_mod
    wl = BASE.with_(T=T, k=k)
    assert T * k > 2 * 8192
    get = _weights(wl)
    x = wl.x()
    x_t = torch.from_numpy(x.view(np.int16)).cuda()
    lg = oracle.router_logits(x, wl.router(), wl.bias())
    idx, w = oracle.route_from_logits(lg, k)
    counts, offsets, pair_row, row_token = oracle.permutation(idx, wl.E)
    assert counts.max() > 8192 // 2 or counts.max() > 2 * counts.mean()
    for e_begin, n_local in ((0, 0), (4, 4)):
        layer = make_layer(wl, max_tokens=T, e_begin=e_begin, n_local=n_local or wl.E)
        try:
            load_workload_host(layer, wl)
            nl = n_local or wl.E
            c, o, pr, rtok = oracle.permutation(idx, wl.E, e_begin, nl)
            # given logits: bit-exact ids, weights within 2e-6, permutation
            got = layer.routing_tensors(layer.route(0, x_t, logits_in=torch.from_numpy(lg).cuda()))
            assert np.array_equal(got["idx"], idx)
            assert np.abs(got["w"] - w).max() <= 2e-6
            for name, ref in (("counts", c), ("offsets", o), ("pair_row", pr),
                              ("row_token", rtok)):
                assert np.array_equal(got[name], ref), name
            # from x, then the layer on that routing
            rt = layer.routing_tensors(layer.route(0, x_t))
            assert np.array_equal(rt["idx"], idx) and np.array_equal(rt["pair_row"], pr)
            y = torch.full((T, wl.d), 0x3F80, dtype=torch.int16, device="cuda")
            layer.forward(0, x_t, y)
            torch.cuda.synchronize()
            y = to_np_u16(y)
            ref = _ref(wl, x, idx, w, get, e_begin, nl)
            has = (pr >= 0).any(axis=1)
            check_layer_output(y[has], ref["y64"][has])
            H, O = read_intermediates(torch, layer, int(o[-1]))
            st = check_chain(x, rt, H, O, y, ref, get)
            assert st["rows"] == int(o[-1])
        finally:
            layer.close()
