"""The layer at the limits the C-ABI accepts: 64 experts (the most a config
may hold) with top-8 and top-64 (every expert selected), a single expert
(top-1: a dense FFN), and the smallest shapes (d = 256, f = 128, so each GEMM
is one feature tile and the down GEMM's two K stages all run after its main
loop).  Token counts cover the decode GEMVs (T <= 16) and the grouped GEMM
(T > 16).  Checked against the oracle: routing ids exactly, weights to fp32
rounding, the output to the layer tolerance."""
import numpy as np
import pytest

import moe_inputs as mi
import oracle
from harness import check_layer_output, load_workload_host, make_layer, x_device

pytestmark = pytest.mark.gpu

BASE = mi.WORKLOADS["tiny"].with_(d=256, f=128)
CASES = [
    ("e64_top8", BASE.with_(E=64, k=8), (1, 16, 17, 200)),
    ("e64_top64", BASE.with_(E=64, k=64), (1, 4, 20)),
    ("e1_top1", BASE.with_(E=1, k=1), (1, 16, 300)),
    ("e8_top2_d512", BASE.with_(E=8, k=2, d=512, f=256), (3, 50)),
]


@pytest.fixture(scope="module")
def torch_mod():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch


def _oracle(wl, x):
    G, U, D = [], [], []
    for e in range(wl.E):
        G.append(wl.gate(e, 0))
        U.append(wl.up(e, 0))
        D.append(wl.down(e, 0))
    return oracle.layer(x, wl.router(0), wl.bias(0), G, U, D, wl.k)


@pytest.mark.parametrize("name,wl,Ts", CASES, ids=[c[0] for c in CASES])
def test_layer_at_limits(torch_mod, name, wl, Ts):
    torch = torch_mod
    layer = make_layer(wl, max_tokens=max(Ts))
    load_workload_host(layer, wl)
    try:
        for T in Ts:
            w = wl.with_(T=T)
            x_t, x = x_device(w)
            got = layer.routing_tensors(layer.route(0, x_t))
            ref = _oracle(w, x)
            assert np.array_equal(got["idx"], ref["idx"]), (name, T)
            assert np.abs(got["w"] - ref["w"]).max() <= 2e-6, (name, T)
            assert np.array_equal(got["counts"], np.bincount(ref["idx"].reshape(-1), minlength=w.E))
            y = torch.full((T, w.d), 0x3F80, dtype=torch.int16, device="cuda")
            layer.forward(0, x_t, y)
            torch.cuda.synchronize()
            check_layer_output(y.cpu().numpy().view(np.uint16), ref["y64"])
    finally:
        layer.close()
