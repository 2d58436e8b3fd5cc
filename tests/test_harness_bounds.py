"""The per-element parity bounds of harness.check_chain, on the CPU: an
independent fp32 emulation of the layer (numpy float32 matmuls, the way the
GPU accumulates) must pass them, and errors the size of a wrong element,
column or row must not.  This keeps the GPU tests' bounds from being either
too tight or vacuous."""
import numpy as np
import pytest

import moe_inputs as mi
import oracle
from harness import bf16_f64, check_chain

WL = mi.WORKLOADS["tiny"].with_(T=24)


def _bf16_bits(a32):
    return oracle.bf16_round(np.asarray(a32, np.float64))


def _emulate(wl, x, idx, w32, e_begin=0, n_local=0):
    """fp32 dataflow of the layer: grouped rows, H, O, y (bits)."""
    nl = n_local or wl.E
    counts, offsets, pair_row, row_token = oracle.permutation(idx, wl.E, e_begin, nl)
    rows = int(offsets[-1])
    H = np.zeros((rows, wl.f), np.uint16)
    O = np.zeros((rows, wl.d), np.float64)
    for e in range(e_begin, e_begin + nl):
        r0, r1 = int(offsets[e]), int(offsets[e + 1])
        if r1 == r0:
            continue
        xr = mi.bf16_bits_to_f32(x[row_token[r0:r1]])
        g = xr @ mi.bf16_bits_to_f32(wl.gate(e))
        u = xr @ mi.bf16_bits_to_f32(wl.up(e))
        h = (g / (np.float32(1) + np.exp(-g)) * u).astype(np.float32)
        H[r0:r1] = _bf16_bits(h)
        O[r0:r1] = mi.bf16_bits_to_f32(H[r0:r1]) @ mi.bf16_bits_to_f32(wl.down(e))
    acc = np.zeros((x.shape[0], wl.d), np.float32)
    for j in range(idx.shape[1]):
        loc = pair_row[:, j] >= 0
        acc[loc] = acc[loc] + w32[loc, j:j + 1] * O[pair_row[loc, j]].astype(np.float32)
    rt = {"idx": idx, "w": w32, "pair_row": pair_row, "offsets": offsets,
          "row_token": row_token}
    return rt, H, O, acc


def _ref(wl, x, idx, w, e_begin=0, n_local=0):
    G = [wl.gate(e) for e in range(wl.E)]
    U = [wl.up(e) for e in range(wl.E)]
    D = [wl.down(e) for e in range(wl.E)]
    y64, y16, hb = oracle.layer_with_routing_ex(x, idx, w, G, U, D, e_begin=e_begin,
                                                n_local=n_local, want_hb=True)
    return {"y64": y64, "y16": y16, "hb": hb, "w": w}


@pytest.fixture(scope="module")
def case():
    x = WL.x()
    lg = oracle.router_logits(x, WL.router())
    idx, w = oracle.route_from_logits(lg, WL.k)
    return x, idx, w


def _weights(e):
    return WL.gate(e), WL.up(e), WL.down(e)


@pytest.mark.parametrize("share", [None, (2, 2)])
def test_fp32_emulation_passes(case, share):
    x, idx, w = case
    eb, nl = share or (0, 0)
    w32 = w.astype(np.float32)
    rt, H, O, acc = _emulate(WL, x, idx, w32, eb, nl)
    ref = _ref(WL, x, idx, w, eb, nl)
    st = check_chain(x, rt, H, O, _bf16_bits(acc), ref, _weights)
    assert st["rows"] == int(rt["offsets"][-1]) and st["h_exact"] > 0.9
    st32 = check_chain(x, rt, H, O, acc, ref, _weights, y_f32=True)
    assert st32["combine_worst"] <= 1.0


@pytest.mark.parametrize("where", ["h_element", "o_column", "y_column", "y_token", "weight"])
def test_planted_errors_fail(case, where):
    x, idx, w = case
    w32 = w.astype(np.float32)
    rt, H, O, acc = _emulate(WL, x, idx, w32)
    ref = _ref(WL, x, idx, w)
    y = _bf16_bits(acc)
    if where == "h_element":
        H[3, 7] = _bf16_bits(bf16_f64(H[3:4, 7]) * 1.02 + 0.05)[0]
    elif where == "o_column":
        O[:, 11] *= 1.01
    elif where == "y_column":
        y[:, 5] = _bf16_bits(bf16_f64(y[:, 5]) * 1.03)
    elif where == "y_token":
        y[4] = 0
    else:
        rt = dict(rt, w=w32 * np.float32(1.001))
    with pytest.raises(AssertionError):
        check_chain(x, rt, H, O, y, ref, _weights)
