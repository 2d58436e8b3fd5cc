"""Shared test helpers: put a synthetic workload into a MoeLayer (device side)
and compute the matching oracle results (host side).  Inputs come only from
moe_inputs; expected values come only from oracle/."""
from __future__ import annotations

import numpy as np

import moe_inputs as mi


def rel_l2(got, ref) -> float:
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    den = np.linalg.norm(ref)
    return float(np.linalg.norm(got - ref) / den) if den > 0 else float(np.linalg.norm(got))


def bf16_f64(bits) -> np.ndarray:
    return mi.bf16_bits_to_f32(np.asarray(bits, np.uint16)).astype(np.float64)


def check_layer_output(y_bits, y64_ref, rel_tol=2e-3, abs_tol=1e-2):
    """The parity bar for layer outputs: relative L2 <= 2e-3 and max-abs
    <= 1e-2 * max(1, max|y_ref|) against the oracle's fp64 result."""
    got = bf16_f64(y_bits)
    r = rel_l2(got, y64_ref)
    scale = max(1.0, float(np.abs(y64_ref).max()) if y64_ref.size else 1.0)
    ma = float(np.abs(got - y64_ref).max()) if got.size else 0.0
    assert r <= rel_tol, f"relative L2 {r:.3e} > {rel_tol}"
    assert ma <= abs_tol * scale, f"max abs {ma:.3e} > {abs_tol} * {scale:.3e}"
    return r, ma


def make_layer(wl: mi.Workload, max_tokens=None, e_begin=None, n_local=None, n_layers=None,
               flags=0):
    import paper_2506_23635_amd as moe
    cfg = moe.make_config(wl.d, wl.f, wl.E, wl.k,
                          expert_begin=wl.e_begin if e_begin is None else e_begin,
                          n_local_experts=(wl.local if n_local is None else n_local),
                          n_layers=wl.n_layers if n_layers is None else n_layers,
                          max_tokens=max_tokens or wl.T, flags=flags)
    return moe.MoeLayer(cfg)


def load_workload_host(layer, wl: mi.Workload, layer_idx=0, experts=None, arena_layer=None):
    """Generate on the host and upload (small shapes)."""
    import torch
    dev = layer.device
    al = layer_idx if arena_layer is None else arena_layer
    wr = torch.from_numpy(wl.router(layer_idx)).to(dev)
    b = wl.bias(layer_idx)
    layer.load_router(al, wr, torch.from_numpy(b).to(dev) if b is not None else None)
    c = layer.cfg
    es = experts if experts is not None else range(c.expert_begin, c.expert_begin + c.n_local_experts)
    for e in es:
        g = torch.from_numpy(wl.gate(e, layer_idx).view(np.int16)).to(dev)
        u = torch.from_numpy(wl.up(e, layer_idx).view(np.int16)).to(dev)
        dn = torch.from_numpy(wl.down(e, layer_idx).view(np.int16)).to(dev)
        layer.load_expert(al, e, g, u, dn)
    torch.cuda.synchronize()


def load_workload_device(layer, wl: mi.Workload, layer_idx=0, arena_layer=None, staging=None):
    """Generate every tensor straight into HBM with the device generator (same
    bits as the host generator) and prestack it through moe_load_expert."""
    import torch
    dev = layer.device
    al = layer_idx if arena_layer is None else arena_layer
    s = layer.stream
    d, f, E = wl.d, wl.f, wl.E
    wr = torch.empty(d * E, dtype=torch.float32, device=dev)
    mi.gen_f32_device(wl.seed, mi.stream_id(mi.KIND_ROUTER, layer_idx), d * E, wl.sigma_r,
                      wr.data_ptr(), s)
    b = None
    if wl.sigma_b:
        b = torch.empty(E, dtype=torch.float32, device=dev)
        mi.gen_f32_device(wl.seed, mi.stream_id(mi.KIND_BIAS, layer_idx), E, wl.sigma_b,
                          b.data_ptr(), s)
    layer.load_router(al, wr, b)
    if staging is None:
        staging = torch.empty(3 * d * f, dtype=torch.int16, device=dev)
    g, u, dn = staging[: d * f], staging[d * f: 2 * d * f], staging[2 * d * f:]
    c = layer.cfg
    for e in range(c.expert_begin, c.expert_begin + c.n_local_experts):
        mi.gen_bf16_device(wl.seed, mi.stream_id(mi.KIND_GATE, layer_idx, e), d * f, wl.sigma_w,
                           g.data_ptr(), s)
        mi.gen_bf16_device(wl.seed, mi.stream_id(mi.KIND_UP, layer_idx, e), d * f, wl.sigma_w,
                           u.data_ptr(), s)
        mi.gen_bf16_device(wl.seed, mi.stream_id(mi.KIND_DOWN, layer_idx, e), d * f, wl.sigma_w,
                           dn.data_ptr(), s)
        layer.load_expert(al, e, g, u, dn)
    torch.cuda.synchronize()
    return staging


def x_device(wl: mi.Workload, layer_idx=0, T=None):
    import torch
    x = wl.x(layer_idx) if T is None else wl.with_(T=T).x(layer_idx)
    return torch.from_numpy(x.view(np.int16)).cuda(), x


def host_experts(wl: mi.Workload, experts, layer_idx=0):
    """Host copies of the weights of the given experts (others None)."""
    G = [None] * wl.E
    U = [None] * wl.E
    D = [None] * wl.E
    for e in experts:
        G[e] = wl.gate(e, layer_idx)
        U[e] = wl.up(e, layer_idx)
        D[e] = wl.down(e, layer_idx)
    return G, U, D


def to_np_u16(t) -> np.ndarray:
    return t.cpu().numpy().view(np.uint16)


# ------------------------------------------------------ per-element chain --

U32 = 2.0 ** -24


def gamma(n) -> float:
    """gamma_n = n u / (1 - n u) for fp32 (u = 2^-24): the relative error bound
    of an n-term fp32 sum (of exact products) in any order."""
    return n * U32 / (1 - n * U32)


def bf16_step(v) -> np.ndarray:
    """The spacing of bf16 values at |v| (fp32 spacing times 2^16)."""
    return np.spacing(np.abs(np.asarray(v, np.float64)).astype(np.float32)).astype(np.float64) * 65536.0


def ordered(bits) -> np.ndarray:
    """bf16 bit patterns as integers ordered like their values (+0 == -0)."""
    b = np.asarray(bits, np.uint16).astype(np.int32)
    mag = b & 0x7FFF
    return np.where(b & 0x8000, -mag, mag)


def read_intermediates(torch, layer, rows):
    """H (bf16 bits [rows, f]) and O (fp64 [rows, d]) of the layer's last
    forward, copied back through moe_intermediates."""
    import paper_2506_23635_amd as moe
    d, f = layer.cfg.d_model, layer.cfg.ffn_dim
    hptr, optr = moe.moe_intermediates(layer.ctx)
    H = torch.empty((max(rows, 1), f), dtype=torch.int16, device=layer.device)
    O = torch.empty((max(rows, 1), d), dtype=torch.float32, device=layer.device)
    if rows:
        moe._copy_dev(H.data_ptr(), hptr, rows * f * 2)
        moe._copy_dev(O.data_ptr(), optr, rows * d * 4)
    torch.cuda.synchronize()
    return H.cpu().numpy().view(np.uint16)[:rows], O.cpu().numpy().astype(np.float64)[:rows]


def check_chain(x, rt, H, O, y, ref, weights, tokens=None, y_f32=False):
    """Per-element parity of every stage of the layer for the given tokens
    (default: all), each stage against the oracle or against the GPU's own
    input to that stage, with bounds derived from fp32 arithmetic:

    H   vs the oracle's hb (same routing): one bf16 step of hb plus the fp32
        dot-product bound gamma_d sum|x||w| carried through silu(g) u to first
        order, plus a few fp32 ulps for the logistic;
    O   vs the fp64 product of the GPU's own H with w2: gamma_f sum|h||w2|
        (bf16 x bf16 products are exact in fp32, only the sum rounds);
    y   vs the fp64 combine of the GPU's own O and fp32 weights, in slot
        order: half a bf16 step (bf16 output) plus gamma_k sum|w o|;
    y   vs the oracle's fp64 y (before its rounding): the combine bound plus,
        per slot, |w - w_oracle||o| and |w_oracle| (gamma_f sum|h||w2| +
        sum|h - hb||w2|), i.e. the H differences found above carried through
        the down projection.
    Tokens with no local slot must give exact zeros.

    x: bf16 bits [T, d]; rt: the GPU routing (routing_tensors); H, O: the
    GPU's intermediates; y: GPU output, bf16 bits or fp32 [T, d]; ref:
    {"y64": [T, d], "hb": [T, k, f] bf16 bits, "w": [T, k]} from
    oracle.layer_with_routing_ex on the same ids; weights(e) -> (gate, up,
    down) bf16 bits.  Returns a dict of statistics, with "y_bound" the
    per-element bound on |y - y_oracle| for the chosen tokens."""
    T, k = rt["idx"].shape
    d = x.shape[1]
    tokens = np.arange(T) if tokens is None else np.asarray(sorted(tokens))
    pair_row, idx = rt["pair_row"], rt["idx"]
    w32 = rt["w"].astype(np.float64)
    w64 = np.asarray(ref["w"], np.float64)
    # (row -> pair) for the local pairs of the chosen tokens, grouped by expert
    by_e = {}
    for t in tokens:
        for j in range(k):
            r = int(pair_row[t, j])
            if r >= 0:
                by_e.setdefault(int(idx[t, j]), []).append((r, int(t), j))
    f = H.shape[1] if H.size else 0
    tpos = np.full(T, -1)
    tpos[tokens] = np.arange(len(tokens))
    habs = np.zeros((len(tokens), k, d))   # sum_n |h_n| |w2[n, :]| per pair
    dh = np.zeros((len(tokens), k, d))     # sum_n |h_n - hb_n| |w2[n, :]| per pair
    gd, gf = gamma(d), gamma(f)
    h_exact, h_worst, o_worst = [], 0.0, 0.0
    for e, plist in sorted(by_e.items()):
        rows = np.array([p[0] for p in plist])
        pt = np.array([p[1] for p in plist])
        pj = np.array([p[2] for p in plist])
        g_w, u_w, d_w = weights(e)
        xf = bf16_f64(x[pt])
        w1 = bf16_f64(g_w)
        g = xf @ w1
        s1 = np.abs(xf) @ np.abs(w1)
        del w1
        v1 = bf16_f64(u_w)
        u = xf @ v1
        s2 = np.abs(xf) @ np.abs(v1)
        del v1
        sig = 1.0 / (1.0 + np.exp(-g))
        silu, dsilu = g * sig, sig * (1.0 + g * (1.0 - sig))
        hb = ref["hb"][pt, pj]
        href = bf16_f64(hb)
        hbound = (bf16_step(href) + gd * (np.abs(dsilu * u) * s1 + np.abs(silu) * s2)
                  + 8 * U32 * np.abs(silu * u))
        del g, u, s1, s2, sig, silu, dsilu
        hg = bf16_f64(H[rows])
        herr = np.abs(hg - href)
        assert np.all(herr <= hbound), ("H", e, float((herr / hbound).max()))
        h_worst = max(h_worst, float((herr / hbound).max()))
        h_exact.append(np.mean(ordered(H[rows]) == ordered(hb)))
        w2 = bf16_f64(d_w)
        aw2 = np.abs(w2)
        o_ref = hg @ w2
        hab = np.abs(hg) @ aw2
        ob = gf * hab + 1e-30
        oerr = np.abs(O[rows] - o_ref)
        assert np.all(oerr <= ob), ("O", e, float((oerr / ob).max()))
        o_worst = max(o_worst, float((oerr / ob).max()))
        habs[tpos[pt], pj] = hab
        dh[tpos[pt], pj] = herr @ aw2
        del w2, aw2, o_ref
    gk = gamma(k)
    yv = np.asarray(y)
    ygot = yv[tokens].astype(np.float64) if y_f32 else bf16_f64(yv[tokens])
    s64 = np.zeros((len(tokens), d))
    sabs = np.zeros((len(tokens), d))
    wdiff = np.zeros((len(tokens), d))
    down = np.zeros((len(tokens), d))
    for j in range(k):
        r = pair_row[tokens, j]
        loc = r >= 0
        if not loc.any():
            continue
        oj = np.zeros((len(tokens), d))
        oj[loc] = O[r[loc]]
        wj = np.where(loc, w32[tokens, j], 0.0)[:, None]
        s64 += wj * oj
        sabs += np.abs(wj * oj)
        wdiff += np.abs(wj - np.where(loc, w64[tokens, j], 0.0)[:, None]) * np.abs(oj)
        down += np.abs(np.where(loc, w64[tokens, j], 0.0))[:, None] * (gf * habs[:, j] + dh[:, j])
    half = 0.0 if y_f32 else 0.5 * bf16_step(np.maximum(np.abs(ygot), np.abs(s64)))
    cb = half + gk * sabs + 1e-30
    cerr = np.abs(ygot - s64)
    assert np.all(cerr <= cb), ("combine", float((cerr / cb).max()))
    none = ~(pair_row[tokens] >= 0).any(axis=1)
    assert np.all(ygot[none] == 0.0)
    yb = cb + wdiff + down
    yerr = np.abs(ygot - ref["y64"][tokens])
    assert np.all(yerr <= yb), ("y vs oracle", float((yerr / yb).max()))
    out = {"h_exact": float(np.mean(h_exact)) if h_exact else 1.0, "h_worst": h_worst,
           "o_worst": o_worst, "combine_worst": float((cerr / cb).max()),
           "y_worst": float((yerr / yb).max()), "rows": int(sum(len(v) for v in by_e.values())),
           "y_bound": yb}
    if not y_f32:
        out["y_bits_equal"] = float(np.mean(ordered(yv[tokens]) == ordered(ref["y16"][tokens])))
    return out
