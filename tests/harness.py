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


def make_layer(wl: mi.Workload, max_tokens=None, e_begin=None, n_local=None, n_layers=None):
    import paper_2506_23635_amd as moe
    cfg = moe.make_config(wl.d, wl.f, wl.E, wl.k,
                          expert_begin=wl.e_begin if e_begin is None else e_begin,
                          n_local_experts=(wl.local if n_local is None else n_local),
                          n_layers=wl.n_layers if n_layers is None else n_layers,
                          max_tokens=max_tokens or wl.T)
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
