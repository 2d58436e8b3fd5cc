"""TEST INFRASTRUCTURE ONLY: ctypes binding of the fp64 CPU oracles (the MoE
layer in moe_oracle.c, the self-attention block in attn_oracle.c).

Only the test-suite, the smoke check and the benchmark's CPU-baseline leg may
import this package.  The product library never loads it, and it never loads
the product library.  The arithmetic lives in ``moe_oracle.c``; this file only
marshals numpy arrays.

Layouts: x bf16 bits [T,d]; router fp32 [d,E]; bias fp32 [E] or None;
gate/up bf16 bits [d,f]; down bf16 bits [f,d]; y bf16 bits [T,d].
Weights are passed as a list of E arrays (None for experts the call never
uses).
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

from . import build as _build

_LIB = None

_p = ctypes.c_void_p
_i = ctypes.c_int


def lib():
    global _LIB
    if _LIB is None:
        path = _build.build(force=False)
        L = ctypes.CDLL(path)
        L.oracle_f64_from_bf16.argtypes = [ctypes.c_uint16]
        L.oracle_f64_from_bf16.restype = ctypes.c_double
        L.oracle_bf16_from_f64.argtypes = [ctypes.c_double]
        L.oracle_bf16_from_f64.restype = ctypes.c_uint16
        L.oracle_bf16_round_array.argtypes = [_p, _p, ctypes.c_int64]
        L.oracle_router_logits.argtypes = [_i, _i, _i, _p, _p, _p, _p]
        L.oracle_route_from_logits.argtypes = [_i, _i, _i, _p, _p, _p]
        L.oracle_permutation.argtypes = [_i, _i, _i, _i, _i, _p, _p, _p, _p, _p]
        L.oracle_expert_glu.argtypes = [_i, _i, _i, _p, _p, _p, _p, _p, _p]
        L.oracle_layer_with_routing.argtypes = [_i] * 7 + [_p] * 8
        L.oracle_layer_with_routing_ex.argtypes = [_i] * 7 + [_p] * 6 + [_i] + [_p] * 3
        L.oracle_layer.argtypes = [_i] * 7 + [_p] * 11
        L.oracle_layer_dense.argtypes = [_i] * 5 + [_p] * 7
        L.oracle_residual_add.argtypes = [_p, _p, _p, ctypes.c_int64]
        L.oracle_layernorm.argtypes = [_i, _i, _p, _p, ctypes.c_double, _p]
        L.oracle_rope.argtypes = [_i, _i, _p, _p, ctypes.c_double, _p]
        L.oracle_attention_core.argtypes = [_i] * 5 + [_p] * 5
        L.oracle_attention_block.argtypes = ([_i] * 6 + [_p, _p, ctypes.c_double, ctypes.c_double] +
                                             [_p] * 11)
        for fn in ("oracle_layernorm", "oracle_rope", "oracle_attention_core",
                   "oracle_attention_block"):
            getattr(L, fn).restype = ctypes.c_int
        for fn in ("oracle_router_logits", "oracle_route_from_logits", "oracle_permutation",
                   "oracle_expert_glu", "oracle_layer_with_routing",
                   "oracle_layer_with_routing_ex", "oracle_layer",
                   "oracle_layer_dense"):
            getattr(L, fn).restype = ctypes.c_int
        _LIB = L
    return _LIB


def _c(a, dtype):
    a = np.ascontiguousarray(a, dtype=dtype)
    return a, a.ctypes.data


def _check(rc, what):
    if rc != 0:
        raise ValueError(f"{what}: oracle rejected the arguments (rc={rc})")


def _ptr_array(arrs, E):
    keep = []
    ptrs = (ctypes.c_void_p * E)()
    for e in range(E):
        a = arrs[e] if e < len(arrs) else None
        if a is None:
            ptrs[e] = None
        else:
            a = np.ascontiguousarray(a, dtype=np.uint16)
            keep.append(a)
            ptrs[e] = a.ctypes.data
    return ptrs, keep


def f64_from_bf16(b: int) -> float:
    return lib().oracle_f64_from_bf16(int(b))


def bf16_from_f64(v: float) -> int:
    return int(lib().oracle_bf16_from_f64(float(v)))


def bf16_round(a) -> np.ndarray:
    a, pa = _c(a, np.float64)
    out = np.empty(a.shape, dtype=np.uint16)
    lib().oracle_bf16_round_array(pa, out.ctypes.data, a.size)
    return out


def router_logits(x, wr, bias=None) -> np.ndarray:
    x, px = _c(x, np.uint16)
    wr, pw = _c(wr, np.float32)
    T, d = x.shape
    E = wr.shape[1]
    assert wr.shape[0] == d
    pb = None
    if bias is not None:
        bias, pb = _c(bias, np.float32)
    out = np.empty((T, E), dtype=np.float32)
    _check(lib().oracle_router_logits(T, d, E, px, pw, pb, out.ctypes.data), "router_logits")
    return out


def route_from_logits(logits, k: int):
    logits, pl = _c(logits, np.float32)
    T, E = logits.shape
    idx = np.empty((T, k), dtype=np.int32)
    w = np.empty((T, k), dtype=np.float64)
    _check(lib().oracle_route_from_logits(T, E, k, pl, idx.ctypes.data, w.ctypes.data),
           "route_from_logits")
    return idx, w


def permutation(idx, E: int, e_begin: int = 0, n_local: int = 0):
    idx, pi = _c(idx, np.int32)
    T, k = idx.shape
    nl = n_local or E
    counts = np.empty(E, dtype=np.int32)
    offsets = np.empty(E + 1, dtype=np.int32)
    pair_row = np.empty((T, k), dtype=np.int32)
    row_token = np.full(max(T * k, 1), -1, dtype=np.int32)
    _check(lib().oracle_permutation(T, E, k, e_begin, nl, pi, counts.ctypes.data,
                                    offsets.ctypes.data, pair_row.ctypes.data,
                                    row_token.ctypes.data), "permutation")
    return counts, offsets, pair_row, row_token[: int(offsets[E])]


def expert_glu(xrows, gate, up, down):
    """Returns (hb bf16 bits [m,f], o fp64 [m,d]) for one expert."""
    xrows, px = _c(xrows, np.uint16)
    gate, pg = _c(gate, np.uint16)
    up, pu = _c(up, np.uint16)
    down, pd = _c(down, np.uint16)
    m, d = xrows.shape
    f = gate.shape[1]
    assert gate.shape == (d, f) and up.shape == (d, f) and down.shape == (f, d)
    hb = np.empty((m, f), dtype=np.uint16)
    o = np.empty((m, d), dtype=np.float64)
    _check(lib().oracle_expert_glu(m, d, f, px, pg, pu, pd, hb.ctypes.data, o.ctypes.data),
           "expert_glu")
    return hb, o


def layer_with_routing(x, idx, w, gates, ups, downs, e_begin: int = 0, n_local: int = 0):
    """Returns (y64 fp64 [T,d] before rounding, y bf16 bits [T,d])."""
    x, px = _c(x, np.uint16)
    idx, pi = _c(idx, np.int32)
    w, pw = _c(w, np.float64)
    T, d = x.shape
    k = idx.shape[1]
    E = len(gates)
    f = next(g for g in gates if g is not None).shape[1]
    nl = n_local or E
    pg, kg = _ptr_array(gates, E)
    pu, ku = _ptr_array(ups, E)
    pd, kd = _ptr_array(downs, E)
    y64 = np.empty((T, d), dtype=np.float64)
    y16 = np.empty((T, d), dtype=np.uint16)
    _check(lib().oracle_layer_with_routing(T, d, f, E, k, e_begin, nl, px, pi, pw, pg, pu, pd,
                                           y64.ctypes.data, y16.ctypes.data),
           "layer_with_routing")
    return y64, y16


def layer_with_routing_ex(x, idx, w, gates, ups, downs, e_begin: int = 0, n_local: int = 0,
                          round_h: bool = True, want_hb: bool = False):
    """layer_with_routing with the per-pair H and the exact form.

    Returns (y64, y16, hb): hb is bf16 bits [T, k, f] (pair (t, j)'s H when
    its expert is local, 0 otherwise) or None.  round_h=False is the
    information-only exact form: H is not rounded before the down
    projection, so y64 carries no intermediate rounding at all."""
    x, px = _c(x, np.uint16)
    idx, pi = _c(idx, np.int32)
    w, pw = _c(w, np.float64)
    T, d = x.shape
    k = idx.shape[1]
    E = len(gates)
    f = next(g for g in gates if g is not None).shape[1]
    nl = n_local or E
    pg, kg = _ptr_array(gates, E)
    pu, ku = _ptr_array(ups, E)
    pd, kd = _ptr_array(downs, E)
    y64 = np.empty((T, d), dtype=np.float64)
    y16 = np.empty((T, d), dtype=np.uint16)
    hb = np.zeros((T, k, f), dtype=np.uint16) if want_hb else None
    _check(lib().oracle_layer_with_routing_ex(T, d, f, E, k, e_begin, nl, px, pi, pw, pg, pu, pd,
                                              int(round_h), y64.ctypes.data, y16.ctypes.data,
                                              hb.ctypes.data if want_hb else None),
           "layer_with_routing_ex")
    return y64, y16, hb


def layer(x, wr, bias, gates, ups, downs, k: int, e_begin: int = 0, n_local: int = 0):
    """The whole layer.  Returns dict with logits, idx, w, y64, y."""
    x, px = _c(x, np.uint16)
    wr, pr = _c(wr, np.float32)
    pb = None
    if bias is not None:
        bias, pb = _c(bias, np.float32)
    T, d = x.shape
    E = wr.shape[1]
    f = next(g for g in gates if g is not None).shape[1]
    nl = n_local or E
    pg, kg = _ptr_array(gates, E)
    pu, ku = _ptr_array(ups, E)
    pd, kd = _ptr_array(downs, E)
    logits = np.empty((T, E), dtype=np.float32)
    idx = np.empty((T, k), dtype=np.int32)
    w = np.empty((T, k), dtype=np.float64)
    y64 = np.empty((T, d), dtype=np.float64)
    y16 = np.empty((T, d), dtype=np.uint16)
    _check(lib().oracle_layer(T, d, f, E, k, e_begin, nl, px, pr, pb, pg, pu, pd,
                              logits.ctypes.data, idx.ctypes.data, w.ctypes.data,
                              y64.ctypes.data, y16.ctypes.data), "layer")
    return {"logits": logits, "idx": idx, "w": w, "y64": y64, "y": y16}


def layer_dense(x, idx, w, gates, ups, downs):
    """Busy-full-loading form: all experts, unselected weights zero.  fp64 [T,d]."""
    x, px = _c(x, np.uint16)
    idx, pi = _c(idx, np.int32)
    w, pw = _c(w, np.float64)
    T, d = x.shape
    k = idx.shape[1]
    E = len(gates)
    f = gates[0].shape[1]
    pg, kg = _ptr_array(gates, E)
    pu, ku = _ptr_array(ups, E)
    pd, kd = _ptr_array(downs, E)
    y64 = np.empty((T, d), dtype=np.float64)
    _check(lib().oracle_layer_dense(T, d, f, E, k, px, pi, pw, pg, pu, pd, y64.ctypes.data),
           "layer_dense")
    return y64


def residual_add(x, y) -> np.ndarray:
    x, px = _c(x, np.uint16)
    y, py = _c(y, np.uint16)
    assert x.shape == y.shape
    out = np.empty(x.shape, dtype=np.uint16)
    lib().oracle_residual_add(px, py, out.ctypes.data, x.size)
    return out


# ------------------------------------------------------------ attention --
# Layouts: x bf16 [T, d]; gamma fp32 [d]; wqkv bf16 [d, (H + 2 G) hd];
# wo bf16 [H hd, d]; k/v caches bf16 [L, G, hd] (position-major), H query
# heads, G key/value heads.


def layernorm(x, gamma, eps: float) -> np.ndarray:
    x, px = _c(x, np.uint16)
    gamma, pg = _c(gamma, np.float32)
    T, d = x.shape
    h = np.empty((T, d), dtype=np.uint16)
    _check(lib().oracle_layernorm(T, d, px, pg, float(eps), h.ctypes.data), "layernorm")
    return h


def rope(v, pos, theta: float) -> np.ndarray:
    """Rotary encoding of head vectors v [n, hd] (fp64) at positions pos [n]."""
    v, pv = _c(v, np.float64)
    pos, pp = _c(pos, np.int32)
    n, hd = v.shape
    out = np.empty_like(v)
    _check(lib().oracle_rope(n, hd, pv, pp, float(theta), out.ctypes.data), "rope")
    return out


def attention_core(q, k_cache, v_cache, pos0: int):
    """Causal grouped-query attention of q [T, H, hd] (bf16 bits) over caches
    [L, G, hd] holding positions 0 .. pos0+T-1.  Returns (attn bf16
    [T, H*hd], attn64 fp64 [T, H*hd])."""
    q, pq = _c(q, np.uint16)
    k_cache, pk = _c(k_cache, np.uint16)
    v_cache, pv = _c(v_cache, np.uint16)
    T, H, hd = q.shape
    G = k_cache.shape[1]
    assert k_cache.shape[0] >= pos0 + T and v_cache.shape == k_cache.shape
    out = np.empty((T, H * hd), dtype=np.uint16)
    out64 = np.empty((T, H * hd), dtype=np.float64)
    _check(lib().oracle_attention_core(T, H, G, hd, pos0, pq, pk, pv, out.ctypes.data,
                                       out64.ctypes.data), "attention_core")
    return out, out64


def attention_block(x, gamma, wqkv, wo, k_cache, v_cache, pos0: int, n_heads: int, n_kv: int,
                    eps: float, theta: float):
    """The block on x [T, d] at positions pos0 ..; k_cache / v_cache
    [L, G, hd] bf16 bits are updated in place (positions pos0 .. pos0+T-1).
    Returns a dict of h, qkv64, q, attn, o64, y64, y (see attn_oracle.c)."""
    x, px = _c(x, np.uint16)
    gamma, pg = _c(gamma, np.float32)
    wqkv, pq = _c(wqkv, np.uint16)
    wo, pw = _c(wo, np.uint16)
    assert k_cache.dtype == np.uint16 and v_cache.dtype == np.uint16
    assert k_cache.flags.c_contiguous and v_cache.flags.c_contiguous
    T, d = x.shape
    hd = wo.shape[0] // n_heads
    nqkv = (n_heads + 2 * n_kv) * hd
    assert wqkv.shape == (d, nqkv) and wo.shape == (n_heads * hd, d)
    assert k_cache.shape[1:] == (n_kv, hd) and k_cache.shape[0] >= pos0 + T
    out = {"h": np.empty((T, d), np.uint16), "qkv64": np.empty((T, nqkv), np.float64),
           "q": np.empty((T, n_heads * hd), np.uint16), "attn": np.empty((T, n_heads * hd), np.uint16),
           "o64": np.empty((T, d), np.float64), "y64": np.empty((T, d), np.float64),
           "y": np.empty((T, d), np.uint16)}
    _check(lib().oracle_attention_block(
        T, d, n_heads, n_kv, hd, pos0, px, pg, float(eps), float(theta), pq, pw,
        k_cache.ctypes.data, v_cache.ctypes.data, out["h"].ctypes.data, out["qkv64"].ctypes.data,
        out["q"].ctypes.data, out["attn"].ctypes.data, out["o64"].ctypes.data,
        out["y64"].ctypes.data, out["y"].ctypes.data), "attention_block")
    return out
