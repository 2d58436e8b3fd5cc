"""Pins of the fp64 attention-block oracle (oracle/attn_oracle.c) against what
mathematics and library routines fix, independent of the oracle itself:

- layer norm: torch.nn.functional.layer_norm in fp64, and closed forms;
- rotary encoding: closed forms for head widths 2 and 4 (which fix the
  "rotate half" pairing and the frequency schedule), norm preservation,
  position 0 as identity, and the relative-position property;
- attention: torch's scaled_dot_product_attention in fp64 (grouped-query,
  with an explicit causal mask that puts token t at position pos0 + t),
  uniform weights for equal keys, the key/value head each query head uses,
  and a dominant key;
- the block: causality (a later token never changes an earlier one), T tokens
  at once equal T single-token steps, zero input, and agreement with a
  composition of library routines (torch layer_norm and SDPA, numpy matmul,
  the pinned rotary encoding).

The paper fixes only the widths (Table tab:vars) and that the block is
replicated per node; the head split, norm, rotary encoding and rounding
points are readings (A1..A8 in attn_oracle.c), so agreement with DBRX's own
numerics is parity unpinned."""
import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import moe_inputs as mi
import oracle


def f64(b):
    return mi.bf16_bits_to_f32(np.asarray(b, np.uint16)).astype(np.float64)


TINY = mi.ATTN_WORKLOADS["attn_tiny"]


# ------------------------------------------------------------- layer norm --

def test_layernorm_vs_torch():
    x = mi.gen_bf16(1, mi.stream_id(mi.KIND_ATTN_X), (7, 384), 2.0)
    g = TINY.with_(d=384).gamma()
    h = oracle.layernorm(x, g, 1e-5)
    ref = F.layer_norm(torch.from_numpy(f64(x)), (384,), weight=torch.from_numpy(g.astype(np.float64)),
                       bias=None, eps=1e-5).numpy()
    want = oracle.bf16_round(ref)
    # the same fp64 value rounded once: equal except where the two fp64
    # evaluations straddle a bf16 midpoint
    assert np.mean(want == h) > 0.999
    assert np.all(np.abs(f64(h) - ref) <= np.spacing(np.abs(ref).astype(np.float32)) * 65536)


def test_layernorm_closed_forms():
    d = 64
    x = np.full((1, d), 0x4040, np.uint16)          # constant 3.0 -> zero after centring
    g = np.full(d, 2.5, np.float32)
    assert np.all((oracle.layernorm(x, g, 1e-5) & 0x7FFF) == 0)
    alt = np.where(np.arange(d) % 2 == 0, 0x4000, 0xC000).astype(np.uint16)[None, :]   # +-2
    h = f64(oracle.layernorm(alt, g, 0.0))          # mean 0, var 4: exactly +-1 * gamma
    assert np.array_equal(h[0], np.where(np.arange(d) % 2 == 0, 2.5, -2.5))


# ---------------------------------------------------------------- rotary --

def test_rope_closed_forms_fix_pairing_and_frequencies():
    theta = 100.0
    p = np.array([3], np.int32)
    out = oracle.rope(np.array([[1.0, 0.0]]), p, theta)
    assert np.allclose(out, [[math.cos(3), math.sin(3)]], atol=1e-15)
    # width 4: component i pairs with i + 2 (rotate half), frequencies
    # theta^0 and theta^(-1/2)
    w = theta ** -0.5
    e0 = oracle.rope(np.array([[1.0, 0.0, 0.0, 0.0]]), p, theta)
    e1 = oracle.rope(np.array([[0.0, 1.0, 0.0, 0.0]]), p, theta)
    e2 = oracle.rope(np.array([[0.0, 0.0, 1.0, 0.0]]), p, theta)
    assert np.allclose(e0, [[math.cos(3), 0, math.sin(3), 0]], atol=1e-15)
    assert np.allclose(e1, [[0, math.cos(3 * w), 0, math.sin(3 * w)]], atol=1e-15)
    assert np.allclose(e2, [[-math.sin(3), 0, math.cos(3), 0]], atol=1e-15)


def test_rope_identity_norm_and_relative_position():
    rng = np.random.default_rng(0)
    hd, theta = 128, 5e5
    q = rng.standard_normal((5, hd))
    k = rng.standard_normal((5, hd))
    assert np.array_equal(oracle.rope(q, np.zeros(5, np.int32), theta), q)
    pos = np.array([0, 7, 100, 2047, 4000], np.int32)
    rq = oracle.rope(q, pos, theta)
    assert np.allclose(np.linalg.norm(rq, axis=1), np.linalg.norm(q, axis=1), rtol=1e-13)
    # <R(m) q, R(n) k> depends on m - n only
    for m, n in ((5, 2), (300, 17), (2047, 0)):
        base = np.sum(oracle.rope(q, np.full(5, m, np.int32), theta) *
                      oracle.rope(k, np.full(5, n, np.int32), theta), axis=1)
        for s in (1, 64, 999):
            sh = np.sum(oracle.rope(q, np.full(5, m + s, np.int32), theta) *
                        oracle.rope(k, np.full(5, n + s, np.int32), theta), axis=1)
            assert np.allclose(sh, base, rtol=1e-9, atol=1e-9)


# ------------------------------------------------------------- attention --

def _sdpa(q, kc, vc, pos0):
    """torch fp64 scaled_dot_product_attention, grouped-query, with token t
    of q at position pos0 + t (explicit mask)."""
    T, H, hd = q.shape
    L = pos0 + T
    qt = torch.from_numpy(f64(q)).permute(1, 0, 2)[None]            # [1, H, T, hd]
    kt = torch.from_numpy(f64(kc[:L])).permute(1, 0, 2)[None]       # [1, G, L, hd]
    vt = torch.from_numpy(f64(vc[:L])).permute(1, 0, 2)[None]
    mask = torch.arange(L)[None, :] <= (pos0 + torch.arange(T))[:, None]
    out = F.scaled_dot_product_attention(qt, kt, vt, attn_mask=mask, enable_gqa=True)
    return out[0].permute(1, 0, 2).reshape(T, H * hd).numpy()


@pytest.mark.parametrize("T,pos0,H,G,hd", [(1, 0, 4, 2, 16), (3, 10, 6, 2, 32), (5, 40, 8, 8, 64),
                                           (2, 100, 48, 8, 128)])
def test_attention_core_vs_torch_sdpa(T, pos0, H, G, hd):
    rng = np.random.default_rng(T + pos0)
    q = oracle.bf16_round(rng.standard_normal((T, H, hd)) * 1.5)
    kc = oracle.bf16_round(rng.standard_normal((pos0 + T, G, hd)) * 1.5)
    vc = oracle.bf16_round(rng.standard_normal((pos0 + T, G, hd)))
    out, out64 = oracle.attention_core(q, kc, vc, pos0)
    ref = _sdpa(q, kc, vc, pos0)
    assert np.allclose(out64, ref, rtol=1e-12, atol=1e-12)
    assert np.array_equal(out, oracle.bf16_round(out64))


def test_attention_equal_keys_average_values():
    T, pos0, H, G, hd = 2, 9, 4, 2, 8
    rng = np.random.default_rng(3)
    q = oracle.bf16_round(rng.standard_normal((T, H, hd)))
    kc = np.tile(oracle.bf16_round(rng.standard_normal((1, G, hd))), (pos0 + T, 1, 1))
    vc = oracle.bf16_round(rng.standard_normal((pos0 + T, G, hd)))
    _, out64 = oracle.attention_core(q, kc, vc, pos0)
    for t in range(T):
        mean = f64(vc[: pos0 + t + 1]).mean(axis=0)            # [G, hd]
        for j in range(H):
            assert np.allclose(out64[t, j * hd:(j + 1) * hd], mean[j // (H // G)], rtol=1e-13)


def test_attention_query_head_uses_its_group():
    T, pos0, H, G, hd = 1, 5, 6, 3, 4
    q = oracle.bf16_round(np.random.default_rng(1).standard_normal((T, H, hd)))
    kc = oracle.bf16_round(np.random.default_rng(2).standard_normal((pos0 + T, G, hd)))
    vc = np.zeros((pos0 + T, G, hd), np.uint16)
    for g in range(G):
        vc[:, g, :] = oracle.bf16_round(np.array([g + 1.0]))[0]
    _, out64 = oracle.attention_core(q, kc, vc, pos0)
    for j in range(H):
        assert np.allclose(out64[0, j * hd:(j + 1) * hd], j // 2 + 1.0, rtol=1e-14)


def test_attention_dominant_key_selects_its_value():
    T, pos0, H, G, hd = 1, 20, 2, 1, 16
    q = np.zeros((T, H, hd), np.uint16)
    q[0, :, 0] = oracle.bf16_round(np.array([8.0]))[0]
    kc = np.zeros((pos0 + T, G, hd), np.uint16)
    kc[13, 0, 0] = oracle.bf16_round(np.array([16.0]))[0]     # score 128 / 4 = 32 vs 0
    vc = oracle.bf16_round(np.random.default_rng(4).standard_normal((pos0 + T, G, hd)))
    _, out64 = oracle.attention_core(q, kc, vc, pos0)
    assert np.allclose(out64[0, :hd], f64(vc[13, 0]), rtol=1e-12, atol=1e-12)


# ----------------------------------------------------------------- block --

def _block(wl, x=None, T=None, pos0=None, caches=None):
    T = wl.T if T is None else T
    pos0 = wl.pos0 if pos0 is None else pos0
    wl = wl.with_(T=T, pos0=pos0)
    if caches is None:
        k0, v0 = wl.cache_prefix()
        kc = np.zeros((wl.max_seq, wl.n_kv, wl.hd), np.uint16)
        vc = np.zeros_like(kc)
        kc[:pos0], vc[:pos0] = k0, v0
    else:
        kc, vc = caches
    x = wl.x() if x is None else x
    r = oracle.attention_block(x, wl.gamma(), wl.wqkv(), wl.wo(), kc, vc, pos0, wl.n_heads,
                               wl.n_kv, wl.eps, wl.theta)
    return r, kc, vc


def test_block_tokens_at_once_equal_single_steps_and_are_causal():
    wl = TINY
    r, kc, vc = _block(wl)
    # the same tokens one at a time, each appending to the cache
    k0, v0 = wl.cache_prefix()
    kc2 = np.zeros_like(kc)
    vc2 = np.zeros_like(vc)
    kc2[:wl.pos0], vc2[:wl.pos0] = k0, v0
    x = wl.x()
    for t in range(wl.T):
        rt, _, _ = _block(wl, x=x[t:t + 1], T=1, pos0=wl.pos0 + t, caches=(kc2, vc2))
        assert np.array_equal(rt["y"][0], r["y"][t])
        assert np.array_equal(rt["attn"][0], r["attn"][t])
    assert np.array_equal(kc, kc2) and np.array_equal(vc, vc2)
    # a later token's input does not change an earlier token's output
    x3 = x.copy()
    x3[-1] ^= 0x0040
    r3, _, _ = _block(wl, x=x3)
    assert np.array_equal(r3["y"][:-1], r["y"][:-1]) and not np.array_equal(r3["y"][-1], r["y"][-1])


def test_block_zero_input():
    """x = 0: the norm gives 0, so q, k, v of the new token are 0, every
    score is 0 and each head averages the cached values with the new zero
    value; y = o = that average times wo."""
    wl = TINY.with_(T=1)
    x = np.zeros((1, wl.d), np.uint16)
    r, kc, vc = _block(wl, x=x)
    assert np.all((r["h"] & 0x7FFF) == 0) and np.all(r["qkv64"] == 0.0)
    L = wl.pos0 + 1
    mean = f64(vc[:L]).sum(axis=0) / L                        # [G, hd]
    group = wl.n_heads // wl.n_kv
    att = np.concatenate([mean[j // group] for j in range(wl.n_heads)])
    # one rounding of the average (summing a/L * v or v then / L may differ
    # in the last fp64 bits, so a midpoint may round either way)
    step = np.spacing(np.abs(att).astype(np.float32)).astype(np.float64) * 65536
    assert np.all(np.abs(f64(r["attn"][0]) - att) <= 0.5 * step * (1 + 1e-9))
    assert np.mean(r["attn"][0] == oracle.bf16_round(att)) > 0.95
    o = f64(r["attn"][0]) @ f64(wl.wo())
    assert np.allclose(r["o64"][0], o, rtol=1e-12, atol=1e-14)
    assert np.array_equal(r["y64"], r["o64"])


@pytest.mark.parametrize("wl", [TINY, TINY.with_(T=3, pos0=0, n_heads=6, n_kv=3, hd=32, d=192)])
def test_block_vs_library_composition(wl):
    """layer_norm (torch, fp64) -> bf16 -> numpy fp64 projection -> the pinned
    rotary encoding -> bf16 -> SDPA (torch, fp64, grouped, causal by position)
    -> bf16 -> numpy fp64 output projection -> + x.  Intermediate bf16 values
    may flip by one step where the two fp64 evaluations straddle a midpoint,
    so the comparison is tight but not bitwise."""
    r, kc, vc = _block(wl)
    x, g = wl.x(), wl.gamma()
    h = oracle.bf16_round(F.layer_norm(torch.from_numpy(f64(x)), (wl.d,),
                                       weight=torch.from_numpy(g.astype(np.float64)), eps=wl.eps).numpy())
    assert np.mean(h == r["h"]) > 0.995
    proj = f64(r["h"]) @ f64(wl.wqkv())
    assert np.allclose(proj, r["qkv64"], rtol=1e-12, atol=1e-12)
    H, G, hd, T = wl.n_heads, wl.n_kv, wl.hd, wl.T
    pos = np.repeat(np.arange(wl.pos0, wl.pos0 + T, dtype=np.int32), H)
    q = oracle.bf16_round(oracle.rope(proj[:, :H * hd].reshape(T * H, hd), pos, wl.theta))
    assert np.array_equal(q.reshape(T, H * hd), r["q"])
    posk = np.repeat(np.arange(wl.pos0, wl.pos0 + T, dtype=np.int32), G)
    k = oracle.bf16_round(oracle.rope(proj[:, H * hd:(H + G) * hd].reshape(T * G, hd), posk, wl.theta))
    assert np.array_equal(k.reshape(T, G, hd), kc[wl.pos0:wl.pos0 + T])
    v = oracle.bf16_round(proj[:, (H + G) * hd:])
    assert np.array_equal(v.reshape(T, G, hd), vc[wl.pos0:wl.pos0 + T])
    att = _sdpa(q.reshape(T, H, hd), kc, vc, wl.pos0)
    assert np.mean(oracle.bf16_round(att) == r["attn"]) > 0.995
    y = f64(x) + f64(r["attn"]) @ f64(wl.wo())
    assert np.allclose(r["y64"], y, rtol=1e-12, atol=1e-12)
    assert np.array_equal(r["y"], oracle.bf16_round(r["y64"]))
