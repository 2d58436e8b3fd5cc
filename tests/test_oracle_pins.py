"""Pins of the fp64 CPU oracle against what the paper and mathematics fix:
library routines, brute force, closed forms, invariants and special cases.
None of these use the GPU library."""
import itertools
import math
import os
from fractions import Fraction

import numpy as np
import pytest
import scipy.special
import torch

import moe_inputs as mi
import oracle

# ------------------------------------------------------------------ bf16 ----


def test_bf16_from_f64_matches_torch_on_fp32_patterns():
    """For every fp32 high half and a set of low halves that contains the
    rounding edges (0, 1, just below/at/above the tie, all ones), the oracle's
    double->bf16 equals torch's fp32->bf16 round-to-nearest-even."""
    hi = np.arange(1 << 16, dtype=np.uint32) << 16
    lows = np.array([0x0000, 0x0001, 0x3FFF, 0x7FFF, 0x8000, 0x8001, 0xC000, 0xFFFF] +
                    list(np.random.default_rng(0).integers(0, 1 << 16, 24)), dtype=np.uint32)
    bits = (hi[:, None] | lows[None, :]).reshape(-1)
    f = bits.view(np.float32)
    finite = np.isfinite(f)
    want = torch.from_numpy(f.copy()).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    with np.errstate(invalid="ignore"):
        got = oracle.bf16_round(f.astype(np.float64))
    assert np.array_equal(got[finite], want[finite])
    nan = np.isnan(f)
    gotf = mi.bf16_bits_to_f32(got[nan])
    assert np.all(np.isnan(gotf))


def _nearest_even_bf16(v):
    x = Fraction(v)
    b0 = int(np.array([v], np.float32).view(np.uint32)[0] >> 16)
    best = None
    for b in range(max(0, b0 - 2), min(0xFFFF, b0 + 2) + 1):
        if (b & 0x7F80) == 0x7F80:
            continue
        val = Fraction(float(mi.bf16_bits_to_f32(np.array([b], np.uint16))[0]))
        key = (abs(val - x), b & 1)
        if best is None or key < best[0]:
            best = (key, b)
    return best[1]


def test_bf16_from_f64_brute_force_near_ties():
    rng = np.random.default_rng(5)
    vals = []
    for v in np.concatenate([rng.standard_normal(200), rng.standard_normal(50) * 1e-38,
                             rng.standard_normal(50) * 1e30]):
        b = int(np.array([abs(v)], np.float32).view(np.uint32)[0] >> 16)
        lo = float(mi.bf16_bits_to_f32(np.array([b], np.uint16))[0])
        hi = float(mi.bf16_bits_to_f32(np.array([b + 1], np.uint16))[0])
        mid = (lo + hi) / 2
        vals += [mid, math.nextafter(mid, math.inf), math.nextafter(mid, -math.inf)]
    for v in vals:
        assert oracle.bf16_from_f64(v) == _nearest_even_bf16(v), v


def test_bf16_special_values():
    assert oracle.bf16_from_f64(0.0) == 0x0000
    assert oracle.bf16_from_f64(-0.0) == 0x8000
    assert oracle.bf16_from_f64(math.inf) == 0x7F80
    assert oracle.bf16_from_f64(-math.inf) == 0xFF80
    assert oracle.bf16_from_f64(1e39) == 0x7F80          # beyond the bf16 range
    assert oracle.bf16_from_f64(2.0 ** -134) == 0x0000     # half the smallest subnormal: even
    assert oracle.bf16_from_f64(2.0 ** -134 * 1.5) == 0x0001
    assert oracle.bf16_from_f64(1.0) == 0x3F80
    assert oracle.bf16_from_f64(1.0 + 2 ** -8) == 0x3F80   # tie, even stays
    assert oracle.bf16_from_f64(1.0 + 3 * 2 ** -8) == 0x3F82  # tie, odd goes up


def test_bf16_two_independent_roundings_agree():
    """The generator's integer rounding and the oracle's rint-based one are
    written independently; they must agree on arbitrary doubles."""
    rng = np.random.default_rng(9)
    v = np.concatenate([rng.standard_normal(5000) * s for s in (1e-40, 1e-3, 1.0, 1e5, 1e37)])
    got = oracle.bf16_round(v)
    for i in range(0, v.size, 7):
        assert got[i] == mi.bf16_rne(float(v[i]))

# ---------------------------------------------------------------- router ----


def test_logits_one_hot_router_picks_x_entries():
    T, d, E = 5, 64, 8
    x = mi.gen_bf16(0, mi.stream_id(mi.KIND_X), (T, d), 1.0)
    pos = [3, 60, 0, 17, 17, 42, 9, 63]
    wr = np.zeros((d, E), np.float32)
    for e, p in enumerate(pos):
        wr[p, e] = 1.0
    lg = oracle.router_logits(x, wr)
    xf = mi.bf16_bits_to_f32(x)
    for e, p in enumerate(pos):
        assert np.array_equal(lg[:, e], xf[:, p])


def test_logits_vs_numpy_matmul():
    T, d, E = 16, 256, 8
    x = mi.gen_bf16(0, mi.stream_id(mi.KIND_X), (T, d), 1.0)
    wr = mi.gen_f32(0, mi.stream_id(mi.KIND_ROUTER), (d, E), 0.02)
    lg = oracle.router_logits(x, wr)
    ref = (mi.bf16_bits_to_f32(x).astype(np.float64) @ wr.astype(np.float64)).astype(np.float32)
    ulp = np.spacing(np.abs(ref))
    assert np.all(np.abs(lg - ref) <= ulp)
    assert np.mean(lg == ref) > 0.95


def test_logits_bias_added_in_fp32_after_rounding():
    T, d, E = 8, 128, 16
    x = mi.gen_bf16(2, mi.stream_id(mi.KIND_X), (T, d), 1.0)
    wr = mi.gen_f32(2, mi.stream_id(mi.KIND_ROUTER), (d, E), 0.02)
    b = mi.gen_f32(2, mi.stream_id(mi.KIND_BIAS), (E,), 1.0)
    l0 = oracle.router_logits(x, wr)
    l1 = oracle.router_logits(x, wr, b)
    assert np.array_equal(l1, (l0 + b[None, :]).astype(np.float32))

# ------------------------------------------------------------ selection -----


def _brute_topk(l, k):
    """Subset with the largest exact sum; among equal sums the one whose
    sorted ids are lexicographically smallest.  Slot order: logit desc, id asc."""
    E = len(l)
    best = None
    for s in itertools.combinations(range(E), k):
        tot = sum(Fraction(float(l[e])) for e in s)
        key = (-tot, s)
        if best is None or key < best[0]:
            best = (key, s)
    s = best[1]
    return sorted(s, key=lambda e: (-Fraction(float(l[e])), e))


@pytest.mark.parametrize("E,k", [(8, 2), (16, 4), (6, 6), (5, 1)])
def test_topk_brute_force_continuous(E, k):
    rng = np.random.default_rng(E * 100 + k)
    lg = rng.standard_normal((40, E)).astype(np.float32)
    idx, w = oracle.route_from_logits(lg, k)
    for t in range(lg.shape[0]):
        assert list(idx[t]) == _brute_topk(lg[t], k)


@pytest.mark.parametrize("E,k", [(8, 2), (16, 4), (7, 3)])
def test_topk_brute_force_with_ties(E, k):
    rng = np.random.default_rng(E + k)
    lg = rng.integers(-2, 3, size=(60, E)).astype(np.float32)   # many ties
    idx, _ = oracle.route_from_logits(lg, k)
    for t in range(lg.shape[0]):
        assert list(idx[t]) == _brute_topk(lg[t], k)


def test_topk_invariants_dbrx_width():
    E, k = 16, 4
    lg = mi.gen_f32(4, mi.stream_id(mi.KIND_ROUTER), (500, E), 1.0)
    idx, w = oracle.route_from_logits(lg, k)
    for t in range(500):
        s = set(idx[t].tolist())
        assert len(s) == k
        sel_min = min(lg[t, e] for e in s)
        assert all(lg[t, e] <= sel_min for e in range(E) if e not in s)
        assert all(lg[t, idx[t, j]] >= lg[t, idx[t, j + 1]] for j in range(k - 1))
    assert np.allclose(w.sum(1), 1.0, rtol=0, atol=1e-15)


def test_topk_signed_zero_and_constructed_ties():
    lg = np.array([[-0.0, 0.0, -1.0, -1.0],
                   [0.5, 0.5, 0.5, 0.5],
                   [-1.0, 2.0, 2.0, -3.0]], np.float32)
    idx, w = oracle.route_from_logits(lg, 2)
    assert idx.tolist() == [[0, 1], [0, 1], [1, 2]]
    assert np.allclose(w, 0.5, rtol=0, atol=1e-16)


def test_topk_rejects_non_finite():
    with pytest.raises(ValueError):
        oracle.route_from_logits(np.array([[0.0, np.nan, 1.0]], np.float32), 1)
    with pytest.raises(ValueError):
        oracle.route_from_logits(np.array([[0.0, np.inf, 1.0]], np.float32), 1)


def test_weights_closed_forms():
    # equal selected logits -> 1/k
    idx, w = oracle.route_from_logits(np.array([[1.0, 1.0, 1.0, 1.0, -5.0]], np.float32), 4)
    assert np.allclose(w, 0.25, rtol=0, atol=1e-16)
    # two selected logits that differ by ln 3 -> 3/4 and 1/4
    a = np.float32(0.25)
    b = np.float32(float(a) - math.log(3.0))
    idx, w = oracle.route_from_logits(np.array([[b, -9.0, a]], np.float32), 2)
    assert idx.tolist() == [[2, 0]]
    gap = float(a) - float(b)   # the fp32 gap, close to ln 3
    assert abs(w[0, 0] - 1.0 / (1.0 + math.exp(-gap))) < 1e-15
    assert abs(w[0, 0] - 0.75) < 1e-7 and abs(w[0, 1] - 0.25) < 1e-7


def test_weights_vs_scipy_softmax_and_renormalised_full_softmax():
    E, k = 16, 4
    lg = mi.gen_f32(8, mi.stream_id(mi.KIND_ROUTER), (200, E), 1.5)
    idx, w = oracle.route_from_logits(lg, k)
    sel = np.take_along_axis(lg.astype(np.float64), idx, axis=1)
    assert np.allclose(w, scipy.special.softmax(sel, axis=1), rtol=1e-14, atol=0)
    full = scipy.special.softmax(lg.astype(np.float64), axis=1)
    psel = np.take_along_axis(full, idx, axis=1)
    assert np.allclose(w, psel / psel.sum(1, keepdims=True), rtol=1e-13, atol=0)

# ---------------------------------------------------------- permutation -----


@pytest.mark.parametrize("T,E,k,e0,nl", [(16, 8, 2, 0, 8), (33, 16, 4, 4, 4), (1, 16, 4, 12, 4),
                                         (64, 16, 4, 0, 16), (0, 8, 2, 0, 8)])
def test_permutation_vs_stable_sort(T, E, k, e0, nl):
    rng = np.random.default_rng(T + E)
    idx = np.array([rng.permutation(E)[:k] for _ in range(T)], np.int32).reshape(T, k)
    counts, offsets, pair_row, row_token = oracle.permutation(idx, E, e0, nl)
    flat_e = idx.reshape(-1)
    flat_t = np.repeat(np.arange(T), k)
    local = (flat_e >= e0) & (flat_e < e0 + nl)
    order = np.argsort(flat_e[local], kind="stable")      # numpy stable sort
    want_tokens = flat_t[local][order]
    assert np.array_equal(row_token, want_tokens)
    assert np.array_equal(counts, np.bincount(flat_e[local], minlength=E))
    assert offsets[0] == 0 and np.array_equal(np.diff(offsets), counts)
    # pair_row is a bijection onto the rows, -1 exactly off the share
    pr = pair_row.reshape(-1)
    assert np.all((pr == -1) == ~local)
    assert sorted(pr[local].tolist()) == list(range(int(local.sum())))
    # unpermute(permute(pairs)) is the identity on (token, expert)
    for p in np.nonzero(local)[0]:
        r = pr[p]
        assert row_token[r] == flat_t[p]
        assert offsets[flat_e[p]] <= r < offsets[flat_e[p] + 1]

# ------------------------------------------------------------ expert GLU ----


def _rand_expert(seed, d, f, e=0, sigma=0.05):
    return (mi.gen_bf16(seed, mi.stream_id(mi.KIND_GATE, 0, e), (d, f), sigma),
            mi.gen_bf16(seed, mi.stream_id(mi.KIND_UP, 0, e), (d, f), sigma),
            mi.gen_bf16(seed, mi.stream_id(mi.KIND_DOWN, 0, e), (f, d), sigma))


def _f64(b):
    return mi.bf16_bits_to_f32(b).astype(np.float64)


def test_expert_glu_vs_numpy_swiglu():
    """SwiGLU with library matmul and scipy's logistic sigmoid; w1 is the gate,
    v1 the up projection, w2 the down projection (shapes d x f, d x f, f x d)."""
    m, d, f = 6, 96, 160
    x = mi.gen_bf16(1, mi.stream_id(mi.KIND_X), (m, d), 1.0)
    g_w, u_w, d_w = _rand_expert(1, d, f, sigma=0.2)
    hb, o = oracle.expert_glu(x, g_w, u_w, d_w)
    g = _f64(x) @ _f64(g_w)
    u = _f64(x) @ _f64(u_w)
    h = g * scipy.special.expit(g) * u
    h_t = torch.from_numpy(h).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    # torch narrows double via float (two roundings); disagreements are at
    # most one bf16 step and only where h sits next to a bf16 midpoint
    diff = hb != h_t
    assert diff.mean() < 0.002
    assert np.all(np.abs(hb[diff].astype(np.int32) - h_t[diff].astype(np.int32)) == 1)
    assert np.allclose(_f64(hb), h, rtol=2 ** -8, atol=1e-30)
    assert np.allclose(o, _f64(hb) @ _f64(d_w), rtol=1e-12, atol=1e-12)


def test_expert_glu_swapped_roles_differ():
    m, d, f = 2, 32, 48
    x = mi.gen_bf16(3, mi.stream_id(mi.KIND_X), (m, d), 1.0)
    g_w, u_w, d_w = _rand_expert(3, d, f, sigma=0.3)
    _, o1 = oracle.expert_glu(x, g_w, u_w, d_w)
    _, o2 = oracle.expert_glu(x, u_w, g_w, d_w)
    assert not np.allclose(o1, o2)


def test_expert_glu_zero_and_one_hot_input():
    d, f = 40, 24
    g_w, u_w, d_w = _rand_expert(4, d, f, sigma=1.0)
    hb, o = oracle.expert_glu(np.zeros((1, d), np.uint16), g_w, u_w, d_w)
    assert np.all(o == 0.0) and np.all((hb & 0x7FFF) == 0)
    i = 13
    xh = np.zeros((1, d), np.uint16)
    xh[0, i] = 0x3F80                                   # x = e_i
    hb, o = oracle.expert_glu(xh, g_w, u_w, d_w)
    g = _f64(g_w[i])
    u = _f64(u_w[i])
    want = g / (1.0 + np.exp(-g)) * u                  # silu(w1[i,:]) * v1[i,:]
    assert np.allclose(_f64(hb[0]), want, rtol=2 ** -8, atol=0)
    assert np.allclose(o[0], _f64(hb[0]) @ _f64(d_w), rtol=1e-13, atol=1e-13)


def test_expert_glu_overflow_safe_silu():
    d, f = 4, 3
    g_w = np.full((d, f), 0x4300, np.uint16)   # 128.0
    g_w[:, 1] = 0xC300                         # -128.0
    u_w = np.full((d, f), 0x3F80, np.uint16)   # 1.0
    d_w = np.full((f, d), 0x3F80, np.uint16)
    x = np.full((1, d), 0x4000, np.uint16)     # 2.0 -> g = +-1024, u = 8
    hb, o = oracle.expert_glu(x, g_w, u_w, d_w)
    h = _f64(hb[0])
    assert h[0] == 8192.0 and h[2] == 8192.0    # silu(1024) * 8
    assert h[1] == 0.0                          # silu(-1024) underflows to -0
    assert np.all(np.isfinite(o))

# ----------------------------------------------------------------- layer ----


def _tiny_inputs(T=16, d=64, f=96, E=8, seed=0, sigma_w=0.05):
    x = mi.gen_bf16(seed, mi.stream_id(mi.KIND_X), (T, d), 1.0)
    wr = mi.gen_f32(seed, mi.stream_id(mi.KIND_ROUTER), (d, E), 0.2)
    ex = [_rand_expert(seed, d, f, e, sigma_w) for e in range(E)]
    return x, wr, [a for a, _, _ in ex], [b for _, b, _ in ex], [c for _, _, c in ex]


def test_layer_single_expert_is_plain_swiglu_ffn():
    T, d, f = 5, 48, 80
    x = mi.gen_bf16(6, mi.stream_id(mi.KIND_X), (T, d), 1.0)
    wr = mi.gen_f32(6, mi.stream_id(mi.KIND_ROUTER), (d, 1), 0.2)
    g_w, u_w, d_w = _rand_expert(6, d, f, sigma=0.1)
    r = oracle.layer(x, wr, None, [g_w], [u_w], [d_w], k=1)
    assert np.all(r["idx"] == 0) and np.all(r["w"] == 1.0)
    hb, o = oracle.expert_glu(x, g_w, u_w, d_w)
    assert np.array_equal(r["y64"], o)
    g = _f64(x) @ _f64(g_w)
    u = _f64(x) @ _f64(u_w)
    h = g * scipy.special.expit(g) * u
    ref = h @ _f64(d_w)                  # no H rounding: within the bf16 step of H
    rel = np.linalg.norm(r["y64"] - ref) / np.linalg.norm(ref)
    assert rel < 4e-3
    assert np.array_equal(r["y"], oracle.bf16_round(r["y64"]))


def test_layer_exact_form_single_expert_is_unrounded_swiglu():
    """The information-only exact form (no H rounding) of E = 1, k = 1 is the
    textbook SwiGLU FFN in fp64 (library matmul, scipy's logistic) to
    rounding; the per-pair H it returns is the rounded form's hb."""
    T, d, f = 5, 48, 80
    x = mi.gen_bf16(6, mi.stream_id(mi.KIND_X), (T, d), 1.0)
    g_w, u_w, d_w = _rand_expert(6, d, f, sigma=0.1)
    idx = np.zeros((T, 1), np.int32)
    w = np.ones((T, 1))
    y64, y16, hb = oracle.layer_with_routing_ex(x, idx, w, [g_w], [u_w], [d_w], round_h=False,
                                                want_hb=True)
    g = _f64(x) @ _f64(g_w)
    u = _f64(x) @ _f64(u_w)
    ref = (g * scipy.special.expit(g) * u) @ _f64(d_w)
    assert np.allclose(y64, ref, rtol=1e-12, atol=1e-12)
    assert np.array_equal(y16, oracle.bf16_round(y64))
    hb1, _ = oracle.expert_glu(x, g_w, u_w, d_w)
    assert np.array_equal(hb[:, 0, :], hb1)


def test_layer_with_routing_ex_rounded_form_is_the_layer():
    """With H rounded, the extended entry point gives the layer's bits, and
    each local pair's H row is that expert's hb for the token (rows of
    non-local pairs stay zero)."""
    x, wr, G, U, D = _tiny_inputs(T=9)
    r = oracle.layer(x, wr, None, G, U, D, k=2, e_begin=2, n_local=4)
    y64, y16, hb = oracle.layer_with_routing_ex(x, r["idx"], r["w"], G, U, D, e_begin=2,
                                                n_local=4, want_hb=True)
    assert np.array_equal(y64, r["y64"]) and np.array_equal(y16, r["y"])
    for t in range(9):
        for j in range(2):
            e = r["idx"][t, j]
            if 2 <= e < 6:
                h1, _ = oracle.expert_glu(x[t:t + 1], G[e], U[e], D[e])
                assert np.array_equal(hb[t, j], h1[0])
            else:
                assert np.all(hb[t, j] == 0)
    # the exact form differs from the rounded one by about the bf16 step of H
    e64, _, _ = oracle.layer_with_routing_ex(x, r["idx"], r["w"], G, U, D, e_begin=2, n_local=4,
                                             round_h=False)
    rel = np.linalg.norm(y64 - e64) / np.linalg.norm(e64)
    assert 1e-5 < rel < 4e-3


def test_layer_zero_input_gives_zero():
    x, wr, G, U, D = _tiny_inputs()
    x[:] = 0
    r = oracle.layer(x, wr, None, G, U, D, k=2)
    assert np.all(r["y64"] == 0.0)


def test_layer_sparse_equals_busy_full_loading_dense():
    """Sec. 4.2 busy full loading: all experts run, unselected zeroed."""
    x, wr, G, U, D = _tiny_inputs()
    r = oracle.layer(x, wr, None, G, U, D, k=2)
    dense = oracle.layer_dense(x, r["idx"], r["w"], G, U, D)
    assert np.allclose(r["y64"], dense, rtol=1e-13, atol=1e-15)


def test_layer_combine_is_weighted_sum_of_expert_outputs():
    x, wr, G, U, D = _tiny_inputs(T=6)
    r = oracle.layer(x, wr, None, G, U, D, k=3)
    for t in range(6):
        acc = np.zeros(x.shape[1])
        for j in range(3):
            e = r["idx"][t, j]
            _, o = oracle.expert_glu(x[t:t + 1], G[e], U[e], D[e])
            acc += r["w"][t, j] * o[0]
        assert np.allclose(r["y64"][t], acc, rtol=1e-14, atol=1e-16)


def test_layer_k_equals_E_is_soft_moe():
    x, wr, G, U, D = _tiny_inputs(T=4, E=4)
    r = oracle.layer(x, wr, None, G, U, D, k=4)
    p = scipy.special.softmax(r["logits"].astype(np.float64), axis=1)
    acc = np.zeros_like(r["y64"])
    for e in range(4):
        _, o = oracle.expert_glu(x, G[e], U[e], D[e])
        acc += p[:, e:e + 1] * o
    assert np.allclose(r["y64"], acc, rtol=1e-13, atol=1e-16)


def test_expert_parallel_shares_sum_to_full_layer():
    """Sec. 2.2 / Sec. 4.3: the all-reduce of the shares' partial outputs is
    the full layer's weighted sum."""
    x, wr, G, U, D = _tiny_inputs(T=12, E=8)
    full = oracle.layer(x, wr, None, G, U, D, k=2)
    tot = np.zeros_like(full["y64"])
    for s in range(4):
        part = oracle.layer(x, wr, None, G, U, D, k=2, e_begin=2 * s, n_local=2)
        assert np.array_equal(part["idx"], full["idx"])
        tot += part["y64"]
        # tokens with no slot in the share get exact zeros
        has = np.any((full["idx"] >= 2 * s) & (full["idx"] < 2 * s + 2), axis=1)
        assert np.all(part["y64"][~has] == 0.0)
    assert np.allclose(tot, full["y64"], rtol=1e-13, atol=1e-16)


def test_layer_unused_experts_may_be_absent():
    x, wr, G, U, D = _tiny_inputs(T=3)
    r = oracle.layer(x, wr, None, G, U, D, k=2)
    used = set(r["idx"].reshape(-1).tolist())
    G2 = [g if e in used else None for e, g in enumerate(G)]
    r2 = oracle.layer(x, wr, None, G2, U, D, k=2)
    assert np.array_equal(r["y"], r2["y"])


def test_residual_add_brute_force():
    rng = np.random.default_rng(11)
    x = mi.gen_bf16(0, mi.stream_id(mi.KIND_X), (300,), 1.0)
    y = mi.gen_bf16(0, mi.stream_id(mi.KIND_X, 1), (300,), 0.01)
    y[:10] = x[:10] ^ 0x8000                      # exact cancellation
    got = oracle.residual_add(x, y)
    for i in range(300):
        s = float(mi.bf16_bits_to_f32(x[i:i + 1])[0]) + float(mi.bf16_bits_to_f32(y[i:i + 1])[0])
        assert got[i] == _nearest_even_bf16(s) or (s == 0.0 and (got[i] & 0x7FFF) == 0)
    assert rng is not None


def test_bf16_from_f64_matches_torch_on_every_fp32_pattern():
    """Exhaustive: for all 2^32 fp32 bit patterns, the oracle's double->bf16
    (every fp32 value is exact in fp64) equals torch's fp32->bf16
    round-to-nearest-even; NaN stays NaN."""
    from concurrent.futures import ThreadPoolExecutor
    chunk = 1 << 24
    base = np.arange(chunk, dtype=np.uint32)

    def check(start):
        f = (base + np.uint32(start)).view(np.float32)
        want = torch.from_numpy(f).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
        with np.errstate(invalid="ignore"):
            got = oracle.bf16_round(f.astype(np.float64))
        nan = np.isnan(f)
        if not nan.any():
            return bool(np.array_equal(got, want))
        return bool(np.array_equal(got[~nan], want[~nan]) and
                    np.all(np.isnan(mi.bf16_bits_to_f32(got[nan]))))

    torch.set_num_threads(1)
    try:
        with ThreadPoolExecutor(min(8, os.cpu_count() or 1)) as ex:
            bad = [hex(s) for s, ok in zip(range(0, 1 << 32, chunk),
                                           ex.map(check, range(0, 1 << 32, chunk))) if not ok]
    finally:
        torch.set_num_threads(os.cpu_count() or 1)
    assert not bad, bad[:8]
