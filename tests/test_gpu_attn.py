"""GPU parity of the self-attention block (include/attn.h) through the C-ABI,
against the fp64 oracle (oracle/attn_oracle.c).

Every stage is checked per element, against the oracle or against an fp64
evaluation of the GPU's own input to that stage, with bounds from fp32
arithmetic:
  h    vs the oracle's layer norm: within one bf16 step (fp32 statistics);
  qkv  vs h_gpu Wqkv in fp64: gamma_d sum |h||w|;
  q, k vs the pinned rotary encoding of the GPU's own qkv, rounded: one bf16
       step (fp32 rotation); v likewise without rotation;
  a    vs the oracle's attention on the GPU's own q and cache: half a bf16
       step plus the fp32 score error carried through the softmax;
  o    vs a_gpu Wo in fp64: gamma_nq sum |a||w|;
  y    = bf16(fp32(x + o_gpu)) exactly (the kernel's residual rounding);
and end to end: o and y against the oracle block (relative L2 <= 2e-3,
max-abs <= 1e-2 max(1, max|ref|)).  T tokens at once equal T single-token
steps bit for bit, the cache changes only at the new positions, and repeated
calls give the same bits."""
import numpy as np
import pytest

import moe_inputs as mi
import oracle
import paper_2506_23635_amd as moe
from harness import bf16_step, check_layer_output, gamma, rel_l2

pytestmark = pytest.mark.gpu

TINY = mi.ATTN_WORKLOADS["attn_tiny"]
DBRX = mi.ATTN_WORKLOADS["attn_decode"]
U32 = 2.0 ** -24


@pytest.fixture(scope="module")
def torch_mod():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch


def f64(b):
    return mi.bf16_bits_to_f32(np.asarray(b, np.uint16)).astype(np.float64)


class Case:
    """An AttnLayer holding one layer of a workload, its cache prefix written
    (positions < pos0), and the host copies the oracle needs."""

    def __init__(self, torch, wl, max_tokens=16, on_device=False):
        self.torch, self.wl = torch, wl
        cfg = moe.make_attn_config(wl.d, wl.n_heads, wl.n_kv, wl.hd, n_layers=1,
                                   max_seq=wl.max_seq, max_tokens=max_tokens,
                                   rope_theta=wl.theta, norm_eps=wl.eps)
        self.layer = moe.AttnLayer(cfg)
        self.gamma, self.wqkv, self.wo = wl.gamma(), wl.wqkv(), wl.wo()
        dev = "cuda" if on_device else "cpu"
        self.layer.load_layer(0, torch.from_numpy(self.gamma).to(dev),
                              torch.from_numpy(self.wqkv.view(np.int16)).to(dev),
                              torch.from_numpy(self.wo.view(np.int16)).to(dev))
        k0, v0 = wl.cache_prefix()
        K, V = self.layer.cache_views(0)
        # a pattern everywhere, then the prefix: writes past the new
        # positions would show
        K.fill_(0x1234)
        V.fill_(0x1234)
        K[:, :wl.pos0] = torch.from_numpy(np.ascontiguousarray(k0.transpose(1, 0, 2)).view(np.int16)).cuda()
        V[:, :wl.pos0] = torch.from_numpy(np.ascontiguousarray(v0.transpose(1, 0, 2)).view(np.int16)).cuda()
        torch.cuda.synchronize()
        # host caches in the oracle's position-major layout
        self.kc = np.zeros((wl.max_seq, wl.n_kv, wl.hd), np.uint16)
        self.vc = np.zeros_like(self.kc)
        self.kc[:wl.pos0], self.vc[:wl.pos0] = k0, v0

    def cache(self):
        K, V = self.layer.cache_views(0)
        self.torch.cuda.synchronize()
        return (K.cpu().numpy().view(np.uint16).transpose(1, 0, 2),
                V.cpu().numpy().view(np.uint16).transpose(1, 0, 2))

    def forward(self, x, pos0, out=None):
        torch = self.torch
        x_t = torch.from_numpy(x.view(np.int16)).cuda()
        y_t = torch.full_like(x_t, 0x3F80) if out is None else out
        self.layer.forward(0, x_t, y_t, pos0)
        torch.cuda.synchronize()
        return y_t.cpu().numpy().view(np.uint16)

    def close(self):
        self.layer.close()


def check_block(case, x, pos0, y, inter, kc_gpu, vc_gpu, tokens=None):
    """The per-element chain and the end-to-end comparison for one call
    (the attention bound on `tokens` only, when given)."""
    wl = case.wl
    T, d, H, G, hd = x.shape[0], wl.d, wl.n_heads, wl.n_kv, wl.hd
    nq, nkv = H * hd, G * hd
    ref = oracle.attention_block(x, case.gamma, case.wqkv, case.wo, case.kc, case.vc, pos0, H, G,
                                 wl.eps, wl.theta)
    # h: fp32 statistics against fp64 ones, one bf16 step at most
    hg, hr = f64(inter["h"]), f64(ref["h"])
    assert np.all(np.abs(hg - hr) <= bf16_step(np.maximum(np.abs(hg), np.abs(hr))) * (1 + 1e-9))
    assert np.mean(inter["h"] == ref["h"]) > 0.98
    # qkv against the GPU's own h
    w = f64(case.wqkv)
    qkv_ref = hg @ w
    bound = gamma(d) * (np.abs(hg) @ np.abs(w)) + 1e-30
    err = np.abs(inter["qkv"] - qkv_ref)
    assert np.all(err <= bound), float((err / bound).max())
    # rotation and rounding of the GPU's own qkv
    qkv = inter["qkv"].astype(np.float64)
    pos = np.repeat(np.arange(pos0, pos0 + T, dtype=np.int32), H)
    q_ref = oracle.rope(qkv[:, :nq].reshape(T * H, hd), pos, wl.theta).reshape(T, nq)
    posk = np.repeat(np.arange(pos0, pos0 + T, dtype=np.int32), G)
    k_ref = oracle.rope(qkv[:, nq:nq + nkv].reshape(T * G, hd), posk, wl.theta).reshape(T, G, hd)
    v_ref = qkv[:, nq + nkv:].reshape(T, G, hd)

    def pair_abs(v, n_heads):
        # |x_i| + |x_{i+hd/2}| for both members of each rotated pair: the fp32
        # rotation (rounded cos/sin, two products and a sum) errs by at most
        # 4 u times this, however much the result cancels
        a = np.abs(v.reshape(T, n_heads, 2, hd // 2))
        return np.repeat((a[:, :, 0] + a[:, :, 1])[:, :, None, :], 2, axis=2).reshape(T, n_heads * hd)

    rot_q = 4 * U32 * pair_abs(qkv[:, :nq], H)
    rot_k = 4 * U32 * pair_abs(qkv[:, nq:nq + nkv], G).reshape(T, G, hd)
    for got, want, rot in ((inter["q"], q_ref, rot_q), (kc_gpu[pos0:pos0 + T], k_ref, rot_k),
                           (vc_gpu[pos0:pos0 + T], v_ref, 0.0)):
        gv = f64(got)
        b = 0.5 * bf16_step(np.maximum(np.abs(gv), np.abs(want))) + rot + 1e-30
        assert np.all(np.abs(gv - want) <= b * (1 + 1e-9)), float((np.abs(gv - want) / b).max())
    # the cache holds the prefix and the new keys/values only
    assert np.array_equal(kc_gpu[:pos0], case.kc[:pos0]) and np.array_equal(vc_gpu[:pos0], case.vc[:pos0])
    assert np.all(kc_gpu[pos0 + T:] == 0x1234) and np.all(vc_gpu[pos0 + T:] == 0x1234)
    # attention on the GPU's own q and cache
    q3 = inter["q"].reshape(T, H, hd)
    a_ref_bits, a64 = oracle.attention_core(q3, kc_gpu, vc_gpu, pos0)
    group = H // G
    ag = f64(inter["a"])
    # per head, for all chosen tokens at once: es[t] = the fp32 score error
    # bound gamma_hd max_p |k_p| . |q_t| / sqrt(hd) over the token's visible
    # positions, vmax[t] = max |v| over them (a running maximum)
    toks = np.arange(T) if tokens is None else np.asarray(tokens)
    n_pos = pos0 + toks + 1
    P = pos0 + T
    kk = np.abs(f64(kc_gpu[:P]))                                   # [P, G, hd]
    vcm = np.maximum.accumulate(np.abs(f64(vc_gpu[:P])), axis=0)   # running max over positions
    visible = np.arange(P)[None, :] < n_pos[:, None]               # [tokens, P]
    for j in range(H):
        g = j // group
        qa = np.abs(f64(q3[toks, j]))                              # [tokens, hd]
        es = gamma(hd) * np.where(visible, qa @ kk[:, g, :].T, 0.0).max(axis=1) / np.sqrt(hd)
        vmax = vcm[n_pos - 1, g, :]                                 # [tokens, hd]
        sl = slice(j * hd, (j + 1) * hd)
        # half a bf16 step, the fp32 score error through the softmax, and
        # 2^-15 vmax for the prefill path's P (two bf16 terms, 16 bits)
        b = (0.5 * bf16_step(np.maximum(np.abs(ag[toks, sl]), np.abs(a64[toks, sl]))) +
             (2 * es[:, None] + (n_pos[:, None] + 64) * U32) * 2 * vmax + 2.0 ** -15 * vmax + 1e-30)
        e = np.abs(ag[toks, sl] - a64[toks, sl])
        ok = e <= b
        if not ok.all():
            i, dd = np.argwhere(~ok)[0]
            raise AssertionError((int(toks[i]), j, int(dd), float((e / b).max())))
    sel = slice(None) if tokens is None else np.asarray(tokens)
    assert np.mean(inter["a"][sel] == a_ref_bits[sel]) > 0.9
    # o against the GPU's own a
    wo = f64(case.wo)
    o_ref = ag @ wo
    ob = gamma(nq) * (np.abs(ag) @ np.abs(wo)) + 1e-30
    assert np.all(np.abs(inter["o"] - o_ref) <= ob)
    # the residual rounding of the kernel, exactly
    xs = mi.bf16_bits_to_f32(x)
    want = oracle.bf16_round((xs + inter["o"].astype(np.float32)).astype(np.float64))
    assert np.array_equal(y, want)
    # end to end against the oracle block
    og = inter["o"].astype(np.float64)
    assert rel_l2(og, ref["o64"]) <= 2e-3
    assert np.abs(og - ref["o64"]).max() <= 1e-2 * max(1.0, np.abs(ref["o64"]).max())
    check_layer_output(y, ref["y64"])
    return ref


@pytest.mark.parametrize("T,pos0,on_device", [(4, 29, False), (1, 0, True), (16, 250, True),
                                              (3, 253, False)])
def test_small_block(torch_mod, T, pos0, on_device):
    torch = torch_mod
    wl = TINY.with_(T=T, pos0=pos0)
    case = Case(torch, wl, on_device=on_device)
    try:
        x = wl.x()
        y = case.forward(x, pos0)
        kc, vc = case.cache()
        check_block(case, x, pos0, y, case.layer.intermediates(T), kc, vc)
    finally:
        case.close()


def test_tokens_at_once_equal_single_steps(torch_mod):
    """T = 6 tokens in one call (crossing a 256-position chunk) give the same
    bits as six single-token calls, and so does the cache."""
    torch = torch_mod
    wl = TINY.with_(T=6, pos0=252)
    x = wl.x()
    a = Case(torch, wl)
    b = Case(torch, wl)
    try:
        ya = a.forward(x, wl.pos0)
        yb = np.concatenate([b.forward(x[t:t + 1], wl.pos0 + t) for t in range(6)])
        assert np.array_equal(ya, yb)
        ka, va = a.cache()
        kb, vb = b.cache()
        assert np.array_equal(ka, kb) and np.array_equal(va, vb)
        # and again, the same bits
        a.forward(x, wl.pos0)
        assert np.array_equal(a.forward(x, wl.pos0), ya)
    finally:
        a.close()
        b.close()


@pytest.mark.parametrize("T,pos0", [(1, 2047), (4, 100), (16, 1000)])
def test_dbrx_block(torch_mod, T, pos0):
    """DBRX widths: d 6144, 48 query heads and 8 key/value heads of 128
    (D_qkv_hidden 8192), one decode token after 2047 cached positions, and
    4 and 16 tokens (16 query rows per key/value head, 96 in all)."""
    torch = torch_mod
    wl = DBRX.with_(T=T, pos0=pos0)
    case = Case(torch, wl, on_device=True)
    try:
        x = wl.x()
        y = case.forward(x, pos0)
        kc, vc = case.cache()
        check_block(case, x, pos0, y, case.layer.intermediates(T), kc, vc)
        assert np.array_equal(case.forward(x, pos0), y)
    finally:
        case.close()


@pytest.mark.parametrize("d,H,G,hd,T", [(2048, 32, 8, 64, 2), (2048, 64, 8, 128, 1),
                                         (4096, 32, 4, 128, 4), (8192, 16, 2, 128, 5)])
def test_projection_shapes(torch_mod, d, H, G, hd, T):
    """Widths whose K loops run 1, 2 and 4 full weight batches per wave in
    the two projections (K = 2048, 4096, 8192 for q|k|v; 2048, 4096, 8192
    for the output), besides the 0 of the small block and the 3 of the DBRX
    block; T = 5 takes the separate norm kernel."""
    torch = torch_mod
    wl = TINY.with_(d=d, n_heads=H, n_kv=G, hd=hd, T=T, pos0=70)
    case = Case(torch, wl)
    try:
        x = wl.x()
        y = case.forward(x, wl.pos0)
        kc, vc = case.cache()
        check_block(case, x, wl.pos0, y, case.layer.intermediates(T), kc, vc)
    finally:
        case.close()


@pytest.mark.parametrize("d,H,G,hd,T,pos0", [(2048, 32, 8, 64, 40, 70), (1024, 8, 8, 128, 150, 30),
                                               (1024, 8, 1, 128, 150, 30), (4096, 32, 4, 128, 200, 0)])
def test_prefill_shapes(torch_mod, d, H, G, hd, T, pos0):
    """The prefill path on other head layouts, every stage per element:
    head_dim 64 at four query heads per key/value head, one query head per
    key/value head (multi-head attention) and one key/value head for all
    (multi-query), and eight per head at d 4096; the causal attention's
    workgroup numbering then maps 1, 4 or 8 query heads to a key/value head."""
    torch = torch_mod
    wl = TINY.with_(d=d, n_heads=H, n_kv=G, hd=hd, T=T, pos0=pos0)
    case = Case(torch, wl, max_tokens=256)
    try:
        x = wl.x()
        y = case.forward(x, pos0)
        kc, vc = case.cache()
        check_block(case, x, pos0, y, case.layer.intermediates(T), kc, vc)
    finally:
        case.close()


@pytest.mark.parametrize("T,pos0", [(17, 0), (64, 37), (100, 200), (130, 0), (171, 341)])
def test_prefill_small_block(torch_mod, T, pos0):
    """More than 16 new tokens: the prefill path (projection GEMMs, rotation
    and cache append, causal attention on the matrix cores), every stage
    per element; T spans partial 128-token query blocks, partial 64-position
    steps and 256-row GEMM tiles, pos0 a cached prefix or none; the last
    case ends exactly at the cache's last position (pos0 + T = max_seq =
    512), so the last query block's K/V loads reach the end of the cache."""
    torch = torch_mod
    wl = TINY.with_(T=T, pos0=pos0)
    case = Case(torch, wl, max_tokens=256)
    try:
        x = wl.x()
        y = case.forward(x, pos0)
        kc, vc = case.cache()
        check_block(case, x, pos0, y, case.layer.intermediates(T), kc, vc)
        assert np.array_equal(case.forward(x, pos0), y)
    finally:
        case.close()


@pytest.mark.parametrize("T,pos0", [(300, 1000), (2048, 0)])
def test_prefill_dbrx_block(torch_mod, T, pos0):
    """DBRX widths through the prefill path: 300 tokens after 1000 cached
    positions, and the whole 2048-token prompt of the long-prompt workload
    from an empty cache.  Every stage per element, the attention on every
    token and head."""
    torch = torch_mod
    wl = DBRX.with_(T=T, pos0=pos0)
    case = Case(torch, wl, max_tokens=2048, on_device=True)
    try:
        x = wl.x()
        y = case.forward(x, pos0)
        kc, vc = case.cache()
        check_block(case, x, pos0, y, case.layer.intermediates(T), kc, vc)
    finally:
        case.close()


def test_prefill_then_decode(torch_mod):
    """A 40-token prompt through the prefill path fills the cache that the
    next token's decode call reads: the decode step checks per element
    against the oracle on that cache."""
    torch = torch_mod
    wl = TINY.with_(T=40, pos0=0)
    case = Case(torch, wl, max_tokens=64)
    try:
        x = wl.x()
        y = case.forward(x, 0)
        kc, vc = case.cache()
        check_block(case, x, 0, y, case.layer.intermediates(40), kc, vc)
        # the oracle's host caches take the prompt's keys and values as the GPU wrote them
        case.kc[:40], case.vc[:40] = kc[:40], vc[:40]
        x1 = TINY.with_(T=1).x(1)
        y1 = case.forward(x1, 40)
        kc1, vc1 = case.cache()
        check_block(case, x1, 40, y1, case.layer.intermediates(1), kc1, vc1)
    finally:
        case.close()


def test_in_place_and_rejections(torch_mod):
    torch = torch_mod
    wl = TINY.with_(T=2, pos0=10)
    case = Case(torch, wl)
    try:
        x = wl.x()
        y = case.forward(x, wl.pos0)
        xt = torch.from_numpy(x.view(np.int16)).cuda()
        case.layer.forward(0, xt, xt, wl.pos0)        # y may be x
        torch.cuda.synchronize()
        assert np.array_equal(xt.cpu().numpy().view(np.uint16), y)
        for T, p0 in ((17, 0), (2, wl.max_seq - 1)):      # past max_tokens, past max_seq
            xx = torch.zeros((T, wl.d), dtype=torch.int16, device="cuda")
            yy = torch.full_like(xx, 7)
            with pytest.raises(moe.MoeError) as ei:
                case.layer.forward(0, xx, yy, p0)
            assert ei.value.status == -4
            torch.cuda.synchronize()
            assert bool((yy == 7).all())
    finally:
        case.close()
