"""A decoder stack through both C-ABIs, each layer as DBRX arranges it (Sec.
2.1's decoder layer: self-attention, then the MoE FFN on a normalised input):
attn_forward_norm gives y = bf16(x + attn_l(norm1(x))) (its key/value cache
appended) and z = norm2(y); moe_forward_residual then adds the MoE layer's
output on z into the stream, x = bf16(y + bf16(moe_l(z))).  Each piece is
checked against the oracle on the GPU's own input to it (teacher forcing),
the caches hold exactly the appended positions, and the chain repeats bit for
bit -- at decode (T = 3) and through the prefill path (T = 40)."""
import numpy as np
import pytest

import moe_inputs as mi
import oracle
import paper_2506_23635_amd as moe
from harness import (bf16_f64, bf16_step, check_layer_output, host_experts, load_workload_host,
                     make_layer, rel_l2)

pytestmark = pytest.mark.gpu

N_LAYERS = 3
MOE_WL = mi.WORKLOADS["tiny"].with_(T=3, n_layers=N_LAYERS)
ATTN_WL = mi.ATTN_WORKLOADS["attn_tiny"].with_(T=3, pos0=61)


@pytest.fixture(scope="module")
def torch_mod():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch


def _build(torch, aw, max_tokens=4):
    mw = MOE_WL
    assert aw.d == mw.d
    cfg = moe.make_attn_config(aw.d, aw.n_heads, aw.n_kv, aw.hd, n_layers=N_LAYERS,
                               max_seq=aw.max_seq, max_tokens=max(16, max_tokens),
                               rope_theta=aw.theta, norm_eps=aw.eps)
    att = moe.AttnLayer(cfg)
    caches = []
    for li in range(N_LAYERS):
        att.load_layer(li, torch.from_numpy(aw.gamma(li)), torch.from_numpy(aw.wqkv(li).view(np.int16)),
                       torch.from_numpy(aw.wo(li).view(np.int16)))
        att.load_post_norm(li, torch.from_numpy(aw.gamma2(li)))
        k0, v0 = aw.cache_prefix(li)
        K, V = att.cache_views(li)
        K.zero_()
        V.zero_()
        K[:, :aw.pos0] = torch.from_numpy(np.ascontiguousarray(k0.transpose(1, 0, 2)).view(np.int16)).cuda()
        V[:, :aw.pos0] = torch.from_numpy(np.ascontiguousarray(v0.transpose(1, 0, 2)).view(np.int16)).cuda()
        kc = np.zeros((aw.max_seq, aw.n_kv, aw.hd), np.uint16)
        vc = np.zeros_like(kc)
        kc[:aw.pos0], vc[:aw.pos0] = k0, v0
        caches.append((kc, vc))
    ffn = make_layer(mw, max_tokens=max_tokens, n_layers=N_LAYERS)
    for li in range(N_LAYERS):
        load_workload_host(ffn, mw, layer_idx=li)
    torch.cuda.synchronize()
    return att, ffn, caches


def _run(torch, att, ffn, x0, pos0):
    """The chain; per layer the block input, y and z (bf16 bits), then the
    final stream."""
    x = torch.from_numpy(x0.view(np.int16)).cuda()
    z = torch.empty_like(x)
    seen = []
    for li in range(N_LAYERS):
        xin = x.cpu().numpy().view(np.uint16).copy()
        att.forward_norm(li, x, x, z, pos0)
        torch.cuda.synchronize()
        seen.append((xin, x.cpu().numpy().view(np.uint16).copy(), z.cpu().numpy().view(np.uint16).copy()))
        ffn.forward_residual(li, z, x)
        torch.cuda.synchronize()
    return seen, x.cpu().numpy().view(np.uint16).copy()


@pytest.mark.parametrize("T,pos0", [(3, 61), (40, 0)])
def test_decoder_chain_layer_by_layer(torch_mod, T, pos0):
    torch = torch_mod
    aw, mw = ATTN_WL.with_(T=T, pos0=pos0), MOE_WL.with_(T=T)
    att, ffn, caches = _build(torch, aw, max_tokens=max(4, T))
    try:
        x0 = mw.x()
        seen, final = _run(torch, att, ffn, x0, pos0)
        for li in range(N_LAYERS):
            xin, y, z = seen[li]
            xout = seen[li + 1][0] if li + 1 < N_LAYERS else final
            kc, vc = caches[li]
            ref = oracle.attention_block(xin, aw.gamma(li), aw.wqkv(li), aw.wo(li), kc.copy(),
                                         vc.copy(), pos0, aw.n_heads, aw.n_kv, aw.eps, aw.theta)
            check_layer_output(y, ref["y64"])
            # z: the post-attention norm of the GPU's own y, within one bf16 step
            zr = bf16_f64(oracle.layernorm(y, aw.gamma2(li), aw.eps))
            zg = bf16_f64(z)
            assert np.all(np.abs(zg - zr) <= bf16_step(np.maximum(np.abs(zg), np.abs(zr))) * (1 + 1e-9))
            G, U, D = host_experts(mw, range(mw.E), li)
            r = oracle.layer(z, mw.router(li), mw.bias(li), G, U, D, mw.k)
            check_layer_output(xout, bf16_f64(y) + r["y64"])
            # the cache holds the prefix and exactly the appended positions
            K, V = att.cache_views(li)
            torch.cuda.synchronize()
            kg = K.cpu().numpy().view(np.uint16).transpose(1, 0, 2)
            assert np.array_equal(kg[:pos0], kc[:pos0])
            assert np.all(kg[pos0 + T:] == 0)
            assert not np.all(kg[pos0:pos0 + T] == 0)
        # the chain again (it rewrites the same cache positions): the same bits
        again, final2 = _run(torch, att, ffn, x0, pos0)
        for a, b in zip(seen, again):
            for u, v in zip(a, b):
                assert np.array_equal(u, v)
        assert np.array_equal(final, final2)
        assert rel_l2(bf16_f64(final), bf16_f64(x0)) > 1e-3     # the layers did something
    finally:
        att.close()
        ffn.close()
