"""A decoder stack through both C-ABIs: for each layer l, the self-attention
block of attn.h (x = bf16(x + attn_l(x)), its key/value cache appended) and
then the MoE layer of moe.h (moe_forward_layers: x = bf16(x + moe_l(x))), the
order of Sec. 2.1's decoder layer.  Each block is checked against the oracle
on the GPU's own input to it (teacher forcing: the attention block and the
MoE layer of the oracle, end-to-end bar on the block's output), the caches
hold exactly the appended positions, and the chain repeats bit for bit."""
import numpy as np
import pytest

import moe_inputs as mi
import oracle
import paper_2506_23635_amd as moe
from harness import (bf16_f64, check_layer_output, host_experts, load_workload_host,
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


def _build(torch):
    aw, mw = ATTN_WL, MOE_WL
    assert aw.d == mw.d
    cfg = moe.make_attn_config(aw.d, aw.n_heads, aw.n_kv, aw.hd, n_layers=N_LAYERS,
                               max_seq=aw.max_seq, max_tokens=16, rope_theta=aw.theta,
                               norm_eps=aw.eps)
    att = moe.AttnLayer(cfg)
    caches = []
    for li in range(N_LAYERS):
        att.load_layer(li, torch.from_numpy(aw.gamma(li)), torch.from_numpy(aw.wqkv(li).view(np.int16)),
                       torch.from_numpy(aw.wo(li).view(np.int16)))
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
    ffn = make_layer(mw, max_tokens=4, n_layers=N_LAYERS)
    for li in range(N_LAYERS):
        load_workload_host(ffn, mw, layer_idx=li)
    torch.cuda.synchronize()
    return att, ffn, caches


def _run(torch, att, ffn, x0):
    """The chain; returns the input of every block (bf16 bits)."""
    x = torch.from_numpy(x0.view(np.int16)).cuda()
    seen = []
    for li in range(N_LAYERS):
        seen.append(x.cpu().numpy().view(np.uint16).copy())
        att.forward(li, x, x, ATTN_WL.pos0)
        torch.cuda.synchronize()
        seen.append(x.cpu().numpy().view(np.uint16).copy())
        ffn.forward_layers(li, 1, x)
        torch.cuda.synchronize()
    seen.append(x.cpu().numpy().view(np.uint16).copy())
    return seen


def test_decoder_chain_layer_by_layer(torch_mod):
    torch = torch_mod
    aw, mw = ATTN_WL, MOE_WL
    att, ffn, caches = _build(torch)
    try:
        x0 = mw.x()
        seen = _run(torch, att, ffn, x0)
        for li in range(N_LAYERS):
            xin, xmid, xout = seen[2 * li], seen[2 * li + 1], seen[2 * li + 2]
            kc, vc = caches[li]
            ref = oracle.attention_block(xin, aw.gamma(li), aw.wqkv(li), aw.wo(li), kc.copy(),
                                         vc.copy(), aw.pos0, aw.n_heads, aw.n_kv, aw.eps, aw.theta)
            check_layer_output(xmid, ref["y64"])
            G, U, D = host_experts(mw, range(mw.E), li)
            r = oracle.layer(xmid, mw.router(li), mw.bias(li), G, U, D, mw.k)
            want = bf16_f64(xmid) + r["y64"]
            check_layer_output(xout, want)
            # the cache holds the prefix and exactly the appended positions
            K, V = att.cache_views(li)
            torch.cuda.synchronize()
            kg = K.cpu().numpy().view(np.uint16).transpose(1, 0, 2)
            assert np.array_equal(kg[:aw.pos0], kc[:aw.pos0])
            assert np.all(kg[aw.pos0 + aw.T:] == 0)
            assert not np.all(kg[aw.pos0:aw.pos0 + aw.T] == 0)
        # the chain again (it rewrites the same cache positions): the same bits
        again = _run(torch, att, ffn, x0)
        for a, b in zip(seen, again):
            assert np.array_equal(a, b)
        assert rel_l2(bf16_f64(seen[-1]), bf16_f64(x0)) > 1e-3     # the layers did something
    finally:
        att.close()
        ffn.close()
