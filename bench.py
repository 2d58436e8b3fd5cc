"""Benchmark of the DBRX-shaped MoE layer on one MI355X.

Headline workload: one decode token through the whole 16-expert layer
(d_model 6144, ffn 10752, top-4, bf16 weights ~N(0, 0.006)); one step = one
moe_forward (router, selection, permutation, gate/up + SiLU, down, weighted
combine) on inputs already resident in HBM.  The prefill layer (2048 tokens,
N(0,1) weights, skewed routing) is timed in the same run and reported under
"prefill".  The fp64 CPU oracle is timed on a bounded sample of the decode
workload as a baseline.

Prints one JSON line.  Usage: python bench.py [--gpus 1] [--steps K] [--warmup W]
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "DBRX-shape MoE layer: decode µs/layer + HBM GB/s; prefill tokens/s + MFMA %"
N_ROT = 4                      # independently seeded layers the decode timing rotates over
HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, GB/s
MFMA_BF16_PEAK_TFLOPS = 2500.0  # MI355X dense bf16 matrix, TFLOP/s


def log(msg):
    print(msg, file=sys.stderr, flush=True)


# One device allocation made before any section runs; every section carves
# its weight arena, workspace and staging buffers from it after a reset.
# Measured: an arena allocated into memory that an earlier section had
# allocated and freed streams 2-4 % slower (the decode step after the 4 GiB
# read buffer 249.3 vs 239.5 us, expert-parallel shares after the decode
# layer up to 4 %), so without the pool each figure would depend on what ran
# before it in the process.
_POOL = None
_POOL_OFF = 0


def pool_init(nbytes):
    global _POOL, _POOL_OFF
    import torch
    _POOL = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    _POOL_OFF = 0


def pool_reset():
    """Starts a section: the previous section's work has finished before
    its memory is handed out again."""
    global _POOL_OFF
    import torch
    torch.cuda.synchronize()
    _POOL_OFF = 0


def pool_take(nbytes):
    """A 256-byte-aligned uint8 view of the pool (a plain allocation when
    no pool was made, e.g. for helper scripts)."""
    global _POOL_OFF
    import torch
    if _POOL is None:
        return torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    off = (_POOL_OFF + 255) // 256 * 256
    if off + nbytes > _POOL.numel():
        raise RuntimeError(f"bench pool exhausted ({off + nbytes} of {_POOL.numel()} bytes)")
    _POOL_OFF = off + nbytes
    return _POOL[off: off + nbytes]


def pool_release():
    """Ends the run's device work explicitly: waits for the stream, drops the
    pool and returns torch's cached blocks, so that no device memory is freed
    during interpreter shutdown (after a profiler's own exit handlers)."""
    global _POOL, _POOL_OFF
    import torch
    torch.cuda.synchronize()
    _POOL = None
    _POOL_OFF = 0
    torch.cuda.empty_cache()
    torch.cuda.synchronize()


def pool_layer(cfg):
    import paper_2506_23635_amd as moe
    return moe.MoeLayer(cfg, arena=pool_take(moe.moe_weight_bytes(cfg)),
                        workspace=pool_take(moe.moe_workspace_bytes(cfg)))


def staging_buffer(wl):
    import torch
    return pool_take(3 * wl.d * wl.f * 2).view(torch.int16)


def section_bytes(cfg, wl):
    """Pool bytes one section takes: arena, workspace, staging, alignment."""
    import paper_2506_23635_amd as moe
    return moe.moe_weight_bytes(cfg) + moe.moe_workspace_bytes(cfg) + 3 * wl.d * wl.f * 2 + (16 << 20)


def setup_layer(wl, max_tokens):
    import torch
    import moe_inputs as mi
    import paper_2506_23635_amd as moe
    cfg = moe.make_config(wl.d, wl.f, wl.E, wl.k, max_tokens=max_tokens)
    pool_reset()
    layer = pool_layer(cfg)
    s = layer.stream
    d, f, E = wl.d, wl.f, wl.E
    wr = torch.empty(d * E, dtype=torch.float32, device="cuda")
    mi.gen_f32_device(wl.seed, mi.stream_id(mi.KIND_ROUTER), d * E, wl.sigma_r, wr.data_ptr(), s)
    b = None
    if wl.sigma_b:
        b = torch.empty(E, dtype=torch.float32, device="cuda")
        mi.gen_f32_device(wl.seed, mi.stream_id(mi.KIND_BIAS), E, wl.sigma_b, b.data_ptr(), s)
    layer.load_router(0, wr, b)
    stg = staging_buffer(wl)
    g, u, dn = stg[: d * f], stg[d * f: 2 * d * f], stg[2 * d * f:]
    for e in range(E):
        mi.gen_bf16_device(wl.seed, mi.stream_id(mi.KIND_GATE, 0, e), d * f, wl.sigma_w, g.data_ptr(), s)
        mi.gen_bf16_device(wl.seed, mi.stream_id(mi.KIND_UP, 0, e), d * f, wl.sigma_w, u.data_ptr(), s)
        mi.gen_bf16_device(wl.seed, mi.stream_id(mi.KIND_DOWN, 0, e), d * f, wl.sigma_w, dn.data_ptr(), s)
        layer.load_expert(0, e, g, u, dn)
    x = torch.empty(wl.T * d, dtype=torch.int16, device="cuda")
    mi.gen_bf16_device(wl.seed, mi.stream_id(mi.KIND_X), wl.T * d, wl.sigma_x, x.data_ptr(), s)
    torch.cuda.synchronize()
    del stg
    return layer, x.view(wl.T, d)


def setup_rotation(wl, n_rot, max_tokens):
    """The whole 16-expert layer held n_rot times, each copy an independently
    seeded layer (router and experts of layer index 0..n_rot-1), so that a
    timed step rotating over them re-reads no weight byte within
    (n_rot - 1) layers (~19 GB at DBRX shape): the 256 MB last-level cache
    cannot serve repeats.  The input x is the same for every copy."""
    import torch
    import moe_inputs as mi
    import paper_2506_23635_amd as moe
    cfg = moe.make_config(wl.d, wl.f, wl.E, wl.k, n_layers=n_rot, max_tokens=max_tokens)
    pool_reset()
    layer = pool_layer(cfg)
    staging = staging_buffer(wl)
    for li in range(n_rot):
        load_layer_device(layer, wl, li, li, staging)
    x = torch.empty(wl.T * wl.d, dtype=torch.int16, device="cuda")
    mi.gen_bf16_device(wl.seed, mi.stream_id(mi.KIND_X), wl.T * wl.d, wl.sigma_x, x.data_ptr(),
                       layer.stream)
    torch.cuda.synchronize()
    del staging
    return layer, x.view(wl.T, wl.d)


def time_layer(layer, x, steps, warmup, kernel_events=True, n_rot=1):
    """Runs warmup + timed steps, step i on arena layer i % n_rot; returns
    (ms_per_step, per-kernel ms/launch, routing of layer 0, dropped)."""
    import torch
    import paper_2506_23635_amd as moe
    T = x.shape[0]
    y = torch.empty((T, layer.cfg.d_model), dtype=torch.int16, device="cuda")
    for i in range(max(warmup, n_rot)):
        layer.forward(i % n_rot, x, y)
    torch.cuda.synchronize()
    steps = max(steps - steps % n_rot, n_rot)
    moe.moe_profile_enable(layer.ctx, 8 * steps + 8 if kernel_events else 0)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(steps):
        layer.forward(i % n_rot, x, y)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    prof, dropped = moe.moe_profile_read(layer.ctx)
    moe.moe_profile_enable(layer.ctx, 0)
    r = layer.route(0, x)
    rt = layer.routing_tensors(r)
    if not kernel_events:
        prof = {}
    per_kernel = {k: {"ms_per_launch": v[0] / v[1], "launches": v[1]}
                  for k, v in prof.items() if v[1]}
    return (t1 - t0) * 1e3 / steps, per_kernel, rt, dropped


def graph_ms(fn, steps, warmup):
    """Captures one call of fn in a HIP graph and times `steps` replays
    (after `warmup` replays) with events; ms per replay."""
    import torch
    fn()
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        fn()
    for _ in range(warmup):
        g.replay()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(steps):
        g.replay()
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / steps
    del g
    return ms


def load_layer_device(layer, wl, layer_idx, arena_layer, staging):
    """Router and the context's local experts of layer `layer_idx` of `wl`,
    generated on the device into `arena_layer` of the context."""
    import torch
    import moe_inputs as mi
    s = layer.stream
    d, f, E = wl.d, wl.f, wl.E
    wr = torch.empty(d * E, dtype=torch.float32, device="cuda")
    mi.gen_f32_device(wl.seed, mi.stream_id(mi.KIND_ROUTER, layer_idx), d * E, wl.sigma_r,
                      wr.data_ptr(), s)
    b = None
    if wl.sigma_b:
        b = torch.empty(E, dtype=torch.float32, device="cuda")
        mi.gen_f32_device(wl.seed, mi.stream_id(mi.KIND_BIAS, layer_idx), E, wl.sigma_b,
                          b.data_ptr(), s)
    layer.load_router(arena_layer, wr, b)
    g, u, dn = staging[: d * f], staging[d * f: 2 * d * f], staging[2 * d * f:]
    c = layer.cfg
    for e in range(c.expert_begin, c.expert_begin + c.n_local_experts):
        mi.gen_bf16_device(wl.seed, mi.stream_id(mi.KIND_GATE, layer_idx, e), d * f, wl.sigma_w,
                           g.data_ptr(), s)
        mi.gen_bf16_device(wl.seed, mi.stream_id(mi.KIND_UP, layer_idx, e), d * f, wl.sigma_w,
                           u.data_ptr(), s)
        mi.gen_bf16_device(wl.seed, mi.stream_id(mi.KIND_DOWN, layer_idx, e), d * f, wl.sigma_w,
                           dn.data_ptr(), s)
        layer.load_expert(arena_layer, e, g, u, dn)


def bf16_residual(x, y):
    """bf16(x + y) for bf16 bit tensors (int16 views): the fp64 sum of two
    bf16 values is exact and is rounded once, to 8 significant bits with ties
    to even.  Used only to follow the chain for the traffic figure."""
    import torch
    v = x.view(torch.bfloat16).double() + y.view(torch.bfloat16).double()
    m, ex = torch.frexp(v)
    r = torch.ldexp(torch.round(m * 256.0), ex - 8)
    return r.to(torch.bfloat16).view(torch.int16)


def ep_share_section(steps):
    """One node's 4-of-16 expert-parallel share (experts 4s..4s+3, s = 0..3)
    at T = 1, 4, 8: routing from the full 16-way logits, only the local
    experts computed.  Each share holds 4 independently seeded layers and the
    timed steps rotate over them, so no weight byte is re-read within 1.5 GB
    (the 256 MB last-level cache cannot serve repeats).  Timed as HIP graph
    replays of the 4 rotating layers (direct launches reported beside)."""
    import torch
    import moe_inputs as mi
    import paper_2506_23635_amd as moe
    sw = mi.WORKLOADS["ep_share"]
    n_rot = 4
    expert_bytes = 3 * sw.d * sw.f * 2
    rows = []
    for s in range(4):
        cfg = moe.make_config(sw.d, sw.f, sw.E, sw.k, expert_begin=4 * s, n_local_experts=4,
                              n_layers=n_rot, max_tokens=8)
        pool_reset()
        layer = pool_layer(cfg)
        staging = staging_buffer(sw)
        for li in range(n_rot):
            load_layer_device(layer, sw, li, li, staging)
        torch.cuda.synchronize()
        for T in (1, 4, 8):
            x = torch.empty(T * sw.d, dtype=torch.int16, device="cuda")
            mi.gen_bf16_device(sw.seed, mi.stream_id(mi.KIND_X), T * sw.d, sw.sigma_x, x.data_ptr(),
                               layer.stream)
            x = x.view(T, sw.d)
            y = torch.empty((T, sw.d), dtype=torch.int16, device="cuda")
            touched = []
            for li in range(n_rot):
                rt = layer.routing_tensors(layer.route(li, x))
                touched.append(int((rt["counts"][4 * s: 4 * s + 4] > 0).sum()))
            for i in range(2 * n_rot):
                layer.forward(i % n_rot, x, y)
            torch.cuda.synchronize()
            n = steps - steps % n_rot
            t0 = time.perf_counter()
            for i in range(n):
                layer.forward(i % n_rot, x, y)
            torch.cuda.synchronize()
            ms_direct = (time.perf_counter() - t0) * 1e3 / n

            def step():
                for li in range(n_rot):
                    layer.forward(li, x, y)

            # one replay runs the 4 rotating layers
            ms = graph_ms(step, max(n // n_rot, 5), 2) / n_rot
            bytes_step = sum(touched) / n_rot * expert_bytes + sw.d * sw.E * 4
            # the rate over the layers that touch a local expert: a layer with
            # none (routing and combine only, no weights) is timed alone, as
            # its own graph, and its time taken out
            idle_ms = 0.0
            for li in range(n_rot):
                if touched[li] == 0:
                    idle_ms += graph_ms(lambda li=li: layer.forward(li, x, y), 40, 5)
            busy = [li for li in range(n_rot) if touched[li] > 0]
            busy_ms = ms * n_rot - idle_ms
            rows.append({"share": s, "experts": [4 * s, 4 * s + 3], "T": T,
                         "local_experts_touched": touched, "us_per_step": ms * 1e3,
                         "us_per_step_direct_launch": ms_direct * 1e3,
                         "hbm_gbs": (bytes_step / (ms * 1e-3) / 1e9) if sum(touched) else None,
                         "hbm_gbs_touched_layers":
                             ((sum(touched) * expert_bytes + len(busy) * sw.d * sw.E * 4)
                              / (busy_ms * 1e-3) / 1e9) if busy else None})
            log(f"ep share {s} T={T}: {ms * 1e3:.1f} us graph, {ms_direct * 1e3:.1f} direct, touched {touched}")
        layer.close()
        del layer, staging
    torch.cuda.empty_cache()
    return rows


def stack_section(steps, warmup):
    """32 chained layers, all 16 experts of every layer resident (203 GB), 4
    decode tokens: moe_forward_stack timed as HIP graph replays."""
    import torch
    import moe_inputs as mi
    import paper_2506_23635_amd as moe
    sw = mi.WORKLOADS["stack"]
    expert_bytes = 3 * sw.d * sw.f * 2
    cfg = moe.make_config(sw.d, sw.f, sw.E, sw.k, n_layers=sw.n_layers, max_tokens=sw.T)
    need = section_bytes(cfg, sw)
    have = _POOL.numel() if _POOL is not None else torch.cuda.mem_get_info()[0] - (8 << 30)
    if have < need:
        log(f"stack: skipped ({have / 1e9:.0f} GB available, {need / 1e9:.0f} GB needed)")
        return None
    pool_reset()
    layer = pool_layer(cfg)
    staging = staging_buffer(sw)
    t0 = time.perf_counter()
    for li in range(sw.n_layers):
        load_layer_device(layer, sw, li, li, staging)
    torch.cuda.synchronize()
    log(f"stack: 32 layers generated and prestacked in {time.perf_counter() - t0:.1f} s")
    del staging
    x0 = torch.empty(sw.T * sw.d, dtype=torch.int16, device="cuda")
    mi.gen_bf16_device(sw.seed, mi.stream_id(mi.KIND_X), sw.T * sw.d, sw.sigma_x, x0.data_ptr(),
                       layer.stream)
    x0 = x0.view(sw.T, sw.d)
    # touched experts per layer along the chain (for the traffic figure)
    touched = []
    cur = x0.clone()
    y = torch.empty_like(cur)
    for li in range(sw.n_layers):
        rt = layer.routing_tensors(layer.route(li, cur))
        touched.append(int((rt["counts"] > 0).sum()))
        layer.forward(li, cur, y)
        cur = bf16_residual(cur, y)
    xs = x0.clone()

    def step():
        xs.copy_(x0)
        layer.forward_stack(xs)

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        step()
    torch.cuda.synchronize()
    ms_direct = (time.perf_counter() - t0) * 1e3 / steps
    ms_graph = graph_ms(step, steps, warmup)
    ms = ms_graph
    bytes_step = sum(touched) * expert_bytes + sw.n_layers * sw.d * sw.E * 4
    out = {"workload": "dbrx_moe_stack_32_layers", "T": sw.T, "n_layers": sw.n_layers,
           "resident_gb": sw.n_layers * sw.E * expert_bytes / 1e9,
           "ms_per_step": ms, "ms_per_step_direct_launch": ms_direct,
           "tokens_per_s": sw.T / (ms * 1e-3), "touched_experts_per_layer": touched,
           "hbm_gb_per_step": bytes_step / 1e9, "hbm_gbs": bytes_step / (ms * 1e-3) / 1e9,
           "hbm_frac": bytes_step / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS}
    log(f"stack: {ms:.2f} ms/step graph, {ms_direct:.2f} direct, {out['hbm_gbs']:.0f} GB/s")
    layer.close()
    del layer, x0, xs, cur, y
    torch.cuda.empty_cache()
    return out


DECODER_LAYERS = 40     # DBRX's layer count (Table tab:vars)
DECODER_PROMPT = 2048   # the long-prompt workload's prompt (2000 tokens), rounded


def decoder_bytes():
    """Pool bytes of the decoder section: the 40 MoE layers' arena and
    workspace, the 40 attention layers' arena, cache and workspace, and the
    staging buffers."""
    import moe_inputs as mi
    import paper_2506_23635_amd as moe
    sw = mi.WORKLOADS["stack"].with_(n_layers=DECODER_LAYERS, T=1)
    aw = mi.ATTN_WORKLOADS["attn_decode"]
    mcfg = moe.make_config(sw.d, sw.f, sw.E, sw.k, n_layers=DECODER_LAYERS,
                           max_tokens=DECODER_PROMPT)
    acfg = moe.make_attn_config(aw.d, aw.n_heads, aw.n_kv, aw.hd, n_layers=DECODER_LAYERS,
                                max_seq=aw.max_seq, max_tokens=DECODER_PROMPT,
                                rope_theta=aw.theta, norm_eps=aw.eps)
    return (section_bytes(mcfg, sw) + 2 * DECODER_PROMPT * aw.d * 2 + moe.attn_weight_bytes(acfg) + moe.attn_cache_bytes(acfg) +
            moe.attn_workspace_bytes(acfg) + (aw.d * aw.nqkv + aw.n_heads * aw.hd * aw.d) * 2 +
            (64 << 20))


def decoder_section(steps, warmup):
    """A whole DBRX-shaped decoder on one GPU: 40 layers, each as DBRX
    arranges it -- norm, self-attention (one token after 2047 cached
    positions) and residual, norm, the 16-expert MoE layer and residual
    (attn_forward_norm, moe_forward_residual) -- every weight resident
    (254 GB of experts + 7 GB of attention).  One step is
    one generated token through all 40 layers; timed with direct launches
    and as HIP graph replays of the whole step.  HBM bytes per token: the
    touched experts (4 per layer at T = 1), the routers, and each layer's
    attention bytes (Wqkv, Wo, gamma, the 2048 positions' keys and values)."""
    import numpy as np
    import torch
    import moe_inputs as mi
    import paper_2506_23635_amd as moe
    sw = mi.WORKLOADS["stack"].with_(n_layers=DECODER_LAYERS, T=1)
    aw = mi.ATTN_WORKLOADS["attn_decode"]
    need = decoder_bytes()
    have = _POOL.numel() if _POOL is not None else 0
    if have < need:
        log(f"decoder: skipped ({have / 1e9:.0f} GB of pool, {need / 1e9:.0f} GB needed)")
        return None
    pool_reset()
    mcfg = moe.make_config(sw.d, sw.f, sw.E, sw.k, n_layers=DECODER_LAYERS,
                           max_tokens=DECODER_PROMPT)
    ffn = pool_layer(mcfg)
    acfg = moe.make_attn_config(aw.d, aw.n_heads, aw.n_kv, aw.hd, n_layers=DECODER_LAYERS,
                                max_seq=aw.max_seq, max_tokens=DECODER_PROMPT,
                                rope_theta=aw.theta, norm_eps=aw.eps)
    att = moe.AttnLayer(acfg, arena=pool_take(moe.attn_weight_bytes(acfg)),
                        cache=pool_take(moe.attn_cache_bytes(acfg)),
                        workspace=pool_take(moe.attn_workspace_bytes(acfg)))
    staging = staging_buffer(sw)
    stg = pool_take(aw.d * aw.nqkv * 2).view(torch.int16)
    stg2 = pool_take(aw.n_heads * aw.hd * aw.d * 2).view(torch.int16)
    s = ffn.stream
    t0 = time.perf_counter()
    for li in range(DECODER_LAYERS):
        load_layer_device(ffn, sw, li, li, staging)
        mi.gen_bf16_device(aw.seed, mi.stream_id(mi.KIND_WQKV, li), aw.d * aw.nqkv, aw.sigma_qkv,
                           stg.data_ptr(), s)
        mi.gen_bf16_device(aw.seed, mi.stream_id(mi.KIND_WO, li), aw.n_heads * aw.hd * aw.d,
                           aw.sigma_o, stg2.data_ptr(), s)
        att.load_layer(li, torch.from_numpy(aw.gamma(li)).cuda(), stg, stg2)
        att.load_post_norm(li, torch.from_numpy(aw.gamma2(li)).cuda())
        K, V = att.cache_views(li)
        mi.gen_bf16_device(aw.seed, mi.stream_id(mi.KIND_KCACHE, li), K.numel(), aw.sigma_cache,
                           K.data_ptr(), s)
        mi.gen_bf16_device(aw.seed, mi.stream_id(mi.KIND_VCACHE, li), V.numel(), aw.sigma_cache,
                           V.data_ptr(), s)
    torch.cuda.synchronize()
    log(f"decoder: {DECODER_LAYERS} layers generated and prestacked in {time.perf_counter() - t0:.1f} s")
    del staging, stg, stg2
    x0 = torch.from_numpy(aw.x().view(np.int16)).cuda()
    pos0 = aw.pos0
    # touched experts per layer along the chain; a layer is DBRX's: y =
    # x + attention(norm1(x)), z = norm2(y), x = y + moe(z)
    touched = []
    x = x0.clone()
    z = torch.empty_like(x)
    for li in range(DECODER_LAYERS):
        att.forward_norm(li, x, x, z, pos0)
        rt = ffn.routing_tensors(ffn.route(li, z))
        touched.append(int((rt["counts"] > 0).sum()))
        ffn.forward_residual(li, z, x)
    torch.cuda.synchronize()
    out_bits = x.cpu().numpy().view(np.uint16)
    finite = bool(np.isfinite(mi.bf16_bits_to_f32(out_bits)).all())

    def step():
        x.copy_(x0)
        for li in range(DECODER_LAYERS):
            att.forward_norm(li, x, x, z, pos0)
            ffn.forward_residual(li, z, x)

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        step()
    torch.cuda.synchronize()
    ms_direct = (time.perf_counter() - t0) * 1e3 / steps
    ms_graph = graph_ms(step, steps, warmup)
    ms = min(ms_direct, ms_graph)
    expert_bytes = 3 * sw.d * sw.f * 2
    attn_b = (aw.d * aw.nqkv * 2 + aw.n_heads * aw.hd * aw.d * 2 + aw.d * 4 +
              2 * aw.n_kv * (pos0 + 1) * aw.hd * 2)
    bytes_tok = sum(touched) * expert_bytes + DECODER_LAYERS * (sw.d * sw.E * 4 + attn_b)
    out = {"workload": "dbrx_decoder_40_layers", "T": 1, "context": pos0 + 1,
           "n_layers": DECODER_LAYERS,
           "resident_gb": (DECODER_LAYERS * sw.E * expert_bytes + moe.attn_weight_bytes(acfg)) / 1e9,
           "ms_per_token": ms, "ms_graph": ms_graph, "ms_direct_launch": ms_direct,
           "tokens_per_s": 1e3 / ms, "touched_experts_per_layer": touched,
           "hbm_gb_per_token": bytes_tok / 1e9, "hbm_gbs": bytes_tok / (ms * 1e-3) / 1e9,
           "hbm_frac": bytes_tok / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS, "output_finite": finite}
    log(f"decoder: {ms:.2f} ms/token ({1e3 / ms:.1f} tok/s), graph {ms_graph:.2f}, "
        f"direct {ms_direct:.2f}, {out['hbm_gbs']:.0f} GB/s")
    # prompt evaluation: a 2048-token prompt from an empty cache through all
    # 40 layers (attention on the prefill path, the MoE on the grouped GEMM)
    P = DECODER_PROMPT
    xp0 = pool_take(P * aw.d * 2).view(torch.int16).view(P, aw.d)
    mi.gen_bf16_device(aw.seed, mi.stream_id(mi.KIND_ATTN_X, 1), P * aw.d, aw.sigma_x,
                       xp0.data_ptr(), s)
    xp = xp0.clone()
    zp = pool_take(P * aw.d * 2).view(torch.int16).view(P, aw.d)

    def prompt():
        xp.copy_(xp0)
        for li in range(DECODER_LAYERS):
            att.forward_norm(li, xp, xp, zp, 0)
            ffn.forward_residual(li, zp, xp)

    prompt()
    torch.cuda.synchronize()
    n_pr = 3
    t0 = time.perf_counter()
    for _ in range(n_pr):
        prompt()
    torch.cuda.synchronize()
    ms_prompt = (time.perf_counter() - t0) * 1e3 / n_pr
    pf = np.isfinite(mi.bf16_bits_to_f32(xp.cpu().numpy().view(np.uint16))).all()
    attn_f = (2.0 * P * aw.d * aw.nqkv + 2.0 * P * aw.n_heads * aw.hd * aw.d +
              4.0 * aw.n_heads * aw.hd * P * (P + 1) / 2)
    moe_f = 2.0 * P * sw.k * 3 * sw.d * sw.f
    pflops = DECODER_LAYERS * (attn_f + moe_f)
    out["prompt"] = {"T": P, "ms_per_prompt": ms_prompt, "tokens_per_s": P / (ms_prompt * 1e-3),
                     "tflops": pflops / (ms_prompt * 1e-3) / 1e12,
                     "mfma_frac": pflops / (ms_prompt * 1e-3) / 1e12 / MFMA_BF16_PEAK_TFLOPS,
                     "output_finite": bool(pf)}
    log(f"decoder prompt: {ms_prompt:.1f} ms for {P} tokens ({P / (ms_prompt * 1e-3):.0f} tok/s, "
        f"{out['prompt']['tflops']:.0f} TFLOP/s)")
    ffn.close()
    att.close()
    del ffn, att, x, x0, z, xp, xp0, zp
    return out


def gemm_timeline(layer, x):
    """One forward with the per-workgroup GEMM timeline on
    (moe_profile_gemm_timeline), its two GEMMs also event-timed: for each
    grouped GEMM, the clock its tiles ran at (shader-clock cycles over the
    constant wall-clock counter, whose rate the runtime reports, so no
    profiler offset enters), the span, how busy the CUs were, the mean tile
    time per number of 64-row pairs, the gap between consecutive tiles on a
    CU, and the MFMA fraction against the spec peak and against the peak at
    the measured clock."""
    import numpy as np
    import torch
    import paper_2506_23635_amd as moe
    n = 8192
    bufs = [torch.zeros(n * 8, dtype=torch.int64, device="cuda") for _ in range(2)]
    y = torch.empty((x.shape[0], layer.cfg.d_model), dtype=torch.int16, device="cuda")
    layer.forward(0, x, y)
    torch.cuda.synchronize()
    moe.moe_profile_gemm_timeline(layer.ctx, bufs[0].data_ptr(), bufs[1].data_ptr(), n)
    moe.moe_profile_enable(layer.ctx, 16)
    layer.forward(0, x, y)
    torch.cuda.synchronize()
    prof, _ = moe.moe_profile_read(layer.ctx)
    moe.moe_profile_enable(layer.ctx, 0)
    moe.moe_profile_gemm_timeline(layer.ctx, None, None, 0)
    d, f = layer.cfg.d_model, layer.cfg.ffn_dim
    # the counter's rate from this launch: its ticks over the same GEMM's
    # event time (the runtime's wall-clock attribute does not describe this
    # counter on this part: it reports 30 MHz, the ticks run at 100 MHz)
    t0 = bufs[0].cpu().numpy().view(np.uint64).reshape(n, 8)
    t0 = t0[t0[:, 1] > 0]
    ev0 = prof["gemm_gateup"][0] / max(prof["gemm_gateup"][1], 1) * 1e-3
    hz = float(t0[:, 1].max() - t0[:, 0].min()) / ev0
    out = {"counter_mhz": hz / 1e6}
    for name, buf, K in (("gemm_gateup", bufs[0], d), ("gemm_down", bufs[1], f)):
        t = buf.cpu().numpy().view(np.uint64).reshape(n, 8)
        t = t[t[:, 1] > 0]
        r0, r1 = t[:, 0].astype(np.int64), t[:, 1].astype(np.int64)
        c0, c1 = t[:, 2].astype(np.int64), t[:, 3].astype(np.int64)
        hw, xcc = t[:, 4] & 0xFFFFFFFF, t[:, 4] >> 32
        rows = ((t[:, 5] >> 32) & 0xFFFF).astype(np.int64)
        cu = (xcc << 8) | ((hw >> 8) & 0xFF)
        tick_us = 1e6 / hz
        dur_us = (r1 - r0) * tick_us
        span_us = (r1.max() - r0.min()) * tick_us
        n_cu = len(np.unique(cu))
        clock = (c1 - c0).sum() / ((r1 - r0).sum() / hz) / 1e9
        per_wg_clock = (c1 - c0) / ((r1 - r0) / hz) / 1e9
        gaps = []
        for u in np.unique(cu):
            sel = np.nonzero(cu == u)[0]
            order = sel[np.argsort(r0[sel])]
            gaps.extend(((r0[order[1:]] - r1[order[:-1]]) * tick_us).tolist())
        pairs = (rows + 63) // 64
        flops = float(rows.sum()) * 256 * K * 2        # each workgroup: rows x 256 features x K
        ev_ms = prof[name][0] / max(prof[name][1], 1)
        tf = flops / (ev_ms * 1e-3) / 1e12
        out[name] = {
            "workgroups": int(len(t)), "cus": int(n_cu), "span_us": float(span_us),
            "event_us": ev_ms * 1e3,
            "clock_ghz": float(clock), "clock_ghz_p5_p95": [float(np.percentile(per_wg_clock, 5)),
                                                            float(np.percentile(per_wg_clock, 95))],
            "cu_busy_frac": float(dur_us.sum() / (n_cu * span_us)),
            "tile_us_by_pairs": {int(p): float(dur_us[pairs == p].mean()) for p in np.unique(pairs)},
            "tiles_by_pairs": {int(p): int((pairs == p).sum()) for p in np.unique(pairs)},
            "gap_us_mean": float(np.mean(gaps)) if gaps else 0.0,
            "tflops": tf, "mfma_frac": tf / MFMA_BF16_PEAK_TFLOPS,
            "mfma_frac_at_clock": tf / (MFMA_BF16_PEAK_TFLOPS * clock / 2.4),
        }
    del bufs
    return out


def attn_section(steps, warmup, n_rot=N_ROT):
    """The DBRX self-attention block on one decode token after 2047 cached
    positions (the paper's long-prompt workload has 2000 input tokens): layer
    norm, fused projection (D_qkv_hidden 8192), rotary encoding and cache
    append, attention over 2048 positions, output projection and residual.
    n_rot independently seeded layers, step i on layer i % n_rot, so no
    weight byte is re-read within 0.5 GB.  HBM bytes per step: Wqkv + Wo +
    gamma + the keys and values of the 2048 positions + x and y."""
    import numpy as np
    import torch
    import moe_inputs as mi
    import paper_2506_23635_amd as moe
    wl = mi.ATTN_WORKLOADS["attn_decode"]
    cfg = moe.make_attn_config(wl.d, wl.n_heads, wl.n_kv, wl.hd, n_layers=n_rot,
                               max_seq=wl.max_seq, max_tokens=16, rope_theta=wl.theta,
                               norm_eps=wl.eps)
    pool_reset()
    layer = moe.AttnLayer(cfg, arena=pool_take(moe.attn_weight_bytes(cfg)),
                          cache=pool_take(moe.attn_cache_bytes(cfg)),
                          workspace=pool_take(moe.attn_workspace_bytes(cfg)))
    s = layer.stream
    stg = pool_take(wl.d * wl.nqkv * 2).view(torch.int16)
    stg2 = pool_take(wl.n_heads * wl.hd * wl.d * 2).view(torch.int16)
    for li in range(n_rot):
        mi.gen_bf16_device(wl.seed, mi.stream_id(mi.KIND_WQKV, li), wl.d * wl.nqkv, wl.sigma_qkv,
                           stg.data_ptr(), s)
        mi.gen_bf16_device(wl.seed, mi.stream_id(mi.KIND_WO, li), wl.n_heads * wl.hd * wl.d,
                           wl.sigma_o, stg2.data_ptr(), s)
        layer.load_layer(li, torch.from_numpy(wl.gamma(li)).cuda(), stg, stg2)
        K, V = layer.cache_views(li)
        mi.gen_bf16_device(wl.seed, mi.stream_id(mi.KIND_KCACHE, li), K.numel(), wl.sigma_cache,
                           K.data_ptr(), s)
        mi.gen_bf16_device(wl.seed, mi.stream_id(mi.KIND_VCACHE, li), V.numel(), wl.sigma_cache,
                           V.data_ptr(), s)
    x = torch.from_numpy(wl.x().view(np.int16)).cuda()
    y = torch.empty_like(x)
    torch.cuda.synchronize()
    pos0 = wl.pos0
    for i in range(max(warmup, n_rot)):
        layer.forward(i % n_rot, x, y, pos0)
    torch.cuda.synchronize()
    n = max(steps - steps % n_rot, n_rot)
    t0 = time.perf_counter()
    for i in range(n):
        layer.forward(i % n_rot, x, y, pos0)
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1e3 / n

    def step():
        for li in range(n_rot):
            layer.forward(li, x, y, pos0)

    ms_graph = graph_ms(step, max(n // n_rot, 5), 2) / n_rot
    moe.attn_profile_enable(layer.ctx, 8 * n + 8)
    for i in range(n):
        layer.forward(i % n_rot, x, y, pos0)
    torch.cuda.synchronize()
    prof, _ = moe.attn_profile_read(layer.ctx)
    moe.attn_profile_enable(layer.ctx, 0)
    kern = {k: v[0] / v[1] * 1e3 for k, v in prof.items() if v[1]}
    wqkv_b, wo_b = wl.d * wl.nqkv * 2, wl.n_heads * wl.hd * wl.d * 2
    kv_b = 2 * wl.n_kv * (pos0 + 1) * wl.hd * 2
    step_b = wqkv_b + wo_b + wl.d * 4 + kv_b + 2 * wl.d * 2
    # the projection's own bytes: Wqkv, x and gamma (it forms the norm
    # itself at T = 1) and the bf16 q, k, v it writes
    qkv_b = wqkv_b + wl.d * 2 + wl.d * 4 + wl.nqkv * 2
    best = min(ms, ms_graph)
    out = {"workload": "dbrx_attention_decode", "T": 1, "context": pos0 + 1,
           "rotation_layers": n_rot, "us_per_layer": best * 1e3, "us_direct_launch": ms * 1e3,
           "us_graph": ms_graph * 1e3, "hbm_bytes_per_step": step_b,
           "hbm_gbs": step_b / (best * 1e-3) / 1e9,
           "hbm_frac": step_b / (best * 1e-3) / 1e9 / HBM_PEAK_GBS, "kernels_us": kern,
           "roofline": {"bound": "hbm", "kernel": "qkv", "achieved": qkv_b / (kern["qkv"] * 1e-6) / 1e9,
                        "peak": HBM_PEAK_GBS, "unit": "GB/s",
                        "frac": qkv_b / (kern["qkv"] * 1e-6) / 1e9 / HBM_PEAK_GBS,
                        "traffic": measured_traffic("attn_qkv", "attn.hip"),
                        "algorithmic_bytes": qkv_b}}
    log(f"attention decode: {best * 1e3:.1f} us/layer ({out['hbm_gbs']:.0f} GB/s), kernels {kern}")
    layer.close()
    del layer, stg, stg2, x, y
    return out


def attn_prefill_section(steps, warmup, n_rot=N_ROT, T=2048):
    """The DBRX self-attention block on a 2048-token prompt from an empty
    cache (the long-prompt workload's prompt evaluation): norm, the q|k|v
    and output projections on the grouped GEMM (matrix cores), rotation and
    cache append, causal attention on the matrix cores, residual.  n_rot
    seeded layers in turn.  FLOPs per step: the two projections
    (2 T d (H + 2G) hd + 2 T H hd d) and the causal attention
    (4 H hd sum_t (t + 1), scores and P V)."""
    import numpy as np
    import torch
    import moe_inputs as mi
    import paper_2506_23635_amd as moe
    aw = mi.ATTN_WORKLOADS["attn_decode"].with_(T=T, pos0=0)
    cfg = moe.make_attn_config(aw.d, aw.n_heads, aw.n_kv, aw.hd, n_layers=n_rot,
                               max_seq=aw.max_seq, max_tokens=T, rope_theta=aw.theta,
                               norm_eps=aw.eps)
    pool_reset()
    layer = moe.AttnLayer(cfg, arena=pool_take(moe.attn_weight_bytes(cfg)),
                          cache=pool_take(moe.attn_cache_bytes(cfg)),
                          workspace=pool_take(moe.attn_workspace_bytes(cfg)))
    s = layer.stream
    stg = pool_take(aw.d * aw.nqkv * 2).view(torch.int16)
    stg2 = pool_take(aw.n_heads * aw.hd * aw.d * 2).view(torch.int16)
    for li in range(n_rot):
        mi.gen_bf16_device(aw.seed, mi.stream_id(mi.KIND_WQKV, li), aw.d * aw.nqkv, aw.sigma_qkv,
                           stg.data_ptr(), s)
        mi.gen_bf16_device(aw.seed, mi.stream_id(mi.KIND_WO, li), aw.n_heads * aw.hd * aw.d,
                           aw.sigma_o, stg2.data_ptr(), s)
        layer.load_layer(li, torch.from_numpy(aw.gamma(li)).cuda(), stg, stg2)
    x = torch.from_numpy(aw.x().view(np.int16)).cuda()
    y = torch.empty_like(x)
    torch.cuda.synchronize()
    for i in range(max(warmup, n_rot)):
        layer.forward(i % n_rot, x, y, 0)
    torch.cuda.synchronize()
    n = max(steps - steps % n_rot, n_rot)
    t0 = time.perf_counter()
    for i in range(n):
        layer.forward(i % n_rot, x, y, 0)
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1e3 / n
    moe.attn_profile_enable(layer.ctx, 8 * n + 8)
    for i in range(n):
        layer.forward(i % n_rot, x, y, 0)
    torch.cuda.synchronize()
    prof, _ = moe.attn_profile_read(layer.ctx)
    moe.attn_profile_enable(layer.ctx, 0)
    kern = {k: v[0] / v[1] for k, v in prof.items() if v[1]}
    d, nq, nqkv = aw.d, aw.n_heads * aw.hd, aw.nqkv
    f_qkv = 2.0 * T * d * nqkv
    f_out = 2.0 * T * nq * d
    f_att = 4.0 * aw.n_heads * aw.hd * (T * (T + 1) / 2)
    flops = f_qkv + f_out + f_att
    out = {"workload": "dbrx_attention_prefill", "T": T, "context": T, "rotation_layers": n_rot,
           "ms_per_layer": ms, "tokens_per_s": T / (ms * 1e-3), "tflops": flops / (ms * 1e-3) / 1e12,
           "mfma_frac": flops / (ms * 1e-3) / 1e12 / MFMA_BF16_PEAK_TFLOPS,
           "kernels_ms": kern,
           "roofline": {"bound": "mfma", "kernel": "qkv", "achieved": f_qkv / (kern["qkv"] * 1e-3) / 1e12,
                        "peak": MFMA_BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                        "frac": f_qkv / (kern["qkv"] * 1e-3) / 1e12 / MFMA_BF16_PEAK_TFLOPS,
                        "algorithmic_flops": f_qkv},
           "attention_core_tflops": f_att / (kern["score"] * 1e-3) / 1e12}
    log(f"attention prefill: {ms:.3f} ms/layer ({out['tflops']:.0f} TFLOP/s), kernels "
        f"{ {k: round(v, 3) for k, v in kern.items()} }")
    layer.close()
    del layer, stg, stg2, x, y
    return out


def stream_read_gbs(nbytes=4 << 30, reps=20):
    """GB/s of the library's plain streaming read (moe_diag_stream_read) over
    a 4 GiB buffer, far past the 256 MB last-level cache: the achievable HBM
    read rate, reported beside the 8 TB/s spec peak."""
    import torch
    import paper_2506_23635_amd as moe
    pool_reset()
    buf = pool_take(nbytes)
    out = torch.zeros(4 * moe.DIAG_MAX_WG, dtype=torch.int32, device="cuda")
    s = torch.cuda.current_stream().cuda_stream
    for _ in range(3):
        moe.moe_diag_stream_read(buf.data_ptr(), nbytes, out.data_ptr(), s)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        moe.moe_diag_stream_read(buf.data_ptr(), nbytes, out.data_ptr(), s)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    del buf, out
    torch.cuda.empty_cache()
    return nbytes / (ms * 1e-3) / 1e9


def measured_traffic(kernel="decode_gateup", source="moe_decode.hip"):
    """HBM bytes per launch of the dominant kernel from the committed counter
    summary (raw fabric read/write requests), or None when the kernel source
    has changed since those counters were taken."""
    import hashlib
    path = os.path.join(ROOT, "profiles", "dbrx_moe_layer_counters.txt")
    src = os.path.join(ROOT, "paper_2506_23635_amd", "csrc", source)
    if not (os.path.exists(path) and os.path.exists(src)):
        return None
    digest = hashlib.sha256(open(src, "rb").read()).hexdigest()
    for line in open(path):
        f = line.split()
        if len(f) >= 10 and f[0] == "traffic_bytes_per_launch" and f[1] == kernel:
            return int(f[2]) if f[-1] == digest else None
    return None


def cpu_baseline(wl, budget_s=10.0):
    """The fp64 oracle on the decode token of the workload, repeated for about
    budget_s seconds of host time (weights generated before the clock)."""
    import numpy as np
    import moe_inputs as mi
    import oracle
    x = wl.x()
    lg = oracle.router_logits(x, wl.router())
    idx, _ = oracle.route_from_logits(lg, wl.k)
    used = sorted(set(idx.reshape(-1).tolist()))
    G = [None] * wl.E
    U = [None] * wl.E
    D = [None] * wl.E
    for e in used:
        G[e], U[e], D[e] = wl.gate(e), wl.up(e), wl.down(e)
    wr = wl.router()
    reps = 0
    t0 = time.perf_counter()
    while True:
        oracle.layer(x, wr, wl.bias(), G, U, D, wl.k)
        reps += 1
        el = time.perf_counter() - t0
        if el >= budget_s or reps >= 1000:
            break
    omp = os.environ.get("OMP_NUM_THREADS")
    threads = int(omp or 0) or os.cpu_count()
    assert np.isfinite(el)
    return {"value": reps * wl.T / el, "unit": "tokens/s", "cores": threads, "kind": "oracle",
            "cpu_model": cpu_model(), "omp_num_threads": omp, "nproc": os.cpu_count(),
            "sample": f"decode token (T={wl.T}) through the full 16-expert layer, {reps} "
                      f"repetitions, {el:.1f} s of host time, fp64 oracle with OpenMP"}


def cpu_model():
    try:
        with open("/proc/cpuinfo") as fh:
            return next((ln.split(":", 1)[1].strip() for ln in fh if ln.startswith("model name")),
                        "")
    except OSError:
        return ""


def cpu_oracle_all():
    """The fp64 oracle on the host cores for every workload, input generation
    excluded from the clock: the small layer, the decode token, each
    expert-parallel share at T = 1, 4, 8, and bounded samples of the
    2048-token prefill layer and of the 32-layer stack (the whole of either
    takes far longer than a run here: the oracle is deliberately plain).
    A reported baseline, printed as one JSON line; no GPU is used."""
    import numpy as np
    import moe_inputs as mi
    import oracle
    out = {"metric": "fp64 oracle on the host cores (baseline only)", "cpu_model": cpu_model(),
           "nproc": os.cpu_count(), "omp_num_threads": os.environ.get("OMP_NUM_THREADS"),
           "workloads": {}}

    def experts(wl, ids, layer=0):
        G, U, D = [None] * wl.E, [None] * wl.E, [None] * wl.E
        for e in ids:
            G[e], U[e], D[e] = wl.gate(e, layer), wl.up(e, layer), wl.down(e, layer)
        return G, U, D

    def clock(fn, min_s=2.0, max_reps=50):
        reps, t0 = 0, time.perf_counter()
        while True:
            fn()
            reps += 1
            el = time.perf_counter() - t0
            if el >= min_s or reps >= max_reps:
                return el / reps, reps

    def row(name, T, sec, reps, sample, **kw):
        out["workloads"][name] = {"T": T, "s_per_call": sec, "tokens_per_s": T / sec,
                                  "reps": reps, "sample": sample, **kw}
        log(f"oracle {name}: {sec:.3f} s per call")

    wl = mi.WORKLOADS["tiny"]
    x = wl.x()
    G, U, D = experts(wl, range(wl.E))
    sec, reps = clock(lambda: oracle.layer(x, wl.router(), wl.bias(), G, U, D, wl.k))
    row("tiny", wl.T, sec, reps, "the whole layer (16 tokens)")

    wl = mi.WORKLOADS["decode"]
    x, wr = wl.x(), wl.router()
    idx, _ = oracle.route_from_logits(oracle.router_logits(x, wr), wl.k)
    G, U, D = experts(wl, sorted(set(idx.reshape(-1).tolist())))
    sec, reps = clock(lambda: oracle.layer(x, wr, wl.bias(), G, U, D, wl.k), min_s=5.0)
    row("decode", 1, sec, reps, "the whole layer (1 token, 4 experts)")

    sw = mi.WORKLOADS["ep_share"]
    wr = sw.router()
    for s in range(4):
        G, U, D = experts(sw, range(4 * s, 4 * s + 4))
        for T in (1, 4, 8):
            x = mi.gen_bf16(sw.seed, mi.stream_id(mi.KIND_X), (T, sw.d), sw.sigma_x)
            idx, _ = oracle.route_from_logits(oracle.router_logits(x, wr), sw.k)
            touched = len({e for e in idx.reshape(-1).tolist() if 4 * s <= e < 4 * s + 4})
            sec, reps = clock(lambda: oracle.layer(x, wr, None, G, U, D, sw.k, e_begin=4 * s,
                                                   n_local=4), min_s=1.0, max_reps=10)
            row(f"ep_share{s}_T{T}", T, sec, reps, "the whole share (layer 0)",
                local_experts_touched=touched)

    wl = mi.WORKLOADS["prefill"]
    n = 64
    x = wl.x()[:n]
    idx, _ = oracle.route_from_logits(oracle.router_logits(x, wl.router(), wl.bias()), wl.k)
    G, U, D = experts(wl, sorted(set(idx.reshape(-1).tolist())))
    sec, reps = clock(lambda: oracle.layer(x, wl.router(), wl.bias(), G, U, D, wl.k), min_s=0.0,
                      max_reps=1)
    row("prefill", n, sec, reps, f"the first {n} of the 2048 tokens through the whole layer; "
        f"the full layer scales with the tokens (x {wl.T // n})")
    del G, U, D

    wl = mi.WORKLOADS["stack"]
    n_l = 8
    x = wl.x()
    sec = 0.0
    for li in range(n_l):
        wr = wl.router(li)
        idx, _ = oracle.route_from_logits(oracle.router_logits(x, wr), wl.k)
        G, U, D = experts(wl, sorted(set(idx.reshape(-1).tolist())), li)
        t0 = time.perf_counter()
        r = oracle.layer(x, wr, None, G, U, D, wl.k)
        x = oracle.residual_add(x, r["y"])
        sec += time.perf_counter() - t0
    row("stack", wl.T, sec * wl.n_layers / n_l, 1,
        f"the first {n_l} of the 32 layers, scaled to the step (x {wl.n_layers // n_l})")
    print(json.dumps(out), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--prefill-steps", type=int, default=20)
    ap.add_argument("--no-prefill", action="store_true")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-ep-share", action="store_true")
    ap.add_argument("--no-stack", action="store_true")
    ap.add_argument("--no-attn", action="store_true")
    ap.add_argument("--no-decoder", action="store_true")
    ap.add_argument("--attn-only", action="store_true",
                    help="time only the attention block (for profiling)")
    ap.add_argument("--stack-steps", type=int, default=20)
    ap.add_argument("--prefill-only", action="store_true",
                    help="time only the prefill layer (for counter collection)")
    ap.add_argument("--timeline", action="store_true",
                    help="with --prefill-only: also record the per-workgroup GEMM timeline")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="also run one 1 GiB device copy of known size (counter calibration)")
    ap.add_argument("--cpu-oracle-all", action="store_true",
                    help="only time the fp64 oracle on every workload on the host (no GPU)")
    args = ap.parse_args()
    if args.cpu_oracle_all:
        cpu_oracle_all()
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU only: this build has no multi-GPU path "
              f"(--gpus {args.gpus} requested)", file=sys.stderr)
        sys.exit(2)

    import torch
    import moe_inputs as mi
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    import paper_2506_23635_amd as moe
    moe.lib()   # raises if the HIP library is not built

    # the device pool, sized for the largest section that will run
    def cfg_of(w, **kw):
        return moe.make_config(w.d, w.f, w.E, w.k, **kw)
    dw, pw0, sw0, kw0 = (mi.WORKLOADS[n] for n in ("decode", "prefill", "ep_share", "stack"))
    sizes = [4 << 30, 2 << 30,
             section_bytes(cfg_of(dw, max_tokens=dw.T, n_layers=N_ROT), dw)]
    if not args.no_prefill or args.prefill_only:
        sizes.append(section_bytes(cfg_of(pw0, max_tokens=pw0.T), pw0))
    if not args.no_ep_share:
        sizes.append(section_bytes(cfg_of(sw0, expert_begin=0, n_local_experts=4, n_layers=4,
                                          max_tokens=8), sw0))
    if not args.no_stack and not args.prefill_only:
        stack_need = section_bytes(cfg_of(kw0, n_layers=kw0.n_layers, max_tokens=kw0.T), kw0)
        if stack_need + (8 << 30) <= torch.cuda.mem_get_info()[0]:
            sizes.append(stack_need)
    if not args.no_decoder and not args.prefill_only and not args.attn_only:
        dec_need = decoder_bytes()
        if dec_need + (8 << 30) <= torch.cuda.mem_get_info()[0]:
            sizes.append(dec_need)
    pool_init(max(sizes))

    if args.calibrate_copy:
        pool_reset()
        src, dst = pool_take(1 << 30), pool_take(1 << 30)
        dst.copy_(src)          # reads 1 GiB, writes 1 GiB
        pool_reset()
    if args.attn_only:
        print(json.dumps({"attention": attn_section(args.steps, args.warmup),
                          "attention_prefill": attn_prefill_section(8, 2)}), flush=True)
        pool_release()
        return
    if args.prefill_only:
        pw = mi.WORKLOADS["prefill"]
        player, px = setup_layer(pw, max_tokens=pw.T)
        pms, pkern, prt, _ = time_layer(player, px, args.prefill_steps, 2)
        rows = int(prt["offsets"][-1])
        tl = None
        if args.timeline:
            # after a pause, then back to back: the clock the power
            # controller grants moves from one GEMM to the next
            time.sleep(1.0)
            tl = [gemm_timeline(player, px) for _ in range(5)]
        print(json.dumps({"prefill_ms": pms, "tflops": 2.0 * rows * 3 * pw.d * pw.f / (pms * 1e-3) / 1e12,
                          "kernels_ms": {k: v["ms_per_launch"] for k, v in pkern.items()},
                          "timeline": tl}),
              flush=True)
        player.close()
        del player, px
        pool_release()
        return

    wl = mi.WORKLOADS["decode"]
    log(f"setup decode layers ({N_ROT} seeded copies of the 16-expert layer, "
        f"{N_ROT * 6.34:.0f} GB) ...")
    layer, x = setup_rotation(wl, N_ROT, max_tokens=wl.T)
    log("timing decode ...")
    # the step time comes from a region without per-kernel events (each event
    # pair adds a few microseconds to a ~0.24 ms step); a second timed region
    # of the same steps brackets every kernel with events for the roofline.
    # Step i runs layer i % N_ROT.
    ms, _, rt, _ = time_layer(layer, x, args.steps, args.warmup, kernel_events=False, n_rot=N_ROT)
    ms_ev, kern, _, dropped = time_layer(layer, x, args.steps, 0, kernel_events=True, n_rot=N_ROT)
    touched_per_layer = []
    for li in range(N_ROT):
        rtl = layer.routing_tensors(layer.route(li, x))
        touched_per_layer.append(int((rtl["counts"] > 0).sum()))
    log(f"decode ms/step {ms:.4f} (with per-kernel events {ms_ev:.4f})")
    touched = sum(touched_per_layer) / N_ROT
    expert_bytes = 3 * wl.d * wl.f * 2
    gu_unit = 2 * wl.d * wl.f * 2                     # one touched expert's gate+up
    layer_bytes = touched * expert_bytes + wl.d * wl.E * 4 + 2 * wl.T * wl.d * 2
    us = ms * 1e3
    hbm_gbs = layer_bytes / (ms * 1e-3) / 1e9
    gu = kern["decode_gateup"]
    gu_bytes = touched * gu_unit + wl.T * wl.d * 2
    gu_gbs = gu_bytes / (gu["ms_per_launch"] * 1e-3) / 1e9
    layer.close()
    del layer, x
    log("timing the plain streaming read (4 GiB) ...")
    read_gbs = stream_read_gbs()
    log(f"streaming read {read_gbs:.0f} GB/s")

    prefill = None
    if not args.no_prefill:
        pw = mi.WORKLOADS["prefill"]
        log("setup prefill layer ...")
        player, px = setup_layer(pw, max_tokens=pw.T)
        log("timing prefill ...")
        pms, _, prt, _ = time_layer(player, px, args.prefill_steps, 3, kernel_events=False)
        _, pkern, _, _ = time_layer(player, px, args.prefill_steps, 0, kernel_events=True)
        rows = int(prt["offsets"][-1])
        flops = 2.0 * rows * 3 * pw.d * pw.f
        tflops = flops / (pms * 1e-3) / 1e12
        g1 = pkern["gemm_gateup"]
        g1_flops = 2.0 * rows * 2 * pw.d * pw.f
        log("prefill GEMM timeline ...")
        tl = gemm_timeline(player, px)
        prefill = {
            "timeline": tl,
            "workload": "dbrx_moe_layer_prefill", "T": pw.T, "tokens_per_s": pw.T / (pms * 1e-3),
            "ms_per_layer": pms, "tflops": tflops, "mfma_frac": tflops / MFMA_BF16_PEAK_TFLOPS,
            "expert_counts": prt["counts"].tolist(),
            "kernels_ms": {k: v["ms_per_launch"] for k, v in pkern.items()},
            "gemm_gateup_tflops": g1_flops / (g1["ms_per_launch"] * 1e-3) / 1e12,
        }
        player.close()
        del player, px
        torch.cuda.empty_cache()

    attention = None
    if not args.no_attn:
        log("timing the attention block (decode) ...")
        attention = attn_section(args.steps, args.warmup)
        log("timing the attention block (prefill) ...")
        attention["prefill"] = attn_prefill_section(8, 2)

    ep_share = None
    if not args.no_ep_share:
        log("timing the expert-parallel shares ...")
        ep_share = ep_share_section(args.steps)

    stack = None
    if not args.no_stack:
        log("setup and timing of the 32-layer stack ...")
        stack = stack_section(args.stack_steps, 3)

    decoder = None
    if not args.no_decoder:
        log("setup and timing of the 40-layer decoder ...")
        decoder = decoder_section(args.stack_steps, 3)

    cpu = None
    if not args.no_cpu_baseline:
        log("timing the CPU oracle ...")
        cpu = cpu_baseline(wl)

    # Eq. (eq:pm) for the full 40-layer DBRX on 1..8 MI355X from this GPU's
    # measured streaming and matrix rates (collective latency and link
    # bandwidth are assumed: one GPU cannot measure them)
    from paper_2506_23635_amd import perf_model, placement
    bw_meas = stack["hbm_gbs"] if stack else hbm_gbs
    tf_meas = prefill["tflops"] if prefill else MFMA_BF16_PEAK_TFLOPS * 0.4
    model = {"inputs": {"hbm_gbs_measured": bw_meas, "mfma_tflops_measured": tf_meas,
                        "collective_latency_s_assumed": 20e-6, "link_gbs_assumed": 150.0},
             "predictions": perf_model.mi355x_predictions(bw_meas, tf_meas),
             "placements": placement.mi355x_placement_predictions(bw_meas, tf_meas)}
    if decoder:
        # the one-GPU prediction beside the measured 40-layer decoder token
        # (the model leaves out the per-kernel fixed costs)
        pred = model["predictions"]["1"]["ms_per_token"]
        model["measured_1gpu"] = {"ms_per_token": decoder["ms_per_token"],
                                  "predicted_ms_per_token": pred,
                                  "measured_over_predicted": decoder["ms_per_token"] / pred}

    out = {
        "metric": METRIC,
        "value": wl.T / (ms * 1e-3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": "dbrx_moe_layer_decode", "T": wl.T, "d_model": wl.d,
                   "ffn_dim": wl.f, "n_experts": wl.E, "top_k": wl.k, "parallelism": "none"},
        "us_per_layer": us,
        "hbm_gbs": hbm_gbs,
        "hbm_frac": hbm_gbs / HBM_PEAK_GBS,
        "hbm_read_ceiling_gbs": read_gbs,
        "hbm_frac_of_ceiling": hbm_gbs / read_gbs,
        "touched_experts": touched,
        "decode_rotation_layers": N_ROT,
        "roofline": {"bound": "hbm", "kernel": "decode_gateup", "achieved": gu_gbs,
                     "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": gu_gbs / HBM_PEAK_GBS,
                     "traffic": measured_traffic(), "algorithmic_bytes": gu_bytes},
        "kernels_us": {k: v["ms_per_launch"] * 1e3 for k, v in kern.items()},
        "ms_per_step_with_kernel_events": ms_ev,
        "profile_dropped": dropped,
        "cpu_baseline": cpu,
        "prefill": prefill,
        "ep_share": ep_share,
        "attention": attention,
        "stack": stack,
        "decoder": decoder,
        "perf_model": model,
    }
    pool_release()
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
