"""The C-ABI library on the host (no GPU needed): it loads, exports every
symbol include/moe.h declares, and rejects bad arguments with the documented
status codes before launching anything."""
import ctypes
import os
import re

import pytest

import paper_2506_23635_amd as moe

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADERS = [os.path.join(ROOT, "include", h) for h in ("moe.h", "attn.h")]

E_ARG, E_SHAPE, E_ALIGN, E_CAPACITY, E_STATE = -1, -2, -3, -4, -5


def declared_functions():
    text = "".join(open(h).read() for h in HEADERS)
    return sorted(set(re.findall(r"MOE_API\s+[\w\s\*]*?\b((?:moe|attn)_\w+)\s*\(", text)))


def test_header_declares_the_boundary():
    names = declared_functions()
    for must in ("moe_init", "moe_route", "moe_forward", "moe_load_expert", "moe_load_router",
                 "moe_weight_bytes", "moe_workspace_bytes", "moe_forward_stack", "moe_destroy",
                 "moe_last_error"):
        assert must in names
    assert sorted(moe.EXPORTED) == names


def test_library_exports_every_declared_symbol():
    lib = moe.lib()
    for name in declared_functions():
        assert hasattr(lib, name), name


def dbrx(**kw):
    base = dict(d_model=6144, ffn_dim=10752, n_experts=16, top_k=4, n_layers=1, max_tokens=2048)
    base.update(kw)
    return moe.make_config(**base)


def test_largest_max_tokens_accepted():
    # 174762 tokens of 6144 bf16 values stay below 2^31 bytes
    assert moe.moe_workspace_bytes(dbrx(max_tokens=174762)) > 0


def test_weight_bytes_formula():
    cfg = dbrx()
    expert = 3 * 6144 * 10752 * 2
    router = 6144 * 16 * 4 + 256
    assert moe.moe_weight_bytes(cfg) == 16 * expert + router
    share = dbrx(expert_begin=4, n_local_experts=4, n_layers=32)
    assert moe.moe_weight_bytes(share) == 32 * (4 * expert + router)
    assert moe.moe_workspace_bytes(cfg) > 2048 * 4 * (10752 * 2 + 6144 * 4)


@pytest.mark.parametrize("bad", [dict(d_model=100), dict(d_model=0), dict(ffn_dim=96),
                                 dict(n_experts=0), dict(n_experts=65), dict(top_k=0),
                                 dict(top_k=17), dict(expert_begin=13, n_local_experts=4),
                                 dict(n_layers=0), dict(max_tokens=0), dict(flags=2),
                                 dict(flags=-1),
                                 dict(max_tokens=174763), dict(ffn_dim=87424)])
def test_bad_configs_rejected(bad):
    # max_tokens 174763: x is then 2^31 bytes or more, past the GEMM's 32-bit gather offsets;
    # ffn_dim 87424: one expert's gate/up slab (4 * d * f bytes) is 2^31 bytes or more
    cfg = dbrx(**bad)
    if bad.get("n_experts") == 0:
        cfg.n_local_experts = 0
    assert moe.moe_weight_bytes(cfg) == 0
    assert moe.moe_workspace_bytes(cfg) == 0
    out = ctypes.c_void_p()
    rc = moe.lib().moe_init(ctypes.byref(cfg), 4096, 8192, ctypes.byref(out))
    assert rc == E_SHAPE and out.value is None
    assert moe.moe_last_error(None)


def test_partial_f32_flag_accepted():
    cfg = dbrx(expert_begin=4, n_local_experts=4, flags=moe.MOE_PARTIAL_F32)
    assert moe.moe_workspace_bytes(cfg) == moe.moe_workspace_bytes(dbrx(expert_begin=4,
                                                                        n_local_experts=4))


@pytest.mark.parametrize("kw", [dict(), dict(max_tokens=1), dict(expert_begin=4, n_local_experts=4),
                                dict(d_model=256, ffn_dim=512, n_experts=8, top_k=2, max_tokens=300)])
def test_workspace_map(kw):
    """Regions in declaration order, each inside the workspace, none
    overlapping, with the sizes the routing and intermediates need."""
    cfg = dbrx(**kw)
    m = moe.moe_workspace_map(cfg)
    total = moe.moe_workspace_bytes(cfg)
    assert list(m) == moe.WS_REGIONS
    end = 0
    for name in moe.WS_REGIONS:
        off, n = m[name]
        assert off >= end and off % 256 == 0 and n > 0, name
        end = off + n
    assert end <= total
    T, E, k, d, f = cfg.max_tokens, cfg.n_experts, cfg.top_k, cfg.d_model, cfg.ffn_dim
    rows = T * min(k, cfg.n_local_experts)
    assert m["logits"][1] == T * E * 4
    for name in ("topk_idx", "topk_w", "pair_row", "row_token"):
        assert m[name][1] == T * k * 4
    assert m["counts"][1] == E * 4 and m["offsets"][1] == (E + 1) * 4
    assert m["h"][1] == rows * f * 2 and m["o"][1] == rows * d * 4
    bad = dbrx(flags=2)
    with pytest.raises(moe.MoeError):
        moe.moe_workspace_map(bad)


def test_init_pointer_checks():
    cfg = moe.make_config(256, 512, 8, 2, max_tokens=16)
    out = ctypes.c_void_p()
    assert moe.lib().moe_init(ctypes.byref(cfg), None, 4096, ctypes.byref(out)) == E_ARG
    assert moe.lib().moe_init(ctypes.byref(cfg), 4096 + 16, 8192, ctypes.byref(out)) == E_ALIGN
    assert moe.lib().moe_init(ctypes.byref(cfg), 4096, 8192, None) == E_ARG


@pytest.fixture
def fake_ctx():
    # fake 256-aligned device addresses: nothing below ever dereferences them,
    # because every call here fails validation before launching
    cfg = moe.make_config(256, 512, 8, 2, expert_begin=2, n_local_experts=4, n_layers=2,
                          max_tokens=16)
    ctx = moe.moe_init(cfg, 1 << 20, 1 << 24)
    yield ctx
    moe.moe_destroy(ctx)


def rc_of(fn, *args):
    return getattr(moe.lib(), fn)(*args)


def test_ctx_validation_before_any_launch(fake_ctx):
    L = moe.lib()
    r = moe.MoeRouting()
    # layer out of range, router not loaded, capacity
    assert L.moe_route(fake_ctx, 2, 4096, 1, None, ctypes.byref(r), None) == E_ARG
    assert L.moe_route(fake_ctx, 0, 4096, 1, None, ctypes.byref(r), None) == E_STATE
    assert "router" in moe.moe_last_error(fake_ctx)
    assert L.moe_route(fake_ctx, 0, 4096, 17, None, ctypes.byref(r), None) == E_CAPACITY
    assert L.moe_route(fake_ctx, 0, 4096, -1, None, ctypes.byref(r), None) == E_ARG
    assert L.moe_route(fake_ctx, 0, 4096, 1, None, None, None) == E_ARG
    # forward before loading
    assert L.moe_forward(fake_ctx, 0, 4096, 1, None, 8192, None) == E_STATE
    assert L.moe_forward(fake_ctx, 5, 4096, 1, None, 8192, None) == E_ARG
    assert L.moe_forward(fake_ctx, 0, 4096, 99, None, 8192, None) == E_CAPACITY
    assert L.moe_forward_stack(fake_ctx, 4096, 1, None) == E_STATE
    assert L.moe_forward_layers(fake_ctx, 0, 1, 4096, 1, None) == E_STATE
    assert L.moe_forward_layers(fake_ctx, 1, 2, 4096, 1, None) == E_ARG      # past n_layers
    assert L.moe_forward_layers(fake_ctx, -1, 1, 4096, 1, None) == E_ARG
    assert L.moe_forward_layers(fake_ctx, 0, -1, 4096, 1, None) == E_ARG
    assert L.moe_forward_layers(fake_ctx, 0, 0, 4096, 1, None) == 0          # empty range
    assert L.moe_forward_layers(fake_ctx, 0, 1, 4096, 99, None) == E_CAPACITY
    assert L.moe_forward_residual(fake_ctx, 0, 4096, 8192, 1, None) == E_STATE
    assert L.moe_forward_residual(fake_ctx, 2, 4096, 8192, 1, None) == E_ARG
    assert L.moe_forward_residual(fake_ctx, 0, 4096, 8192, 99, None) == E_CAPACITY
    # experts outside the local range [2, 6), null and misaligned pointers
    assert L.moe_load_expert(fake_ctx, 0, 1, 4096, 4096, 4096, 1, None) == E_ARG
    assert L.moe_load_expert(fake_ctx, 0, 6, 4096, 4096, 4096, 1, None) == E_ARG
    assert L.moe_load_expert(fake_ctx, 2, 3, 4096, 4096, 4096, 1, None) == E_ARG
    assert L.moe_load_expert(fake_ctx, 0, 3, None, 4096, 4096, 1, None) == E_ARG
    assert L.moe_load_expert(fake_ctx, 0, 3, 4096 + 2, 4096, 4096, 1, None) == E_ALIGN
    assert L.moe_load_router(fake_ctx, 0, None, None, 1, None) == E_ARG
    assert L.moe_load_router(fake_ctx, -1, 4096, None, 1, None) == E_ARG


def test_zero_tokens_route_is_empty_without_launch(fake_ctx):
    # a zero-token call needs the router loaded but launches nothing; with
    # the router not loaded it is a state error
    r = moe.MoeRouting()
    assert moe.lib().moe_route(fake_ctx, 0, None, 0, None, ctypes.byref(r), None) == E_STATE


def test_status_strings():
    L = moe.lib()
    assert L.moe_status_string(0) == b"MOE_OK"
    assert L.moe_status_string(-4) == b"MOE_E_CAPACITY"


def test_diag_stream_read_rejects_bad_arguments():
    # argument checks run before any launch (no GPU needed)
    lib = moe.lib()
    aligned = 1 << 20
    assert lib.moe_diag_stream_read(None, 16, aligned, None) == E_ARG
    assert lib.moe_diag_stream_read(aligned, 16, None, None) == E_ARG
    assert lib.moe_diag_stream_read(aligned + 8, 16, aligned, None) == E_ARG
    assert lib.moe_diag_stream_read(aligned, 17, aligned, None) == E_ARG
    assert lib.moe_diag_stream_read(aligned, 16, aligned + 4, None) == E_ARG
    assert lib.moe_diag_stream_read(aligned, 0, aligned, None) == moe.MOE_OK


def test_diag_bf16_rejects_bad_arguments():
    lib = moe.lib()
    aligned = 1 << 20
    assert lib.moe_diag_bf16(None, aligned, 2, None) == E_ARG
    assert lib.moe_diag_bf16(aligned, None, 2, None) == E_ARG
    assert lib.moe_diag_bf16(aligned + 4, aligned, 2, None) == E_ARG
    assert lib.moe_diag_bf16(aligned, aligned + 2, 2, None) == E_ARG
    assert lib.moe_diag_bf16(aligned, aligned, 3, None) == E_ARG
    assert lib.moe_diag_bf16(aligned, aligned, 0, None) == moe.MOE_OK


def test_binding_checks_tensors_before_the_abi():
    """The C-ABI takes plain pointers and cannot see sizes, so the binding
    rejects a tensor of the wrong dtype, a strided view, a tensor on another
    device or one with fewer elements than the call uses."""
    import torch
    ptr = moe._tensor_ptr
    bf = moe._bf16_types(torch)
    cpu = torch.device("cpu")
    x = torch.zeros(4, 8, dtype=torch.int16)
    assert ptr(x, "x", 32, bf, cpu) == x.data_ptr()
    assert ptr(x.view(torch.bfloat16), "x", 32, bf, None) == x.data_ptr()
    assert ptr(torch.zeros(0, 8, dtype=torch.int16), "x", 0, bf, cpu) is not None
    bad = [
        (None, 0, "is None"),
        (x.view(torch.float16), 32, "dtype"),
        (x.float(), 32, "dtype"),
        (x.t(), 32, "contiguous"),
        (x[:, ::2], 16, "contiguous"),
        (x, 33, "elements"),
    ]
    for t, n, what in bad:
        with pytest.raises(moe.MoeError, match=what):
            ptr(t, "x", n, bf, cpu)
    with pytest.raises(moe.MoeError, match="expected cuda:0"):
        ptr(x, "x", 32, bf, torch.device("cuda", 0))
    assert ptr(torch.zeros(16), "wr", 16, (torch.float32,), cpu)
    with pytest.raises(moe.MoeError, match="dtype"):
        ptr(torch.zeros(16, dtype=torch.float64), "wr", 16, (torch.float32,), cpu)


def test_layer_needs_a_gpu_device():
    with pytest.raises(moe.MoeError, match="runs on a GPU"):
        moe.MoeLayer(moe.make_config(256, 128, 8, 2), device="cpu")


def test_binding_constants_match_the_header():
    text = open(HEADERS[0]).read()
    assert int(re.search(r"#define MOE_DIAG_MAX_WG (\d+)", text).group(1)) == moe.DIAG_MAX_WG
    assert int(re.search(r"#define MOE_PARTIAL_F32 0x(\d+)", text).group(1), 16) == moe.MOE_PARTIAL_F32
    for name, value in moe.STATUS_NAMES.items():
        assert re.search(rf"\b{value}\s*=\s*{name}\b", text), value
    def enum_body(src, name):
        end = src.index("} %s;" % name)
        return src[src.rindex("typedef enum {", 0, end):end]
    regions = enum_body(text, "moe_ws_region")
    names = [n.lower()[len("moe_ws_"):] for n in re.findall(r"\b(MOE_WS_\w+)", regions)]
    assert names[:-1] == moe.WS_REGIONS and names[-1] == "count"
    atext = open(HEADERS[1]).read()
    kinds = enum_body(atext, "attn_kernel_kind")
    knames = [n.lower()[len("attn_k_"):] for n in re.findall(r"\b(ATTN_K_\w+)", kinds)]
    assert knames[:-1] == moe.ATTN_KERNEL_KINDS and knames[-1] == "count"


def _attn_cfg(**kw):
    base = dict(d_model=6144, n_heads=48, n_kv_heads=8, head_dim=128, n_layers=1, max_seq=4096,
                max_tokens=16)
    base.update(kw)
    return moe.make_attn_config(**base)


def test_attn_sizes():
    cfg = _attn_cfg()
    layer = 6144 * 4 + 512 + 6144 * 4 + (6144 * 8192 + 6144 * 6144) * 2   # gamma, frequencies, gamma2, Wqkv, Wo
    assert moe.attn_weight_bytes(cfg) == layer
    assert moe.attn_cache_bytes(_attn_cfg(n_layers=3)) == 3 * 2 * 8 * 4096 * 128 * 2
    assert moe.attn_workspace_bytes(cfg) > 16 * (6144 * 2 + 8192 * 4)


@pytest.mark.parametrize("bad", [dict(d_model=200), dict(d_model=8448), dict(head_dim=96), dict(n_kv_heads=5),
                                 dict(n_heads=64, n_kv_heads=4), dict(max_tokens=32769),
                                 dict(n_heads=4, n_kv_heads=1, head_dim=64, max_tokens=17),
                                 dict(max_tokens=0), dict(max_seq=0), dict(n_layers=0),
                                 dict(rope_theta=1.0), dict(norm_eps=-1.0), dict(flags=1),
                                 dict(n_heads=3, n_kv_heads=1, head_dim=64)])
def test_attn_bad_configs_rejected(bad):
    # n_heads 64 over 4 key/value heads: 16 query heads share one, past the
    # attention kernel's 8; 3 heads of 64: the output projection's K (192) is
    # not a multiple of 256; 4 + 2 heads of 64 (384 fused rows) cannot take
    # the prefill GEMM's 256-row tiles, so such a config is limited to 16
    # tokens
    cfg = _attn_cfg(**bad)
    assert moe.attn_weight_bytes(cfg) == 0
    out = ctypes.c_void_p()
    assert moe.lib().attn_init(ctypes.byref(cfg), 4096, 8192, 16384, ctypes.byref(out)) == E_SHAPE
    assert out.value is None and moe.lib().attn_last_error(None)


def test_attn_validation_before_any_launch():
    cfg = _attn_cfg(d_model=256, n_heads=4, n_kv_heads=2, head_dim=64, n_layers=2, max_seq=64,
                    max_tokens=4)
    L = moe.lib()
    out = ctypes.c_void_p()
    assert L.attn_init(ctypes.byref(cfg), 4096 + 16, 8192, 16384, ctypes.byref(out)) == E_ALIGN
    assert L.attn_init(ctypes.byref(cfg), None, 8192, 16384, ctypes.byref(out)) == E_ARG
    ctx = moe.attn_init(cfg, 1 << 20, 1 << 24, 1 << 26)
    try:
        assert L.attn_forward(ctx, 0, 4096, 4096, 1, 0, None) == E_STATE      # not loaded
        assert L.attn_forward(ctx, 2, 4096, 4096, 1, 0, None) == E_ARG
        assert L.attn_forward(ctx, 0, 4096, 4096, 5, 0, None) == E_CAPACITY   # T > max_tokens
        assert L.attn_forward(ctx, 0, 4096, 4096, 2, 63, None) == E_CAPACITY  # past max_seq
        assert L.attn_forward(ctx, 0, 4096, 4096, 1, -1, None) == E_ARG
        assert L.attn_load_layer(ctx, 0, None, 4096, 4096, 1, None) == E_ARG
        assert L.attn_load_layer(ctx, 0, 4096 + 4, 4096, 4096, 1, None) == E_ALIGN
        assert L.attn_load_layer(ctx, 5, 4096, 4096, 4096, 1, None) == E_ARG
        assert "range" in moe.lib().attn_last_error(ctx).decode()
        assert L.attn_forward_norm(ctx, 0, 4096, 4096, 4096, 1, 0, None) == E_STATE
        assert L.attn_load_post_norm(ctx, 0, None, 1, None) == E_ARG
        assert L.attn_load_post_norm(ctx, 0, 4096 + 4, 1, None) == E_ALIGN
        assert L.attn_load_post_norm(ctx, 2, 4096, 1, None) == E_ARG
    finally:
        L.attn_destroy(ctx)
