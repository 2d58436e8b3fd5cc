// attn_capi.cpp -- the C-ABI of include/attn.h: configuration checks, the
// carve-up of the caller's weight arena, cache and workspace, the one-time
// weight repack (the query and key heads of Wqkv with their rotation pairs
// in one tile), and the launch sequences of the block: up to 16 tokens
// (decode) norm, inside the projection up to 4 tokens -> fused projection +
// rotary + cache append -> attention over position chunks -> merge ->
// output projection + residual; above 16 (prefill) norm -> projection GEMM
// -> rotary + cache append -> causal attention -> output GEMM -> residual.
// Nothing here allocates device memory.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstring>
#include <cstdint>
#include <new>
#include <string>
#include <vector>

#include "../../include/attn.h"
#include "moe_common.h"

namespace {

constexpr size_t kAlign = 256;
constexpr int kDecodeTokens = 16;  // up to here the decode path (token columns of one MFMA B operand)
constexpr int kMaxTokens = 32768;  // the prefill path's bound (activation buffers below 2^31 bytes)
constexpr int kMaxGroup = 8;       // query heads per key/value head (attention LDS rows)

size_t align_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

struct Layout {
    size_t gamma_bytes, freq_off, gamma2_off, wqkv_off, wqkv_bytes, wo_off, wo_bytes, layer_bytes,
        arena_bytes;
    size_t cache_head_elems, cache_layer_bytes, cache_bytes;
    size_t h_off, qkv_off, q_off, part_off, a_off, o_off, qkvp_off, plan_off, ws_bytes;
    int nqkv, nq, n_chunks, max_tiles;
};

const char* check_config(const attn_config* c)
{
    if (!c) return "config is NULL";
    if (c->d_model <= 0 || c->d_model % 256 || c->d_model > 8192)
        return "d_model must be a multiple of 256 in [256, 8192]";
    if (c->head_dim != 64 && c->head_dim != 128) return "head_dim must be 64 or 128";
    if (c->n_heads < 1 || c->n_kv_heads < 1 || c->n_heads % c->n_kv_heads)
        return "n_kv_heads must divide n_heads";
    if (c->n_heads / c->n_kv_heads > kMaxGroup) return "at most 8 query heads per key/value head";
    if ((int64_t)c->n_heads * c->head_dim % 256) return "n_heads * head_dim must be a multiple of 256";
    if ((int64_t)(c->n_heads + 2 * c->n_kv_heads) * c->head_dim * c->d_model * 2 > INT32_MAX)
        return "the fused projection must stay below 2^31 bytes";
    if ((int64_t)c->n_heads * c->head_dim > 65536) return "n_heads * head_dim too large";
    if (c->n_layers < 1 || c->n_layers > 1024) return "n_layers must be in [1, 1024]";
    if (c->max_seq < 1 || c->max_seq > (1 << 20)) return "max_seq must be in [1, 2^20]";
    if (c->max_tokens < 1 || c->max_tokens > kMaxTokens) return "max_tokens must be in [1, 32768]";
    if (c->max_tokens > kDecodeTokens && (int64_t)(c->n_heads + 2 * c->n_kv_heads) * c->head_dim % 256)
        return "above 16 tokens (n_heads + 2 n_kv_heads) * head_dim must be a multiple of 256";
    if (!(c->rope_theta > 1.0f) || !std::isfinite(c->rope_theta)) return "rope_theta must be > 1";
    if (!(c->norm_eps >= 0.0f) || !std::isfinite(c->norm_eps)) return "norm_eps must be >= 0";
    if (c->flags != 0) return "flags must be 0";
    return nullptr;
}

Layout make_layout(const attn_config* c)
{
    Layout L{};
    const size_t d = c->d_model, hd = c->head_dim, H = c->n_heads, G = c->n_kv_heads;
    L.nq = (int)(H * hd);
    L.nqkv = (int)((H + 2 * G) * hd);
    L.gamma_bytes = align_up(d * 4, kAlign);
    L.freq_off = L.gamma_bytes;
    L.gamma2_off = L.freq_off + align_up(hd / 2 * 8, kAlign);
    L.wqkv_off = L.gamma2_off + L.gamma_bytes;
    L.wqkv_bytes = d * L.nqkv * 2;
    L.wo_off = L.wqkv_off + align_up(L.wqkv_bytes, kAlign);
    L.wo_bytes = (size_t)L.nq * d * 2;
    L.layer_bytes = L.wo_off + align_up(L.wo_bytes, kAlign);
    L.arena_bytes = L.layer_bytes * c->n_layers;
    L.cache_head_elems = (size_t)c->max_seq * hd;
    L.cache_layer_bytes = 2 * G * L.cache_head_elems * 2;
    L.cache_bytes = L.cache_layer_bytes * c->n_layers;
    L.n_chunks = attn_chunks(c->max_seq);
    const size_t Tm = c->max_tokens;
    const size_t Td = std::min<size_t>(Tm, kDecodeTokens);
    const int tile_rows = moe_prefill_tile_rows();
    L.max_tiles = (int)((Tm + tile_rows - 1) / tile_rows);
    size_t off = 0;
    auto take = [&](size_t bytes) { size_t o = off; off = align_up(off + bytes, kAlign); return o; };
    L.h_off = take(Tm * d * 2);
    L.qkv_off = take(Tm * L.nqkv * 4);
    L.q_off = take(Tm * L.nq * 2);
    L.part_off = take(Td * H * L.n_chunks * attn_part_stride((int)hd) * 4);
    L.a_off = take(Tm * L.nq * 2);
    L.o_off = take(Tm * d * 4);
    if (Tm > (size_t)kDecodeTokens) {
        L.qkvp_off = take(Tm * L.nqkv * 4);
        // the projection GEMMs' tile table: (0, 256 i) per token tile, then
        // per T: offsets {0, T} and the tile count
        L.plan_off = take((size_t)L.max_tiles * 8 + (Tm + 1) * 16);
    }
    L.ws_bytes = off;
    return L;
}

thread_local std::string g_init_error;

}  // namespace

struct attn_ctx {
    attn_config cfg;
    Layout L;
    uint8_t* arena;
    uint8_t* cache;
    uint8_t* ws;
    std::vector<uint8_t> loaded;
    std::vector<uint8_t> post_loaded;
    bool prof_on;
    std::vector<hipEvent_t> prof_events;
    std::vector<int> prof_kinds;
    int64_t prof_dropped;
    std::string err;
};

namespace {

moe_status fail(attn_ctx* ctx, moe_status s, const std::string& msg)
{
    if (ctx) ctx->err = msg;
    else g_init_error = msg;
    return s;
}

moe_status hip_fail(attn_ctx* ctx, hipError_t e, const char* what)
{
    return fail(ctx, MOE_E_HIP, std::string(what) + ": " + hipGetErrorString(e));
}

bool misaligned(const void* p) { return ((uintptr_t)p & 15u) != 0; }

template <class F>
hipError_t timed(attn_ctx* c, int kind, hipStream_t s, F&& launch)
{
    if (!c->prof_on) return launch();
    const size_t slot = c->prof_kinds.size();
    if (2 * slot + 1 >= c->prof_events.size()) {
        ++c->prof_dropped;
        return launch();
    }
    hipError_t e = hipEventRecord(c->prof_events[2 * slot], s);
    if (e != hipSuccess) return e;
    e = launch();
    if (e != hipSuccess) return e;
    e = hipEventRecord(c->prof_events[2 * slot + 1], s);
    if (e == hipSuccess) c->prof_kinds.push_back(kind);
    return e;
}

uint8_t* layer_w(attn_ctx* c, int l) { return c->arena + (size_t)l * c->L.layer_bytes; }
uint16_t* layer_k(attn_ctx* c, int l)
{
    return reinterpret_cast<uint16_t*>(c->cache + (size_t)l * c->L.cache_layer_bytes);
}
uint16_t* layer_v(attn_ctx* c, int l)
{
    return layer_k(c, l) + (size_t)c->cfg.n_kv_heads * c->L.cache_head_elems;
}

// One plain GEMM out = in W^T on the grouped GEMM's down mode: a single
// "expert" whose rows are the T tokens, its weight the packed N x K matrix.
hipError_t project(attn_ctx* c, const uint8_t* wpk, const uint16_t* in, int K, int N, float* out,
                   int T, hipStream_t s)
{
    const Layout& L = c->L;
    int32_t* plan = reinterpret_cast<int32_t*>(c->ws + L.plan_off);
    moe::GemmArgs g{};
    g.experts = wpk;
    g.expert_bytes = (uint64_t)N * K * 2;
    g.gu_bytes = 0;
    g.H = const_cast<uint16_t*>(in);
    g.O = out;
    g.tiles = plan;
    g.offsets = plan + (size_t)L.max_tiles * 2 + (size_t)T * 4;
    g.n_tiles = g.offsets + 2;
    g.d = N;
    g.f = K;
    g.e_begin = 0;
    g.max_tiles = (T + moe_prefill_tile_rows() - 1) / moe_prefill_tile_rows();
    g.T = T;
    return moe_launch_gemm_down(&g, s);
}

// The block for T > 16 new tokens: norm -> q|k|v (GEMM) -> rotation and
// cache append -> causal attention -> o = a Wo (GEMM) -> residual.
moe_status prefill(attn_ctx* ctx, int layer, const uint16_t* x, uint16_t* y, int T, int pos0,
                   hipStream_t s)
{
    const attn_config& c = ctx->cfg;
    const Layout& L = ctx->L;
    uint8_t* w = layer_w(ctx, layer);
    uint16_t* h = reinterpret_cast<uint16_t*>(ctx->ws + L.h_off);
    float* qkv = reinterpret_cast<float*>(ctx->ws + L.qkv_off);
    float* qkvp = reinterpret_cast<float*>(ctx->ws + L.qkvp_off);
    uint16_t* q = reinterpret_cast<uint16_t*>(ctx->ws + L.q_off);
    uint16_t* a = reinterpret_cast<uint16_t*>(ctx->ws + L.a_off);
    float* o = reinterpret_cast<float*>(ctx->ws + L.o_off);
    const int d = c.d_model;
    const float* gamma = reinterpret_cast<const float*>(w);
    hipError_t e = timed(ctx, ATTN_K_NORM, s, [&] {
        return attn_launch_norm(x, gamma, T, d, c.norm_eps, h, s);
    });
    if (e != hipSuccess) return hip_fail(ctx, e, "norm kernel launch");
    e = timed(ctx, ATTN_K_QKV, s, [&] { return project(ctx, w + L.wqkv_off, h, d, L.nqkv, qkvp, T, s); });
    if (e != hipSuccess) return hip_fail(ctx, e, "projection GEMM launch");
    e = timed(ctx, ATTN_K_ROPE, s, [&] {
        return attn_launch_rope(qkvp, reinterpret_cast<const double*>(w + L.freq_off), qkv, q,
                                layer_k(ctx, layer), layer_v(ctx, layer), T, c.n_heads,
                                c.n_kv_heads, c.head_dim, c.max_seq, pos0, s);
    });
    if (e != hipSuccess) return hip_fail(ctx, e, "rotation kernel launch");
    e = timed(ctx, ATTN_K_SCORE, s, [&] {
        return attn_launch_flash(q, layer_k(ctx, layer), layer_v(ctx, layer), a, T, c.n_heads,
                                 c.n_kv_heads, c.head_dim, c.max_seq, pos0, s);
    });
    if (e != hipSuccess) return hip_fail(ctx, e, "attention kernel launch");
    e = timed(ctx, ATTN_K_OUT, s, [&] { return project(ctx, w + L.wo_off, a, L.nq, d, o, T, s); });
    if (e != hipSuccess) return hip_fail(ctx, e, "output projection GEMM launch");
    e = timed(ctx, ATTN_K_RESIDUAL, s, [&] {
        return attn_launch_residual(x, o, y, (int64_t)T * d, s);
    });
    if (e != hipSuccess) return hip_fail(ctx, e, "residual kernel launch");
    return MOE_OK;
}

}  // namespace

namespace {

moe_status check_forward(attn_ctx* ctx, int32_t layer, const uint16_t* x, uint16_t* y, int32_t T,
                         int32_t pos0)
{
    const attn_config& c = ctx->cfg;
    if (layer < 0 || layer >= c.n_layers) return fail(ctx, MOE_E_ARG, "layer out of range");
    if (T < 0 || pos0 < 0) return fail(ctx, MOE_E_ARG, "T and pos0 must be non-negative");
    if (T > c.max_tokens) return fail(ctx, MOE_E_CAPACITY, "T exceeds max_tokens");
    if ((int64_t)pos0 + T > c.max_seq) return fail(ctx, MOE_E_CAPACITY, "pos0 + T exceeds max_seq");
    if (!ctx->loaded[layer]) return fail(ctx, MOE_E_STATE, "layer weights not loaded");
    if (T == 0) return MOE_OK;
    if (!x || !y) return fail(ctx, MOE_E_ARG, "x or y is NULL");
    if (misaligned(x) || misaligned(y)) return fail(ctx, MOE_E_ALIGN, "x and y must be 16-byte aligned");
    return MOE_OK;
}

moe_status forward_impl(attn_ctx* ctx, int32_t layer, const uint16_t* x, uint16_t* y, int32_t T,
                        int32_t pos0, hipStream_t s)
{
    const attn_config& c = ctx->cfg;
    const Layout& L = ctx->L;
    uint8_t* w = layer_w(ctx, layer);
    uint16_t* h = reinterpret_cast<uint16_t*>(ctx->ws + L.h_off);
    float* qkv = reinterpret_cast<float*>(ctx->ws + L.qkv_off);
    uint16_t* q = reinterpret_cast<uint16_t*>(ctx->ws + L.q_off);
    float* part = reinterpret_cast<float*>(ctx->ws + L.part_off);
    uint16_t* a = reinterpret_cast<uint16_t*>(ctx->ws + L.a_off);
    float* o = reinterpret_cast<float*>(ctx->ws + L.o_off);
    const int d = c.d_model;
    const float* gamma = reinterpret_cast<const float*>(w);
    hipError_t e = hipSuccess;
    if (T > kDecodeTokens) return prefill(ctx, layer, x, y, T, pos0, s);
    if (!attn_norm_in_projection(T)) {
        e = timed(ctx, ATTN_K_NORM, s, [&] {
            return attn_launch_norm(x, gamma, T, d, c.norm_eps, h, s);
        });
        if (e != hipSuccess) return hip_fail(ctx, e, "norm kernel launch");
    }
    e = timed(ctx, ATTN_K_QKV, s, [&] {
        return attn_launch_qkv(w + L.wqkv_off, h, x, gamma, c.norm_eps,
                               reinterpret_cast<const double*>(w + L.freq_off), qkv, q,
                               layer_k(ctx, layer), layer_v(ctx, layer), T, d, c.n_heads,
                               c.n_kv_heads, c.head_dim, c.max_seq, pos0, s);
    });
    if (e != hipSuccess) return hip_fail(ctx, e, "projection kernel launch");
    e = timed(ctx, ATTN_K_SCORE, s, [&] {
        return attn_launch_score(q, layer_k(ctx, layer), layer_v(ctx, layer), part, T, c.n_heads,
                                 c.n_kv_heads, c.head_dim, c.max_seq, pos0, L.n_chunks, s);
    });
    if (e != hipSuccess) return hip_fail(ctx, e, "attention kernel launch");
    e = timed(ctx, ATTN_K_COMBINE, s, [&] {
        return attn_launch_combine(part, a, T, c.n_heads, c.head_dim, pos0, L.n_chunks, s);
    });
    if (e != hipSuccess) return hip_fail(ctx, e, "merge kernel launch");
    e = timed(ctx, ATTN_K_OUT, s, [&] {
        return attn_launch_out(w + L.wo_off, a, T, L.nq, d, o, x, y, s);
    });
    if (e != hipSuccess) return hip_fail(ctx, e, "output projection kernel launch");
    return MOE_OK;
}

}  // namespace

extern "C" {

size_t attn_weight_bytes(const attn_config* cfg)
{
    return check_config(cfg) ? 0 : make_layout(cfg).arena_bytes;
}

size_t attn_cache_bytes(const attn_config* cfg)
{
    return check_config(cfg) ? 0 : make_layout(cfg).cache_bytes;
}

size_t attn_workspace_bytes(const attn_config* cfg)
{
    return check_config(cfg) ? 0 : make_layout(cfg).ws_bytes;
}

moe_status attn_init(const attn_config* cfg, void* weight_arena, void* kv_cache, void* workspace,
                     attn_ctx** out)
{
    if (!out) return fail(nullptr, MOE_E_ARG, "out is NULL");
    *out = nullptr;
    if (const char* why = check_config(cfg)) return fail(nullptr, MOE_E_SHAPE, why);
    if (!weight_arena || !kv_cache || !workspace)
        return fail(nullptr, MOE_E_ARG, "arena, cache or workspace is NULL");
    if (((uintptr_t)weight_arena | (uintptr_t)kv_cache | (uintptr_t)workspace) & (kAlign - 1))
        return fail(nullptr, MOE_E_ALIGN, "arena, cache and workspace must be 256-byte aligned");
    attn_ctx* c = new (std::nothrow) attn_ctx();
    if (!c) return fail(nullptr, MOE_E_ARG, "out of host memory");
    c->cfg = *cfg;
    c->L = make_layout(cfg);
    c->arena = static_cast<uint8_t*>(weight_arena);
    c->cache = static_cast<uint8_t*>(kv_cache);
    c->ws = static_cast<uint8_t*>(workspace);
    if (cfg->max_tokens > kDecodeTokens) {
        // the prefill projections' tile table, written once into the workspace
        const int tile_rows = moe_prefill_tile_rows();
        std::vector<int32_t> plan((size_t)c->L.max_tiles * 2 + ((size_t)cfg->max_tokens + 1) * 4, 0);
        for (int i = 0; i < c->L.max_tiles; ++i) plan[2 * i + 1] = i * tile_rows;
        for (int T = 0; T <= cfg->max_tokens; ++T) {
            int32_t* e = &plan[(size_t)c->L.max_tiles * 2 + (size_t)T * 4];
            e[1] = T;
            e[2] = (T + tile_rows - 1) / tile_rows;
        }
        const hipError_t e = hipMemcpy(c->ws + c->L.plan_off, plan.data(), plan.size() * 4,
                                       hipMemcpyHostToDevice);
        if (e != hipSuccess) {
            delete c;
            return fail(nullptr, MOE_E_HIP, std::string("tile table copy: ") + hipGetErrorString(e));
        }
    }
    c->loaded.assign(cfg->n_layers, 0);
    c->post_loaded.assign(cfg->n_layers, 0);
    c->prof_on = false;
    c->prof_dropped = 0;
    *out = c;
    return MOE_OK;
}

moe_status attn_load_layer(attn_ctx* ctx, int32_t layer, const float* gamma, const uint16_t* wqkv,
                           const uint16_t* wo, int32_t src_on_device, moe_stream_t stream)
{
    if (!ctx) return MOE_E_ARG;
    const attn_config& c = ctx->cfg;
    const Layout& L = ctx->L;
    if (layer < 0 || layer >= c.n_layers) return fail(ctx, MOE_E_ARG, "layer out of range");
    if (!gamma || !wqkv || !wo) return fail(ctx, MOE_E_ARG, "weight pointer is NULL");
    hipStream_t s = static_cast<hipStream_t>(stream);
    uint8_t* base = layer_w(ctx, layer);
    const int d = c.d_model;
    // the rotary frequencies theta^(-2f/hd), once per layer beside gamma
    std::vector<double> freq(c.head_dim / 2);
    for (int f = 0; f < c.head_dim / 2; ++f)
        freq[f] = std::pow((double)c.rope_theta, -2.0 * f / c.head_dim);
    hipError_t e;
    if (src_on_device) {
        if (misaligned(gamma) || misaligned(wqkv) || misaligned(wo))
            return fail(ctx, MOE_E_ALIGN, "device weight pointers must be 16-byte aligned");
        e = hipMemcpyAsync(base, gamma, (size_t)d * 4, hipMemcpyDeviceToDevice, s);
        if (e == hipSuccess)
            e = hipMemcpyAsync(base + L.freq_off, freq.data(), freq.size() * 8,
                               hipMemcpyHostToDevice, s);
        if (e == hipSuccess) e = hipStreamSynchronize(s);   // freq is a host temporary
        if (e == hipSuccess)
            e = timed(ctx, ATTN_K_PACK, s, [&] {
                return moe_launch_pack_perm(wqkv, d, L.nqkv, base + L.wqkv_off, 1, 0, c.head_dim,
                                            (c.n_heads + c.n_kv_heads) * c.head_dim, s);
            });
        if (e == hipSuccess)
            e = timed(ctx, ATTN_K_PACK, s, [&] {
                return moe_launch_pack(wo, L.nq, d, base + L.wo_off, 1, 0, s);
            });
        if (e != hipSuccess) return hip_fail(ctx, e, "attention weight repack");
    } else {
        std::vector<uint8_t> tmp;
        try {
            tmp.resize(L.layer_bytes);
        } catch (...) {
            return fail(ctx, MOE_E_ARG, "out of host memory for the host repack");
        }
        std::memcpy(tmp.data(), gamma, (size_t)d * 4);
        std::memcpy(tmp.data() + L.freq_off, freq.data(), freq.size() * 8);
        moe_pack_host_perm(wqkv, d, L.nqkv, tmp.data() + L.wqkv_off, 1, 0, c.head_dim,
                           (c.n_heads + c.n_kv_heads) * c.head_dim);
        moe_pack_host(wo, L.nq, d, tmp.data() + L.wo_off, 1, 0);
        e = hipMemcpyAsync(base, tmp.data(), tmp.size(), hipMemcpyHostToDevice, s);
        if (e == hipSuccess) e = hipStreamSynchronize(s);
        if (e != hipSuccess) return hip_fail(ctx, e, "host-to-device copy of the attention weights");
    }
    ctx->loaded[layer] = 1;
    return MOE_OK;
}

moe_status attn_load_post_norm(attn_ctx* ctx, int32_t layer, const float* gamma2,
                               int32_t src_on_device, moe_stream_t stream)
{
    if (!ctx) return MOE_E_ARG;
    if (layer < 0 || layer >= ctx->cfg.n_layers) return fail(ctx, MOE_E_ARG, "layer out of range");
    if (!gamma2) return fail(ctx, MOE_E_ARG, "gamma2 is NULL");
    hipStream_t s = static_cast<hipStream_t>(stream);
    uint8_t* dst = layer_w(ctx, layer) + ctx->L.gamma2_off;
    const size_t bytes = (size_t)ctx->cfg.d_model * 4;
    hipError_t e;
    if (src_on_device) {
        if (misaligned(gamma2)) return fail(ctx, MOE_E_ALIGN, "gamma2 must be 16-byte aligned");
        e = hipMemcpyAsync(dst, gamma2, bytes, hipMemcpyDeviceToDevice, s);
    } else {
        e = hipMemcpyAsync(dst, gamma2, bytes, hipMemcpyHostToDevice, s);
        if (e == hipSuccess) e = hipStreamSynchronize(s);
    }
    if (e != hipSuccess) return hip_fail(ctx, e, "post-attention norm load");
    ctx->post_loaded[layer] = 1;
    return MOE_OK;
}

moe_status attn_forward(attn_ctx* ctx, int32_t layer, const uint16_t* x, uint16_t* y, int32_t T,
                        int32_t pos0, moe_stream_t stream)
{
    if (!ctx) return MOE_E_ARG;
    moe_status st = check_forward(ctx, layer, x, y, T, pos0);
    if (st != MOE_OK || T == 0) return st;
    return forward_impl(ctx, layer, x, y, T, pos0, static_cast<hipStream_t>(stream));
}

moe_status attn_forward_norm(attn_ctx* ctx, int32_t layer, const uint16_t* x, uint16_t* y,
                             uint16_t* z, int32_t T, int32_t pos0, moe_stream_t stream)
{
    if (!ctx) return MOE_E_ARG;
    moe_status st = check_forward(ctx, layer, x, y, T, pos0);
    if (st != MOE_OK) return st;
    if (!ctx->post_loaded[layer]) return fail(ctx, MOE_E_STATE, "post-attention norm not loaded");
    if (T == 0) return MOE_OK;
    if (!z) return fail(ctx, MOE_E_ARG, "z is NULL");
    if (misaligned(z)) return fail(ctx, MOE_E_ALIGN, "z must be 16-byte aligned");
    hipStream_t s = static_cast<hipStream_t>(stream);
    st = forward_impl(ctx, layer, x, y, T, pos0, s);
    if (st != MOE_OK) return st;
    const float* gamma2 = reinterpret_cast<const float*>(layer_w(ctx, layer) + ctx->L.gamma2_off);
    const hipError_t e = timed(ctx, ATTN_K_POST_NORM, s, [&] {
        return attn_launch_norm(y, gamma2, T, ctx->cfg.d_model, ctx->cfg.norm_eps, z, s);
    });
    if (e != hipSuccess) return hip_fail(ctx, e, "post-attention norm launch");
    return MOE_OK;
}

moe_status attn_intermediates(const attn_ctx* ctx, const uint16_t** h, const float** qkv,
                              const uint16_t** q, const uint16_t** a, const float** o)
{
    if (!ctx) return MOE_E_ARG;
    const Layout& L = ctx->L;
    if (h) *h = reinterpret_cast<const uint16_t*>(ctx->ws + L.h_off);
    if (qkv) *qkv = reinterpret_cast<const float*>(ctx->ws + L.qkv_off);
    if (q) *q = reinterpret_cast<const uint16_t*>(ctx->ws + L.q_off);
    if (a) *a = reinterpret_cast<const uint16_t*>(ctx->ws + L.a_off);
    if (o) *o = reinterpret_cast<const float*>(ctx->ws + L.o_off);
    return MOE_OK;
}

moe_status attn_profile_enable(attn_ctx* ctx, int32_t max_launches)
{
    if (!ctx) return MOE_E_ARG;
    if (max_launches < 0) return fail(ctx, MOE_E_ARG, "max_launches is negative");
    for (hipEvent_t ev : ctx->prof_events)
        if (ev) (void)hipEventDestroy(ev);
    ctx->prof_events.clear();
    ctx->prof_kinds.clear();
    ctx->prof_dropped = 0;
    ctx->prof_on = false;
    if (max_launches == 0) return MOE_OK;
    ctx->prof_events.resize(2 * (size_t)max_launches);
    for (auto& ev : ctx->prof_events) {
        hipError_t e = hipEventCreate(&ev);
        if (e != hipSuccess) {
            ev = nullptr;
            return hip_fail(ctx, e, "event creation");
        }
    }
    ctx->prof_kinds.reserve(max_launches);
    ctx->prof_on = true;
    return MOE_OK;
}

moe_status attn_profile_read(attn_ctx* ctx, double* total_ms, int64_t* launches, int64_t* dropped)
{
    if (!ctx) return MOE_E_ARG;
    if (!total_ms || !launches) return fail(ctx, MOE_E_ARG, "output array is NULL");
    for (int k = 0; k < ATTN_K_COUNT; ++k) { total_ms[k] = 0.0; launches[k] = 0; }
    for (size_t i = 0; i < ctx->prof_kinds.size(); ++i) {
        hipError_t e = hipEventSynchronize(ctx->prof_events[2 * i + 1]);
        float ms = 0.f;
        if (e == hipSuccess)
            e = hipEventElapsedTime(&ms, ctx->prof_events[2 * i], ctx->prof_events[2 * i + 1]);
        if (e != hipSuccess) return hip_fail(ctx, e, "event timing");
        total_ms[ctx->prof_kinds[i]] += ms;
        launches[ctx->prof_kinds[i]] += 1;
    }
    if (dropped) *dropped = ctx->prof_dropped;
    ctx->prof_kinds.clear();
    ctx->prof_dropped = 0;
    return MOE_OK;
}

void attn_destroy(attn_ctx* ctx)
{
    if (!ctx) return;
    for (hipEvent_t ev : ctx->prof_events)
        if (ev) (void)hipEventDestroy(ev);
    delete ctx;
}

const char* attn_last_error(const attn_ctx* ctx) { return ctx ? ctx->err.c_str() : g_init_error.c_str(); }

}  // extern "C"
