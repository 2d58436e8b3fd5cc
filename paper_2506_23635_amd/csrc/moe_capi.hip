// moe_capi.cpp -- the C-ABI declared in include/moe.h: configuration checks,
// arena and workspace carve-up, prestacking of experts, and the launch
// sequence of one layer (router -> selection/permutation -> expert FFN ->
// weighted combine).  No device memory is allocated here: the weight arena
// and the workspace are the caller's (paper Sec. 4.1: weights are prestacked
// once into a persistent array and indexed per layer).
#include <hip/hip_runtime.h>

#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <new>
#include <string>
#include <algorithm>
#include <vector>

#include "../../include/moe.h"
#include "moe_common.h"

namespace {

constexpr int kDecodeMaxTokens = 16;   // token columns of one MFMA B operand
constexpr size_t kAlign = 256;

size_t align_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

struct Layout {
    // arena
    size_t router_bytes, bias_off, gu_bytes, dn_bytes, expert_bytes, experts_off, layer_bytes;
    size_t arena_bytes;
    // workspace
    size_t dpart_off, logits_off, idx_off, w_off, counts_off, offsets_off, pair_row_off,
        row_token_off, active_off, tiles_off, n_tiles_off, h_off, o_off, ws_bytes;
    size_t region_off[MOE_WS_COUNT], region_bytes[MOE_WS_COUNT];   // moe_workspace_map
    int rows_max, max_tiles;
};

const char* check_config(const moe_config* c)
{
    if (!c) return "config is NULL";
    if (c->d_model <= 0 || c->d_model % 256) return "d_model must be a positive multiple of 256";
    if (c->ffn_dim <= 0 || c->ffn_dim % 128) return "ffn_dim must be a positive multiple of 128";
    if (c->n_experts < 1 || c->n_experts > 64) return "n_experts must be in [1, 64]";
    if (c->top_k < 1 || c->top_k > c->n_experts) return "top_k must be in [1, n_experts]";
    if (c->expert_begin < 0 || c->n_local_experts < 1 ||
        c->expert_begin + c->n_local_experts > c->n_experts)
        return "local expert range outside [0, n_experts)";
    if (c->n_layers < 1 || c->n_layers > 1024) return "n_layers must be in [1, 1024]";
    if (c->max_tokens < 1 || c->max_tokens > (1 << 20)) return "max_tokens must be in [1, 2^20]";
    if ((int64_t)c->max_tokens * c->d_model * 2 > INT32_MAX)
        return "max_tokens * d_model * 2 must stay below 2^31 (32-bit gather offsets)";
    if ((int64_t)c->d_model * c->ffn_dim * 4 > INT32_MAX)
        return "d_model * ffn_dim * 4 (one expert's gate/up slab) must stay below 2^31";
    if (c->flags & ~MOE_PARTIAL_F32) return "flags: only MOE_PARTIAL_F32 is defined";
    return nullptr;
}

Layout make_layout(const moe_config* c)
{
    Layout L{};
    const size_t d = c->d_model, f = c->ffn_dim, E = c->n_experts, k = c->top_k;
    const size_t Tm = c->max_tokens, nl = c->n_local_experts;
    L.router_bytes = align_up(d * E * 4, kAlign);
    L.bias_off = L.router_bytes;
    L.experts_off = L.router_bytes + align_up(E * 4, kAlign);
    L.gu_bytes = 2 * f * d * 2;
    L.dn_bytes = d * f * 2;
    L.expert_bytes = L.gu_bytes + L.dn_bytes;
    L.layer_bytes = L.experts_off + nl * L.expert_bytes;
    L.arena_bytes = L.layer_bytes * (size_t)c->n_layers;

    const size_t kl = k < nl ? k : nl;
    L.rows_max = (int)(Tm * kl);
    const int tile_rows = moe_prefill_tile_rows();
    L.max_tiles = (int)((L.rows_max + tile_rows - 1) / tile_rows + nl);
    size_t off = 0;
    auto take = [&](int region, size_t bytes) {
        size_t o = off;
        off = align_up(off + bytes, kAlign);
        L.region_off[region] = o;
        L.region_bytes[region] = bytes;
        return o;
    };
    L.dpart_off = take(MOE_WS_ROUTE_PARTIALS, (size_t)moe_route_decode_wgs(c->d_model) * 16 * 16 * 8);
    L.logits_off = take(MOE_WS_LOGITS, Tm * E * 4);
    L.idx_off = take(MOE_WS_TOPK_IDX, Tm * k * 4);
    L.w_off = take(MOE_WS_TOPK_W, Tm * k * 4);
    L.counts_off = take(MOE_WS_COUNTS, E * 4);
    L.offsets_off = take(MOE_WS_OFFSETS, (E + 1) * 4);
    L.pair_row_off = take(MOE_WS_PAIR_ROW, Tm * k * 4);
    L.row_token_off = take(MOE_WS_ROW_TOKEN, Tm * k * 4);
    L.active_off = take(MOE_WS_ACTIVE, (E + 1) * 4);
    L.tiles_off = take(MOE_WS_TILES, (size_t)L.max_tiles * 2 * 4);
    L.n_tiles_off = take(MOE_WS_N_TILES, 4);
    L.h_off = take(MOE_WS_H, (size_t)L.rows_max * f * 2);
    L.o_off = take(MOE_WS_O, (size_t)L.rows_max * d * 4);
    L.ws_bytes = off;
    return L;
}

thread_local std::string g_init_error;

// Device views of one workspace: the context's own, or the library's static
// scratch (moe_forward_static).
struct WsView {
    uint8_t* base;
    size_t dpart_off, h_off, o_off;
    moe::RouteView rv;
};

WsView make_ws_view(uint8_t* w, const Layout& L)
{
    WsView v{};
    v.base = w;
    v.dpart_off = L.dpart_off;
    v.h_off = L.h_off;
    v.o_off = L.o_off;
    v.rv.logits = reinterpret_cast<float*>(w + L.logits_off);
    v.rv.topk_idx = reinterpret_cast<int32_t*>(w + L.idx_off);
    v.rv.topk_w = reinterpret_cast<float*>(w + L.w_off);
    v.rv.counts = reinterpret_cast<int32_t*>(w + L.counts_off);
    v.rv.offsets = reinterpret_cast<int32_t*>(w + L.offsets_off);
    v.rv.pair_row = reinterpret_cast<int32_t*>(w + L.pair_row_off);
    v.rv.row_token = reinterpret_cast<int32_t*>(w + L.row_token_off);
    v.rv.active = reinterpret_cast<int32_t*>(w + L.active_off);
    v.rv.tiles = reinterpret_cast<int32_t*>(w + L.tiles_off);
    v.rv.n_tiles = reinterpret_cast<int32_t*>(w + L.n_tiles_off);
    return v;
}

}  // namespace

struct moe_ctx {
    moe_config cfg;
    Layout L;
    uint8_t* arena;
    WsView ws;                            // the caller's workspace
    std::vector<uint8_t> router_loaded;   // [n_layers]
    std::vector<uint8_t> has_bias;        // [n_layers]
    std::vector<uint8_t> expert_loaded;   // [n_layers * n_local]
    // per-kernel timing (moe_profile_*): an event pair around each launch
    bool prof_on;
    std::vector<hipEvent_t> prof_events;   // 2 per launch slot
    std::vector<int> prof_kinds;           // kind of each recorded launch
    int64_t prof_dropped;
    uint64_t* tl_gateup;   // GEMM timelines (moe_profile_gemm_timeline), or NULL
    uint64_t* tl_down;
    int tl_max;
    // the routing that the last moe_route returned (moe_forward accepts it
    // while nothing has overwritten or outdated it)
    bool route_valid;
    int route_layer, route_T;
    const uint16_t* route_x;   // the x it was computed from; NULL for given logits
    std::string err;
};

namespace {

moe_status fail(moe_ctx* ctx, moe_status s, const std::string& msg)
{
    if (ctx) ctx->err = msg;
    else g_init_error = msg;
    return s;
}

bool misaligned(const void* p) { return ((uintptr_t)p & 15u) != 0; }

moe_status hip_fail(moe_ctx* ctx, hipError_t e, const char* what)
{
    return fail(ctx, MOE_E_HIP, std::string(what) + ": " + hipGetErrorString(e));
}

// Runs one launch; with profiling on, brackets it with a pair of events on
// the launch stream.
template <class F>
hipError_t timed(moe_ctx* c, int kind, hipStream_t s, F&& launch)
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

uint8_t* layer_base(moe_ctx* c, int layer) { return c->arena + (size_t)layer * c->L.layer_bytes; }

moe_status check_layer(moe_ctx* ctx, int layer)
{
    if (layer < 0 || layer >= ctx->cfg.n_layers) return fail(ctx, MOE_E_ARG, "layer out of range");
    if (!ctx->router_loaded[layer]) return fail(ctx, MOE_E_STATE, "router of this layer not loaded");
    for (int i = 0; i < ctx->cfg.n_local_experts; ++i)
        if (!ctx->expert_loaded[(size_t)layer * ctx->cfg.n_local_experts + i])
            return fail(ctx, MOE_E_STATE, "a local expert of this layer is not loaded");
    return MOE_OK;
}

moe_status do_route(moe_ctx* ctx, const WsView& ws, int layer, const uint16_t* x, int T,
                    const float* logits_in, hipStream_t s)
{
    const moe_config& c = ctx->cfg;
    uint8_t* lb = layer_base(ctx, layer);
    const float* wrT = reinterpret_cast<const float*>(lb);
    const float* bias = ctx->has_bias[layer] ? reinterpret_cast<const float*>(lb + ctx->L.bias_off)
                                             : nullptr;
    const int tile_rows = moe_prefill_tile_rows();
    hipError_t e;
    if (!logits_in && moe_route_decode_ok(T, c.n_experts, c.top_k)) {
        double* dpart = reinterpret_cast<double*>(ws.base + ws.dpart_off);
        e = timed(ctx, MOE_K_ROUTE, s, [&] {
            return moe_launch_route_decode(x, wrT, bias, dpart, T, c.d_model, c.n_experts,
                                           c.top_k, c.expert_begin, c.n_local_experts, tile_rows,
                                           &ws.rv, s);
        });
        if (e != hipSuccess) return hip_fail(ctx, e, "route kernel launch");
    } else {
        if (!logits_in) {
            e = timed(ctx, MOE_K_ROUTER, s, [&] {
                return moe_launch_router_select(x, wrT, bias, T, c.d_model, c.n_experts,
                                                c.top_k, &ws.rv, s);
            });
            if (e != hipSuccess) return hip_fail(ctx, e, "router kernel launch");
        }
        e = timed(ctx, MOE_K_ROUTE, s, [&] {
            return moe_launch_route(logits_in, T, c.n_experts, c.top_k, c.expert_begin,
                                    c.n_local_experts, tile_rows, &ws.rv, s);
        });
        if (e != hipSuccess) return hip_fail(ctx, e, "route kernel launch");
    }
    return MOE_OK;
}

void fill_routing(moe_ctx* ctx, int layer, int T, moe_routing* out)
{
    const moe::RouteView& rv = ctx->ws.rv;
    out->logits = rv.logits;
    out->topk_idx = rv.topk_idx;
    out->topk_w = rv.topk_w;
    out->counts = rv.counts;
    out->offsets = rv.offsets;
    out->pair_row = rv.pair_row;
    out->row_token = rv.row_token;
    out->T = T;
    out->layer = layer;
}

moe_status run_experts(moe_ctx* ctx, const WsView& ws, int layer, const uint16_t* x, int T,
                       hipStream_t s)
{
    const moe_config& c = ctx->cfg;
    const uint8_t* experts = layer_base(ctx, layer) + ctx->L.experts_off;
    uint16_t* H = reinterpret_cast<uint16_t*>(ws.base + ws.h_off);
    float* O = reinterpret_cast<float*>(ws.base + ws.o_off);
    hipError_t e;
    if (T <= kDecodeMaxTokens) {
        moe::DecodeArgs a;
        a.experts = experts;
        a.expert_bytes = ctx->L.expert_bytes;
        a.gu_bytes = ctx->L.gu_bytes;
        a.x = x;
        a.H = H;
        a.O = O;
        a.active = ws.rv.active;
        a.counts = ws.rv.counts;
        a.offsets = ws.rv.offsets;
        a.row_token = ws.rv.row_token;
        a.d = c.d_model;
        a.f = c.ffn_dim;
        a.e_begin = c.expert_begin;
        int slots = std::min(c.n_local_experts, T * c.top_k);
        e = timed(ctx, MOE_K_DECODE_GATEUP, s, [&] { return moe_launch_decode_gateup(&a, slots, s); });
        if (e != hipSuccess) return hip_fail(ctx, e, "decode gate/up kernel launch");
        e = timed(ctx, MOE_K_DECODE_DOWN, s, [&] { return moe_launch_decode_down(&a, slots, s); });
        if (e != hipSuccess) return hip_fail(ctx, e, "decode down kernel launch");
    } else {
        moe::GemmArgs a;
        a.experts = experts;
        a.expert_bytes = ctx->L.expert_bytes;
        a.gu_bytes = ctx->L.gu_bytes;
        a.x = x;
        a.H = H;
        a.O = O;
        a.offsets = ws.rv.offsets;
        a.row_token = ws.rv.row_token;
        a.tiles = ws.rv.tiles;
        a.n_tiles = ws.rv.n_tiles;
        a.d = c.d_model;
        a.f = c.ffn_dim;
        a.e_begin = c.expert_begin;
        a.T = T;
        a.max_stamps = ctx->tl_max;
        const int tile_rows = moe_prefill_tile_rows();
        const int kl = std::min(c.top_k, c.n_local_experts);
        a.max_tiles = (T * kl + tile_rows - 1) / tile_rows + c.n_local_experts;
        a.stamps = ctx->tl_gateup;
        e = timed(ctx, MOE_K_GEMM_GATEUP, s, [&] { return moe_launch_gemm_gateup(&a, s); });
        if (e != hipSuccess) return hip_fail(ctx, e, "grouped GEMM gate/up kernel launch");
        a.stamps = ctx->tl_down;
        e = timed(ctx, MOE_K_GEMM_DOWN, s, [&] { return moe_launch_gemm_down(&a, s); });
        if (e != hipSuccess) return hip_fail(ctx, e, "grouped GEMM down kernel launch");
    }
    return MOE_OK;
}

// The weighted combine of the routed rows of ws: into y (bf16), y32 (fp32)
// or, with x_residual, in place x = bf16(x + y).
moe_status combine(moe_ctx* ctx, const WsView& ws, int T, uint16_t* y, float* y32,
                   uint16_t* x_residual, hipStream_t s)
{
    hipError_t e = timed(ctx, MOE_K_COMBINE, s, [&] {
        return moe_launch_combine(reinterpret_cast<const float*>(ws.base + ws.o_off),
                                  ws.rv.pair_row, ws.rv.topk_w, T, ctx->cfg.d_model,
                                  ctx->cfg.top_k, y, y32, x_residual, s);
    });
    if (e != hipSuccess) return hip_fail(ctx, e, "combine kernel launch");
    return MOE_OK;
}

// The static scratch of moe_forward_static: one array per GPU, held until
// the process ends.  Host code never uses the array's name as an address
// (on the host it is only a stand-in for the device symbol); the device
// address is looked up once per device and kept in g_scratch_ptr.
static __device__ __align__(256) uint8_t scratch[MOE_STATIC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices];

// The current device's address of `scratch`, looked up on the first call
// on that device (with the device current), then reused.
moe_status scratch_ptr(moe_ctx* ctx, uint8_t** out)
{
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(ctx, e, "hipGetDevice");
    if (dev < 0 || dev >= kMaxDevices) return fail(ctx, MOE_E_HIP, "device index past the scratch table");
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return hip_fail(ctx, e, "hipGetSymbolAddress of the static scratch");
        if (!p) return fail(ctx, MOE_E_HIP, "hipGetSymbolAddress returned NULL for the static scratch");
        g_scratch_ptr[dev] = p;
    }
    *out = static_cast<uint8_t*>(g_scratch_ptr[dev]);
    return MOE_OK;
}

}  // namespace

extern "C" {

size_t moe_weight_bytes(const moe_config* cfg)
{
    if (check_config(cfg)) return 0;
    return make_layout(cfg).arena_bytes;
}

size_t moe_workspace_bytes(const moe_config* cfg)
{
    if (check_config(cfg)) return 0;
    return make_layout(cfg).ws_bytes;
}

int32_t moe_workspace_map(const moe_config* cfg, uint64_t* offset, uint64_t* bytes, int32_t n)
{
    if (check_config(cfg)) return 0;
    const Layout L = make_layout(cfg);
    for (int i = 0; i < n && i < MOE_WS_COUNT; ++i) {
        if (offset) offset[i] = L.region_off[i];
        if (bytes) bytes[i] = L.region_bytes[i];
    }
    return MOE_WS_COUNT;
}

moe_status moe_init(const moe_config* cfg, void* weight_arena, void* workspace, moe_ctx** out)
{
    if (!out) return fail(nullptr, MOE_E_ARG, "out is NULL");
    *out = nullptr;
    if (const char* why = check_config(cfg)) return fail(nullptr, MOE_E_SHAPE, why);
    if (!weight_arena || !workspace) return fail(nullptr, MOE_E_ARG, "arena or workspace is NULL");
    if (((uintptr_t)weight_arena & (kAlign - 1)) || ((uintptr_t)workspace & (kAlign - 1)))
        return fail(nullptr, MOE_E_ALIGN, "arena and workspace must be 256-byte aligned");
    moe_ctx* c = new (std::nothrow) moe_ctx();
    if (!c) return fail(nullptr, MOE_E_ARG, "out of host memory");
    c->cfg = *cfg;
    c->L = make_layout(cfg);
    c->arena = static_cast<uint8_t*>(weight_arena);
    c->ws = make_ws_view(static_cast<uint8_t*>(workspace), c->L);
    c->router_loaded.assign(cfg->n_layers, 0);
    c->has_bias.assign(cfg->n_layers, 0);
    c->expert_loaded.assign((size_t)cfg->n_layers * cfg->n_local_experts, 0);
    c->route_valid = false;
    c->route_layer = -1;
    c->route_T = 0;
    c->route_x = nullptr;
    c->prof_on = false;
    c->prof_dropped = 0;
    c->tl_gateup = c->tl_down = nullptr;
    c->tl_max = 0;
    *out = c;
    return MOE_OK;
}

moe_status moe_load_expert(moe_ctx* ctx, int32_t layer, int32_t expert, const uint16_t* gate,
                           const uint16_t* up, const uint16_t* down, int32_t src_on_device,
                           moe_stream_t stream)
{
    if (!ctx) return MOE_E_ARG;
    const moe_config& c = ctx->cfg;
    if (layer < 0 || layer >= c.n_layers) return fail(ctx, MOE_E_ARG, "layer out of range");
    if (expert < c.expert_begin || expert >= c.expert_begin + c.n_local_experts)
        return fail(ctx, MOE_E_ARG, "expert is not in the local range");
    if (!gate || !up || !down) return fail(ctx, MOE_E_ARG, "weight pointer is NULL");
    uint8_t* dst = layer_base(ctx, layer) + ctx->L.experts_off +
                   (size_t)(expert - c.expert_begin) * ctx->L.expert_bytes;
    hipStream_t s = static_cast<hipStream_t>(stream);
    const int d = c.d_model, f = c.ffn_dim;
    if (src_on_device) {
        if (misaligned(gate) || misaligned(up) || misaligned(down))
            return fail(ctx, MOE_E_ALIGN, "device weight pointers must be 16-byte aligned");
        hipError_t e;
        auto pk = [&](const uint16_t* src, int K, int N, uint8_t* to, int mul, int add) {
            return timed(ctx, MOE_K_PACK, s, [&] { return moe_launch_pack(src, K, N, to, mul, add, s); });
        };
        if ((e = pk(gate, d, f, dst, 2, 0)) != hipSuccess ||
            (e = pk(up, d, f, dst, 2, 1)) != hipSuccess ||
            (e = pk(down, f, d, dst + ctx->L.gu_bytes, 1, 0)) != hipSuccess)
            return hip_fail(ctx, e, "pack kernel launch");
    } else {
        std::vector<uint8_t> tmp;
        try {
            tmp.resize(ctx->L.expert_bytes);
        } catch (...) {
            return fail(ctx, MOE_E_ARG, "out of host memory for the host repack");
        }
        moe_pack_host(gate, d, f, tmp.data(), 2, 0);
        moe_pack_host(up, d, f, tmp.data(), 2, 1);
        moe_pack_host(down, f, d, tmp.data() + ctx->L.gu_bytes, 1, 0);
        hipError_t e = hipMemcpyAsync(dst, tmp.data(), tmp.size(), hipMemcpyHostToDevice, s);
        if (e == hipSuccess) e = hipStreamSynchronize(s);
        if (e != hipSuccess) return hip_fail(ctx, e, "host-to-device copy of packed expert");
    }
    ctx->expert_loaded[(size_t)layer * c.n_local_experts + (expert - c.expert_begin)] = 1;
    return MOE_OK;
}

moe_status moe_load_router(moe_ctx* ctx, int32_t layer, const float* wr, const float* bias,
                           int32_t src_on_device, moe_stream_t stream)
{
    if (!ctx) return MOE_E_ARG;
    const moe_config& c = ctx->cfg;
    if (layer < 0 || layer >= c.n_layers) return fail(ctx, MOE_E_ARG, "layer out of range");
    if (!wr) return fail(ctx, MOE_E_ARG, "router weight is NULL");
    if (ctx->route_layer == layer) ctx->route_valid = false;
    uint8_t* lb = layer_base(ctx, layer);
    hipStream_t s = static_cast<hipStream_t>(stream);
    const int d = c.d_model, E = c.n_experts;
    float* wrT = reinterpret_cast<float*>(lb);
    hipError_t e;
    if (src_on_device) {
        if (misaligned(wr) || (bias && misaligned(bias)))
            return fail(ctx, MOE_E_ALIGN, "device router pointers must be 16-byte aligned");
        e = timed(ctx, MOE_K_PACK, s, [&] { return moe_launch_transpose_router(wr, d, E, wrT, s); });
        if (e == hipSuccess && bias)
            e = hipMemcpyAsync(lb + ctx->L.bias_off, bias, (size_t)E * 4, hipMemcpyDeviceToDevice, s);
    } else {
        std::vector<float> tmp;
        try {
            tmp.resize((size_t)d * E);
        } catch (...) {
            return fail(ctx, MOE_E_ARG, "out of host memory for the router transpose");
        }
        for (int i = 0; i < d; ++i)
            for (int ee = 0; ee < E; ++ee) tmp[(size_t)ee * d + i] = wr[(size_t)i * E + ee];
        e = hipMemcpyAsync(wrT, tmp.data(), tmp.size() * 4, hipMemcpyHostToDevice, s);
        if (e == hipSuccess && bias)
            e = hipMemcpyAsync(lb + ctx->L.bias_off, bias, (size_t)E * 4, hipMemcpyHostToDevice, s);
        if (e == hipSuccess) e = hipStreamSynchronize(s);
    }
    if (e != hipSuccess) return hip_fail(ctx, e, "router load");
    if (ctx->route_layer == layer) ctx->route_valid = false;   // routed with the old router
    ctx->router_loaded[layer] = 1;
    ctx->has_bias[layer] = bias ? 1 : 0;
    return MOE_OK;
}

moe_status moe_route(moe_ctx* ctx, int32_t layer, const uint16_t* x, int32_t T,
                     const float* logits_in, moe_routing* out, moe_stream_t stream)
{
    if (!ctx) return MOE_E_ARG;
    if (!out) return fail(ctx, MOE_E_ARG, "out is NULL");
    if (layer < 0 || layer >= ctx->cfg.n_layers) return fail(ctx, MOE_E_ARG, "layer out of range");
    if (T < 0) return fail(ctx, MOE_E_ARG, "T is negative");
    if (T > ctx->cfg.max_tokens) return fail(ctx, MOE_E_CAPACITY, "T exceeds max_tokens");
    if (!ctx->router_loaded[layer]) return fail(ctx, MOE_E_STATE, "router of this layer not loaded");
    ctx->route_valid = false;
    if (T == 0) {
        fill_routing(ctx, layer, 0, out);
        return MOE_OK;
    }
    if (!logits_in) {
        if (!x) return fail(ctx, MOE_E_ARG, "x is NULL");
        if (misaligned(x)) return fail(ctx, MOE_E_ALIGN, "x must be 16-byte aligned");
    } else if (misaligned(logits_in)) {
        return fail(ctx, MOE_E_ALIGN, "logits_in must be 16-byte aligned");
    }
    moe_status st = do_route(ctx, ctx->ws, layer, x, T, logits_in, static_cast<hipStream_t>(stream));
    if (st != MOE_OK) return st;
    ctx->route_valid = true;
    ctx->route_layer = layer;
    ctx->route_T = T;
    ctx->route_x = logits_in ? nullptr : x;
    fill_routing(ctx, layer, T, out);
    return MOE_OK;
}

moe_status moe_forward(moe_ctx* ctx, int32_t layer, const uint16_t* x, int32_t T,
                       const moe_routing* r, void* y, moe_stream_t stream)
{
    if (!ctx) return MOE_E_ARG;
    if (T < 0) return fail(ctx, MOE_E_ARG, "T is negative");
    if (T > ctx->cfg.max_tokens) return fail(ctx, MOE_E_CAPACITY, "T exceeds max_tokens");
    moe_status st = check_layer(ctx, layer);
    if (st != MOE_OK) return st;
    if (T == 0) return MOE_OK;
    if (!x || !y) return fail(ctx, MOE_E_ARG, "x or y is NULL");
    if (misaligned(x) || misaligned(y)) return fail(ctx, MOE_E_ALIGN, "x and y must be 16-byte aligned");
    hipStream_t s = static_cast<hipStream_t>(stream);
    if (r) {
        if (!ctx->route_valid || r->T != T || r->layer != layer || r->logits != ctx->ws.rv.logits ||
            ctx->route_T != T || ctx->route_layer != layer)
            return fail(ctx, MOE_E_STATE,
                        "routing is not the current result of the last moe_route for this layer and T");
        if (ctx->route_x && ctx->route_x != x)
            return fail(ctx, MOE_E_STATE, "routing was computed from a different x");
    } else {
        ctx->route_valid = false;   // the views are about to be overwritten
        st = do_route(ctx, ctx->ws, layer, x, T, nullptr, s);
        if (st != MOE_OK) return st;
    }
    st = run_experts(ctx, ctx->ws, layer, x, T, s);
    if (st != MOE_OK) return st;
    const bool f32_out = (ctx->cfg.flags & MOE_PARTIAL_F32) != 0;
    return combine(ctx, ctx->ws, T, f32_out ? nullptr : static_cast<uint16_t*>(y),
                   f32_out ? static_cast<float*>(y) : nullptr, nullptr, s);
}

moe_status moe_forward_layers(moe_ctx* ctx, int32_t first, int32_t n, uint16_t* x_inout,
                              int32_t T, moe_stream_t stream)
{
    if (!ctx) return MOE_E_ARG;
    if (first < 0 || n < 0 || (int64_t)first + n > ctx->cfg.n_layers)
        return fail(ctx, MOE_E_ARG, "layer range outside [0, n_layers)");
    if (T < 0) return fail(ctx, MOE_E_ARG, "T is negative");
    if (T > ctx->cfg.max_tokens) return fail(ctx, MOE_E_CAPACITY, "T exceeds max_tokens");
    for (int l = first; l < first + n; ++l) {
        moe_status st = check_layer(ctx, l);
        if (st != MOE_OK) return st;
    }
    if (T == 0 || n == 0) return MOE_OK;
    if (!x_inout) return fail(ctx, MOE_E_ARG, "x is NULL");
    if (misaligned(x_inout)) return fail(ctx, MOE_E_ALIGN, "x must be 16-byte aligned");
    hipStream_t s = static_cast<hipStream_t>(stream);
    ctx->route_valid = false;   // the routing views are overwritten layer by layer
    for (int l = first; l < first + n; ++l) {
        moe_status st = do_route(ctx, ctx->ws, l, x_inout, T, nullptr, s);
        if (st != MOE_OK) return st;
        st = run_experts(ctx, ctx->ws, l, x_inout, T, s);
        if (st != MOE_OK) return st;
        st = combine(ctx, ctx->ws, T, nullptr, nullptr, x_inout, s);
        if (st != MOE_OK) return st;
    }
    return MOE_OK;
}

moe_status moe_forward_residual(moe_ctx* ctx, int32_t layer, const uint16_t* x, uint16_t* r_inout,
                                int32_t T, moe_stream_t stream)
{
    if (!ctx) return MOE_E_ARG;
    if (layer < 0 || layer >= ctx->cfg.n_layers) return fail(ctx, MOE_E_ARG, "layer out of range");
    if (T < 0) return fail(ctx, MOE_E_ARG, "T is negative");
    if (T > ctx->cfg.max_tokens) return fail(ctx, MOE_E_CAPACITY, "T exceeds max_tokens");
    moe_status st = check_layer(ctx, layer);
    if (st != MOE_OK) return st;
    if (T == 0) return MOE_OK;
    if (!x || !r_inout) return fail(ctx, MOE_E_ARG, "x or r is NULL");
    if (misaligned(x) || misaligned(r_inout)) return fail(ctx, MOE_E_ALIGN, "x and r must be 16-byte aligned");
    hipStream_t s = static_cast<hipStream_t>(stream);
    ctx->route_valid = false;   // the routing views are about to be overwritten
    st = do_route(ctx, ctx->ws, layer, x, T, nullptr, s);
    if (st != MOE_OK) return st;
    st = run_experts(ctx, ctx->ws, layer, x, T, s);
    if (st != MOE_OK) return st;
    return combine(ctx, ctx->ws, T, nullptr, nullptr, r_inout, s);
}

moe_status moe_forward_stack(moe_ctx* ctx, uint16_t* x_inout, int32_t T, moe_stream_t stream)
{
    if (!ctx) return MOE_E_ARG;
    return moe_forward_layers(ctx, 0, ctx->cfg.n_layers, x_inout, T, stream);
}

moe_status moe_forward_static(moe_ctx* ctx, int32_t layer, const uint16_t* x, int32_t T, void* y,
                              moe_stream_t stream)
{
    if (!ctx) return MOE_E_ARG;
    if (T < 0) return fail(ctx, MOE_E_ARG, "T is negative");
    if (T > ctx->cfg.max_tokens) return fail(ctx, MOE_E_CAPACITY, "T exceeds max_tokens");
    moe_status st = check_layer(ctx, layer);
    if (st != MOE_OK) return st;
    if (T == 0) return MOE_OK;
    if (!x || !y) return fail(ctx, MOE_E_ARG, "x or y is NULL");
    if (misaligned(x) || misaligned(y)) return fail(ctx, MOE_E_ALIGN, "x and y must be 16-byte aligned");
    // the workspace layout of this T, carved from the static scratch
    moe_config c = ctx->cfg;
    c.max_tokens = T;
    const Layout L = make_layout(&c);
    if (L.ws_bytes > MOE_STATIC_SCRATCH_BYTES)
        return fail(ctx, MOE_E_CAPACITY,
                    "T needs " + std::to_string(L.ws_bytes) + " bytes of scratch; the static scratch holds " +
                        std::to_string((size_t)MOE_STATIC_SCRATCH_BYTES));
    uint8_t* base = nullptr;
    st = scratch_ptr(ctx, &base);
    if (st != MOE_OK) return st;
    const WsView ws = make_ws_view(base, L);
    hipStream_t s = static_cast<hipStream_t>(stream);
    st = do_route(ctx, ws, layer, x, T, nullptr, s);
    if (st != MOE_OK) return st;
    st = run_experts(ctx, ws, layer, x, T, s);
    if (st != MOE_OK) return st;
    const bool f32_out = (ctx->cfg.flags & MOE_PARTIAL_F32) != 0;
    return combine(ctx, ws, T, f32_out ? nullptr : static_cast<uint16_t*>(y),
                   f32_out ? static_cast<float*>(y) : nullptr, nullptr, s);
}

moe_status moe_intermediates(const moe_ctx* ctx, const uint16_t** h, const float** o)
{
    if (!ctx) return MOE_E_ARG;
    if (h) *h = reinterpret_cast<const uint16_t*>(ctx->ws.base + ctx->ws.h_off);
    if (o) *o = reinterpret_cast<const float*>(ctx->ws.base + ctx->ws.o_off);
    return MOE_OK;
}

moe_status moe_profile_enable(moe_ctx* ctx, int32_t max_launches)
{
    if (!ctx) return MOE_E_ARG;
    if (max_launches < 0) return fail(ctx, MOE_E_ARG, "max_launches is negative");
    for (hipEvent_t ev : ctx->prof_events) (void)hipEventDestroy(ev);
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

moe_status moe_profile_gemm_timeline(moe_ctx* ctx, uint64_t* gateup, uint64_t* down,
                                     int32_t max_wg)
{
    if (!ctx) return MOE_E_ARG;
    if (max_wg < 0) return fail(ctx, MOE_E_ARG, "max_wg is negative");
    if ((gateup && misaligned(gateup)) || (down && misaligned(down)))
        return fail(ctx, MOE_E_ALIGN, "timeline buffers must be 16-byte aligned");
    ctx->tl_gateup = max_wg ? gateup : nullptr;
    ctx->tl_down = max_wg ? down : nullptr;
    ctx->tl_max = max_wg;
    return MOE_OK;
}

moe_status moe_profile_read(moe_ctx* ctx, double* total_ms, int64_t* launches, int64_t* dropped)
{
    if (!ctx) return MOE_E_ARG;
    if (!total_ms || !launches) return fail(ctx, MOE_E_ARG, "output array is NULL");
    for (int k = 0; k < MOE_K_COUNT; ++k) { total_ms[k] = 0.0; launches[k] = 0; }
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

void moe_destroy(moe_ctx* ctx)
{
    if (!ctx) return;
    for (hipEvent_t ev : ctx->prof_events)
        if (ev) (void)hipEventDestroy(ev);
    delete ctx;
}

const char* moe_last_error(const moe_ctx* ctx)
{
    return ctx ? ctx->err.c_str() : g_init_error.c_str();
}

const char* moe_status_string(moe_status s)
{
    switch (s) {
    case MOE_OK: return "MOE_OK";
    case MOE_E_ARG: return "MOE_E_ARG";
    case MOE_E_SHAPE: return "MOE_E_SHAPE";
    case MOE_E_ALIGN: return "MOE_E_ALIGN";
    case MOE_E_CAPACITY: return "MOE_E_CAPACITY";
    case MOE_E_STATE: return "MOE_E_STATE";
    case MOE_E_HIP: return "MOE_E_HIP";
    }
    return "unknown";
}

}  // extern "C"
