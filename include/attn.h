/*
 * attn.h -- C-ABI of the MI355X (gfx950) DBRX-style self-attention block, the
 * other half of a decoder layer beside the MoE FFN of moe.h (Chen et al.,
 * RACS'24: Sec. 2.1 and its decoder-layer figure -- self-attention then the
 * MoE FFN; Table tab:vars -- D_embed 6144, D_qkv_hidden 8192, and note (b):
 * a D_qkv_hidden x D_embed fused query/key/value projection plus a
 * D_embed x D_embed output projection per layer; Sec. 4.3 -- the block is
 * replicated on every node, so one device computes it whole).
 *
 * For T new tokens at positions pos0 .. pos0+T-1 of one sequence, per layer:
 *   h      = bf16( (x - mean) / sqrt(var + eps) * gamma )        layer norm
 *   q|k|v  = h Wqkv   (n_heads, n_kv_heads, n_kv_heads heads of head_dim)
 *   q, k   rotated by position (rotary encoding, pairs i and i + head_dim/2,
 *          angle pos * theta^(-2i/head_dim)), then q, k, v rounded to bf16;
 *          k and v are appended to the layer's cache
 *   a_j    = bf16( softmax_p(q_j . k_p / sqrt(head_dim)) v_p ), p over
 *          positions 0 .. pos of the token; query head j uses key/value head
 *          j / (n_heads / n_kv_heads)
 *   o      = a Wo (fp32)           y = bf16(x + o)
 * The paper fixes the widths; the head split, the norm, the rotary encoding
 * and the rounding points are this library's readings.
 *
 * Conventions are those of moe.h: bf16 as uint16_t bits, device pointers
 * owned by the caller and 16-byte aligned, work enqueued on `stream`, every
 * argument checked on the host before any launch, a moe_status returned and
 * a message kept for attn_last_error.  A context is used by one host thread
 * and one stream at a time.
 */
#ifndef ATTN_H
#define ATTN_H

#include "moe.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef struct attn_ctx attn_ctx;

/* Block configuration.
 *   d_model    : D_embed, a multiple of 256, at most 8192.
 *   n_heads, n_kv_heads, head_dim : query heads, key/value heads (dividing
 *                n_heads) and their width, 64 or 128; (n_heads + 2
 *                n_kv_heads) head_dim is D_qkv_hidden, a multiple of 16, and
 *                n_heads head_dim a multiple of 256.
 *   n_layers   : layers held in the weight arena and the cache (>= 1).
 *   max_seq    : cache positions per layer (>= 1).
 *   max_tokens : largest T of a call, 1 .. 32768.  Up to 16 tokens a call
 *                takes the decode path (weight-streaming GEMVs, attention
 *                over position chunks); above, the prefill path (matrix-core
 *                GEMMs for the projections, causal attention on the matrix
 *                cores), which needs (n_heads + 2 n_kv_heads) head_dim to be
 *                a multiple of 256 when max_tokens > 16.
 *   rope_theta : base of the rotary frequencies (> 1).
 *   norm_eps   : layer-norm epsilon (>= 0).
 *   flags      : must be 0. */
typedef struct {
    int32_t d_model, n_heads, n_kv_heads, head_dim;
    int32_t n_layers, max_seq, max_tokens;
    float rope_theta, norm_eps;
    int32_t flags;
} attn_config;

/* Bytes of the caller-allocated weight arena (per layer: gamma fp32 [d]
 * padded to 256 B, the rotary frequencies fp64 [head_dim/2] padded to 256 B,
 * the post-attention norm's gamma2 fp32 [d] padded to 256 B,
 * then Wqkv and Wo repacked into the fragment-tiled layout
 * of moe.h's experts, the query and key rows of Wqkv reordered within each
 * head so that the two members of every rotation pair share a 16-row tile),
 * of the key/value cache, and of the workspace (which, when max_tokens > 16,
 * also holds a small tile table that attn_init writes); 0 if cfg is
 * invalid.  Cache layout, per layer l: K then V, each bf16
 * [n_kv_heads][max_seq][head_dim] (head-major, positions contiguous), so K of
 * layer l head g position p starts at element
 * ((l * 2 + 0) * n_kv_heads + g) * max_seq * head_dim + p * head_dim.  A
 * caller may write earlier positions' keys and values there directly. */
MOE_API size_t attn_weight_bytes(const attn_config *cfg);
MOE_API size_t attn_cache_bytes(const attn_config *cfg);
MOE_API size_t attn_workspace_bytes(const attn_config *cfg);

/* Sec. 4.1's persistent buffers, applied to the block: validates cfg and
 * records the three caller-allocated device buffers (256-byte aligned, kept
 * until attn_destroy).  Allocates only the host-side context; when
 * max_tokens > 16 it also copies the prefill tile table into the workspace
 * (a synchronous copy; MOE_E_HIP if it fails).  Errors as moe_init; the
 * message is readable through attn_last_error(NULL). */
MOE_API moe_status attn_init(const attn_config *cfg, void *weight_arena, void *kv_cache,
                             void *workspace, attn_ctx **out);

/* Table tab:vars note (b): loads one layer's weights, repacking them once
 * into the arena.  gamma fp32 [d]; wqkv bf16 [d][(n_heads + 2 n_kv_heads)
 * head_dim] row-major (h wqkv gives q | k | v, heads in order); wo bf16
 * [n_heads head_dim][d] row-major (a wo gives o).  src_on_device as in
 * moe_load_expert (1: device pointers, kernels enqueued on stream; 0: host
 * pointers, repacked on the host and copied before returning). */
MOE_API moe_status attn_load_layer(attn_ctx *ctx, int32_t layer, const float *gamma,
                                   const uint16_t *wqkv, const uint16_t *wo,
                                   int32_t src_on_device, moe_stream_t stream);

/* Sec. 2.1 / Sec. 4.3: the block on T tokens x (bf16 [T, d]) at positions
 * pos0 .. pos0+T-1 of layer `layer`'s cache, which must already hold
 * positions 0 .. pos0-1; writes the tokens' keys and values at their
 * positions and y = bf16(x + o) (bf16 [T, d]; y may be x).  Requires
 * 1 <= T <= max_tokens (T == 0: no-op), pos0 >= 0, pos0 + T <= max_seq
 * (MOE_E_CAPACITY otherwise) and the layer loaded (MOE_E_STATE). */
MOE_API moe_status attn_forward(attn_ctx *ctx, int32_t layer, const uint16_t *x, uint16_t *y,
                                int32_t T, int32_t pos0, moe_stream_t stream);

/* The post-attention norm of a DBRX decoder layer (its attention part is
 * norm, attention, norm; Sec. 2.1's decoder layer feeds the MoE FFN the
 * block's output): loads gamma2 fp32 [d] of layer `layer` (src_on_device as
 * attn_load_layer). */
MOE_API moe_status attn_load_post_norm(attn_ctx *ctx, int32_t layer, const float *gamma2,
                                       int32_t src_on_device, moe_stream_t stream);

/* attn_forward, then z = bf16((y - mean) / sqrt(var + eps) * gamma2) (bf16
 * [T, d]), the normalised input of the layer's MoE FFN; z may be y.
 * Requires attn_load_post_norm of the layer (MOE_E_STATE). */
MOE_API moe_status attn_forward_norm(attn_ctx *ctx, int32_t layer, const uint16_t *x, uint16_t *y,
                                     uint16_t *z, int32_t T, int32_t pos0, moe_stream_t stream);

/* Introspection for tests: device pointers into the workspace with the last
 * forward's intermediates, valid until the next forward: h bf16 [T, d],
 * qkv fp32 [T, (n_heads + 2 n_kv_heads) head_dim] (before rotation), q bf16
 * [T, n_heads head_dim] (rotated), a bf16 [T, n_heads head_dim] (attention
 * output), o fp32 [T, d].  Any pointer may be NULL. */
MOE_API moe_status attn_intermediates(const attn_ctx *ctx, const uint16_t **h, const float **qkv,
                                      const uint16_t **q, const uint16_t **a, const float **o);

/* Per-kernel timing, as moe_profile_enable / moe_profile_read, with the
 * kinds of attn_kernel_kind. */
typedef enum {
    ATTN_K_NORM = 0,       /* layer norm */
    ATTN_K_QKV = 1,        /* fused projection (+ rotary + cache append in decode) */
    ATTN_K_SCORE = 2,      /* attention (over position chunks in decode, causal in prefill) */
    ATTN_K_COMBINE = 3,    /* merge of the chunks (decode) */
    ATTN_K_OUT = 4,        /* output projection (+ residual in decode) */
    ATTN_K_PACK = 5,       /* weight repacking */
    ATTN_K_ROPE = 6,       /* rotary + cache append (prefill) */
    ATTN_K_RESIDUAL = 7,   /* y = bf16(x + o) (prefill) */
    ATTN_K_POST_NORM = 8,  /* z = norm(y) (attn_forward_norm) */
    ATTN_K_COUNT = 9
} attn_kernel_kind;
MOE_API moe_status attn_profile_enable(attn_ctx *ctx, int32_t max_launches);
MOE_API moe_status attn_profile_read(attn_ctx *ctx, double *total_ms, int64_t *launches,
                                     int64_t *dropped);

/* Frees the host-side context (never the caller's buffers). */
MOE_API void attn_destroy(attn_ctx *ctx);

/* Message of the last failing call on ctx; with ctx == NULL, of the last
 * failing attn_init on this thread. */
MOE_API const char *attn_last_error(const attn_ctx *ctx);

#ifdef __cplusplus
}
#endif

#endif /* ATTN_H */
