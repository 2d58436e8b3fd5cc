/*
 * moe.h -- C-ABI of the MI355X (gfx950) DBRX-style Mixture-of-Experts layer.
 *
 * The layer (Chen et al., RACS'24, "Towards Building Private LLMs: Exploring
 * Multi-Node Expert Parallelism on Apple Silicon for Mixture-of-Experts Large
 * Language Model"):
 *   - Sec. 2.1: each decoder layer holds 16 FFN experts, of which the router
 *     selects 4 per token;
 *   - Sec. 2.2: the selected experts' outputs are combined by a weighted sum;
 *   - Table tab:vars note (e): an expert is three D_embed x D_ffn matrices
 *     v1, w1, w2 (here: w1 = gate with SiLU, v1 = up, w2 = down);
 *   - Sec. 3.1 / Sec. 4.3: under expert parallelism each node holds a subset
 *     of the experts, the router is replicated, and each node returns the
 *     partial weighted sum of its local experts (an all-reduce adds them).
 *   - Sec. 4.1: the weights of an expert are prestacked once into one
 *     persistent array and indexed per layer; here moe_init takes one
 *     caller-allocated weight arena and one workspace, and no call after it
 *     allocates device memory.
 *
 * Per token t with bf16 input x[t, 0:d]:
 *   logits[t,e] = fp32(sum_i x[t,i] * wr[i,e]) (+ bias[e], added in fp32)
 *   S_t         = the k experts with the largest logits (ties: lower id),
 *                 slot order = logit descending, id ascending
 *   w[t,j]      = softmax over the k selected logits
 *   h_j         = bf16( silu(x W1_j) * (x V1_j) )              [f]
 *   o_j         = h_j W2_j  (fp32 accumulation)                 [d]
 *   y[t]        = bf16( sum over local slots j of w[t,j] * o_j )
 * The stacked form chains layers as x_next = bf16(x + y).
 *
 * Conventions for every entry point
 *   - bf16 tensors are passed as uint16_t bit patterns.
 *   - Tensor pointers are HIP device pointers unless a parameter says host;
 *     the caller owns them.  Device tensor pointers must be 16-byte aligned.
 *   - stream is a hipStream_t handle (NULL = the default stream).  MOE_OK
 *     means the work was enqueued on that stream; device-side faults surface
 *     as HIP errors at the caller's next synchronisation.
 *   - Every argument is validated on the host before anything is launched; a
 *     failing call enqueues nothing, returns a negative moe_status and
 *     records a message readable through moe_last_error().  Nothing throws
 *     or aborts across this interface.
 *   - A context is used by one host thread and one stream at a time.
 */
#ifndef MOE_H
#define MOE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#if defined(__GNUC__)
#define MOE_API __attribute__((visibility("default")))
#else
#define MOE_API
#endif

typedef struct moe_ctx moe_ctx;
typedef void *moe_stream_t; /* a hipStream_t */

typedef enum {
    MOE_OK = 0,
    MOE_E_ARG = -1,      /* null/invalid pointer or out-of-range index */
    MOE_E_SHAPE = -2,    /* config or size not supported */
    MOE_E_ALIGN = -3,    /* device pointer not 16-byte aligned */
    MOE_E_CAPACITY = -4, /* T above the config's max_tokens */
    MOE_E_STATE = -5,    /* call out of order (e.g. forward before load) */
    MOE_E_HIP = -6       /* a HIP runtime call failed */
} moe_status;

/* Configuration flags (moe_config.flags). */
#define MOE_PARTIAL_F32 0x1 /* moe_forward writes y as fp32 [T, d], unrounded
                               (an expert-parallel share's partial sum that a
                               cross-device all-reduce adds, Sec. 4.3) */

/* Layer configuration.
 *   d_model, ffn_dim : D_embed and D_ffn (Table tab:vars: 6144 and 10752).
 *                      d_model must be a multiple of 256, ffn_dim of 128.
 *   n_experts, top_k : E and k (Sec. 2.1: 16 and 4); 1 <= k <= E <= 64.
 *   expert_begin, n_local_experts : the experts resident on this device,
 *                      [expert_begin, expert_begin + n_local_experts).  The
 *                      whole layer is 0, n_experts; a node's expert-parallel
 *                      share is a sub-range (Sec. 3.1, Sec. 4.3).
 *   n_layers         : layers held in the arena (>= 1).
 *   max_tokens       : largest T any call will pass; sizes the workspace.
 *                      max_tokens * d_model * 2 must stay below 2^31.
 *   d_model * ffn_dim * 4 (one expert's packed gate/up bytes) must stay
 *                      below 2^31.
 *   flags            : 0 or MOE_PARTIAL_F32; any other bit is rejected. */
typedef struct {
    int32_t d_model, ffn_dim, n_experts, top_k;
    int32_t expert_begin, n_local_experts;
    int32_t n_layers, max_tokens;
    int32_t flags;
} moe_config;

/* Routing of the last moe_route / moe_forward call on a context.  Every
 * pointer is a device view into the workspace, valid until the next
 * moe_route / moe_forward / moe_forward_stack / moe_forward_layers on the
 * same context.
 *   logits   fp32 [T, E]      topk_idx int32 [T, k]   topk_w fp32 [T, k]
 *   counts   int32 [E]        pairs routed to each local expert (0 off-share)
 *   offsets  int32 [E + 1]    exclusive prefix sum of counts
 *   pair_row int32 [T, k]     row of pair (t, j) in expert-grouped order, or
 *                             -1 when its expert is not local
 *   row_token int32 [offsets[E]]  token of each grouped row
 * Rows are grouped by expert ascending, then token ascending. */
typedef struct {
    float *logits;
    int32_t *topk_idx;
    float *topk_w;
    int32_t *counts;
    int32_t *offsets;
    int32_t *pair_row;
    int32_t *row_token;
    int32_t T;
    int32_t layer;
} moe_routing;

/* Bytes of the persistent weight arena / workspace for cfg (0 if cfg is
 * invalid).  The arena holds, per layer, the router (fp32) and every local
 * expert's three matrices repacked into the kernels' tiled layout (Sec. 4.1:
 * the weights are stacked once into one persistent array). */
MOE_API size_t moe_weight_bytes(const moe_config *cfg);
MOE_API size_t moe_workspace_bytes(const moe_config *cfg);

/* Sec. 4.1 (prestacking: buffers set up once, so that no call afterwards
 * pays for memory management) and Sec. 3.1 / Sec. 4.3 (a node holds a range
 * of the experts).  Validates cfg, records the caller-allocated device
 * buffers (sizes from the functions above, both 256-byte aligned; they must
 * stay allocated and unmoved until moe_destroy) and returns a new context in
 * *out.  Allocates only the host-side context.  Errors: MOE_E_SHAPE for an
 * invalid cfg, MOE_E_ARG for a NULL buffer or out, MOE_E_ALIGN; *out is then
 * NULL and moe_last_error(NULL) holds the reason.
 * The weight stream is sensitive to where the arena lands: measured, an arena
 * placed in memory that earlier allocations had used and freed streams 2-4 %
 * slower than one carved from a single large allocation made up front. */
MOE_API moe_status moe_init(const moe_config *cfg, void *weight_arena, void *workspace,
                    moe_ctx **out);

/* Prestacking (Sec. 4.1): repacks one local expert of one layer into the
 * arena.  gate and up are [d, f] row-major (x gate gives the gate
 * pre-activation), down is [f, d] row-major, all bf16.  src_on_device != 0:
 * the three pointers are device memory and the repack is a kernel enqueued
 * on stream; 0: they are host memory, repacked on the host and copied
 * synchronously (the call returns after the copy).  expert is a global id
 * inside the local range. */
MOE_API moe_status moe_load_expert(moe_ctx *ctx, int32_t layer, int32_t expert,
                           const uint16_t *gate, const uint16_t *up,
                           const uint16_t *down, int32_t src_on_device,
                           moe_stream_t stream);

/* Sec. 3.1 and Sec. 4.3 (the router decides where each token goes; every
 * node holds a full copy of it).  Loads one layer's router: wr fp32 [d, E]
 * row-major, bias fp32 [E] or NULL (no bias).  Same src_on_device rule as
 * moe_load_expert.  A routing returned for this layer before the call is no
 * longer accepted by moe_forward. */
MOE_API moe_status moe_load_router(moe_ctx *ctx, int32_t layer, const float *wr,
                           const float *bias, int32_t src_on_device,
                           moe_stream_t stream);

/* Sec. 2.1 (the router selects 4 of the 16 experts per token), Sec. 3.1
 * (its output decides which experts, and so which nodes, receive a token).
 * Router, selection and permutation for T tokens of x (bf16 [T, d]).  If
 * logits_in (fp32 [T, E], device) is not NULL it is routed as given and the
 * router product is skipped (x may then be NULL).  On MOE_OK, *out describes
 * the routing (views into the workspace).  T == 0 is a no-op that reports an
 * empty routing.  Errors: MOE_E_ARG (layer, T < 0, NULL out or x),
 * MOE_E_CAPACITY (T > max_tokens), MOE_E_STATE (router not loaded),
 * MOE_E_ALIGN. */
MOE_API moe_status moe_route(moe_ctx *ctx, int32_t layer, const uint16_t *x, int32_t T,
                     const float *logits_in, moe_routing *out,
                     moe_stream_t stream);

/* Sec. 2.1 (the selected experts are GLU FFNs, Table tab:vars (e)), Sec. 2.2
 * (their outputs are combined by a weighted sum), Sec. 4.3 (a node computes
 * only its local experts and returns their partial sum).
 * The layer: y = weighted sum of the local selected experts, bf16 [T, d], or
 * fp32 [T, d] (unrounded) when the config has MOE_PARTIAL_F32.  If r is NULL
 * the routing is computed first (as moe_route with NULL logits_in);
 * otherwise r must be the routing that the last moe_route on this context
 * returned, for the same layer and T, and -- if it was computed from x rather
 * than given logits -- the same x; a forward with internal routing, a stack
 * forward or a moe_load_router of that layer in between invalidates it
 * (MOE_E_STATE).  For an expert-parallel share, y is the partial sum of the
 * local slots (zero rows for tokens with no local slot).  Requires the
 * layer's router and local experts loaded (MOE_E_STATE otherwise). */
MOE_API moe_status moe_forward(moe_ctx *ctx, int32_t layer, const uint16_t *x,
                       int32_t T, const moe_routing *r, void *y,
                       moe_stream_t stream);

/* For callers that cannot allocate device memory when they call (code under
 * HIP graph capture, tight serving loops, harnesses that forbid allocation).
 * Same as moe_forward(ctx, layer, x, T, NULL, y, stream) -- routing, experts
 * and combine; y bf16 [T, d], or fp32 with MOE_PARTIAL_F32 -- but the
 * routing arrays and the intermediates H and O live in a static device array
 * of MOE_STATIC_SCRATCH_BYTES that the library holds on each GPU it runs on
 * until the process ends, not in the context's workspace.  The call leaves
 * the workspace untouched (a routing from moe_route stays valid) and calls no
 * allocating routine.  T is limited by max_tokens and by the scratch: the
 * workspace that moe_workspace_bytes reports for max_tokens = T must fit in
 * MOE_STATIC_SCRATCH_BYTES (T <= 40 at d 6144, f 10752, 16 experts, top-4);
 * beyond either, MOE_E_CAPACITY and nothing is enqueued.  The context's
 * device must be current.  Every call on a GPU shares that GPU's array and
 * leaves its contents behind: calls that overlap on one GPU (two streams, two
 * host threads) race and must be ordered by the caller.  The first call on a
 * device looks up the array's device address (a runtime query, no
 * allocation); its failure returns MOE_E_HIP. */
#define MOE_STATIC_SCRATCH_BYTES (8u << 20)
MOE_API moe_status moe_forward_static(moe_ctx *ctx, int32_t layer, const uint16_t *x,
                                      int32_t T, void *y, moe_stream_t stream);

/* Sec. 4.1 (all layers' experts resident in one prestacked array, indexed
 * per layer) and Sec. 2.1 (one MoE FFN per decoder layer).  All n_layers
 * layers in order on T tokens, in place: for each layer l,
 * x = bf16(x + layer_l(x)), always bf16 (MOE_PARTIAL_F32 does not apply).
 * x_inout is bf16 [T, d].  Requires every layer loaded (MOE_E_STATE). */
MOE_API moe_status moe_forward_stack(moe_ctx *ctx, uint16_t *x_inout, int32_t T,
                             moe_stream_t stream);

/* Sec. 2.1 (a decoder layer is self-attention followed by the MoE FFN): the
 * same as moe_forward_stack for the n consecutive layers first .. first+n-1
 * only, so that a caller can interleave other blocks (the self-attention of
 * attn.h) between MoE layers: for each of them x = bf16(x + layer_l(x)), in
 * place, bf16 [T, d].  moe_forward_stack(ctx, x, T, s) is
 * moe_forward_layers(ctx, 0, n_layers, x, T, s).  Requires 0 <= first,
 * n >= 0, first + n <= n_layers (MOE_E_ARG) and those layers loaded
 * (MOE_E_STATE); n == 0 or T == 0 is a no-op. */
MOE_API moe_status moe_forward_layers(moe_ctx *ctx, int32_t first, int32_t n, uint16_t *x_inout,
                                      int32_t T, moe_stream_t stream);

/* Sec. 2.1's decoder layer with the FFN fed a normalised input: layer
 * `layer` on x (bf16 [T, d], routed and computed as moe_forward), its output
 * added into the residual stream r_inout = bf16(r_inout + bf16(y)) in place
 * (bf16 [T, d]; r_inout may be x, which is then one layer of
 * moe_forward_layers).  Errors as moe_forward_layers. */
MOE_API moe_status moe_forward_residual(moe_ctx *ctx, int32_t layer, const uint16_t *x,
                                        uint16_t *r_inout, int32_t T, moe_stream_t stream);

/* Workspace map for a caller that owns the workspace and wants to inspect or
 * guard its parts: region i (moe_ws_region order) starts offset[i] bytes
 * into the workspace and holds bytes[i] bytes; the gaps between regions
 * (alignment padding) are never written.  Fills min(n, MOE_WS_COUNT)
 * entries and returns MOE_WS_COUNT, or 0 if cfg is invalid. */
typedef enum {
    MOE_WS_ROUTE_PARTIALS = 0, /* fp64 partial logits of the small-T router */
    MOE_WS_LOGITS, MOE_WS_TOPK_IDX, MOE_WS_TOPK_W, MOE_WS_COUNTS, MOE_WS_OFFSETS,
    MOE_WS_PAIR_ROW, MOE_WS_ROW_TOKEN,
    MOE_WS_ACTIVE,             /* int32 [1 + E]: #active local experts, their ids */
    MOE_WS_TILES,              /* int32 [max_tiles][2]: GEMM token tiles */
    MOE_WS_N_TILES,            /* int32 [1] */
    MOE_WS_H,                  /* bf16 [rows_max, f] */
    MOE_WS_O,                  /* fp32 [rows_max, d] */
    MOE_WS_COUNT
} moe_ws_region;
MOE_API int32_t moe_workspace_map(const moe_config *cfg, uint64_t *offset, uint64_t *bytes,
                                  int32_t n);

/* Introspection for tests: device pointers to the intermediates of the last
 * forward on ctx, valid until the next forward.  h: bf16 [rows, f], the
 * SiLU-gated activations of each grouped row; o: fp32 [rows, d], each grouped
 * row's expert output before the routing weight.  Rows follow the routing's
 * pair_row / offsets.  Either pointer may be NULL. */
MOE_API moe_status moe_intermediates(const moe_ctx *ctx, const uint16_t **h,
                             const float **o);

/* Per-kernel timing for measurement harnesses.  moe_profile_enable(ctx, n)
 * with n > 0 creates 2n HIP events and from then on brackets each kernel
 * launch of the context with an event pair on the launch stream (at most n
 * launches between reads; later ones run untimed and are counted as
 * dropped); n == 0 turns timing off and frees the events.
 * moe_profile_read waits for the recorded launches, writes per kind the total
 * milliseconds and the launch count (arrays of MOE_K_COUNT), the number of
 * dropped launches (may be NULL), and starts a new recording. */
typedef enum {
    MOE_K_ROUTER = 0,        /* router logits, fp64 partial sums */
    MOE_K_ROUTE = 1,         /* selection, weights, permutation */
    MOE_K_DECODE_GATEUP = 2, /* small-T gate/up + SiLU */
    MOE_K_DECODE_DOWN = 3,   /* small-T down projection */
    MOE_K_GEMM_GATEUP = 4,   /* grouped GEMM gate/up + SiLU */
    MOE_K_GEMM_DOWN = 5,     /* grouped GEMM down projection */
    MOE_K_COMBINE = 6,       /* weighted combine (and residual) */
    MOE_K_PACK = 7,          /* expert prestacking */
    MOE_K_COUNT = 8
} moe_kernel_kind;
MOE_API moe_status moe_profile_enable(moe_ctx *ctx, int32_t max_launches);
MOE_API moe_status moe_profile_read(moe_ctx *ctx, double *total_ms,
                                    int64_t *launches, int64_t *dropped);

/* Measurement: a per-workgroup timeline of the grouped GEMMs (T > 16).
 * With buffers set (device, uint64 [max_wg][8] each, zeroed by the caller;
 * either may be NULL), every later forward on ctx that takes the GEMM path
 * records, for each GEMM workgroup b < max_wg that has a tile: [0], [1] the
 * constant 100 MHz counter at the tile's start and end, [2], [3] the shader
 * clock counter at start and end (so [3]-[2] over ([1]-[0]) / 1e8 s is the
 * clock the tile ran at), [4] HW_ID | XCC_ID << 32 of its CU, [5] feature
 * tile | token tile << 16 | rows << 32 | expert << 48.  Workgroups without a
 * tile leave their entry untouched.  max_wg == 0 turns it off.  The
 * recording adds one barrier per workgroup. */
MOE_API moe_status moe_profile_gemm_timeline(moe_ctx *ctx, uint64_t *gateup, uint64_t *down,
                                             int32_t max_wg);

/* Frees the host-side context and its profiling events (never the caller's
 * device buffers). */
MOE_API void moe_destroy(moe_ctx *ctx);

/* Message of the last failing call on ctx ("" if none); with ctx == NULL,
 * the message of the last failing moe_init on this thread. */
MOE_API const char *moe_last_error(const moe_ctx *ctx);

/* Static name of a status code. */
MOE_API const char *moe_status_string(moe_status s);

/* Diagnostics, beside the layer: one plain streaming read of `bytes` bytes of
 * device memory at src, every 16-byte word loaded once (nontemporal, 1 KiB
 * contiguous per wave-load, the decode GEMVs' pattern), to measure the HBM
 * read rate the layer's weight streams can reach on this device.  So that no
 * load is dead, workgroup b (of at most MOE_DIAG_MAX_WG) writes the XOR of
 * the words it read to out[4b .. 4b+3] (device, MOE_DIAG_MAX_WG x 4 uint32,
 * zeroed by the caller: the XOR of all of out is then the buffer's XOR).
 * Enqueued on stream; allocates nothing.  src and out 16-byte aligned and
 * bytes a multiple of 16, else MOE_E_ARG (nothing enqueued); bytes == 0
 * enqueues nothing. */
#define MOE_DIAG_MAX_WG 512
MOE_API moe_status moe_diag_stream_read(const void *src, uint64_t bytes, uint32_t *out,
                                        moe_stream_t stream);

/* Diagnostics: dst[i] = bf16(src[i]) for i < n by the hardware conversion
 * that the grouped GEMM's gate/up epilogue applies to H (R5: round to
 * nearest even; a NaN stays a NaN), so that a test can hold it against the
 * integer rounding on every fp32 pattern.  src fp32 [n] and dst bf16 [n],
 * device memory; src 8-byte and dst 4-byte aligned and n even, else
 * MOE_E_ARG (nothing enqueued); n == 0 enqueues nothing.  Enqueued on
 * stream; allocates nothing. */
MOE_API moe_status moe_diag_bf16(const float *src, uint16_t *dst, uint64_t n, moe_stream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* MOE_H */
