// moe_prefill.hip -- the expert FFN for many tokens (prefill): a grouped GEMM
// on the bf16 matrix cores (v_mfma_f32_32x32x16_bf16).
//
// A workgroup computes a BM x BN = 256 x 256 tile of C = W X^T for one
// expert: W (the A operand) is 256 output features of the expert's packed
// weights, X (the B operand) is 256 of the expert's token rows (K
// contiguous).  Four waves split the features (4 x 64); each wave owns a
// 64-feature x 256-token block (2 x 8 MFMA blocks of 32 x 32, all 256
// accumulator registers), so each weight slab is re-read by only
// ceil(tokens / 256) workgroups.  One workgroup per CU (128 KiB of LDS),
// one wave per SIMD: latency is hidden by software pipelining alone.
//
//  - A never touches LDS: the packed layout already holds every 32 x 16
//    fragment as 1 KiB in lane order, each fragment is used by exactly one
//    wave, and the wave loads it straight into registers through a ring of
//    three 64-wide K stages.
//  - B (the gathered token rows, shared by all four waves) goes from HBM to
//    LDS by buffer loads with the LDS-direct option, four stages deep; each
//    load reads whole 128-byte lines and the chunks of each row are
//    XOR-swizzled in LDS so that the fragment reads are conflict-free.  The
//    fragments are read into a small register window a few MFMAs ahead,
//    also across stage boundaries.
//  - An expert's partial last token tile skips the MFMAs of token-block
//    pairs past its last row (the padding waste is under 64 rows).
//  - Workgroups are numbered so that consecutive tiles (same weight slab,
//    consecutive token tiles) land on the same XCD and share its L2.
//
// gemm<kGateUp>: A = GU slab (gate and up row tiles interleaved), X = the
//   expert's rows of x gathered through row_token; epilogue
//   H = bf16(silu(G) * U) (paper Table tab:vars (e): w1 gate, v1 up).
// gemm<kDown>:   A = DN slab, X = the expert's rows of H; epilogue O fp32.
//
// Token tiles (expert, first grouped row) come from the routing kernel; the
// grid is sized for the worst case and surplus workgroups exit at once.
#include <type_traits>

#include "moe_common.h"

namespace moe {

constexpr int BM = 256;         // features per workgroup tile
constexpr int BN = 256;         // token rows per workgroup tile
constexpr int BK = 64;          // K per stage (four 16-K MFMA steps)
constexpr int kThreads = 256;   // 4 waves, one per 64-feature slab
constexpr int FB = 2;           // 32-feature MFMA blocks per wave
constexpr int kWaveRt = 2 * FB; // 16-row weight tiles per wave
constexpr int TB = BN / 32;     // 32-token MFMA blocks per tile
constexpr int KS = BK / 16;     // 16-K MFMA steps per stage
constexpr int kRingA = 3;       // register ring of A stages
constexpr int kRingB = 4;       // LDS ring of B stages
constexpr int A_FRAGS = FB * KS;                  // 8 A fragments per wave per stage
constexpr int B_FRAGS = TB * KS;                  // 32 B fragments per stage
constexpr int B_LOADS = B_FRAGS * 64 / kThreads;  // 8 per thread
constexpr int B_STAGE_BYTES = B_FRAGS * kTileBytes;  // 32 KiB
constexpr int kXcds = 8;
constexpr int kBufferFlags = 0x00020000;   // buffer descriptor word 3 (raw dword data, gfx9 family)
constexpr int kWaitAll = (0x7 << 4) | (0xF << 8);   // vmcnt 0
static_assert(kRingA == 3, "the K loop is unrolled by three stages");
static_assert(kRingB == 4, "stage s reads B(s), publishes B(s+1), loads B(s+2)");

typedef __attribute__((__vector_size__(16 * sizeof(float)))) float f32x16_t;

__device__ inline f32x16_t mfma32x32x16(const u32x4_t a, const u32x4_t b, f32x16_t c)
{
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                   __builtin_bit_cast(bf16x8_t, b), c, 0, 0, 0);
}

enum { kGateUp = 0, kDown = 1 };

// chunk swizzle of B row R in LDS (a function of R mod 16 only, so 32-row
// token blocks share it): rows 0..7 take eight distinct slots, and rows
// 8..15 the complementary (row parity, slot) pairs, so any 8 consecutive
// rows or 16 consecutive rows at one chunk hit distinct banks
__device__ __forceinline__ int b_swizzle(int R) { return (R & 7) ^ ((R >> 3) & 1); }

struct TileCtx {
    __amdgpu_buffer_rsrc_t a_rsrc;  // buffer over the expert's packed slab (GU or DN)
    uint32_t a_off[FB];        // this lane's A byte offset per feature block (stage 0, step 0)
    __amdgpu_buffer_rsrc_t b_rsrc;  // buffer over x (gate/up) or over the tile's rows of H
    uint32_t b_off[B_LOADS];   // byte offsets in b_rsrc of this lane's 16-byte chunk, per load
    uint32_t rd_off[KS];       // LDS byte offsets of this lane's B fragment piece, per K step
    int n_stages;
    int w, lane;
};

// The K loop of one tile on v_mfma_f32_32x32x16_bf16.  A 32 x 16 operand
// fragment is 1 KiB in lane order (lane l: row l%32, K 8(l/32)..+7).
//
// A stage is 32 units (16-K step j, 32-token block t), j-major; a unit is
// one B fragment read from LDS and the two MFMAs (both feature blocks) that
// use it.  B fragments are read kLook units ahead through a small register
// window, also across stage boundaries: the barrier that publishes the next
// stage's B sits kLook units before the end of the current stage.
//
// The global loads are spread over the units (a burst of them would stall
// the wave's in-order issue behind the address unit): stage s issues load q
// of B(s+2) at unit 4q + 1 (into the LDS buffer that stage s-2 used, free
// since stage s-1's barrier), and refills A fragment (fb, j) with A(s+3) two
// units after the last MFMA that reads it.
// kFull: every token block holds rows (branch-free loop); otherwise only the
// first n_pairs pairs of token blocks run their MFMAs.
constexpr int kUnits = KS * TB;   // 32 units per stage
constexpr int kLook = 3;          // B fragments in flight ahead of their MFMAs
constexpr int kWin = kLook + 1;   // B register window
constexpr int kBarrierUnit = kUnits - kLook;
static_assert(kUnits % kWin == 0, "the window index must repeat per stage");
static_assert(kUnits == 4 * B_LOADS, "one B load every four units");

// the unit at which stage s issues B load q of B(s+2)
constexpr int b_load_unit(int q) { return 4 * q + 1; }
// the unit at which stage s refills A fragment (fb, j) with A(s+3): the
// units of K step j are 8j .. 8j+7; the last K step's fragments go after
// the stage (unit kUnits)
constexpr int a_load_unit(int fb, int j) { return j + 1 < KS ? 8 * (j + 1) + 2 * fb : kUnits; }
// vector-memory ops issued after the last load of B(s+1) (stage s-1, unit
// b_load_unit(B_LOADS-1)) up to stage s's barrier; vector-memory ops
// complete in order, so waiting until at most this many are outstanding
// means this wave's part of B(s+1) is in LDS.  The stages after the main
// loop (kTail) issue no A refills: their registers are never read again, and
// the compiler would drop them as dead loads anyway.  The stage before a tail
// stage may be one too, so there only the stage's own B loads before the
// barrier are certain to follow B(s+1).
constexpr int vm_after_last_b(bool kTail)
{
    int n = 0;
    for (int q = 0; q < B_LOADS; ++q)
        if (b_load_unit(q) < kBarrierUnit) ++n;
    if (kTail) return n;
    for (int fb = 0; fb < FB; ++fb)
        for (int j = 0; j < KS; ++j) {
            const int u = a_load_unit(fb, j);
            if (u > b_load_unit(B_LOADS - 1)) ++n;   // rest of stage s-1
            if (u < kBarrierUnit) ++n;               // stage s before the barrier
        }
    return n;
}
static_assert(b_load_unit(B_LOADS - 1) >= kBarrierUnit, "every B(s+1) load precedes the count");
static_assert(vm_after_last_b(false) < 64, "vmcnt holds 6 bits");
// s_waitcnt immediate (gfx9 layout: vmcnt[3:0] | expcnt[6:4] | lgkmcnt[11:8] |
// vmcnt[15:14])
constexpr int wait_vm(int n) { return (n & 0xF) | ((n >> 4) << 14) | (0x7 << 4) | (0xF << 8); }
constexpr int kWaitBStage = wait_vm(vm_after_last_b(false));
constexpr int kWaitBTail = wait_vm(vm_after_last_b(true));

template <bool kFull>
__device__ __forceinline__ void tile_loop(const TileCtx& c, int n_pairs, uint8_t* lds,
                                          f32x16_t (&acc)[FB][TB])
{
    const int n_stages = c.n_stages;
    const int w = c.w;
    u32x4_t ra[kRingA][A_FRAGS];
    u32x4_t bw[kWin];
    // A fragment (fb, j) of stage s: K step j lives in K tile 2s + j/2,
    // second half of the tile for odd j (512 bytes on)
    auto load_a1 = [&](int s, int fb, int j, u32x4_t& dst) {
        dst = __builtin_bit_cast(u32x4_t, __builtin_amdgcn_raw_buffer_load_b128(
                                              c.a_rsrc, c.a_off[fb] + (j / 2) * kTileBytes + (j % 2) * (kTileBytes / 2),
                                              (uint32_t)s * (2 * kTileBytes), 0));
    };
    // B goes global -> LDS directly through buffer loads: a stage of B is
    // 256 rows x 128 bytes (64 K), row-major in LDS with the eight 16-byte
    // chunks of each row XOR-swizzled (see process_tile).  Load q of wave w
    // fills rows 64w + 8q .. +7, so every load reads whole 128-byte lines.
    // Buffer (not global) loads: the compiler counts them in vmcnt only, so
    // the LDS reads of the B window keep exact lgkmcnt waits.
    auto load_b1 = [&](int s, int buf, int q) {
        __builtin_amdgcn_raw_ptr_buffer_load_lds(
            c.b_rsrc,
            (__attribute__((address_space(3))) void*)(&lds[buf * B_STAGE_BYTES +
                                                           (w * B_LOADS + q) * kTileBytes]),
            16, c.b_off[q], (uint32_t)s * (BK * 2), 0, 0);
    };
    // the B fragment of unit u: token block t (rows 32t..), K step j
    auto read_unit = [&](const uint8_t* bbuf, int u) {
        const int j = u / TB, t = u % TB;
        bw[u % kWin] = *reinterpret_cast<const u32x4_t*>(&bbuf[c.rd_off[j] + t * 32 * (BK * 2)]);
    };
    // explicit partial wait + bare barrier: a __syncthreads() release fence
    // would wait for every outstanding LDS DMA (vmcnt 0); the empty asm
    // statements keep the compiler from moving memory operations across it
    auto wait_and_barrier = [&](auto tail) {
        __builtin_amdgcn_s_waitcnt(decltype(tail)::value ? kWaitBTail : kWaitBStage);
        asm volatile("" ::: "memory");
        __builtin_amdgcn_s_barrier();
        asm volatile("" ::: "memory");
    };
    // stage s (A in A, B in LDS buffer s % 4).  B loads past the last stage
    // re-read the last stage into buffers no stage reads; A refills are
    // issued in the main loop only (tail is std::true_type after it).
    auto stage = [&](int s, u32x4_t (&A)[A_FRAGS], auto tail) {
        constexpr bool kTail = decltype(tail)::value;
        const uint8_t* bcur = lds + (s % kRingB) * B_STAGE_BYTES;
        const uint8_t* bnext = lds + ((s + 1) % kRingB) * B_STAGE_BYTES;
        const int sb = min(s + 2, n_stages - 1), bbuf = (s + 2) % kRingB;
        const int sa = min(s + kRingA, n_stages - 1);
#pragma unroll
        for (int u = 0; u < kUnits; ++u) {
            if (u == kBarrierUnit) wait_and_barrier(tail);
            if (u % 4 == 1) load_b1(sb, bbuf, u / 4);
#pragma unroll
            for (int fb = 0; fb < FB; ++fb)
#pragma unroll
                for (int j = 0; j < KS; ++j)
                    if (!kTail && a_load_unit(fb, j) == u) load_a1(sa, fb, j, A[fb * KS + j]);
            if (u + kLook < kUnits)
                read_unit(bcur, u + kLook);
            else
                read_unit(bnext, u + kLook - kUnits);
            __builtin_amdgcn_sched_barrier(0);
            const int j = u / TB, t = u % TB;
            if (kFull || t / 2 < n_pairs) {
#pragma unroll
                for (int fb = 0; fb < FB; ++fb)
                    acc[fb][t] = mfma32x32x16(A[fb * KS + j], bw[u % kWin], acc[fb][t]);
            }
            __builtin_amdgcn_sched_barrier(0);
        }
#pragma unroll
        for (int fb = 0; fb < FB; ++fb)
#pragma unroll
            for (int j = 0; j < KS; ++j)
                if (!kTail && a_load_unit(fb, j) == kUnits) load_a1(sa, fb, j, A[fb * KS + j]);
    };

    // prologue: B(0), B(1) and A(0..2); wait for them, then read the first
    // kLook units of stage 0
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int q = 0; q < B_LOADS; ++q) load_b1(min(i, n_stages - 1), i, q);
#pragma unroll
    for (int i = 0; i < kRingA; ++i)
#pragma unroll
        for (int fb = 0; fb < FB; ++fb)
#pragma unroll
            for (int j = 0; j < KS; ++j) load_a1(min(i, n_stages - 1), fb, j, ra[i][fb * KS + j]);
    __builtin_amdgcn_s_waitcnt(kWaitAll);
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
#pragma unroll
    for (int u = 0; u < kLook; ++u) read_unit(lds, u);
    // three stages per iteration, so that the A ring is indexed statically
    int s = 0;
    for (; s + kRingA <= n_stages; s += kRingA) {
        stage(s + 0, ra[0], std::false_type{});
        stage(s + 1, ra[1], std::false_type{});
        stage(s + 2, ra[2], std::false_type{});
    }
    if (s < n_stages) {
        stage(s, ra[0], std::true_type{});
        if (s + 1 < n_stages) stage(s + 1, ra[1], std::true_type{});
    }
    // the last stages re-issued dummy B loads into LDS: drain them before the
    // workgroup can finish and its LDS be handed to another workgroup
    __builtin_amdgcn_s_waitcnt(kWaitAll);
    __builtin_amdgcn_s_barrier();
}

// One BM x BN tile (feature tile ft, token tile tt) of the grouped GEMM.
template <int kMode>
__device__ __forceinline__ void process_tile(const GemmArgs& a, int ft, int tt, uint8_t* lds)
{
    const int e = a.tiles[2 * tt];
    const int row_start = a.tiles[2 * tt + 1];
    const int row_end = min(row_start + BN, a.offsets[e + 1]);
    const int ntb = (row_end - row_start + 31) / 32;   // 32-token blocks with rows

    const int K = kMode == kGateUp ? a.d : a.f;
    const uint64_t KT = (uint64_t)K / kTileK;
    const uint8_t* wbase = a.experts + (uint64_t)(e - a.e_begin) * a.expert_bytes +
                           (kMode == kGateUp ? 0 : a.gu_bytes);

    TileCtx c;
    c.n_stages = K / BK;
    c.lane = threadIdx.x & 63;
    c.w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);   // wave-uniform, in an SGPR
    const int lane = c.lane, w = c.w;
    // M is a multiple of BM (the library requires d % 256 == 0 and
    // f % 128 == 0), so every wave's 64-feature slab lies inside the matrix
    const uint64_t rt0 = (uint64_t)ft * (BM / 16) + w * kWaveRt;
    // A: lane l of a 32 x 16 fragment reads row l%32 of the block (row tile
    // rt0 + 2 fb + (l%32)/16, granule row l%16) at K group l/32 of the step.
    // Buffer loads over the expert's slab (the library caps a slab below
    // 2^31 bytes, so offsets fit 32 bits; the size bounds every load).
    const uint64_t slab_bytes = kMode == kGateUp ? a.gu_bytes : a.expert_bytes - a.gu_bytes;
    c.a_rsrc = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint8_t*>(wbase), 0, (int)slab_bytes,
                                                 kBufferFlags);
#pragma unroll
    for (int fb = 0; fb < FB; ++fb)
        c.a_off[fb] = (uint32_t)tile_offset(rt0 + 2 * fb + ((lane & 31) >> 4), 0, KT) +
                      (uint32_t)(((lane >> 5) * 16) + (lane & 15)) * 16;
    // B: a stage holds, for each of the 256 token rows R of the tile, the
    // 128 bytes of K [64 s, 64 s + 64) as eight 16-byte chunks; chunk c sits
    // in slot c ^ swz(R) so that the MFMA reads (8 consecutive rows at one
    // chunk) fall in distinct LDS banks.  Load q of wave w: lane l reads row
    // R = 64w + 8q + l/8, slot l%8, i.e. chunk (l%8) ^ swz(R).  Gate/up
    // gathers rows of x (the library caps T*d*2 below 2^31, so byte offsets
    // fit 32 bits); down reads the tile's own rows of H through a buffer
    // based at the tile's first row.  The buffer size bounds every load
    // (out-of-range reads return zero).
    if (kMode == kGateUp)
        c.b_rsrc = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(a.x), 0,
                                                     a.T * a.d * 2, kBufferFlags);
    else
        c.b_rsrc = __builtin_amdgcn_make_buffer_rsrc(a.H + (int64_t)row_start * a.f, 0,
                                                     (row_end - row_start) * a.f * 2, kBufferFlags);
#pragma unroll
    for (int q = 0; q < B_LOADS; ++q) {
        const int R = w * 64 + q * 8 + (lane >> 3);
        const int row = row_start + R;
        const int rr = row < row_end ? row : row_start;   // rows past the end: any valid row
        const uint32_t chunk = (uint32_t)((lane & 7) ^ b_swizzle(R)) * 16;
        if (kMode == kGateUp)
            c.b_off[q] = (uint32_t)a.row_token[rr] * (uint32_t)a.d * 2 + chunk;
        else
            c.b_off[q] = (uint32_t)(rr - row_start) * (uint32_t)a.f * 2 + chunk;
    }
    // MFMA B operand of K step j, token block t: lane l takes row
    // R = 32t + l%32, chunk 2j + l/32 (swz(R) does not depend on t)
#pragma unroll
    for (int j = 0; j < KS; ++j) {
        const int R = lane & 31;
        c.rd_off[j] = (uint32_t)R * (BK * 2) + (uint32_t)(((2 * j + (lane >> 5)) ^ b_swizzle(R)) * 16);
    }

    f32x16_t acc[FB][TB];
#pragma unroll
    for (int fb = 0; fb < FB; ++fb)
#pragma unroll
        for (int tb = 0; tb < TB; ++tb) acc[fb][tb] = f32x16_t{};

    // full tiles take the branch-free loop; an expert's partial last tile
    // skips the MFMAs of token-block pairs past its last row
    if (ntb == TB)
        tile_loop<true>(c, TB / 2, lds, acc);
    else
        tile_loop<false>(c, (ntb + 1) / 2, lds, acc);

    // epilogue: in a 32 x 32 block lane l holds token column l%32 and rows
    // 8g + 4(l/32) + r in register 4g + r (g, r = 0..3).  A 32-row block is
    // row tiles (rt, rt + 1): for the gate/up GEMM that is 16 gate rows
    // (g = 0, 1) and the 16 up rows of the same features (g = 2, 3).
    const int half = lane >> 5;
    const int jcol = lane & 31;
#pragma unroll
    for (int tb = 0; tb < TB; ++tb) {
        const int row = row_start + tb * 32 + jcol;
        if (row >= row_end) continue;
#pragma unroll
        for (int fb = 0; fb < FB; ++fb) {
            const f32x16_t v = acc[fb][tb];
            const uint64_t rt = rt0 + 2 * fb;
            if (kMode == kGateUp) {
#pragma unroll
                for (int g = 0; g < 2; ++g) {
                    const int feat = (int)(rt / 2) * 16 + 8 * g + 4 * half;
                    const uint32_t h01 = cvt_pk_bf16(silu_mul(v[4 * g + 0], v[4 * g + 8]),
                                                     silu_mul(v[4 * g + 1], v[4 * g + 9]));
                    const uint32_t h23 = cvt_pk_bf16(silu_mul(v[4 * g + 2], v[4 * g + 10]),
                                                     silu_mul(v[4 * g + 3], v[4 * g + 11]));
                    *reinterpret_cast<uint2*>(a.H + (int64_t)row * a.f + feat) = make_uint2(h01, h23);
                }
            } else {
#pragma unroll
                for (int g = 0; g < 4; ++g) {
                    const int feat = (int)rt * 16 + 8 * g + 4 * half;
                    *reinterpret_cast<float4*>(a.O + (int64_t)row * a.d + feat) =
                        make_float4(v[4 * g], v[4 * g + 1], v[4 * g + 2], v[4 * g + 3]);
                }
            }
        }
    }
}

template <int kMode>
__global__ __launch_bounds__(kThreads) void gemm_kernel(GemmArgs a)
{
    __shared__ __attribute__((aligned(16))) uint8_t lds[kRingB * B_STAGE_BYTES];
    const int M = kMode == kGateUp ? 2 * a.f : a.d;   // a multiple of BM
    const int n_ftiles = M / BM;
    // XCD-aware numbering: hardware hands block b to XCD b % 8; each XCD
    // gets a contiguous run of logical tiles (feature tile major, token tile
    // fastest over the max_tiles slots the grid is sized for), so the
    // workgroups running together on an XCD work on consecutive token tiles
    // of one feature slab and share the weight slabs of their experts (A) in
    // its L2.  Slots past the routing's token tiles exit at once.  (Splitting
    // only the live tiles evenly over the XCDs measured no better: the XCDs'
    // finish times differ by the mix of full and partial tiles they get.)
    const int per_xcd = gridDim.x / kXcds;
    const int logical = (blockIdx.x % kXcds) * per_xcd + blockIdx.x / kXcds;
    const int ft = logical / a.max_tiles, tt = logical % a.max_tiles;
    if (ft >= n_ftiles || tt >= *a.n_tiles) return;
    // measurement only (a.stamps set by moe_profile_gemm_timeline): the
    // constant 100 MHz counter and the shader-clock counter around the tile
    const bool stamp = a.stamps != nullptr && (int)blockIdx.x < a.max_stamps;
    uint64_t r0 = 0, c0 = 0;
    if (stamp) {
        r0 = __builtin_amdgcn_s_memrealtime();
        c0 = __builtin_amdgcn_s_memtime();
    }
    process_tile<kMode>(a, ft, tt, lds);
    if (stamp) {
        __syncthreads();
        if (threadIdx.x == 0) {
            const uint64_t r1 = __builtin_amdgcn_s_memrealtime();
            const uint64_t c1 = __builtin_amdgcn_s_memtime();
            uint32_t hw, xcc;
            asm volatile("s_getreg_b32 %0, hwreg(HW_REG_HW_ID)" : "=s"(hw));
            asm volatile("s_getreg_b32 %0, hwreg(HW_REG_XCC_ID)" : "=s"(xcc));
            const int e = a.tiles[2 * tt], row0 = a.tiles[2 * tt + 1];
            const int rows = min(row0 + BN, a.offsets[e + 1]) - row0;
            uint64_t* out = a.stamps + (uint64_t)blockIdx.x * 8;
            out[0] = r0;
            out[1] = r1;
            out[2] = c0;
            out[3] = c1;
            out[4] = (uint64_t)hw | ((uint64_t)xcc << 32);
            out[5] = (uint64_t)ft | ((uint64_t)tt << 16) | ((uint64_t)rows << 32) |
                     ((uint64_t)e << 48);
        }
    }
}

}  // namespace moe

extern "C" int moe_prefill_tile_rows() { return moe::BN; }

template <int kMode>
static hipError_t launch_gemm(const moe::GemmArgs* a, hipStream_t s)
{
    const int M = kMode == moe::kGateUp ? 2 * a->f : a->d;
    const int n = M / moe::BM * a->max_tiles;
    const int grid = (n + moe::kXcds - 1) / moe::kXcds * moe::kXcds;
    hipLaunchKernelGGL((moe::gemm_kernel<kMode>), dim3(grid), dim3(moe::kThreads), 0, s, *a);
    return hipGetLastError();
}

extern "C" hipError_t moe_launch_gemm_gateup(const moe::GemmArgs* a, hipStream_t s)
{
    return launch_gemm<moe::kGateUp>(a, s);
}

extern "C" hipError_t moe_launch_gemm_down(const moe::GemmArgs* a, hipStream_t s)
{
    return launch_gemm<moe::kDown>(a, s);
}

