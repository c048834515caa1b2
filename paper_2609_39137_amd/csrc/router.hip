// Fused router step for gfx950: gate contraction z = W_r x on MFMA (Sec. 2.2),
// sigmoid scores, bias-adjusted Top-K (Eq. pid-routing), gate weights from the
// unbiased scores and per-expert load counts (Eq. pid-error).  The T x E score
// matrix stays in registers and LDS.
//
// Tiling.  A workgroup owns BT tokens and one slice of BE experts; each wave
// owns all BT tokens and its own WE = BE / WAVES experts.  The wave's router
// rows are private to it and go straight from global memory into MFMA
// A-operand registers; the token tile is shared by the waves through LDS.
// The contraction runs over 128-byte chunks of each row.  Two contraction
// kernels share the selection epilogue:
//   - 32x32x16 tiles (router32_kernel): WE = 32 NBLK, BT = 32 TBW; also the
//     fp32-input path (32x32x2 MFMAs).
//   - 16x16x32 tiles (router16_kernel): WE = 16 ET, BT = 16 TT.  With 8 waves
//     of 48 experts x 128 tokens each wave needs only 96 accumulators, so two
//     waves share a SIMD while every router byte is still loaded once per
//     workgroup.
// In both, lanes of a wave consume the same k bytes of a chunk for both
// operands, so the k order agrees between A and B.
//
// Token tile: staged through registers into two LDS stages of 160-byte rows
// (128 bytes + 32 of padding, which measured fastest for the B-operand reads
// and the staging writes), loaded two chunks ahead of use.
//
// Router matrix: either row-major [E][d] or the packed layout written by
// idb_router_pack_weight: for every 16-expert block b, chunk c and 64-byte
// half s of the chunk, one contiguous 1 KB piece holds, for lane l < 64, bytes
// [c*128 + 64 s + 16 (l/16), +16) of row 16 b + l%16 (exactly one 16x16x32
// A operand; a 32x32x16 A operand is four 256-byte runs of it).
//
// MFMA output layouts (C = W_tile x_tile^T): 32x32 - lane l holds token l%32
// of the block and experts 8 (r/4) + 4 (l/32) + r%4, r < 16; 16x16 - lane l
// holds token l%16 of the tile and experts 4 (l/16) + r, r < 4.
//
// Epilogue: epilogue.h, steps A-G; step A (sigmoid of the accumulators into
// the LDS score matrix) is the contraction kernel's, as it depends on the MFMA
// layout.  Several slices: router_merge_kernel combines their candidates.

#include "common.h"
#include "controller_block.h"
#include "epilogue.h"
#include "internal.h"

#include <hip/hip_ext.h>
#include <type_traits>

#pragma clang fp contract(off)

namespace idb {

namespace {

constexpr int kRowPad = 160;  // LDS bytes per staged token row (128 + 32 pad)
constexpr int kMaxSlices = 8;

// One 16-byte unit of both operands: bf16 -> one 32x32x16 MFMA; fp32 -> four
// 32x32x2 MFMAs, float i of each lane's unit feeding the i-th.
template <bool F32>
__device__ __forceinline__ floatx16 mfma_unit(uint4 a, uint4 b, floatx16 c) {
    if constexpr (F32) {
        c = __builtin_amdgcn_mfma_f32_32x32x2f32(__builtin_bit_cast(float, a.x), __builtin_bit_cast(float, b.x), c,
                                                 0, 0, 0);
        c = __builtin_amdgcn_mfma_f32_32x32x2f32(__builtin_bit_cast(float, a.y), __builtin_bit_cast(float, b.y), c,
                                                 0, 0, 0);
        c = __builtin_amdgcn_mfma_f32_32x32x2f32(__builtin_bit_cast(float, a.z), __builtin_bit_cast(float, b.z), c,
                                                 0, 0, 0);
        c = __builtin_amdgcn_mfma_f32_32x32x2f32(__builtin_bit_cast(float, a.w), __builtin_bit_cast(float, b.w), c,
                                                 0, 0, 0);
        return c;
    } else {
        return __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(a), as_bf16x8(b), c, 0, 0, 0);
    }
}

// XCD-aware block order: consecutive blocks land on different XCDs, so remap
// to give each XCD a contiguous run of (tile, slice) pairs; the slices of one
// token tile then share their token rows in that XCD's L2.
__device__ __forceinline__ int xcd_block_order() {
    const int nb = gridDim.x;
    int L = blockIdx.x;
    if ((nb & 7) == 0) L = (blockIdx.x & 7) * (nb >> 3) + (blockIdx.x >> 3);
    return L;
}

template <bool F32, int WAVES, int TBW, int NBLK>
struct Cfg32 {
    static constexpr int NT = WAVES * 64;
    static constexpr int BT = 32 * TBW;
    static constexpr int WE = 32 * NBLK;
    static constexpr int BE = WAVES * WE;
    static constexpr int PPT = BT * 8 / NT;  // 16-byte token-tile pieces per thread per chunk
    static constexpr int STAGE = BT * kRowPad;
    static constexpr int MAIN_LDS = 2 * STAGE;
    using Epi = EpiCfg<NT, BT, BE, MAIN_LDS>;
    static_assert(PPT * NT == BT * 8, "token-tile pieces must split evenly over threads");
};

template <bool F32, bool PACKED, int WAVES, int TBW, int NBLK, bool SM>
__global__ __launch_bounds__(WAVES * 64) void router32_kernel(RouterArgs a, int NS) {
    using C = Cfg32<F32, WAVES, TBW, NBLK>;
    using EC = typename C::Epi;
    __shared__ __attribute__((aligned(16))) unsigned char smem[EC::LDS];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform: keep it scalar
    const int h = lane >> 5;
    const int l32 = lane & 31;
    const int L = xcd_block_order();
    const int tile = L / NS;
    const int slice = L - tile * NS;

    const int64_t T = a.T;
    const int E = a.E;
    const int64_t tok0 = (int64_t)tile * C::BT;
    const int e_wave0 = slice * C::BE + wave * C::WE;
    const int64_t RB = (int64_t)a.d * (F32 ? 4 : 2);
    const int NCH = (int)(RB / 128);

    if (a.zero_counts && blockIdx.x == 0)
        for (int e = tid; e < E; e += C::NT) a.counts[e] = 0;
    if (a.ticket && blockIdx.x == 0 && tid == 0) *a.ticket = 0u;  // the merge's or the statistics kernel's
    const int sbase = slice * C::BE;
    float breg[EC::NBIAS];
    prefetch_bias<EC, SM>(a, sbase, breg);

    // ---------------------------------------------------------------- contraction
    // Operands are fetched with buffer loads: a scalar resource per operand
    // and a 32-bit per-lane offset, with the chunk and block advance in the
    // scalar offset, so the unrolled loads need no 64-bit address registers.
    // Every load stays inside its resource by construction (the scalar offset
    // is not range-checked).
    //
    // A operands (router rows): lane (h, m = l32) reads row 32 blk + m, bytes
    // c*128 + 64 h + 16 u.  Packed: the piece of 16-row block 2 blk + m/16,
    // chunk c and half h, at lane slot m%16 + 16 u.  A chunk adds WCH bytes to
    // the scalar offset, a unit WU to the lane offset.
    constexpr int WU = PACKED ? 256 : 16;
    constexpr int WCH = PACKED ? 2048 : 128;
    const __amdgpu_buffer_rsrc_t wres = make_rsrc(a.W, (int64_t)E * RB);
    const int wvoff = PACKED ? (l32 >> 4) * NCH * 2048 + h * 1024 + (l32 & 15) * 16 : l32 * (int)RB + 64 * h;
    int wsoff[NBLK];
#pragma unroll
    for (int nbk = 0; nbk < NBLK; ++nbk) {
        int blk = (e_wave0 + nbk * 32) / 32;
        blk = blk < E / 32 ? blk : E / 32 - 1;  // padding blocks read a valid block; masked later
        wsoff[nbk] = PACKED ? blk * NCH * 4096 : blk * 32 * (int)RB;
    }
    // Token-tile pieces: thread piece p = tid + NT*q covers row p/8, bytes
    // 16*(p%8) of the chunk.  Rows past T re-read row T-1 (never output).
    const int nrows = (int)((T - tok0) < C::BT ? (T - tok0) : C::BT);
    const __amdgpu_buffer_rsrc_t xres =
        make_rsrc(reinterpret_cast<const char*>(a.x) + tok0 * RB, (int64_t)nrows * RB);
    int xvoff[C::PPT];
    int xdst[C::PPT];
#pragma unroll
    for (int q = 0; q < C::PPT; ++q) {
        const int p = tid + C::NT * q;
        const int row = p >> 3, c16 = p & 7;
        const int rowc = row < nrows ? row : nrows - 1;
        xvoff[q] = rowc * (int)RB + c16 * 16;
        xdst[q] = row * kRowPad + c16 * 16;
    }
    const int boff = l32 * kRowPad + 64 * h;

    floatx16 acc[TBW][NBLK];
#pragma unroll
    for (int tb = 0; tb < TBW; ++tb)
#pragma unroll
        for (int nbk = 0; nbk < NBLK; ++nbk)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[tb][nbk][r] = 0.0f;

    // Software pipeline, two chunks deep for both operands.  W operands: two
    // register sets; right after the MFMAs of unit u of chunk c, set c&1
    // starts loading unit u of chunk c+2.  Token tile: two sets of staging
    // registers; the top of chunk c loads chunk c+2 into the set that held
    // chunk c, and the end of chunk c stores chunk c+1 (loaded a whole chunk
    // earlier) into the idle LDS stage.  Every fetch thus has about two
    // chunks of MFMA work to arrive.
    //
    // The loop body is branch-free so that the compiler's vector-memory wait
    // counts stay exact (loads complete in order; a conditional load would
    // make every later wait drain the queue): prefetch targets are clamped
    // to the last chunk (a cached re-read at the end), the last store goes to
    // a stage that is never read, and an odd last chunk is peeled.
    uint4 w[2][NBLK][4], xr[2][C::PPT];
    auto load_x = [&](int c, int j) {
#pragma unroll
        for (int q = 0; q < C::PPT; ++q) xr[j][q] = bload16(xres, xvoff[q], c * 128);
    };
    auto store_x = [&](int stage, int j) {
#pragma unroll
        for (int q = 0; q < C::PPT; ++q) *reinterpret_cast<uint4*>(smem + stage * C::STAGE + xdst[q]) = xr[j][q];
    };
    auto load_w = [&](int c, int j) {
#pragma unroll
        for (int nbk = 0; nbk < NBLK; ++nbk)
#pragma unroll
            for (int u = 0; u < 4; ++u) w[j][nbk][u] = bload16(wres, wvoff + WU * u, wsoff[nbk] + c * WCH);
    };
    // MFMAs of one chunk from LDS stage / W set j; with prefetch, each W unit
    // is refilled from chunk cn right after its MFMAs.
    auto compute = [&](int j, bool prefetch, int cn) {
        const unsigned char* st = smem + j * C::STAGE + boff;
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            uint4 bx[TBW];
#pragma unroll
            for (int tb = 0; tb < TBW; ++tb) bx[tb] = *reinterpret_cast<const uint4*>(st + tb * 32 * kRowPad + 16 * u);
#pragma unroll
            for (int tb = 0; tb < TBW; ++tb)
#pragma unroll
                for (int nbk = 0; nbk < NBLK; ++nbk) acc[tb][nbk] = mfma_unit<F32>(w[j][nbk][u], bx[tb], acc[tb][nbk]);
            if (prefetch) {
#pragma unroll
                for (int nbk = 0; nbk < NBLK; ++nbk) w[j][nbk][u] = bload16(wres, wvoff + WU * u, wsoff[nbk] + cn * WCH);
            }
        }
    };

    const int last = NCH - 1;
    load_x(0, 0);
    load_w(0, 0);
    load_x(last < 1 ? last : 1, 1);
    load_w(last < 1 ? last : 1, 1);
    store_x(0, 0);
    __syncthreads();
    for (int c0 = 0; c0 + 1 < NCH; c0 += 2) {
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            const int c = c0 + j;
            const int cn = c + 2 < last ? c + 2 : last;
            load_x(cn, j);
            compute(j, true, cn);
            store_x(1 - j, 1 - j);
            __syncthreads();
        }
    }
    if (NCH & 1) {
        compute(0, false, 0);
        __syncthreads();
    }

    // ---------------------------------------------------------------- selection
    // Slice column of accumulator (nbk, r): wave*WE + 4 h + 32 nbk + 8 (r/4) +
    // (r%4).  E is a multiple of 32, so a whole 32-expert block is real or
    // padding.
    const int ccol = wave * C::WE + 4 * h;
    // score activation; auxiliary-loss routing (SM) ranks the logits themselves
    auto act = [&](float z) {
        if constexpr (SM) return z;
        else return sigmoid_fast(z);
    };
    auto store_pass = [&](int pass, float* sc) {
        constexpr int PB = EC::TPP / 32;
#pragma unroll
        for (int pb = 0; pb < PB; ++pb) {
            const int tb = pass * PB + pb;
            const int row = pb * 32 + l32;
            const int64_t tok = tok0 + tb * 32 + l32;
#pragma unroll
            for (int nbk = 0; nbk < NBLK; ++nbk) {
                const bool real = sbase + wave * C::WE + nbk * 32 < E;
#pragma unroll
                for (int r4 = 0; r4 < 4; ++r4) {
                    float4 s4;
                    s4.x = real ? act(acc[tb][nbk][4 * r4 + 0]) : -INFINITY;
                    s4.y = real ? act(acc[tb][nbk][4 * r4 + 1]) : -INFINITY;
                    s4.z = real ? act(acc[tb][nbk][4 * r4 + 2]) : -INFINITY;
                    s4.w = real ? act(acc[tb][nbk][4 * r4 + 3]) : -INFINITY;
                    const int col = ccol + nbk * 32 + 8 * r4;
                    *reinterpret_cast<float4*>(sc + row * EC::RS + col) = s4;
                    if (a.dump && real && tok < T) *reinterpret_cast<float4*>(a.dump + tok * E + sbase + col) = s4;
                }
            }
        }
    };
    select_epilogue<EC, SM>(a, NS, slice, tok0, smem, breg, store_pass);
}

template <int WAVES, int TT, int ET>
struct Cfg16 {
    static constexpr int NT = WAVES * 64;
    static constexpr int BT = 16 * TT;
    static constexpr int WE = 16 * ET;
    static constexpr int BE = WAVES * WE;
    static constexpr int PPT = BT * 8 / NT;  // 16-byte token-tile pieces per thread per chunk
    static constexpr int STAGE = BT * kRowPad;
    static constexpr int MAIN_LDS = 2 * STAGE;
    using Epi = EpiCfg<NT, BT, BE, MAIN_LDS>;
    static_assert(PPT * NT == BT * 8, "token-tile pieces must split evenly over threads");
};

template <bool PACKED, int WAVES, int TT, int ET, bool SM>
__global__ __launch_bounds__(WAVES * 64) void router16_kernel(RouterArgs a, int NS) {
    using C = Cfg16<WAVES, TT, ET>;
    using EC = typename C::Epi;
    __shared__ __attribute__((aligned(16))) unsigned char smem[EC::LDS];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform: keep it scalar
    const int l16 = lane & 15, g4 = lane >> 4;
    const int L = xcd_block_order();
    const int tile = L / NS;
    const int slice = L - tile * NS;

    const int64_t T = a.T;
    const int E = a.E;
    const int64_t tok0 = (int64_t)tile * C::BT;
    const int e_wave0 = slice * C::BE + wave * C::WE;
    const int64_t RB = (int64_t)a.d * 2;
    const int NCH = (int)(RB / 128);

    if (a.zero_counts && blockIdx.x == 0)
        for (int e = tid; e < E; e += C::NT) a.counts[e] = 0;
    if (a.ticket && blockIdx.x == 0 && tid == 0) *a.ticket = 0u;  // the merge's or the statistics kernel's
    const int sbase = slice * C::BE;
    float breg[EC::NBIAS];
    prefetch_bias<EC, SM>(a, sbase, breg);

    // ---------------------------------------------------------------- contraction
    // Buffer loads as in router32_kernel.  A operand of expert tile et, chunk
    // c, half s (k bytes [64 s, 64 s + 64) of the chunk): lane l reads row
    // 16 b + l%16, bytes c*128 + 64 s + 16 (l/16) of its 16-row block b.
    // Packed, that is the piece of (b, c, s) at lane slot l.
    constexpr int WS = PACKED ? 1024 : 64;     // lane-offset step of a half
    constexpr int WCH = PACKED ? 2048 : 128;   // scalar-offset step of a chunk
    const __amdgpu_buffer_rsrc_t wres = make_rsrc(a.W, (int64_t)E * RB);
    const int wvoff = PACKED ? lane * 16 : l16 * (int)RB + 16 * g4;
    int wsoff[ET];
#pragma unroll
    for (int et = 0; et < ET; ++et) {
        int blk = (e_wave0 + et * 16) / 16;
        blk = blk < E / 16 ? blk : E / 16 - 1;  // padding tiles read a valid block; masked later
        wsoff[et] = PACKED ? blk * NCH * 2048 : blk * 16 * (int)RB;
    }
    // Token-tile pieces: thread piece p = tid + NT*q covers row p/8, bytes
    // 16*(p%8) of the chunk.  Rows past T re-read row T-1 (never output).
    const int nrows = (int)((T - tok0) < C::BT ? (T - tok0) : C::BT);
    const __amdgpu_buffer_rsrc_t xres =
        make_rsrc(reinterpret_cast<const char*>(a.x) + tok0 * RB, (int64_t)nrows * RB);
    int xvoff[C::PPT];
    int xdst[C::PPT];
#pragma unroll
    for (int q = 0; q < C::PPT; ++q) {
        const int p = tid + C::NT * q;
        const int row = p >> 3, c16 = p & 7;
        const int rowc = row < nrows ? row : nrows - 1;
        xvoff[q] = rowc * (int)RB + c16 * 16;
        xdst[q] = row * kRowPad + c16 * 16;
    }
    // B operand of token tile tt, half s: token 16 tt + l%16, bytes 64 s + 16 (l/16).
    const int boff = l16 * kRowPad + 16 * g4;

    floatx4 acc[TT][ET];
#pragma unroll
    for (int tt = 0; tt < TT; ++tt)
#pragma unroll
        for (int et = 0; et < ET; ++et) acc[tt][et] = floatx4{0.0f, 0.0f, 0.0f, 0.0f};

    // Software pipeline as in router32_kernel: two W register sets and two
    // token-tile staging sets, two chunks deep, branch-free loop body.
    uint4 w[2][ET][2], xr[2][C::PPT];
    auto load_x = [&](int c, int j) {
#pragma unroll
        for (int q = 0; q < C::PPT; ++q) xr[j][q] = bload16(xres, xvoff[q], c * 128);
    };
    auto store_x = [&](int stage, int j) {
#pragma unroll
        for (int q = 0; q < C::PPT; ++q) *reinterpret_cast<uint4*>(smem + stage * C::STAGE + xdst[q]) = xr[j][q];
    };
    auto load_w = [&](int c, int j) {
#pragma unroll
        for (int et = 0; et < ET; ++et)
#pragma unroll
            for (int s = 0; s < 2; ++s) w[j][et][s] = bload16(wres, wvoff + WS * s, wsoff[et] + c * WCH);
    };
    auto compute = [&](int j, bool prefetch, int cn) {
        const unsigned char* st = smem + j * C::STAGE + boff;
#pragma unroll
        for (int s = 0; s < 2; ++s) {
            // all of the half's B operands first, so their LDS latencies overlap
            uint4 bx[TT];
#pragma unroll
            for (int tt = 0; tt < TT; ++tt) bx[tt] = *reinterpret_cast<const uint4*>(st + tt * 16 * kRowPad + 64 * s);
#pragma unroll
            for (int tt = 0; tt < TT; ++tt)
#pragma unroll
                for (int et = 0; et < ET; ++et)
                    acc[tt][et] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(w[j][et][s]), as_bf16x8(bx[tt]),
                                                                          acc[tt][et], 0, 0, 0);
            if (prefetch) {
#pragma unroll
                for (int et = 0; et < ET; ++et) w[j][et][s] = bload16(wres, wvoff + WS * s, wsoff[et] + cn * WCH);
            }
        }
        // Schedule: half 0's TT B-operand reads, then its MFMAs with half 1's
        // reads interleaved one per ET MFMAs, then half 1's MFMAs, so no
        // group of MFMAs waits for a fresh LDS read.
        __builtin_amdgcn_sched_group_barrier(0x100, TT, 0);  // LDS reads
#pragma unroll
        for (int i = 0; i < TT; ++i) {
            __builtin_amdgcn_sched_group_barrier(0x008, ET, 0);  // MFMA
            __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
        }
        __builtin_amdgcn_sched_group_barrier(0x008, TT * ET, 0);
    };

    const int last = NCH - 1;
    load_x(0, 0);
    load_w(0, 0);
    load_x(last < 1 ? last : 1, 1);
    load_w(last < 1 ? last : 1, 1);
    store_x(0, 0);
    __syncthreads();
    for (int c0 = 0; c0 + 1 < NCH; c0 += 2) {
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            const int c = c0 + j;
            const int cn = c + 2 < last ? c + 2 : last;
            load_x(cn, j);
            compute(j, true, cn);
            store_x(1 - j, 1 - j);
            __syncthreads();
        }
    }
    if (NCH & 1) {
        compute(0, false, 0);
        __syncthreads();
    }

    // ---------------------------------------------------------------- selection
    // Slice column of accumulator (et, r): wave*WE + 16 et + 4 (l/16) + r.
    // E is a multiple of 32, so a whole 16-expert tile is real or padding.
    // score activation; auxiliary-loss routing (SM) ranks the logits themselves
    auto act = [&](float z) {
        if constexpr (SM) return z;
        else return sigmoid_fast(z);
    };
    // The wave's expert tiles are all real unless the slice ends inside them;
    // without a dump and with all tiles real the store loop needs no checks
    // (both conditions are uniform over the workgroup).
    const bool all_real = sbase + wave * C::WE + C::WE <= E;
    auto store_tiles = [&](int pass, float* sc, auto checked) {
        constexpr int PT = EC::TPP / 16;  // token tiles per pass
#pragma unroll
        for (int pt = 0; pt < PT; ++pt) {
            const int tt = pass * PT + pt;
            const int row = pt * 16 + l16;
            const int64_t tok = tok0 + tt * 16 + l16;
#pragma unroll
            for (int et = 0; et < ET; ++et) {
                const int col = wave * C::WE + et * 16 + 4 * g4;
                float4 s4;
                if constexpr (decltype(checked)::value) {
                    const bool real = sbase + wave * C::WE + et * 16 < E;
                    s4.x = real ? act(acc[tt][et][0]) : -INFINITY;
                    s4.y = real ? act(acc[tt][et][1]) : -INFINITY;
                    s4.z = real ? act(acc[tt][et][2]) : -INFINITY;
                    s4.w = real ? act(acc[tt][et][3]) : -INFINITY;
                    *reinterpret_cast<float4*>(sc + row * EC::RS + col) = s4;
                    if (a.dump && real && tok < T) *reinterpret_cast<float4*>(a.dump + tok * E + sbase + col) = s4;
                } else {
                    s4.x = act(acc[tt][et][0]);
                    s4.y = act(acc[tt][et][1]);
                    s4.z = act(acc[tt][et][2]);
                    s4.w = act(acc[tt][et][3]);
                    *reinterpret_cast<float4*>(sc + row * EC::RS + col) = s4;
                }
            }
        }
    };
    auto store_pass = [&](int pass, float* sc) {
        if (!a.dump && all_real) store_tiles(pass, sc, std::false_type{});
        else store_tiles(pass, sc, std::true_type{});
    };
    select_epilogue<EC, SM>(a, NS, slice, tok0, smem, breg, store_pass);
}

// Merge the slices' rank-ordered candidate lists into the final Top-K, compute
// the gate weights and count the assignments.  One thread per candidate: its
// final rank is its position in its own slice's list plus the number of the
// other slices' candidates that rank above it (keys are distinct: every
// candidate is a different expert).  A workgroup takes groups of
// kMergeThreads / (NS*K) tokens in a grid-stride loop and flushes one LDS
// histogram at the end.
constexpr int kMergeThreads = 256;
constexpr int kMergeBlocks = 512;

__global__ __launch_bounds__(kMergeThreads) void router_merge_kernel(RouterArgs a, int NS, CtrlArgs c) {
    __shared__ int hist[1024];
    __shared__ unsigned long long key[kMergeThreads];
    __shared__ float sel[kMergeThreads];  // selected scores, [token of the group][rank]
    const int E = a.E, K = a.K;
    const int KL = a.alpha ? K + 1 : K;  // candidates per slice
    const int per_tok = NS * KL;         // <= kMaxSlices * kMaxK = kMergeThreads
    const int tpg = kMergeThreads / per_tok;
    const int tid = threadIdx.x;
    const int tt = tid / per_tok, pos = tid - tt * per_tok;
    const int sl = pos / KL, r = pos - sl * KL;
    for (int e = tid; e < E; e += kMergeThreads) hist[e] = 0;
    const int64_t groups = (a.T + tpg - 1) / tpg;
    for (int64_t g = blockIdx.x; g < groups; g += gridDim.x) {
        const int64_t tok = g * tpg + tt;
        const bool act = tt < tpg && tok < a.T;
        float s = 0.0f;
        int e = 0;
        unsigned long long k = 0ull;
        if (act) {
            const int64_t gi = tok * per_tok + pos;
            s = a.cand_s[gi];
            e = a.cand_i[gi];
            k = rank_key(a.cand_v[gi], e);
        }
        __syncthreads();  // the previous group is done with key[] and sel[]
        key[tid] = k;
        __syncthreads();
        int rank = r;
        if (act) {
            for (int o = 0; o < NS; ++o) {
                if (o == sl) continue;
                const int b = tt * per_tok + o * KL;
                for (int j = 0; j < KL; ++j) rank += (key[b + j] > k) ? 1 : 0;
            }
            if (rank < K) {
                sel[tt * K + rank] = s;
                a.idx[tok * K + rank] = e;
                atomicAdd(&hist[e], 1);
            } else if (rank == K && a.alpha) {
                a.alpha[tok] = rank_key_value(k);  // the cutoff: the biased value of rank K
            }
        }
        __syncthreads();
        if (act && rank < K) {
            // den: fp32 sum of the selected unbiased scores in rank order
            float den = 0.0f;
            for (int j = 0; j < K; ++j) den = den + sel[tt * K + j];
            a.w[tok * K + rank] = (den == 0.0f) ? 1.0f / (float)K : s / den;
        }
    }
    __syncthreads();
    flush_hist(hist, a.counts, E);
    if (c.ticket) {
        __shared__ CtrlScratch csh;
        controller_tail<1024 / kMergeThreads>(a.counts, E, c.Ki, c.Kd, c.sign_mode, c.center, c.bias, c.e_prev,
                                          c.step, c.status, c.stats, c.ticket, csh);
    }
}

// Merge by token tile (NS*K <= 64): a few workgroups walk the 128-token tiles
// in a grid-stride loop.  A tile's NS*K candidates per token go to LDS; each
// candidate's final rank is its position in its slice's list plus the other
// slices' candidates above it (keys are distinct, as the experts are).  The
// next tile's candidates are fetched into registers while the current one is
// ranked.  The workgroup's histogram is flushed once, right after its last
// tile's ranking, so the count atomics overlap that tile's output stores (few
// workgroups: few, spread-out flushes instead of a burst on the same
// counters).
constexpr int kTileThreads = 512;
constexpr int kTileTokens = 128;

__global__ __launch_bounds__(kTileThreads) void router_merge_tile_kernel(RouterArgs a, int NS, CtrlArgs c) {
    __shared__ int hist[1024];
    __shared__ unsigned long long mk[kTileTokens * 64];
    __shared__ float ms[kTileTokens * 64];
    __shared__ float msel[kTileTokens * kMaxK];
    __shared__ int midx[kTileTokens * kMaxK];
    __shared__ float mden[kTileTokens];  // per token: the fp32 sum of its selected scores in rank order
    const int E = a.E, K = a.K;
    const int KL = a.alpha ? K + 1 : K;  // candidates per slice
    const int NSK = NS * KL;             // <= 64
    const int tid = threadIdx.x;
    for (int e = tid; e < E; e += kTileThreads) hist[e] = 0;
    const int64_t ntiles = (a.T + kTileTokens - 1) / kTileTokens;

    // A thread's candidates of tile g (slots past the tile's candidates are
    // neither loaded nor used).
    constexpr int kIt = kTileTokens * 64 / kTileThreads;
    float cv[kIt], cs[kIt];
    int ci[kIt];
    auto fetch = [&](int64_t g) {
        const int64_t t0 = g * kTileTokens;
        const int nt = (int)((a.T - t0) < kTileTokens ? (a.T - t0) : kTileTokens);
        const int n = nt * NSK;
#pragma unroll
        for (int it = 0; it < kIt; ++it) {
            const int c = tid + it * kTileThreads;
            if (c < n) {
                const int64_t gi = t0 * NSK + c;  // candidates of token t: [t][slice][K]
                cv[it] = a.cand_v[gi];
                cs[it] = a.cand_s[gi];
                ci[it] = a.cand_i[gi];
            }
        }
    };
    int64_t g = blockIdx.x;
    if (g < ntiles) fetch(g);
    for (; g < ntiles; g += gridDim.x) {
        const int64_t tok0 = g * kTileTokens;
        const int ntok = (int)((a.T - tok0) < kTileTokens ? (a.T - tok0) : kTileTokens);
        const int n = ntok * NSK;
        __syncthreads();  // the previous tile is done with the LDS arrays
#pragma unroll
        for (int it = 0; it < kIt; ++it) {
            const int c = tid + it * kTileThreads;
            if (c < n) {
                mk[c] = rank_key(cv[it], ci[it]);
                ms[c] = cs[it];
            }
        }
        if (g + gridDim.x < ntiles) fetch(g + gridDim.x);
        __syncthreads();
        if (NS == 2) {
            // Each slice's list is in rank order: a two-pointer merge per
            // token (the lists hold KL distinct keys each; key 0 marks an
            // exhausted list).  Each list's key after its head is read ahead,
            // and the gate weights' denominator is summed in rank order on
            // the way.
            for (int t = tid; t < ntok; t += kTileThreads) {
                const unsigned long long* L0 = mk + t * NSK;
                const unsigned long long* L1 = L0 + KL;
                const float* S0 = ms + t * NSK;
                const float* S1 = S0 + KL;
                int p0 = 0, p1 = 0;
                unsigned long long k0 = L0[0], k1 = L1[0];
                for (int r = 0; r < K; ++r) {
                    const bool take0 = k0 > k1;
                    const unsigned long long k = take0 ? k0 : k1;
                    msel[t * kMaxK + r] = take0 ? S0[p0] : S1[p1];
                    midx[t * kMaxK + r] = (int)~(unsigned)k;
                    atomicAdd(&hist[(int)~(unsigned)k], 1);
                    if (take0) {
                        ++p0;
                        k0 = p0 < KL ? L0[p0] : 0ull;
                    } else {
                        ++p1;
                        k1 = p1 < KL ? L1[p1] : 0ull;
                    }
                }
                // the cutoff: the biased value of rank K
                if (a.alpha) a.alpha[tok0 + t] = rank_key_value(k0 > k1 ? k0 : k1);
            }
        } else {
            // A candidate's final rank: its rank in its own slice plus the
            // other slices' candidates above it.
            for (int c = tid; c < n; c += kTileThreads) {
                const int t = c / NSK, pos = c - t * NSK;
                const int sl = pos / KL, r = pos - sl * KL;
                const unsigned long long k = mk[c];
                int rank = r;
                for (int o = 0; o < NS; ++o) {
                    if (o == sl) continue;
                    const unsigned long long* lo = mk + t * NSK + o * KL;
#pragma unroll 8
                    for (int j = 0; j < KL; ++j) rank += (lo[j] > k) ? 1 : 0;
                }
                if (rank < K) {
                    msel[t * kMaxK + rank] = ms[c];
                    midx[t * kMaxK + rank] = (int)~(unsigned)k;
                    atomicAdd(&hist[(int)~(unsigned)k], 1);
                } else if (rank == K && a.alpha) {
                    a.alpha[tok0 + t] = rank_key_value(k);
                }
            }
            __syncthreads();
            for (int t = tid; t < ntok; t += kTileThreads) {
                float den = 0.0f;
                for (int j = 0; j < K; ++j) den = den + msel[t * kMaxK + j];
                mden[t] = den;
            }
        }
        __syncthreads();
        // The histogram is complete after the last tile's merge: its global
        // flush overlaps the output stores below.
        if (g + gridDim.x >= ntiles) flush_hist(hist, a.counts, E);
        // gate weights: den is the fp32 sum of the selected unbiased scores
        // in rank order
        for (int c = tid; c < ntok * K; c += kTileThreads) {
            const int t = c / K, r = c - t * K;
            float den = 0.0f;
#pragma unroll 8
            for (int j = 0; j < K; ++j) den = den + msel[t * kMaxK + j];
            const int e = midx[t * kMaxK + r];
            const int64_t tok = tok0 + t;
            a.idx[tok * K + r] = e;
            a.w[tok * K + r] = (den == 0.0f) ? 1.0f / (float)K : msel[t * kMaxK + r] / den;
        }
    }
    if (c.ticket) {
        __shared__ CtrlScratch csh;
        controller_tail<1024 / kTileThreads>(a.counts, E, c.Ki, c.Kd, c.sign_mode, c.center, c.bias, c.e_prev,
                                          c.step, c.status, c.stats, c.ticket, csh);
    }
}

// Router matrix [E][d] -> packed layout: output piece p (16 bytes) = lane
// slot l = p%64 of the 1 KB piece (b, c, s) with p/64 = (b*NCH + c)*2 + s,
// i.e. row 16 b + l%16, bytes c*128 + 64 s + 16 (l/16).
__global__ void pack_weight_kernel(const char* __restrict__ W, char* __restrict__ P, int64_t RB, int64_t pieces) {
    const int64_t nch = RB / 128;
    for (int64_t o = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; o < pieces;
         o += (int64_t)gridDim.x * blockDim.x) {
        const int l = (int)(o & 63), s = (int)((o >> 6) & 1);
        const int64_t c = (o >> 7) % nch, b = (o >> 7) / nch;
        const int64_t src = (b * 16 + (l & 15)) * RB + c * 128 + 64 * s + 16 * (l >> 4);
        *reinterpret_cast<uint4*>(P + o * 16) = *reinterpret_cast<const uint4*>(W + src);
    }
}

// One launch of kernel k; with an event set, an extended launch that records
// the kernel's own start and end timestamps in them.
template <class Kern>
hipError_t launch_kernel(Kern k, int64_t blocks, int threads, const RouterArgs& a, int NS, hipStream_t stream,
                         hipEvent_t start, hipEvent_t stop) {
    if (start || stop)
        hipExtLaunchKernelGGL(k, dim3((unsigned)blocks), dim3(threads), 0, stream, start, stop, 0, a, NS);
    else
        hipLaunchKernelGGL(k, dim3((unsigned)blocks), dim3(threads), 0, stream, a, NS);
    return hipGetLastError();
}

template <bool F32, bool PACKED, int WAVES, int TBW, int NBLK, bool SM = false>
hipError_t launch32(const RouterArgs& a, int NS, hipStream_t stream, hipEvent_t start, hipEvent_t stop) {
    using C = Cfg32<F32, WAVES, TBW, NBLK>;
    const int64_t blocks = (a.T + C::BT - 1) / C::BT * NS;
    return launch_kernel(router32_kernel<F32, PACKED, WAVES, TBW, NBLK, SM>, blocks, C::NT, a, NS, stream, start,
                         stop);
}

template <bool PACKED, int WAVES, int TT, int ET, bool SM = false>
hipError_t launch16(const RouterArgs& a, int NS, hipStream_t stream, hipEvent_t start, hipEvent_t stop) {
    using C = Cfg16<WAVES, TT, ET>;
    const int64_t blocks = (a.T + C::BT - 1) / C::BT * NS;
    return launch_kernel(router16_kernel<PACKED, WAVES, TT, ET, SM>, blocks, C::NT, a, NS, stream, start, stop);
}

template <bool PACKED>
hipError_t launch_layout(const RouterTiling& t, const RouterArgs& a, int NS, hipStream_t stream, hipEvent_t e0,
                         hipEvent_t e1) {
    if (a.softmax) {
        // softmax mode: compiled for the tilings marked in kTilings only
        switch (t.id) {
            case 2: return launch32<false, PACKED, 8, 2, 3, true>(a, NS, stream, e0, e1);
            case 4: return launch32<false, PACKED, 4, 4, 1, true>(a, NS, stream, e0, e1);
            case 5: return launch32<true, PACKED, 4, 4, 1, true>(a, NS, stream, e0, e1);
            case 7: return launch16<PACKED, 8, 4, 6, true>(a, NS, stream, e0, e1);
            default: return hipErrorInvalidValue;
        }
    }
    switch (t.id) {
        case 1: return launch32<false, PACKED, 4, 4, 3>(a, NS, stream, e0, e1);
        case 2: return launch32<false, PACKED, 8, 2, 3>(a, NS, stream, e0, e1);
        case 3: return launch32<false, PACKED, 4, 4, 2>(a, NS, stream, e0, e1);
        case 4: return launch32<false, PACKED, 4, 4, 1>(a, NS, stream, e0, e1);
        case 5: return launch32<true, PACKED, 4, 4, 1>(a, NS, stream, e0, e1);
        case 6: return launch16<PACKED, 8, 8, 3>(a, NS, stream, e0, e1);
        case 7: return launch16<PACKED, 8, 4, 6>(a, NS, stream, e0, e1);
        default: return hipErrorInvalidValue;
    }
}

// id, fp32 input, waves, tokens per workgroup, experts per wave, preference
// among tilings with equally few padded experts (lower first), softmax mode
// compiled.
const RouterTiling kTilings[] = {
    {1, 0, 4, 128, 96, 2, 0},  // bf16 32x32 tiles: 128 tokens x 384 experts per workgroup
    {2, 0, 8, 64, 96, 5, 1},   // bf16 32x32 tiles: 64 tokens x 768 experts
    {3, 0, 4, 128, 64, 3, 0},  // bf16 32x32 tiles: 128 tokens x 256 experts
    {4, 0, 4, 128, 32, 4, 1},  // bf16 32x32 tiles: 128 tokens x 128 experts
    {5, 1, 4, 128, 32, 0, 1},  // fp32 32x32 tiles: 128 tokens x 128 experts
    {6, 0, 8, 128, 48, 0, 0},  // bf16 16x16 tiles: 128 tokens x 384 experts, two waves per SIMD
    {7, 0, 8, 64, 96, 1, 1},   // bf16 16x16 tiles: 64 tokens x 768 experts, two waves per SIMD
};

}  // namespace

int router_tiling_count() { return (int)(sizeof(kTilings) / sizeof(kTilings[0])); }
RouterTiling router_tiling(int i) { return kTilings[i]; }

hipError_t launch_router_score_select(const RouterTiling& t, const RouterArgs& a, hipStream_t stream,
                                      hipEvent_t start, hipEvent_t stop) {
    const int NS = router_slices(t, a.E);
    return a.w_packed ? launch_layout<true>(t, a, NS, stream, start, stop)
                      : launch_layout<false>(t, a, NS, stream, start, stop);
}

hipError_t launch_router_merge(const RouterTiling& t, const RouterArgs& a, const CtrlArgs* ctrl,
                               hipStream_t stream) {
    const int NS = router_slices(t, a.E);
    if (NS <= 1) return hipSuccess;
    CtrlArgs c{};
    if (ctrl) c = *ctrl;
    const int KL = a.alpha ? a.K + 1 : a.K;
    if (NS * KL <= 64) {
        // one workgroup per CU at most (its LDS takes most of one): larger
        // batches walk several tiles per workgroup, each next tile's
        // candidates fetched during the current one's merge
        int cus = 0, dev = 0;
        if (hipGetDevice(&dev) != hipSuccess ||
            hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus < 1)
            cus = 256;
        int64_t blocks = (a.T + kTileTokens - 1) / kTileTokens;
        if (blocks > cus) blocks = cus;
        hipLaunchKernelGGL(router_merge_tile_kernel, dim3((unsigned)blocks), dim3(kTileThreads), 0, stream, a, NS,
                           c);
        return hipGetLastError();
    }
    const int tpg = kMergeThreads / (NS * KL);
    int64_t groups = (a.T + tpg - 1) / tpg;
    if (groups > kMergeBlocks) groups = kMergeBlocks;
    hipLaunchKernelGGL(router_merge_kernel, dim3((unsigned)groups), dim3(kMergeThreads), 0, stream, a, NS, c);
    return hipGetLastError();
}

hipError_t launch_pack_weight(const void* W, void* P, int E, int64_t row_bytes, hipStream_t stream) {
    const int64_t pieces = (int64_t)E * row_bytes / 16;
    int64_t blocks = (pieces + 255) / 256;
    if (blocks > 4096) blocks = 4096;
    hipLaunchKernelGGL(pack_weight_kernel, dim3((unsigned)blocks), dim3(256), 0, stream,
                       reinterpret_cast<const char*>(W), reinterpret_cast<char*>(P), row_bytes, pieces);
    return hipGetLastError();
}

}  // namespace idb
