// Fused router step for gfx950: gate contraction z = W_r x on MFMA (Sec. 2.2),
// sigmoid scores, bias-adjusted Top-K (Eq. pid-routing), gate weights from the
// unbiased scores and per-expert load counts (Eq. pid-error).  The T x E score
// matrix stays in registers and LDS.
//
// Tiling.  A workgroup owns BT = 32*TBW tokens and one slice of BE =
// WAVES*32*NBLK experts.  Each wave owns all BT tokens and its own 32*NBLK
// experts: its router rows are private to it and go straight from global
// memory into MFMA A-operand registers, while the token tile is shared by the
// waves through LDS.  The contraction runs over 128-byte chunks of each row.
// Within a chunk, lane half h of every 32-lane group consumes bytes
// [64h, 64h + 64) in four 16-byte units, identically for both operands, so the
// k order agrees between them.
//
// Token tile: staged through registers into two LDS stages of 144-byte rows
// (128 bytes + 16 of padding, so the MFMA B-operand reads of 32 rows are free
// of bank conflicts), loaded one chunk ahead of use.
//
// Router matrix: either row-major [E][d] (each A-operand load touches 32 rows)
// or the packed layout written by idb_router_pack_weight, in which the 64
// lanes' 16-byte A operands of one (32-expert block, chunk, unit) are one
// contiguous 1 KB piece.
//
// MFMA 32x32 output layout (C = W_block * x_block^T): lane l holds token
// (l % 32) of the block and experts 8*(r/4) + 4*(l/32) + (r%4), r < 16.  So a
// token's BE scores are spread over 2*WAVES lanes, 16*NBLK per lane.
//
// Epilogue per token and slice (exact for any input):
//   1. s = sigmoid(z) (computed once), v = fl32(s + b).
//   2. Each lane splits its values into G groups, 16 group maxima per token;
//      tau = the K-th largest group maximum <= the token's K-th largest v.
//   3. Each lane counts its values >= tau; a prefix over the token's lanes
//      gives every lane its write offset, and the candidates (typically about
//      K + 5) are written to an LDS list without atomics.
//   4. Candidate rank = number of candidates above it in the order (v desc,
//      index asc); ranks < K are the slice's selection, in rank order.
//   5. Lists that would overflow (heavy ties, K > 16) are resolved one token
//      at a time: the token's values are gathered into an LDS row and one wave
//      takes K rounds of wave-wide argmax.
//   6. One slice: gate weights, outputs and an LDS histogram flushed with one
//      atomic per non-zero bin.  Several slices: the slice's K candidates go
//      to the workspace and router_merge_kernel combines them.
#include "common.h"
#include "internal.h"

#pragma clang fp contract(off)

namespace idb {

namespace {

constexpr int kCap = 32;     // candidate list capacity per token and slice
constexpr int kRowPad = 144;  // LDS bytes per staged token row (128 + 16 pad)
constexpr int kMaxSlices = 8;

template <bool F32, int WAVES, int TBW, int NBLK>
struct Cfg {
    static constexpr int NT = WAVES * 64;
    static constexpr int BT = 32 * TBW;
    static constexpr int WE = 32 * NBLK;
    static constexpr int BE = WAVES * WE;
    static constexpr int NV = 16 * NBLK;     // values per lane per token
    static constexpr int G = 8 / WAVES;      // groups per lane: 2*WAVES*G = 16
    static constexpr int GS = NV / G;        // values per group
    static constexpr int TPT = NT / BT;      // threads per token in the ranking
    static constexpr int NLANES = 2 * WAVES;  // lanes holding one token's slice
    static constexpr int PPT = BT * 8 / NT;  // 16-byte token-tile pieces per thread per chunk
    static constexpr int STAGE = BT * kRowPad;
    static constexpr int MAIN_LDS = 2 * STAGE;
    // epilogue LDS layout (bytes).  Per-token rows are padded (17, NLANES+1 and
    // 36 words) so the 32 tokens of a wave fall on different LDS banks; the
    // 36-word rows are also 16-byte aligned for vector reads.
    static constexpr int GMS = 17;            // group-maximum row stride (words)
    static constexpr int CNS = NLANES + 1;    // count row stride
    static constexpr int LST = kCap + 4;      // candidate / selection row stride
    static constexpr int OFF_GM = 0;
    static constexpr int OFF_TAU = OFF_GM + BT * GMS * 4;
    static constexpr int OFF_CNT = OFF_TAU + BT * 4;
    static constexpr int OFF_LV = ((OFF_CNT + BT * CNS * 4) + 15) / 16 * 16;
    static constexpr int OFF_LS = OFF_LV + BT * LST * 4;
    static constexpr int OFF_LI = OFF_LS + BT * LST * 4;
    static constexpr int OFF_SV = OFF_LI + BT * LST * 4;
    static constexpr int OFF_SS = OFF_SV + BT * LST * 4;
    static constexpr int OFF_SI = OFF_SS + BT * LST * 4;
    static constexpr int OFF_OVF = OFF_SI + BT * LST * 4;
    static constexpr int OFF_ROWV = OFF_OVF + 16 * 4;
    static constexpr int OFF_ROWS = OFF_ROWV + BE * 4;
    static constexpr int OFF_HIST = OFF_ROWS + BE * 4;
    static constexpr int EPI_LDS = OFF_HIST + 1024 * 4;
    static constexpr int LDS = MAIN_LDS > EPI_LDS ? MAIN_LDS : EPI_LDS;
    static_assert(BT <= NT, "one thread per token in the threshold step");
    static_assert(NV % G == 0, "groups must split a lane's values evenly");
    static_assert(PPT * NT == BT * 8, "token-tile pieces must split evenly over threads");
    static_assert(BT <= 16 * 32, "overflow bitmask size");
    static_assert(BE % 64 == 0, "overflow gather row is read 64 lanes at a time");
};

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

__device__ __forceinline__ float comp4(const float4& f, int i) {
    return i == 0 ? f.x : (i == 1 ? f.y : (i == 2 ? f.z : f.w));
}

template <bool F32, bool PACKED, int WAVES, int TBW, int NBLK>
__global__ __launch_bounds__(WAVES * 64) void router_score_select_kernel(RouterArgs a, int NS) {
    using C = Cfg<F32, WAVES, TBW, NBLK>;
    __shared__ __attribute__((aligned(16))) unsigned char smem[C::LDS];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int h = lane >> 5;
    const int l32 = lane & 31;

    // XCD-aware block order: consecutive blocks land on different XCDs, so
    // remap to give each XCD a contiguous run of (tile, slice) pairs; the
    // slices of one token tile then share their token rows in that XCD's L2.
    const int nb = gridDim.x;
    int L = blockIdx.x;
    if ((nb & 7) == 0) L = (blockIdx.x & 7) * (nb >> 3) + (blockIdx.x >> 3);
    const int tile = L / NS;
    const int slice = L - tile * NS;

    const int64_t T = a.T;
    const int E = a.E;
    const int K = a.K;
    const int64_t tok0 = (int64_t)tile * C::BT;
    const int e_wave0 = slice * C::BE + wave * C::WE;
    const int64_t RB = (int64_t)a.d * (F32 ? 4 : 2);
    const int NCH = (int)(RB / 128);

    if (a.zero_counts && blockIdx.x == 0)
        for (int e = tid; e < E; e += C::NT) a.counts[e] = 0;

    // ---------------------------------------------------------------- contraction
    // A operands (router rows): byte strides of a chunk and of a unit.
    constexpr int WU = PACKED ? 1024 : 16;
    constexpr int64_t WCH = PACKED ? 4096 : 128;
    const char* wrow[NBLK];
#pragma unroll
    for (int nbk = 0; nbk < NBLK; ++nbk) {
        int blk = (e_wave0 + nbk * 32) / 32;
        blk = blk < E / 32 ? blk : E / 32 - 1;  // padding blocks read a valid block; masked later
        if constexpr (PACKED)
            wrow[nbk] = reinterpret_cast<const char*>(a.W) + (int64_t)blk * NCH * 4096 + lane * 16;
        else
            wrow[nbk] = reinterpret_cast<const char*>(a.W) + (int64_t)(blk * 32 + l32) * RB + 64 * h;
    }
    // Token-tile pieces: thread piece p = tid + NT*q covers row p/8, bytes
    // 16*(p%8) of the chunk.  Rows past T re-read row T-1 (never output).
    const char* xsrc[C::PPT];
    int xdst[C::PPT];
#pragma unroll
    for (int q = 0; q < C::PPT; ++q) {
        const int p = tid + C::NT * q;
        const int row = p >> 3, c16 = p & 7;
        int64_t tok = tok0 + row;
        tok = tok < T ? tok : T - 1;
        xsrc[q] = reinterpret_cast<const char*>(a.x) + tok * RB + c16 * 16;
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

    // Software pipeline.  W operands: one register set refilled unit by unit
    // (right after the MFMAs of unit u of chunk c, the same registers start
    // loading unit u of chunk c+1).  Token tile: loaded into staging registers
    // at the top of chunk c for chunk c+1, stored into the idle LDS stage at
    // the end of chunk c.  Vector-memory loads complete in order, and in this
    // issue order each wait the compiler inserts covers only the data about
    // to be used.
    uint4 w[NBLK][4], xr[C::PPT];
    auto load_x = [&](int c) {
#pragma unroll
        for (int q = 0; q < C::PPT; ++q) xr[q] = ld16(xsrc[q] + c * 128);
    };
    auto store_x = [&](int stage) {
#pragma unroll
        for (int q = 0; q < C::PPT; ++q) *reinterpret_cast<uint4*>(smem + stage * C::STAGE + xdst[q]) = xr[q];
    };

    load_x(0);
#pragma unroll
    for (int nbk = 0; nbk < NBLK; ++nbk)
#pragma unroll
        for (int u = 0; u < 4; ++u) w[nbk][u] = ld16(wrow[nbk] + WU * u);
    store_x(0);
    __syncthreads();
    for (int c = 0; c < NCH; ++c) {
        const bool more = c + 1 < NCH;
        if (more) load_x(c + 1);
        const unsigned char* st = smem + (c & 1) * C::STAGE + boff;
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            uint4 bx[TBW];
#pragma unroll
            for (int tb = 0; tb < TBW; ++tb) bx[tb] = *reinterpret_cast<const uint4*>(st + tb * 32 * kRowPad + 16 * u);
#pragma unroll
            for (int tb = 0; tb < TBW; ++tb)
#pragma unroll
                for (int nbk = 0; nbk < NBLK; ++nbk) acc[tb][nbk] = mfma_unit<F32>(w[nbk][u], bx[tb], acc[tb][nbk]);
            if (more) {
#pragma unroll
                for (int nbk = 0; nbk < NBLK; ++nbk) w[nbk][u] = ld16(wrow[nbk] + (c + 1) * WCH + WU * u);
            }
        }
        if (more) store_x((c + 1) & 1);
        __syncthreads();
    }

    // ---------------------------------------------------------------- epilogue
    float* gm = reinterpret_cast<float*>(smem + C::OFF_GM);
    float* tau_s = reinterpret_cast<float*>(smem + C::OFF_TAU);
    int* cnt = reinterpret_cast<int*>(smem + C::OFF_CNT);
    float* lv = reinterpret_cast<float*>(smem + C::OFF_LV);
    float* ls = reinterpret_cast<float*>(smem + C::OFF_LS);
    int* li = reinterpret_cast<int*>(smem + C::OFF_LI);
    float* sv = reinterpret_cast<float*>(smem + C::OFF_SV);
    float* ss = reinterpret_cast<float*>(smem + C::OFF_SS);
    int* si = reinterpret_cast<int*>(smem + C::OFF_SI);
    unsigned* ovf = reinterpret_cast<unsigned*>(smem + C::OFF_OVF);
    float* rowv = reinterpret_cast<float*>(smem + C::OFF_ROWV);
    float* rows = reinterpret_cast<float*>(smem + C::OFF_ROWS);
    int* hist = reinterpret_cast<int*>(smem + C::OFF_HIST);

    // Expert of accumulator (nbk, r): ebase + 32 nbk + 8 (r/4) + (r%4).  E is a
    // multiple of 32, so a whole 32-expert block is either real or padding.
    const int ebase = e_wave0 + 4 * h;
    auto blk_real = [&](int nbk) { return e_wave0 + nbk * 32 < E; };
    const int slot = wave * 2 + h;  // this lane's position among the token's lanes

    // this lane's bias values, four consecutive experts per (nbk, r/4)
    float4 b4[NBLK][4];
#pragma unroll
    for (int nbk = 0; nbk < NBLK; ++nbk)
#pragma unroll
        for (int r4 = 0; r4 < 4; ++r4) {
            const int e = ebase + nbk * 32 + 8 * r4;
            b4[nbk][r4] = blk_real(nbk) ? make_float4(a.bias[e], a.bias[e + 1], a.bias[e + 2], a.bias[e + 3])
                                        : make_float4(0.f, 0.f, 0.f, 0.f);
        }
    for (int e = tid; e < 1024; e += C::NT) hist[e] = 0;
    if (tid < 16) ovf[tid] = 0;

    // 1. scores, once (and the optional debug dump of exactly these values)
#pragma unroll
    for (int tb = 0; tb < TBW; ++tb)
#pragma unroll
        for (int nbk = 0; nbk < NBLK; ++nbk)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[tb][nbk][r] = sigmoid_fast(acc[tb][nbk][r]);
    if (a.dump) {
#pragma unroll
        for (int tb = 0; tb < TBW; ++tb) {
            const int64_t tok = tok0 + tb * 32 + l32;
            if (tok < T) {
#pragma unroll
                for (int nbk = 0; nbk < NBLK; ++nbk)
                    if (blk_real(nbk)) {
#pragma unroll
                        for (int r4 = 0; r4 < 4; ++r4)
                            *reinterpret_cast<float4*>(a.dump + tok * E + ebase + nbk * 32 + 8 * r4) =
                                make_float4(acc[tb][nbk][4 * r4], acc[tb][nbk][4 * r4 + 1], acc[tb][nbk][4 * r4 + 2],
                                            acc[tb][nbk][4 * r4 + 3]);
                    }
            }
        }
    }

    // 2. group maxima of v = s + b
#pragma unroll
    for (int tb = 0; tb < TBW; ++tb) {
        float gmx[C::G];
#pragma unroll
        for (int g = 0; g < C::G; ++g) gmx[g] = -INFINITY;
#pragma unroll
        for (int nbk = 0; nbk < NBLK; ++nbk) {
            if (!blk_real(nbk)) continue;
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int g = (nbk * 16 + r) / C::GS;
                gmx[g] = fmaxf(gmx[g], acc[tb][nbk][r] + comp4(b4[nbk][r >> 2], r & 3));
            }
        }
#pragma unroll
        for (int g = 0; g < C::G; ++g) gm[(tb * 32 + l32) * C::GMS + slot * C::G + g] = gmx[g];
    }
    __syncthreads();

    // 3. per-token threshold
    if (tid < C::BT) {
        float g16[16];
#pragma unroll
        for (int i = 0; i < 16; ++i) g16[i] = gm[tid * C::GMS + i];
        sort16_ascending(g16);
        float tau = -INFINITY;
        if (K <= 16) {
#pragma unroll
            for (int i = 0; i < 16; ++i)
                if (i == 16 - K) tau = g16[i];
        }
        tau_s[tid] = tau;
    }
    __syncthreads();

    // 4. candidates v >= tau: count, prefix over the token's lanes, write
    float taus[TBW];
#pragma unroll
    for (int tb = 0; tb < TBW; ++tb) {
        const int tl = tb * 32 + l32;
        taus[tb] = tau_s[tl];
        int n = 0;
#pragma unroll
        for (int nbk = 0; nbk < NBLK; ++nbk) {
            if (!blk_real(nbk)) continue;
#pragma unroll
            for (int r = 0; r < 16; ++r) n += (acc[tb][nbk][r] + comp4(b4[nbk][r >> 2], r & 3) >= taus[tb]) ? 1 : 0;
        }
        cnt[tl * C::CNS + slot] = n;
    }
    __syncthreads();
#pragma unroll
    for (int tb = 0; tb < TBW; ++tb) {
        const int tl = tb * 32 + l32;
        int off = 0, total = 0;
#pragma unroll
        for (int o = 0; o < C::NLANES; ++o) {
            const int n = cnt[tl * C::CNS + o];
            off += (o < slot) ? n : 0;
            total += n;
        }
        if (total > kCap) {
            if (slot == 0) atomicOr(&ovf[tl >> 5], 1u << (tl & 31));
            continue;
        }
        if (tok0 + tl >= T) continue;
        const float tau = taus[tb];
#pragma unroll
        for (int nbk = 0; nbk < NBLK; ++nbk) {
            if (!blk_real(nbk)) continue;
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const float s = acc[tb][nbk][r];
                const float v = s + comp4(b4[nbk][r >> 2], r & 3);
                if (v >= tau) {
                    lv[tl * C::LST + off] = v;
                    ls[tl * C::LST + off] = s;
                    li[tl * C::LST + off] = ebase + nbk * 32 + 8 * (r >> 2) + (r & 3);
                    ++off;
                }
            }
        }
    }
    __syncthreads();

    // 5. rank the candidates of every token whose list did not overflow.  The
    // token's threads hold its whole list in registers (entries past n read
    // as (-inf, INT_MAX), which rank below everything) and count, for each of
    // their candidates, the entries that rank above it.
    {
        const int tl = tid / C::TPT, q = tid % C::TPT;
        int n = 0;
#pragma unroll
        for (int o = 0; o < C::NLANES; ++o) n += cnt[tl * C::CNS + o];
        if (n <= kCap) {
            float cv[kCap];
            int ci[kCap];
#pragma unroll
            for (int o4 = 0; o4 < kCap / 4; ++o4) {
                const float4 v4 = *reinterpret_cast<const float4*>(lv + tl * C::LST + 4 * o4);
                const int4 i4 = *reinterpret_cast<const int4*>(li + tl * C::LST + 4 * o4);
                cv[4 * o4] = v4.x; cv[4 * o4 + 1] = v4.y; cv[4 * o4 + 2] = v4.z; cv[4 * o4 + 3] = v4.w;
                ci[4 * o4] = i4.x; ci[4 * o4 + 1] = i4.y; ci[4 * o4 + 2] = i4.z; ci[4 * o4 + 3] = i4.w;
            }
#pragma unroll
            for (int o = 0; o < kCap; ++o)
                if (o >= n) {
                    cv[o] = -INFINITY;
                    ci[o] = 0x7fffffff;
                }
            for (int c = q; c < n; c += C::TPT) {
                const float vc = lv[tl * C::LST + c];
                const int ic = li[tl * C::LST + c];
                int rank = 0;
#pragma unroll
                for (int o = 0; o < kCap; ++o) rank += ranks_above(cv[o], ci[o], vc, ic) ? 1 : 0;
                if (rank < K) {
                    sv[tl * C::LST + rank] = vc;
                    ss[tl * C::LST + rank] = ls[tl * C::LST + c];
                    si[tl * C::LST + rank] = ic;
                }
            }
        }
    }

    // 6. overflowing tokens, one at a time: gather the token's slice into an
    // LDS row, then wave 0 takes K rounds of wave-wide argmax over it.
    for (int word = 0; word < C::BT / 32; ++word) {
        unsigned bits = ovf[word];  // uniform: written before the last barrier
        while (bits) {
            const int tl = word * 32 + __builtin_ctz(bits);
            bits &= bits - 1;
            const int tb = tl >> 5;
            if ((tl & 31) == l32) {
#pragma unroll
                for (int tbb = 0; tbb < TBW; ++tbb) {
                    if (tbb != tb) continue;
#pragma unroll
                    for (int nbk = 0; nbk < NBLK; ++nbk)
#pragma unroll
                        for (int r = 0; r < 16; ++r) {
                            const int p = wave * C::WE + nbk * 32 + 8 * (r >> 2) + 4 * h + (r & 3);
                            const float s = acc[tbb][nbk][r];
                            rows[p] = s;
                            rowv[p] = blk_real(nbk) ? s + comp4(b4[nbk][r >> 2], r & 3) : -INFINITY;
                        }
                }
            }
            __syncthreads();
            if (wave == 0) {
                unsigned taken = 0;
                for (int r = 0; r < K; ++r) {
                    float bv = -INFINITY, bs = 0.0f;
                    int bi = 0x7fffffff, bq = -1;
#pragma unroll
                    for (int q = 0; q < C::BE / 64; ++q) {
                        const int p = lane + 64 * q;
                        const float v = rowv[p];
                        const int e = slice * C::BE + p;
                        if (!((taken >> q) & 1u) && v != -INFINITY && ranks_above(v, e, bv, bi)) {
                            bv = v;
                            bs = rows[p];
                            bi = e;
                            bq = q;
                        }
                    }
                    float wv = bv, ws = bs;
                    int wi = bi;
#pragma unroll
                    for (int off = 32; off >= 1; off >>= 1) {
                        const float ov = __shfl_xor(wv, off);
                        const float os = __shfl_xor(ws, off);
                        const int oi = __shfl_xor(wi, off);
                        if (ranks_above(ov, oi, wv, wi)) {
                            wv = ov;
                            ws = os;
                            wi = oi;
                        }
                    }
                    if (bi == wi && bq >= 0) taken |= 1u << bq;
                    if (lane == 0) {
                        sv[tl * C::LST + r] = wv;
                        ss[tl * C::LST + r] = ws;
                        si[tl * C::LST + r] = wi;
                    }
                }
            }
            __syncthreads();
        }
    }
    __syncthreads();

    // 7. outputs
    {
        const int tl = tid / C::TPT, q = tid % C::TPT;
        const int64_t tok = tok0 + tl;
        if (tok < T) {
            if (NS > 1) {
                const int64_t base = (tok * NS + slice) * K;
                for (int r = q; r < K; r += C::TPT) {
                    a.cand_v[base + r] = sv[tl * C::LST + r];
                    a.cand_s[base + r] = ss[tl * C::LST + r];
                    a.cand_i[base + r] = si[tl * C::LST + r];
                }
            } else {
                // gate weights: den is the fp32 sum of the selected unbiased
                // scores in rank order
                float den = 0.0f;
#pragma unroll
                for (int r = 0; r < kMaxK; ++r)
                    if (r < K) den = den + ss[tl * C::LST + r];
                for (int r = q; r < K; r += C::TPT) {
                    const int e = si[tl * C::LST + r];
                    a.idx[tok * K + r] = e;
                    a.w[tok * K + r] = (den == 0.0f) ? 1.0f / (float)K : ss[tl * C::LST + r] / den;
                    if ((unsigned)e < (unsigned)E) atomicAdd(&hist[e], 1);
                }
            }
        }
    }
    if (NS == 1) {
        __syncthreads();
        for (int e = tid; e < E; e += C::NT)
            if (hist[e] != 0) atomicAdd(&a.counts[e], hist[e]);
    }
}

// Merge the slices' rank-ordered candidate lists into the final Top-K, compute
// the gate weights and count the assignments.  The workgroup copies its
// tokens' candidates into LDS with coalesced loads, then each thread merges
// one token.
constexpr int kMergeThreads = 256;

__global__ __launch_bounds__(kMergeThreads) void router_merge_kernel(RouterArgs a, int NS, int tokens_per_wg) {
    extern __shared__ __attribute__((aligned(16))) unsigned char dyn[];
    int* hist = reinterpret_cast<int*>(dyn);
    const int E = a.E, K = a.K;
    const int per_tok = NS * K;
    float* cv = reinterpret_cast<float*>(dyn + 4096);
    float* cs = cv + tokens_per_wg * per_tok;
    int* ci = reinterpret_cast<int*>(cs + tokens_per_wg * per_tok);
    const int tid = threadIdx.x;
    for (int e = tid; e < E; e += kMergeThreads) hist[e] = 0;
    for (int64_t tok_base = (int64_t)blockIdx.x * tokens_per_wg; tok_base < a.T;
         tok_base += (int64_t)gridDim.x * tokens_per_wg) {
        const int ntok = (int)((a.T - tok_base) < tokens_per_wg ? (a.T - tok_base) : tokens_per_wg);
        const int64_t g0 = tok_base * per_tok;
        __syncthreads();
        for (int i = tid; i < ntok * per_tok; i += kMergeThreads) {
            cv[i] = a.cand_v[g0 + i];
            cs[i] = a.cand_s[g0 + i];
            ci[i] = a.cand_i[g0 + i];
        }
        __syncthreads();
        for (int t = tid; t < ntok; t += kMergeThreads) {
            const int base = t * per_tok;
            int head[kMaxSlices];
#pragma unroll
            for (int s = 0; s < kMaxSlices; ++s) head[s] = 0;
            float sel_s[kMaxK];
            const int64_t tok = tok_base + t;
#pragma unroll
            for (int r = 0; r < kMaxK; ++r) {
                if (r < K) {
                    float bv = -INFINITY, bs = 0.0f;
                    int bi = 0x7fffffff, bsl = 0;
#pragma unroll
                    for (int s = 0; s < kMaxSlices; ++s) {
                        if (s < NS && head[s] < K) {
                            const int o = base + s * K + head[s];
                            if (ranks_above(cv[o], ci[o], bv, bi)) {
                                bv = cv[o];
                                bi = ci[o];
                                bs = cs[o];
                                bsl = s;
                            }
                        }
                    }
#pragma unroll
                    for (int s = 0; s < kMaxSlices; ++s) head[s] += (s == bsl) ? 1 : 0;
                    sel_s[r] = bs;
                    a.idx[tok * K + r] = bi;
                    if ((unsigned)bi < (unsigned)E) atomicAdd(&hist[bi], 1);
                }
            }
            float den = 0.0f;
#pragma unroll
            for (int r = 0; r < kMaxK; ++r)
                if (r < K) den = den + sel_s[r];
#pragma unroll
            for (int r = 0; r < kMaxK; ++r)
                if (r < K) a.w[tok * K + r] = (den == 0.0f) ? 1.0f / (float)K : sel_s[r] / den;
        }
    }
    __syncthreads();
    for (int e = tid; e < E; e += kMergeThreads)
        if (hist[e] != 0) atomicAdd(&a.counts[e], hist[e]);
}

// Router matrix [E][d] -> packed layout: for 32-expert block b, chunk c
// (128 bytes of each row), unit u (16 bytes), lane l = 32h + m, the 16 bytes
// at ((b*NCH + c)*4 + u)*1024 + 16 l are row 32b + m, bytes c*128 + 64h + 16u.
__global__ void pack_weight_kernel(const char* __restrict__ W, char* __restrict__ P, int64_t RB, int64_t pieces) {
    const int64_t nch = RB / 128;
    for (int64_t o = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; o < pieces;
         o += (int64_t)gridDim.x * blockDim.x) {
        const int l = (int)(o & 63), u = (int)((o >> 6) & 3);
        const int64_t c = (o >> 8) % nch, b = (o >> 8) / nch;
        const int m = l & 31, hh = l >> 5;
        const int64_t src = (b * 32 + m) * RB + c * 128 + 64 * hh + 16 * u;
        *reinterpret_cast<uint4*>(P + o * 16) = *reinterpret_cast<const uint4*>(W + src);
    }
}

template <bool F32, bool PACKED, int WAVES, int TBW, int NBLK>
hipError_t launch_tiling(const RouterArgs& a, int NS, hipStream_t stream) {
    using C = Cfg<F32, WAVES, TBW, NBLK>;
    const int64_t tiles = (a.T + C::BT - 1) / C::BT;
    const int64_t blocks = tiles * NS;
    hipLaunchKernelGGL((router_score_select_kernel<F32, PACKED, WAVES, TBW, NBLK>), dim3((unsigned)blocks),
                       dim3(C::NT), 0, stream, a, NS);
    return hipGetLastError();
}

template <bool PACKED>
hipError_t launch_layout(const RouterTiling& t, const RouterArgs& a, int NS, hipStream_t stream) {
    switch (t.id) {
        case 1: return launch_tiling<false, PACKED, 4, 4, 3>(a, NS, stream);
        case 2: return launch_tiling<false, PACKED, 8, 2, 3>(a, NS, stream);
        case 3: return launch_tiling<false, PACKED, 4, 4, 2>(a, NS, stream);
        case 4: return launch_tiling<false, PACKED, 4, 4, 1>(a, NS, stream);
        case 5: return launch_tiling<true, PACKED, 4, 4, 1>(a, NS, stream);
        default: return hipErrorInvalidValue;
    }
}

const RouterTiling kTilings[] = {
    {1, 0, 4, 4, 3},  // bf16: 128 tokens x 384 experts per workgroup
    {2, 0, 8, 2, 3},  // bf16: 64 tokens x 768 experts per workgroup
    {3, 0, 4, 4, 2},  // bf16: 128 tokens x 256 experts
    {4, 0, 4, 4, 1},  // bf16: 128 tokens x 128 experts
    {5, 1, 4, 4, 1},  // fp32: 128 tokens x 128 experts
};

}  // namespace

int router_tiling_count() { return (int)(sizeof(kTilings) / sizeof(kTilings[0])); }
RouterTiling router_tiling(int i) { return kTilings[i]; }

hipError_t launch_router_score_select(const RouterTiling& t, const RouterArgs& a, hipStream_t stream) {
    const int NS = router_slices(t, a.E);
    return a.w_packed ? launch_layout<true>(t, a, NS, stream) : launch_layout<false>(t, a, NS, stream);
}

hipError_t launch_router_merge(const RouterTiling& t, const RouterArgs& a, hipStream_t stream) {
    const int NS = router_slices(t, a.E);
    if (NS <= 1) return hipSuccess;
    const int per_tok_bytes = NS * a.K * 12;
    int tpw = 49152 / per_tok_bytes;
    tpw = tpw > 256 ? 256 : tpw;
    tpw = tpw < 1 ? 1 : tpw;
    int64_t blocks = (a.T + tpw - 1) / tpw;
    if (blocks > 1024) blocks = 1024;
    const size_t lds = 4096 + (size_t)tpw * per_tok_bytes;
    hipLaunchKernelGGL(router_merge_kernel, dim3((unsigned)blocks), dim3(kMergeThreads), lds, stream, a, NS, tpw);
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
