// Fused router step for gfx950: gate contraction z = W_r x on MFMA (Sec. 2.2),
// sigmoid scores, bias-adjusted Top-K (Eq. pid-routing), gate weights from the
// unbiased scores and per-expert load counts (Eq. pid-error).  The T x E score
// matrix stays in registers and LDS.
//
// Tiling.  A workgroup owns BT = 32*TBW tokens and one slice of BE =
// WAVES*32*NBLK experts.  Each wave owns all BT tokens and its own 32*NBLK
// experts, so the router rows it multiplies are private to it and come
// straight from global memory into MFMA A-operand registers, while the token
// tile is shared by the waves through a double-buffered LDS stage.  The
// contraction runs over 128-byte chunks of each row; within a chunk, lane half
// h of every 32-lane group consumes bytes [64h, 64h + 64) in four 16-byte
// units, for both operands, so the k order is consistent between them.
//
// MFMA 32x32 output layout (C = W_block * x_block^T): lane l holds token
// (l % 32) of the block and experts 8*(r/4) + 4*(l/32) + (r%4), r < 16.  So a
// token's BE scores are spread over 2*WAVES lanes, 16*NBLK per lane.
//
// Epilogue per token and slice (exact for any input):
//   1. s = sigmoid(z), v = fl32(s + b).
//   2. Each lane splits its values into G groups (16 group maxima per token);
//      tau = the K-th largest group maximum <= the token's K-th largest v.
//   3. Values >= tau go to an LDS candidate list (about K + 5 of them).
//   4. Candidate rank = number of candidates above it in the order (v desc,
//      index asc); ranks < K form the slice's selection in rank order.
//   5. Overflowing lists (ties, K > 16) fall back to K rounds of "best value
//      strictly below the previous pick" over all the token's lanes.
//   6. One slice: gate weights, outputs and an LDS histogram flushed with one
//      atomic per non-zero bin.  Several slices: the slice's K candidates go
//      to the workspace and router_merge_kernel combines them.
#include "common.h"
#include "internal.h"

#pragma clang fp contract(off)

namespace idb {

namespace {

constexpr int kCap = 32;      // candidate list capacity per token and slice
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
    static constexpr int PPT = BT * 8 / NT;  // 16-byte x pieces per thread per chunk
    static constexpr int STAGE = BT * kRowPad;
    static constexpr int MAIN_LDS = 2 * STAGE;
    static constexpr int NLANES = 2 * WAVES;  // lanes holding one token's slice
    // epilogue LDS layout (bytes)
    static constexpr int OFF_GM = 0;
    static constexpr int OFF_TAU = OFF_GM + BT * 16 * 4;
    static constexpr int OFF_CNT = OFF_TAU + BT * 4;
    static constexpr int OFF_PV = OFF_CNT + BT * 4;
    static constexpr int OFF_PI = OFF_PV + BT * 4;
    static constexpr int OFF_LV = OFF_PI + BT * 4;
    static constexpr int OFF_LS = OFF_LV + BT * kCap * 4;
    static constexpr int OFF_LI = OFF_LS + BT * kCap * 4;
    static constexpr int OFF_SV = OFF_LI + BT * kCap * 4;
    static constexpr int OFF_SS = OFF_SV + BT * kMaxK * 4;
    static constexpr int OFF_SI = OFF_SS + BT * kMaxK * 4;
    static constexpr int OFF_RV = OFF_SI + BT * kMaxK * 4;
    static constexpr int OFF_RS = OFF_RV + BT * NLANES * 4;
    static constexpr int OFF_RI = OFF_RS + BT * NLANES * 4;
    static constexpr int OFF_HIST = OFF_RI + BT * NLANES * 4;
    static constexpr int OFF_FLAG = OFF_HIST + 1024 * 4;
    static constexpr int OFF_BIAS = OFF_FLAG + 16;
    static constexpr int EPI_LDS = OFF_BIAS + BE * 4;
    static constexpr int LDS = MAIN_LDS > EPI_LDS ? MAIN_LDS : EPI_LDS;
    static_assert(BT <= NT, "one thread per token in the threshold step");
    static_assert(NV % G == 0, "groups must split a lane's values evenly");
    static_assert(PPT * NT == BT * 8, "x pieces must split evenly");
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

template <bool F32, int WAVES, int TBW, int NBLK>
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
    // slices of one token tile then share their x rows in that XCD's L2.
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
    const char* wrow[NBLK];
#pragma unroll
    for (int nbk = 0; nbk < NBLK; ++nbk) {
        int e = e_wave0 + nbk * 32 + l32;
        e = e < E ? e : E - 1;  // rows past E are loaded from a valid row and masked later
        wrow[nbk] = reinterpret_cast<const char*>(a.W) + (int64_t)e * RB + 64 * h;
    }
    const char* xsrc[C::PPT];
    int xdst[C::PPT];
    bool xok[C::PPT];
#pragma unroll
    for (int q = 0; q < C::PPT; ++q) {
        const int p = tid + C::NT * q;
        const int row = p >> 3, c16 = p & 7;
        const int64_t tok = tok0 + row;
        xok[q] = tok < T;
        xsrc[q] = reinterpret_cast<const char*>(a.x) + (xok[q] ? tok : 0) * RB + c16 * 16;
        xdst[q] = row * kRowPad + c16 * 16;
    }

    floatx16 acc[TBW][NBLK];
#pragma unroll
    for (int tb = 0; tb < TBW; ++tb)
#pragma unroll
        for (int nbk = 0; nbk < NBLK; ++nbk)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[tb][nbk][r] = 0.0f;

    // W operands: one register set, refilled unit by unit.  Right after the
    // MFMAs of unit u of chunk c are issued, the same registers start loading
    // unit u of chunk c+1, which gives each load a whole chunk of MFMA work to
    // arrive.
    uint4 w[NBLK][4], xr[C::PPT];

    auto load_x = [&](int c) {
#pragma unroll
        for (int q = 0; q < C::PPT; ++q) xr[q] = xok[q] ? ld16(xsrc[q] + c * 128) : make_uint4(0, 0, 0, 0);
    };
    auto store_x = [&](int stage) {
#pragma unroll
        for (int q = 0; q < C::PPT; ++q)
            *reinterpret_cast<uint4*>(smem + stage * C::STAGE + xdst[q]) = xr[q];
    };

    load_x(0);
#pragma unroll
    for (int nbk = 0; nbk < NBLK; ++nbk)
#pragma unroll
        for (int u = 0; u < 4; ++u) w[nbk][u] = ld16(wrow[nbk] + 16 * u);
    store_x(0);
    __syncthreads();
    for (int c = 0; c < NCH; ++c) {
        const bool more = c + 1 < NCH;
        if (more) load_x(c + 1);
        const unsigned char* st = smem + (c & 1) * C::STAGE + l32 * kRowPad + 64 * h;
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
                for (int nbk = 0; nbk < NBLK; ++nbk) w[nbk][u] = ld16(wrow[nbk] + (c + 1) * 128 + 16 * u);
            }
        }
        if (more) store_x((c + 1) & 1);
        __syncthreads();
    }

    // ---------------------------------------------------------------- epilogue
    float* gm = reinterpret_cast<float*>(smem + C::OFF_GM);
    float* tau_s = reinterpret_cast<float*>(smem + C::OFF_TAU);
    int* cnt = reinterpret_cast<int*>(smem + C::OFF_CNT);
    float* pvs = reinterpret_cast<float*>(smem + C::OFF_PV);
    int* pis = reinterpret_cast<int*>(smem + C::OFF_PI);
    float* lv = reinterpret_cast<float*>(smem + C::OFF_LV);
    float* ls = reinterpret_cast<float*>(smem + C::OFF_LS);
    int* li = reinterpret_cast<int*>(smem + C::OFF_LI);
    float* sv = reinterpret_cast<float*>(smem + C::OFF_SV);
    float* ss = reinterpret_cast<float*>(smem + C::OFF_SS);
    int* si = reinterpret_cast<int*>(smem + C::OFF_SI);
    float* rv = reinterpret_cast<float*>(smem + C::OFF_RV);
    float* rs = reinterpret_cast<float*>(smem + C::OFF_RS);
    int* ri = reinterpret_cast<int*>(smem + C::OFF_RI);
    int* hist = reinterpret_cast<int*>(smem + C::OFF_HIST);
    int* flag = reinterpret_cast<int*>(smem + C::OFF_FLAG);
    float* bias_s = reinterpret_cast<float*>(smem + C::OFF_BIAS);

    // Expert of accumulator (nbk, r): ebase + 32 nbk + 8 (r/4) + (r%4).  E is a
    // multiple of 32, so a whole 32-expert block is either real or padding.
    const int ebase = e_wave0 + 4 * h;
    auto blk_real = [&](int nbk) { return e_wave0 + nbk * 32 < E; };
    // The slice's bias, staged once; lane reads 4 consecutive experts at a time.
    for (int j = tid; j < C::BE; j += C::NT) {
        const int e = slice * C::BE + j;
        bias_s[j] = e < E ? a.bias[e] : 0.0f;
    }
    for (int e = tid; e < 1024; e += C::NT) hist[e] = 0;
    if (tid == 0) flag[0] = 0;
    auto bias4 = [&](int nbk, int r4) {
        return *reinterpret_cast<const float4*>(bias_s + wave * C::WE + nbk * 32 + 8 * r4 + 4 * h);
    };
    auto comp = [](const float4& f, int i) { return i == 0 ? f.x : (i == 1 ? f.y : (i == 2 ? f.z : f.w)); };

    // 1. scores s = sigmoid(z).  The accumulators keep z; every step below
    // recomputes s from it with the same instructions, so the values the
    // selection compares and the optional debug dump are identical.
    auto score = [&](int tb, int nbk, int r) { return sigmoid_fast(acc[tb][nbk][r]); };
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
                                make_float4(score(tb, nbk, 4 * r4), score(tb, nbk, 4 * r4 + 1),
                                            score(tb, nbk, 4 * r4 + 2), score(tb, nbk, 4 * r4 + 3));
                    }
            }
        }
    }
    __syncthreads();

    // 2. group maxima of v = s + b
    {
        float gmx[TBW][C::G];
#pragma unroll
        for (int tb = 0; tb < TBW; ++tb)
#pragma unroll
            for (int g = 0; g < C::G; ++g) gmx[tb][g] = -INFINITY;
#pragma unroll
        for (int nbk = 0; nbk < NBLK; ++nbk) {
            if (!blk_real(nbk)) continue;
            float4 b4[4];
#pragma unroll
            for (int r4 = 0; r4 < 4; ++r4) b4[r4] = bias4(nbk, r4);
#pragma unroll
            for (int tb = 0; tb < TBW; ++tb)
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const int g = (nbk * 16 + r) / C::GS;
                    gmx[tb][g] = fmaxf(gmx[tb][g], score(tb, nbk, r) + comp(b4[r >> 2], r & 3));
                }
        }
#pragma unroll
        for (int tb = 0; tb < TBW; ++tb)
#pragma unroll
            for (int g = 0; g < C::G; ++g) gm[(tb * 32 + l32) * 16 + (wave * 2 + h) * C::G + g] = gmx[tb][g];
    }
    __syncthreads();

    // 3. per-token threshold
    if (tid < C::BT) {
        float g16[16];
#pragma unroll
        for (int i = 0; i < 16; ++i) g16[i] = gm[tid * 16 + i];
        sort16_ascending(g16);
        float tau = -INFINITY;
        if (K <= 16) {
#pragma unroll
            for (int i = 0; i < 16; ++i)
                if (i == 16 - K) tau = g16[i];
        }
        tau_s[tid] = tau;
        cnt[tid] = 0;
    }
    __syncthreads();

    // 4. candidates v >= tau
    {
        float taus[TBW];
        bool live[TBW];
#pragma unroll
        for (int tb = 0; tb < TBW; ++tb) {
            taus[tb] = tau_s[tb * 32 + l32];
            live[tb] = tok0 + tb * 32 + l32 < T;
        }
#pragma unroll
        for (int nbk = 0; nbk < NBLK; ++nbk) {
            if (!blk_real(nbk)) continue;
            float4 b4[4];
#pragma unroll
            for (int r4 = 0; r4 < 4; ++r4) b4[r4] = bias4(nbk, r4);
#pragma unroll
            for (int tb = 0; tb < TBW; ++tb) {
                const int tl = tb * 32 + l32;
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const float s = score(tb, nbk, r);
                    const float v = s + comp(b4[r >> 2], r & 3);
                    if (live[tb] && v >= taus[tb]) {
                        const int p = atomicAdd(&cnt[tl], 1);
                        if (p < kCap) {
                            lv[tl * kCap + p] = v;
                            ls[tl * kCap + p] = s;
                            li[tl * kCap + p] = ebase + nbk * 32 + 8 * (r >> 2) + (r & 3);
                        }
                    }
                }
            }
        }
    }
    __syncthreads();

    // 5. rank the candidates of every token whose list did not overflow
    {
        const int tl = tid / C::TPT, q = tid % C::TPT;
        const int n = cnt[tl];
        if (n > kCap) {
            flag[0] = 1;
        } else {
            for (int c = q; c < n; c += C::TPT) {
                const float vc = lv[tl * kCap + c];
                const int ic = li[tl * kCap + c];
                int rank = 0;
                for (int o = 0; o < n; ++o) rank += ranks_above(lv[tl * kCap + o], li[tl * kCap + o], vc, ic) ? 1 : 0;
                if (rank < K) {
                    sv[tl * kMaxK + rank] = vc;
                    ss[tl * kMaxK + rank] = ls[tl * kCap + c];
                    si[tl * kMaxK + rank] = ic;
                }
            }
        }
    }
    __syncthreads();

    // 6. exact fallback for overflowing tokens: K rounds of "best value
    // strictly below the previous pick", reduced over the token's lanes.
    if (flag[0]) {
        if (tid < C::BT) {
            pvs[tid] = INFINITY;
            pis[tid] = -1;
        }
        __syncthreads();
        for (int r = 0; r < K; ++r) {
#pragma unroll
            for (int tb = 0; tb < TBW; ++tb) {
                const int tl = tb * 32 + l32;
                if (cnt[tl] > kCap) {
                    const float pv = pvs[tl];
                    const int pi = pis[tl];
                    float bv = -INFINITY, bs = 0.0f;
                    int bi = 0x7fffffff;
#pragma unroll
                    for (int nbk = 0; nbk < NBLK; ++nbk) {
                        if (!blk_real(nbk)) continue;
#pragma unroll
                        for (int rr = 0; rr < 16; ++rr) {
                            const float s = score(tb, nbk, rr);
                            const float v = s + bias_s[wave * C::WE + nbk * 32 + 8 * (rr >> 2) + 4 * h + (rr & 3)];
                            const int e = ebase + nbk * 32 + 8 * (rr >> 2) + (rr & 3);
                            const bool below = (pi < 0) || ranks_above(pv, pi, v, e);
                            if (below && ranks_above(v, e, bv, bi)) {
                                bv = v;
                                bs = s;
                                bi = e;
                            }
                        }
                    }
                    const int o = tl * C::NLANES + wave * 2 + h;
                    rv[o] = bv;
                    rs[o] = bs;
                    ri[o] = bi;
                }
            }
            __syncthreads();
            if (tid < C::BT && cnt[tid] > kCap) {
                float bv = -INFINITY, bs = 0.0f;
                int bi = 0x7fffffff;
                for (int o = 0; o < C::NLANES; ++o) {
                    const int k = tid * C::NLANES + o;
                    if (ranks_above(rv[k], ri[k], bv, bi)) {
                        bv = rv[k];
                        bs = rs[k];
                        bi = ri[k];
                    }
                }
                sv[tid * kMaxK + r] = bv;
                ss[tid * kMaxK + r] = bs;
                si[tid * kMaxK + r] = bi;
                pvs[tid] = bv;
                pis[tid] = bi;
            }
            __syncthreads();
        }
    }

    // 7. outputs
    {
        const int tl = tid / C::TPT, q = tid % C::TPT;
        const int64_t tok = tok0 + tl;
        if (tok < T) {
            if (NS > 1) {
                const int64_t base = (tok * NS + slice) * K;
                for (int r = q; r < K; r += C::TPT) {
                    a.cand_v[base + r] = sv[tl * kMaxK + r];
                    a.cand_s[base + r] = ss[tl * kMaxK + r];
                    a.cand_i[base + r] = si[tl * kMaxK + r];
                }
            } else {
                for (int r = q; r < K; r += C::TPT) {
                    const int e = si[tl * kMaxK + r];
                    a.idx[tok * K + r] = e;
                    a.w[tok * K + r] = gate_weight(ss + tl * kMaxK, K, r);
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
// the gate weights and count the assignments.  One thread per token.
constexpr int kMergeThreads = 256;

__global__ __launch_bounds__(kMergeThreads) void router_merge_kernel(RouterArgs a, int NS) {
    __shared__ int hist[1024];
    const int tid = threadIdx.x;
    const int E = a.E, K = a.K;
    for (int e = tid; e < E; e += kMergeThreads) hist[e] = 0;
    __syncthreads();
    for (int64_t tok = (int64_t)blockIdx.x * kMergeThreads + tid; tok < a.T;
         tok += (int64_t)gridDim.x * kMergeThreads) {
        const int64_t base = tok * NS * K;
        int head[kMaxSlices];
#pragma unroll
        for (int s = 0; s < kMaxSlices; ++s) head[s] = 0;
        float sel_s[kMaxK];
#pragma unroll
        for (int r = 0; r < kMaxK; ++r) {
            if (r < K) {
                float bv = -INFINITY, bs = 0.0f;
                int bi = 0x7fffffff, bsl = 0;
#pragma unroll
                for (int s = 0; s < kMaxSlices; ++s) {
                    if (s < NS && head[s] < K) {
                        const int64_t o = base + (int64_t)s * K + head[s];
                        const float v = a.cand_v[o];
                        const int i = a.cand_i[o];
                        if (ranks_above(v, i, bv, bi)) {
                            bv = v;
                            bi = i;
                            bs = a.cand_s[o];
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
    __syncthreads();
    for (int e = tid; e < E; e += kMergeThreads)
        if (hist[e] != 0) atomicAdd(&a.counts[e], hist[e]);
}

template <bool F32, int WAVES, int TBW, int NBLK>
hipError_t launch_tiling(const RouterArgs& a, int NS, hipStream_t stream) {
    using C = Cfg<F32, WAVES, TBW, NBLK>;
    const int64_t tiles = (a.T + C::BT - 1) / C::BT;
    const int64_t blocks = tiles * NS;
    hipLaunchKernelGGL((router_score_select_kernel<F32, WAVES, TBW, NBLK>), dim3((unsigned)blocks), dim3(C::NT), 0,
                       stream, a, NS);
    return hipGetLastError();
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
    switch (t.id) {
        case 1: return launch_tiling<false, 4, 4, 3>(a, NS, stream);
        case 2: return launch_tiling<false, 8, 2, 3>(a, NS, stream);
        case 3: return launch_tiling<false, 4, 4, 2>(a, NS, stream);
        case 4: return launch_tiling<false, 4, 4, 1>(a, NS, stream);
        case 5: return launch_tiling<true, 4, 4, 1>(a, NS, stream);
        default: return hipErrorInvalidValue;
    }
}

hipError_t launch_router_merge(const RouterTiling& t, const RouterArgs& a, hipStream_t stream) {
    const int NS = router_slices(t, a.E);
    if (NS <= 1) return hipSuccess;
    int64_t blocks = (a.T + kMergeThreads - 1) / kMergeThreads;
    if (blocks > 64) blocks = 64;
    hipLaunchKernelGGL(router_merge_kernel, dim3((unsigned)blocks), dim3(kMergeThreads), 0, stream, a, NS);
    return hipGetLastError();
}

}  // namespace idb
