// Bias-adjusted Top-K selection from given fp32 scores (Eq. pid-routing), gate
// weights from the unbiased scores (Sec. 2.2) and per-expert load counts
// (Eq. pid-error): the router step without the gate contraction, an HBM-bound
// pass over a materialised T x E score matrix.
//
// Two kernels:
//  * select_reg_kernel (K <= 10, E % 4 == 0, 16-byte aligned scores): 16 lanes
//    (one DPP row) per token, each holding every 16th float4 of the row in
//    registers.  The K-th largest of the 16 lane maxima is a lower bound tau of
//    the token's K-th largest biased score; only the float4 chunks whose
//    maximum reaches tau are read again, and their values >= tau go to a short
//    LDS list whose entries are ranked by counting.  A token whose list would
//    overflow takes K exact argmax rounds over its row instead.
//  * select_kernel (every other case): a workgroup of 512 threads walks tiles
//    of 32 tokens (grid-stride, one workgroup per CU: the score rows of a tile
//    take most of the LDS).  A tile's scores go from registers into the LDS
//    score rows of the selection epilogue (epilogue.h, one slice of BE >= E
//    experts, padding -inf); right after, the next tile's scores are loaded
//    into the same registers, so their HBM reads overlap the selection of the
//    current tile.
// Both flush their LDS histogram once per workgroup.
#include "common.h"
#include "epilogue.h"
#include "internal.h"

#include <utility>

#pragma clang fp contract(off)

namespace idb {

namespace {

constexpr int kSelThreads = 512;
constexpr int kSelTile = 32;  // tokens per tile
// LDS for a tile's score rows: 32 rows of 1028 floats at BE = 1024 (131.6 KB);
// the epilogue's other arrays fit in the remaining 29 KB of the 160 KB.
constexpr int kSelScoreLds = 160 * 1024 - 29 * 1024;

__global__ void fill_i32_kernel(int32_t* p, int32_t value, int64_t n) {
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
        p[i] = value;
}

// BE: the slice width (a multiple of 256 >= E); VEC: E % 4 == 0 and 16-byte
// aligned scores, so a tile row is read as float4 pieces.
template <int BE, bool VEC>
__global__ __launch_bounds__(kSelThreads) void select_kernel(RouterArgs a, const float* __restrict__ scores) {
    using EC = EpiCfg<kSelThreads, kSelTile, BE, 0, kSelScoreLds>;
    static_assert(EC::NPASS == 1, "one pass per tile");
    __shared__ __attribute__((aligned(16))) unsigned char smem[EC::LDS];
    constexpr int PIECES = kSelTile * BE / 4;      // float4 pieces of a tile
    constexpr int PER = PIECES / kSelThreads;      // per thread
    static_assert(PER * kSelThreads == PIECES, "tile pieces split evenly");
    const int tid = threadIdx.x;
    const int64_t T = a.T;
    const int E = a.E;

    float breg[EC::NBIAS];
    prefetch_bias<EC>(a, 0, breg);
    epi_begin<EC>(smem, breg);

    // piece p = tid + kSelThreads * i: tile row p / (BE/4), columns 4 (p % (BE/4)) + c
    float4 r[PER];
    auto load = [&](int64_t tile) {
#pragma unroll
        for (int i = 0; i < PER; ++i) {
            const int p = tid + kSelThreads * i;
            const int row = p / (BE / 4), c4 = 4 * (p % (BE / 4));
            const int64_t t = tile * kSelTile + row;
            float4 f = make_float4(-INFINITY, -INFINITY, -INFINITY, -INFINITY);
            if (t < T) {
                const float* src = scores + t * (int64_t)E + c4;
                if (VEC) {
                    if (c4 < E) f = *reinterpret_cast<const float4*>(src);
                } else {
                    if (c4 + 0 < E) f.x = src[0];
                    if (c4 + 1 < E) f.y = src[1];
                    if (c4 + 2 < E) f.z = src[2];
                    if (c4 + 3 < E) f.w = src[3];
                }
            }
            r[i] = f;
        }
    };
    const int64_t ntiles = (T + kSelTile - 1) / kSelTile;
    int64_t tile = blockIdx.x;
    if (tile < ntiles) load(tile);
    for (; tile < ntiles; tile += gridDim.x) {
        const int64_t next = tile + gridDim.x;
        auto store_pass = [&](int, float* sc) {
#pragma unroll
            for (int i = 0; i < PER; ++i) {
                const int p = tid + kSelThreads * i;
                const int row = p / (BE / 4), c4 = 4 * (p % (BE / 4));
                *reinterpret_cast<float4*>(sc + row * EC::RS + c4) = r[i];
            }
            if (next < ntiles) load(next);
        };
        epi_tile<EC, false>(a, 1, 0, tile * kSelTile, smem, store_pass);
    }
    flush_hist(reinterpret_cast<const int*>(smem + EC::OFF_HIST), a.counts, E);
}

template <int BE>
hipError_t launch_select_be(const RouterArgs& a, const float* scores, hipStream_t stream) {
    const int64_t ntiles = (a.T + kSelTile - 1) / kSelTile;
    int cus = 0;
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus < 1)
        cus = 256;
    const int grid = (int)(ntiles < cus ? ntiles : cus);
    const bool vec = (a.E % 4 == 0) && ((reinterpret_cast<uintptr_t>(scores) & 15) == 0);
    if (vec)
        hipLaunchKernelGGL((select_kernel<BE, true>), dim3(grid), dim3(kSelThreads), 0, stream, a, scores);
    else
        hipLaunchKernelGGL((select_kernel<BE, false>), dim3(grid), dim3(kSelThreads), 0, stream, a, scores);
    return hipGetLastError();
}


// ---------------------------------------------------------------------------
// Register-resident selection.
constexpr int kRegMaxK = 10;   // largest K of this kernel
constexpr int kRegCap = 64;    // candidate list entries per token
constexpr int kRegStage = 4;   // marked chunks per lane staged in LDS

// DPP rotation by R lanes inside each 16-lane row.
template <int R>
__device__ __forceinline__ unsigned row_ror(unsigned x) {
    return (unsigned)__builtin_amdgcn_update_dpp(0, (int)x, 0x120 + R, 0xF, 0xF, false);
}
template <int R>
__device__ __forceinline__ float row_rorf(float x) {
    return __uint_as_float(row_ror<R>(__float_as_uint(x)));
}

// Number of lanes of the row whose value is strictly greater than this lane's.
template <int... R>
__device__ __forceinline__ int row_count_greater(float m, std::integer_sequence<int, R...>) {
    return ((row_rorf<R + 1>(m) > m ? 1 : 0) + ...);
}

__device__ __forceinline__ float row_min(float x) {
    x = fminf(x, row_rorf<8>(x));
    x = fminf(x, row_rorf<4>(x));
    x = fminf(x, row_rorf<2>(x));
    return fminf(x, row_rorf<1>(x));
}

// Row-wide maximum of a 64-bit rank key; every lane of the row gets it.
template <int R>
__device__ __forceinline__ void row_max_key_step(unsigned long long& k) {
    const unsigned lo = row_ror<R>((unsigned)k), hi = row_ror<R>((unsigned)(k >> 32));
    const unsigned long long o = ((unsigned long long)hi << 32) | lo;
    k = o > k ? o : k;
}
__device__ __forceinline__ unsigned long long row_max_key(unsigned long long k) {
    row_max_key_step<8>(k);
    row_max_key_step<4>(k);
    row_max_key_step<2>(k);
    row_max_key_step<1>(k);
    return k;
}

__device__ __forceinline__ float f4_at(const float4& v, int q) {
    return q == 0 ? v.x : q == 1 ? v.y : q == 2 ? v.z : v.w;
}

// Heavy ties (a candidate list that would overflow): K rounds over the row's
// biased scores by the token's 16 lanes (one DPP row, all active).  Round r
// takes the largest rank key strictly below the previous round's pick.  Rank
// keys order (v descending, index ascending) with -0 == +0, and every real
// column's key is above the key 0 a round starts from -- -inf included, so a
// row with fewer than K finite biased scores still picks its -inf columns by
// lowest index.  Each round reads the row again, one float4 at a time (from
// L2), so that this rare path adds few registers to the main path's.
template <int NV>
__device__ __forceinline__ void overflow_select(const float* row, const float* bias_s, unsigned vmask, int j, int K,
                                                int* sel_i, float* sel_s) {
    unsigned long long prev = ~0ull;
    int mine = 0;
    for (int r = 0; r < K; ++r) {
        unsigned long long best = 0ull;
#pragma unroll 1
        for (int c = 0; c < NV; ++c) {
            if ((vmask >> c) & 1u) {
                const int col0 = 4 * (16 * c + j);
                const float4 s4 = *reinterpret_cast<const float4*>(row + col0);
                const float4 b4 = *reinterpret_cast<const float4*>(bias_s + col0);
                const float4 v4 = make_float4(s4.x + b4.x, s4.y + b4.y, s4.z + b4.z, s4.w + b4.w);
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const unsigned long long kk = rank_key(f4_at(v4, q), col0 + q);
                    if (kk < prev && kk > best) best = kk;
                }
            }
        }
        best = row_max_key(best);
        prev = best;
        if (j == r) mine = (int)~(unsigned)best;
    }
    if (j < K) {
        sel_i[j] = mine;
        sel_s[j] = row[mine];
    }
}

// NV: float4 chunks per lane (64 NV >= E).  Lane j of a token's row owns the
// columns 4 (16 c + j) .. +3 for c < NV.
template <int NV, int WAVES>
__global__ __launch_bounds__(64 * WAVES) void select_reg_kernel(RouterArgs a, const float* __restrict__ scores) {
    constexpr int BE = 64 * NV;
    constexpr int TPB = 4 * WAVES;  // tokens per workgroup tile (4 per wave)
    __shared__ __attribute__((aligned(16))) float bias_s[BE];
    __shared__ int hist[BE];
    __shared__ int cnt[TPB];
    __shared__ unsigned long long lkey[TPB][kRegCap];
    __shared__ float lsc[TPB][kRegCap];
    __shared__ int sel_i[TPB][kRegMaxK];
    __shared__ float sel_s[TPB][kRegMaxK];
    // each lane's first kRegStage marked chunks, copied from its registers
    // (slot-major, so a wave's copies are consecutive 16-byte units)
    __shared__ float4 staged[kRegStage][64 * WAVES];

    const int tid = threadIdx.x;
    const int E = a.E, K = a.K;
    const int64_t T = a.T;
    for (int i = tid; i < BE; i += blockDim.x) {
        bias_s[i] = i < E ? a.bias[i] : 0.0f;
        hist[i] = 0;
    }
    __syncthreads();

    const int lane = tid & 63;
    const int j = lane & 15;
    const int slot = (tid >> 6) * 4 + (lane >> 4);  // token of the tile
    unsigned vmask = 0;                              // chunks holding real columns
#pragma unroll
    for (int c = 0; c < NV; ++c) vmask |= (4 * (16 * c + j) < E ? 1u : 0u) << c;

    const int64_t ntiles = (T + TPB - 1) / TPB;
    for (int64_t tile = blockIdx.x; tile < ntiles; tile += gridDim.x) {
        const int64_t t = tile * TPB + slot;
        const bool valid = t < T;  // uniform over the row
        const float* row = scores + (valid ? t : 0) * (int64_t)E;

        float4 sv[NV];
        // a tile of real tokens whose rows fill all 64 NV columns loads
        // without per-chunk conditions (uniform over the workgroup)
        if (64 * NV == E && (tile + 1) * TPB <= T) {
#pragma unroll
            for (int c = 0; c < NV; ++c) sv[c] = *reinterpret_cast<const float4*>(row + 4 * (16 * c + j));
        } else {
#pragma unroll
            for (int c = 0; c < NV; ++c) {
                sv[c] = make_float4(-INFINITY, -INFINITY, -INFINITY, -INFINITY);
                if (valid && ((vmask >> c) & 1u)) sv[c] = *reinterpret_cast<const float4*>(row + 4 * (16 * c + j));
            }
        }
        // chunk and lane maxima of v = s + b
        float cm[NV];
        float m = -INFINITY;
#pragma unroll
        for (int c = 0; c < NV; ++c) {
            const float4 b4 = *reinterpret_cast<const float4*>(bias_s + 4 * (16 * c + j));
            const float v0 = sv[c].x + b4.x, v1 = sv[c].y + b4.y, v2 = sv[c].z + b4.z, v3 = sv[c].w + b4.w;
            cm[c] = fmaxf(fmaxf(v0, v1), fmaxf(v2, v3));
            m = fmaxf(m, cm[c]);
        }
        // tau = the K-th largest lane maximum: K distinct elements reach it, so
        // every element of the top-K does.  Padding lanes (-inf) make tau -inf
        // when fewer than K lanes hold real columns.
        const int gt = row_count_greater(m, std::make_integer_sequence<int, 15>{});
        const float tau = row_min(gt < K ? m : INFINITY);

        unsigned cmask = 0;
#pragma unroll
        for (int c = 0; c < NV; ++c) cmask |= (cm[c] >= tau ? 1u : 0u) << c;
        cmask &= valid ? vmask : 0u;

        if (j == 0) cnt[slot] = 0;
        // the first kRegStage marked chunks go from registers to LDS, in
        // ascending chunk order (the order the loop below takes them)
        {
            int k = 0;
#pragma unroll
            for (int c = 0; c < NV; ++c) {
                if ((cmask >> c) & 1u) {
                    if (k < kRegStage) staged[k][tid] = sv[c];
                    ++k;
                }
            }
        }
        wave_sync();
        // candidates: the values >= tau of the marked chunks, appended to the
        // token's list (list order is irrelevant: ranks are counted below);
        // a lane's chunks past the staged ones are read again from memory
        int taken = 0;
        while (__ballot(cmask != 0u) != 0) {
            if (cmask != 0u) {
                const int c = __ffs(cmask) - 1;
                cmask &= cmask - 1u;
                const int col0 = 4 * (16 * c + j);
                const float4 s4 = taken < kRegStage ? staged[taken][tid]
                                                    : *reinterpret_cast<const float4*>(row + col0);
                ++taken;
                const float4 b4 = *reinterpret_cast<const float4*>(bias_s + col0);
                const float4 v4 = make_float4(s4.x + b4.x, s4.y + b4.y, s4.z + b4.z, s4.w + b4.w);
                const int n4 = (v4.x >= tau) + (v4.y >= tau) + (v4.z >= tau) + (v4.w >= tau);
                int p = atomicAdd(&cnt[slot], n4);
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    if (f4_at(v4, q) >= tau) {
                        if (p < kRegCap) {
                            lkey[slot][p] = rank_key(f4_at(v4, q), col0 + q);
                            lsc[slot][p] = f4_at(s4, q);
                        }
                        ++p;
                    }
                }
            }
        }
        wave_sync();

        const int n = cnt[slot];
        const bool over = n > kRegCap;  // uniform over the row
        const int nl = over ? 0 : n;
        int nmax = __builtin_amdgcn_readlane(nl, 0);
        nmax = max(nmax, __builtin_amdgcn_readlane(nl, 16));
        nmax = max(nmax, __builtin_amdgcn_readlane(nl, 32));
        nmax = max(nmax, __builtin_amdgcn_readlane(nl, 48));
        // rank of each listed candidate = the number of list keys above it;
        // the lanes take the entries in groups of 16
        for (int base = 0; base < nmax; base += 16) {
            const int me = base + j;
            const unsigned long long km = me < nl ? lkey[slot][me] : 0ull;
            int rk = 0;
            int e = 0;
            for (; e + 4 <= nmax; e += 4) {
                const unsigned long long q0 = lkey[slot][e], q1 = lkey[slot][e + 1];
                const unsigned long long q2 = lkey[slot][e + 2], q3 = lkey[slot][e + 3];
                rk += (e < nl && q0 > km) ? 1 : 0;
                rk += (e + 1 < nl && q1 > km) ? 1 : 0;
                rk += (e + 2 < nl && q2 > km) ? 1 : 0;
                rk += (e + 3 < nl && q3 > km) ? 1 : 0;
            }
            for (; e < nmax; ++e) rk += (e < nl && lkey[slot][e] > km) ? 1 : 0;
            if (me < nl && rk < K) {
                sel_i[slot][rk] = (int)~(unsigned)km;
                sel_s[slot][rk] = lsc[slot][me];
            }
        }

        if (over) {
            overflow_select<NV>(row, bias_s, vmask, j, K, &sel_i[slot][0], &sel_s[slot][0]);
        }
        wave_sync();

        if (valid && j < K) {
            const int idx = sel_i[slot][j];
            const float w = gate_weight(&sel_s[slot][0], K, j);
            a.idx[t * K + j] = idx;
            a.w[t * K + j] = w;
            atomicAdd(&hist[idx], 1);
        }
        wave_sync();
    }
    __syncthreads();
    flush_hist(hist, a.counts, E);
}

// Workgroup shape: waves per workgroup and resident workgroups per CU.  Every
// workgroup flushes its histogram with one device atomic per non-zero bin, so
// fewer, larger workgroups issue fewer atomics.
constexpr int kRegWaves = 16;
constexpr int kRegWgPerCu = 1;

template <int NV>
hipError_t launch_select_reg(const RouterArgs& a, const float* scores, hipStream_t stream) {
    constexpr int TPB = 4 * kRegWaves;
    const int64_t ntiles = (a.T + TPB - 1) / TPB;
    int cus = 0;
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus < 1)
        cus = 256;
    // one round of workgroups over the CUs; more tiles are walked grid-stride
    const int64_t cap = (int64_t)cus * kRegWgPerCu;
    const int grid = (int)(ntiles < cap ? ntiles : cap);
    hipLaunchKernelGGL((select_reg_kernel<NV, kRegWaves>), dim3(grid), dim3(64 * kRegWaves), 0, stream, a, scores);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_fill_i32(int32_t* p, int32_t value, int64_t n, hipStream_t stream) {
    int64_t blocks = (n + 255) / 256;
    if (blocks > 1024) blocks = 1024;
    if (blocks < 1) blocks = 1;
    hipLaunchKernelGGL(fill_i32_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, p, value, n);
    return hipGetLastError();
}

hipError_t launch_select_from_scores(const float* scores, const float* bias, int64_t T, int E, int K, int32_t* idx,
                                     float* w, int32_t* counts, hipStream_t stream) {
    RouterArgs a{};
    a.bias = bias;
    a.T = T;
    a.E = E;
    a.K = K;
    a.idx = idx;
    a.w = w;
    a.counts = counts;
    if (K <= kRegMaxK && E % 4 == 0 && (reinterpret_cast<uintptr_t>(scores) & 15) == 0) {
        if (E <= 256) return launch_select_reg<4>(a, scores, stream);
        if (E <= 512) return launch_select_reg<8>(a, scores, stream);
        if (E <= 768) return launch_select_reg<12>(a, scores, stream);
        return launch_select_reg<16>(a, scores, stream);
    }
    if (E <= 256) return launch_select_be<256>(a, scores, stream);
    if (E <= 512) return launch_select_be<512>(a, scores, stream);
    if (E <= 768) return launch_select_be<768>(a, scores, stream);
    return launch_select_be<1024>(a, scores, stream);
}

}  // namespace idb
