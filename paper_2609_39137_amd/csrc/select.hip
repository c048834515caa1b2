// Bias-adjusted Top-K selection from given fp32 scores (Eq. pid-routing), gate
// weights from the unbiased scores (Sec. 2.2) and per-expert load counts
// (Eq. pid-error).  This is the router step without the gate contraction: an
// HBM-bound pass over a materialised T x E score matrix.
//
// Layout: a 16-lane row of a wave owns one token.  Lane `sub` of the row holds
// experts 4*(sub + 16 j) + c (j < CH, c < 4), so each row reads its token's
// scores with coalesced 16-byte loads, and the lane keeps the bias of its
// experts in registers for every token it visits.
//
// Selection, exact for any input:
//   1. v = fl32(s + b); each lane takes the max of its values.
//   2. tau = K-th largest of the row's 16 lane maxima.  Those are 16 distinct
//      elements, so tau <= the token's K-th largest v and every selected
//      expert has v >= tau.
//   3. Experts with v >= tau are appended to an LDS candidate list (typically
//      about K + 5 of them).
//   4. Each candidate's rank = number of candidates above it in the strict
//      order (v desc, index asc); ranks < K are the selection, in rank order.
//   5. If the list overflowed (ties, or K > 16), the row instead takes K rounds
//      of "best expert strictly below the previous one" over all its values.
#include "common.h"
#include "internal.h"

#pragma clang fp contract(off)

namespace idb {

namespace {

constexpr int kRowTokensPerWave = 4;
constexpr int kSelThreads = 256;
constexpr int kTokensPerIter = kRowTokensPerWave * (kSelThreads / 64);  // 16
constexpr int kSelCap = 64;

__global__ void fill_i32_kernel(int32_t* p, int32_t value, int64_t n) {
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
        p[i] = value;
}

template <int CH, bool VEC>
__global__ __launch_bounds__(kSelThreads) void select_kernel(const float* __restrict__ scores,
                                                             const float* __restrict__ bias, int64_t T, int E, int K,
                                                             int32_t* __restrict__ idx_out,
                                                             float* __restrict__ w_out,
                                                             int32_t* __restrict__ counts) {
    constexpr int NV = 4 * CH;
    __shared__ float lv[kTokensPerIter][kSelCap];
    __shared__ float ls[kTokensPerIter][kSelCap];
    __shared__ int li[kTokensPerIter][kSelCap];
    __shared__ int lcnt[kTokensPerIter];
    __shared__ float sel_v[kTokensPerIter][kMaxK];
    __shared__ float sel_s[kTokensPerIter][kMaxK];
    __shared__ int sel_i[kTokensPerIter][kMaxK];
    __shared__ int hist[1024];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int sub = lane & 15;
    const int slot = (tid >> 6) * kRowTokensPerWave + (lane >> 4);

    int ex[NV];
    float bv[NV];
#pragma unroll
    for (int j = 0; j < NV; ++j) {
        ex[j] = 4 * (sub + 16 * (j / 4)) + (j % 4);
        bv[j] = (ex[j] < E) ? bias[ex[j]] : 0.0f;
    }
    for (int e = tid; e < E; e += kSelThreads) hist[e] = 0;

    for (int64_t base = (int64_t)blockIdx.x * kTokensPerIter; base < T;
         base += (int64_t)gridDim.x * kTokensPerIter) {
        const int64_t t = base + slot;
        const bool valid = t < T;
        float s[NV];
        const float* row = scores + (valid ? t : 0) * (int64_t)E;
        if (VEC) {
#pragma unroll
            for (int j = 0; j < CH; ++j) {
                const int q = sub + 16 * j;
                float4 f = make_float4(0.f, 0.f, 0.f, 0.f);
                if (valid && 4 * q < E) f = *reinterpret_cast<const float4*>(row + 4 * q);
                s[4 * j + 0] = f.x;
                s[4 * j + 1] = f.y;
                s[4 * j + 2] = f.z;
                s[4 * j + 3] = f.w;
            }
        } else {
#pragma unroll
            for (int j = 0; j < NV; ++j) s[j] = (valid && ex[j] < E) ? row[ex[j]] : 0.0f;
        }
        // 1. lane maximum of v = s + b over real experts
        float m = -INFINITY;
#pragma unroll
        for (int j = 0; j < NV; ++j)
            if (valid && ex[j] < E) m = fmaxf(m, s[j] + bv[j]);
        // 2. threshold from the row's 16 lane maxima
        float tau = row16_sorted_ascending_at(m, 16 - (K <= 16 ? K : 16));
        if (K > 16) tau = -INFINITY;
        if (sub == 0) lcnt[slot] = 0;
        __syncthreads();
        // 3. candidates v >= tau
        if (valid) {
#pragma unroll
            for (int j = 0; j < NV; ++j) {
                const float v = s[j] + bv[j];
                if (ex[j] < E && v >= tau) {
                    const int p = atomicAdd(&lcnt[slot], 1);
                    if (p < kSelCap) {
                        lv[slot][p] = v;
                        ls[slot][p] = s[j];
                        li[slot][p] = ex[j];
                    }
                }
            }
        }
        __syncthreads();
        const int C = lcnt[slot];
        if (valid && C <= kSelCap) {
            // 4. rank each candidate against the others
            for (int c = sub; c < C; c += 16) {
                const float vc = lv[slot][c];
                const int ic = li[slot][c];
                int rank = 0;
                for (int o = 0; o < C; ++o) rank += ranks_above(lv[slot][o], li[slot][o], vc, ic) ? 1 : 0;
                if (rank < K) {
                    sel_v[slot][rank] = vc;
                    sel_s[slot][rank] = ls[slot][c];
                    sel_i[slot][rank] = ic;
                }
            }
        } else if (valid) {
            // 5. overflow: K rounds of "best strictly below the previous pick"
            float pv = INFINITY;
            int pi = -1;
            for (int r = 0; r < K; ++r) {
                float bvv = -INFINITY, bs = 0.0f;
                int bi = 0x7fffffff;
#pragma unroll
                for (int j = 0; j < NV; ++j) {
                    const float v = s[j] + bv[j];
                    const bool below = (pi < 0) || ranks_above(pv, pi, v, ex[j]);
                    if (ex[j] < E && below && ranks_above(v, ex[j], bvv, bi)) {
                        bvv = v;
                        bs = s[j];
                        bi = ex[j];
                    }
                }
#pragma unroll
                for (int off = 8; off >= 1; off >>= 1) {
                    const float ov = __shfl_xor(bvv, off, 16);
                    const float os = __shfl_xor(bs, off, 16);
                    const int oi = __shfl_xor(bi, off, 16);
                    if (ranks_above(ov, oi, bvv, bi)) {
                        bvv = ov;
                        bs = os;
                        bi = oi;
                    }
                }
                if (sub == 0) {
                    sel_v[slot][r] = bvv;
                    sel_s[slot][r] = bs;
                    sel_i[slot][r] = bi;
                }
                pv = bvv;
                pi = bi;
            }
        }
        __syncthreads();
        if (valid) {
            for (int r = sub; r < K; r += 16) {
                const int e = sel_i[slot][r];
                idx_out[t * K + r] = e;
                w_out[t * K + r] = gate_weight(sel_s[slot], K, r);
                if ((unsigned)e < (unsigned)E) atomicAdd(&hist[e], 1);
            }
        }
        __syncthreads();
    }
    for (int e = tid; e < E; e += kSelThreads)
        if (hist[e] != 0) atomicAdd(&counts[e], hist[e]);
}

template <int CH>
hipError_t launch_select_ch(const float* scores, const float* bias, int64_t T, int E, int K, int32_t* idx, float* w,
                            int32_t* counts, hipStream_t stream) {
    const int64_t iters = (T + kTokensPerIter - 1) / kTokensPerIter;
    const int grid = (int)(iters < 512 ? iters : 512);
    const bool vec = (E % 4 == 0) && ((reinterpret_cast<uintptr_t>(scores) & 15) == 0);
    if (vec)
        hipLaunchKernelGGL((select_kernel<CH, true>), dim3(grid), dim3(kSelThreads), 0, stream, scores, bias, T, E,
                           K, idx, w, counts);
    else
        hipLaunchKernelGGL((select_kernel<CH, false>), dim3(grid), dim3(kSelThreads), 0, stream, scores, bias, T,
                           E, K, idx, w, counts);
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
    const int ch = (E + 63) / 64;  // float4 chunks per lane
    if (ch <= 1) return launch_select_ch<1>(scores, bias, T, E, K, idx, w, counts, stream);
    if (ch <= 2) return launch_select_ch<2>(scores, bias, T, E, K, idx, w, counts, stream);
    if (ch <= 4) return launch_select_ch<4>(scores, bias, T, E, K, idx, w, counts, stream);
    if (ch <= 8) return launch_select_ch<8>(scores, bias, T, E, K, idx, w, counts, stream);
    if (ch <= 12) return launch_select_ch<12>(scores, bias, T, E, K, idx, w, counts, stream);
    return launch_select_ch<16>(scores, bias, T, E, K, idx, w, counts, stream);
}

}  // namespace idb
