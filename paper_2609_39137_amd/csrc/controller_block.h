// The ID bias controller update (Algorithm 1, Eq. rapid-update), the load
// statistics (Eq. vio) and the update's diagnostics as device functions: run
// by one workgroup (the stand-alone controller kernel and the router tail
// that runs it after the last slice-merge workgroup), or by one wave
// (controller_wave: the batched kernel of many layers, one wave each).
#pragma once

#include "common.h"

namespace idb {

// LDS scratch of controller_block.
struct CtrlScratch {
    long long w_sum[16];
    int w_max[16], w_min[16], w_neg[16];
    float tree[1024];
};

// LDS scratch of the diagnostics (controller_block with a diag pointer).
struct DiagScratch {
    int wcnt[2][16];  // per-wave counts of the threshold search (two banks, alternating)
    double tree[1024];
};

// Sum of one value per thread over the workgroup (exact for integers).
__device__ inline long long block_sum(long long v, CtrlScratch& sh) {
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6, nw = blockDim.x >> 6;
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o);
    __syncthreads();  // w_sum is free
    if (lane == 0) sh.w_sum[wv] = v;
    __syncthreads();
    long long t = 0;
    for (int w = 0; w < nw; ++w) t += sh.w_sum[w];
    return t;
}

// Leaves of the centering tree: the next power of two >= E.
__host__ __device__ inline int ctrl_tree_size(int E) {
    int P = 1;
    while (P < E) P <<= 1;
    return P;
}

// The whole O(E) update on one workgroup whose size is a multiple of 64, each
// thread taking experts i, i + blockDim, ... (kPer of them): needs
// kPer * blockDim >= P, the centering tree's size below, and E <= 1024.  With a
// non-null stats pointer it also writes MaxVio/MinVio of the same counts;
// with a non-null diag pointer (and dsh), the update's diagnostics: diag[0]
// the active-gate fraction #{g_i = 1}/E, diag[1] the share of the assignments
// on the m = ceil(E/10) busiest experts (the sum of the m largest counts over
// S), diag[2] the inactive-expert ratio #{n_i = 0}/E, diag[3] the mean
// |b_new - b_old| summed in fp64 over the same pairwise tree; NaN x 4 when the
// update does not run.
// Reductions: exact integer sums/extrema across waves (order-free); the
// centering mean with the fixed pairwise tree (level h adds a_{j+h} into a_j
// for j < h, P = next power of two >= E), levels h >= 64 in LDS, the last
// six inside wave 0 by shuffles (same pairs, same order).
template <int kPer, bool kCoherentCounts = false>
__device__ inline void controller_block(const int32_t* __restrict__ counts, int E, int P, float Ki, float Kd,
                                        int sign_mode, int center, float* __restrict__ bias,
                                        float* __restrict__ e_prev, int64_t* __restrict__ step,
                                        int32_t* __restrict__ status, double* __restrict__ stats,
                                        CtrlScratch& sh, double* __restrict__ diag = nullptr,
                                        DiagScratch* dsh = nullptr) {
#pragma clang fp contract(off)
    const int i0 = threadIdx.x, nt = blockDim.x;
    const int lane = i0 & 63, wv = i0 >> 6, nw = nt >> 6;
    int n[kPer];
    float b0[kPer], ep0[kPer];  // state, loaded together with the counts
    long long sum = 0;
    int mx = INT32_MIN, mn = INT32_MAX, neg = 0;
#pragma unroll
    for (int q = 0; q < kPer; ++q) {
        const int i = i0 + q * nt;
        // counts written by atomics of other workgroups of the same launch
        // are read with agent-scope loads.
        n[q] = (i >= E) ? 0
               : kCoherentCounts ? __hip_atomic_load(counts + i, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)
                                 : counts[i];
        b0[q] = (i < E) ? bias[i] : 0.0f;
        ep0[q] = (i < E) ? e_prev[i] : 0.0f;
        if (i < E) {
            sum += n[q];
            mx = max(mx, n[q]);
            mn = min(mn, n[q]);
            neg |= n[q] < 0 ? 1 : 0;
        }
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) {
        sum += __shfl_xor(sum, o);
        mx = max(mx, __shfl_xor(mx, o));
        mn = min(mn, __shfl_xor(mn, o));
        neg |= __shfl_xor(neg, o);
    }
    if (lane == 0) {
        sh.w_sum[wv] = sum;
        sh.w_max[wv] = mx;
        sh.w_min[wv] = mn;
        sh.w_neg[wv] = neg;
    }
    __syncthreads();
    // Total assignments S = E * nbar (Eq. pid-error).
    long long S = 0;
    int any_negative = 0;
    mx = INT32_MIN;
    mn = INT32_MAX;
    for (int w = 0; w < nw; ++w) {
        S += sh.w_sum[w];
        mx = max(mx, sh.w_max[w]);
        mn = min(mn, sh.w_min[w]);
        any_negative |= sh.w_neg[w];
    }
    if (stats && i0 == nt - 1) {
        // MaxVio, MinVio (Eq. vio): one fp64 division of an exact integer
        // numerator each; NaN for an empty batch.  (The last wave: wave 0
        // has the centering tree's serial part.)
        if (S == 0) {
            stats[0] = __builtin_nan("");
            stats[1] = __builtin_nan("");
        } else {
            stats[0] = (double)((long long)E * mx - S) / (double)S;
            stats[1] = (double)(S - (long long)E * mn) / (double)S;
        }
    }
    if (any_negative || S == 0) {
        // Invalid or empty batch: report it and leave the state untouched.
        if (i0 == 0) {
            *status = any_negative ? kStatusInvalid : kStatusEmpty;
            if (diag)
                for (int q = 0; q < 4; ++q) diag[q] = __builtin_nan("");
        }
        return;
    }
    float e[kPer], b[kPer];
    int gates = 0;
#pragma unroll
    for (int q = 0; q < kPer; ++q) {
        const int i = i0 + q * nt;
        e[q] = 0.0f;
        b[q] = 0.0f;
        if (i < E) {
            // Normalised load error e = (nbar - n)/nbar = (S - E n)/S: exact
            // integer numerator, one correctly rounded fp64 division, then fp32.
            const long long num = S - (long long)E * (long long)n[q];
            e[q] = (float)((double)num / (double)S);
            const float ep = ep0[q];
            const float de = e[q] - ep;  // Eq. rapid-delta
            // Worsening gate (Eq. rapid-gate) as a sign test: open iff the
            // previous error and its change are both positive or both negative.
            const bool g = (ep > 0.0f && de > 0.0f) || (ep < 0.0f && de < 0.0f);
            float u;
            if (sign_mode) {
                const float sg = (e[q] > 0.0f) ? 1.0f : ((e[q] < 0.0f) ? -1.0f : 0.0f);
                u = Ki * sg;  // DeepSeek fixed-step integral
            } else {
                u = Ki * e[q];  // magnitude-aware integral
            }
            b[q] = b0[q] + u;
            if (g) {
                const float dterm = Kd * de;  // gated, accumulated derivative
                b[q] = b[q] + dterm;
            }
            gates += g ? 1 : 0;
        }
    }
    // Zero-mean centering (second line of Eq. rapid-update): the fixed
    // pairwise tree over the P leaves (level h adds leaf j + h into leaf j for
    // j < h).  Levels h >= nt pair two leaves of one thread (registers);
    // levels nt/2 .. 64 pair the same lane of two waves (one LDS exchange,
    // then wave 0 in registers); the last six run inside wave 0 by shuffles.
    float m = 0.0f;
    if (center) {
        float v[kPer];
#pragma unroll
        for (int q = 0; q < kPer; ++q) v[q] = (i0 + q * nt < E) ? b[q] : 0.0f;
#pragma unroll
        for (int d = kPer / 2; d >= 1; d >>= 1)
            if (2 * d * nt <= P)
#pragma unroll
                for (int q = 0; q < d; ++q) v[q] = v[q] + v[q + d];
        const int NP = P < nt ? P : nt;  // tree nodes left, node i0 in thread i0
        float a = 0.0f;
        if (NP > 64) {
            if (i0 < NP) sh.tree[i0] = v[0];
            __syncthreads();
            if (wv == 0) {
                float r[16];  // node 64 w + lane, w < NP / 64 <= 16
#pragma unroll
                for (int w = 0; w < 16; ++w) r[w] = (w < NP / 64) ? sh.tree[64 * w + lane] : 0.0f;
#pragma unroll
                for (int hw = 8; hw >= 1; hw >>= 1)
                    if (hw < NP / 64)
#pragma unroll
                        for (int w = 0; w < hw; ++w) r[w] = r[w] + r[w + hw];
                a = r[0];
            }
        } else if (wv == 0) {
            a = (lane < NP) ? v[0] : 0.0f;
        }
        if (wv == 0) {
            for (int h = (NP < 64 ? NP : 64) >> 1; h >= 1; h >>= 1) {
                const float up = __shfl_down(a, h);
                if (lane < h) a = a + up;
            }
            if (lane == 0) sh.tree[1024 - 1] = a;  // a slot no other thread reads before the barrier
        }
        __syncthreads();
        m = sh.tree[1024 - 1] / (float)E;
    }
#pragma unroll
    for (int q = 0; q < kPer; ++q) {
        const int i = i0 + q * nt;
        if (i < E) {
            bias[i] = center ? (b[q] - m) : b[q];
            e_prev[i] = e[q];
        }
    }
    if (i0 == 0) {
        *step = *step + 1;
        *status = kStatusOk;
    }
    if (!diag) return;
    // diagnostics of this update
    int zeros = 0;
#pragma unroll
    for (int q = 0; q < kPer; ++q) {
        const int i = i0 + q * nt;
        if (i < E) zeros += n[q] == 0 ? 1 : 0;
        if (i < P) {
            const float nb = (i < E) ? (center ? (b[q] - m) : b[q]) : 0.0f;
            dsh->tree[i] = (i < E) ? (double)fabsf(nb - b0[q]) : 0.0;
        }
    }
    const long long G = block_sum(gates, sh);  // its barriers also publish tree[]
    const long long Z = block_sum(zeros, sh);
    // The m = ceil(E/10) largest counts: their sum does not depend on how ties
    // are ranked, so it is sum(n_i > th) + (m - #{n_i > th}) th with th the
    // m-th largest count, the largest v with #{n_i >= v} >= m, found bit by bit
    // from the top (counts are >= 0 here, mx the largest).
    const int mtop = (E + 9) / 10;
    int th = 0;
    for (int bit = 31 - __builtin_clz((unsigned)mx | 1u), bank = 0; bit >= 0; --bit, bank ^= 1) {
        const int cand = th | (1 << bit);
        int c = 0;
#pragma unroll
        for (int q = 0; q < kPer; ++q) {
            const int i = i0 + q * nt;
            c += __builtin_popcountll(__builtin_amdgcn_ballot_w64(i < E && n[q] >= cand));
        }
        if (lane == 0) dsh->wcnt[bank][wv] = c;
        __syncthreads();  // the other bank was last read before the previous barrier
        int tot = 0;
        for (int w = 0; w < nw; ++w) tot += dsh->wcnt[bank][w];
        if (tot >= mtop) th = cand;
    }
    long long above = 0, nabove = 0;
#pragma unroll
    for (int q = 0; q < kPer; ++q) {
        const int i = i0 + q * nt;
        if (i < E && n[q] > th) {
            above += n[q];
            nabove += 1;
        }
    }
    const long long sum_above = block_sum(above, sh);
    const long long TOP = sum_above + (mtop - block_sum(nabove, sh)) * (long long)th;
    int h = P >> 1;
    for (; h >= 64; h >>= 1) {
        for (int i = i0; i < h; i += nt) dsh->tree[i] = dsh->tree[i] + dsh->tree[i + h];
        __syncthreads();
    }
    if (wv == 0) {
        double a = (lane < P) ? dsh->tree[lane] : 0.0;
        for (; h >= 1; h >>= 1) {
            const double up = __shfl_down(a, h);
            if (lane < h) a = a + up;
        }
        if (lane == 0) {
            diag[0] = (double)G / (double)E;
            diag[1] = (double)TOP / (double)S;
            diag[2] = (double)Z / (double)E;
            diag[3] = a / (double)E;
        }
    }
}

// ---------------------------------------------------------------- one wave

constexpr int kCtrlPer = 16;  // experts per lane: E <= 64 * 16

// Butterfly sum over the wave: every lane ends with the same bits (each step
// adds a pair of equal partial sums in either order, and addition commutes).
template <class V>
__device__ inline V wave_sum(V v) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) v = v + __shfl_xor(v, o);
    return v;
}

// The fixed pairwise tree over P leaves (P a power of two, <= 1024), leaf
// l + 64 q in register q of lane l: level h adds leaf j + h into leaf j for
// j < h, h = P/2, ..., 1.  Levels h >= 64 add register q + h/64 into register
// q of the same lane; the last six use shuffles inside register 0.  Returns
// the root (leaf 0) in every lane.
template <class V>
__device__ inline V wave_tree_sum(V (&a)[kCtrlPer], int P) {
    const int lane = threadIdx.x & 63;
#pragma unroll
    for (int H = 512; H >= 64; H >>= 1) {
        if (H < P) {
#pragma unroll
            for (int q = 0; q < H / 64; ++q) a[q] = a[q] + a[q + H / 64];
        }
    }
    V r = a[0];
    for (int h = (P >> 1) < 32 ? (P >> 1) : 32; h >= 1; h >>= 1) {
        const V up = __shfl_down(r, h);
        if (lane < h) r = r + up;
    }
    return __shfl(r, 0);
}

// A lane's experts' bias and previous error.
__device__ inline void controller_load_state(const float* __restrict__ bias, const float* __restrict__ e_prev, int E,
                                             float (&b0)[kCtrlPer], float (&ep0)[kCtrlPer]) {
    const int lane = threadIdx.x & 63;
#pragma unroll
    for (int q = 0; q < kCtrlPer; ++q) {
        const int i = lane + 64 * q;
        b0[q] = (i < E) ? bias[i] : 0.0f;
        ep0[q] = (i < E) ? e_prev[i] : 0.0f;
    }
}

// controller_wave: the same update as controller_block (the same arithmetic
// and the same fixed trees, so the same bits) by one full wave, lane l
// holding experts l, l + 64, ... (E <= 1024), from the state b0, ep0
// (controller_load_state), with no LDS array and no barrier: one wave per
// layer when many layers update at once.  With a non-null stats pointer it also writes
// MaxVio/MinVio of the same counts; with a non-null diag pointer, the update's
// diagnostics: diag[0] the active-gate fraction #{g_i = 1}/E, diag[1] the
// share of the assignments on the m = ceil(E/10) busiest experts, diag[2] the
// inactive-expert ratio #{n_i = 0}/E, diag[3] the mean |b_new - b_old| summed
// in fp64 over the same pairwise tree; NaN x 4 when the update does not run.
// Counts written by atomics of other workgroups of the same launch are read
// with agent-scope loads (kCoherentCounts).
template <bool kCoherentCounts = false>
__device__ inline void controller_wave(const int32_t* __restrict__ counts, int E, float Ki, float Kd, int sign_mode,
                                       int center, const float (&b0)[kCtrlPer], const float (&ep0)[kCtrlPer],
                                       float* __restrict__ bias, float* __restrict__ e_prev,
                                       int64_t* __restrict__ step, int32_t* __restrict__ status,
                                       double* __restrict__ stats, double* __restrict__ diag = nullptr) {
#pragma clang fp contract(off)
    const int lane = threadIdx.x & 63;
    const int P = ctrl_tree_size(E);
    int n[kCtrlPer];
    long long sum = 0;
    int mx = INT32_MIN, mn = INT32_MAX, neg = 0;
#pragma unroll
    for (int q = 0; q < kCtrlPer; ++q) {
        const int i = lane + 64 * q;
        n[q] = (i >= E) ? 0
               : kCoherentCounts ? __hip_atomic_load(counts + i, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)
                                 : counts[i];
        if (i < E) {
            sum += n[q];
            mx = max(mx, n[q]);
            mn = min(mn, n[q]);
            neg |= n[q] < 0 ? 1 : 0;
        }
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) {
        sum += __shfl_xor(sum, o);
        mx = max(mx, __shfl_xor(mx, o));
        mn = min(mn, __shfl_xor(mn, o));
        neg |= __shfl_xor(neg, o);
    }
    const long long S = sum;  // total assignments S = E * nbar (Eq. pid-error)
    if (stats && lane == 0) {
        // MaxVio, MinVio (Eq. vio): one fp64 division of an exact integer
        // numerator each; NaN for an empty batch.
        if (S == 0) {
            stats[0] = __builtin_nan("");
            stats[1] = __builtin_nan("");
        } else {
            stats[0] = (double)((long long)E * mx - S) / (double)S;
            stats[1] = (double)(S - (long long)E * mn) / (double)S;
        }
    }
    if (neg || S == 0) {
        // Invalid or empty batch: report it and leave the state untouched.
        if (lane == 0) {
            *status = neg ? kStatusInvalid : kStatusEmpty;
            if (diag)
                for (int q = 0; q < 4; ++q) diag[q] = __builtin_nan("");
        }
        return;
    }
    float e[kCtrlPer], b[kCtrlPer];
    int gates = 0;
#pragma unroll
    for (int q = 0; q < kCtrlPer; ++q) {
        const int i = lane + 64 * q;
        e[q] = 0.0f;
        b[q] = 0.0f;
        if (i < E) {
            // Normalised load error e = (nbar - n)/nbar = (S - E n)/S: exact
            // integer numerator, one correctly rounded fp64 division, then fp32.
            const long long num = S - (long long)E * (long long)n[q];
            e[q] = (float)((double)num / (double)S);
            const float ep = ep0[q];
            const float de = e[q] - ep;  // Eq. rapid-delta
            // Worsening gate (Eq. rapid-gate) as a sign test: open iff the
            // previous error and its change are both positive or both negative.
            const bool g = (ep > 0.0f && de > 0.0f) || (ep < 0.0f && de < 0.0f);
            float u;
            if (sign_mode) {
                const float sg = (e[q] > 0.0f) ? 1.0f : ((e[q] < 0.0f) ? -1.0f : 0.0f);
                u = Ki * sg;  // DeepSeek fixed-step integral
            } else {
                u = Ki * e[q];  // magnitude-aware integral
            }
            b[q] = b0[q] + u;
            if (g) {
                const float dterm = Kd * de;  // gated, accumulated derivative
                b[q] = b[q] + dterm;
            }
            gates += g ? 1 : 0;
        }
    }
    // Zero-mean centering (second line of Eq. rapid-update): the mean of b~
    // over the fixed pairwise tree, padded with +0 to P leaves.
    float m = 0.0f;
    if (center) {
        float t[kCtrlPer];
#pragma unroll
        for (int q = 0; q < kCtrlPer; ++q) t[q] = (lane + 64 * q < E) ? b[q] : 0.0f;
        m = wave_tree_sum(t, P) / (float)E;
    }
    float nb[kCtrlPer];
#pragma unroll
    for (int q = 0; q < kCtrlPer; ++q) {
        const int i = lane + 64 * q;
        nb[q] = center ? (b[q] - m) : b[q];
        if (i < E) {
            bias[i] = nb[q];
            e_prev[i] = e[q];
        }
    }
    if (lane == 0) {
        *step = *step + 1;
        *status = kStatusOk;
    }
    if (!diag) return;
    // diagnostics of this update
    int zeros = 0;
    double d[kCtrlPer];
#pragma unroll
    for (int q = 0; q < kCtrlPer; ++q) {
        const bool real = lane + 64 * q < E;
        zeros += (real && n[q] == 0) ? 1 : 0;
        d[q] = real ? (double)fabsf(nb[q] - b0[q]) : 0.0;
    }
    const int G = wave_sum(gates);
    const int Z = wave_sum(zeros);
    // The m = ceil(E/10) largest counts: their sum does not depend on how ties
    // are ranked, so it is sum(n_i > th) + (m - #{n_i > th}) th with th the
    // m-th largest count, the largest v with #{n_i >= v} >= m, found bit by bit
    // from the top (counts are >= 0 here, mx the largest).
    const int mtop = (E + 9) / 10;
    int th = 0;
    for (int bit = 31 - __builtin_clz((unsigned)mx | 1u); bit >= 0; --bit) {
        const int cand = th | (1 << bit);
        int c = 0;
#pragma unroll
        for (int q = 0; q < kCtrlPer; ++q)
            c += __builtin_popcountll(__builtin_amdgcn_ballot_w64(lane + 64 * q < E && n[q] >= cand));
        if (c >= mtop) th = cand;
    }
    long long above = 0;
    int nabove = 0;
#pragma unroll
    for (int q = 0; q < kCtrlPer; ++q) {
        if (lane + 64 * q < E && n[q] > th) {
            above += n[q];
            nabove += 1;
        }
    }
    const long long TOP = wave_sum(above) + (long long)(mtop - wave_sum(nabove)) * (long long)th;
    const double drift = wave_tree_sum(d, P);
    if (lane == 0) {
        diag[0] = (double)G / (double)E;
        diag[1] = (double)TOP / (double)S;
        diag[2] = (double)Z / (double)E;
        diag[3] = drift / (double)E;
    }
}

// Run by every thread of each workgroup of a launch once it is done with
// counts: the workgroup that finishes last (ticket) runs controller_block on
// the complete counts.  The counts are written only by agent-scope atomics
// (performed at the device's coherence point) and read only by agent-scope
// loads (served there too), so no cache write-back or invalidation is needed:
// every wave waits for its own memory operations (the count atomics) to
// complete, the barrier collects the workgroup, and one thread takes the
// ticket; the last workgroup reads the counts after its ticket returns.  The
// controller state it reads is written by no other workgroup of the launch.
template <int kPer>
__device__ inline void controller_tail(const int32_t* counts, int E, float Ki, float Kd, int sign_mode, int center,
                                       float* bias, float* e_prev, int64_t* step, int32_t* status, double* stats,
                                       unsigned* ticket, CtrlScratch& sh) {
    __shared__ int last;
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (threadIdx.x == 0)
        last = __hip_atomic_fetch_add(ticket, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == gridDim.x - 1;
    __syncthreads();
    if (!last) return;
    controller_block<kPer, true>(counts, E, ctrl_tree_size(E), Ki, Kd, sign_mode, center, bias, e_prev, step, status,
                           stats, sh);
}

}  // namespace idb
