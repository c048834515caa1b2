// ID controller update (Alg. 1; Eq. rapid-integral, rapid-delta, rapid-gate,
// rapid-update; SIGN mode: Eq. pid-deepseek) and MaxVio/MinVio (Eq. vio).
//
// Both are O(E) single-workgroup kernels: the controller holds one expert per
// thread (E <= 1024) and reduces in LDS with fixed trees, so the result is
// bit-reproducible.  fp32 steps are evaluated exactly as written: no FMA
// contraction in this file.
#include "common.h"
#include "internal.h"

#pragma clang fp contract(off)

namespace idb {

// One workgroup, one expert per thread.  With a non-null stats pointer it
// also writes MaxVio/MinVio of the same counts (as load_stats_kernel), so a
// step needs one launch for both.
__global__ __launch_bounds__(1024) void controller_update_kernel(const int32_t* __restrict__ counts, int E, int P,
                                                                 float Ki, float Kd, int sign_mode, int center,
                                                                 float* __restrict__ bias,
                                                                 float* __restrict__ e_prev,
                                                                 int64_t* __restrict__ step,
                                                                 int32_t* __restrict__ status,
                                                                 double* __restrict__ stats) {
    __shared__ long long w_sum[16];
    __shared__ int w_max[16], w_min[16], w_neg[16];
    __shared__ float tree[1024];
    const int i = threadIdx.x;
    const int lane = i & 63, wv = i >> 6, nw = blockDim.x >> 6;
    const int n = (i < E) ? counts[i] : 0;
    // Total assignments S = E * nbar (Eq. pid-error), and the largest and
    // smallest count: exact integer reductions (order-free), across the wave
    // by shuffles, then across the waves.
    long long sum = n;
    int mx = (i < E) ? n : INT32_MIN, mn = (i < E) ? n : INT32_MAX, neg = n < 0 ? 1 : 0;
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) {
        sum += __shfl_xor(sum, o);
        mx = max(mx, __shfl_xor(mx, o));
        mn = min(mn, __shfl_xor(mn, o));
        neg |= __shfl_xor(neg, o);
    }
    if (lane == 0) {
        w_sum[wv] = sum;
        w_max[wv] = mx;
        w_min[wv] = mn;
        w_neg[wv] = neg;
    }
    __syncthreads();
    long long S = 0;
    int any_negative = 0;
    mx = INT32_MIN;
    mn = INT32_MAX;
    for (int w = 0; w < nw; ++w) {
        S += w_sum[w];
        mx = max(mx, w_max[w]);
        mn = min(mn, w_min[w]);
        any_negative |= w_neg[w];
    }
    if (stats && i == 0) {
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
    if (any_negative || S == 0) {
        // Invalid or empty batch: report it and leave the state untouched.
        if (i == 0) *status = any_negative ? kStatusInvalid : kStatusEmpty;
        return;
    }
    float e = 0.0f, b = 0.0f;
    if (i < E) {
        // Normalised load error e = (nbar - n)/nbar = (S - E n)/S: exact integer
        // numerator, one correctly rounded fp64 division, then fp32.
        const long long num = S - (long long)E * (long long)n;
        e = (float)((double)num / (double)S);
        const float ep = e_prev[i];
        const float de = e - ep;  // Eq. rapid-delta
        // Worsening gate (Eq. rapid-gate) as a sign test: open iff the previous
        // error and its change are both positive or both negative.
        const bool g = (ep > 0.0f && de > 0.0f) || (ep < 0.0f && de < 0.0f);
        float u;
        if (sign_mode) {
            const float sg = (e > 0.0f) ? 1.0f : ((e < 0.0f) ? -1.0f : 0.0f);
            u = Ki * sg;  // DeepSeek fixed-step integral
        } else {
            u = Ki * e;  // magnitude-aware integral
        }
        b = bias[i] + u;
        if (g) {
            const float dterm = Kd * de;  // gated, accumulated derivative
            b = b + dterm;
        }
    }
    // Zero-mean centering (second line of Eq. rapid-update): fixed pairwise
    // tree over b~ padded with +0 to P = next power of two >= E, level h
    // adding a_{j+h} into a_j for j < h.  Levels h >= 64 go through LDS, the
    // last six inside wave 0 by shuffles (same pairs, same order).
    float m = 0.0f;
    if (center) {
        if (i < P) tree[i] = (i < E) ? b : 0.0f;
        __syncthreads();
        int h = P >> 1;
        for (; h >= 64; h >>= 1) {
            if (i < h) tree[i] = tree[i] + tree[i + h];
            __syncthreads();
        }
        if (wv == 0) {
            float a = (lane < P) ? tree[lane] : 0.0f;
            for (; h >= 1; h >>= 1) {
                const float up = __shfl_down(a, h);
                if (lane < h) a = a + up;
            }
            if (lane == 0) tree[0] = a;
        }
        __syncthreads();
        m = tree[0] / (float)E;
    }
    if (i < E) {
        bias[i] = center ? (b - m) : b;
        e_prev[i] = e;
    }
    if (i == 0) {
        *step = *step + 1;
        *status = kStatusOk;
    }
}

// MaxVio = (E max n - S)/S, MinVio = (S - E min n)/S (Eq. vio), one fp64
// division each of an exact integer numerator.  NaN for an empty batch.
__global__ __launch_bounds__(1024) void load_stats_kernel(const int32_t* __restrict__ counts, int E,
                                                          double* __restrict__ out) {
    __shared__ long long s_sum[1024];
    __shared__ int s_max[1024];
    __shared__ int s_min[1024];
    const int i = threadIdx.x;
    long long S = 0;
    int mx = INT32_MIN, mn = INT32_MAX;
    for (int j = i; j < E; j += blockDim.x) {
        const int n = counts[j];
        S += n;
        mx = max(mx, n);
        mn = min(mn, n);
    }
    s_sum[i] = S;
    s_max[i] = mx;
    s_min[i] = mn;
    __syncthreads();
    for (int h = blockDim.x >> 1; h >= 1; h >>= 1) {
        if (i < h) {
            s_sum[i] += s_sum[i + h];
            s_max[i] = max(s_max[i], s_max[i + h]);
            s_min[i] = min(s_min[i], s_min[i + h]);
        }
        __syncthreads();
    }
    if (i == 0) {
        const long long tot = s_sum[0];
        if (tot == 0) {
            out[0] = __builtin_nan("");
            out[1] = __builtin_nan("");
        } else {
            out[0] = (double)((long long)E * s_max[0] - tot) / (double)tot;
            out[1] = (double)(tot - (long long)E * s_min[0]) / (double)tot;
        }
    }
}

hipError_t launch_controller_update(const int32_t* counts, int E, float Ki, float Kd, int sign_mode, int center,
                                    float* bias, float* e_prev, int64_t* step, int32_t* status, double* stats,
                                    hipStream_t stream) {
    int P = 1;
    while (P < E) P <<= 1;
    const int threads = P < 64 ? 64 : P;
    hipLaunchKernelGGL(controller_update_kernel, dim3(1), dim3(threads), 0, stream, counts, E, P, Ki, Kd,
                       sign_mode, center, bias, e_prev, step, status, stats);
    return hipGetLastError();
}

hipError_t launch_load_stats(const int32_t* counts, int E, double* out, hipStream_t stream) {
    hipLaunchKernelGGL(load_stats_kernel, dim3(1), dim3(1024), 0, stream, counts, E, out);
    return hipGetLastError();
}

}  // namespace idb
