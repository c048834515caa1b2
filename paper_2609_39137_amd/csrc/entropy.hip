// Routing entropies (Sec. 4.3), averaged over the tokens of a batch:
//   H_topK = -sum_r w_r log w_r over a token's gate weights (0 log 0 = 0),
//            natural logarithms in fp64;
//   H_full = -sum_e p_e log p_e, p_e = c_e / C, c_e = max(fl32(s_e + b_e), 0),
//            C = sum_e c_e, evaluated as log C - ln 2 (sum_e c_e log2 c_e) / C
//            (H_full = 0 when C = 0), each c_e log2 c_e with the hardware
//            fp32 log2 and summed in fp64 (terms with c_e below the smallest
//            normal fp32 count as 0).
// The softmax form (the auxiliary-loss router, whose selection scores are the
// softmax probabilities of its logits): H_full = log Z - (sum_e t_e (z_e - M))
// / Z with M the token's largest logit, t_e = exp(z_e - M) from the hardware
// exp2 in fp32 and Z = sum_e t_e, both sums in fp64.
// Deterministic: a fixed grid of kEntropyBlocks workgroups with fixed token
// assignments and fixed reduction trees writes per-workgroup partial sums,
// which one wave adds in a fixed order.
#include "common.h"
#include "internal.h"

#pragma clang fp contract(off)

namespace idb {

namespace {

constexpr int kEntThreads = 256;
constexpr int kEntWaves = kEntThreads / 64;
constexpr int kEntPerLane = 16;  // scores per lane and token: E <= 1024

__device__ inline double block_sum_fixed(double v, double* red) {
    // fixed butterfly inside each wave, then the waves in order
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o);
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
    if (lane == 0) red[wv] = v;
    __syncthreads();
    double t = 0.0;
    for (int w = 0; w < kEntWaves; ++w) t += red[w];
    __syncthreads();
    return t;
}

// c log2 c of one clamped biased score, as an fp64 term (0 for c = 0 and for
// c below the smallest normal fp32, whose term is below 2^-119 in size).
__device__ inline double clog2c(float c) {
    return c >= 1.17549435e-38f ? (double)c * (double)__builtin_amdgcn_logf(c) : 0.0;
}

// One token's H_full over the softmax of its logits z (one wave, lane l
// holding z_{l + 64 j}; padding lanes -inf).
__device__ inline double softmax_entropy_wave(const float (&z)[kEntPerLane]) {
    float m = -INFINITY;
#pragma unroll
    for (int j = 0; j < kEntPerLane; ++j) m = fmaxf(m, z[j]);
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) m = fmaxf(m, __shfl_xor(m, o));
    double Z = 0.0, D = 0.0;
#pragma unroll
    for (int j = 0; j < kEntPerLane; ++j) {
        if (z[j] != -INFINITY) {
            const float x = z[j] - m;
            const float t = __builtin_amdgcn_exp2f(x * 1.4426950408889634f);
            Z += (double)t;
            D += (double)t * (double)x;
        }
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) {
        Z += __shfl_xor(Z, o);
        D += __shfl_xor(D, o);
    }
    return log(Z) - D / Z;
}

template <bool SOFTMAX>
__global__ __launch_bounds__(kEntThreads) void entropy_partial_kernel(const float* __restrict__ w, int64_t T, int K,
                                                                      const float* __restrict__ scores,
                                                                      const float* __restrict__ bias, int E,
                                                                      double* __restrict__ partial) {
    __shared__ double red[kEntWaves];
    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    // H_topK: one thread per token
    double htop = 0.0;
    for (int64_t t = (int64_t)blockIdx.x * kEntThreads + tid; t < T; t += (int64_t)gridDim.x * kEntThreads) {
        double h = 0.0;
        for (int r = 0; r < K; ++r) {
            const double x = (double)w[t * K + r];
            if (x > 0.0) h -= x * log(x);
        }
        htop += h;
    }
    const double stop = block_sum_fixed(htop, red);
    // H_full: one wave per token, a lane's experts lane, lane + 64, ...; the
    // bias stays in registers, and two tokens' scores are loaded at once
    double hfull = 0.0;
    if (SOFTMAX) {
        // one wave per token, a lane's logits lane, lane + 64, ...
        for (int64_t t = (int64_t)blockIdx.x * kEntWaves + wv; t < T; t += (int64_t)gridDim.x * kEntWaves) {
            float z[kEntPerLane];
#pragma unroll
            for (int j = 0; j < kEntPerLane; ++j) {
                const int e = lane + 64 * j;
                z[j] = e < E ? scores[t * E + e] : -INFINITY;
            }
            const double h = softmax_entropy_wave(z);
            if (lane == 0) hfull += h;
        }
    } else if (scores) {
        float b[kEntPerLane];
#pragma unroll
        for (int j = 0; j < kEntPerLane; ++j) b[j] = lane + 64 * j < E ? bias[lane + 64 * j] : 0.0f;
        const int64_t step = (int64_t)gridDim.x * kEntWaves;
        for (int64_t t0 = (int64_t)blockIdx.x * kEntWaves + wv; t0 < T; t0 += 2 * step) {
            const int64_t t1 = t0 + step;
            float s0[kEntPerLane], s1[kEntPerLane];
#pragma unroll
            for (int j = 0; j < kEntPerLane; ++j) {
                const int e = lane + 64 * j;
                s0[j] = e < E ? scores[t0 * E + e] : 0.0f;
                s1[j] = (e < E && t1 < T) ? scores[t1 * E + e] : 0.0f;
            }
            double C0 = 0.0, D0 = 0.0, C1 = 0.0, D1 = 0.0;
#pragma unroll
            for (int j = 0; j < kEntPerLane; ++j) {
                if (lane + 64 * j < E) {
                    const float c0 = fmaxf(s0[j] + b[j], 0.0f), c1 = fmaxf(s1[j] + b[j], 0.0f);
                    C0 += (double)c0;
                    D0 += clog2c(c0);
                    C1 += (double)c1;
                    D1 += clog2c(c1);
                }
            }
#pragma unroll
            for (int o = 32; o >= 1; o >>= 1) {
                C0 += __shfl_xor(C0, o);
                D0 += __shfl_xor(D0, o);
                C1 += __shfl_xor(C1, o);
                D1 += __shfl_xor(D1, o);
            }
            constexpr double kLn2 = 0.69314718055994530942;
            if (lane == 0) {
                hfull += C0 > 0.0 ? log(C0) - kLn2 * D0 / C0 : 0.0;
                if (t1 < T) hfull += C1 > 0.0 ? log(C1) - kLn2 * D1 / C1 : 0.0;
            }
        }
    }
    const double sfull = block_sum_fixed(hfull, red);
    if (tid == 0) {
        partial[2 * blockIdx.x] = stop;
        partial[2 * blockIdx.x + 1] = sfull;
    }
}

// One wave: lane l adds the partials l, l + 64, ... in order, then a fixed
// butterfly over the lanes.
__global__ __launch_bounds__(64) void entropy_final_kernel(const double* __restrict__ partial, int nblk, int64_t T,
                                                          int has_scores, double* __restrict__ out) {
    const int lane = threadIdx.x;
    double a = 0.0, b = 0.0;
#pragma unroll 8
    for (int i = lane; i < nblk; i += 64) {
        a += partial[2 * i];
        b += partial[2 * i + 1];
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) {
        a += __shfl_xor(a, o);
        b += __shfl_xor(b, o);
    }
    if (lane == 0) {
        out[0] = a / (double)T;
        out[1] = has_scores ? b / (double)T : __builtin_nan("");
    }
}

}  // namespace

hipError_t launch_routing_entropy(const float* gate_w, int64_t T, int K, const float* scores, const float* bias,
                                  int E, int softmax, double* partial, double* out, hipStream_t stream) {
    if (softmax)
        hipLaunchKernelGGL(entropy_partial_kernel<true>, dim3(kEntropyBlocks), dim3(kEntThreads), 0, stream, gate_w,
                           T, K, scores, bias, E, partial);
    else
        hipLaunchKernelGGL(entropy_partial_kernel<false>, dim3(kEntropyBlocks), dim3(kEntThreads), 0, stream, gate_w,
                           T, K, scores, bias, E, partial);
    hipLaunchKernelGGL(entropy_final_kernel, dim3(1), dim3(64), 0, stream, partial, kEntropyBlocks, T,
                       scores ? 1 : 0, out);
    return hipGetLastError();
}

}  // namespace idb
