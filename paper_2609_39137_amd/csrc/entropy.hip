// Routing entropies (Sec. 4.3), averaged over the tokens of a batch:
//   H_topK = -sum_r w_r log w_r over a token's gate weights (0 log 0 = 0);
//   H_full = -sum_e p_e log p_e, p_e = c_e / C, c_e = max(fl32(s_e + b_e), 0),
//            C = sum_e c_e, evaluated as log C - (sum_e c_e log c_e) / C
//            (H_full = 0 when C = 0).
// Natural logarithms in fp64.  Deterministic: a fixed grid of kEntropyBlocks
// workgroups with fixed token assignments and fixed reduction trees writes
// per-workgroup partial sums, and one thread adds them in order.
#include "common.h"
#include "internal.h"

#pragma clang fp contract(off)

namespace idb {

namespace {

constexpr int kEntThreads = 256;
constexpr int kEntWaves = kEntThreads / 64;

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
    // H_full: one wave per token
    double hfull = 0.0;
    if (scores) {
        for (int64_t t = (int64_t)blockIdx.x * kEntWaves + wv; t < T; t += (int64_t)gridDim.x * kEntWaves) {
            double C = 0.0, D = 0.0;
            for (int e = lane; e < E; e += 64) {
                const float v = scores[t * E + e] + bias[e];
                if (v > 0.0f) {
                    const double c = (double)v;
                    C += c;
                    D += c * log(c);
                }
            }
#pragma unroll
            for (int o = 32; o >= 1; o >>= 1) {
                C += __shfl_xor(C, o);
                D += __shfl_xor(D, o);
            }
            if (lane == 0) hfull += C > 0.0 ? log(C) - D / C : 0.0;
        }
    }
    const double sfull = block_sum_fixed(hfull, red);
    if (tid == 0) {
        partial[2 * blockIdx.x] = stop;
        partial[2 * blockIdx.x + 1] = sfull;
    }
}

__global__ void entropy_final_kernel(const double* __restrict__ partial, int nblk, int64_t T, int has_scores,
                                     double* __restrict__ out) {
    if (threadIdx.x != 0) return;
    double a = 0.0, b = 0.0;
    for (int i = 0; i < nblk; ++i) {
        a += partial[2 * i];
        b += partial[2 * i + 1];
    }
    out[0] = a / (double)T;
    out[1] = has_scores ? b / (double)T : __builtin_nan("");
}

}  // namespace

hipError_t launch_routing_entropy(const float* gate_w, int64_t T, int K, const float* scores, const float* bias,
                                  int E, double* partial, double* out, hipStream_t stream) {
    hipLaunchKernelGGL(entropy_partial_kernel, dim3(kEntropyBlocks), dim3(kEntThreads), 0, stream, gate_w, T, K,
                       scores, bias, E, partial);
    hipLaunchKernelGGL(entropy_final_kernel, dim3(1), dim3(64), 0, stream, partial, kEntropyBlocks, T,
                       scores ? 1 : 0, out);
    return hipGetLastError();
}

}  // namespace idb
