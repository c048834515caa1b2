// ID controller update (Alg. 1; Eq. rapid-integral, rapid-delta, rapid-gate,
// rapid-update; SIGN mode: Eq. pid-deepseek) and MaxVio/MinVio (Eq. vio).
//
// The single-layer controller holds one expert per thread of one workgroup
// (E <= 1024) and reduces in LDS with fixed trees; the batched kernel runs one
// wave per layer with the same trees in registers; both are bit-reproducible
// and give the same bits.  fp32 steps are evaluated exactly as written: no FMA
// contraction in this file.
#include "common.h"
#include "controller_block.h"
#include "internal.h"

#pragma clang fp contract(off)

namespace idb {

__global__ __launch_bounds__(1024) void controller_update_kernel(const int32_t* __restrict__ counts, int E, int P,
                                                                 float Ki, float Kd, int sign_mode, int center,
                                                                 float* __restrict__ bias,
                                                                 float* __restrict__ e_prev,
                                                                 int64_t* __restrict__ step,
                                                                 int32_t* __restrict__ status,
                                                                 double* __restrict__ stats) {
    __shared__ CtrlScratch sh;
    controller_block<1>(counts, E, P, Ki, Kd, sign_mode, center, bias, e_prev, step, status, stats, sh);
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

// L layers' updates in one launch, one wave per layer (Alg. 1 runs once per
// MoE layer and iteration): counts, bias and e_prev [L][E], step and status
// [L], stats [L][2] and diag [L][4] (both nullable).  The same bits as the
// single-layer update.
__global__ __launch_bounds__(64) void controller_layers_kernel(const int32_t* __restrict__ counts, int E, float Ki,
                                                               float Kd, int sign_mode, int center,
                                                               float* __restrict__ bias, float* __restrict__ e_prev,
                                                               int64_t* __restrict__ step,
                                                               int32_t* __restrict__ status,
                                                               double* __restrict__ stats,
                                                               double* __restrict__ diag) {
    const int64_t l = blockIdx.x;
    float b0[kCtrlPer], ep0[kCtrlPer];
    controller_load_state(bias + l * E, e_prev + l * E, E, b0, ep0);
    controller_wave(counts + l * E, E, Ki, Kd, sign_mode, center, b0, ep0, bias + l * E, e_prev + l * E, step + l,
                    status + l, stats ? stats + 2 * l : nullptr, diag ? diag + 4 * l : nullptr);
}

hipError_t launch_controller_update(const int32_t* counts, int E, float Ki, float Kd, int sign_mode, int center,
                                    float* bias, float* e_prev, int64_t* step, int32_t* status, double* stats,
                                    hipStream_t stream) {
    const int P = ctrl_tree_size(E);
    const int threads = P < 64 ? 64 : P;
    hipLaunchKernelGGL(controller_update_kernel, dim3(1), dim3(threads), 0, stream, counts, E, P, Ki, Kd,
                       sign_mode, center, bias, e_prev, step, status, stats);
    return hipGetLastError();
}

hipError_t launch_controller_layers(const int32_t* counts, int L, int E, float Ki, float Kd, int sign_mode,
                                    int center, float* bias, float* e_prev, int64_t* step, int32_t* status,
                                    double* stats, double* diag, hipStream_t stream) {
    hipLaunchKernelGGL(controller_layers_kernel, dim3((unsigned)L), dim3(64), 0, stream, counts, E, Ki, Kd, sign_mode,
                       center, bias, e_prev, step, status, stats, diag);
    return hipGetLastError();
}

hipError_t launch_load_stats(const int32_t* counts, int E, double* out, hipStream_t stream) {
    hipLaunchKernelGGL(load_stats_kernel, dim3(1), dim3(1024), 0, stream, counts, E, out);
    return hipGetLastError();
}

}  // namespace idb
