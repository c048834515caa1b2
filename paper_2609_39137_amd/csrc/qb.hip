// Quantile Balancing's bias update (Eq. pid-quantile, Eq. pid-quantile-def),
// with the EMA variant the paper uses as a diagnostic: for each expert j,
//   d_ij = fl32(s_ij - alpha_i)                   (margins, -0 read as +0)
//   q_j  = quantile_{1-K/E}(d_.j) = the k-th smallest margin,
//          k = ceil(T (E - K) / E)                (inverted empirical CDF)
//   b_j  = -q_j, or fl32(fl32(rho b_j) + fl32(fl32(1 - rho) (-q_j))) for rho > 0.
// s comes expert-major ([E][T], written by the router in its Quantile
// Balancing mode) and alpha [T] is each token's (K+1)-th largest biased score.
//
// One workgroup per expert finds the exact k-th smallest margin by an
// MSB-first radix select over the margins' order-preserving 32-bit keys: four
// passes of 8-bit digits, each a histogram of the keys that match the digits
// found so far (one LDS histogram per wave, then summed), the digit taken
// where the running count reaches the rank still wanted.  Up to 32768 tokens
// the keys are computed once into LDS (NK slots); beyond, each pass
// recomputes them from global memory.
#include "common.h"
#include "internal.h"

#pragma clang fp contract(off)

namespace idb {

namespace {

constexpr int kQbThreads = 512;
constexpr int kQbWaves = kQbThreads / 64;

// Order-preserving key of a float (after -0 -> +0): a < b iff key(a) < key(b).
__device__ __forceinline__ unsigned order_key(float d) {
    const unsigned u = __float_as_uint(d + 0.0f);
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ __forceinline__ float key_value(unsigned o) {
    return __uint_as_float((o & 0x80000000u) ? (o & 0x7fffffffu) : ~o);
}

template <int NK>  // LDS key slots (T <= NK), or 0: keys recomputed per pass
__global__ __launch_bounds__(kQbThreads) void qb_update_kernel(const float* __restrict__ scores_t,
                                                               const float* __restrict__ alpha, int64_t T, int E,
                                                               int K, float rho, float* __restrict__ bias) {
    constexpr bool IN_LDS = NK > 0;
    __shared__ unsigned keys[IN_LDS ? NK : 1];
    __shared__ unsigned hist[kQbWaves][256];
    __shared__ unsigned pick[2];  // digit, count below it
    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int j = blockIdx.x;
    const float* row = scores_t + (int64_t)j * T;
    auto margin_key = [&](int64_t t) { return order_key(row[t] - alpha[t]); };
    if (IN_LDS) {
        for (int64_t t = tid; t < T; t += kQbThreads) keys[t] = margin_key(t);
    }
    // rank wanted, 1-based ascending; T <= 2^26 keeps every count in 32 bits
    unsigned kleft = (unsigned)((T * (int64_t)(E - K) + E - 1) / E);
    unsigned prefix = 0u, mask = 0u;
    for (int shift = 24; shift >= 0; shift -= 8) {
        for (int i = tid; i < kQbWaves * 256; i += kQbThreads) (&hist[0][0])[i] = 0u;
        __syncthreads();
        for (int64_t t = tid; t < T; t += kQbThreads) {
            const unsigned u = IN_LDS ? keys[t] : margin_key(t);
            if ((u & mask) == prefix) atomicAdd(&hist[wave][(u >> shift) & 255u], 1u);
        }
        __syncthreads();
        if (wave == 0) {
            // lane l owns digits 4l .. 4l+3; an inclusive scan over the lanes
            // finds the digit where the count reaches kleft
            unsigned c[4], tot = 0u;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                unsigned n = 0u;
#pragma unroll
                for (int w = 0; w < kQbWaves; ++w) n += hist[w][4 * lane + i];
                c[i] = n;
                tot += n;
            }
            unsigned incl = tot;
#pragma unroll
            for (int o = 1; o < 64; o <<= 1) {
                const unsigned up = __shfl_up(incl, o);
                if (lane >= o) incl += up;
            }
            unsigned run = incl - tot;  // keys in lower digits
            if (run < kleft && kleft <= incl) {
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    if (run < kleft && kleft <= run + c[i]) {
                        pick[0] = (unsigned)(4 * lane + i);
                        pick[1] = run;
                    }
                    run += c[i];
                }
            }
        }
        __syncthreads();
        prefix |= pick[0] << shift;
        mask |= 255u << shift;
        kleft -= pick[1];
        __syncthreads();  // pick[] is rewritten by the next pass
    }
    if (tid == 0) {
        const float Q = -key_value(prefix);
        if (rho == 0.0f) {
            bias[j] = Q;
        } else {
            const float keep = rho * bias[j];
            const float take = (1.0f - rho) * Q;
            bias[j] = keep + take;
        }
    }
}

}  // namespace

hipError_t launch_qb_update(const float* scores_t, const float* alpha, int64_t T, int E, int K, float rho,
                            float* bias, hipStream_t stream) {
    if (T <= 16384)
        hipLaunchKernelGGL(qb_update_kernel<16384>, dim3((unsigned)E), dim3(kQbThreads), 0, stream, scores_t, alpha,
                           T, E, K, rho, bias);
    else if (T <= 32768)
        hipLaunchKernelGGL(qb_update_kernel<32768>, dim3((unsigned)E), dim3(kQbThreads), 0, stream, scores_t, alpha,
                           T, E, K, rho, bias);
    else
        hipLaunchKernelGGL(qb_update_kernel<0>, dim3((unsigned)E), dim3(kQbThreads), 0, stream, scores_t, alpha, T,
                           E, K, rho, bias);
    return hipGetLastError();
}

}  // namespace idb
