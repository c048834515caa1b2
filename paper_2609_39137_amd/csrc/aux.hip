// Auxiliary-loss balancing's forward statistics (Eq. pid-auxloss) from the
// fused router's per-tile rows: the softmax column sums and the expert counts
// of every token tile.  Writes counts n_i, f_i = n_i / T, P_i = (1/T) times
// the sum of p_i over the batch, the loss alpha * sum_i f_i P_i and, when
// asked, MaxVio/MinVio (Eq. vio).  Fixed summation orders throughout
// (deterministic), fp64 above the per-tile fp32 sums.
#include "common.h"
#include "internal.h"

namespace idb {
namespace {

constexpr int kAuxThreads = 1024;
constexpr int kAuxWaves = kAuxThreads / 64;
constexpr int kAuxBatch = 16;  // tile rows a wave has in flight

// One workgroup per 64 experts, lane = expert.  Wave w adds the tiles w,
// w + 16, ... in order (kAuxBatch rows in flight); wave 0 adds the wave sums
// in order and reduces over its experts; the workgroup that finishes last
// adds the workgroups' records in order.
__global__ __launch_bounds__(kAuxThreads) void aux_stats_kernel(const float* __restrict__ part,
                                                                const int32_t* __restrict__ cpart, int tiles,
                                                                int64_t T, int E, double alpha,
                                                                int32_t* __restrict__ counts, double* __restrict__ f,
                                                                double* __restrict__ P, double* __restrict__ loss,
                                                                double* __restrict__ stats,
                                                                AuxPartial* __restrict__ partial,
                                                                unsigned* __restrict__ ticket) {
    __shared__ double red[kAuxWaves][64];
    __shared__ long long cred[kAuxWaves][64];
    __shared__ int last;
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
    const int i = blockIdx.x * 64 + lane;
    const bool real = i < E;
    const int ic = real ? i : E - 1;  // padding lanes read a valid column, then drop it
    double acc = 0.0;
    long long cacc = 0;
    for (int r0 = wv; r0 < tiles; r0 += kAuxWaves * kAuxBatch) {
        float v[kAuxBatch];
        int c[kAuxBatch];
#pragma unroll
        for (int j = 0; j < kAuxBatch; ++j) {
            const int r = r0 + kAuxWaves * j;
            const int rr = r < tiles ? r : tiles - 1;
            v[j] = part[(int64_t)rr * E + ic];
            c[j] = cpart[(int64_t)rr * E + ic];
        }
#pragma unroll
        for (int j = 0; j < kAuxBatch; ++j) {
            if (r0 + kAuxWaves * j < tiles) {
                acc = acc + (double)v[j];
                cacc += c[j];
            }
        }
    }
    red[wv][lane] = acc;
    cred[wv][lane] = cacc;
    __syncthreads();
    if (wv == 0) {
        double s = 0.0;
        long long n = 0;
#pragma unroll
        for (int w = 0; w < kAuxWaves; ++w) {
            s = s + red[w][lane];
            n += cred[w][lane];
        }
        double fp = 0.0;
        long long nsum = 0;
        int mx = INT32_MIN, mn = INT32_MAX;
        if (real) {
            const double Pi = s / (double)T;
            const double fi = (double)n / (double)T;
            counts[i] = (int32_t)n;
            P[i] = Pi;
            f[i] = fi;
            fp = fi * Pi;
            nsum = n;
            mx = mn = (int)n;
        }
#pragma unroll
        for (int o = 32; o >= 1; o >>= 1) {
            fp = fp + __shfl_xor(fp, o);
            nsum += __shfl_xor(nsum, o);
            mx = max(mx, __shfl_xor(mx, o));
            mn = min(mn, __shfl_xor(mn, o));
        }
        if (lane == 0) {
            // agent-scope stores: coherent across the XCDs' L2s without a
            // cache write-back
            __hip_atomic_store(&partial[blockIdx.x].fp, fp, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            __hip_atomic_store(&partial[blockIdx.x].sum, nsum, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            __hip_atomic_store(&partial[blockIdx.x].max, mx, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            __hip_atomic_store(&partial[blockIdx.x].min, mn, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
    }
    // The records are written and read only by agent-scope atomic accesses:
    // a workgroup waits for its own stores to complete before it takes a
    // ticket (a relaxed increment), and the workgroup that takes the last one
    // reads the records after its ticket, so no cache write-back or
    // invalidation is needed around the ticket.
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (threadIdx.x == 0)
        last = __hip_atomic_fetch_add(ticket, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == gridDim.x - 1;
    __syncthreads();
    if (!last) return;
    if (threadIdx.x == 0) {
        double L = 0.0;
        long long S = 0;
        int mx = INT32_MIN, mn = INT32_MAX;
        for (int q = 0; q < (int)gridDim.x; ++q) {
            L = L + __hip_atomic_load(&partial[q].fp, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            S += __hip_atomic_load(&partial[q].sum, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            mx = max(mx, __hip_atomic_load(&partial[q].max, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
            mn = min(mn, __hip_atomic_load(&partial[q].min, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
        }
        *loss = alpha * L;
        if (stats) {
            // MaxVio, MinVio: one fp64 division of an exact integer numerator each
            stats[0] = (double)((long long)E * mx - S) / (double)S;
            stats[1] = (double)(S - (long long)E * mn) / (double)S;
        }
    }
}

}  // namespace

hipError_t launch_aux_stats(const float* prob_part, const int32_t* cnt_part, int tiles, int64_t T, int E,
                            double alpha, int32_t* counts, double* f, double* P, double* loss, double* stats,
                            AuxPartial* partial, unsigned* ticket, hipStream_t stream) {
    const int blocks = (E + 63) / 64;  // <= kAuxMaxBlocks for E <= 1024
    hipLaunchKernelGGL(aux_stats_kernel, dim3((unsigned)blocks), dim3(kAuxThreads), 0, stream, prob_part, cnt_part,
                       tiles, T, E, alpha, counts, f, P, loss, stats, partial, ticket);
    return hipGetLastError();
}

}  // namespace idb
