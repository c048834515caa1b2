// Bias-adjusted Top-K selection from given fp32 scores (Eq. pid-routing), gate
// weights from the unbiased scores (Sec. 2.2) and per-expert load counts
// (Eq. pid-error): the router step without the gate contraction, an HBM-bound
// pass over a materialised T x E score matrix.
//
// A workgroup of 512 threads walks tiles of 32 tokens (grid-stride, one
// workgroup per CU: the score rows of a tile take most of the LDS).  A tile's scores go from registers into the LDS score
// rows of the selection epilogue (epilogue.h, one slice of BE >= E experts,
// padding -inf); right after, the next tile's scores are loaded into the same
// registers, so their HBM reads overlap the selection of the current tile.
// The LDS histogram is flushed once per workgroup.
#include "common.h"
#include "epilogue.h"
#include "internal.h"

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
    if (E <= 256) return launch_select_be<256>(a, scores, stream);
    if (E <= 512) return launch_select_be<512>(a, scores, stream);
    if (E <= 768) return launch_select_be<768>(a, scores, stream);
    return launch_select_be<1024>(a, scores, stream);
}

}  // namespace idb
