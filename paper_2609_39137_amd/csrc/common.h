// Internal helpers shared by the gfx950 kernels of the ID Balancing router
// step.  Device code only; the C ABI lives in abi.cpp.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace idb {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef float floatx4 __attribute__((ext_vector_type(4)));

// Device status codes (same values as idb_status in include/idb.h).
constexpr int32_t kStatusOk = 0;
constexpr int32_t kStatusInvalid = 1;
constexpr int32_t kStatusEmpty = 3;

// Largest number of experts selected per token on the GPU paths.
constexpr int kMaxK = 32;

// Strict total order of the biased-score ranking (Eq. pid-routing) with the
// lowest expert index winning ties: does (va, ia) rank above (vb, ib)?
// IEEE comparisons, so -0 == +0.
__device__ __forceinline__ bool ranks_above(float va, int ia, float vb, int ib) {
    return (va > vb) || (va == vb && ia < ib);
}

// The same order as one unsigned 64-bit key: key(a) > key(b) exactly when
// ranks_above(a, b).  High word: the float's bits mapped to an unsigned order
// (after -0 -> +0, so equal values get equal words); low word: ~index, so the
// lower index wins ties.  Key 0 ranks below every finite or infinite value and
// serves as "no entry".
__device__ __forceinline__ unsigned long long rank_key(float v, int idx) {
    const unsigned u = __float_as_uint(v + 0.0f);  // -0 + +0 = +0
    const unsigned o = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
    return ((unsigned long long)o << 32) | (unsigned)(~(unsigned)idx);
}

// The value of a rank key (inverse of its high word; -0 comes back as +0).
__device__ __forceinline__ float rank_key_value(unsigned long long key) {
    const unsigned o = (unsigned)(key >> 32);
    return __uint_as_float((o & 0x80000000u) ? (o & 0x7fffffffu) : ~o);
}

// Orders a wave's LDS writes before the same wave's later LDS reads of what
// other lanes wrote: one wave's LDS instructions execute in issue order, so
// only the compiler has to be kept from moving memory operations across.
__device__ __forceinline__ void wave_sync() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Score activation s = sigmoid(z) = 1 / (1 + 2^(-z log2 e)) with the hardware
// exp2 and reciprocal (each about 1 ulp).  Saturates to exactly 0 and 1.
__device__ __forceinline__ float sigmoid_fast(float z) {
    float e = __builtin_amdgcn_exp2f(z * -1.4426950408889634f);
    return __builtin_amdgcn_rcpf(1.0f + e);
}

// 16 values held one per lane in each 16-lane row of a wave: the value of
// rank `r` in ascending order (bitonic sort across the row).  Every lane of the
// row gets the result.  All 16 lanes of the row must be active.
__device__ __forceinline__ float row16_sorted_ascending_at(float x, int r) {
    const int lane = threadIdx.x & 15;
#pragma unroll
    for (int k = 2; k <= 16; k <<= 1) {
#pragma unroll
        for (int j = k >> 1; j > 0; j >>= 1) {
            float o = __shfl_xor(x, j, 16);
            bool lower = (lane & j) == 0;
            bool up = (lane & k) == 0;
            float lo = fminf(x, o), hi = fmaxf(x, o);
            x = (lower == up) ? lo : hi;
        }
    }
    return __shfl(x, r, 16);
}

// Sort N (a power of two) register values ascending in place (fixed bitonic
// network).
template <int N>
__device__ __forceinline__ void sort_ascending(float (&a)[N]) {
    static_assert((N & (N - 1)) == 0, "bitonic network needs a power of two");
#pragma unroll
    for (int k = 2; k <= N; k <<= 1) {
#pragma unroll
        for (int j = k >> 1; j > 0; j >>= 1) {
#pragma unroll
            for (int i = 0; i < N; ++i) {
                const int l = i ^ j;
                if (l > i) {
                    const float lo = fminf(a[i], a[l]), hi = fmaxf(a[i], a[l]);
                    if ((i & k) == 0) {
                        a[i] = lo;
                        a[l] = hi;
                    } else {
                        a[i] = hi;
                        a[l] = lo;
                    }
                }
            }
        }
    }
}

__device__ __forceinline__ uint4 ld16(const void* p) { return *reinterpret_cast<const uint4*>(p); }

// Raw buffer resource over [base, base + bytes) (bytes < 2^32) and a 16-byte
// load at per-lane offset voff plus scalar offset soff.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, int64_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, (int)bytes, 0x00020000);
}
__device__ __forceinline__ uint4 bload16(__amdgpu_buffer_rsrc_t r, int voff, int soff) {
    const auto v = __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, 0);
    return make_uint4(v[0], v[1], v[2], v[3]);
}

__device__ __forceinline__ bf16x8 as_bf16x8(uint4 u) { return __builtin_bit_cast(bf16x8, u); }

// Gate weights of one token from its selected unbiased scores in rank order:
// den is the fp32 sum in rank order; w_r = s_r / den (IEEE division); den == 0
// gives 1/K.
__device__ __forceinline__ float gate_weight(const float* sel_s, int K, int r) {
    float den = 0.0f;
    for (int q = 0; q < K; ++q) den = den + sel_s[q];
    return (den == 0.0f) ? 1.0f / (float)K : sel_s[r] / den;
}

}  // namespace idb
