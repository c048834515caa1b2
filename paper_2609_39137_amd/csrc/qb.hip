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
// each thread keeps its keys in registers (R <= 32 of them, 512 or 1024
// threads) and the selection first narrows the keys to the few near the top
// (see qb_update_reg_kernel).  Beyond 32768 tokens each pass recomputes the
// keys from global memory.
//
// With a counts pointer, workgroup 0 also writes MaxVio/MinVio of the step's
// counts (Eq. vio), as the stand-alone statistics kernel does: exact integer
// sum, maximum and minimum, one fp64 division each (NaN for an empty batch),
// after its own expert's selection (loading the counts at launch instead keeps
// them in registers through the selection: more spills, slower).
#include "common.h"
#include "internal.h"

#pragma clang fp contract(off)

namespace idb {

namespace {

constexpr int kQbThreads = 512;  // the global-memory kernel's workgroup
constexpr int kQbList = 4096;    // compacted keys after the first pass

// Order-preserving key of a float (after -0 -> +0): a < b iff key(a) < key(b).
__device__ __forceinline__ unsigned order_key(float d) {
    const unsigned u = __float_as_uint(d + 0.0f);
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ __forceinline__ float key_value(unsigned o) {
    return __uint_as_float((o & 0x80000000u) ? (o & 0x7fffffffu) : ~o);
}

// Counts of digits into a wave's histogram.  The margins crowd into a few
// digits (the high byte is mostly sign and exponent), so runs of equal digits
// are counted in a two-entry cache and added with one LDS atomic each.
struct DigitCounter {
    unsigned d0 = 256u, c0 = 0u, d1 = 256u, c1 = 0u;  // digit 256: empty entry
    __device__ __forceinline__ void add(unsigned* h, unsigned dg) {
        if (dg == d0) {
            ++c0;
        } else if (dg == d1) {
            ++c1;
        } else {
            if (c1) atomicAdd(&h[d1], c1);
            d1 = d0;
            c1 = c0;
            d0 = dg;
            c0 = 1u;
        }
    }
    __device__ __forceinline__ void flush(unsigned* h) {
        if (c0) atomicAdd(&h[d0], c0);
        if (c1) atomicAdd(&h[d1], c1);
    }
};

// After a pass's histogram is complete, run by wave 0: the digit where the
// running count reaches kleft (lane l owns digits 4l .. 4l+3), published with
// the count of the keys below it and in it.
template <int NW>
__device__ __forceinline__ void pick_digit(unsigned (&hist)[NW][256], unsigned kleft, unsigned* pick) {
    const int lane = threadIdx.x & 63;
    unsigned c[4], tot = 0u;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        unsigned n = 0u;
#pragma unroll
        for (int w = 0; w < NW; ++w) n += hist[w][4 * lane + i];
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
                pick[2] = c[i];
            }
            run += c[i];
        }
    }
}

__device__ __forceinline__ void write_bias(float* bias, int j, unsigned key, float rho) {
    const float Q = -key_value(key);
    if (rho == 0.0f) {
        bias[j] = Q;
    } else {
        const float keep = rho * bias[j];
        const float take = (1.0f - rho) * Q;
        bias[j] = keep + take;
    }
}

// Orders the LDS accesses of one wave's lanes (a code-motion barrier; a wave's
// LDS operations execute in order).
__device__ __forceinline__ void wave_sync() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Radix select run by one wave over n keys in LDS: the key of ascending rank
// kleft (1-based), returned to every lane.  h: the wave's 256-bin histogram.
__device__ unsigned wave_select(const unsigned* vals, unsigned n, unsigned kleft, unsigned* h) {
    const int lane = threadIdx.x & 63;
    unsigned prefix = 0u, mask = 0u;
    for (int shift = 24; shift >= 0; shift -= 8) {
#pragma unroll
        for (int i = 0; i < 4; ++i) h[4 * lane + i] = 0u;
        wave_sync();
        DigitCounter dc;
        for (unsigned i = lane; i < n; i += 64) {
            const unsigned u = vals[i];
            if ((u & mask) == prefix) dc.add(h, (u >> shift) & 255u);
        }
        dc.flush(h);
        wave_sync();
        unsigned c[4], tot = 0u;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            c[i] = h[4 * lane + i];
            tot += c[i];
        }
        unsigned incl = tot;
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
            const unsigned up = __shfl_up(incl, o);
            if (lane >= o) incl += up;
        }
        unsigned run = incl - tot, digit = 0u, below = 0u;
        const bool mine = run < kleft && kleft <= incl;
        if (mine) {
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                if (run < kleft && kleft <= run + c[i]) {
                    digit = (unsigned)(4 * lane + i);
                    below = run;
                }
                run += c[i];
            }
        }
        const int src = __builtin_ctzll(__ballot(mine));
        digit = __shfl(digit, src);
        below = __shfl(below, src);
        prefix |= digit << shift;
        mask |= 255u << shift;
        kleft -= below;
        wave_sync();  // the histogram is reset by the next pass
    }
    return prefix;
}

// The same selection for n <= 64 * V keys: each lane loads its V keys once
// and every pass reads registers only.
// With LOW > 0 the passes stop above bit LOW: the result is the selected
// key's high bits with the low LOW bits zero, a lower bound of the key.
template <int V, int LOW = 0>
__device__ unsigned wave_select_reg(const unsigned* vals, unsigned n, unsigned kleft, unsigned* h) {
    const int lane = threadIdx.x & 63;
    unsigned v[V];
#pragma unroll
    for (int i = 0; i < V; ++i) {
        const unsigned idx = (unsigned)lane + 64u * i;
        v[i] = idx < n ? vals[idx] : 0u;
    }
    unsigned prefix = 0u, mask = 0u;
    for (int shift = 24; shift >= LOW; shift -= 8) {
#pragma unroll
        for (int i = 0; i < 4; ++i) h[4 * lane + i] = 0u;
        wave_sync();
        DigitCounter dc;
#pragma unroll
        for (int i = 0; i < V; ++i)
            if ((unsigned)lane + 64u * i < n && (v[i] & mask) == prefix) dc.add(h, (v[i] >> shift) & 255u);
        dc.flush(h);
        wave_sync();
        unsigned c[4], tot = 0u;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            c[i] = h[4 * lane + i];
            tot += c[i];
        }
        unsigned incl = tot;
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
            const unsigned up = __shfl_up(incl, o);
            if (lane >= o) incl += up;
        }
        unsigned run = incl - tot, digit = 0u, below = 0u;
        const bool mine = run < kleft && kleft <= incl;
        if (mine) {
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                if (run < kleft && kleft <= run + c[i]) {
                    digit = (unsigned)(4 * lane + i);
                    below = run;
                }
                run += c[i];
            }
        }
        const int src = __builtin_ctzll(__ballot(mine));
        digit = __shfl(digit, src);
        below = __shfl(below, src);
        prefix |= digit << shift;
        mask |= 255u << shift;
        kleft -= below;
        wave_sync();  // the histogram is reset by the next pass
    }
    return prefix;
}

// MaxVio, MinVio of counts whose entries i = tid + NT q (q < NQ) thread tid
// holds in n[] (0 past E), over a workgroup of NT threads.
template <int NT, int NQ>
__device__ void qb_block_stats(const int (&n)[NQ], int E, double* __restrict__ out) {
    constexpr int NW = NT / 64;
    __shared__ long long w_sum[NW];
    __shared__ int w_max[NW], w_min[NW];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    long long S = 0;
    int mx = INT32_MIN, mn = INT32_MAX;
#pragma unroll
    for (int q = 0; q < NQ; ++q)
        if (tid + NT * q < E) {
            S += n[q];
            mx = max(mx, n[q]);
            mn = min(mn, n[q]);
        }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) {
        S += __shfl_xor(S, o);
        mx = max(mx, __shfl_xor(mx, o));
        mn = min(mn, __shfl_xor(mn, o));
    }
    if (lane == 0) {
        w_sum[wave] = S;
        w_max[wave] = mx;
        w_min[wave] = mn;
    }
    __syncthreads();
    if (tid == 0) {
        for (int w = 1; w < NW; ++w) {
            S += w_sum[w];
            mx = max(mx, w_max[w]);
            mn = min(mn, w_min[w]);
        }
        if (S == 0) {
            out[0] = __builtin_nan("");
            out[1] = __builtin_nan("");
        } else {
            out[0] = (double)((long long)E * mx - S) / (double)S;
            out[1] = (double)(S - (long long)E * mn) / (double)S;
        }
    }
}

// The counts that thread tid of workgroup 0 holds for qb_block_stats.
template <int NT, int NQ>
__device__ __forceinline__ void qb_stats_load(const int32_t* __restrict__ counts, int E, int (&n)[NQ]) {
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
        const int i = threadIdx.x + NT * q;
        n[q] = i < E ? counts[i] : 0;
    }
}

// NT threads, R keys per thread in registers (T <= R * NT).  The wanted key
// is the r-th largest, r = T - k + 1, normally far fewer than T.  When r <=
// NT: tau = the r-th largest of the threads' maxima with its 16 low bits
// cleared (at least r keys are >= tau, so the wanted key is one of them, and
// its rank from the top is the same within the keys >= tau); those keys go to
// an LDS list and one wave selects the exact key from it (both small
// selections run in one wave on registers; a longer list is read from LDS
// each pass).  Otherwise, or when the list would overflow, a full radix
// select over the registers.
template <int NT, int R, bool VEC>
__global__ __launch_bounds__(NT) __attribute__((amdgpu_waves_per_eu(NT == 512 ? 6 : 1)))
void qb_update_reg_kernel(const float* __restrict__ scores_t,
                                                           const float* __restrict__ alpha, int64_t T, int E, int K,
                                                           float rho, float* __restrict__ bias,
                                                           const int32_t* __restrict__ counts,
                                                           double* __restrict__ stats) {
    constexpr int NW = NT / 64;
    constexpr int NQ = (1024 + NT - 1) / NT;  // counts per thread of workgroup 0 (E <= 1024)
    __shared__ unsigned hist[NW][256];
    __shared__ unsigned list[kQbList];
    __shared__ unsigned maxima[NT];
    __shared__ unsigned pick[3];  // digit, keys below it, keys in it
    __shared__ unsigned nlist, tau_s;
    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int j = blockIdx.x;
    const float* row = scores_t + (int64_t)j * T;
    const bool with_stats = counts && j == 0;  // uniform over the workgroup

    // Key slot r holds token tok(r): with VEC (T % 4 == 0) the tokens
    // 4 (tid + NT i) + c for r = 4 i + c, read as float4 pieces, every load of
    // the thread in flight at once; else tid + NT r.  Slots past T are never
    // counted.
    unsigned key[R];
    auto tok = [&](int r) -> int64_t {
        return VEC ? 4 * (tid + (int64_t)(r / 4) * NT) + (r % 4) : tid + (int64_t)r * NT;
    };
    if (VEC) {
        constexpr int Q = R / 4;
        const float4* row4 = reinterpret_cast<const float4*>(row);
        const float4* alpha4 = reinterpret_cast<const float4*>(alpha);
        const int64_t last = T / 4 - 1;
        float4 sv[Q], av[Q];
#pragma unroll
        for (int i = 0; i < Q; ++i) {
            int64_t q = tid + (int64_t)i * NT;
            q = q < last ? q : last;
            sv[i] = row4[q];
            av[i] = alpha4[q];
        }
#pragma unroll
        for (int i = 0; i < Q; ++i) {
            key[4 * i + 0] = order_key(sv[i].x - av[i].x);
            key[4 * i + 1] = order_key(sv[i].y - av[i].y);
            key[4 * i + 2] = order_key(sv[i].z - av[i].z);
            key[4 * i + 3] = order_key(sv[i].w - av[i].w);
        }
    } else {
        constexpr int H = R < 16 ? R : 16;  // loads in flight per batch
#pragma unroll
        for (int h = 0; h < R; h += H) {
            float sv[H], av[H];
#pragma unroll
            for (int r = 0; r < H; ++r) {
                int64_t t = tid + (int64_t)(h + r) * NT;
                t = t < T ? t : T - 1;
                sv[r] = row[t];
                av[r] = alpha[t];
            }
#pragma unroll
            for (int r = 0; r < H; ++r) key[h + r] = order_key(sv[r] - av[r]);
        }
    }
    auto live = [&](int r) { return tok(r) < T; };

    const unsigned k = (unsigned)((T * (int64_t)(E - K) + E - 1) / E);  // 1-based ascending rank
    const unsigned r_top = (unsigned)T - k + 1u;                       // the same key's rank from the top
    const int64_t holders = VEC ? (T + 3) / 4 : T;                      // threads holding at least one key
    const unsigned nvalid = (unsigned)(holders < NT ? holders : NT);
    bool done = false;
    unsigned result = 0u;
    if (r_top <= nvalid) {
        unsigned m = 0u;
#pragma unroll
        for (int r = 0; r < R; ++r)
            if (live(r)) m = key[r] > m ? key[r] : m;
        maxima[tid] = m;  // meaningful for tid < nvalid
        if (tid == 0) nlist = 0u;
        __syncthreads();
        if (wave == 0) {
            // 16 high bits suffice: a lower bound of the r-th largest maximum
            const unsigned t = wave_select_reg<NT / 64, 16>(maxima, nvalid, nvalid - r_top + 1u, hist[0]);
            if (lane == 0) tau_s = t;
        }
        __syncthreads();
        const unsigned tau = tau_s;
        // the keys >= tau into the list: counts, a scan over the wave, one
        // LDS atomic per wave for its base
        unsigned c = 0u;
#pragma unroll
        for (int r = 0; r < R; ++r) c += (live(r) && key[r] >= tau) ? 1u : 0u;
        unsigned incl = c;
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
            const unsigned up = __shfl_up(incl, o);
            if (lane >= o) incl += up;
        }
        unsigned base = 0u;
        if (lane == 63) base = atomicAdd(&nlist, incl);
        unsigned pos = __shfl(base, 63) + incl - c;
#pragma unroll
        for (int r = 0; r < R; ++r)
            if (live(r) && key[r] >= tau) {
                if (pos < (unsigned)kQbList) list[pos] = key[r];
                ++pos;
            }
        __syncthreads();
        const unsigned n = nlist;
        if (n <= (unsigned)NT) {
            if (wave == 0) {
                result = wave_select_reg<NT / 64>(list, n, n - r_top + 1u, hist[0]);
                if (lane == 0) write_bias(bias, j, result, rho);
            }
            done = true;
        } else if (n <= (unsigned)kQbList) {
            if (wave == 0) {
                result = wave_select(list, n, n - r_top + 1u, hist[0]);
                if (lane == 0) write_bias(bias, j, result, rho);
            }
            done = true;
        }
    }
    if (!done) {
        // full radix select over the registers
        unsigned kleft = k, prefix = 0u, mask = 0u;
        for (int shift = 24; shift >= 0; shift -= 8) {
            __syncthreads();
            for (int i = tid; i < NW * 256; i += NT) (&hist[0][0])[i] = 0u;
            __syncthreads();
            DigitCounter dc;
#pragma unroll
            for (int r = 0; r < R; ++r)
                if (live(r) && (key[r] & mask) == prefix) dc.add(hist[wave], (key[r] >> shift) & 255u);
            dc.flush(hist[wave]);
            __syncthreads();
            if (wave == 0) pick_digit(hist, kleft, pick);
            __syncthreads();
            prefix |= pick[0] << shift;
            mask |= 255u << shift;
            kleft -= pick[1];
        }
        result = prefix;
        if (tid == 0) write_bias(bias, j, result, rho);
    }
    if (with_stats) {
        int cnt[NQ];
        qb_stats_load<NT>(counts, E, cnt);
        qb_block_stats<NT>(cnt, E, stats);
    }
}

// Any T: the keys are recomputed from global memory in every pass.
__global__ __launch_bounds__(kQbThreads) void qb_update_global_kernel(const float* __restrict__ scores_t,
                                                                      const float* __restrict__ alpha, int64_t T,
                                                                      int E, int K, float rho,
                                                                      float* __restrict__ bias,
                                                                      const int32_t* __restrict__ counts,
                                                                      double* __restrict__ stats) {
    constexpr int NW = kQbThreads / 64;
    constexpr int NQ = (1024 + kQbThreads - 1) / kQbThreads;
    __shared__ unsigned hist[NW][256];
    __shared__ unsigned pick[3];
    const int tid = threadIdx.x;
    const int wave = tid >> 6;
    const int j = blockIdx.x;
    const bool with_stats = counts && j == 0;
    int cnt[NQ];
    if (with_stats) qb_stats_load<kQbThreads>(counts, E, cnt);
    const float* row = scores_t + (int64_t)j * T;
    unsigned kleft = (unsigned)((T * (int64_t)(E - K) + E - 1) / E);
    unsigned prefix = 0u, mask = 0u;
    for (int shift = 24; shift >= 0; shift -= 8) {
        for (int i = tid; i < NW * 256; i += kQbThreads) (&hist[0][0])[i] = 0u;
        __syncthreads();
        DigitCounter dc;
        for (int64_t t = tid; t < T; t += kQbThreads) {
            const unsigned u = order_key(row[t] - alpha[t]);
            if ((u & mask) == prefix) dc.add(hist[wave], (u >> shift) & 255u);
        }
        dc.flush(hist[wave]);
        __syncthreads();
        if (wave == 0) pick_digit(hist, kleft, pick);
        __syncthreads();
        prefix |= pick[0] << shift;
        mask |= 255u << shift;
        kleft -= pick[1];
        __syncthreads();  // pick[] is rewritten by the next pass
    }
    if (tid == 0) write_bias(bias, j, prefix, rho);
    if (with_stats) qb_block_stats<kQbThreads>(cnt, E, stats);
}

template <int NT, int R>
void launch_reg(const float* scores_t, const float* alpha, int64_t T, int E, int K, float rho, float* bias,
                const int32_t* counts, double* stats, hipStream_t stream) {
    // float4 pieces need T % 4 == 0 (16-byte aligned rows) and aligned buffers
    const bool vec = (T % 4 == 0) && ((reinterpret_cast<uintptr_t>(scores_t) | reinterpret_cast<uintptr_t>(alpha)) &
                                      15) == 0;
    if (vec)
        hipLaunchKernelGGL((qb_update_reg_kernel<NT, R, true>), dim3((unsigned)E), dim3(NT), 0, stream, scores_t,
                           alpha, T, E, K, rho, bias, counts, stats);
    else
        hipLaunchKernelGGL((qb_update_reg_kernel<NT, R, false>), dim3((unsigned)E), dim3(NT), 0, stream, scores_t,
                           alpha, T, E, K, rho, bias, counts, stats);
}

}  // namespace

hipError_t launch_qb_update(const float* scores_t, const float* alpha, int64_t T, int E, int K, float rho,
                            float* bias, const int32_t* counts, double* stats, hipStream_t stream) {
    if (T <= 16 * 512)
        launch_reg<512, 16>(scores_t, alpha, T, E, K, rho, bias, counts, stats, stream);
    else if (T <= 32 * 512)
        launch_reg<512, 32>(scores_t, alpha, T, E, K, rho, bias, counts, stats, stream);
    else if (T <= 32 * 1024)
        launch_reg<1024, 32>(scores_t, alpha, T, E, K, rho, bias, counts, stats, stream);
    else
        hipLaunchKernelGGL(qb_update_global_kernel, dim3((unsigned)E), dim3(kQbThreads), 0, stream, scores_t, alpha,
                           T, E, K, rho, bias, counts, stats);
    return hipGetLastError();
}

}  // namespace idb
