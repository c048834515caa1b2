// Selection epilogue shared by the fused router kernels (router.hip) and the
// selection from given scores (select.hip): bias-adjusted Top-K (Eq.
// pid-routing), gate weights from the unbiased scores (Sec. 2.2) and the load
// histogram (Eq. pid-error) for a tile of tokens whose scores sit in LDS.
//
// The scores of TPP tokens at a time are written token-major into LDS; TPT
// adjacent threads then own one token, each every TPT-th block of 16 experts
// (so a wave's LDS reads of the score rows hit distinct banks).  A token's
// threads share one wave, so after step A only wave-level ordering is needed
// between the steps.  Exact for any input:
//   A. the scores into the LDS score matrix (the caller's store_pass; padding
//      experts -inf).
//   B. v = fl32(s + b) into registers; NG <= 32 group maxima per token.
//   C. tau = the K-th largest group maximum, <= the token's K-th largest v;
//      each thread marks its values >= tau in a bitmask and counts them.
//   D. A prefix over the token's threads gives write offsets; the candidates
//      (typically about K + 2) go to an LDS list as 64-bit rank keys.
//   E. Candidate rank = number of list keys above it; ranks < K are the
//      slice's selection, in rank order.
//   F. Tokens whose list would overflow (heavy ties, large K) are resolved by
//      their own wave, one at a time: K rounds of "best key strictly below
//      the previous pick" over the token's LDS score row.
//   G. One slice: gate weights, outputs and an LDS histogram flushed with one
//      atomic per non-zero bin.  Several slices: the slice's K candidates go
//      to the workspace for the slice merge.
// With a.alpha set (Quantile Balancing), K + 1 candidates are kept in steps
// C-G and the biased value of rank K (the cutoff alpha of Eq.
// pid-quantile-def) is written per token; with a.scores_t set, the scores are
// also written expert-major after step A.
// In softmax mode (SM; auxiliary-loss routing, one slice) the LDS matrix holds
// logits and the bias is zero: step C also finds each token's largest logit
// M and Z = sum exp(z - M), the gate weights are exp(z_r - z_top) over their
// sum, and with a.prob_part set the tile's column sums of exp(z - M) / Z go
// out per token tile.
#pragma once

#include "common.h"
#include "internal.h"

namespace idb {
namespace {

constexpr int kCap = 32;      // candidate list capacity per token and slice
constexpr int kShortList = 16;  // lists up to this length are ranked in one unrolled sweep
constexpr float kLog2e = 1.4426950408889634f;

// exp(x) as 2^(x log2 e) with the hardware exp2 (about 1 ulp; exp(-inf) = 0).
__device__ __forceinline__ float exp_fast(float x) { return __builtin_amdgcn_exp2f(x * kLog2e); }
constexpr int kScoreLds = 100000;  // LDS budget of the epilogue's score matrix

// Epilogue layout for NT threads, BT tokens, BE experts per workgroup; the
// contraction's MAIN_LDS bytes of LDS are reused, and the score rows of a pass
// take at most SCORE_LDS bytes.
template <int NT_, int BT_, int BE_, int MAIN_LDS_, int SCORE_LDS = kScoreLds>
struct EpiCfg {
    static constexpr int NT = NT_;
    static constexpr int BT = BT_;
    static constexpr int BE = BE_;
    static constexpr int RS = BE + 4;  // score row stride in floats (odd number of 16-byte units)
    // tokens per pass: the largest of BT, BT/2, BT/4 whose score rows fit
    static constexpr int TPP = (BT * RS * 4 <= SCORE_LDS && BT <= NT) ? BT
                               : ((BT / 2) * RS * 4 <= SCORE_LDS && BT / 2 <= NT) ? BT / 2 : BT / 4;
    static constexpr int NPASS = BT / TPP;
    static constexpr int TPT = NT / TPP;
    static constexpr int VPT = BE / TPT;  // slice columns per thread: every TPT-th 16-column block
    static constexpr int NBL = VPT / 16;  // 16-column blocks per thread
    // group maxima per token: one per 16-column block when that makes 24 to
    // 32 of them (a multiple of 4), else 32
    static constexpr int NG = (TPT * NBL >= 24 && TPT * NBL <= 32 && (TPT * NBL) % 4 == 0) ? TPT * NBL : 32;
    static constexpr int GPT = NG / TPT;  // group maxima per thread
    static constexpr int GSZ = VPT / GPT;
    static constexpr int MW = (VPT + 31) / 32;          // candidate mask words
    static constexpr int NCI = (kCap + TPT - 1) / TPT;  // list entries ranked per thread
    static constexpr int NBIAS = (BE + NT - 1) / NT;    // bias values staged per thread
    static constexpr int GMS = NG + 4;                  // group-maximum row stride (words, 16-byte aligned)
    static constexpr int CNS = TPT + 1;                 // count row stride
    static constexpr int LKS = kCap + 2;                // candidate-key row stride (8-byte keys)
    static constexpr int LSS = kMaxK + 4;               // selection row stride
    static constexpr int OFF_SC = 0;
    static constexpr int OFF_BIAS = OFF_SC + TPP * RS * 4;
    static constexpr int OFF_GM = OFF_BIAS + BE * 4;
    static constexpr int OFF_CNT = OFF_GM + TPP * GMS * 4;
    static constexpr int OFF_LK = (OFF_CNT + TPP * CNS * 4 + 15) / 16 * 16;
    static constexpr int OFF_SI = OFF_LK + TPP * LKS * 8;
    static constexpr int OFF_HIST = OFF_SI + TPP * LSS * 4;
    static constexpr int EPI_LDS = OFF_HIST + 1024 * 4;
    static constexpr int LDS = MAIN_LDS_ > EPI_LDS ? MAIN_LDS_ : EPI_LDS;
    static_assert(NPASS * TPP == BT && TPP % 16 == 0, "passes of whole 16-token groups");
    static_assert(TPT * TPP == NT && TPT <= 16 && 16 % TPT == 0, "a token's threads share one wave");
    static_assert(VPT * TPT == BE && VPT % 16 == 0 && GSZ * GPT == VPT && GPT * TPT == NG, "columns split evenly");
    static_assert(TPP * RS * 4 <= SCORE_LDS, "score rows of a pass fit");
    static_assert(NT % TPP == 0, "whole token rows per thread group");
    static_assert(LDS <= 160 * 1024, "LDS of one workgroup");
};

// Adds a workgroup's LDS histogram into the global counts, one atomic per
// non-zero bin.  Each workgroup starts at a different bin, so workgroups that
// finish together do not queue on the same counter.
__device__ __forceinline__ void flush_hist(const int* hist, int32_t* counts, int E) {
    const int rot = (int)((blockIdx.x * 97u) % (unsigned)E);
    for (int i = threadIdx.x; i < E; i += blockDim.x) {
        int e = i + rot;
        e = e < E ? e : e - E;
        if (hist[e] != 0) atomicAdd(&counts[e], hist[e]);
    }
}

// Loads the slice's bias into registers (issued before the contraction, so
// it arrives meanwhile); the epilogue moves it to LDS.
template <class EC, bool SM = false>
__device__ __forceinline__ void prefetch_bias(const RouterArgs& a, int sbase, float (&breg)[EC::NBIAS]) {
#pragma unroll
    for (int i = 0; i < EC::NBIAS; ++i) {
        const int c = threadIdx.x + EC::NT * i;
        // softmax mode (auxiliary-loss routing) keeps no bias
        breg[i] = (!SM && c < EC::BE && sbase + c < a.E) ? a.bias[sbase + c] : 0.0f;
    }
}

// Start of the epilogue: the slice's bias (from prefetch_bias registers) into
// LDS, the LDS histogram zeroed.  The first pass's barrier orders both.
template <class EC>
__device__ __forceinline__ void epi_begin(unsigned char* smem, const float (&breg)[EC::NBIAS]) {
    float* bias_s = reinterpret_cast<float*>(smem + EC::OFF_BIAS);
    int* hist = reinterpret_cast<int*>(smem + EC::OFF_HIST);
#pragma unroll
    for (int i = 0; i < EC::NBIAS; ++i) {
        const int c = threadIdx.x + EC::NT * i;
        if (c < EC::BE) bias_s[c] = breg[i];
    }
    for (int e = threadIdx.x; e < 1024; e += EC::NT) hist[e] = 0;
}

// Steps A-G for BT tokens from tok0 of one slice.  store_pass(pass, sc)
// writes the scores of tokens [pass*TPP, (pass+1)*TPP) of the tile into rows
// 0..TPP-1 of the LDS score matrix sc (padding experts: -inf).  One slice:
// outputs and the LDS histogram; several: the slice's candidates.  Ends with a
// barrier.
template <class EC, bool SM, class StoreFn>
__device__ __forceinline__ void epi_tile(const RouterArgs& a, int NS, int slice, int64_t tok0, unsigned char* smem,
                                         StoreFn&& store_pass) {
    using C = EC;
    constexpr int WAVES = C::NT / 64;
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int64_t T = a.T;
    const int E = a.E;
    const int K = a.K;        // experts selected per token
    const int KL = a.alpha ? K + 1 : K;  // candidates kept per token (the (K+1)-th gives the cutoff)
    const int sbase = slice * C::BE;
    float* sc = reinterpret_cast<float*>(smem + C::OFF_SC);
    float* bias_s = reinterpret_cast<float*>(smem + C::OFF_BIAS);
    float* gm = reinterpret_cast<float*>(smem + C::OFF_GM);
    int* cnt = reinterpret_cast<int*>(smem + C::OFF_CNT);
    unsigned long long* lk = reinterpret_cast<unsigned long long*>(smem + C::OFF_LK);
    int* si = reinterpret_cast<int*>(smem + C::OFF_SI);
    int* hist = reinterpret_cast<int*>(smem + C::OFF_HIST);

    const int tl = tid / C::TPT, q = tid % C::TPT;  // token of the pass and part, in steps B-G
    // This thread's value j sits in slice column col(j) = 16 (q + TPT (j/16)) + j%16.
    auto col_of = [&](int j) { return 16 * (q + C::TPT * (j >> 4)) + (j & 15); };
    unsigned valid[C::MW];  // bit j: column j is a real expert
    {
#pragma unroll
        for (int w = 0; w < C::MW; ++w) valid[w] = 0u;
#pragma unroll
        for (int m = 0; m < C::NBL; ++m) {
            const int nreal = E - sbase - 16 * (q + C::TPT * m);  // may be <= 0 or >= 16
            const unsigned bits = nreal >= 16 ? 0xffffu : (nreal <= 0 ? 0u : ((1u << nreal) - 1u));
            valid[m >> 1] |= bits << (16 * (m & 1));
        }
    }

    float pacc[C::NBIAS];  // softmax column sums of the tile (prob_part)
#pragma unroll
    for (int i = 0; i < C::NBIAS; ++i) pacc[i] = 0.0f;

#pragma unroll
    for (int pass = 0; pass < C::NPASS; ++pass) {
        // A. scores of the pass's tokens into the LDS score matrix
        store_pass(pass, sc);
        __syncthreads();

        // The scores also go out expert-major, [E][T] (Quantile Balancing's
        // input): a thread takes a token row and every (NT/TPP)-th group of 4
        // experts, so each store instruction covers TPP consecutive tokens.
        if (a.scores_t) {
            const int row = tid % C::TPP;
            const int64_t tok = tok0 + pass * C::TPP + row;
            if (tok < T) {
                for (int c4 = 4 * (tid / C::TPP); c4 < C::BE; c4 += 4 * (C::NT / C::TPP)) {
                    const int e = sbase + c4;
                    if (e < E) {
                        const float4 v4 = *reinterpret_cast<const float4*>(sc + row * C::RS + c4);
                        a.scores_t[(int64_t)e * T + tok] = v4.x;
                        if (e + 1 < E) a.scores_t[(int64_t)(e + 1) * T + tok] = v4.y;
                        if (e + 2 < E) a.scores_t[(int64_t)(e + 2) * T + tok] = v4.z;
                        if (e + 3 < E) a.scores_t[(int64_t)(e + 3) * T + tok] = v4.w;
                    }
                }
            }
        }

        // B. biased values of this thread's columns; group maxima
        float v[C::VPT];
#pragma unroll
        for (int m = 0; m < C::NBL; ++m)
#pragma unroll
            for (int i4 = 0; i4 < 4; ++i4) {
                const int col = 16 * (q + C::TPT * m) + 4 * i4;
                const float4 s4 = *reinterpret_cast<const float4*>(sc + tl * C::RS + col);
                const float4 b4 = *reinterpret_cast<const float4*>(bias_s + col);
                const int j = 16 * m + 4 * i4;
                v[j + 0] = s4.x + b4.x;
                v[j + 1] = s4.y + b4.y;
                v[j + 2] = s4.z + b4.z;
                v[j + 3] = s4.w + b4.w;
            }
        float own[C::GPT];
#pragma unroll
        for (int g = 0; g < C::GPT; ++g) {
            float mx = -INFINITY;
#pragma unroll
            for (int j = 0; j < C::GSZ; ++j) mx = fmaxf(mx, v[g * C::GSZ + j]);
            own[g] = mx;
            gm[tl * C::GMS + q * C::GPT + g] = mx;
        }
        wave_sync();

        // C. threshold; candidate masks and counts
        // tau = the K-th largest of the token's NG group maxima, i.e. the
        // largest maximum m with #{maxima >= m} >= K (for K > NG no maximum
        // qualifies: tau = -inf and the token takes step F): each thread
        // tests its own maxima against all NG, a max over the token's lanes
        // combines them.
        float tau = -INFINITY;
        float zmax = 0.0f, zsum = 0.0f;  // softmax mode
        {
            float g[C::NG];
#pragma unroll
            for (int i4 = 0; i4 < C::NG / 4; ++i4) {
                const float4 t4 = *reinterpret_cast<const float4*>(gm + tl * C::GMS + 4 * i4);
                g[4 * i4 + 0] = t4.x;
                g[4 * i4 + 1] = t4.y;
                g[4 * i4 + 2] = t4.z;
                g[4 * i4 + 3] = t4.w;
            }
#pragma unroll
            for (int i = 0; i < C::GPT; ++i) {
                int ge = 0;
#pragma unroll
                for (int j = 0; j < C::NG; ++j) ge += (g[j] >= own[i]) ? 1 : 0;
                if (ge >= KL) tau = fmaxf(tau, own[i]);
            }
#pragma unroll
            for (int o = 1; o < C::TPT; o <<= 1) tau = fmaxf(tau, __shfl_xor(tau, o));
            if constexpr (SM) {
                // the token's largest logit and Z = sum exp(z - M): each
                // thread over its columns in order (padding: exp(-inf) = 0),
                // then a butterfly over the token's threads (every lane ends
                // with the same bits: fp32 addition commutes)
                zmax = g[0];
#pragma unroll
                for (int j = 1; j < C::NG; ++j) zmax = fmaxf(zmax, g[j]);
#pragma unroll
                for (int j = 0; j < C::VPT; ++j) zsum = zsum + exp_fast(v[j] - zmax);
#pragma unroll
                for (int o = 1; o < C::TPT; o <<= 1) zsum = zsum + __shfl_xor(zsum, o);
            }
        }
        // Bit j: v_j >= tau, an IEEE comparison (-0 == +0; every real value
        // reaches tau = -inf).  Padding columns are masked out.
        unsigned msk[C::MW];
#pragma unroll
        for (int w = 0; w < C::MW; ++w) msk[w] = 0u;
#pragma unroll
        for (int j = 0; j < C::VPT; ++j) msk[j / 32] |= (v[j] >= tau ? 1u : 0u) << (j % 32);
        int mine_n = 0;
#pragma unroll
        for (int w = 0; w < C::MW; ++w) {
            msk[w] &= valid[w];
            mine_n += __builtin_popcount(msk[w]);
        }
        cnt[tl * C::CNS + q] = mine_n;
        wave_sync();

        // D. write offsets; candidate keys into the token's list
        int off = 0, n = 0;
#pragma unroll
        for (int o = 0; o < C::TPT; ++o) {
            const int m = cnt[tl * C::CNS + o];
            off += (o < q) ? m : 0;
            n += m;
        }
        if (SM && q == 0) {
            // the group maxima are no longer read: the row keeps M and 1/Z
            gm[tl * C::GMS + 0] = zmax;
            gm[tl * C::GMS + 1] = 1.0f / zsum;
        }
        const bool listed = n <= kCap;
        if (listed) {
#pragma unroll
            for (int w = 0; w < C::MW; ++w) {
                unsigned m = msk[w];
                while (m) {
                    const int col = col_of(w * 32 + __builtin_ctz(m));
                    m &= m - 1u;
                    lk[tl * C::LKS + off] = rank_key(sc[tl * C::RS + col] + bias_s[col], sbase + col);
                    ++off;
                }
            }
            // short lists are padded with key 0 (below every key) to kShortList
            for (int c = n + q; c < kShortList; c += C::TPT) lk[tl * C::LKS + c] = 0ull;
        }
        wave_sync();

        // E. ranks of the listed candidates: thread q ranks entries q, q+TPT, ...
        // against the n list keys, reading each list key once.  When no list
        // of the wave is longer than kShortList, one unrolled sweep over the
        // padded kShortList keys (the padding ranks below every entry).
        if (listed && __ballot(n > kShortList) == 0) {
            constexpr int NSH = (kShortList + C::TPT - 1) / C::TPT;
            unsigned long long mine[NSH];
            int rank[NSH];
#pragma unroll
            for (int i = 0; i < NSH; ++i) {
                const int c = q + C::TPT * i;
                mine[i] = c < kShortList ? lk[tl * C::LKS + c] : 0ull;
                rank[i] = 0;
            }
#pragma unroll
            for (int o = 0; o < kShortList; ++o) {
                const unsigned long long ko = lk[tl * C::LKS + o];
#pragma unroll
                for (int i = 0; i < NSH; ++i) rank[i] += (ko > mine[i]) ? 1 : 0;
            }
#pragma unroll
            for (int i = 0; i < NSH; ++i)
                if (q + C::TPT * i < n && rank[i] < KL) si[tl * C::LSS + rank[i]] = (int)~(unsigned)mine[i];
        } else if (listed) {
            unsigned long long mine[C::NCI];
            int rank[C::NCI];
#pragma unroll
            for (int i = 0; i < C::NCI; ++i) {
                const int c = q + C::TPT * i;
                mine[i] = c < n ? lk[tl * C::LKS + c] : ~0ull;  // ~0: beyond the list, never written
                rank[i] = 0;
            }
#pragma unroll 4
            for (int o = 0; o < n; ++o) {
                const unsigned long long ko = lk[tl * C::LKS + o];
#pragma unroll
                for (int i = 0; i < C::NCI; ++i) rank[i] += (ko > mine[i]) ? 1 : 0;
            }
#pragma unroll
            for (int i = 0; i < C::NCI; ++i)
                if (q + C::TPT * i < n && rank[i] < KL) si[tl * C::LSS + rank[i]] = (int)~(unsigned)mine[i];
        }

        // F. this wave's overflowing tokens, one at a time by the whole wave
        {
            unsigned long long lead = __ballot(!listed && q == 0);  // wave-uniform
            while (lead) {
                const int t = (wave * 64 + __builtin_ctzll(lead)) / C::TPT;
                lead &= lead - 1ull;
                unsigned long long prev = ~0ull;
                for (int r = 0; r < KL; ++r) {
                    unsigned long long best = 0ull;
                    for (int c = lane; c < C::BE; c += 64) {
                        if (sbase + c < E) {
                            const unsigned long long kk = rank_key(sc[t * C::RS + c] + bias_s[c], sbase + c);
                            if (kk < prev && kk > best) best = kk;
                        }
                    }
#pragma unroll
                    for (int o = 32; o >= 1; o >>= 1) {
                        const unsigned lo = __shfl_xor((unsigned)best, o);
                        const unsigned hi = __shfl_xor((unsigned)(best >> 32), o);
                        const unsigned long long other = ((unsigned long long)hi << 32) | lo;
                        best = other > best ? other : best;
                    }
                    prev = best;
                    if (lane == 0) si[t * C::LSS + r] = (int)~(unsigned)best;
                }
            }
        }
        wave_sync();

        // G. outputs of the pass's tokens (selected scores read back from the
        // token's LDS score row)
        {
            const int64_t tok = tok0 + pass * C::TPP + tl;
            if (tok < T) {
                if (NS > 1) {
                    const int64_t base = (tok * NS + slice) * KL;
                    for (int r = q; r < KL; r += C::TPT) {
                        const int e = si[tl * C::LSS + r];
                        const float s = sc[tl * C::RS + (e - sbase)];
                        a.cand_v[base + r] = s + bias_s[e - sbase];
                        a.cand_s[base + r] = s;
                        a.cand_i[base + r] = e;
                    }
                } else {
                    if constexpr (SM) {
                        // gate weights: the selected probabilities
                        // renormalised, exp(z_r - z_top) over their fp32 sum
                        // in rank order (the first term is exactly 1)
                        const float ztop = sc[tl * C::RS + (si[tl * C::LSS + 0] - sbase)];
                        float den = 0.0f;
#pragma unroll 8
                        for (int r = 0; r < K; ++r)
                            den = den + exp_fast(sc[tl * C::RS + (si[tl * C::LSS + r] - sbase)] - ztop);
                        for (int r = q; r < K; r += C::TPT) {
                            const int e = si[tl * C::LSS + r];
                            a.idx[tok * K + r] = e;
                            a.w[tok * K + r] = exp_fast(sc[tl * C::RS + (e - sbase)] - ztop) / den;
                            atomicAdd(&hist[e], 1);
                        }
                    } else {
                    // gate weights: den is the fp32 sum of the selected
                    // unbiased scores in rank order
                    float den = 0.0f;
#pragma unroll 8
                    for (int r = 0; r < K; ++r) den = den + sc[tl * C::RS + (si[tl * C::LSS + r] - sbase)];
                    for (int r = q; r < K; r += C::TPT) {
                        const int e = si[tl * C::LSS + r];
                        const float s = sc[tl * C::RS + (e - sbase)];
                        a.idx[tok * K + r] = e;
                        a.w[tok * K + r] = (den == 0.0f) ? 1.0f / (float)K : s / den;
                        atomicAdd(&hist[e], 1);
                    }
                    }
                    if (a.alpha && q == 0) {
                        // cutoff: the biased value of rank K
                        const int e = si[tl * C::LSS + K];
                        a.alpha[tok] = (sc[tl * C::RS + (e - sbase)] + bias_s[e - sbase]) + 0.0f;
                    }
                }
            }
        }
        if (SM && NS == 1 && a.prob_part) {
            // column sums of the pass's probabilities p = exp(z - M) / Z,
            // tokens in order; a thread owns columns tid, tid + NT, ...
            // (every token's M and 1/Z row is complete after the barrier)
            __syncthreads();
            const int64_t left = T - (tok0 + pass * C::TPP);
            const int rows = left < C::TPP ? (int)left : C::TPP;
#pragma unroll
            for (int i = 0; i < C::NBIAS; ++i) {
                const int c = tid + C::NT * i;
                if (c < C::BE && sbase + c < E) {
                    float s = 0.0f;
                    for (int row = 0; row < rows; ++row)
                        s = s + exp_fast(sc[row * C::RS + c] - gm[row * C::GMS + 0]) * gm[row * C::GMS + 1];
                    pacc[i] = pacc[i] + s;
                }
            }
        }
        __syncthreads();
    }
    if (SM && NS == 1 && a.prob_part) {
        float* out = a.prob_part + (tok0 / C::BT) * (int64_t)E + sbase;
#pragma unroll
        for (int i = 0; i < C::NBIAS; ++i) {
            const int c = tid + C::NT * i;
            if (c < C::BE && sbase + c < E) out[c] = pacc[i];
        }
    }
}

// The whole epilogue of one workgroup tile (the fused router kernels); SM:
// the softmax mode of auxiliary-loss routing.
template <class EC, bool SM, class StoreFn>
__device__ __forceinline__ void select_epilogue(const RouterArgs& a, int NS, int slice, int64_t tok0,
                                                unsigned char* smem, const float (&breg)[EC::NBIAS],
                                                StoreFn&& store_pass) {
    epi_begin<EC>(smem, breg);
    epi_tile<EC, SM>(a, NS, slice, tok0, smem, store_pass);
    if (NS != 1) return;
    const int* hist = reinterpret_cast<const int*>(smem + EC::OFF_HIST);
    if (SM && a.cnt_part) {
        // the tile's counts as one row (summed in order by the statistics kernel)
        int32_t* row = a.cnt_part + (tok0 / EC::BT) * (int64_t)a.E;
        for (int e = threadIdx.x; e < a.E; e += EC::NT) row[e] = hist[e];
    } else {
        flush_hist(hist, a.counts, a.E);
    }
}

}  // namespace
}  // namespace idb
