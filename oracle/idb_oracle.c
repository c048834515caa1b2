/*
 * CPU oracle for the ID Balancing router step and bias controller.
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the plain, slow, obviously correct
 * reference that the GPU library is checked against.  Only the test suite,
 * the smoke check and the benchmark's CPU-baseline leg may load it.  It shares
 * no source, header, helper or table with the GPU library.
 *
 * What it computes, and the passage of "ID Balancing: Stable Training of
 * Extremely Sparse MoE via PID-Based Load Control" each step follows:
 *
 *   R1  logits z = W_r x                                   (Sec. 2.2)
 *   R2  scores s_i = sigma(z_i), logistic sigmoid          (Sec. 2.2; Sec. 4.3 scores
 *                                                            loss-free routers with the
 *                                                            sigmoid plus the bias)
 *   R3  biased score v_i = s_i + b_i, one fp32 addition    (Eq. pid-routing)
 *   R4  T(x) = the K largest v_i                           (Eq. pid-routing)
 *   R5  gate weights: selected s_i normalised, no bias     (Sec. 2.2, text after
 *                                                            Eq. pid-routing)
 *   R6  n_i = number of tokens assigned to expert i        (Eq. pid-error; Alg. 1)
 *   C1..C7 the ID bias update                              (Alg. 1; Eq. rapid-integral,
 *                                                            rapid-delta, rapid-gate,
 *                                                            rapid-update)
 *   SIGN mode: DeepSeek's fixed-step integral rule         (Eq. pid-deepseek)
 *   S1  MaxVio / MinVio                                    (Sec. 4.1, Eq. vio)
 *   D1..D4 controller diagnostics: active-gate fraction,  (Sec. 3 text after Eq.
 *          busiest-10% share, inactive-expert ratio, mean    rapid-gate and its figure;
 *          absolute bias change                              Sec. 4.3; Sec. 3 bias drift)
 *   H1, H2 top-K and full-pool score entropy               (Sec. 4.3)
 *   H3  full-pool entropy of the softmax router scores     (Sec. 4.3)
 *   Q1..Q4 Quantile Balancing's target bias, with the EMA   (Eq. pid-quantile,
 *          variant used as a diagnostic                      Eq. pid-quantile-def; Sec. 3,
 *                                                            EMA smoothing of the target)
 *   X1..X5 auxiliary-loss balancing, forward statistics:   (Eq. pid-auxloss)
 *          softmax router probabilities, Top-K, assigned
 *          fractions f_i, mean probabilities P_i, the loss
 *
 * Readings of points the paper leaves open (each is listed in the design
 * notes of the repository):
 *   - Top-K ties go to the lowest expert index; the selected experts are
 *     reported in rank order (v descending, index ascending).
 *   - IEEE comparison of v, so -0 == +0.
 *   - gate weight w_r = s_r / den with den the fp32 sum of the selected
 *     unbiased scores taken in rank order; den == 0 gives w = 1/K.
 *   - e_i = (nbar - n_i)/nbar evaluated as one correctly rounded fp64 division
 *     of the exact integer numerator S - E*n_i by S, then rounded to fp32.
 *   - the gate is the sign test (e_prev > 0 and de > 0) or (e_prev < 0 and
 *     de < 0), i.e. the truth value of e_prev * de > 0 without an fp32 product.
 *   - b + K_i e + K_d g de is evaluated left to right in fp32, each product and
 *     sum rounded, the derivative added only when the gate is open, no FMA.
 *   - the centering mean uses a fixed pairwise tree: pad b~ with +0 to the next
 *     power of two P >= E, then a_j <- a_j + a_{j+h} for h = P/2, ..., 1.
 *   - an empty batch (sum of counts == 0) leaves the state untouched and
 *     reports status 3; a negative count reports status 1.
 *   - Diagnostics of one update: the active-gate fraction is #{g_i = 1} / E;
 *     the busiest-10% share is the sum of the m = ceil(E / 10) largest counts
 *     over S; the inactive-expert ratio is #{n_i = 0} / E; the mean absolute
 *     bias change is (1/E) sum |fl32(b_new - b_old)| summed in fp64 over the
 *     fixed pairwise tree (padded with +0 to a power of two); each ratio is one
 *     fp64 division.  All four are NaN when the update does not run.
 *   - Entropies in nats with natural logarithms in fp64: H_topK = -sum_r w_r
 *     log w_r over a token's gate weights (0 log 0 = 0); H_full = -sum_e p_e
 *     log p_e with p_e = max(s_e + b_e, 0) / sum of those (the biased sigmoid
 *     score clamped at zero, normalised; H_full = 0 when the sum is 0); both
 *     averaged over the tokens in fp64, tokens in order.
 *   - Quantile Balancing: the cutoff alpha_i is the (K+1)-th largest biased
 *     score fl32(s + b) of token i; margins are fl32(s_ij - alpha_i) with -0
 *     read as +0; quantile_{1-K/E} over the m tokens of a batch is the
 *     inverted empirical CDF, i.e. the k-th smallest margin with
 *     k = ceil(m (E - K) / E) computed in exact integers; the target is its
 *     negation.  The EMA variant is fl32(fl32(rho b) + fl32(fl32(1 - rho) Q)),
 *     and rho == 0 is the plain target b = Q.
 *   - Auxiliary-loss routers keep no bias: p = softmax(z) over all E experts
 *     in fp64 (max subtracted first); T(x) = the K largest p, ranked on the
 *     logits rounded to fp32 (softmax preserves their order; fp32 is the
 *     precision the GPU decides in) with ties to the lowest index; gate
 *     weights w_r = p_r / sum of the selected p in rank order, in fp64, then
 *     fp32; f_i = n_i / T; P_i = (1/T) sum over tokens of p_i, tokens in
 *     order; the loss alpha * sum_i f_i P_i, experts in order.
 *
 * Build: gcc -O2 -ffp-contract=off -fopenmp -shared -fPIC (never -ffast-math:
 * the fp32 steps must round exactly as written).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <time.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define ORACLE_DTYPE_BF16 0
#define ORACLE_DTYPE_F32 1

#define ORACLE_MODE_ERROR 0 /* ID: integral step K_i * e      */
#define ORACLE_MODE_SIGN 1  /* DeepSeek: integral step K_i * sign(e) */

#define ORACLE_STATUS_OK 0
#define ORACLE_STATUS_INVALID 1
#define ORACLE_STATUS_EMPTY 3

int oracle_num_threads(void) {
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* Threads of the following OpenMP loops (timing a single-thread rate). */
void oracle_set_num_threads(int n) {
#ifdef _OPENMP
    omp_set_num_threads(n);
#else
    (void)n;
#endif
}

/* Exact widening of one input element to double.  bf16 is the upper half of
 * an IEEE binary32, so shifting its 16 bits up gives the same value. */
static double load_elem(const void* base, int dtype, int64_t i) {
    if (dtype == ORACLE_DTYPE_BF16) {
        uint32_t bits = ((uint32_t)((const uint16_t*)base)[i]) << 16;
        float f;
        memcpy(&f, &bits, sizeof f);
        return (double)f;
    }
    return (double)((const float*)base)[i];
}

/* R1 for one token: z_i = sum_k x_k W_ik, products and sum in double,
 * k ascending.  x is [T][d] row-major, W is [E][d] row-major. */
static double logit(const void* x, const void* W, int dtype, int64_t t, int32_t d, int32_t i) {
    double acc = 0.0;
    for (int32_t k = 0; k < d; ++k) {
        double xv = load_elem(x, dtype, t * (int64_t)d + k);
        double wv = load_elem(W, dtype, (int64_t)i * d + k);
        acc = acc + xv * wv;
    }
    return acc;
}

/* R2: logistic sigmoid in double, rounded once to fp32. */
static float sigmoid_ref(double z) {
    return (float)(1.0 / (1.0 + exp(-z)));
}

/* R1 (+ R2) for the listed rows (all rows when rows == NULL).
 * z_out (nullable) gets [nrows][E] doubles; s_out (nullable) gets fp32 scores. */
void oracle_router_scores(const void* x, const void* W, int dtype, int64_t T, int32_t d, int32_t E,
                          const int64_t* rows, int64_t nrows, double* z_out, float* s_out) {
    if (rows == NULL) nrows = T;
#pragma omp parallel for schedule(dynamic, 4)
    for (int64_t r = 0; r < nrows; ++r) {
        int64_t t = rows ? rows[r] : r;
        for (int32_t i = 0; i < E; ++i) {
            double z = logit(x, W, dtype, t, d, i);
            if (z_out) z_out[r * E + i] = z;
            if (s_out) s_out[r * E + i] = sigmoid_ref(z);
        }
    }
}

/* Strict total order of Eq. pid-routing with the lowest-index tie-break:
 * does (va, ia) rank above (vb, ib)?  IEEE comparison, so -0 == +0. */
static int ranks_above(float va, int32_t ia, float vb, int32_t ib) {
    if (va > vb) return 1;
    if (va < vb) return 0;
    return ia < ib;
}

/* R3-R5 for one token: K passes of "best expert not yet taken". */
static void select_token(const float* s, const float* bias, int32_t E, int32_t K, unsigned char* taken,
                         int32_t* idx, float* w) {
    memset(taken, 0, (size_t)E);
    for (int32_t r = 0; r < K; ++r) {
        int32_t best = -1;
        float best_v = 0.0f;
        for (int32_t i = 0; i < E; ++i) {
            if (taken[i]) continue;
            float v = s[i] + bias[i]; /* R3: exactly one fp32 addition */
            if (best < 0 || ranks_above(v, i, best_v, best)) {
                best = i;
                best_v = v;
            }
        }
        taken[best] = 1;
        idx[r] = best;
    }
    /* R5: weights from the unbiased scores, normalised over the selected set. */
    float den = 0.0f;
    for (int32_t r = 0; r < K; ++r) den = den + s[idx[r]];
    for (int32_t r = 0; r < K; ++r) w[r] = (den == 0.0f) ? 1.0f / (float)K : s[idx[r]] / den;
}

/* R3-R6 given fp32 scores s [T][E] and bias [E].  idx, w are [T][K] in rank
 * order; counts [E] is zeroed first unless accumulate != 0. */
void oracle_select(const float* s, const float* bias, int64_t T, int32_t E, int32_t K, int32_t* idx, float* w,
                   int32_t* counts, int accumulate) {
#pragma omp parallel
    {
        unsigned char* taken = (unsigned char*)malloc((size_t)E);
#pragma omp for schedule(static)
        for (int64_t t = 0; t < T; ++t)
            select_token(s + t * (int64_t)E, bias, E, K, taken, idx + t * (int64_t)K, w + t * (int64_t)K);
        free(taken);
    }
    if (!accumulate)
        for (int32_t i = 0; i < E; ++i) counts[i] = 0;
    for (int64_t t = 0; t < T; ++t)
        for (int32_t r = 0; r < K; ++r) counts[idx[t * (int64_t)K + r]] += 1; /* R6 */
}

/* R1-R6 in one call: the whole router step for T tokens (used for timing the
 * CPU baseline and for free-running closed loops).  s_out is nullable. */
void oracle_router(const void* x, const void* W, int dtype, const float* bias, int64_t T, int32_t d, int32_t E,
                   int32_t K, int32_t* idx, float* w, int32_t* counts, int accumulate, float* s_out) {
#pragma omp parallel
    {
        float* s = (float*)malloc(sizeof(float) * (size_t)E);
        unsigned char* taken = (unsigned char*)malloc((size_t)E);
#pragma omp for schedule(dynamic, 4)
        for (int64_t t = 0; t < T; ++t) {
            for (int32_t i = 0; i < E; ++i) s[i] = sigmoid_ref(logit(x, W, dtype, t, d, i));
            if (s_out) memcpy(s_out + t * (int64_t)E, s, sizeof(float) * (size_t)E);
            select_token(s, bias, E, K, taken, idx + t * (int64_t)K, w + t * (int64_t)K);
        }
        free(taken);
        free(s);
    }
    if (!accumulate)
        for (int32_t i = 0; i < E; ++i) counts[i] = 0;
    for (int64_t t = 0; t < T; ++t)
        for (int32_t r = 0; r < K; ++r) counts[idx[t * (int64_t)K + r]] += 1;
}

/* Sign with sign(0) = 0 (Eq. pid-deepseek applies it elementwise). */
static float sign_of(float e) {
    if (e > 0.0f) return 1.0f;
    if (e < 0.0f) return -1.0f;
    return 0.0f;
}

/* Fixed pairwise tree sum used by the centering step. */
static float tree_sum(const float* v, int32_t E) {
    int32_t P = 1;
    while (P < E) P *= 2;
    float* a = (float*)malloc(sizeof(float) * (size_t)P);
    for (int32_t j = 0; j < P; ++j) a[j] = (j < E) ? v[j] : 0.0f;
    for (int32_t h = P / 2; h >= 1; h /= 2)
        for (int32_t j = 0; j < h; ++j) a[j] = a[j] + a[j + h];
    float sum = a[0];
    free(a);
    return sum;
}

/* One controller call (Alg. 1, one iteration, one layer).
 * State (bias, e_prev, step) is updated in place; returns and stores status. */
int oracle_controller(const int32_t* counts, int32_t E, float Ki, float Kd, int mode, int center, float* bias,
                      float* e_prev, int64_t* step, int32_t* status) {
    /* C1: total assignments S = E * nbar (Eq. pid-error needs S > 0). */
    int64_t S = 0;
    for (int32_t i = 0; i < E; ++i) {
        if (counts[i] < 0) {
            *status = ORACLE_STATUS_INVALID;
            return *status;
        }
        S += counts[i];
    }
    if (S == 0) {
        *status = ORACLE_STATUS_EMPTY;
        return *status;
    }
    float* bt = (float*)malloc(sizeof(float) * (size_t)E);
    float* e = (float*)malloc(sizeof(float) * (size_t)E);
    for (int32_t i = 0; i < E; ++i) {
        /* C2: e_i = (nbar - n_i) / nbar = (S - E n_i) / S (Eq. pid-error). */
        int64_t num = S - (int64_t)E * (int64_t)counts[i];
        e[i] = (float)((double)num / (double)S);
        /* C3: change of error (Eq. rapid-delta); e_prev starts at 0. */
        float de = e[i] - e_prev[i];
        /* C4: worsening gate (Eq. rapid-gate). */
        int g = (e_prev[i] > 0.0f && de > 0.0f) || (e_prev[i] < 0.0f && de < 0.0f);
        /* C5: integral step (Eq. rapid-integral, or Eq. pid-deepseek in SIGN
         * mode) then the gated derivative step (Eq. rapid-update). */
        float u = (mode == ORACLE_MODE_SIGN) ? Ki * sign_of(e[i]) : Ki * e[i];
        float b = bias[i] + u;
        if (g) {
            float dterm = Kd * de;
            b = b + dterm;
        }
        bt[i] = b;
    }
    /* C6: subtract the mean of b~ (second line of Eq. rapid-update). */
    if (center) {
        float m = tree_sum(bt, E) / (float)E;
        for (int32_t i = 0; i < E; ++i) bias[i] = bt[i] - m;
    } else {
        for (int32_t i = 0; i < E; ++i) bias[i] = bt[i];
    }
    /* C7 */
    for (int32_t i = 0; i < E; ++i) e_prev[i] = e[i];
    *step += 1;
    *status = ORACLE_STATUS_OK;
    free(e);
    free(bt);
    return *status;
}

static int cmp_int_desc(const void* a, const void* b) {
    int32_t x = *(const int32_t*)a, y = *(const int32_t*)b;
    return (x < y) - (x > y);
}

/* One controller call (as oracle_controller) plus its diagnostics D1-D4:
 * diag[0] active-gate fraction (Eq. rapid-gate; Sec. 3 reports its
 * trajectory), diag[1] share of the assignments on the busiest 10% of
 * experts, diag[2] inactive-expert ratio (Sec. 4.3), diag[3] mean absolute
 * bias change of this update.  NaN x 4 when the update does not run. */
int oracle_controller_diag(const int32_t* counts, int32_t E, float Ki, float Kd, int mode, int center, float* bias,
                           float* e_prev, int64_t* step, int32_t* status, double* diag) {
    float* b_old = (float*)malloc(sizeof(float) * (size_t)E);
    float* ep_old = (float*)malloc(sizeof(float) * (size_t)E);
    memcpy(b_old, bias, sizeof(float) * (size_t)E);
    memcpy(ep_old, e_prev, sizeof(float) * (size_t)E);
    int st = oracle_controller(counts, E, Ki, Kd, mode, center, bias, e_prev, step, status);
    if (st != ORACLE_STATUS_OK) {
        for (int q = 0; q < 4; ++q) diag[q] = NAN;
        free(b_old);
        free(ep_old);
        return st;
    }
    int64_t S = 0;
    int32_t gates = 0, zeros = 0;
    for (int32_t i = 0; i < E; ++i) S += counts[i];
    for (int32_t i = 0; i < E; ++i) {
        /* D1: the gate of this update, from the error it used (C2-C4) */
        int64_t num = S - (int64_t)E * (int64_t)counts[i];
        float e = (float)((double)num / (double)S);
        float de = e - ep_old[i];
        gates += (ep_old[i] > 0.0f && de > 0.0f) || (ep_old[i] < 0.0f && de < 0.0f);
        zeros += counts[i] == 0; /* D3 */
    }
    /* D2: the m = ceil(E / 10) largest counts */
    int32_t* sorted = (int32_t*)malloc(sizeof(int32_t) * (size_t)E);
    memcpy(sorted, counts, sizeof(int32_t) * (size_t)E);
    qsort(sorted, (size_t)E, sizeof(int32_t), cmp_int_desc);
    const int32_t m = (E + 9) / 10;
    int64_t top = 0;
    for (int32_t i = 0; i < m; ++i) top += sorted[i];
    /* D4: mean |b_new - b_old|, fp64 pairwise tree */
    int32_t P = 1;
    while (P < E) P *= 2;
    double* a = (double*)malloc(sizeof(double) * (size_t)P);
    for (int32_t j = 0; j < P; ++j) a[j] = (j < E) ? (double)fabsf(bias[j] - b_old[j]) : 0.0;
    for (int32_t h = P / 2; h >= 1; h /= 2)
        for (int32_t j = 0; j < h; ++j) a[j] = a[j] + a[j + h];
    diag[0] = (double)gates / (double)E;
    diag[1] = (double)top / (double)S;
    diag[2] = (double)zeros / (double)E;
    diag[3] = a[0] / (double)E;
    free(a);
    free(sorted);
    free(b_old);
    free(ep_old);
    return st;
}

/* H1: mean over T tokens of H_topK = -sum_r w_r log w_r (nats), w [T][K]. */
double oracle_topk_entropy(const float* w, int64_t T, int32_t K) {
    double acc = 0.0;
    for (int64_t t = 0; t < T; ++t) {
        double h = 0.0;
        for (int32_t r = 0; r < K; ++r) {
            double x = (double)w[t * (int64_t)K + r];
            if (x > 0.0) h -= x * log(x);
        }
        acc += h;
    }
    return acc / (double)T;
}

/* H2: mean over T tokens of H_full = -sum_e p_e log p_e, p_e = c_e / sum c,
 * c_e = max(fl32(s_e + b_e), 0) (the clamped biased sigmoid score). */
double oracle_full_entropy(const float* s, const float* bias, int64_t T, int32_t E) {
    double acc = 0.0;
    for (int64_t t = 0; t < T; ++t) {
        double C = 0.0;
        for (int32_t e = 0; e < E; ++e) {
            float v = s[t * (int64_t)E + e] + bias[e];
            if (v > 0.0f) C += (double)v;
        }
        double h = 0.0;
        if (C > 0.0)
            for (int32_t e = 0; e < E; ++e) {
                float v = s[t * (int64_t)E + e] + bias[e];
                if (v > 0.0f) {
                    double p = (double)v / C;
                    h -= p * log(p);
                }
            }
        acc += h;
    }
    return acc / (double)T;
}

/* H3: mean over T tokens of H_full for the auxiliary-loss router, whose
 * selection scores are the softmax probabilities over the router logits
 * (Sec. 4.3): p_e = exp(z_e - M) / sum_e' exp(z_e' - M) with M the token's
 * largest logit, H_full = -sum_e p_e log p_e (0 log 0 = 0), all in fp64 from
 * the fp32 logits z [T][E]. */
double oracle_softmax_entropy(const float* z, int64_t T, int32_t E) {
    double acc = 0.0;
    for (int64_t t = 0; t < T; ++t) {
        const float* zt = z + t * (int64_t)E;
        double m = (double)zt[0];
        for (int32_t e = 1; e < E; ++e)
            if ((double)zt[e] > m) m = (double)zt[e];
        double Z = 0.0;
        for (int32_t e = 0; e < E; ++e) Z += exp((double)zt[e] - m);
        double h = 0.0;
        for (int32_t e = 0; e < E; ++e) {
            const double p = exp((double)zt[e] - m) / Z;
            if (p > 0.0) h -= p * log(p);
        }
        acc += h;
    }
    return acc / (double)T;
}

/* S1: MaxVio = (max n - nbar)/nbar, MinVio = (nbar - min n)/nbar (Eq. vio),
 * each as one fp64 division of an exact integer numerator.  out[0] = MaxVio,
 * out[1] = MinVio; both NaN for an empty batch. */
void oracle_load_stats(const int32_t* counts, int32_t E, double* out) {
    int64_t S = 0;
    int32_t mx = counts[0], mn = counts[0];
    for (int32_t i = 0; i < E; ++i) {
        S += counts[i];
        if (counts[i] > mx) mx = counts[i];
        if (counts[i] < mn) mn = counts[i];
    }
    if (S == 0) {
        out[0] = NAN;
        out[1] = NAN;
        return;
    }
    out[0] = (double)((int64_t)E * mx - S) / (double)S;
    out[1] = (double)(S - (int64_t)E * mn) / (double)S;
}

/* Q1: the cutoff of Eq. pid-quantile-def for each token: the (K+1)-th largest
 * biased score fl32(s + b) in the order of Eq. pid-routing (K + 1 passes of
 * "best not yet taken"; K + 1 <= E). */
void oracle_qb_alpha(const float* s, const float* bias, int64_t T, int32_t E, int32_t K, float* alpha) {
#pragma omp parallel
    {
        unsigned char* taken = (unsigned char*)malloc((size_t)E);
#pragma omp for schedule(static)
        for (int64_t t = 0; t < T; ++t) {
            const float* st = s + t * (int64_t)E;
            memset(taken, 0, (size_t)E);
            float pick = 0.0f;
            for (int32_t r = 0; r <= K; ++r) {
                int32_t best = -1;
                float best_v = 0.0f;
                for (int32_t i = 0; i < E; ++i) {
                    if (taken[i]) continue;
                    float v = st[i] + bias[i];
                    if (best < 0 || ranks_above(v, i, best_v, best)) {
                        best = i;
                        best_v = v;
                    }
                }
                taken[best] = 1;
                pick = best_v;
            }
            alpha[t] = pick + 0.0f; /* -0 read as +0 */
        }
        free(taken);
    }
}

static int cmp_float_asc(const void* a, const void* b) {
    float x = *(const float*)a, y = *(const float*)b;
    return (x > y) - (x < y);
}

/* Q2-Q4: Quantile Balancing's bias update (Eq. pid-quantile) from the batch's
 * scores s [T][E] and cutoffs alpha [T].  For each expert j: the margins
 * d_ij = fl32(s_ij - alpha_i) (-0 read as +0), their (1 - K/E) quantile q_j
 * as the k-th smallest with k = ceil(T (E - K) / E), the target Q_j = -q_j
 * (Eq. pid-quantile-def), then b_j = Q_j for rho == 0, else the EMA
 * fl32(fl32(rho b_j) + fl32(fl32(1 - rho) Q_j)).  1 <= K < E. */
void oracle_qb_update(const float* s, const float* alpha, int64_t T, int32_t E, int32_t K, float rho, float* bias) {
    const int64_t k = (T * (int64_t)(E - K) + E - 1) / E; /* ceil(T (E-K) / E), 1-based */
#pragma omp parallel
    {
        float* d = (float*)malloc(sizeof(float) * (size_t)T);
#pragma omp for schedule(static)
        for (int32_t j = 0; j < E; ++j) {
            for (int64_t t = 0; t < T; ++t) d[t] = (s[t * (int64_t)E + j] - alpha[t]) + 0.0f;
            qsort(d, (size_t)T, sizeof(float), cmp_float_asc);
            const float q = d[k - 1];
            const float Q = -q;
            if (rho == 0.0f) {
                bias[j] = Q;
            } else {
                const float keep = rho * bias[j];
                const float take = (1.0f - rho) * Q;
                bias[j] = keep + take;
            }
        }
        free(d);
    }
}

/* Wall-clock seconds of one whole oracle step (R1-R6, C1-C7, S1) on the host,
 * for the CPU baseline.  Uses the OpenMP thread count in effect. */
/* X1-X5 from logits z [T][E] (fp64): the auxiliary-loss router's forward
 * statistics (Eq. pid-auxloss).  idx, w [T][K] in rank order; counts [E];
 * f, P [E]; *loss = alpha sum_i f_i P_i. */
void oracle_aux_stats(const double* z, int64_t T, int32_t E, int32_t K, double alpha, int32_t* idx, float* w,
                      int32_t* counts, double* f, double* P, double* loss) {
    double* p = (double*)malloc((size_t)T * E * sizeof(double));
#pragma omp parallel
    {
        unsigned char* taken = (unsigned char*)malloc((size_t)E);
#pragma omp for schedule(static)
        for (int64_t t = 0; t < T; ++t) {
            const double* zt = z + t * (int64_t)E;
            double* pt = p + t * (int64_t)E;
            /* X1: softmax, the largest logit subtracted so exp cannot overflow */
            double m = zt[0];
            for (int32_t i = 1; i < E; ++i)
                if (zt[i] > m) m = zt[i];
            double Z = 0.0;
            for (int32_t i = 0; i < E; ++i) {
                pt[i] = exp(zt[i] - m);
                Z = Z + pt[i];
            }
            for (int32_t i = 0; i < E; ++i) pt[i] = pt[i] / Z;
            /* X2: Top-K on the fp32 logits, lowest index first among equals */
            memset(taken, 0, (size_t)E);
            int32_t* it = idx + t * (int64_t)K;
            for (int32_t r = 0; r < K; ++r) {
                int32_t best = -1;
                float best_v = 0.0f;
                for (int32_t i = 0; i < E; ++i) {
                    if (taken[i]) continue;
                    const float v = (float)zt[i];
                    if (best < 0 || ranks_above(v, i, best_v, best)) {
                        best = i;
                        best_v = v;
                    }
                }
                taken[best] = 1;
                it[r] = best;
            }
            /* X3: gate weights, the selected probabilities renormalised */
            double den = 0.0;
            for (int32_t r = 0; r < K; ++r) den = den + pt[it[r]];
            for (int32_t r = 0; r < K; ++r) w[t * (int64_t)K + r] = (float)(pt[it[r]] / den);
        }
        free(taken);
    }
    /* X4: assignment counts and fractions */
    for (int32_t i = 0; i < E; ++i) counts[i] = 0;
    for (int64_t t = 0; t < T; ++t)
        for (int32_t r = 0; r < K; ++r) counts[idx[t * (int64_t)K + r]] += 1;
    /* X5: mean probabilities and the loss */
    for (int32_t i = 0; i < E; ++i) {
        double acc = 0.0;
        for (int64_t t = 0; t < T; ++t) acc = acc + p[t * (int64_t)E + i];
        P[i] = acc / (double)T;
        f[i] = (double)counts[i] / (double)T;
    }
    double L = 0.0;
    for (int32_t i = 0; i < E; ++i) L = L + f[i] * P[i];
    *loss = alpha * L;
    free(p);
}

double oracle_step_seconds(const void* x, const void* W, int dtype, int64_t T, int32_t d, int32_t E, int32_t K,
                           float Ki, float Kd, float* bias, float* e_prev, int64_t* step, int32_t* status,
                           int32_t* idx, float* w, int32_t* counts, double* stats) {
    struct timespec t0, t1;
    clock_gettime(CLOCK_MONOTONIC, &t0);
    oracle_router(x, W, dtype, bias, T, d, E, K, idx, w, counts, 0, NULL);
    oracle_controller(counts, E, Ki, Kd, ORACLE_MODE_ERROR, 1, bias, e_prev, step, status);
    oracle_load_stats(counts, E, stats);
    clock_gettime(CLOCK_MONOTONIC, &t1);
    return (double)(t1.tv_sec - t0.tv_sec) + 1e-9 * (double)(t1.tv_nsec - t0.tv_nsec);
}
