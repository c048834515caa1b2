// Host-side launchers of the gfx950 kernels, called by the C ABI (abi.cpp).
// Arguments are validated by the caller; these only enqueue work.
#pragma once

#include <hip/hip_runtime_api.h>
#include <stddef.h>
#include <stdint.h>

namespace idb {

// stats: nullable device double[2]; when set, MaxVio/MinVio of counts too.
hipError_t launch_controller_update(const int32_t* counts, int E, float Ki, float Kd, int sign_mode, int center,
                                    float* bias, float* e_prev, int64_t* step, int32_t* status, double* stats,
                                    hipStream_t stream);
hipError_t launch_load_stats(const int32_t* counts, int E, double* out, hipStream_t stream);
// L layers' controller updates in one launch; stats [L][2], diag [L][4] nullable.
hipError_t launch_controller_layers(const int32_t* counts, int L, int E, float Ki, float Kd, int sign_mode,
                                    int center, float* bias, float* e_prev, int64_t* step, int32_t* status,
                                    double* stats, double* diag, hipStream_t stream);
// Routing entropies: partial sums into workspace [kEntropyBlocks][2], then the means into out[2]; softmax:
// H_full over the softmax of the logits in scores (bias unused).
constexpr int kEntropyBlocks = 512;
hipError_t launch_routing_entropy(const float* gate_w, int64_t T, int K, const float* scores, const float* bias,
                                  int E, int softmax, double* partial, double* out, hipStream_t stream);

// Auxiliary-loss statistics from the router's per-tile softmax column sums
// prob_part [tiles][E] and counts cnt_part [tiles][E]: counts [E], f [E],
// P [E], loss, and (stats nullable) MaxVio/MinVio.  partial holds
// kAuxMaxBlocks block records; the ticket must be zero (the router kernel
// zeroes it).
constexpr int kAuxMaxBlocks = 16;  // expert blocks of 64 for E <= 1024
struct AuxPartial {
    double fp;  // sum of f_i P_i over the block's experts
    long long sum;
    int max, min;
};
hipError_t launch_aux_stats(const float* prob_part, const int32_t* cnt_part, int tiles, int64_t T, int E,
                            double alpha, int32_t* counts, double* f, double* P, double* loss, double* stats,
                            AuxPartial* partial, unsigned* ticket, hipStream_t stream);

// Fixed scratch of idb_router_step_noalloc (noalloc.hip): its size, and its
// device address on `device` (which must be the current device; the address
// is looked up once per device and kept).
size_t noalloc_scratch_bytes();
hipError_t noalloc_scratch(int device, void** out);

hipError_t launch_fill_i32(int32_t* p, int32_t value, int64_t n, hipStream_t stream);
// Quantile Balancing's bias update from expert-major scores and cutoffs;
// with counts (nullable), workgroup 0 also writes MaxVio/MinVio to stats.
hipError_t launch_qb_update(const float* scores_t, const float* alpha, int64_t T, int E, int K, float rho,
                            float* bias, const int32_t* counts, double* stats, hipStream_t stream);
// Selection from given scores; counts must already hold the starting values.
hipError_t launch_select_from_scores(const float* scores, const float* bias, int64_t T, int E, int K,
                                     int32_t* idx, float* w, int32_t* counts, hipStream_t stream);

// Tilings of the fused router kernel.
struct RouterTiling {
    int id;       // variant id (1-based)
    int is_f32;   // input dtype of this tiling
    int waves;    // waves per workgroup
    int bt;       // tokens per workgroup
    int we;       // experts per wave (a workgroup's slice is waves * we experts)
    int rank;     // preference among tilings with equally few padded experts (lower first)
    int softmax;  // the softmax mode (auxiliary-loss routing) is compiled for this tiling
};

// Number of known tilings and the i-th one (0-based).
int router_tiling_count();
RouterTiling router_tiling(int i);

struct RouterArgs {
    const void* x;
    const void* W;
    int w_packed;  // W is in the packed layout of launch_pack_weight
    const float* bias;
    int64_t T;
    int d;
    int E;
    int K;
    int32_t* idx;
    float* w;
    int32_t* counts;
    int zero_counts;  // workgroup 0 of the multi-slice kernel zeroes counts
    unsigned* ticket;  // nullable; workgroup 0 of the multi-slice kernel zeroes it
    float* dump;
    // multi-slice candidates in the workspace: [T][slices][KL], KL = K, or
    // K + 1 with alpha set
    float* cand_v;
    float* cand_s;
    int32_t* cand_i;
    // Quantile Balancing (Eq. pid-quantile-def), both nullable: alpha [T] the
    // (K+1)-th largest biased score per token; scores_t [E][T] the scores.
    float* alpha;
    float* scores_t;
    // Auxiliary-loss routing (Eq. pid-auxloss; one-slice tilings only): the
    // logits themselves are ranked (bias null: no bias), the gate weights are
    // the selected softmax probabilities renormalised, and with prob_part set
    // each token tile's column sums of the full softmax go to [tiles][E].
    int softmax;
    float* prob_part;
    // softmax mode: each token tile's expert counts go to cnt_part [tiles][E]
    // (no atomics; the statistics kernel sums them into counts)
    int32_t* cnt_part;
};

// Slices of E covered by one workgroup column for tiling t.
inline int router_slices(const RouterTiling& t, int E) {
    const int be = t.waves * t.we;
    return (E + be - 1) / be;
}

// Controller update run by the last workgroup of the slice merge (after every
// other workgroup has flushed its counts); the ticket counts finished
// workgroups and must be zero at the merge launch.
struct CtrlArgs {
    float Ki, Kd;
    int sign_mode, center;
    float* bias;
    float* e_prev;
    int64_t* step;
    int32_t* status;
    double* stats;  // nullable
    unsigned* ticket;
};

// start/stop: nullable events that take the kernel's own start and end
// timestamps (an extended launch; measurement only).
hipError_t launch_router_score_select(const RouterTiling& t, const RouterArgs& a, hipStream_t stream,
                                      hipEvent_t start = nullptr, hipEvent_t stop = nullptr);
// ctrl: nullable; with it, the merge also runs the controller update on the
// finished counts (multi-slice tilings only).
hipError_t launch_router_merge(const RouterTiling& t, const RouterArgs& a, const CtrlArgs* ctrl,
                               hipStream_t stream);
// Router matrix [E][d] (row_bytes per row) -> the packed A-operand layout.
hipError_t launch_pack_weight(const void* W, void* P, int E, int64_t row_bytes, hipStream_t stream);

}  // namespace idb
