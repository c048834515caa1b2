// C ABI of the ID Balancing router step (declared in include/idb.h): argument
// checks, tiling choice and kernel launches.  Every check runs before any HIP
// call, so an invalid call enqueues nothing and touches no output.
#include "idb.h"

#include <math.h>
#include <stdarg.h>
#include <stdio.h>

#include "internal.h"

namespace {

thread_local char g_last_error[256] = "";

idb_status fail(idb_status s, const char* fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_last_error, sizeof g_last_error, fmt, ap);
    va_end(ap);
    return s;
}

idb_status hip_result(hipError_t e, const char* what) {
    if (e == hipSuccess) return IDB_OK;
    return fail(IDB_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) == 0; }

constexpr int64_t kMaxTokens = int64_t(1) << 26;
constexpr int kMaxExperts = 1024;
constexpr int kMaxSlices = 8;
constexpr int kMaxKGpu = 32;

size_t round_up(size_t n) { return (n + 255) & ~size_t(255); }

// Resolve a router variant for a shape; returns IDB_OK and the tiling, or an error.
// one_slice: only tilings whose workgroups cover all E experts and that have
// the softmax mode (the auxiliary-loss statistics need each token's whole
// softmax in one workgroup).
idb_status resolve_tiling(int32_t E, idb_dtype dtype, int32_t variant, idb::RouterTiling* out,
                          bool one_slice = false) {
    const int n = idb::router_tiling_count();
    const int want_f32 = dtype == IDB_DTYPE_F32;
    const int max_slices = one_slice ? 1 : kMaxSlices;
    if (variant != 0) {
        if (variant < 1 || variant > n) return fail(IDB_ERR_INVALID_ARG, "router variant %d out of range", variant);
        idb::RouterTiling t = idb::router_tiling(variant - 1);
        if (t.is_f32 != want_f32) return fail(IDB_ERR_UNSUPPORTED, "router variant %d is for another dtype", variant);
        if (idb::router_slices(t, E) > max_slices)
            return fail(IDB_ERR_UNSUPPORTED, "router variant %d needs more than %d expert slice(s) for E=%d",
                        variant, max_slices, E);
        if (one_slice && !t.softmax)
            return fail(IDB_ERR_UNSUPPORTED, "router variant %d has no softmax mode", variant);
        *out = t;
        return IDB_OK;
    }
    // Automatic: among the tilings of this dtype, the fewest padded experts,
    // then the preferred one (the ranking follows measured throughput).
    bool found = false;
    idb::RouterTiling best{};
    long best_waste = 0;
    for (int i = 0; i < n; ++i) {
        idb::RouterTiling t = idb::router_tiling(i);
        if (t.is_f32 != want_f32) continue;
        const int ns = idb::router_slices(t, E);
        if (ns > max_slices || (one_slice && !t.softmax)) continue;
        const long waste = (long)ns * t.waves * t.we - E;
        if (!found || waste < best_waste || (waste == best_waste && t.rank < best.rank)) {
            best = t;
            best_waste = waste;
            found = true;
        }
    }
    if (!found)
        return fail(IDB_ERR_UNSUPPORTED, one_slice ? "no one-slice router tiling for E=%d" : "no router tiling for E=%d",
                    E);
    *out = best;
    return IDB_OK;
}

idb_status check_router_shape(int64_t T, int32_t d, int32_t E, int32_t K, idb_dtype dtype) {
    if (dtype != IDB_DTYPE_BF16 && dtype != IDB_DTYPE_F32) return fail(IDB_ERR_INVALID_ARG, "unknown dtype %d", dtype);
    if (T < 1 || T > kMaxTokens) return fail(IDB_ERR_INVALID_ARG, "T=%lld out of [1, 2^26]", (long long)T);
    // d <= 65536 and E <= 1024 keep every operand byte offset of the fused
    // kernel (at most E * d * 4 = 2^28) inside its 32-bit buffer addressing.
    if (d < 1 || d > 65536) return fail(IDB_ERR_INVALID_ARG, "d=%d out of [1, 65536]", d);
    if (E < 1 || K < 1 || K > E) return fail(IDB_ERR_INVALID_ARG, "need 1 <= K <= E (K=%d, E=%d)", K, E);
    if (E > kMaxExperts) return fail(IDB_ERR_UNSUPPORTED, "E=%d above %d", E, kMaxExperts);
    if (E % 32 != 0) return fail(IDB_ERR_UNSUPPORTED, "E=%d is not a multiple of 32", E);
    if (K > kMaxKGpu) return fail(IDB_ERR_UNSUPPORTED, "K=%d above %d", K, kMaxKGpu);
    const int dmul = dtype == IDB_DTYPE_BF16 ? 64 : 32;
    if (d % dmul != 0) return fail(IDB_ERR_UNSUPPORTED, "d=%d is not a multiple of %d", d, dmul);
    return IDB_OK;
}

size_t router_ws_bytes(int64_t T, int32_t E, int32_t K, const idb::RouterTiling& t) {
    const int ns = idb::router_slices(t, E);
    if (ns <= 1) return 0;
    // candidates (value, score, index) [T][ns][K], then the merge's ticket
    return 3 * round_up((size_t)T * ns * K * 4) + 256;
}

// Auxiliary-loss statistics: per-tile softmax column sums [tiles][E] fp32,
// per-tile counts [tiles][E] int32, kAuxMaxBlocks block records, the ticket.
size_t aux_rows_bytes(int64_t T, int32_t E, const idb::RouterTiling& t) {
    return round_up((size_t)((T + t.bt - 1) / t.bt) * E * 4);
}
size_t aux_ws_bytes(int64_t T, int32_t E, const idb::RouterTiling& t) {
    return 2 * aux_rows_bytes(T, E, t) + round_up(idb::kAuxMaxBlocks * sizeof(idb::AuxPartial)) + 256;
}

struct RouterCall {
    idb::RouterTiling tiling;
    idb::RouterArgs args;
    unsigned* ticket;  // the merge's (multi-slice tilings) or the statistics kernel's ticket
    idb::AuxPartial* aux_partial;  // auxiliary-loss statistics: block records
};

idb_status prepare_router(const void* x, const void* W_g, idb_dtype dtype, idb_weight_layout layout,
                          const float* bias, int64_t T, int32_t d,
                          int32_t E, int32_t K, int32_t* expert_idx, float* gate_w, int32_t* counts,
                          int32_t accumulate_counts, float* scores_dump, void* workspace, size_t workspace_bytes,
                          int32_t variant, bool need_inputs, RouterCall* call, bool qb = false,
                          bool aux = false) {
    // Quantile Balancing keeps K + 1 candidates per token (the (K+1)-th is the cutoff)
    const int32_t KL = qb ? K + 1 : K;
    idb_status st = check_router_shape(T, d, E, KL, dtype);
    if (st != IDB_OK) return st;
    if (layout != IDB_WEIGHT_ROW_MAJOR && layout != IDB_WEIGHT_PACKED)
        return fail(IDB_ERR_INVALID_ARG, "unknown weight layout %d", layout);
    if (need_inputs) {
        if (!x || !W_g || (!bias && !aux)) return fail(IDB_ERR_INVALID_ARG, "null input pointer");
        if (!aligned(x, 16) || !aligned(W_g, 16)) return fail(IDB_ERR_INVALID_ARG, "x and W_g must be 16-byte aligned");
        if (bias && !aligned(bias, 4)) return fail(IDB_ERR_INVALID_ARG, "bias must be 4-byte aligned");
        if (scores_dump && !aligned(scores_dump, 16))
            return fail(IDB_ERR_INVALID_ARG, "scores_dump must be 16-byte aligned");
    }
    if (!expert_idx || !gate_w || !counts) return fail(IDB_ERR_INVALID_ARG, "null output pointer");
    if (!aligned(expert_idx, 4) || !aligned(gate_w, 4) || !aligned(counts, 4))
        return fail(IDB_ERR_INVALID_ARG, "outputs must be 4-byte aligned");
    st = resolve_tiling(E, dtype, variant, &call->tiling, aux);
    if (st != IDB_OK) return st;
    const size_t need = aux ? aux_ws_bytes(T, E, call->tiling) : router_ws_bytes(T, E, KL, call->tiling);
    if (need > 0) {
        if (!workspace || workspace_bytes < need)
            return fail(IDB_ERR_INVALID_ARG, "workspace of %zu bytes needed, %zu given", need, workspace_bytes);
        if (!aligned(workspace, 16)) return fail(IDB_ERR_INVALID_ARG, "workspace must be 16-byte aligned");
    }
    idb::RouterArgs& a = call->args;
    a.x = x;
    a.W = W_g;
    a.w_packed = layout == IDB_WEIGHT_PACKED;
    a.bias = bias;
    a.T = T;
    a.d = d;
    a.E = E;
    a.K = K;
    a.idx = expert_idx;
    a.w = gate_w;
    a.counts = counts;
    a.dump = scores_dump;
    const int ns = idb::router_slices(call->tiling, E);
    a.zero_counts = (!accumulate_counts && ns > 1) ? 1 : 0;
    const size_t part = round_up((size_t)T * ns * KL * 4);
    char* ws = static_cast<char*>(workspace);
    a.cand_v = need ? reinterpret_cast<float*>(ws) : nullptr;
    a.cand_s = need ? reinterpret_cast<float*>(ws + part) : nullptr;
    a.cand_i = need ? reinterpret_cast<int32_t*>(ws + 2 * part) : nullptr;
    // the merge's ticket slot; the router kernel's first workgroup zeroes it,
    // so a merge that applies the controller update may follow any router call
    a.ticket = need ? reinterpret_cast<unsigned*>(ws + 3 * part) : nullptr;
    a.alpha = nullptr;
    a.scores_t = nullptr;
    a.softmax = aux ? 1 : 0;
    a.prob_part = nullptr;
    a.cnt_part = nullptr;
    call->ticket = need ? reinterpret_cast<unsigned*>(ws + 3 * part) : nullptr;
    call->aux_partial = nullptr;
    if (aux) {
        // one slice: no candidates; the statistics' per-tile rows instead
        const size_t rows = aux_rows_bytes(T, E, call->tiling);
        a.bias = nullptr;
        a.cand_v = a.cand_s = nullptr;
        a.cand_i = nullptr;
        a.prob_part = reinterpret_cast<float*>(ws);
        a.cnt_part = reinterpret_cast<int32_t*>(ws + rows);
        call->aux_partial = reinterpret_cast<idb::AuxPartial*>(ws + 2 * rows);
        call->ticket =
            reinterpret_cast<unsigned*>(ws + 2 * rows + round_up(idb::kAuxMaxBlocks * sizeof(idb::AuxPartial)));
        a.ticket = call->ticket;  // zeroed by the router kernel, taken by the statistics kernel
    }
    return IDB_OK;
}

idb_status enqueue_score_select(const RouterCall& c, int32_t accumulate_counts, hipStream_t stream,
                                hipEvent_t start = nullptr, hipEvent_t stop = nullptr) {
    const int ns = idb::router_slices(c.tiling, c.args.E);
    if (ns <= 1 && !accumulate_counts && !c.args.cnt_part) {
        idb_status st = hip_result(idb::launch_fill_i32(c.args.counts, 0, c.args.E, stream), "zero counts");
        if (st != IDB_OK) return st;
    }
    return hip_result(idb::launch_router_score_select(c.tiling, c.args, stream, start, stop),
                      "router score/select launch");
}

}  // namespace

extern "C" {

size_t idb_router_workspace_bytes(int64_t T, int32_t d, int32_t E, int32_t K, idb_dtype dtype, int32_t variant) {
    if (check_router_shape(T, d, E, K, dtype) != IDB_OK) return 0;
    idb::RouterTiling t;
    if (resolve_tiling(E, dtype, variant, &t) != IDB_OK) return 0;
    return router_ws_bytes(T, E, K, t);
}

idb_status idb_router_variant_info(int64_t T, int32_t d, int32_t E, int32_t K, idb_dtype dtype, int32_t variant,
                                   int32_t out[5]) {
    if (!out) return fail(IDB_ERR_INVALID_ARG, "null out");
    idb_status st = check_router_shape(T, d, E, K, dtype);
    if (st != IDB_OK) return st;
    idb::RouterTiling t;
    st = resolve_tiling(E, dtype, variant, &t);
    if (st != IDB_OK) return st;
    out[0] = t.bt;
    out[1] = idb::router_slices(t, E);
    out[2] = t.waves;
    out[3] = t.we;
    out[4] = t.id;
    return IDB_OK;
}

idb_status idb_router_score_select(const void* x, const void* W_g, idb_dtype dtype, idb_weight_layout weight_layout,
                                   const float* bias, int64_t T, int32_t d, int32_t E, int32_t K, int32_t* expert_idx,
                                   float* gate_w, int32_t* counts, int32_t accumulate_counts, float* scores_dump,
                                   void* workspace, size_t workspace_bytes, int32_t variant, hipStream_t stream) {
    RouterCall c;
    idb_status st = prepare_router(x, W_g, dtype, weight_layout, bias, T, d, E, K, expert_idx, gate_w, counts, accumulate_counts,
                                   scores_dump, workspace, workspace_bytes, variant, true, &c);
    if (st != IDB_OK) return st;
    return enqueue_score_select(c, accumulate_counts, stream);
}

idb_status idb_router_score_select_timed(const void* x, const void* W_g, idb_dtype dtype,
                                         idb_weight_layout weight_layout, const float* bias, int64_t T, int32_t d,
                                         int32_t E, int32_t K, int32_t* expert_idx, float* gate_w, int32_t* counts,
                                         int32_t accumulate_counts, float* scores_dump, void* workspace,
                                         size_t workspace_bytes, int32_t variant, hipStream_t stream,
                                         hipEvent_t start_event, hipEvent_t stop_event) {
    RouterCall c;
    idb_status st = prepare_router(x, W_g, dtype, weight_layout, bias, T, d, E, K, expert_idx, gate_w, counts, accumulate_counts,
                                   scores_dump, workspace, workspace_bytes, variant, true, &c);
    if (st != IDB_OK) return st;
    return enqueue_score_select(c, accumulate_counts, stream, start_event, stop_event);
}

idb_status idb_router_merge(int64_t T, int32_t d, int32_t E, int32_t K, idb_dtype dtype, int32_t* expert_idx,
                            float* gate_w, int32_t* counts, void* workspace, size_t workspace_bytes, int32_t variant,
                            hipStream_t stream) {
    RouterCall c;
    idb_status st = prepare_router(nullptr, nullptr, dtype, IDB_WEIGHT_ROW_MAJOR, nullptr, T, d, E, K, expert_idx, gate_w, counts, 1,
                                   nullptr, workspace, workspace_bytes, variant, false, &c);
    if (st != IDB_OK) return st;
    return hip_result(idb::launch_router_merge(c.tiling, c.args, nullptr, stream), "router merge launch");
}

idb_status idb_router_forward(const void* x, const void* W_g, idb_dtype dtype, idb_weight_layout weight_layout,
                              const float* bias, int64_t T, int32_t d, int32_t E, int32_t K, int32_t* expert_idx,
                              float* gate_w, int32_t* counts, int32_t accumulate_counts, float* scores_dump,
                              void* workspace, size_t workspace_bytes, int32_t variant, hipStream_t stream) {
    RouterCall c;
    idb_status st = prepare_router(x, W_g, dtype, weight_layout, bias, T, d, E, K, expert_idx, gate_w, counts, accumulate_counts,
                                   scores_dump, workspace, workspace_bytes, variant, true, &c);
    if (st != IDB_OK) return st;
    st = enqueue_score_select(c, accumulate_counts, stream);
    if (st != IDB_OK) return st;
    return hip_result(idb::launch_router_merge(c.tiling, c.args, nullptr, stream), "router merge launch");
}

size_t idb_router_packed_weight_bytes(int32_t E, int32_t d, idb_dtype dtype) {
    if (check_router_shape(1, d, E, 1, dtype) != IDB_OK) return 0;
    return (size_t)E * d * (dtype == IDB_DTYPE_BF16 ? 2 : 4);
}

idb_status idb_router_pack_weight(const void* W_g, idb_dtype dtype, int32_t E, int32_t d, void* W_packed,
                                  hipStream_t stream) {
    idb_status st = check_router_shape(1, d, E, 1, dtype);
    if (st != IDB_OK) return st;
    if (!W_g || !W_packed) return fail(IDB_ERR_INVALID_ARG, "null pointer");
    if (!aligned(W_g, 16) || !aligned(W_packed, 16)) return fail(IDB_ERR_INVALID_ARG, "W_g and W_packed must be 16-byte aligned");
    const size_t bytes = (size_t)E * d * (dtype == IDB_DTYPE_BF16 ? 2 : 4);
    const char* a0 = static_cast<const char*>(W_g);
    const char* b0 = static_cast<const char*>(W_packed);
    if (a0 < b0 + bytes && b0 < a0 + bytes) return fail(IDB_ERR_INVALID_ARG, "W_packed overlaps W_g");
    const int64_t rb = (int64_t)d * (dtype == IDB_DTYPE_BF16 ? 2 : 4);
    return hip_result(idb::launch_pack_weight(W_g, W_packed, E, rb, stream), "pack weight launch");
}

idb_status idb_select_from_scores(const float* scores, const float* bias, int64_t T, int32_t E, int32_t K,
                                  int32_t* expert_idx, float* gate_w, int32_t* counts, int32_t accumulate_counts,
                                  hipStream_t stream) {
    if (!scores || !bias || !expert_idx || !gate_w || !counts) return fail(IDB_ERR_INVALID_ARG, "null pointer");
    if (T < 1 || T > kMaxTokens) return fail(IDB_ERR_INVALID_ARG, "T=%lld out of [1, 2^26]", (long long)T);
    if (E < 1 || K < 1 || K > E) return fail(IDB_ERR_INVALID_ARG, "need 1 <= K <= E (K=%d, E=%d)", K, E);
    if (E > kMaxExperts) return fail(IDB_ERR_UNSUPPORTED, "E=%d above %d", E, kMaxExperts);
    if (K > kMaxKGpu) return fail(IDB_ERR_UNSUPPORTED, "K=%d above %d", K, kMaxKGpu);
    if (!aligned(scores, 4) || !aligned(bias, 4) || !aligned(expert_idx, 4) || !aligned(gate_w, 4) ||
        !aligned(counts, 4))
        return fail(IDB_ERR_INVALID_ARG, "buffers must be 4-byte aligned");
    if (!accumulate_counts) {
        idb_status st = hip_result(idb::launch_fill_i32(counts, 0, E, stream), "zero counts");
        if (st != IDB_OK) return st;
    }
    return hip_result(idb::launch_select_from_scores(scores, bias, T, E, K, expert_idx, gate_w, counts, stream),
                      "select launch");
}

namespace {
idb_status check_controller(const idb_controller_cfg* cfg, const idb_controller_state* state, const double* stats) {
    if (!cfg || !state) return fail(IDB_ERR_INVALID_ARG, "null pointer");
    if (!state->bias || !state->e_prev || !state->step || !state->status)
        return fail(IDB_ERR_INVALID_ARG, "null state buffer");
    if (cfg->E < 1 || cfg->E > kMaxExperts) return fail(IDB_ERR_INVALID_ARG, "E=%d out of [1, 1024]", cfg->E);
    if (!(cfg->Ki >= 0.0f) || !(cfg->Kd >= 0.0f) || !isfinite(cfg->Ki) || !isfinite(cfg->Kd))
        return fail(IDB_ERR_INVALID_ARG, "gains must be finite and >= 0");
    if (cfg->integral_mode != IDB_INTEGRAL_ERROR && cfg->integral_mode != IDB_INTEGRAL_SIGN)
        return fail(IDB_ERR_INVALID_ARG, "unknown integral mode %d", cfg->integral_mode);
    if (cfg->center != 0 && cfg->center != 1) return fail(IDB_ERR_INVALID_ARG, "center must be 0 or 1");
    if (!aligned(state->bias, 4) || !aligned(state->e_prev, 4) || !aligned(state->step, 8) ||
        !aligned(state->status, 4) || (stats && !aligned(stats, 8)))
        return fail(IDB_ERR_INVALID_ARG, "misaligned buffer");
    return IDB_OK;
}

idb_status enqueue_controller(const int32_t* counts, const idb_controller_cfg* cfg, const idb_controller_state* state,
                              double* stats, hipStream_t stream) {
    return hip_result(idb::launch_controller_update(counts, cfg->E, cfg->Ki, cfg->Kd,
                                                    cfg->integral_mode == IDB_INTEGRAL_SIGN, cfg->center,
                                                    state->bias, state->e_prev, state->step, state->status, stats,
                                                    stream),
                      "controller launch");
}

idb_status controller_call(const int32_t* counts, const idb_controller_cfg* cfg, const idb_controller_state* state,
                           double* stats, hipStream_t stream) {
    if (!counts) return fail(IDB_ERR_INVALID_ARG, "null pointer");
    idb_status st = check_controller(cfg, state, stats);
    if (st != IDB_OK) return st;
    if (!aligned(counts, 4)) return fail(IDB_ERR_INVALID_ARG, "misaligned buffer");
    return enqueue_controller(counts, cfg, state, stats, stream);
}
// The second launch of idb_router_step: the slice merge whose last workgroup
// applies the update (multi-slice tilings), or the controller step launch
// (one-slice tilings, whose router kernel finished the counts itself).
idb_status enqueue_merge_step(const RouterCall& c, const idb_controller_cfg* cfg, const idb_controller_state* state,
                              double* out_maxvio_minvio, hipStream_t stream) {
    if (!c.ticket) return enqueue_controller(c.args.counts, cfg, state, out_maxvio_minvio, stream);
    idb::CtrlArgs k;
    k.Ki = cfg->Ki;
    k.Kd = cfg->Kd;
    k.sign_mode = cfg->integral_mode == IDB_INTEGRAL_SIGN;
    k.center = cfg->center;
    k.bias = state->bias;
    k.e_prev = state->e_prev;
    k.step = state->step;
    k.status = state->status;
    k.stats = out_maxvio_minvio;
    k.ticket = c.ticket;
    return hip_result(idb::launch_router_merge(c.tiling, c.args, &k, stream), "router merge launch");
}


}  // namespace

idb_status idb_controller_update(const int32_t* counts, const idb_controller_cfg* cfg,
                                 const idb_controller_state* state, hipStream_t stream) {
    return controller_call(counts, cfg, state, nullptr, stream);
}

idb_status idb_controller_step(const int32_t* counts, const idb_controller_cfg* cfg,
                               const idb_controller_state* state, double* out_maxvio_minvio, hipStream_t stream) {
    if (!out_maxvio_minvio) return fail(IDB_ERR_INVALID_ARG, "null statistics output");
    return controller_call(counts, cfg, state, out_maxvio_minvio, stream);
}

idb_status idb_router_step(const void* x, const void* W_g, idb_dtype dtype, idb_weight_layout weight_layout,
                           int64_t T, int32_t d, int32_t K, const idb_controller_cfg* cfg,
                           const idb_controller_state* state, int32_t* expert_idx, float* gate_w, int32_t* counts,
                           int32_t accumulate_counts, double* out_maxvio_minvio, void* workspace,
                           size_t workspace_bytes, int32_t variant, hipStream_t stream) {
    idb_status st = check_controller(cfg, state, out_maxvio_minvio);
    if (st != IDB_OK) return st;
    RouterCall c;
    st = prepare_router(x, W_g, dtype, weight_layout, state->bias, T, d, cfg->E, K, expert_idx, gate_w, counts,
                        accumulate_counts, nullptr, workspace, workspace_bytes, variant, true, &c);
    if (st != IDB_OK) return st;
    st = enqueue_score_select(c, accumulate_counts, stream);
    if (st != IDB_OK) return st;
    return enqueue_merge_step(c, cfg, state, out_maxvio_minvio, stream);
}

idb_status idb_router_merge_step(int64_t T, int32_t d, int32_t K, idb_dtype dtype, const idb_controller_cfg* cfg,
                                 const idb_controller_state* state, int32_t* expert_idx, float* gate_w,
                                 int32_t* counts, double* out_maxvio_minvio, void* workspace, size_t workspace_bytes,
                                 int32_t variant, hipStream_t stream) {
    idb_status st = check_controller(cfg, state, out_maxvio_minvio);
    if (st != IDB_OK) return st;
    RouterCall c;
    st = prepare_router(nullptr, nullptr, dtype, IDB_WEIGHT_ROW_MAJOR, nullptr, T, d, cfg->E, K, expert_idx, gate_w,
                        counts, 1, nullptr, workspace, workspace_bytes, variant, false, &c);
    if (st != IDB_OK) return st;
    return enqueue_merge_step(c, cfg, state, out_maxvio_minvio, stream);
}

idb_status idb_router_step_noalloc(const void* x, const void* W_g, idb_dtype dtype, idb_weight_layout weight_layout,
                                   int64_t T, int32_t d, int32_t K, const idb_controller_cfg* cfg,
                                   const idb_controller_state* state, int32_t* expert_idx, float* gate_w,
                                   int32_t* counts, int32_t accumulate_counts, double* out_maxvio_minvio,
                                   int32_t variant, hipStream_t stream) {
    // every argument check of idb_router_step first, without any HIP call
    idb_status st = check_controller(cfg, state, out_maxvio_minvio);
    if (st != IDB_OK) return st;
    st = check_router_shape(T, d, cfg->E, K, dtype);
    if (st != IDB_OK) return st;
    idb::RouterTiling t;
    st = resolve_tiling(cfg->E, dtype, variant, &t);
    if (st != IDB_OK) return st;
    const size_t need = router_ws_bytes(T, cfg->E, K, t);
    const size_t have = idb::noalloc_scratch_bytes();
    if (need > have)
        return fail(IDB_ERR_UNSUPPORTED,
                    "idb_router_step_noalloc: this shape needs %zu bytes of scratch, the fixed scratch holds %zu "
                    "(T=%lld, E=%d, K=%d; use idb_router_step with a workspace)",
                    need, have, (long long)T, cfg->E, K);
    {
        // pointers, alignment and layout as idb_router_step checks them; the
        // workspace stands in as an aligned placeholder (only its size and
        // alignment are checked, nothing is dereferenced)
        RouterCall probe;
        st = prepare_router(x, W_g, dtype, weight_layout, state->bias, T, d, cfg->E, K, expert_idx, gate_w, counts,
                            accumulate_counts, nullptr, reinterpret_cast<void*>(uintptr_t(256)), have, variant, true,
                            &probe);
        if (st != IDB_OK) return st;
    }
    void* ws = nullptr;
    if (need > 0) {
        int dev = -1;
        st = hip_result(hipGetDevice(&dev), "current device");
        if (st != IDB_OK) return st;
        if (stream) {
            hipDevice_t sdev = -1;
            st = hip_result(hipStreamGetDevice(stream, &sdev), "stream device");
            if (st != IDB_OK) return st;
            if ((int)sdev != dev)
                return fail(IDB_ERR_INVALID_ARG, "stream belongs to device %d, current device is %d", (int)sdev, dev);
        }
        st = hip_result(idb::noalloc_scratch(dev, &ws), "scratch address");
        if (st != IDB_OK) return st;
    }
    return idb_router_step(x, W_g, dtype, weight_layout, T, d, K, cfg, state, expert_idx, gate_w, counts,
                           accumulate_counts, out_maxvio_minvio, ws, need > 0 ? have : 0, variant, stream);
}

size_t idb_qb_router_workspace_bytes(int64_t T, int32_t d, int32_t E, int32_t K, idb_dtype dtype,
                                     int32_t variant) {
    if (K < 1 || check_router_shape(T, d, E, K + 1, dtype) != IDB_OK) return 0;
    idb::RouterTiling t;
    if (resolve_tiling(E, dtype, variant, &t) != IDB_OK) return 0;
    return router_ws_bytes(T, E, K + 1, t);
}

idb_status idb_qb_router_forward(const void* x, const void* W_g, idb_dtype dtype, idb_weight_layout weight_layout,
                                 const float* bias, int64_t T, int32_t d, int32_t E, int32_t K, int32_t* expert_idx,
                                 float* gate_w, int32_t* counts, int32_t accumulate_counts, float* scores_t,
                                 float* alpha, void* workspace, size_t workspace_bytes, int32_t variant,
                                 hipStream_t stream) {
    if (K < 1) return fail(IDB_ERR_INVALID_ARG, "K=%d below 1", K);
    if (K + 1 > E) return fail(IDB_ERR_INVALID_ARG, "Quantile Balancing needs K + 1 <= E (K=%d, E=%d)", K, E);
    if (!scores_t || !alpha) return fail(IDB_ERR_INVALID_ARG, "null scores_t or alpha");
    if (!aligned(scores_t, 4) || !aligned(alpha, 4)) return fail(IDB_ERR_INVALID_ARG, "misaligned scores_t or alpha");
    RouterCall c;
    idb_status st = prepare_router(x, W_g, dtype, weight_layout, bias, T, d, E, K, expert_idx, gate_w, counts,
                                   accumulate_counts, nullptr, workspace, workspace_bytes, variant, true, &c, true);
    if (st != IDB_OK) return st;
    c.args.alpha = alpha;
    c.args.scores_t = scores_t;
    st = enqueue_score_select(c, accumulate_counts, stream);
    if (st != IDB_OK) return st;
    return hip_result(idb::launch_router_merge(c.tiling, c.args, nullptr, stream), "router merge launch");
}

idb_status idb_qb_update(const float* scores_t, const float* alpha, int64_t T, int32_t E, int32_t K, float rho,
                         float* bias, const int32_t* counts, double* out_maxvio_minvio, hipStream_t stream) {
    if (!scores_t || !alpha || !bias) return fail(IDB_ERR_INVALID_ARG, "null pointer");
    if (!counts != !out_maxvio_minvio)
        return fail(IDB_ERR_INVALID_ARG, "counts and out_maxvio_minvio go together (both or neither)");
    if (T < 1 || T > kMaxTokens) return fail(IDB_ERR_INVALID_ARG, "T=%lld out of [1, 2^26]", (long long)T);
    if (E < 2 || E > kMaxExperts) return fail(IDB_ERR_INVALID_ARG, "E=%d out of [2, %d]", E, kMaxExperts);
    if (K < 1 || K >= E) return fail(IDB_ERR_INVALID_ARG, "need 1 <= K < E (K=%d, E=%d)", K, E);
    if (!(rho >= 0.0f && rho < 1.0f)) return fail(IDB_ERR_INVALID_ARG, "rho must lie in [0, 1)");
    if (!aligned(scores_t, 4) || !aligned(alpha, 4) || !aligned(bias, 4) || !aligned(counts, 4) ||
        !aligned(out_maxvio_minvio, 8))
        return fail(IDB_ERR_INVALID_ARG, "misaligned buffer");
    return hip_result(idb::launch_qb_update(scores_t, alpha, T, E, K, rho, bias, counts, out_maxvio_minvio, stream),
                      "Quantile Balancing launch");
}

size_t idb_aux_router_workspace_bytes(int64_t T, int32_t d, int32_t E, int32_t K, idb_dtype dtype,
                                      int32_t variant) {
    if (check_router_shape(T, d, E, K, dtype) != IDB_OK) return 0;
    idb::RouterTiling t;
    if (resolve_tiling(E, dtype, variant, &t, true) != IDB_OK) return 0;
    return aux_ws_bytes(T, E, t);
}

idb_status idb_aux_router_forward(const void* x, const void* W_g, idb_dtype dtype, idb_weight_layout weight_layout,
                                  int64_t T, int32_t d, int32_t E, int32_t K, double alpha, int32_t* expert_idx,
                                  float* gate_w, int32_t* counts, double* f, double* P, double* loss,
                                  double* out_maxvio_minvio, float* logits_dump, void* workspace,
                                  size_t workspace_bytes, int32_t variant, hipStream_t stream) {
    if (!f || !P || !loss) return fail(IDB_ERR_INVALID_ARG, "null statistics output");
    if (!aligned(f, 8) || !aligned(P, 8) || !aligned(loss, 8) ||
        (out_maxvio_minvio && !aligned(out_maxvio_minvio, 8)))
        return fail(IDB_ERR_INVALID_ARG, "statistics outputs must be 8-byte aligned");
    if (!isfinite(alpha)) return fail(IDB_ERR_INVALID_ARG, "alpha must be finite");
    RouterCall c;
    idb_status st = prepare_router(x, W_g, dtype, weight_layout, nullptr, T, d, E, K, expert_idx, gate_w, counts, 0,
                                   logits_dump, workspace, workspace_bytes, variant, true, &c, false, true);
    if (st != IDB_OK) return st;
    st = enqueue_score_select(c, 0, stream);
    if (st != IDB_OK) return st;
    const int64_t tiles = (T + c.tiling.bt - 1) / c.tiling.bt;  // <= 2^26 / 64
    return hip_result(idb::launch_aux_stats(c.args.prob_part, c.args.cnt_part, (int)tiles, T, E, alpha, counts, f, P,
                                            loss, out_maxvio_minvio, c.aux_partial, c.ticket, stream),
                      "auxiliary-loss statistics launch");
}

idb_status idb_controller_update_layers(const int32_t* counts, int32_t L, const idb_controller_cfg* cfg,
                                        const idb_controller_state* state, double* out_stats, double* out_diag,
                                        hipStream_t stream) {
    if (!counts) return fail(IDB_ERR_INVALID_ARG, "null pointer");
    if (L < 1 || L > 65535) return fail(IDB_ERR_INVALID_ARG, "L=%d out of [1, 65535]", L);
    idb_status st = check_controller(cfg, state, out_stats);
    if (st != IDB_OK) return st;
    if (!aligned(counts, 4) || (out_diag && !aligned(out_diag, 8))) return fail(IDB_ERR_INVALID_ARG, "misaligned buffer");
    return hip_result(idb::launch_controller_layers(counts, L, cfg->E, cfg->Ki, cfg->Kd,
                                                    cfg->integral_mode == IDB_INTEGRAL_SIGN, cfg->center, state->bias,
                                                    state->e_prev, state->step, state->status, out_stats, out_diag,
                                                    stream),
                      "controller layers launch");
}

size_t idb_routing_entropy_workspace_bytes(void) { return (size_t)idb::kEntropyBlocks * 2 * sizeof(double); }

idb_status idb_routing_entropy(const float* gate_w, int64_t T, int32_t K, const float* scores, const float* bias,
                               int32_t E, void* workspace, size_t workspace_bytes, double* out, hipStream_t stream) {
    if (!gate_w || !out || !workspace) return fail(IDB_ERR_INVALID_ARG, "null pointer");
    if (T < 1 || T > kMaxTokens) return fail(IDB_ERR_INVALID_ARG, "T=%lld out of [1, 2^26]", (long long)T);
    if (K < 1 || K > kMaxKGpu) return fail(IDB_ERR_INVALID_ARG, "K=%d out of [1, %d]", K, kMaxKGpu);
    if (scores && (!bias || E < 1 || E > kMaxExperts))
        return fail(IDB_ERR_INVALID_ARG, "scores need a bias and 1 <= E <= %d", kMaxExperts);
    if (workspace_bytes < idb_routing_entropy_workspace_bytes())
        return fail(IDB_ERR_INVALID_ARG, "workspace of %zu bytes needed", idb_routing_entropy_workspace_bytes());
    if (!aligned(gate_w, 4) || !aligned(out, 8) || !aligned(workspace, 8) || (scores && !aligned(scores, 4)) ||
        (bias && !aligned(bias, 4)))
        return fail(IDB_ERR_INVALID_ARG, "misaligned buffer");
    return hip_result(idb::launch_routing_entropy(gate_w, T, K, scores, bias, E, 0, static_cast<double*>(workspace),
                                                  out, stream),
                      "routing entropy launch");
}

idb_status idb_routing_entropy_softmax(const float* gate_w, int64_t T, int32_t K, const float* logits, int32_t E,
                                       void* workspace, size_t workspace_bytes, double* out, hipStream_t stream) {
    if (!gate_w || !logits || !out || !workspace) return fail(IDB_ERR_INVALID_ARG, "null pointer");
    if (T < 1 || T > kMaxTokens) return fail(IDB_ERR_INVALID_ARG, "T=%lld out of [1, 2^26]", (long long)T);
    if (K < 1 || K > kMaxKGpu) return fail(IDB_ERR_INVALID_ARG, "K=%d out of [1, %d]", K, kMaxKGpu);
    if (E < 1 || E > kMaxExperts) return fail(IDB_ERR_INVALID_ARG, "E=%d out of [1, %d]", E, kMaxExperts);
    if (workspace_bytes < idb_routing_entropy_workspace_bytes())
        return fail(IDB_ERR_INVALID_ARG, "workspace of %zu bytes needed", idb_routing_entropy_workspace_bytes());
    if (!aligned(gate_w, 4) || !aligned(out, 8) || !aligned(workspace, 8) || !aligned(logits, 4))
        return fail(IDB_ERR_INVALID_ARG, "misaligned buffer");
    return hip_result(idb::launch_routing_entropy(gate_w, T, K, logits, nullptr, E, 1,
                                                  static_cast<double*>(workspace), out, stream),
                      "routing entropy launch");
}

idb_status idb_load_stats(const int32_t* counts, int32_t E, double* out_maxvio_minvio, hipStream_t stream) {
    if (!counts || !out_maxvio_minvio) return fail(IDB_ERR_INVALID_ARG, "null pointer");
    if (E < 1 || E > (1 << 20)) return fail(IDB_ERR_INVALID_ARG, "E=%d out of [1, 2^20]", E);
    if (!aligned(counts, 4) || !aligned(out_maxvio_minvio, 8)) return fail(IDB_ERR_INVALID_ARG, "misaligned buffer");
    return hip_result(idb::launch_load_stats(counts, E, out_maxvio_minvio, stream), "load stats launch");
}

const char* idb_status_string(idb_status s) {
    switch (s) {
        case IDB_OK: return "ok";
        case IDB_ERR_INVALID_ARG: return "invalid argument";
        case IDB_ERR_UNSUPPORTED: return "unsupported shape or option";
        case IDB_ERR_EMPTY_BATCH: return "empty batch: every count is zero";
        case IDB_ERR_HIP: return "HIP launch failure";
        default: return "unknown status";
    }
}

const char* idb_last_error(void) { return g_last_error; }

}  // extern "C"
