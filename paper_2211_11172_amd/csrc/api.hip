// libharl C ABI: argument validation and dispatch.  Every host-visible check runs before any HIP
// call, so a rejected call launches nothing and touches no output.
#include <hip/hip_runtime.h>

#include <map>
#include <mutex>
#include <string>

#include <cmath>

#include "internal.hpp"

namespace harl {

static thread_local std::string g_last_error;

int fail(int status, const std::string &msg) {
    g_last_error = msg;
    return status;
}

int hip_fail(hipError_t e, const char *what) {
    g_last_error = std::string(what) + ": " + hipGetErrorString(e);
    return HARL_E_HIP;
}

int ensure_dynamic_lds(const void *kernel, size_t bytes) {
    static std::mutex mu;
    static std::map<std::pair<const void *, int>, size_t> done;
    int dev = 0;
    HARL_HIP_CHECK(hipGetDevice(&dev));
    std::lock_guard<std::mutex> lock(mu);
    size_t &have = done[{kernel, dev}];
    if (have >= bytes) return HARL_OK;
    HARL_HIP_CHECK(hipFuncSetAttribute(kernel, hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes));
    have = bytes;
    return HARL_OK;
}

}  // namespace harl

using harl::aligned;
using harl::fail;

extern "C" {

const char *harl_last_error(void) { return harl::g_last_error.c_str(); }

const char *harl_version(void) { return "harl 0.1 gfx950"; }

int harl_ensemble_create(const harl_ensemble_desc *desc, harl_ensemble **out, void *stream) {
    if (!desc || !out) return fail(HARL_E_INVALID_ARG, "harl_ensemble_create: null desc or out");
    *out = nullptr;
    return harl::pack_ensemble(desc, out, static_cast<hipStream_t>(stream));
}

int harl_ensemble_destroy(harl_ensemble *ens) {
    if (!ens) return HARL_OK;
    harl::free_ensemble(ens);
    return HARL_OK;
}

int harl_ensemble_info(const harl_ensemble *ens, int32_t *n_trees, int32_t *depth, int32_t *n_features) {
    if (!ens) return fail(HARL_E_INVALID_ARG, "harl_ensemble_info: null handle");
    if (n_trees) *n_trees = ens->n_trees;
    if (depth) *depth = ens->depth;
    if (n_features) *n_features = ens->n_features;
    return HARL_OK;
}

size_t harl_score_round_workspace_size(const harl_ensemble *ens, int32_t n_rows, int32_t n_prog) {
    (void)n_prog;
    if (!ens || n_rows < 0) return 0;
    return harl::score_round_ws_bytes(ens, n_rows);
}

int harl_score_round(const harl_ensemble *ens, const float *d_feat, int64_t ld, int32_t n_rows,
                     const int32_t *d_prog_ptr, int32_t n_prog, float *d_prog_score, float *d_stmt_score,
                     void *d_ws, size_t ws_bytes, void *stream) {
    if (!ens) return fail(HARL_E_INVALID_ARG, "harl_score_round: null ensemble");
    if (n_rows < 0 || n_prog < 0) return fail(HARL_E_INVALID_ARG, "harl_score_round: negative size");
    if (n_prog == 0) return HARL_OK;
    if (!d_prog_ptr || !d_prog_score) return fail(HARL_E_INVALID_ARG, "harl_score_round: null prog_ptr or prog_score");
    if (n_rows > 0 && !d_feat) return fail(HARL_E_INVALID_ARG, "harl_score_round: null features");
    if (ld < n_rows) return fail(HARL_E_INVALID_ARG, "harl_score_round: ld must be >= n_rows");
    if (ld > ((int64_t)1 << 40)) return fail(HARL_E_INVALID_ARG, "harl_score_round: ld too large");
    if (d_feat && !aligned(d_feat, 4)) return fail(HARL_E_INVALID_ARG, "harl_score_round: features must be 4-byte aligned");
    if (!aligned(d_prog_ptr, 4) || !aligned(d_prog_score, 4) || (d_stmt_score && !aligned(d_stmt_score, 4)))
        return fail(HARL_E_INVALID_ARG, "harl_score_round: misaligned int32/fp32 array");
    if (!d_ws || !aligned(d_ws, 256)) return fail(HARL_E_INVALID_ARG, "harl_score_round: workspace null or not 256-byte aligned");
    if (ws_bytes < harl::score_round_ws_bytes(ens, n_rows))
        return fail(HARL_E_WORKSPACE, "harl_score_round: workspace smaller than harl_score_round_workspace_size()");
    return harl::score_round_launch(ens, d_feat, ld, n_rows, d_prog_ptr, n_prog, d_prog_score, d_stmt_score, d_ws,
                                    ws_bytes, static_cast<hipStream_t>(stream));
}

int harl_policy_create(const harl_policy_desc *desc, harl_policy **out, void *stream) {
    if (!desc || !out) return fail(HARL_E_INVALID_ARG, "harl_policy_create: null desc or out");
    *out = nullptr;
    return harl::pack_policy(desc, out, static_cast<hipStream_t>(stream));
}

int harl_policy_destroy(harl_policy *pol) {
    if (!pol) return HARL_OK;
    void *ptrs[] = {pol->d_w1, pol->d_w2, pol->d_wh, pol->d_b1, pol->d_b2, pol->d_bh, pol->x32_stream, pol->x32_bias};
    hipError_t first = hipSuccess;
    for (void *p : ptrs) {
        hipError_t e = hipFree(p);
        if (first == hipSuccess) first = e;
    }
    delete pol;
    return first == hipSuccess ? HARL_OK : harl::hip_fail(first, "harl_policy_destroy");
}

int harl_policy_step(const harl_policy *pol, const void *d_states, int32_t B, int32_t *d_action, float *d_value,
                     float *d_probs, float *d_logits, void *stream) {
    if (!pol) return fail(HARL_E_INVALID_ARG, "harl_policy_step: null policy");
    if (B < 0) return fail(HARL_E_INVALID_ARG, "harl_policy_step: negative batch");
    if (B == 0) return HARL_OK;
    if (!d_states || !d_action || !d_value) return fail(HARL_E_INVALID_ARG, "harl_policy_step: null states, action or value");
    const size_t el = pol->dtype == HARL_BF16 ? 2 : 4;
    if (!aligned(d_states, el) || !aligned(d_action, 4) || !aligned(d_value, 4) || (d_probs && !aligned(d_probs, 4)) ||
        (d_logits && !aligned(d_logits, 4)))
        return fail(HARL_E_INVALID_ARG, "harl_policy_step: misaligned array");
    return harl::policy_step_launch(pol, d_states, B, d_action, d_value, d_probs, d_logits,
                                    static_cast<hipStream_t>(stream));
}

size_t harl_topk_workspace_size(int32_t n, int32_t k) {
    if (n < 0 || k < 0) return 0;
    return harl::topk_ws_bytes(n, k);
}

// Checks shared by harl_topk and harl_topk_static (everything but the workspace); *done is set
// when the call is a valid no-op.
static int topk_check(const char *who, const float *d_score, int32_t n, int32_t k, int64_t index_base,
                      const float *d_io_score, const int64_t *d_io_index, uint32_t flags, bool *done) {
    *done = false;
    const std::string w(who);
    if (n < 0 || k < 0) return fail(HARL_E_INVALID_ARG, w + ": negative size");
    if (k > HARL_TOPK_MAX_K) return fail(HARL_E_UNSUPPORTED, w + ": k above HARL_TOPK_MAX_K");
    if (flags & ~HARL_TOPK_MERGE) return fail(HARL_E_INVALID_ARG, w + ": unknown flag");
    if (!(flags & HARL_TOPK_MERGE) && k > n) return fail(HARL_E_INVALID_ARG, w + ": k > n without HARL_TOPK_MERGE");
    if (index_base < 0 || index_base > ((int64_t)1 << 62) - 1 - n)
        return fail(HARL_E_INVALID_ARG, w + ": index_base out of range");
    if (k == 0) {
        *done = true;
        return HARL_OK;
    }
    if (!d_io_score || !d_io_index) return fail(HARL_E_INVALID_ARG, w + ": null output");
    if (!aligned(d_io_score, 4) || !aligned(d_io_index, 8)) return fail(HARL_E_INVALID_ARG, w + ": misaligned output");
    if (n == 0) {  // only reachable with MERGE: nothing to merge
        *done = true;
        return HARL_OK;
    }
    if (!d_score || !aligned(d_score, 4)) return fail(HARL_E_INVALID_ARG, w + ": null or misaligned scores");
    return HARL_OK;
}

int harl_topk(const float *d_score, int32_t n, int32_t k, int64_t index_base, float *d_io_score, int64_t *d_io_index,
              uint32_t flags, void *d_ws, size_t ws_bytes, void *stream) {
    bool done = false;
    if (const int rc = topk_check("harl_topk", d_score, n, k, index_base, d_io_score, d_io_index, flags, &done)) return rc;
    if (done) return HARL_OK;
    if (!d_ws || !aligned(d_ws, 256)) return fail(HARL_E_INVALID_ARG, "harl_topk: workspace null or not 256-byte aligned");
    if (ws_bytes < harl::topk_ws_bytes(n, k))
        return fail(HARL_E_WORKSPACE, "harl_topk: workspace smaller than harl_topk_workspace_size()");
    return harl::topk_launch(d_score, n, k, index_base, d_io_score, d_io_index, flags, d_ws, ws_bytes,
                             static_cast<hipStream_t>(stream));
}

int harl_topk_static(const float *d_score, int32_t n, int32_t k, int64_t index_base, float *d_io_score,
                     int64_t *d_io_index, uint32_t flags, void *stream) {
    bool done = false;
    if (const int rc = topk_check("harl_topk_static", d_score, n, k, index_base, d_io_score, d_io_index, flags, &done))
        return rc;
    if (done) return HARL_OK;
    const size_t need = harl::topk_ws_bytes(n, k);
    if (need > (size_t)HARL_TOPK_STATIC_SCRATCH_BYTES)
        return fail(HARL_E_UNSUPPORTED, "harl_topk_static: n and k need " + std::to_string(need) +
                                            " bytes of scratch, above HARL_TOPK_STATIC_SCRATCH_BYTES (" +
                                            std::to_string((size_t)HARL_TOPK_STATIC_SCRATCH_BYTES) + "); use harl_topk");
    void *ws = nullptr;
    if (const int rc = harl::topk_scratch(&ws)) return rc;
    return harl::topk_launch(d_score, n, k, index_base, d_io_score, d_io_index, flags, ws,
                             (size_t)HARL_TOPK_STATIC_SCRATCH_BYTES, static_cast<hipStream_t>(stream));
}

int harl_topk_reset(float *d_io_score, int64_t *d_io_index, int32_t k, void *stream) {
    if (k < 0 || k > HARL_TOPK_MAX_K) return fail(HARL_E_INVALID_ARG, "harl_topk_reset: k out of range");
    if (k == 0) return HARL_OK;
    if (!d_io_score || !d_io_index || !aligned(d_io_score, 4) || !aligned(d_io_index, 8))
        return fail(HARL_E_INVALID_ARG, "harl_topk_reset: null or misaligned output");
    return harl::topk_reset_launch(d_io_score, d_io_index, k, static_cast<hipStream_t>(stream));
}

int harl_policy_select(const float *d_logits, int32_t B, int32_t a, const int32_t *seg_offsets, int32_t n_seg,
                       uint32_t flags, uint64_t seed, uint64_t counter, int32_t *d_action, float *d_logp, float *d_probs,
                       void *stream) {
    if (B < 0 || a < 1 || a > 4096) return fail(HARL_E_INVALID_ARG, "harl_policy_select: need B >= 0 and 1 <= a <= 4096");
    if (n_seg < 1 || n_seg > HARL_SELECT_MAX_SEGMENTS)
        return fail(HARL_E_INVALID_ARG, "harl_policy_select: n_seg out of range");
    if (flags & ~HARL_SELECT_SAMPLE) return fail(HARL_E_INVALID_ARG, "harl_policy_select: unknown flag");
    if (!seg_offsets || seg_offsets[0] != 0 || seg_offsets[n_seg] != a)
        return fail(HARL_E_INVALID_ARG, "harl_policy_select: segments must run from 0 to a");
    for (int s = 0; s < n_seg; ++s)
        if (seg_offsets[s + 1] <= seg_offsets[s])
            return fail(HARL_E_INVALID_ARG, "harl_policy_select: segment offsets must increase");
    if (B == 0) return HARL_OK;
    if (!d_logits || !aligned(d_logits, 4)) return fail(HARL_E_INVALID_ARG, "harl_policy_select: null or misaligned logits");
    if (!d_action || !aligned(d_action, 4) || (d_logp && !aligned(d_logp, 4)) || (d_probs && !aligned(d_probs, 4)))
        return fail(HARL_E_INVALID_ARG, "harl_policy_select: null or misaligned output");
    return harl::policy_select_launch(d_logits, B, a, seg_offsets, n_seg, flags, seed, counter, d_action, d_logp,
                                      d_probs, static_cast<hipStream_t>(stream));
}

static int ppo_check_config(const harl_ppo_config *c) {
    if (!c) return fail(HARL_E_INVALID_ARG, "harl_ppo: null config");
    if (c->s < 1 || c->s > 1024 || c->h1 < 1 || c->h1 > 4096 || c->h2 < 1 || c->h2 > 4096 || c->a < 1 || c->a > 4096)
        return fail(HARL_E_INVALID_ARG, "harl_ppo: sizes out of range");
    if (c->n_seg < 1 || c->n_seg > HARL_SELECT_MAX_SEGMENTS || c->seg_offsets[0] != 0 || c->seg_offsets[c->n_seg] != c->a)
        return fail(HARL_E_INVALID_ARG, "harl_ppo: segments must run from 0 to a");
    for (int s = 0; s < c->n_seg; ++s)
        if (c->seg_offsets[s + 1] <= c->seg_offsets[s]) return fail(HARL_E_INVALID_ARG, "harl_ppo: segment offsets must increase");
    if (!(c->clip_eps >= 0.f && c->clip_eps < 1.f) || !(c->beta1 >= 0.f && c->beta1 < 1.f) ||
        !(c->beta2 >= 0.f && c->beta2 < 1.f) || !(c->adam_eps > 0.f) || !(c->lr_actor >= 0.f) || !(c->lr_critic >= 0.f) ||
        !(c->w_value >= 0.f) || !(c->w_entropy >= 0.f))
        return fail(HARL_E_INVALID_ARG, "harl_ppo: hyper-parameter out of range");
    return HARL_OK;
}

size_t harl_ppo_param_count(const harl_ppo_config *cfg) {
    if (ppo_check_config(cfg) != HARL_OK) return 0;
    return harl::ppo_param_count(cfg);
}

size_t harl_ppo_workspace_size(const harl_ppo_config *cfg, int32_t M) {
    if (ppo_check_config(cfg) != HARL_OK || M < 0) return 0;
    return harl::ppo_ws_bytes(cfg, M);
}

int harl_ppo_update(const harl_ppo_config *cfg, float *d_params, float *d_adam_m, float *d_adam_v, int32_t step,
                    const float *d_states, const int32_t *d_actions, const float *d_logp_old, const float *d_adv,
                    const float *d_ret, int32_t M, float *d_grad, float *d_loss, void *d_ws, size_t ws_bytes,
                    void *stream) {
    if (const int rc = ppo_check_config(cfg)) return rc;
    if (M < 0 || step < 1) return fail(HARL_E_INVALID_ARG, "harl_ppo_update: need M >= 0 and step >= 1");
    if (M == 0) return HARL_OK;
    const void *in[] = {d_params, d_adam_m, d_adam_v, d_states, d_actions, d_logp_old, d_adv, d_ret};
    for (const void *p : in)
        if (!p || !aligned(p, 4)) return fail(HARL_E_INVALID_ARG, "harl_ppo_update: null or misaligned array");
    if ((d_grad && !aligned(d_grad, 4)) || (d_loss && !aligned(d_loss, 4)))
        return fail(HARL_E_INVALID_ARG, "harl_ppo_update: misaligned output");
    if (!d_ws || !aligned(d_ws, 256)) return fail(HARL_E_INVALID_ARG, "harl_ppo_update: workspace null or not 256-byte aligned");
    if (ws_bytes < harl::ppo_ws_bytes(cfg, M))
        return fail(HARL_E_WORKSPACE, "harl_ppo_update: workspace smaller than harl_ppo_workspace_size()");
    return harl::ppo_update_launch(cfg, d_params, d_adam_m, d_adam_v, step, d_states, d_actions, d_logp_old, d_adv, d_ret,
                                   M, d_grad, d_loss, d_ws, static_cast<hipStream_t>(stream));
}

int harl_track_advantage(const float *d_c_prev, const float *d_c_next, const float *d_v_prev, const float *d_v_next,
                         int32_t n, float gamma, float eps, float *d_reward, float *d_adv, void *stream) {
    if (n < 0) return fail(HARL_E_INVALID_ARG, "harl_track_advantage: negative size");
    if (!(eps > 0.f) || !(eps < INFINITY)) return fail(HARL_E_INVALID_ARG, "harl_track_advantage: eps must be > 0 and finite");
    if (n == 0) return HARL_OK;
    const float *in[] = {d_c_prev, d_c_next, d_v_prev, d_v_next};
    for (const float *p : in)
        if (!p || !aligned(p, 4)) return fail(HARL_E_INVALID_ARG, "harl_track_advantage: null or misaligned input");
    if (!d_adv || !aligned(d_adv, 4) || (d_reward && !aligned(d_reward, 4)))
        return fail(HARL_E_INVALID_ARG, "harl_track_advantage: null or misaligned output");
    return harl::track_advantage_launch(d_c_prev, d_c_next, d_v_prev, d_v_next, n, gamma, eps, d_reward, d_adv,
                                        static_cast<hipStream_t>(stream));
}

int harl_track_keep_count(int32_t n, double rho, int32_t *n_keep) {
    if (!n_keep) return fail(HARL_E_INVALID_ARG, "harl_track_keep_count: null n_keep");
    if (n < 0 || !(rho >= 0.0 && rho <= 1.0)) return fail(HARL_E_INVALID_ARG, "harl_track_keep_count: need n >= 0, 0 <= rho <= 1");
    *n_keep = n - (int32_t)std::floor(rho * (double)n);
    return HARL_OK;
}

size_t harl_track_eliminate_workspace_size(int32_t n) {
    if (n < 0) return 0;
    return harl::track_eliminate_ws_bytes(n);
}

int harl_track_eliminate(const float *d_adv, int32_t n, int32_t n_keep, int32_t *d_keep_index, const void *d_rows,
                         int64_t row_bytes, void *d_rows_out, void *d_ws, size_t ws_bytes, void *stream) {
    if (n < 0 || n_keep < 0 || n_keep > n) return fail(HARL_E_INVALID_ARG, "harl_track_eliminate: need 0 <= n_keep <= n");
    if ((d_rows == nullptr) != (d_rows_out == nullptr))
        return fail(HARL_E_INVALID_ARG, "harl_track_eliminate: give both rows and rows_out, or neither");
    if (d_rows && (row_bytes < 1 || row_bytes > ((int64_t)1 << 40) / (n > 0 ? n : 1)))
        return fail(HARL_E_INVALID_ARG, "harl_track_eliminate: row_bytes out of range");
    if (n_keep == 0) return HARL_OK;
    if (!d_adv || !aligned(d_adv, 4)) return fail(HARL_E_INVALID_ARG, "harl_track_eliminate: null or misaligned advantages");
    if (!d_keep_index || !aligned(d_keep_index, 4))
        return fail(HARL_E_INVALID_ARG, "harl_track_eliminate: null or misaligned keep_index");
    if (d_rows) {
        const char *a = static_cast<const char *>(d_rows), *b = static_cast<const char *>(d_rows_out);
        if (a < b + (int64_t)n_keep * row_bytes && b < a + (int64_t)n * row_bytes)
            return fail(HARL_E_INVALID_ARG, "harl_track_eliminate: rows and rows_out overlap");
    }
    if (n_keep < n) {
        if (!d_ws || !aligned(d_ws, 256))
            return fail(HARL_E_INVALID_ARG, "harl_track_eliminate: workspace null or not 256-byte aligned");
        if (ws_bytes < harl::track_eliminate_ws_bytes(n))
            return fail(HARL_E_WORKSPACE, "harl_track_eliminate: workspace smaller than harl_track_eliminate_workspace_size()");
    }
    return harl::track_eliminate_launch(d_adv, n, n_keep, d_keep_index, d_rows, row_bytes, d_rows_out, d_ws,
                                        static_cast<hipStream_t>(stream));
}

static int gbdt_check_params(const harl_gbdt_params *p) {
    if (!p) return fail(HARL_E_INVALID_ARG, "harl_gbdt: null parameters");
    if (p->max_depth < 1 || p->max_depth > HARL_GBDT_MAX_DEPTH)
        return fail(HARL_E_INVALID_ARG, "harl_gbdt: max_depth out of range");
    if (!(p->reg_lambda > 0.0) || !(p->gamma >= 0.0) || !(p->min_child_weight >= 0.0) || !std::isfinite(p->eta) ||
        !std::isfinite(p->reg_lambda) || !std::isfinite(p->gamma) || !std::isfinite(p->min_child_weight) ||
        !std::isfinite(p->base_score))
        return fail(HARL_E_INVALID_ARG, "harl_gbdt: hyper-parameter out of range");
    return HARL_OK;
}

static bool gbdt_sizes_ok(int32_t F, int32_t N, int32_t P) {
    return F >= 1 && F <= HARL_GBDT_MAX_FEATURES && N >= 0 && N <= (1 << 30) && P >= 0 && P <= (1 << 30);
}

int harl_gbdt_bin(const float *d_feat, int64_t ld_feat, int32_t n_features, int32_t n_rows, const float *d_cuts,
                  int32_t cut_stride, const int32_t *d_n_cuts, uint8_t *d_bins, int64_t ld_bins, void *stream) {
    if (!gbdt_sizes_ok(n_features, n_rows, 0)) return fail(HARL_E_INVALID_ARG, "harl_gbdt_bin: sizes out of range");
    if (ld_feat < n_rows || ld_bins < n_rows || cut_stride < 1)
        return fail(HARL_E_INVALID_ARG, "harl_gbdt_bin: need ld_feat >= n_rows, ld_bins >= n_rows, cut_stride >= 1");
    if (n_rows == 0) return HARL_OK;
    if (!d_feat || !aligned(d_feat, 4) || !d_cuts || !aligned(d_cuts, 4) || !d_n_cuts || !aligned(d_n_cuts, 4))
        return fail(HARL_E_INVALID_ARG, "harl_gbdt_bin: null or misaligned input");
    if (!d_bins || !aligned(d_bins, 8)) return fail(HARL_E_INVALID_ARG, "harl_gbdt_bin: bins null or not 8-byte aligned");
    return harl::gbdt_bin_launch(d_feat, ld_feat, n_features, n_rows, d_cuts, cut_stride, d_n_cuts, d_bins, ld_bins,
                                 static_cast<hipStream_t>(stream));
}

size_t harl_gbdt_round_workspace_size(const harl_gbdt_params *prm, int32_t n_features, int32_t n_rows, int32_t n_prog) {
    if (gbdt_check_params(prm) != HARL_OK || !gbdt_sizes_ok(n_features, n_rows, n_prog)) return 0;
    return harl::gbdt_ws_bytes(n_features, n_rows, n_prog, prm->max_depth);
}

int harl_gbdt_round(const harl_gbdt_params *prm, const uint8_t *d_bins, int64_t ld_bins, int32_t n_features,
                    int32_t n_rows, const float *d_cuts, int32_t cut_stride, const int32_t *d_n_cuts,
                    const int32_t *d_prog_ptr, int32_t n_prog, const float *d_label, const float *d_weight,
                    float *d_margin, int32_t *d_feature, float *d_threshold, int32_t *d_left, int32_t *d_right,
                    uint8_t *d_default_left, float *d_leaf_value, void *d_ws, size_t ws_bytes, void *stream) {
    if (const int rc = gbdt_check_params(prm)) return rc;
    if (!gbdt_sizes_ok(n_features, n_rows, n_prog)) return fail(HARL_E_INVALID_ARG, "harl_gbdt_round: sizes out of range");
    if (ld_bins < n_rows || cut_stride < 1)
        return fail(HARL_E_INVALID_ARG, "harl_gbdt_round: need ld_bins >= n_rows, cut_stride >= 1");
    if (n_rows > 0 && (!d_bins || !aligned(d_bins, 8)))
        return fail(HARL_E_INVALID_ARG, "harl_gbdt_round: bins null or not 8-byte aligned");
    const void *in4[] = {d_cuts, d_n_cuts, d_prog_ptr, d_feature, d_threshold, d_left, d_right, d_leaf_value};
    for (const void *p : in4)
        if (!p || !aligned(p, 4)) return fail(HARL_E_INVALID_ARG, "harl_gbdt_round: null or misaligned array");
    if (!d_default_left) return fail(HARL_E_INVALID_ARG, "harl_gbdt_round: null default_left");
    if (n_prog > 0 && (!d_label || !aligned(d_label, 4) || !d_weight || !aligned(d_weight, 4)))
        return fail(HARL_E_INVALID_ARG, "harl_gbdt_round: null or misaligned label / weight");
    if (n_rows > 0 && (!d_margin || !aligned(d_margin, 4)))
        return fail(HARL_E_INVALID_ARG, "harl_gbdt_round: null or misaligned margin");
    if (!d_ws || !aligned(d_ws, 256)) return fail(HARL_E_INVALID_ARG, "harl_gbdt_round: workspace null or not 256-byte aligned");
    if (ws_bytes < harl::gbdt_ws_bytes(n_features, n_rows, n_prog, prm->max_depth))
        return fail(HARL_E_WORKSPACE, "harl_gbdt_round: workspace smaller than harl_gbdt_round_workspace_size()");
    return harl::gbdt_round_launch(prm, d_bins, ld_bins, n_features, n_rows, d_cuts, cut_stride, d_n_cuts, d_prog_ptr,
                                   n_prog, d_label, d_weight, d_margin, d_feature, d_threshold, d_left, d_right,
                                   d_default_left, d_leaf_value, d_ws, static_cast<hipStream_t>(stream));
}

}  // extern "C"
