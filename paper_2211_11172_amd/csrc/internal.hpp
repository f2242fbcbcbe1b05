// Internal declarations shared by the libharl translation units (not part of the ABI).
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>
#include <string>
#include <vector>

#include "../../include/harl.h"

namespace harl {

// Thread-local error text behind harl_last_error().
int fail(int status, const std::string &msg);
int hip_fail(hipError_t e, const char *what);

#define HARL_HIP_CHECK(expr)                                      \
    do {                                                          \
        hipError_t _e = (expr);                                   \
        if (_e != hipSuccess) return ::harl::hip_fail(_e, #expr); \
    } while (0)

// Raise a kernel's dynamic-LDS limit to at least `bytes` on the current device; the attribute is
// set once per (kernel, device) and remembered, so hot-path launches make no extra runtime call.
int ensure_dynamic_lds(const void *kernel, size_t bytes);

inline bool aligned(const void *p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }
inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }
inline int64_t round_up(int64_t a, int64_t b) { return ceil_div(a, b) * b; }

// ------------------------------------------------------------------------------------------
// Packed GBDT ensemble.  Every tree is stored as a complete binary tree of `depth` split levels
// (an early leaf repeats below dummy splits), in the record layout described in score.hip: 8-byte
// records {threshold, children's feature codes} for the upper levels and 16-byte records
// {threshold, left leaf, right leaf, 0} for the last split level.  A feature code is the split
// feature (< 2^15) with bit 15 set when missing values go left.
// ------------------------------------------------------------------------------------------
constexpr int kMaxDepth = 12;
constexpr int kMaxFeatures = 448;
constexpr int kMinB16Depth = 8, kMaxB16Depth = 10;  // ensemble depths the binned path (score_bin.hip) walks
// Statement rows from which a depth-8 ensemble is scored on the binned path (its binning pass costs
// more than it saves on smaller rounds); deeper ensembles take it at any size.
constexpr int32_t kB16MinRowsDepth8 = 1 << 17;

}  // namespace harl

struct harl_ensemble {
    int32_t n_trees;
    int32_t n_features;
    int32_t depth;
    int32_t tree_stride;  // bytes per packed tree (multiple of 16)
    float base_score;
    int device;
    void *d_trees;        // n_trees * tree_stride bytes
    // launch shape of the fp32 walk, chosen once at create
    int32_t cfg_wp, cfg_a, cfg_b, cfg_c;
    // tree groups forced at create (HARL_SCORE_TREE_GROUPS, for tests of the grouped layout); 0 = automatic
    int32_t tree_groups_override;
    // binned-path row threshold forced at create (HARL_SCORE_BINNED_MIN_ROWS, for tests); -1 = automatic
    int32_t b16_min_rows_override;
    // binned path (score_bin.hip), or null when the ensemble does not qualify: packed trees of
    // b16_stride bytes, per-feature distinct thresholds (offsets and counts per feature)
    void *d_trees_b16;
    float *d_thr_b16;                         // per feature: sorted thresholds + NaN padding
    int32_t *d_thr_off_b16, *d_thr_len_b16;   // their offsets and lengths (padding included)
    int32_t *d_search_b16;                    // per feature: {probes | key shift << 8, bucket base}
    uint16_t *d_lut_b16;                      // per feature: thresholds below each of 4,096 key buckets
    float *d_leaves_b16;                      // tails: per tree level D-2's records and the leaves
    int32_t b16_stride, tree_groups_b16;
    int32_t b16_common_steps;                 // the probe count of the most features
    int32_t b16_min_rows;                     // rounds of fewer statement rows take the fp32 walk
};

// ------------------------------------------------------------------------------------------
// Packed actor/critic.  Weights are pre-tiled into the exact per-lane MFMA operand order of the
// policy kernel (one coalesced load per fragment); see policy.hip for the fragment layouts.
// ------------------------------------------------------------------------------------------
struct harl_policy {
    harl_dtype dtype;
    int32_t s, h1, h2, a;        // logical sizes
    int32_t sp, h1p, h2p, hap;   // padded sizes: input, hidden 1, hidden 2, heads (a+1 rounded)
    int device;
    void *d_w1, *d_w2, *d_wh;    // fragment-ordered weights
    float *d_b1, *d_b2, *d_bh;   // padded biases (bh = [ba; bv; 0...])
    // large-batch bf16 kernel (policy_x32.hip): chunked weight stream and accumulator-order biases;
    // x32_stream is null when the shape is outside that kernel's limits
    void *x32_stream, *x32_bias;
    int32_t x32_ks2, x32_ht, x32_nt1, x32_nt2, x32_chunk;
};

namespace harl {

// Launchers (stream-ordered, no allocation, no sync).  Arguments are already validated.
int score_round_launch(const harl_ensemble *E, const float *X, int64_t ld, int32_t n_rows,
                       const int32_t *prog_ptr, int32_t n_prog, float *prog_score, float *stmt_score,
                       void *ws, size_t ws_bytes, hipStream_t stream);
size_t score_round_ws_bytes(const harl_ensemble *E, int32_t n_rows);
int pack_ensemble(const harl_ensemble_desc *desc, harl_ensemble **out, hipStream_t stream);
void free_ensemble(harl_ensemble *E);
// binned path (score_bin.hip)
int pack_b16(harl_ensemble *E, const std::vector<int32_t> &feat, const std::vector<float> &thr,
             const std::vector<uint8_t> &dleft, const std::vector<float> &leaf, hipStream_t stream);
void free_b16(harl_ensemble *E);
bool score_b16_packed(const harl_ensemble *E);
bool score_b16_usable(const harl_ensemble *E, int32_t n_rows);
size_t score_b16_ws_bytes(const harl_ensemble *E, int32_t n_rows);
int score_b16_launch(const harl_ensemble *E, const float *X, int64_t ld, int32_t n_rows, float **partial_out,
                     int *groups_out, int *tiles_out, int *nbg_out, void *ws, size_t ws_bytes, hipStream_t stream);

int pack_policy(const harl_policy_desc *desc, harl_policy **out, hipStream_t stream);
bool policy_x32_eligible(const harl_policy_desc *desc);
int pack_policy_x32(const harl_policy_desc *desc, harl_policy *P, hipStream_t stream);
int policy_x32_launch(const harl_policy *P, const void *states, int32_t B, int32_t *action, float *value,
                      float *probs, float *logits, hipStream_t stream);
int policy_step_launch(const harl_policy *P, const void *states, int32_t B, int32_t *action,
                       float *value, float *probs, float *logits, hipStream_t stream);

size_t topk_ws_bytes(int32_t n, int32_t k);
int topk_launch(const float *score, int32_t n, int32_t k, int64_t index_base, float *io_score,
                int64_t *io_index, uint32_t flags, void *ws, size_t ws_bytes, hipStream_t stream);
int topk_reset_launch(float *io_score, int64_t *io_index, int32_t k, hipStream_t stream);
int topk_scratch(void **out);

int track_advantage_launch(const float *c_prev, const float *c_next, const float *v_prev, const float *v_next, int32_t n,
                           float gamma, float eps, float *reward, float *adv, hipStream_t stream);
size_t track_eliminate_ws_bytes(int32_t n);
size_t ppo_param_count(const harl_ppo_config *c);
size_t ppo_ws_bytes(const harl_ppo_config *c, int32_t M);
int ppo_update_launch(const harl_ppo_config *c, float *params, float *adam_m, float *adam_v, int32_t step,
                      const float *X, const int32_t *actions, const float *logp_old, const float *adv, const float *ret,
                      int32_t M, float *grad_out, float *loss_out, void *ws, hipStream_t stream);
int policy_select_launch(const float *logits, int32_t B, int32_t a, const int32_t *seg_offsets, int32_t n_seg,
                         uint32_t flags, uint64_t seed, uint64_t counter, int32_t *action, float *logp, float *probs,
                         hipStream_t stream);
int track_eliminate_launch(const float *adv, int32_t n, int32_t n_keep, int32_t *keep_index, const void *rows,
                           int64_t row_bytes, void *rows_out, void *ws, hipStream_t stream);

size_t gbdt_ws_bytes(int32_t F, int32_t N, int32_t P, int32_t depth);
int gbdt_bin_launch(const float *x, int64_t ldx, int32_t F, int32_t N, const float *cuts, int32_t cut_stride,
                    const int32_t *n_cuts, uint8_t *bins, int64_t ld, hipStream_t stream);
int gbdt_round_launch(const harl_gbdt_params *prm, const uint8_t *bins, int64_t ld, int32_t F, int32_t N,
                      const float *cuts, int32_t cut_stride, const int32_t *n_cuts, const int32_t *prog_ptr,
                      int32_t P, const float *label, const float *weight, float *margin, int32_t *feature,
                      float *threshold, int32_t *left, int32_t *right, uint8_t *default_left, float *leaf_value,
                      void *ws, hipStream_t stream);

}  // namespace harl
