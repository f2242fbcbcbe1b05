/*
 * harl.h -- C ABI of libharl: one HARL search round's batched candidate evaluation on an MI355X.
 *
 * HARL (Zhang, He, Zhang, ICPP'22) searches tensor-program schedules with an actor/critic over
 * parameter modifications and scores every visited schedule with a learned cost model
 * (Algorithm 1; Sections 4.3 and 6.1).  One round of that loop, over all live candidates, is:
 *
 *   harl_policy_step  the actor pi_theta(M|S) picks each candidate's next modification and the
 *                     critic V(S) gives its value (Algorithm 1, action selection; Eq. 6);
 *   harl_score_round  the cost model C(S') scores every candidate: a gradient-boosted tree
 *                     ensemble (XGBoost in the paper, Section 6.1, Appendix A.1) applied to each
 *                     statement's feature row and summed over the program's statements;
 *   harl_topk         the top-K candidates by predicted score (Algorithm 1, top-K phase;
 *                     Section 4.3, Top-K Selection Phase), optionally merged into a running top-K
 *                     that plays the heap H accumulating candidates across steps (Algorithm 1).
 *
 * Around the round: harl_track_advantage / harl_track_eliminate (reward, advantage and the
 * adaptive-stopping elimination of schedule tracks; Eq. 6, Section 5), harl_policy_select (one
 * action per modification type, greedy or sampled; Section 4.3), harl_ppo_update (the actor/critic's
 * training step; Section 6.1) and harl_gbdt_bin / harl_gbdt_round (the cost model's refit on
 * measured programs; Algorithm 1, Section 6.1).
 *
 * Conventions for every call:
 *   - Return value is a harl_status; nothing else signals an error and no C++ exception crosses
 *     this interface.  harl_last_error() gives the message of the calling thread's last failure.
 *   - Host-visible arguments (pointers, sizes, workspace size, alignment) are checked before any
 *     HIP call; on failure nothing is launched and no output is touched.
 *   - Pointers named d_* are device pointers (HIP device memory of the current device), owned by
 *     the caller and left untouched beyond the documented outputs.  Pointers in *_desc structs are
 *     host pointers, read only during the create call.
 *   - `stream` is a hipStream_t (NULL = the default stream).  Hot-path calls are asynchronous
 *     and stream-ordered: they enqueue kernels and return; they allocate nothing and never
 *     synchronise.  Create/destroy calls allocate/free device memory and synchronise `stream`.
 *   - Device-content preconditions (e.g. a monotone prog_ptr) are the caller's to uphold; the
 *     kernels clamp every index they derive from device data, so a violation gives wrong numbers,
 *     never an out-of-bounds access.
 *   - Results are deterministic: fixed-order reductions, no floating-point atomics.
 */
#ifndef HARL_H
#define HARL_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    HARL_OK = 0,
    HARL_E_INVALID_ARG = -1, /* a null pointer, bad size, bad alignment or malformed model      */
    HARL_E_UNSUPPORTED = -2, /* a valid request outside what the library implements             */
    HARL_E_WORKSPACE = -3,   /* the workspace is smaller than the matching *_workspace_size()   */
    HARL_E_HIP = -4,         /* a HIP runtime call or kernel launch failed                      */
    HARL_E_NOMEM = -5        /* a device allocation failed (create calls only)                  */
} harl_status;

typedef enum { HARL_F32 = 0, HARL_BF16 = 1 } harl_dtype;

/* Message for the calling thread's last non-OK return ("" if none).  Valid until the next call. */
const char *harl_last_error(void);

/* Library version string, e.g. "harl 0.1 gfx950". */
const char *harl_version(void);

/* ============================================================================================
 * Cost model: a GBDT ensemble (Section 6.1 and Appendix A.1: XGBoost with Ansor's settings).
 * ============================================================================================ */

/*
 * Host description of a tree ensemble, in explicit node arrays over all trees.
 * Node n is a leaf iff feature[n] < 0; a leaf contributes leaf_value[n].  An internal node sends a
 * feature value x to left[n] iff x < threshold[n] (strict; x == threshold goes right); a missing
 * value (NaN) goes left iff default_left[n] != 0.  Tree t starts at node root[t].  Trees may be
 * irregular; a tree whose leaves sit at different depths is packed as a complete tree of its
 * ensemble's largest depth (an early leaf is repeated below dummy splits, which does not change
 * any result).  A NaN threshold sends every non-missing value right.
 * Limits: 1 <= n_trees; 1 <= n_features <= 448 (a 64-row feature tile must fit the LDS);
 * largest root-to-leaf depth <= 12;
 * every child id in [0, n_nodes); every tree acyclic.
 */
typedef struct {
    int32_t n_trees;
    int32_t n_features;
    int32_t n_nodes;              /* total nodes over all trees                                 */
    const int32_t *root;          /* [n_trees]                                                  */
    const int32_t *feature;       /* [n_nodes], < 0 for a leaf                                  */
    const float *threshold;       /* [n_nodes], read for internal nodes                         */
    const int32_t *left;          /* [n_nodes], read for internal nodes                         */
    const int32_t *right;         /* [n_nodes], read for internal nodes                         */
    const uint8_t *default_left;  /* [n_nodes], read for internal nodes                         */
    const float *leaf_value;      /* [n_nodes], read for leaves                                 */
    float base_score;             /* added once to every program's score                        */
} harl_ensemble_desc;

typedef struct harl_ensemble harl_ensemble;

/* Validate and pack `desc` into a library-owned device copy on the current device.  *out
 * receives the handle (NULL on failure).  Synchronises `stream`. */
int harl_ensemble_create(const harl_ensemble_desc *desc, harl_ensemble **out, void *stream);
/* Free a handle (NULL is a no-op).  The caller must not destroy it while work using it runs. */
int harl_ensemble_destroy(harl_ensemble *ens);
/* Packed depth and tree count of a handle (for sizing); returns HARL_E_INVALID_ARG on NULL. */
int harl_ensemble_info(const harl_ensemble *ens, int32_t *n_trees, int32_t *depth, int32_t *n_features);

/* Bytes of device workspace harl_score_round needs for n_rows statement rows. */
size_t harl_score_round_workspace_size(const harl_ensemble *ens, int32_t n_rows, int32_t n_prog);

/*
 * Cost-model scores of one round's candidates (Algorithm 1: C(S') for every new schedule).
 *
 *   d_feat      [n_features][ld] fp32, feature-major: feature f of statement row r is
 *               d_feat[f*ld + r].  4-byte aligned, ld >= n_rows; 16-byte alignment with
 *               ld % 4 == 0 lets the kernel stage rows with 16-byte loads.
 *   n_rows      statement rows in this round (>= 0).
 *   d_prog_ptr  [n_prog+1] int32: program p owns rows [d_prog_ptr[p], d_prog_ptr[p+1]);
 *               0 = d_prog_ptr[0] <= ... <= d_prog_ptr[n_prog] = n_rows (caller's precondition).
 *   d_prog_score [n_prog] fp32 out: base_score + sum of its statements' ensemble sums.
 *   d_stmt_score [n_rows] fp32 out, or NULL: each statement row's ensemble sum.
 *   d_ws, ws_bytes  device workspace of at least harl_score_round_workspace_size() bytes,
 *               256-byte aligned; its contents on entry are ignored.
 * Sums over trees (on the binned path of 8- to 10-level ensembles in fp32 over at most 16 trees
 * at a time, then in fp64) and over a program's statements (fp64) are accumulated in a fixed order
 * and rounded once to fp32.  n_prog == 0 is a no-op.
 */
int harl_score_round(const harl_ensemble *ens, const float *d_feat, int64_t ld, int32_t n_rows,
                     const int32_t *d_prog_ptr, int32_t n_prog, float *d_prog_score,
                     float *d_stmt_score, void *d_ws, size_t ws_bytes, void *stream);

/* ============================================================================================
 * Actor / critic (Section 4.3; Algorithm 1; Eq. 6 defines the critic's use).
 * ============================================================================================ */

/*
 * Host description of the actor/critic: a shared trunk h1 = ReLU(W1 s + b1),
 * h2 = ReLU(W2 h1 + b2), an actor head logits = Wa h2 + ba and a value head v = wv . h2 + bv.
 * Weights are [out][in] row-major (PyTorch nn.Linear layout): fp32 for HARL_F32, raw bf16 bit
 * patterns (uint16) for HARL_BF16.  Biases are fp32.  A HARL_BF16 policy takes bf16 states, uses
 * bf16 x bf16 products with fp32 accumulation, and rounds h1 and h2 to bf16 (nearest, ties to
 * even) after bias and ReLU; a HARL_F32 policy is fp32 throughout.
 * Limits: 1 <= s <= 1024; 1 <= h1, h2 <= 4096; 1 <= a <= 127.
 */
typedef struct {
    harl_dtype dtype;
    int32_t s, h1, h2, a;
    const void *w1;   /* [h1][s]  */
    const float *b1;  /* [h1]     */
    const void *w2;   /* [h2][h1] */
    const float *b2;  /* [h2]     */
    const void *wa;   /* [a][h2]  */
    const float *ba;  /* [a]      */
    const void *wv;   /* [h2]     */
    const float *bv;  /* [1]      */
} harl_policy_desc;

typedef struct harl_policy harl_policy;

/* Validate and pre-tile the weights into a library-owned device copy.  Synchronises `stream`. */
int harl_policy_create(const harl_policy_desc *desc, harl_policy **out, void *stream);
int harl_policy_destroy(harl_policy *pol);

/*
 * Actor/critic forward for B states (Algorithm 1: select M with pi_theta(M|S); critic V(S)).
 *   d_states  [B][s] row-major, fp32 or bf16 bits per the policy's dtype; 16-byte aligned.
 *   d_action  [B] int32 out: the lowest index attaining the largest logit.
 *   d_value   [B] fp32 out: the critic's value.
 *   d_probs   [B][a] fp32 out, or NULL: softmax of the logits.
 *   d_logits  [B][a] fp32 out, or NULL: the actor's logits.
 * B == 0 is a no-op.
 */
int harl_policy_step(const harl_policy *pol, const void *d_states, int32_t B, int32_t *d_action,
                     float *d_value, float *d_probs, float *d_logits, void *stream);

/* ============================================================================================
 * Top-K selection (Algorithm 1, top-K phase) and the running heap H.
 * ============================================================================================ */

#define HARL_TOPK_MAX_K 2048
/* flags for harl_topk */
#define HARL_TOPK_MERGE 1u

/* Bytes of device workspace harl_topk needs for n scores and a given k. */
size_t harl_topk_workspace_size(int32_t n, int32_t k);

/*
 * The k best of n scores, ranked by (score descending, index ascending); score -0 ties +0 and
 * NaN ranks below every number.  Candidate i carries the global index index_base + i.
 *   d_score              [n] fp32 in, 4-byte aligned.
 *   d_io_score/io_index  [k] fp32 / int64.  Without HARL_TOPK_MERGE they receive the top k of
 *                        this call (k <= n required).  With HARL_TOPK_MERGE they must hold a
 *                        running top-k (ranked as above, e.g. from harl_topk_reset or an earlier
 *                        call) and are replaced by the top k of their union with this call's n
 *                        candidates (any n >= 0).  Output scores are bit copies of the inputs.
 *   d_ws, ws_bytes       workspace of at least harl_topk_workspace_size(n, k) bytes,
 *                        256-byte aligned.
 * 1 <= k <= HARL_TOPK_MAX_K (k == 0 is a no-op); n >= 0; index_base >= 0 and
 * index_base + n < 2^62.
 */
int harl_topk(const float *d_score, int32_t n, int32_t k, int64_t index_base, float *d_io_score,
              int64_t *d_io_index, uint32_t flags, void *d_ws, size_t ws_bytes, void *stream);

/* Fill a running top-k with the empty sentinel (-inf, INT64_MAX) in every slot. */
int harl_topk_reset(float *d_io_score, int64_t *d_io_index, int32_t k, void *stream);

/*
 * For callers that cannot allocate device memory (work recorded under stream or graph capture,
 * tight serving loops, harnesses that forbid hipMalloc): harl_topk without a workspace argument.
 * Its candidate buffers are a library-owned device array of HARL_TOPK_STATIC_SCRATCH_BYTES per
 * device, held from the first call on that device until the process ends; the call itself
 * allocates nothing.  Arguments, results and errors as harl_topk, plus HARL_E_UNSUPPORTED when
 * harl_topk_workspace_size(n, k) exceeds HARL_TOPK_STATIC_SCRATCH_BYTES (k = 2048 allows
 * n <= 2,088,960; k = 1024, n <= 4,186,112; k = 128, n <= 33,546,240).  Every call on one device shares that device's
 * array: calls that may overlap on one device (other streams, other host threads) race and must be
 * ordered by the caller; each call writes the buffers before it reads them, so nothing carries over.
 */
#define HARL_TOPK_STATIC_SCRATCH_BYTES (8u << 20)
int harl_topk_static(const float *d_score, int32_t n, int32_t k, int64_t index_base, float *d_io_score,
                     int64_t *d_io_index, uint32_t flags, void *stream);

/* ============================================================================================
 * Per-modification-type action selection (Section 4.3: the best modification of each type;
 * Appendix A.1: num_iters^2 + 1 tile-size actions and 3 per other type; Section 6.1: PPO rollouts
 * sample the actions).
 * ============================================================================================ */

#define HARL_SELECT_MAX_SEGMENTS 32
/* flags for harl_policy_select */
#define HARL_SELECT_SAMPLE 1u

/*
 * One action per modification type from the actor's logits (e.g. the d_logits output of
 * harl_policy_step).  Each row of a logits is cut into n_seg consecutive segments, one per type:
 * segment s holds actions [seg_offsets[s], seg_offsets[s + 1]).  Per state and segment:
 *   action  the lowest index attaining the maximum logit (greedy), or with HARL_SELECT_SAMPLE the
 *           lowest index attaining the maximum of logit + Gumbel noise, a draw from the segment's
 *           softmax.  The noise of logit i of state b is -log(-log(u)), u = (w + 0.5) * 2^-24 with
 *           w the top 24 bits of word i % 4 of Philox4x32-10 (Salmon et al., SC'11) at counter
 *           (i / 4, b, counter low word, counter high word) and key (seed low word, seed high
 *           word); noise and comparison are fp64.  NaN logits never win; a segment without a
 *           number above -inf picks its first action.  Indices are row-global (0 .. a-1).
 *   logp    the chosen action's log-probability under the segment's softmax (fp32).
 *   probs   the segment-wise softmax of the row (fp32).
 *   d_logits       [B][a] fp32 in, 4-byte aligned.
 *   seg_offsets    HOST array [n_seg + 1]: 0 = o_0 < o_1 < ... < o_n_seg = a.
 *   d_action       [B][n_seg] int32 out.
 *   d_logp         [B][n_seg] fp32 out, or NULL.
 *   d_probs        [B][a] fp32 out, or NULL.
 * 1 <= n_seg <= HARL_SELECT_MAX_SEGMENTS; 1 <= a <= 4096; B >= 0 (B == 0 is a no-op); the same
 * (seed, counter) gives the same draws, so a rollout step passes a fresh counter.
 */
int harl_policy_select(const float *d_logits, int32_t B, int32_t a, const int32_t *seg_offsets,
                       int32_t n_seg, uint32_t flags, uint64_t seed, uint64_t counter,
                       int32_t *d_action, float *d_logp, float *d_probs, void *stream);

/* ============================================================================================
 * PPO update of the actor/critic (Algorithm 1: train the actor with the policy gradient of Eq. 5
 * and the critic with the MSE of the advantage Y; Section 6.1: PPO; Table 5: weights and rates).
 * ============================================================================================ */

/* Sizes and hyper-parameters of the trained fp32 network (the shared trunk of harl_policy_desc
 * with the per-type actor head of harl_policy_select and a value head). */
typedef struct {
    int32_t s, h1, h2, a;      /* input, hidden and action sizes: 1..1024, 1..4096, 1..4096, 1..4096 */
    int32_t n_seg;             /* modification types, 1..HARL_SELECT_MAX_SEGMENTS */
    int32_t seg_offsets[HARL_SELECT_MAX_SEGMENTS + 1];  /* 0 = o_0 < ... < o_n_seg = a */
    float clip_eps;            /* PPO clip range (0.2) */
    float w_value, w_entropy;  /* loss weights (0.5, 0.01; Table 5) */
    float lr_actor, lr_critic; /* Adam rates: trunk + actor head, value head (3e-4, 1e-3; Table 5) */
    float beta1, beta2, adam_eps;  /* Adam (0.9, 0.999, 1e-8) */
} harl_ppo_config;

/* Floats of the packed parameters W1 [h1][s], b1, W2 [h2][h1], b2, Wa [a][h2], ba, wv [h2], bv
 * (PyTorch nn.Linear layout, in that order); also the length of the gradient and Adam moments. */
size_t harl_ppo_param_count(const harl_ppo_config *cfg);
/* Bytes of device workspace harl_ppo_update needs for a mini-batch of M transitions. */
size_t harl_ppo_workspace_size(const harl_ppo_config *cfg, int32_t M);

/*
 * One PPO update on a mini-batch of M transitions, in fp32 on the device:
 *   loss = -mean(min(ratio A, clip(ratio, 1 - clip_eps, 1 + clip_eps) A))
 *          + w_value mean((V(s) - R)^2) - w_entropy mean(H),
 *   ratio = exp(logp - logp_old), logp = sum over types of the chosen actions' log-softmax,
 *   H = sum over types of the segment entropies;
 * then its gradient (backpropagation through the trunk; min passes the gradient to the unclipped
 * term on equality, clip inside its closed range, ReLU's derivative at 0 is 0) and one Adam step
 * (bias correction with the 1-based `step`).
 *   d_params [P] in/out, d_adam_m / d_adam_v [P] in/out (zero before the first step),
 *   P = harl_ppo_param_count(cfg).
 *   d_states [M][s] fp32; d_actions [M][n_seg] int32 (row-global indices, each in its segment;
 *   others are clamped into it); d_logp_old, d_adv, d_ret [M] fp32 (the behaviour policy's
 *   log-probability, the advantage of Eq. 6 and the critic's target R).
 *   d_grad   [P] out, or NULL: the gradient of this step.
 *   d_loss   [4] out, or NULL: total, clipped-surrogate, value-MSE and entropy terms.
 *   d_ws, ws_bytes: at least harl_ppo_workspace_size(cfg, M) bytes, 256-byte aligned.
 * All device arrays 4-byte aligned.  M == 0 is a no-op; step >= 1.  Deterministic.
 */
int harl_ppo_update(const harl_ppo_config *cfg, float *d_params, float *d_adam_m, float *d_adam_v,
                    int32_t step, const float *d_states, const int32_t *d_actions,
                    const float *d_logp_old, const float *d_adv, const float *d_ret, int32_t M,
                    float *d_grad, float *d_loss, void *d_ws, size_t ws_bytes, void *stream);

/* ============================================================================================
 * Schedule tracks between rounds: reward and advantage of a modification step (Algorithm 1,
 * Eq. 6) and the adaptive-stopping elimination (Section 5).
 * ============================================================================================ */

/*
 * Reward and advantage of one modification step of n schedule tracks.  Track i moved from state s
 * (cost-model score d_c_prev[i], critic value d_v_prev[i]) to s' (d_c_next[i], d_v_next[i]):
 *   reward     r = (C(s') - C(s)) / max(|C(s)|, eps)     (Algorithm 1's relative score change;
 *                  the denominator is read as max(|C(s)|, eps) so that signed scores keep the sign
 *                  of an improvement and a zero score stays finite)
 *   advantage  A = r + gamma * V(s') - V(s)             (Eq. 6; the paper uses gamma = 0.9)
 * computed in fp32.  All arrays [n] fp32, 4-byte aligned, device memory; d_reward may be NULL.
 * NaN inputs propagate.  n == 0 is a no-op; eps must be > 0 and finite.
 */
int harl_track_advantage(const float *d_c_prev, const float *d_c_next, const float *d_v_prev,
                         const float *d_v_next, int32_t n, float gamma, float eps, float *d_reward,
                         float *d_adv, void *stream);

/*
 * Tracks kept by one adaptive-stopping elimination (Section 5: after every window of lambda steps
 * the proportion rho of the tracks with the lowest advantage is eliminated): the eliminated count
 * is floor(rho * n), computed in double precision, so *n_keep = n - floor(rho * n).  Host-only
 * arithmetic (no device call); 0 <= rho <= 1 (the paper uses rho = 0.5), n >= 0.
 */
int harl_track_keep_count(int32_t n, double rho, int32_t *n_keep);

/* Bytes of device workspace harl_track_eliminate needs for n tracks. */
size_t harl_track_eliminate_workspace_size(int32_t n);

/*
 * Adaptive-stopping elimination (Section 5): rank the n tracks by advantage (descending; NaN
 * behind every number; -0 ties +0; then lower track index) and keep the first n_keep, i.e. drop
 * the n - n_keep of lowest advantage (the paper drops the proportion rho = 0.5 every lambda = 20
 * steps while at least 64 tracks remain; the caller chooses n_keep).
 *   d_adv          [n] fp32 in, 4-byte aligned.
 *   d_keep_index   [n_keep] int32 out: the surviving tracks' indices in ascending order.
 *   d_rows         [n][row_bytes] in, or NULL: per-track rows (e.g. the policy states);
 *   d_rows_out     [n_keep][row_bytes] out, or NULL: the survivors' rows in d_keep_index order
 *                  (both or neither of d_rows / d_rows_out; row_bytes >= 1; no overlap).
 *   d_ws, ws_bytes workspace of at least harl_track_eliminate_workspace_size(n) bytes,
 *                  256-byte aligned; its contents on entry do not matter.
 * 0 <= n_keep <= n; n_keep == 0 is a no-op.  The result is exact and deterministic.
 */
int harl_track_eliminate(const float *d_adv, int32_t n, int32_t n_keep, int32_t *d_keep_index,
                         const void *d_rows, int64_t row_bytes, void *d_rows_out, void *d_ws,
                         size_t ws_bytes, void *stream);

/* ============================================================================================
 * Refit of the cost model on measured programs (Algorithm 1: the top-K states are measured and
 * the cost model is trained on (S^, P); Section 6.1 and Appendix A.1: XGBoost with Ansor's
 * settings).  Histogram-based gradient boosting (Chen and Guestrin, KDD'16, Sections 3 and 3.4).
 * ============================================================================================ */

#define HARL_GBDT_MAX_DEPTH 12
#define HARL_GBDT_MAX_CUTS 254
#define HARL_GBDT_MAX_FEATURES 4096

/*
 * Feature binning.  Feature f of statement row r is d_feat[f*ld_feat + r] (the feature-major
 * layout harl_score_round reads); its cut points are d_cuts[f*cut_stride + i], i < d_n_cuts[f]
 * (strictly increasing, finite; d_n_cuts[f] is clamped to [0, min(254, cut_stride)]).
 *   d_bins  out, in groups of 8 features: the bin of feature f of row r is the byte
 *           d_bins[((f/8)*ld_bins + r)*8 + f%8], the number of cut points <= x, or 255 for NaN
 *           (missing); the bytes of features n_features .. 8*ceil(n_features/8)-1 are 0.  The
 *           array holds ceil(n_features/8) planes of ld_bins rows of 8 bytes; rows >= n_rows are
 *           not written.
 * ld_bins >= n_rows; d_bins 8-byte aligned; other arrays 4-byte aligned.  n_rows == 0 is a
 * no-op.  Exact.
 */
int harl_gbdt_bin(const float *d_feat, int64_t ld_feat, int32_t n_features, int32_t n_rows,
                  const float *d_cuts, int32_t cut_stride, const int32_t *d_n_cuts, uint8_t *d_bins,
                  int64_t ld_bins, void *stream);

/* Boosting hyper-parameters (Ansor's cost model: max_depth 10, eta 0.2, gamma 0.001,
 * min_child_weight 0; XGBoost's default reg_lambda 1). */
typedef struct {
    int32_t max_depth;       /* 1 .. HARL_GBDT_MAX_DEPTH                          */
    double eta;              /* learning rate (shrinkage of the leaf weights)     */
    double reg_lambda;       /* L2 regularisation of the leaf weights, > 0        */
    double gamma;            /* minimum gain of a split, >= 0                      */
    double min_child_weight; /* minimum hessian sum of a child, >= 0               */
    double base_score;       /* added once to every program's prediction          */
} harl_gbdt_params;

/* Bytes of device workspace harl_gbdt_round needs. */
size_t harl_gbdt_round_workspace_size(const harl_gbdt_params *prm, int32_t n_features, int32_t n_rows,
                                      int32_t n_prog);

/*
 * One boosting round on measured programs under the pack-sum squared error: program p's
 * prediction is s_p = base_score + the sum of its statements' margins, the objective
 * 1/2 sum_p w_p (s_p - y_p)^2, so each statement row of p carries gradient w_p (s_p - y_p) and
 * hessian w_p.  The tree grows depth-wise: a node takes the split (feature f, threshold index t
 * in 1 .. n_cuts[f], missing direction) of largest gain
 *   GL^2/(HL + lambda) + GR^2/(HR + lambda) - G^2/(H + lambda)
 * (ties: lowest f, then lowest t, then missing-left) among those whose children's hessian sums
 * reach min_child_weight, and splits iff that gain exceeds gamma; a leaf holds
 * -(G / (H + lambda)) * eta.  Gradient and hessian sums are exact: each program's value is rounded
 * once to the grid 2^-e, e = 62 - ceil(log2 n_rows) - E for the largest magnitude m 2^E
 * (1/2 <= m < 1), and summed as 64-bit integers; gains are fp64.  The result does not depend on
 * scheduling.
 *   d_bins, ld_bins  the bins in harl_gbdt_bin's layout (each byte <= its feature's n_cuts, or
 *              255); 8-byte aligned, ld_bins >= n_rows.
 *   d_cuts, cut_stride, d_n_cuts   the cut points the bins were made with (thresholds).
 *   d_prog_ptr [n_prog+1] int32: program p owns rows [d_prog_ptr[p], d_prog_ptr[p+1]),
 *              0 = d_prog_ptr[0] <= ... <= d_prog_ptr[n_prog] = n_rows.
 *   d_label, d_weight [n_prog] fp32: measured target and weight (finite, weight >= 0).
 *   d_margin   [n_rows] fp32 in/out: each row's sum over the trees so far; the new tree's leaf
 *              value is added (fp32).
 *   d_feature, d_threshold, d_left, d_right, d_default_left, d_leaf_value: the new tree, node
 *              arrays of 2^(max_depth+1) - 1 entries (the harl_ensemble_desc fields), children of
 *              node k at 2k+1 and 2k+2; a split node sends x < threshold left; nodes the tree does
 *              not reach hold feature -1 and leaf value 0.
 *   d_ws, ws_bytes: at least harl_gbdt_round_workspace_size() bytes, 256-byte aligned; contents
 *              on entry do not matter.
 * n_rows == 0 gives a single leaf of value -0.  Errors: HARL_E_INVALID_ARG for sizes, parameters
 * or alignment out of range, HARL_E_WORKSPACE for a short workspace.
 */
int harl_gbdt_round(const harl_gbdt_params *prm, const uint8_t *d_bins, int64_t ld_bins,
                    int32_t n_features, int32_t n_rows, const float *d_cuts, int32_t cut_stride,
                    const int32_t *d_n_cuts, const int32_t *d_prog_ptr, int32_t n_prog,
                    const float *d_label, const float *d_weight, float *d_margin, int32_t *d_feature,
                    float *d_threshold, int32_t *d_left, int32_t *d_right, uint8_t *d_default_left,
                    float *d_leaf_value, void *d_ws, size_t ws_bytes, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* HARL_H */
