/*
 * harl_oracle.c -- TEST INFRASTRUCTURE, not part of the product path.
 *
 * A plain, slow, obviously correct CPU implementation of one HARL search round's candidate
 * evaluation, written from the paper (Zhang, He, Zhang: "HARL: Hierarchical Adaptive
 * Reinforcement Learning Based Auto Scheduler for Neural Networks", ICPP'22):
 *
 *   oracle_score_round   cost-model prediction C(S') of every candidate (Algorithm 1, the reward
 *                        step and the heap-insert step; Section 4.3; the cost model is XGBoost,
 *                        Section 6.1 and Appendix A.1), here a GBDT applied to each statement's
 *                        feature row and summed over the statements of a program;
 *   oracle_policy_step   actor pi_theta(M|S) and critic V(S) forward (Algorithm 1, action
 *                        selection; Eq. 6 for the critic's role; Section 4.3), a shared ReLU
 *                        trunk with a linear actor head and a linear value head;
 *   oracle_topk          "select top-K states from the heap H" (Algorithm 1, top-K phase;
 *                        Section 4.3, Top-K Selection Phase): the K best predicted scores;
 *   oracle_merge         the heap H accumulating candidates across steps (Algorithm 1);
 *   oracle_track_advantage  reward of a modification step (Algorithm 1) and the advantage of
 *                        Eq. 6 for every schedule track;
 *   oracle_track_eliminate  adaptive-stopping elimination of the tracks with the lowest
 *                        advantages (Section 5);
 *   oracle_policy_select  one action per modification type from the actor's logits (Section 4.3:
 *                        the best modification of each type; Appendix A.1: num_iters^2 + 1 tile
 *                        actions and 3 for each other type), greedy or sampled as PPO rollouts
 *                        do (Section 6.1), with the per-type softmax and log-probability;
 *   oracle_philox4x32    the counter-based generator the sampling draws from (Salmon, Moraes,
 *                        Dror, Shaw: "Parallel random numbers: as easy as 1, 2, 3", SC'11).
 *
 * All arithmetic on scores and activations is fp64 over the given fp32 / bf16 input values.
 * Nothing here is blocked, fused or reordered beyond the definitions.  Only tests/, the package's
 * smoke check and bench.py's CPU-baseline leg may load this library; the HIP path shares no code
 * with it.  Built with plain -O2 (never -ffast-math: NaN tests must survive).
 *
 * Readings where the paper is silent:
 *   - a split sends x left iff x < threshold (strict), x == threshold goes right;
 *   - only NaN is missing; a missing value follows the node's default direction;
 *   - a program's score is base_score + the sum of its statements' scores;
 *   - larger score is better; ranking is by (score desc, index asc); -0 ties +0; NaN ranks last;
 *   - bf16 policies round the hidden activations h1, h2 to bf16 (nearest, ties to even) after
 *     bias and ReLU; fp32 policies keep them exact (fp64 here);
 *   - the action is the lowest index attaining the maximum logit; probabilities are the softmax
 *     of the logits;
 *   - the reward's denominator C(s) is taken as max(|C(s)|, eps): the paper's scores are
 *     positive, signed scores keep the sign of an improvement and a zero score stays finite;
 *   - elimination ranks tracks like top-K (advantage desc, NaN last, -0 ties +0, then lower track
 *     index), keeps a given number of them and lists the survivors in ascending track order;
 *   - the actor's logits are one flat row cut into consecutive segments, one per modification
 *     type; a segment's action is the lowest index attaining its maximum (of the logits, or of
 *     logit + Gumbel noise when sampling); NaN logits never win; a segment of only NaN / -inf
 *     logits picks its first action;
 *   - the Gumbel noise of logit i of state b is -log(-log(u)), u = (w + 0.5) * 2^-24 from the top
 *     24 bits w of word i % 4 of Philox4x32-10(counter = (i / 4, b, counter_lo, counter_hi),
 *     key = (seed_lo, seed_hi)).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define ORACLE_OK 0
#define ORACLE_EINVAL (-1)
#define ORACLE_ENOMEM (-5)

static void set_threads(int n_threads) {
#ifdef _OPENMP
    if (n_threads > 0) omp_set_num_threads(n_threads);
#else
    (void)n_threads;
#endif
}

int oracle_max_threads(void) {
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* ------------------------------------------------------------------------------------------- */
/* Cost model: GBDT over per-statement feature rows, summed per program                         */
/* ------------------------------------------------------------------------------------------- */

/* Walk one tree from its root for statement row r; return the reached leaf's node id, or -1 if the
 * walk does not end within n_nodes steps or leaves the node range (a malformed tree). */
static int64_t walk_tree(int32_t root, int32_t n_nodes, const int32_t *feature, const float *threshold,
                         const int32_t *left, const int32_t *right, const uint8_t *default_left,
                         const float *X, int64_t ld, int32_t n_features, int64_t r) {
    int64_t n = root;
    for (int32_t step = 0; step <= n_nodes; ++step) {
        if (n < 0 || n >= n_nodes) return -1;
        int32_t f = feature[n];
        if (f < 0) return n;                       /* a leaf */
        if (f >= n_features) return -1;
        float v = X[(int64_t)f * ld + r];
        if (isnan(v))
            n = default_left[n] ? left[n] : right[n];
        else
            n = (v < threshold[n]) ? left[n] : right[n];
    }
    return -1;
}

/*
 * For every program p and statement row r in [prog_ptr[p], prog_ptr[p+1]):
 *     stmt[r]  = sum over trees t of leaf_t(x_r)                    (fp64)
 *     prog[p]  = base_score + sum over its rows of stmt[r]          (fp64)
 *     scale[p] = |base_score| + sum over its rows and trees of |leaf_t(x_r)|
 * X is feature-major: feature f of row r is X[f*ld + r].  Outputs are fp64; stmt may be NULL.
 * Returns 0, or -1 on a malformed input (bad prog_ptr, malformed tree).
 */
int oracle_score_round(int32_t n_trees, int32_t n_nodes, const int32_t *root, const int32_t *feature,
                       const float *threshold, const int32_t *left, const int32_t *right,
                       const uint8_t *default_left, const float *leaf_value, double base_score,
                       int32_t n_features, const float *X, int64_t ld, int32_t n_rows,
                       const int32_t *prog_ptr, int32_t n_prog,
                       double *prog, double *stmt, double *scale, int n_threads) {
    if (n_prog < 0 || n_rows < 0 || ld < n_rows || n_trees < 0) return ORACLE_EINVAL;
    if (n_prog > 0 && (prog_ptr[0] != 0 || prog_ptr[n_prog] != n_rows)) return ORACLE_EINVAL;
    for (int32_t p = 0; p < n_prog; ++p)
        if (prog_ptr[p + 1] < prog_ptr[p]) return ORACLE_EINVAL;
    set_threads(n_threads);
    int bad = 0;
#pragma omp parallel for schedule(dynamic, 16) reduction(| : bad)
    for (int32_t p = 0; p < n_prog; ++p) {
        double acc = base_score, sc = fabs(base_score);
        for (int64_t r = prog_ptr[p]; r < prog_ptr[p + 1]; ++r) {
            double s = 0.0;
            for (int32_t t = 0; t < n_trees; ++t) {
                int64_t leaf = walk_tree(root[t], n_nodes, feature, threshold, left, right,
                                         default_left, X, ld, n_features, r);
                if (leaf < 0) { bad = 1; break; }
                s += (double)leaf_value[leaf];
                sc += fabs((double)leaf_value[leaf]);
            }
            if (stmt) stmt[r] = s;
            acc += s;
        }
        prog[p] = acc;
        if (scale) scale[p] = sc;
    }
    return bad ? ORACLE_EINVAL : ORACLE_OK;
}

/* ------------------------------------------------------------------------------------------- */
/* Actor / critic forward                                                                       */
/* ------------------------------------------------------------------------------------------- */

/* Value of element i of a weight/state array stored as fp32 (dtype 0) or bf16 bits (dtype 1). */
static double load_val(const void *base, int dtype, int64_t i) {
    if (dtype == 0) return (double)((const float *)base)[i];
    uint32_t bits = (uint32_t)((const uint16_t *)base)[i] << 16;
    float f;
    memcpy(&f, &bits, sizeof f);
    return (double)f;
}

/* Round an fp64 value to the nearest bf16 value (ties to even), returned as fp64.  Works on the
 * exact binary expansion: keep 8 significant bits (1 implicit + 7 stored) of the normalised
 * value; subnormal bf16 values keep fewer bits, with the same rule. */
static double round_to_bf16(double v) {
    if (v == 0.0 || isnan(v) || isinf(v)) return v;
    int e;
    double m = frexp(fabs(v), &e);           /* |v| = m * 2^e, m in [0.5, 1) */
    int keep = 8;                            /* significant bits of a normal bf16 */
    int emin = -125;                         /* smallest normal bf16 is 2^-126 = 0.5 * 2^-125 */
    if (e < emin) keep -= (emin - e);        /* subnormal range loses bits */
    if (keep < 0) return copysign(0.0, v);
    double scaled = ldexp(m, keep);          /* integer part holds the kept bits */
    double fl = floor(scaled);
    double frac = scaled - fl;
    if (frac > 0.5 || (frac == 0.5 && fmod(fl, 2.0) != 0.0)) fl += 1.0;
    double r = ldexp(fl, e - keep);
    if (r > 3.3895313892515355e38) r = INFINITY; /* beyond the largest finite bf16 */
    return copysign(r, v);
}

/* Exported for the tests of the rounding rule itself. */
double oracle_round_bf16(double v) { return round_to_bf16(v); }

/*
 * For each state b (row b of states[B][S]):
 *     h1 = max(0, W1 s + b1),  h2 = max(0, W2 h1 + b2)     (bf16 policies: h rounded to bf16)
 *     logits = Wa h2 + ba,     value = wv . h2 + bv
 *     action = lowest i with logits[i] == max logits;  probs = softmax(logits)
 * Weights are [out][in] row-major.  Scales (for tolerances) are sum_j |W_ij h_j| + |b_i|.
 * logits/probs/logit_scale are [B][A]; any output but action and value may be NULL.
 */
int oracle_policy_step(int dtype, int32_t S, int32_t H1, int32_t H2, int32_t A,
                       const void *w1, const float *b1, const void *w2, const float *b2,
                       const void *wa, const float *ba, const void *wv, const float *bv,
                       const void *states, int32_t B,
                       int32_t *action, double *value, double *logits, double *probs,
                       double *logit_scale, double *value_scale, int n_threads) {
    if ((dtype != 0 && dtype != 1) || S <= 0 || H1 <= 0 || H2 <= 0 || A <= 0 || B < 0)
        return ORACLE_EINVAL;
    set_threads(n_threads);
    int oom = 0;
#pragma omp parallel reduction(| : oom)
    {
        double *h1 = (double *)malloc(sizeof(double) * (size_t)H1);
        double *h2 = (double *)malloc(sizeof(double) * (size_t)H2);
        double *z = (double *)malloc(sizeof(double) * (size_t)A);
        if (!h1 || !h2 || !z) {
            oom = 1;
        } else {
#pragma omp for schedule(static)
            for (int32_t b = 0; b < B; ++b) {
                for (int32_t i = 0; i < H1; ++i) {
                    double acc = b1[i];
                    for (int32_t j = 0; j < S; ++j)
                        acc += load_val(w1, dtype, (int64_t)i * S + j) *
                               load_val(states, dtype, (int64_t)b * S + j);
                    acc = acc > 0.0 ? acc : 0.0;
                    h1[i] = dtype == 1 ? round_to_bf16(acc) : acc;
                }
                for (int32_t i = 0; i < H2; ++i) {
                    double acc = b2[i];
                    for (int32_t j = 0; j < H1; ++j) acc += load_val(w2, dtype, (int64_t)i * H1 + j) * h1[j];
                    acc = acc > 0.0 ? acc : 0.0;
                    h2[i] = dtype == 1 ? round_to_bf16(acc) : acc;
                }
                int32_t best = 0;
                for (int32_t i = 0; i < A; ++i) {
                    double acc = ba[i], sc = fabs((double)ba[i]);
                    for (int32_t j = 0; j < H2; ++j) {
                        double t = load_val(wa, dtype, (int64_t)i * H2 + j) * h2[j];
                        acc += t;
                        sc += fabs(t);
                    }
                    z[i] = acc;
                    if (logits) logits[(int64_t)b * A + i] = acc;
                    if (logit_scale) logit_scale[(int64_t)b * A + i] = sc;
                    if (acc > z[best]) best = i;      /* strict: the lowest index wins ties */
                }
                action[b] = best;
                double v = bv[0], vs = fabs((double)bv[0]);
                for (int32_t j = 0; j < H2; ++j) {
                    double t = load_val(wv, dtype, j) * h2[j];
                    v += t;
                    vs += fabs(t);
                }
                value[b] = v;
                if (value_scale) value_scale[b] = vs;
                if (probs) {
                    double m = z[best], sum = 0.0;
                    for (int32_t i = 0; i < A; ++i) sum += exp(z[i] - m);
                    for (int32_t i = 0; i < A; ++i) probs[(int64_t)b * A + i] = exp(z[i] - m) / sum;
                }
            }
        }
        free(h1);
        free(h2);
        free(z);
    }
    return oom ? ORACLE_ENOMEM : ORACLE_OK;
}

/* ------------------------------------------------------------------------------------------- */
/* Top-K and the running heap                                                                   */
/* ------------------------------------------------------------------------------------------- */

typedef struct {
    float score;
    int64_t index;
} cand_t;

/* Ranking order: higher score first; NaN after every number; -0 and +0 equal; then lower index. */
static int cand_cmp(const void *pa, const void *pb) {
    const cand_t *a = (const cand_t *)pa, *b = (const cand_t *)pb;
    int an = isnan(a->score), bn = isnan(b->score);
    if (an != bn) return an ? 1 : -1;
    if (!an) {
        if (a->score > b->score) return -1;
        if (a->score < b->score) return 1;
    }
    if (a->index < b->index) return -1;
    if (a->index > b->index) return 1;
    return 0;
}

/* The k best of n scores, ranked; candidate i carries index index_base + i.  Requires k <= n. */
int oracle_topk(const float *score, int64_t n, int32_t k, int64_t index_base,
                float *out_score, int64_t *out_index) {
    if (n < 0 || k < 0 || k > n) return ORACLE_EINVAL;
    cand_t *c = (cand_t *)malloc(sizeof(cand_t) * (size_t)(n > 0 ? n : 1));
    if (!c) return ORACLE_ENOMEM;
    for (int64_t i = 0; i < n; ++i) {
        c[i].score = score[i];
        c[i].index = index_base + i;
    }
    qsort(c, (size_t)n, sizeof(cand_t), cand_cmp);
    for (int32_t i = 0; i < k; ++i) {
        out_score[i] = c[i].score;
        out_index[i] = c[i].index;
    }
    free(c);
    return ORACLE_OK;
}

/* running <- the k best of (running's k entries) united with (n new scores, indices index_base+i). */
int oracle_merge(float *run_score, int64_t *run_index, int32_t k,
                 const float *score, int64_t n, int64_t index_base) {
    if (n < 0 || k < 0) return ORACLE_EINVAL;
    int64_t m = (int64_t)k + n;
    cand_t *c = (cand_t *)malloc(sizeof(cand_t) * (size_t)(m > 0 ? m : 1));
    if (!c) return ORACLE_ENOMEM;
    for (int32_t i = 0; i < k; ++i) {
        c[i].score = run_score[i];
        c[i].index = run_index[i];
    }
    for (int64_t i = 0; i < n; ++i) {
        c[k + i].score = score[i];
        c[k + i].index = index_base + i;
    }
    qsort(c, (size_t)m, sizeof(cand_t), cand_cmp);
    for (int32_t i = 0; i < k; ++i) {
        run_score[i] = c[i].score;
        run_index[i] = c[i].index;
    }
    free(c);
    return ORACLE_OK;
}

/* ------------------------------------------------------------------------------------------- */
/* Schedule tracks: reward, advantage and adaptive-stopping elimination                         */
/* ------------------------------------------------------------------------------------------- */

/* One modification step of n schedule tracks.  Track i moved from state s (predicted score
 * c_prev[i], critic value v_prev[i]) to s' (c_next[i], v_next[i]).  Algorithm 1 rewards the step
 * with the relative change of the cost model's score, r = (C(s') - C(s)) / C(s), here with the
 * denominator max(|C(s)|, eps); Eq. 6 gives the advantage A = r + gamma V(s') - V(s).
 * scale[i] = |r| + |gamma V(s')| + |V(s)| bounds the terms of A (scale-relative tolerance). */
int oracle_track_advantage(const float *c_prev, const float *c_next, const float *v_prev,
                           const float *v_next, int64_t n, double gamma, double eps,
                           double *reward, double *adv, double *scale) {
    if (n < 0 || !(eps > 0.0)) return ORACLE_EINVAL;
    for (int64_t i = 0; i < n; ++i) {
        const double c = c_prev[i], cn = c_next[i];
        const double denom = fabs(c) > eps ? fabs(c) : eps;
        const double r = (cn - c) / denom;
        const double g = gamma * (double)v_next[i];
        const double v = v_prev[i];
        reward[i] = r;
        adv[i] = r + g - v;
        scale[i] = fabs(r) + fabs(g) + fabs(v);
    }
    return ORACLE_OK;
}

/* Adaptive-stopping elimination (Section 5): after a window of steps the tracks are ordered by
 * advantage and the ones with the lowest advantages stop.  The n_keep tracks ranked first (the
 * top-K ranking above, on the advantage, track i carrying index i) survive; their indices are
 * written in ascending order, so the surviving tracks keep their relative order. */
int oracle_track_eliminate(const float *adv, int64_t n, int64_t n_keep, int32_t *keep_index) {
    if (n < 0 || n_keep < 0 || n_keep > n || n > INT32_MAX) return ORACLE_EINVAL;
    cand_t *c = (cand_t *)malloc(sizeof(cand_t) * (size_t)(n > 0 ? n : 1));
    unsigned char *keep = (unsigned char *)calloc((size_t)(n > 0 ? n : 1), 1);
    if (!c || !keep) {
        free(c);
        free(keep);
        return ORACLE_ENOMEM;
    }
    for (int64_t i = 0; i < n; ++i) {
        c[i].score = adv[i];
        c[i].index = i;
    }
    qsort(c, (size_t)n, sizeof(cand_t), cand_cmp);
    for (int64_t k = 0; k < n_keep; ++k) keep[c[k].index] = 1;
    int64_t m = 0;
    for (int64_t i = 0; i < n; ++i)
        if (keep[i]) keep_index[m++] = (int32_t)i;
    free(c);
    free(keep);
    return ORACLE_OK;
}

/* ------------------------------------------------------------------------------------------- */
/* Per-type action selection                                                                    */
/* ------------------------------------------------------------------------------------------- */

/* Philox4x32 with 10 rounds, from its published definition: each round multiplies counter words
 * 0 and 2 by two constants into 64-bit products, and the new counter is
 * (hi(M1 c2) ^ c1 ^ k0, lo(M1 c2), hi(M0 c0) ^ c3 ^ k1, lo(M0 c0)); the key is advanced by the
 * Weyl constants between rounds. */
void oracle_philox4x32(const uint32_t ctr_in[4], const uint32_t key_in[2], uint32_t out[4]) {
    const uint32_t M0 = 0xD2511F53u, M1 = 0xCD9E8D57u, W0 = 0x9E3779B9u, W1 = 0xBB67AE85u;
    uint32_t c[4] = {ctr_in[0], ctr_in[1], ctr_in[2], ctr_in[3]};
    uint32_t k[2] = {key_in[0], key_in[1]};
    for (int round = 0; round < 10; ++round) {
        if (round > 0) {
            k[0] += W0;
            k[1] += W1;
        }
        const uint64_t p0 = (uint64_t)M0 * c[0], p1 = (uint64_t)M1 * c[2];
        const uint32_t hi0 = (uint32_t)(p0 >> 32), lo0 = (uint32_t)p0;
        const uint32_t hi1 = (uint32_t)(p1 >> 32), lo1 = (uint32_t)p1;
        const uint32_t n0 = hi1 ^ c[1] ^ k[0], n2 = hi0 ^ c[3] ^ k[1];
        c[0] = n0;
        c[1] = lo1;
        c[2] = n2;
        c[3] = lo0;
    }
    memcpy(out, c, sizeof(c));
}

/* The Gumbel noise of logit i of state b (see the readings above). */
static double gumbel_noise(uint64_t seed, uint64_t counter, int64_t b, int32_t i) {
    const uint32_t ctr[4] = {(uint32_t)(i / 4), (uint32_t)b, (uint32_t)counter, (uint32_t)(counter >> 32)};
    const uint32_t key[2] = {(uint32_t)seed, (uint32_t)(seed >> 32)};
    uint32_t w[4];
    oracle_philox4x32(ctr, key, w);
    const double u = ((double)(w[i % 4] >> 8) + 0.5) * (1.0 / 16777216.0);
    return -log(-log(u));
}

/* For every state b and segment s = [off[s], off[s+1]) of its a logits: the chosen action (the
 * lowest index attaining the maximum of z_i, or of z_i + Gumbel noise when `sample`), its
 * log-probability under the segment's softmax, and the softmax itself (fp64). */
int oracle_policy_select(const float *logits, int64_t B, int32_t a, const int32_t *off, int32_t n_seg,
                         int sample, uint64_t seed, uint64_t counter, int32_t *action, double *logp,
                         double *probs) {
    if (B < 0 || a < 1 || n_seg < 1 || off[0] != 0 || off[n_seg] != a) return ORACLE_EINVAL;
    for (int32_t s = 0; s < n_seg; ++s)
        if (off[s + 1] <= off[s]) return ORACLE_EINVAL;
    for (int64_t b = 0; b < B; ++b) {
        const float *z = logits + b * a;
        for (int32_t s = 0; s < n_seg; ++s) {
            const int32_t lo = off[s], hi = off[s + 1];
            double m = -INFINITY, best = -INFINITY;
            int32_t pick = lo;
            for (int32_t i = lo; i < hi; ++i) {
                const double v = z[i];
                if (v > m) m = v;
                const double key = sample ? v + gumbel_noise(seed, counter, b, i) : v;
                if (key > best) {
                    best = key;
                    pick = i;
                }
            }
            double sum = 0.0;
            for (int32_t i = lo; i < hi; ++i) sum += exp((double)z[i] - m);
            for (int32_t i = lo; i < hi; ++i) probs[b * a + i] = exp((double)z[i] - m) / sum;
            action[b * n_seg + s] = pick;
            logp[b * n_seg + s] = (double)z[pick] - m - log(sum);
        }
    }
    return ORACLE_OK;
}

/* ------------------------------------------------------------------------------------------- */
/* Refit of the cost model on measured programs (Algorithm 1, its last steps: the top-K states
 * are measured and the cost model is trained on (S^, P); Section 6.1 and Appendix A.1: XGBoost
 * with Ansor's settings).  One boosting round of histogram-based gradient boosting (Chen and
 * Guestrin, KDD'16, Section 3: the second-order gain and the optimal leaf weight; Section 3.4:
 * the sparsity-aware default direction) under the pack-sum squared error: a program's prediction
 * is base_score plus the sum of its statements' margins, the objective is
 * 1/2 sum_p w_p (s_p - y_p)^2, so every statement row of program p carries the gradient
 * w_p (s_p - y_p) and the hessian w_p.
 *
 * Readings where the paper is silent:
 *   - features are binned per feature by caller-given increasing cut points: bin(x) = the number
 *     of cut points <= x (0 .. n_cuts), 255 for NaN (missing);
 *   - a candidate split (f, t, dir) sends bins < t left, t in 1 .. n_cuts[f], and the missing
 *     rows left (dir = 1) or right (dir = 0); its node test is x < cuts[f][t - 1];
 *   - gradients and hessians are summed exactly: each program's value is rounded once to a
 *     fixed-point grid 2^-e (e chosen from the largest magnitude and the row count so that no
 *     sum can exceed 2^62) and summed as 64-bit integers;
 *   - gain = GL^2 / (HL + lambda) + GR^2 / (HR + lambda) - G^2 / (H + lambda) in fp64, the node
 *     splits iff the best gain exceeds gamma (pre-pruning) and both children's hessians reach
 *     min_child_weight; the best is the largest gain, ties to the lowest feature, then the lowest
 *     t, then missing-left before missing-right;
 *   - the tree grows depth-wise to max_depth in heap numbering (children of node k are 2k + 1
 *     and 2k + 2); a leaf holds -(G / (H + lambda)) eta rounded to fp32;
 *   - the margins are updated in fp32: margin[r] += leaf value of the row's leaf. */

/* bins[r * ld + f] for statement row r and feature f < F (bytes F .. ld - 1 are zero) from the
 * feature-major values x[f * ldx + r] and the cut points cuts[f * cut_stride + i], i < n_cuts[f]. */
int oracle_gbdt_bin(const float *x, int64_t N, int32_t F, int64_t ldx, const float *cuts,
                    int32_t cut_stride, const int32_t *n_cuts, int64_t ld, uint8_t *bins) {
    if (N < 0 || F < 1 || ld < F || ldx < N || cut_stride < 1) return ORACLE_EINVAL;
    for (int32_t f = 0; f < F; ++f)
        if (n_cuts[f] < 0 || n_cuts[f] > 254 || n_cuts[f] > cut_stride) return ORACLE_EINVAL;
    for (int64_t r = 0; r < N; ++r) {
        for (int64_t f = 0; f < ld; ++f) {
            uint8_t b = 0;
            if (f < F) {
                const float v = x[f * ldx + r];
                int c = 0;
                for (int32_t i = 0; i < n_cuts[f]; ++i)
                    if (cuts[f * cut_stride + i] <= v) ++c;
                b = isnan(v) ? (uint8_t)255 : (uint8_t)c;
            }
            bins[r * ld + f] = b;
        }
    }
    return ORACLE_OK;
}

/* Smallest c with 2^c >= n (n >= 1). */
static int ceil_log2_i64(int64_t n) {
    int c = 0;
    while (((int64_t)1 << c) < n) ++c;
    return c;
}

/* The fixed-point exponent e for values of largest magnitude amax summed over n rows:
 * amax < 2^E (frexp), |v 2^e| <= 2^(62 - ceil_log2(n)). */
static int fixed_exponent(double amax, int64_t n) {
    if (!(amax > 0.0)) return 0;
    int E;
    frexp(amax, &E);
    return 62 - ceil_log2_i64(n > 0 ? n : 1) - E;
}

typedef struct {
    const uint8_t *bins;
    int32_t F;
    int64_t ld;
    const float *cuts;
    int32_t cut_stride;
    const int32_t *n_cuts;
    const int64_t *qg, *qh;  /* per row */
    int eg, eh;
    int32_t max_depth;
    double eta, lambda, gamma, mcw;
    float *margin;
    int32_t *feature;
    float *threshold;
    int32_t *left, *right;
    uint8_t *default_left;
    float *leaf_value;
} gbdt_ctx;

static double node_score(double G, double H, double lambda) { return (G * G) / (H + lambda); }

static int grow(const gbdt_ctx *c, int64_t k, int32_t depth, const int64_t *rows, int64_t n) {
    int64_t Gi = 0, Hi = 0;
    for (int64_t i = 0; i < n; ++i) {
        Gi += c->qg[rows[i]];
        Hi += c->qh[rows[i]];
    }
    const double G = ldexp((double)Gi, -c->eg), H = ldexp((double)Hi, -c->eh);
    int found = 0, bf = 0, bt = 0, bdir = 0;
    double best = 0.0;
    if (depth < c->max_depth) {
        const double parent = node_score(G, H, c->lambda);
        for (int32_t f = 0; f < c->F; ++f) {
            int64_t hg[256], hh[256];
            memset(hg, 0, sizeof hg);
            memset(hh, 0, sizeof hh);
            for (int64_t i = 0; i < n; ++i) {
                const uint8_t b = c->bins[rows[i] * c->ld + f];
                hg[b] += c->qg[rows[i]];
                hh[b] += c->qh[rows[i]];
            }
            int64_t GLi = 0, HLi = 0;
            for (int32_t t = 1; t <= c->n_cuts[f]; ++t) {
                GLi += hg[t - 1];
                HLi += hh[t - 1];
                for (int dir = 1; dir >= 0; --dir) { /* missing-left first */
                    const int64_t gl = GLi + (dir ? hg[255] : 0), hl = HLi + (dir ? hh[255] : 0);
                    const double GL = ldexp((double)gl, -c->eg), HL = ldexp((double)hl, -c->eh);
                    const double GR = ldexp((double)(Gi - gl), -c->eg), HR = ldexp((double)(Hi - hl), -c->eh);
                    if (!(HL >= c->mcw) || !(HR >= c->mcw)) continue;
                    const double gain = (node_score(GL, HL, c->lambda) + node_score(GR, HR, c->lambda)) - parent;
                    if (!found || gain > best) {
                        found = 1;
                        best = gain;
                        bf = f;
                        bt = t;
                        bdir = dir;
                    }
                }
            }
        }
    }
    if (found && best > c->gamma) {
        c->feature[k] = bf;
        c->threshold[k] = c->cuts[(int64_t)bf * c->cut_stride + bt - 1];
        c->left[k] = (int32_t)(2 * k + 1);
        c->right[k] = (int32_t)(2 * k + 2);
        c->default_left[k] = (uint8_t)bdir;
        c->leaf_value[k] = 0.0f;
        int64_t *lr = (int64_t *)malloc(sizeof(int64_t) * (size_t)(n > 0 ? n : 1));
        int64_t *rr = (int64_t *)malloc(sizeof(int64_t) * (size_t)(n > 0 ? n : 1));
        if (!lr || !rr) {
            free(lr);
            free(rr);
            return ORACLE_ENOMEM;
        }
        int64_t nl = 0, nr = 0;
        for (int64_t i = 0; i < n; ++i) {
            const uint8_t b = c->bins[rows[i] * c->ld + bf];
            const int go_left = b == 255 ? bdir : b < bt;
            if (go_left) lr[nl++] = rows[i];
            else rr[nr++] = rows[i];
        }
        int rc = grow(c, 2 * k + 1, depth + 1, lr, nl);
        if (rc == ORACLE_OK) rc = grow(c, 2 * k + 2, depth + 1, rr, nr);
        free(lr);
        free(rr);
        return rc;
    }
    const float w = (float)(-(G / (H + c->lambda)) * c->eta);
    c->feature[k] = -1;
    c->leaf_value[k] = w;
    for (int64_t i = 0; i < n; ++i) c->margin[rows[i]] = c->margin[rows[i]] + w;
    return ORACLE_OK;
}

/* One boosting round.  bins [N][ld] as oracle_gbdt_bin writes them; program p owns rows
 * [prog_ptr[p], prog_ptr[p + 1]); label, weight [P]; margin [N] in/out.  The tree is written to
 * node arrays of 2^(max_depth + 1) - 1 entries in heap numbering; nodes the tree does not reach
 * hold feature -1, leaf value 0.  exps (optional) receives the fixed-point exponents (e_g, e_h). */
int oracle_gbdt_round(const uint8_t *bins, int64_t N, int32_t F, int64_t ld, const float *cuts,
                      int32_t cut_stride, const int32_t *n_cuts, const int32_t *prog_ptr, int64_t P,
                      const float *label, const float *weight, double base_score, int32_t max_depth,
                      double eta, double lambda, double gamma, double min_child_weight, float *margin,
                      int32_t *feature, float *threshold, int32_t *left, int32_t *right,
                      uint8_t *default_left, float *leaf_value, int32_t *exps) {
    if (N < 0 || P < 0 || F < 1 || ld < F || max_depth < 1 || max_depth > 12 || !(lambda > 0.0) ||
        !(gamma >= 0.0) || !(min_child_weight >= 0.0) || cut_stride < 1)
        return ORACLE_EINVAL;
    if (prog_ptr[0] != 0 || prog_ptr[P] != N) return ORACLE_EINVAL;
    const int64_t n_nodes = ((int64_t)1 << (max_depth + 1)) - 1;
    for (int64_t k = 0; k < n_nodes; ++k) {
        feature[k] = -1;
        threshold[k] = 0.0f;
        left[k] = right[k] = 0;
        default_left[k] = 0;
        leaf_value[k] = 0.0f;
    }
    /* pack-sum gradient and hessian per program */
    double *g = (double *)malloc(sizeof(double) * (size_t)(P > 0 ? P : 1));
    double *h = (double *)malloc(sizeof(double) * (size_t)(P > 0 ? P : 1));
    int64_t *qg = (int64_t *)malloc(sizeof(int64_t) * (size_t)(N > 0 ? N : 1));
    int64_t *qh = (int64_t *)malloc(sizeof(int64_t) * (size_t)(N > 0 ? N : 1));
    int64_t *rows = (int64_t *)malloc(sizeof(int64_t) * (size_t)(N > 0 ? N : 1));
    if (!g || !h || !qg || !qh || !rows) {
        free(g); free(h); free(qg); free(qh); free(rows);
        return ORACLE_ENOMEM;
    }
    double gmax = 0.0, hmax = 0.0;
    for (int64_t p = 0; p < P; ++p) {
        double s = base_score;
        for (int32_t r = prog_ptr[p]; r < prog_ptr[p + 1]; ++r) s += (double)margin[r];
        g[p] = (double)weight[p] * (s - (double)label[p]);
        h[p] = (double)weight[p];
        if (prog_ptr[p + 1] > prog_ptr[p]) {
            if (fabs(g[p]) > gmax) gmax = fabs(g[p]);
            if (fabs(h[p]) > hmax) hmax = fabs(h[p]);
        }
    }
    const int eg = fixed_exponent(gmax, N), eh = fixed_exponent(hmax, N);
    for (int64_t p = 0; p < P; ++p)
        for (int32_t r = prog_ptr[p]; r < prog_ptr[p + 1]; ++r) {
            qg[r] = (int64_t)rint(ldexp(g[p], eg));
            qh[r] = (int64_t)rint(ldexp(h[p], eh));
        }
    if (exps) {
        exps[0] = eg;
        exps[1] = eh;
    }
    for (int64_t r = 0; r < N; ++r) rows[r] = r;
    const gbdt_ctx c = {bins, F, ld, cuts, cut_stride, n_cuts, qg, qh, eg, eh, max_depth, eta, lambda,
                        gamma, min_child_weight, margin, feature, threshold, left, right, default_left,
                        leaf_value};
    const int rc = grow(&c, 0, 0, rows, N);
    free(g); free(h); free(qg); free(qh); free(rows);
    return rc;
}
