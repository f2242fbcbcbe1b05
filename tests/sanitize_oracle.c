/* Exercises every entry point of the CPU oracle (oracle/harl_oracle.c) on small inputs and their
 * edge cases (empty programs, zero rows, k = 0 and k = n, NaN / +-inf / +-0 values, irregular trees,
 * every tree depth up to 12, degenerate refit sets) so that a build with -fsanitize=address,undefined
 * reports any out-of-bounds access, leak or undefined behaviour.  Test infrastructure: compiled and
 * run by tests/test_oracle_sanitized.py.  Exits 0 when every call returned as expected. */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

int oracle_score_round(int32_t, int32_t, const int32_t *, const int32_t *, const float *, const int32_t *,
                       const int32_t *, const uint8_t *, const float *, double, int32_t, const float *, int64_t,
                       int32_t, const int32_t *, int32_t, double *, double *, double *, int);
int oracle_policy_step(int, int32_t, int32_t, int32_t, int32_t, const void *, const float *, const void *,
                       const float *, const void *, const float *, const void *, const float *, const void *,
                       int32_t, int32_t *, double *, double *, double *, double *, double *, int);
int oracle_topk(const float *, int64_t, int32_t, int64_t, float *, int64_t *);
int oracle_merge(float *, int64_t *, int32_t, const float *, int64_t, int64_t);
int oracle_track_advantage(const float *, const float *, const float *, const float *, int64_t, double, double,
                           double *, double *, double *);
int oracle_track_eliminate(const float *, int64_t, int64_t, int32_t *);
void oracle_philox4x32(const uint32_t[4], const uint32_t[2], uint32_t[4]);
int oracle_policy_select(const float *, int64_t, int32_t, const int32_t *, int32_t, int, uint64_t, uint64_t,
                         int32_t *, double *, double *);
int oracle_gbdt_bin(const float *, int64_t, int32_t, int64_t, const float *, int32_t, const int32_t *, int64_t,
                    uint8_t *);
int oracle_gbdt_round(const uint8_t *, int64_t, int32_t, int64_t, const float *, int32_t, const int32_t *,
                      const int32_t *, int64_t, const float *, const float *, double, int32_t, double, double,
                      double, double, float *, int32_t *, float *, int32_t *, int32_t *, uint8_t *, float *,
                      int32_t *);
double oracle_round_bf16(double);

static uint64_t rs = 88172645463325252ull;
static uint32_t rnd(void) {
    rs ^= rs << 13;
    rs ^= rs >> 7;
    rs ^= rs << 17;
    return (uint32_t)(rs >> 11);
}
static float uf(void) { return (float)(rnd() % 1000000) / 1000000.0f; }
static float special(void) {
    static const float v[] = {0.0f, -0.0f, 1.5f, -2.25f, 1e-40f, 3e38f};
    const uint32_t r = rnd() % 10;
    if (r == 0) return NAN;
    if (r == 1) return INFINITY;
    if (r == 2) return -INFINITY;
    if (r < 6) return v[rnd() % 6];
    return uf() * 8.0f - 4.0f;
}
static int fails = 0;
static void expect(int cond, const char *what) {
    if (!cond) {
        fprintf(stderr, "unexpected result: %s\n", what);
        ++fails;
    }
}
static uint16_t bf16_bits(float x) {
    uint32_t b;
    memcpy(&b, &x, 4);
    return (uint16_t)(b >> 16);
}

/* a random tree of at most max_depth levels appended to the node arrays; returns its root */
static int32_t build(int32_t *n, int32_t cap, int depth, int max_depth, int F, int32_t *feat, float *thr, int32_t *l,
                     int32_t *r, uint8_t *dl, float *leaf) {
    const int32_t id = (*n)++;
    if (id >= cap) abort();
    feat[id] = -1;
    thr[id] = 0.f;
    l[id] = r[id] = -1;
    dl[id] = 0;
    leaf[id] = uf() - 0.5f;
    if (depth < max_depth && (depth == 0 || rnd() % 4 != 0)) {
        feat[id] = (int32_t)(rnd() % (uint32_t)F);
        thr[id] = special();
        dl[id] = (uint8_t)(rnd() & 1);
        l[id] = build(n, cap, depth + 1, max_depth, F, feat, thr, l, r, dl, leaf);
        r[id] = build(n, cap, depth + 1, max_depth, F, feat, thr, l, r, dl, leaf);
    }
    return id;
}

static void score_cases(void) {
    for (int depth = 1; depth <= 12; ++depth) {
        const int T = 3, F = 7, cap = T * ((1 << (depth + 1)) + 1);
        int32_t *feat = malloc(sizeof(int32_t) * cap), *l = malloc(sizeof(int32_t) * cap), *r = malloc(sizeof(int32_t) * cap);
        float *thr = malloc(sizeof(float) * cap), *leaf = malloc(sizeof(float) * cap);
        uint8_t *dl = malloc(cap);
        int32_t root[3], n = 0;
        for (int t = 0; t < T; ++t) root[t] = build(&n, cap, 0, depth, F, feat, thr, l, r, dl, leaf);
        const int P = 9;
        int32_t ptr[10] = {0, 0, 3, 3, 4, 9, 9, 12, 12, 15};   /* empty programs included */
        const int R = ptr[P], ld = R + 3;
        float *X = malloc(sizeof(float) * F * ld);
        for (int i = 0; i < F * ld; ++i) X[i] = special();
        double prog[9], stmt[15], scale[9];
        expect(oracle_score_round(T, n, root, feat, thr, l, r, dl, leaf, 0.25, F, X, ld, R, ptr, P, prog, stmt, scale, 1) == 0,
               "score_round");
        expect(oracle_score_round(T, n, root, feat, thr, l, r, dl, leaf, 0.0, F, X, ld, 0, ptr, 1, prog, stmt, scale, 2) == 0,
               "score_round with no rows");
        free(feat); free(l); free(r); free(thr); free(leaf); free(dl); free(X);
    }
}

static void policy_cases(void) {
    for (int dtype = 0; dtype <= 1; ++dtype)
        for (int B = 0; B <= 5; B += 5) {
            const int S = 5, H1 = 9, H2 = 6, A = 4;
            float w1f[9 * 5], w2f[6 * 9], waf[4 * 6], wvf[6], stf[5 * 5];
            uint16_t w1h[9 * 5], w2h[6 * 9], wah[4 * 6], wvh[6], sth[5 * 5];
            float b1[9], b2[6], ba[4], bv[1];
            for (int i = 0; i < 45; ++i) w1h[i] = bf16_bits(w1f[i] = uf() - 0.5f);
            for (int i = 0; i < 54; ++i) w2h[i] = bf16_bits(w2f[i] = uf() - 0.5f);
            for (int i = 0; i < 24; ++i) wah[i] = bf16_bits(waf[i] = uf() - 0.5f);
            for (int i = 0; i < 6; ++i) wvh[i] = bf16_bits(wvf[i] = uf() - 0.5f);
            for (int i = 0; i < 25; ++i) sth[i] = bf16_bits(stf[i] = uf() - 0.5f);
            for (int i = 0; i < 9; ++i) b1[i] = uf();
            for (int i = 0; i < 6; ++i) b2[i] = uf();
            for (int i = 0; i < 4; ++i) ba[i] = uf();
            bv[0] = uf();
            int32_t action[5];
            double value[5], logits[20], probs[20], ls[20], vs[5];
            const void *w1 = dtype ? (const void *)w1h : w1f, *w2 = dtype ? (const void *)w2h : w2f;
            const void *wa = dtype ? (const void *)wah : waf, *wv = dtype ? (const void *)wvh : wvf;
            const void *st = dtype ? (const void *)sth : stf;
            expect(oracle_policy_step(dtype, S, H1, H2, A, w1, b1, w2, b2, wa, ba, wv, bv, st, B, action, value, logits,
                                      probs, ls, vs, 1) == 0, "policy_step");
            expect(oracle_policy_step(dtype, S, H1, H2, A, w1, b1, w2, b2, wa, ba, wv, bv, st, B, action, value, logits,
                                      NULL, ls, vs, 2) == 0, "policy_step without probabilities");
        }
    expect(oracle_round_bf16(1.0 + 1.0 / 256) == 1.0, "bf16 rounding ties to even");
}

static void rank_cases(void) {
    for (int n = 0; n <= 40; n += 8) {
        float s[40];
        for (int i = 0; i < n; ++i) s[i] = rnd() % 3 ? special() : 1.0f;
        for (int k = 0; k <= n; k += (n > 0 ? n / 4 + 1 : 1)) {
            float os[41];
            int64_t oi[41];
            expect(oracle_topk(s, n, k, 7, os, oi) == 0, "topk");
            if (k > 0) {
                float rs_[41];
                int64_t ri[41];
                for (int i = 0; i < k; ++i) {
                    rs_[i] = -INFINITY;
                    ri[i] = INT64_MAX;
                }
                expect(oracle_merge(rs_, ri, k, s, n, 100) == 0, "merge");
                expect(oracle_merge(rs_, ri, k, s, n, 200) == 0, "merge again");
            }
        }
        expect(oracle_topk(s, n, n + 1, 0, NULL, NULL) != 0, "topk rejects k > n");
        float cp[40], cn[40], vp[40], vn[40];
        double rw[40], adv[40], sc[40];
        for (int i = 0; i < n; ++i) {
            cp[i] = special();
            cn[i] = special();
            vp[i] = uf();
            vn[i] = uf();
        }
        expect(oracle_track_advantage(cp, cn, vp, vn, n, 0.9, 1e-6, rw, adv, sc) == 0, "track_advantage");
        for (int64_t keep = 0; keep <= n; keep += (n > 0 ? n / 3 + 1 : 1)) {
            int32_t ki[40];
            expect(oracle_track_eliminate(s, n, keep, ki) == 0, "track_eliminate");
        }
        expect(oracle_track_eliminate(s, n, n + 1, NULL) != 0, "track_eliminate rejects n_keep > n");
    }
    uint32_t ctr[4] = {0, 1, 2, 3}, key[2] = {5, 6}, out[4];
    oracle_philox4x32(ctr, key, out);
    for (int B = 0; B <= 9; B += 9) {
        const int32_t off[4] = {0, 5, 8, 11};
        float z[9 * 11];
        for (int i = 0; i < 9 * 11; ++i) z[i] = rnd() % 7 ? uf() * 4 - 2 : special();
        int32_t act[9 * 3];
        double lp[9 * 3], pr[9 * 11];
        for (int sample = 0; sample <= 1; ++sample)
            expect(oracle_policy_select(z, B, 11, off, 3, sample, 42, 7, act, lp, pr) == 0, "policy_select");
    }
}

static void gbdt_cases(void) {
    const int F = 5, cs = 6;
    float cuts[5 * 6];
    int32_t nc[5] = {6, 3, 1, 0, 6};
    for (int f = 0; f < F; ++f)
        for (int j = 0; j < cs; ++j) cuts[f * cs + j] = (float)j - 2.5f + 0.1f * (float)f;
    for (int N = 0; N <= 60; N += 20) {
        const int ld = 8;
        float *x = malloc(sizeof(float) * F * (N + 1));
        for (int i = 0; i < F * (N + 1); ++i) x[i] = special();
        uint8_t *bins = malloc((size_t)(N + 1) * ld);
        expect(oracle_gbdt_bin(x, N, F, N + 1, cuts, cs, nc, ld, bins) == 0, "gbdt_bin");
        const int P = N / 4 + 1;
        int32_t *ptr = malloc(sizeof(int32_t) * (P + 1));
        for (int p = 0; p <= P; ++p) ptr[p] = p == P ? N : (p * N) / P;
        float *label = malloc(sizeof(float) * P), *weight = malloc(sizeof(float) * P), *margin = malloc(sizeof(float) * (N + 1));
        for (int p = 0; p < P; ++p) {
            label[p] = uf();
            weight[p] = uf();
        }
        for (int depth = 1; depth <= 4; ++depth) {
            const int nn = (1 << (depth + 1)) - 1;
            int32_t feat[31], l[31], r[31], exps[2];
            float thr[31], leaf[31];
            uint8_t dl[31];
            for (int i = 0; i < N; ++i) margin[i] = 0.f;
            expect(oracle_gbdt_round(bins, N, F, ld, cuts, cs, nc, ptr, P, label, weight, 0.5, depth, 0.2, 1.0, 0.0, 0.0,
                                     margin, feat, thr, l, r, dl, leaf, exps) == 0, "gbdt_round");
            (void)nn;
        }
        free(x); free(bins); free(ptr); free(label); free(weight); free(margin);
    }
}

int main(void) {
    score_cases();
    policy_cases();
    rank_cases();
    gbdt_cases();
    if (fails) return 1;
    printf("oracle sanitizer run: ok\n");
    return 0;
}
