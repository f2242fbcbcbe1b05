// One PPO update of the actor/critic (HARL paper, Algorithm 1: sample a mini-batch from the replay
// buffer, train the actor with the policy gradient of Eq. 5 and the critic with the MSE of the
// advantage Y of Eq. 6; Section 6.1: PPO; Table 5: value weight 0.5, entropy weight 0.01, learning
// rates 3e-4 / 1e-3).
//
// The network is the shared trunk of the policy kernels in fp32 (W1, W2 with ReLU) with the
// per-type actor head of harl_policy_select and a value head.  One update:
//   forward    h1 = relu(X W1^T + b1), h2 = relu(h1 W2^T + b2), logits = h2 Wa^T + ba
//                                                                      (k_gemm, fused epilogues)
//   objective  per row (k_ppo_heads): v = h2 wv^T + bv, per-type log-softmax and entropy, logp = sum over types of
//              the chosen actions' log-probabilities, ratio = exp(logp - logp_old), the clipped
//              surrogate -min(ratio A, clip(ratio, 1 - eps, 1 + eps) A), w_v (v - R)^2 and the
//              entropy bonus -w_e H, each averaged over the batch; their gradients with respect to
//              the logits and v (min passes the gradient to the unclipped term on equality, clip
//              inside its closed range)
//   backward   dWa = dlogits^T h2, dwv = dv^T h2, dz2 = (dlogits Wa + dv wv) * [h2 > 0],
//              dW2 = dz2^T h1, dz1 = (dz2 W2) * [h1 > 0], dW1 = dz1^T X; each bias gradient is
//              the last column of its weight gradient's GEMM against [B | 1] -- all reductions over
//              the batch in fixed-order split-K pieces summed in order
//   Adam       bias-corrected, the actor's rate for the trunk and actor head, the critic's for the
//              value head (k_adam)
// k_gemm: C[i][j] = sum_p A(i, p) B(p, j) with A(i, p) = A[i a_si + p a_sp], B(p, j) = B[p b_sp +
// j b_sj] (any transpose), fp32 on v_mfma_f32_16x16x4f32: a workgroup of 4 waves owns a 64 x 64
// tile of C (a wave 32 x 32, 2 x 2 MFMA tiles; 32 x 64 when the grid would be small), K is staged through LDS 32 at a time while the next
// 32 are loaded into registers.  No result depends on scheduling.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>

#include "internal.hpp"

namespace harl {
namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kGemmThreads = 256, kTile = 64, kTileK = 32;
constexpr int kMaxSplits = 128;
constexpr int kLossChunk = 4096;  // rows per loss partial (large batches)

enum Epilogue : int { kPlain = 0, kBias = 1, kBiasRelu = 2, kReluMask = 3 };

struct GemmArgs {
    const float *A;  // null: A(i, p) = 1 (column sums)
    int64_t a_si, a_sp;
    const float *B;
    int64_t b_sp, b_sj;
    float *C;  // C[i ldc + j], or partial sums [split][I][J] when split
    int64_t ldc;
    int I, J, P, p_per_split, split;
    int epi;
    const float *bias;            // bias[j]
    const float *mask;            // multiply by [mask[i ldm + j] > 0]
    int64_t ldm;
    int ones;                     // C's last column (j = J - 1) is A's row sums (B has J - 1 columns)
    float *bias_out;              // split only: column J - 1 of rows i < rows_w goes to bias_out[i]
    int rows_w;                   // split only: rows i < rows_w go to C / bias_out (0 = all rows);
    float *last_out;              //   row rows_w, if last_out, to last_out[j]; later rows nowhere
};

// Operand elements of the K step starting at p0 for this thread: A's TI x TK and B's TK x 64
// tiles, the tile index moving fastest along the operand's contiguous direction.  VEC: 16-byte
// loads of 4 elements consecutive along that direction (the host checks that every such group is
// wholly inside or wholly outside the operand and 16-byte aligned); otherwise one element per load.
template <int TI, int TK, bool VEC>
struct Frag {
    static constexpr int W = VEC ? 4 : 1;
    static constexpr int NA = TI * TK / (kGemmThreads * W), NB = kTile * TK / (kGemmThreads * W);
    float a[NA][W], b[NB][W];
};

template <int TI, int TK, bool VEC>
__device__ __forceinline__ void gemm_fetch(const GemmArgs &g, int i0, int j0, int p0, int p_end, Frag<TI, TK, VEC> &f) {
    using F = Frag<TI, TK, VEC>;
    constexpr int W = F::W;
    const int t = threadIdx.x;
    const bool a_i_fast = g.a_si == 1, b_p_fast = g.b_sp == 1;
#pragma unroll
    for (int q = 0; q < F::NA; ++q) {
        const int e = t + kGemmThreads * q;
        // element (ii, pp) is the first of the group
        const int ii = a_i_fast ? (e % (TI / W)) * W : e / (TK / W), pp = a_i_fast ? e / (TI / W) : (e % (TK / W)) * W;
        const int gi = i0 + ii, gp = p0 + pp;
        if constexpr (VEC) {
            float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
            if (gi < g.I && gp < p_end) v = *reinterpret_cast<const float4 *>(g.A + (int64_t)gi * g.a_si + (int64_t)gp * g.a_sp);
            f.a[q][0] = v.x;
            f.a[q][1] = v.y;
            f.a[q][2] = v.z;
            f.a[q][3] = v.w;
        } else {
            float v = 0.f;
            if (gi < g.I && gp < p_end) v = g.A ? g.A[(int64_t)gi * g.a_si + (int64_t)gp * g.a_sp] : 1.f;
            f.a[q][0] = v;
        }
    }
#pragma unroll
    for (int q = 0; q < F::NB; ++q) {
        const int e = t + kGemmThreads * q;
        const int pb = b_p_fast ? (e % (TK / W)) * W : e / (kTile / W), jb = b_p_fast ? e / (TK / W) : (e % (kTile / W)) * W;
        const int gpb = p0 + pb, gj = j0 + jb;
        const int J0 = g.J - g.ones;  // B's columns
        if constexpr (VEC) {
            float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
            if (gpb < p_end && gj < J0)
                v = *reinterpret_cast<const float4 *>(g.B + (int64_t)gpb * g.b_sp + (int64_t)gj * g.b_sj);
            f.b[q][0] = v.x;
            f.b[q][1] = v.y;
            f.b[q][2] = v.z;
            f.b[q][3] = v.w;
        } else {
            f.b[q][0] = (gpb < p_end && gj < J0) ? g.B[(int64_t)gpb * g.b_sp + (int64_t)gj * g.b_sj] : 0.f;
        }
    }
}

// TI rows (64 or 32) by 64 columns of C per workgroup; wave w owns rows (w / 2) TI / 2 .. and
// columns (w % 2) 32 ..
template <int TI, int TK, bool VEC>
__global__ __launch_bounds__(kGemmThreads) void k_gemm(GemmArgs g) {
    using F = Frag<TI, TK, VEC>;
    constexpr int XT = TI / 32, W = F::W;
    __shared__ float As[TI][TK + 1];
    __shared__ float Bs[TK][kTile + 1];
    const int t = threadIdx.x, wv = t / 64, l = t % 64;
    const int i0 = blockIdx.y * TI, j0 = blockIdx.x * kTile;
    const int p_begin = blockIdx.z * g.p_per_split;
    const int p_end = g.P - p_begin < g.p_per_split ? g.P : p_begin + g.p_per_split;
    const int wi = (wv / 2) * (16 * XT), wj = (wv % 2) * 32;
    const bool a_i_fast = g.a_si == 1, b_p_fast = g.b_sp == 1;
    f32x4 acc[XT][2];
#pragma unroll
    for (int x = 0; x < XT; ++x)
#pragma unroll
        for (int y = 0; y < 2; ++y) acc[x][y] = f32x4{0.f, 0.f, 0.f, 0.f};
    F fr;
    // the column-0 workgroups of a GEMM with g.ones also sum A's rows: thread t < TI, row t
    const bool rowsum = g.ones && blockIdx.x == 0 && t < TI;
    float rs = 0.f;
    if (p_begin < p_end) gemm_fetch<TI, TK, VEC>(g, i0, j0, p_begin, p_end, fr);
    for (int p0 = p_begin; p0 < p_end; p0 += TK) {
#pragma unroll
        for (int q = 0; q < F::NA; ++q) {
            const int e = t + kGemmThreads * q;
            const int ii = a_i_fast ? (e % (TI / W)) * W : e / (TK / W), pp = a_i_fast ? e / (TI / W) : (e % (TK / W)) * W;
#pragma unroll
            for (int u = 0; u < W; ++u) As[ii + (a_i_fast ? u : 0)][pp + (a_i_fast ? 0 : u)] = fr.a[q][u];
        }
#pragma unroll
        for (int q = 0; q < F::NB; ++q) {
            const int e = t + kGemmThreads * q;
            const int pb = b_p_fast ? (e % (TK / W)) * W : e / (kTile / W), jb = b_p_fast ? e / (TK / W) : (e % (kTile / W)) * W;
#pragma unroll
            for (int u = 0; u < W; ++u) Bs[pb + (b_p_fast ? u : 0)][jb + (b_p_fast ? 0 : u)] = fr.b[q][u];
        }
        __syncthreads();
        // the next K step's operands are loaded while this one runs on the matrix cores
        if (p0 + TK < p_end) gemm_fetch<TI, TK, VEC>(g, i0, j0, p0 + TK, p_end, fr);
        if (rowsum)
#pragma unroll 8
            for (int kk = 0; kk < TK; ++kk) rs += As[t][kk];  // in p order; staged zeros past p_end
#pragma unroll
        for (int kk = 0; kk < TK; kk += 4) {
            float a[XT], b[2];
#pragma unroll
            for (int x = 0; x < XT; ++x) a[x] = As[wi + 16 * x + l % 16][kk + l / 16];
#pragma unroll
            for (int y = 0; y < 2; ++y) b[y] = Bs[kk + l / 16][wj + 16 * y + l % 16];
#pragma unroll
            for (int x = 0; x < XT; ++x)
#pragma unroll
                for (int y = 0; y < 2; ++y) acc[x][y] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[x], b[y], acc[x][y], 0, 0, 0);
        }
        __syncthreads();
    }
    if (rowsum && i0 + t < g.I) {
        const int i = i0 + t;
        if (g.split) g.C[((int64_t)blockIdx.z * g.I + i) * g.J + g.J - 1] = rs;
        else g.C[(int64_t)i * g.ldc + g.J - 1] = rs;
    }
    // accumulator register r of tile (x, y) is C[wi + 16x + 4(l/16) + r][wj + 16y + l%16]
#pragma unroll
    for (int x = 0; x < XT; ++x)
#pragma unroll
        for (int y = 0; y < 2; ++y)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int i = i0 + wi + 16 * x + 4 * (l / 16) + r, j = j0 + wj + 16 * y + l % 16;
                if (i >= g.I || j >= g.J - g.ones) continue;
                float v = acc[x][y][r];
                if (g.split) {
                    g.C[((int64_t)blockIdx.z * g.I + i) * g.J + j] = v;
                    continue;
                }
                if (g.epi == kBias || g.epi == kBiasRelu) v += g.bias[j];
                if (g.epi == kBiasRelu) v = fmaxf(v, 0.f);
                if (g.epi == kReluMask) v = g.mask[(int64_t)i * g.ldm + j] > 0.f ? v : 0.f;
                g.C[(int64_t)i * g.ldc + j] = v;
            }
}

// The sum over splits (in order) of partial[s][e], e < n = I J, row r = e / J, column c = e % J:
// without bias_out to out[e]; with it, rows r < rows_w send column J - 1 to bias_out[r] and the
// others to out[r (J - 1) + c], row rows_w goes to last_out[c] when last_out is given, and later
// rows are dropped.
__global__ __launch_bounds__(256) void k_split_sum(const float *__restrict__ partial, int splits, int64_t n,
                                                   float *__restrict__ out, int J, float *__restrict__ bias_out,
                                                   int rows_w, float *__restrict__ last_out) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= n) return;
    float s = 0.f;
    int k = 0;
    for (; k + 8 <= splits; k += 8) {  // eight loads in flight, added in split order
        float v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) v[u] = partial[(int64_t)(k + u) * n + i];
#pragma unroll
        for (int u = 0; u < 8; ++u) s += v[u];
    }
    for (; k < splits; ++k) s += partial[(int64_t)k * n + i];
    if (!bias_out) {
        out[i] = s;
        return;
    }
    const int64_t r = i / J, c = i - r * J;
    if (r >= rows_w) {
        if (r == rows_w && last_out) last_out[c] = s;
    } else if (c == J - 1) {
        bias_out[r] = s;
    } else {
        out[r * (J - 1) + c] = s;
    }
}

// Column sums of Y [rows][J] (row stride ldy), each row weighted by w[row] when w is given:

struct HeadArgs {
    const float *logits, *logp_old, *adv, *ret;
    const float *h2, *wv, *bv;  // the value head v = h2 . wv + bv is evaluated here
    int h2n;
    const int32_t *actions;
    int M, a, n_seg;
    int32_t off[HARL_SELECT_MAX_SEGMENTS + 1];
    float clip_eps, w_v, w_e;
    float *dlogits, *rows;  // dlogits: [M][ldd], dv in column a, zeros after; rows: [M][3] (min(s1, s2), (v - R)^2, entropy)
    int ldd;
    const float *wa;        // [a][h2n]: with wv, copied (a row per workgroup) into
    float *wext;            // [ldd][h2n] = [Wa; wv; 0], the B operand of dz2 = [dlogits, dv, 0] wext
};

// Log-sum-exp and entropy of segment [lo, hi) of a logits row.
__device__ __forceinline__ void segment_stats(const float *z, int lo, int hi, float &lse, float &H) {
    float mx = -INFINITY;
    for (int i = lo; i < hi; ++i) mx = fmaxf(mx, z[i]);
    float sum = 0.f;
    for (int i = lo; i < hi; ++i) sum += expf(z[i] - mx);
    lse = mx + logf(sum);
    H = 0.f;
    for (int i = lo; i < hi; ++i) {
        const float ls = z[i] - lse;
        H -= expf(ls) * ls;
    }
}

// A workgroup owns R consecutive rows, staged in LDS with coalesced loads.  Thread (row, segment)
// takes the segment's log-sum-exp, entropy and chosen log-probability; thread (row) adds them over
// the segments in order and forms the clipped surrogate, value and entropy terms; thread (row,
// segment) then overwrites the segment's logits with their gradient, and the rows are stored
// coalesced.  An action outside its segment (a broken device precondition) is clamped into it.
constexpr int kHeadThreads = 256, kHeadLdsFloats = 4096;

__global__ __launch_bounds__(kHeadThreads) void k_ppo_heads(HeadArgs h, int R) {
    __shared__ float zs[kHeadLdsFloats];
    __shared__ float s_lse[kHeadThreads], s_H[kHeadThreads], s_lp[kHeadThreads], s_gl[kHeadThreads];
    __shared__ float s_v[kHeadThreads], s_dv[kHeadThreads];
    const int t = threadIdx.x, a = h.a, ns = h.n_seg;
    const int64_t m0 = (int64_t)blockIdx.x * R;
    const int rows = h.M - m0 < R ? (int)(h.M - m0) : R;
    const int n = rows * a;
    for (int e = t; e < n; e += kHeadThreads) zs[e] = h.logits[m0 * a + e];
    {  // value head: tpr threads per row (a power of two, within one wave), strided partial dot
       // products combined by a butterfly of shuffles (fixed order)
        int tpr = 64;
        while (tpr * R > kHeadThreads) tpr >>= 1;
        const int row = t / tpr, sub = t % tpr;
        float acc = 0.f;
        if (row < rows) {
            const float *x = h.h2 + (m0 + row) * h.h2n;
            for (int k = sub; k < h.h2n; k += tpr) acc += x[k] * h.wv[k];
        }
        for (int off = tpr / 2; off > 0; off >>= 1) acc += __shfl_xor(acc, off, tpr);
        if (sub == 0 && row < rows) s_v[row] = acc + h.bv[0];
    }
    __syncthreads();
    const int p = t, r = p / ns, sg = p - r * ns;
    const bool own = p < rows * ns;
    int lo = 0, hi = 0, act = 0;
    if (own) {
        lo = h.off[sg];
        hi = h.off[sg + 1];
        act = min(max(h.actions[(m0 + r) * ns + sg], lo), hi - 1);
        float lse, H;
        segment_stats(zs + r * a, lo, hi, lse, H);
        s_lse[p] = lse;
        s_H[p] = H;
        s_lp[p] = zs[r * a + act] - lse;
    }
    __syncthreads();
    if (t < rows) {
        const int64_t m = m0 + t;
        float logp = 0.f, ent = 0.f;
        for (int k = 0; k < ns; ++k) {
            ent += s_H[t * ns + k];
            logp += s_lp[t * ns + k];
        }
        const float ratio = expf(logp - h.logp_old[m]);
        const float adv = h.adv[m];
        const float s1 = ratio * adv;
        const float rc = fminf(fmaxf(ratio, 1.f - h.clip_eps), 1.f + h.clip_eps);
        const float s2 = rc * adv;
        const bool inside = ratio >= 1.f - h.clip_eps && ratio <= 1.f + h.clip_eps;
        const float active = s1 <= s2 ? 1.f : (inside ? 1.f : 0.f);
        const float inv_m = 1.f / (float)h.M;
        s_gl[t] = -(adv * ratio * active) * inv_m;
        const float dvv = s_v[t] - h.ret[m];
        s_dv[t] = h.w_v * 2.f * dvv * inv_m;
        float *rw = h.rows + m * 3;
        rw[0] = fminf(s1, s2);
        rw[1] = dvv * dvv;
        rw[2] = ent;
    }
    __syncthreads();
    if (own) {
        const float g_logp = s_gl[r], lse = s_lse[p], H = s_H[p];
        const float we = h.w_e * (1.f / (float)h.M);
        float *z = zs + r * a;
        for (int i = lo; i < hi; ++i) {
            const float ls = z[i] - lse;
            const float pr = expf(ls);
            // g_logp (onehot - p) - (w_e / M) dH/dz, with dH/dz = -p (log p + H)
            z[i] = g_logp * ((i == act ? 1.f : 0.f) - pr) + we * pr * (ls + H);
        }
    }
    __syncthreads();
    for (int e = t; e < rows * h.ldd; e += kHeadThreads) {
        const int r2 = e / h.ldd, c = e - r2 * h.ldd;
        h.dlogits[m0 * h.ldd + e] = c < a ? zs[r2 * a + c] : (c == a ? s_dv[r2] : 0.f);
    }
    for (int r2 = blockIdx.x; r2 < h.ldd; r2 += gridDim.x)  // row r2 of [Wa; wv; 0] by workgroup r2
        for (int c = t; c < h.h2n; c += kHeadThreads)
            h.wext[(int64_t)r2 * h.h2n + c] = r2 < a ? h.wa[(int64_t)r2 * h.h2n + c] : (r2 == a ? h.wv[c] : 0.f);
}

// Sums of the row terms over rows [r0, r1) by one workgroup: thread-strided in row order, then the
// 256 thread sums in order.  Result in out (thread 0).
__device__ void loss_rows(const float *__restrict__ rows, int r0, int r1, double (&out)[3]) {
    __shared__ double part[3][256];
    const int t = threadIdx.x;
    double s[3] = {0.0, 0.0, 0.0};
    int m = r0 + t;
    for (; m + 768 < r1; m += 1024) {  // four rows of this thread in flight, added in row order
        float v[4][3];
#pragma unroll
        for (int u = 0; u < 4; ++u)
#pragma unroll
            for (int c = 0; c < 3; ++c) v[u][c] = rows[(int64_t)(m + 256 * u) * 3 + c];
#pragma unroll
        for (int u = 0; u < 4; ++u)
#pragma unroll
            for (int c = 0; c < 3; ++c) s[c] += (double)v[u][c];
    }
    for (; m < r1; m += 256)
#pragma unroll
        for (int c = 0; c < 3; ++c) s[c] += (double)rows[(int64_t)m * 3 + c];
#pragma unroll
    for (int c = 0; c < 3; ++c) part[c][t] = s[c];
    __syncthreads();
    if (t == 0) {
        out[0] = out[1] = out[2] = 0.0;
        for (int k = 0; k < 256; ++k)
#pragma unroll
            for (int c = 0; c < 3; ++c) out[c] += part[c][k];
    }
}

// Large batches: workgroup b sums rows [b kLossChunk, (b + 1) kLossChunk).
__global__ __launch_bounds__(256) void k_ppo_loss_part(const float *__restrict__ rows, int M, double *__restrict__ lpart) {
    double tot[3];
    const int r0 = blockIdx.x * kLossChunk;
    loss_rows(rows, r0, std::min(M, r0 + kLossChunk), tot);
    if (threadIdx.x == 0)
        for (int c = 0; c < 3; ++c) lpart[blockIdx.x * 3 + c] = tot[c];
}

// loss[0..3] = (total, clip, value, entropy): the means of the row terms; with lpart, the sums of
// n_part chunk sums in chunk order, else the rows summed here.
__global__ __launch_bounds__(256) void k_ppo_loss(const float *__restrict__ rows, int M, const double *__restrict__ lpart,
                                                  int n_part, float w_v, float w_e, float *__restrict__ loss) {
    double tot[3] = {0.0, 0.0, 0.0};
    if (lpart) {
        if (threadIdx.x != 0) return;
        for (int b = 0; b < n_part; ++b)
            for (int c = 0; c < 3; ++c) tot[c] += lpart[b * 3 + c];
    } else {
        loss_rows(rows, 0, M, tot);
    }
    if (threadIdx.x == 0) {
        const double clip = -tot[0] / M, value = tot[1] / M, ent = tot[2] / M;
        loss[0] = (float)(clip + (double)w_v * value - (double)w_e * ent);
        loss[1] = (float)clip;
        loss[2] = (float)value;
        loss[3] = (float)ent;
    }
}

__global__ __launch_bounds__(256) void k_adam(float *__restrict__ p, float *__restrict__ m, float *__restrict__ v,
                                              const float *__restrict__ g, int64_t n, int64_t n_actor, float lr_a,
                                              float lr_c, float b1, float b2, float bc1, float bc2, float eps) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= n) return;
    const float gi = g[i];
    const float mi = b1 * m[i] + (1.f - b1) * gi;
    const float vi = b2 * v[i] + (1.f - b2) * gi * gi;
    m[i] = mi;
    v[i] = vi;
    const float lr = i < n_actor ? lr_a : lr_c;
    p[i] -= lr * (mi / bc1) / (sqrtf(vi / bc2) + eps);
}

struct Layout {
    int64_t w1, b1, w2, b2, wa, ba, wv, bv, n, n_actor;
};

Layout param_layout(const harl_ppo_config *c) {
    Layout L{};
    L.w1 = 0;
    L.b1 = L.w1 + (int64_t)c->h1 * c->s;
    L.w2 = L.b1 + c->h1;
    L.b2 = L.w2 + (int64_t)c->h2 * c->h1;
    L.wa = L.b2 + c->h2;
    L.ba = L.wa + (int64_t)c->a * c->h2;
    L.wv = L.ba + c->a;
    L.bv = L.wv + c->h2;
    L.n = L.bv + 1;
    L.n_actor = L.wv;
    return L;
}

// Split-K pieces of a weight-gradient GEMM: enough for about 1,024 workgroups of 64 x 64 tiles, at
// least 128 rows of the batch per piece, at most kMaxSplits.
int splits_for(int P, int I, int J) {
    const int64_t tiles = ceil_div(J, 64) * ceil_div(I, 64);
    int64_t s = ceil_div(1024, tiles);
    s = std::min<int64_t>(s, ceil_div(P, 128));
    return (int)std::max<int64_t>(1, std::min<int64_t>(s, kMaxSplits));
}


struct Ws {
    float *h1, *h2, *logits, *dlogits, *wext, *dz2, *dz1, *rows, *grad, *partial;
    double *lpart;  // loss partials of row chunks (large batches)
    size_t bytes;
};

Ws ws_layout(const harl_ppo_config *c, int32_t M, char *base) {
    const Layout L = param_layout(c);
    const int64_t Mp = M > 0 ? M : 1;
    int64_t off = 0;
    auto take = [&](int64_t floats) {
        float *p = base ? reinterpret_cast<float *>(base + off) : nullptr;
        off += round_up(floats * 4, 256);
        return p;
    };
    Ws w{};
    w.h1 = take(Mp * c->h1);
    w.h2 = take(Mp * c->h2);
    w.logits = take(Mp * c->a);
    w.dlogits = take(Mp * round_up(c->a + 1, 4));  // [M][a + 1 rounded to 4]: dlogits, dv, zeros
    w.wext = take(round_up(c->a + 1, 4) * c->h2);
    w.lpart = reinterpret_cast<double *>(take(2 * 3 * ceil_div(Mp, kLossChunk)));
    w.dz2 = take(Mp * c->h2);
    w.dz1 = take(Mp * c->h1);
    w.rows = take(Mp * 3);
    w.grad = take(L.n);
    // split-K partials of the weight-gradient GEMMs (each with its bias column), for the piece
    // counts those GEMMs use at this batch size
    const int ldd = (int)round_up(c->a + 1, 4);
    auto need = [&](int I, int J0) { return (int64_t)splits_for((int)Mp, I, J0) * I * (J0 + 1); };
    w.partial = take(std::max(std::max(need(ldd, c->h2), need(c->h2, c->h1)), need(c->h1, c->s)));
    w.bytes = (size_t)off;
    return w;
}

// 16-byte operand loads are safe when each operand's contiguous dimension and other stride are
// multiples of 4 and its base is 16-byte aligned (then a group of 4 is wholly in or out of range).
bool vec_ok(const GemmArgs &g) {
    if (!g.A || !aligned(g.A, 16) || !aligned(g.B, 16)) return false;
    const bool a_ok = g.a_si == 1 ? (g.I % 4 == 0 && g.a_sp % 4 == 0) : (g.a_sp == 1 && g.P % 4 == 0 && g.a_si % 4 == 0);
    const int J0 = g.J - g.ones;  // B's columns
    const bool b_ok = g.b_sp == 1 ? (g.P % 4 == 0 && g.b_sj % 4 == 0) : (g.b_sj == 1 && J0 % 4 == 0 && g.b_sp % 4 == 0);
    return a_ok && b_ok;
}

template <int TK, bool VEC>
void launch_gemm(const GemmArgs &g, unsigned gx, int used, hipStream_t stream) {
    // 32-row tiles when 64-row tiles would leave the machine short of workgroups
    const bool small = (int64_t)gx * ceil_div(g.I, 64) * used < 1024 && g.I > 32;
    if (small)
        hipLaunchKernelGGL((k_gemm<32, TK, VEC>), dim3(gx, (unsigned)ceil_div(g.I, 32), used), dim3(kGemmThreads), 0,
                           stream, g);
    else
        hipLaunchKernelGGL((k_gemm<64, TK, VEC>), dim3(gx, (unsigned)ceil_div(g.I, 64), used), dim3(kGemmThreads), 0,
                           stream, g);
}

int gemm(const GemmArgs &g0, float *partial, hipStream_t stream) {
    GemmArgs g = g0;
    const unsigned gx = (unsigned)ceil_div(g.J - g.ones, kTile);
    const bool vec = vec_ok(g);
    const int tk = vec ? 2 * kTileK : kTileK;  // 64-deep K stages with 16-byte loads, else 32
    int used = 1;
    if (g.split) {
        const int splits = splits_for(g.P, g.I, g.J - g.ones);
        g.p_per_split = (int)round_up(ceil_div(g.P, splits), tk);
        used = (int)ceil_div(g.P, g.p_per_split);
    } else {
        g.p_per_split = (int)round_up(g.P, tk);
    }
    float *out = g.C;
    if (g.split) g.C = partial;
    if (vec)
        launch_gemm<2 * kTileK, true>(g, gx, used, stream);
    else
        launch_gemm<kTileK, false>(g, gx, used, stream);
    HARL_HIP_CHECK(hipGetLastError());
    if (g.split) {
        const int64_t n = (int64_t)g.I * g.J;  // out is contiguous [I][J]
        hipLaunchKernelGGL(k_split_sum, dim3((unsigned)ceil_div(n, 256)), dim3(256), 0, stream, partial, used, n, out,
                           g.J, g.bias_out, g.rows_w ? g.rows_w : g.I, g.last_out);
    }
    HARL_HIP_CHECK(hipGetLastError());
    return HARL_OK;
}

GemmArgs ga(const float *A, int64_t a_si, int64_t a_sp, const float *B, int64_t b_sp, int64_t b_sj, float *C,
            int64_t ldc, int I, int J, int P) {
    GemmArgs g{};
    g.A = A;
    g.a_si = a_si;
    g.a_sp = a_sp;
    g.B = B;
    g.b_sp = b_sp;
    g.b_sj = b_sj;
    g.C = C;
    g.ldc = ldc;
    g.I = I;
    g.J = J;
    g.P = P;
    return g;
}

}  // namespace

size_t ppo_param_count(const harl_ppo_config *c) { return (size_t)param_layout(c).n; }

size_t ppo_ws_bytes(const harl_ppo_config *c, int32_t M) { return ws_layout(c, M, nullptr).bytes; }

int ppo_update_launch(const harl_ppo_config *c, float *params, float *adam_m, float *adam_v, int32_t step,
                      const float *X, const int32_t *actions, const float *logp_old, const float *adv, const float *ret,
                      int32_t M, float *grad_out, float *loss_out, void *ws, hipStream_t stream) {
    const Layout L = param_layout(c);
    const Ws w = ws_layout(c, M, static_cast<char *>(ws));
    float *grad = grad_out ? grad_out : w.grad;
    const int s = c->s, h1 = c->h1, h2 = c->h2, a = c->a;
    const float *W1 = params + L.w1, *W2 = params + L.w2, *Wa = params + L.wa, *wv = params + L.wv;
    int rc;
    // ---- forward ----
    GemmArgs g = ga(X, s, 1, W1, 1, s, w.h1, h1, M, h1, s);
    g.epi = kBiasRelu;
    g.bias = params + L.b1;
    if ((rc = gemm(g, w.partial, stream))) return rc;
    g = ga(w.h1, h1, 1, W2, 1, h1, w.h2, h2, M, h2, h1);
    g.epi = kBiasRelu;
    g.bias = params + L.b2;
    if ((rc = gemm(g, w.partial, stream))) return rc;
    g = ga(w.h2, h2, 1, Wa, 1, h2, w.logits, a, M, a, h2);
    g.epi = kBias;
    g.bias = params + L.ba;
    if ((rc = gemm(g, w.partial, stream))) return rc;
    // ---- objective and its gradient at the logits and the value ----
    HeadArgs h{};
    h.logits = w.logits;
    h.h2 = w.h2;
    h.wv = wv;
    h.bv = params + L.bv;
    h.h2n = h2;
    h.logp_old = logp_old;
    h.adv = adv;
    h.ret = ret;
    h.actions = actions;
    h.M = M;
    h.a = a;
    h.n_seg = c->n_seg;
    for (int k = 0; k <= c->n_seg; ++k) h.off[k] = c->seg_offsets[k];
    h.clip_eps = c->clip_eps;
    h.w_v = c->w_value;
    h.w_e = c->w_entropy;
    h.dlogits = w.dlogits;
    h.ldd = (int)round_up(a + 1, 4);
    h.wa = Wa;
    h.wext = w.wext;
    h.rows = w.rows;
    {
        // rows per workgroup: enough workgroups to cover the machine, at most kHeadLdsFloats logits
        // and kHeadThreads (row, segment) pairs
        int64_t R = ceil_div(M, 512);
        R = std::max<int64_t>(1, std::min<int64_t>({R, kHeadLdsFloats / a, kHeadThreads / c->n_seg}));
        hipLaunchKernelGGL(k_ppo_heads, dim3((unsigned)ceil_div(M, R)), dim3(kHeadThreads), 0, stream, h, (int)R);
    }
    HARL_HIP_CHECK(hipGetLastError());
    if (loss_out) {
        if (M > 4 * kLossChunk) {  // one workgroup per chunk of rows, then the chunk sums in order
            const int nb = (int)ceil_div(M, kLossChunk);
            hipLaunchKernelGGL(k_ppo_loss_part, dim3((unsigned)nb), dim3(256), 0, stream, w.rows, M, w.lpart);
            hipLaunchKernelGGL(k_ppo_loss, dim3(1), dim3(256), 0, stream, w.rows, M, w.lpart, nb, c->w_value,
                               c->w_entropy, loss_out);
        } else {
            hipLaunchKernelGGL(k_ppo_loss, dim3(1), dim3(256), 0, stream, w.rows, M, nullptr, 0, c->w_value,
                               c->w_entropy, loss_out);
        }
        HARL_HIP_CHECK(hipGetLastError());
    }
    // ---- backward: heads ----
    // Each weight gradient's GEMM also returns the row sums of A in a last column of C (the
    // bias gradient): the column-0 workgroups add up the A tiles they stage.
    // [dWa | dba; dwv | dbv] = [dlogits, dv, 0]^T [h2 | 1]: rows < a to Wa's and ba's gradients,
    // row a to wv's and bv's (adjacent in the parameter layout), the zero rows nowhere
    const int ldd = (int)round_up(a + 1, 4);
    g = ga(w.dlogits, 1, ldd, w.h2, h2, 1, grad + L.wa, h2, ldd, h2 + 1, M);
    g.split = 1;
    g.ones = 1;
    g.bias_out = grad + L.ba;
    g.rows_w = a;
    g.last_out = grad + L.wv;
    if ((rc = gemm(g, w.partial, stream))) return rc;
    // dz2 = (dlogits Wa + dv wv) * [h2 > 0], one contraction over the padded columns
    g = ga(w.dlogits, ldd, 1, w.wext, h2, 1, w.dz2, h2, M, h2, ldd);  // [dlogits, dv, 0] [Wa; wv; 0]
    g.epi = kReluMask;
    g.mask = w.h2;
    g.ldm = h2;
    if ((rc = gemm(g, w.partial, stream))) return rc;
    // ---- backward: layer 2 ----
    g = ga(w.dz2, 1, h2, w.h1, h1, 1, grad + L.w2, h1, h2, h1 + 1, M);  // [dW2 | db2] = dz2^T [h1 | 1]
    g.split = 1;
    g.ones = 1;
    g.bias_out = grad + L.b2;
    if ((rc = gemm(g, w.partial, stream))) return rc;
    // dz1 = (dz2 W2) * [h1 > 0]
    g = ga(w.dz2, h2, 1, W2, h1, 1, w.dz1, h1, M, h1, h2);
    g.epi = kReluMask;
    g.mask = w.h1;
    g.ldm = h1;
    if ((rc = gemm(g, w.partial, stream))) return rc;
    // ---- backward: layer 1 ----
    g = ga(w.dz1, 1, h1, X, s, 1, grad + L.w1, s, h1, s + 1, M);  // [dW1 | db1] = dz1^T [X | 1]
    g.split = 1;
    g.ones = 1;
    g.bias_out = grad + L.b1;
    if ((rc = gemm(g, w.partial, stream))) return rc;
    // ---- Adam ----
    const double bc1 = 1.0 - std::pow((double)c->beta1, step), bc2 = 1.0 - std::pow((double)c->beta2, step);
    hipLaunchKernelGGL(k_adam, dim3((unsigned)ceil_div(L.n, 256)), dim3(256), 0, stream, params, adam_m, adam_v, grad,
                       L.n, L.n_actor, c->lr_actor, c->lr_critic, c->beta1, c->beta2, (float)bc1, (float)bc2,
                       c->adam_eps);
    HARL_HIP_CHECK(hipGetLastError());
    return HARL_OK;
}

}  // namespace harl
