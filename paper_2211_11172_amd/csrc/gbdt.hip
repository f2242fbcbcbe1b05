// Refit of the cost model on measured programs (Algorithm 1: the top-K states are measured and
// the cost model is trained on (S^, P); Section 6.1 and Appendix A.2: XGBoost with Ansor's
// settings).  One boosting round of histogram-based gradient boosting under the pack-sum squared
// error 1/2 sum_p w_p (s_p - y_p)^2, s_p = base + the sum of program p's statement margins; the
// gain, leaf weight and learned missing direction follow Chen and Guestrin (KDD'16, Sections 3
// and 3.4).
//
//   k_gb_bin        bins[r][f] = number of cut points <= x (upper bound), 255 for NaN
//   k_gb_prog_grad  per program: s_p (fp64, statements in order), g_p = w_p (s_p - y_p), h_p = w_p,
//                   per-block maxima of |g|, |h|
//   k_gb_exps       the fixed-point exponents: |v 2^e| <= 2^(62 - ceil(log2 N)), so sums of N rows
//                   of 64-bit integers are exact, and no result depends on summation order
//   k_gb_row_q      each statement row's integer gradient and hessian; rows start in the root
//   per depth d < max_depth (rows kept grouped by node in `order`):
//     k_gb_level    one workgroup: node ranges from the parent's partition, the chunk list
//                   (kChunk rows per chunk) and the shared-histogram slots of multi-chunk nodes
//     k_gb_hist     workgroup = (chunk, 8 features): a [2][8][256] int64 histogram in LDS (ds_add
//                   of integers); a one-chunk node evaluates its splits at once, a larger one adds
//                   its histogram into the node's slot (integer atomics: the sum is exact)
//     k_gb_split    the slot nodes' split evaluation from the shared histograms
//     k_gb_decide   per node: best over feature groups, split or leaf, tree arrays, children sums
//     k_gb_flags / scan / k_gb_scatter   stable partition of each split node's rows
//   k_gb_leaves     the last level's leaves;  k_gb_margin  margin[r] += leaf of the row
//
// Split evaluation (thread = (feature, 8 consecutive bins)): an int64 prefix over bins gives GL,
// HL for every threshold index t; the gain GL^2/(HL+l) + GR^2/(HR+l) - G^2/(H+l) is fp64 with
// contraction off, missing rows tried left, then right; the best is the largest gain, ties to the
// lowest (feature, t, missing-left first).  Every decision is therefore bit-identical to a
// sequential evaluation of the same definitions.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>

#include "internal.hpp"

#pragma clang fp contract(off)

namespace harl {
namespace {

constexpr int kThreads = 256;
constexpr int kChunk = 2048;        // rows per histogram workgroup
constexpr int kGroup = 8;           // features per histogram workgroup (one 8-byte load per row)
constexpr int kBins = 256;          // bin 255 holds the missing values
constexpr int kScanBlock = 2048;    // flags per scan block

struct Params {
    double eta, lambda, gamma, mcw, base;
    int depth;
};

// One split candidate's record; key orders candidates: (feature, t, missing-left first).
struct Best {
    double gain;
    int32_t key, valid;
    int64_t GL, HL, G, H;
};

struct Ws {
    double *gp, *hp, *bmax;    // [P], [P], [2][nblk]
    int32_t *exps;             // [2]
    int64_t *qg, *qh;          // [N]
    int32_t *order, *order2, *nid, *flag, *spn, *X, *bsum;  // X: [N + 1]
    int32_t *start, *cnt, *alive, *sf, *st, *sd;             // per heap node
    int64_t *Gt, *Ht;                                        // per heap node
    int32_t *cp, *slot, *slot_node, *lvl;                    // level: [L+1], [L], [S], {chunks, slots}
    Best *best;                                              // [L][n_fg]
    int64_t *hist;                                           // [S][n_fg][2][8][256]
};

__device__ __forceinline__ int ceil_log2(int64_t n) {
    int c = 0;
    while (((int64_t)1 << c) < n) ++c;
    return c;
}

__device__ __forceinline__ double node_score(double G, double H, double lambda) { return (G * G) / (H + lambda); }

__device__ __forceinline__ int clamp_cuts(const int32_t *n_cuts, int f, int cut_stride) {
    int nc = n_cuts[f];
    nc = nc < 0 ? 0 : nc;
    nc = nc > 254 ? 254 : nc;
    return nc > cut_stride ? cut_stride : nc;
}

// a precedes b: larger gain, then the smaller key
__device__ __forceinline__ bool better(const Best &a, const Best &b) {
    if (!a.valid) return false;
    if (!b.valid) return true;
    if (a.gain > b.gain) return true;
    if (a.gain < b.gain) return false;
    return a.key < b.key;
}

// ------------------------------------------------------------------------------------------
// binning
// ------------------------------------------------------------------------------------------
__global__ __launch_bounds__(kThreads) void k_gb_bin(const float *__restrict__ x, int64_t ldx, int F, int N,
                                                     const float *__restrict__ cuts, int cut_stride,
                                                     const int32_t *__restrict__ n_cuts, uint8_t *__restrict__ bins,
                                                     int64_t ld) {
    const int r = blockIdx.x * kThreads + threadIdx.x;
    if (r >= N) return;
    const int g = blockIdx.y;
    uint64_t word = 0;
#pragma unroll
    for (int j = 0; j < kGroup; ++j) {
        const int f = g * kGroup + j;
        if (f >= F) break;
        const float v = x[(int64_t)f * ldx + r];
        const float *c = cuts + (int64_t)f * cut_stride;
        int lo = 0, hi = clamp_cuts(n_cuts, f, cut_stride);
        while (lo < hi) {  // number of cut points <= v
            const int mid = (lo + hi) >> 1;
            if (c[mid] <= v) lo = mid + 1;
            else hi = mid;
        }
        const uint64_t b = v != v ? 255u : (uint64_t)lo;
        word |= b << (8 * j);
    }
    *reinterpret_cast<uint64_t *>(bins + (int64_t)r * ld + (int64_t)g * kGroup) = word;
}

// ------------------------------------------------------------------------------------------
// gradients
// ------------------------------------------------------------------------------------------
__global__ __launch_bounds__(kThreads) void k_gb_prog_grad(const float *__restrict__ margin,
                                                           const int32_t *__restrict__ prog_ptr, int P,
                                                           const float *__restrict__ label,
                                                           const float *__restrict__ weight, double base, Ws w) {
    __shared__ double sg[kThreads], sh[kThreads];
    const int p = blockIdx.x * kThreads + threadIdx.x;
    double ag = 0.0, ah = 0.0;
    if (p < P) {
        const int r0 = prog_ptr[p], r1 = prog_ptr[p + 1];
        double s = base;
        for (int r = r0; r < r1; ++r) s += (double)margin[r];
        const double g = (double)weight[p] * (s - (double)label[p]);
        const double h = (double)weight[p];
        w.gp[p] = g;
        w.hp[p] = h;
        if (r1 > r0) {
            ag = fabs(g);
            ah = fabs(h);
        }
    }
    sg[threadIdx.x] = ag;
    sh[threadIdx.x] = ah;
    __syncthreads();
    for (int s = kThreads / 2; s > 0; s >>= 1) {
        if (threadIdx.x < s) {
            sg[threadIdx.x] = fmax(sg[threadIdx.x], sg[threadIdx.x + s]);
            sh[threadIdx.x] = fmax(sh[threadIdx.x], sh[threadIdx.x + s]);
        }
        __syncthreads();
    }
    if (threadIdx.x == 0) {
        w.bmax[2 * blockIdx.x] = sg[0];
        w.bmax[2 * blockIdx.x + 1] = sh[0];
    }
}

__global__ __launch_bounds__(kThreads) void k_gb_exps(Ws w, int nblk, int64_t N) {
    __shared__ double sg[kThreads], sh[kThreads];
    double ag = 0.0, ah = 0.0;
    for (int b = threadIdx.x; b < nblk; b += kThreads) {
        ag = fmax(ag, w.bmax[2 * b]);
        ah = fmax(ah, w.bmax[2 * b + 1]);
    }
    sg[threadIdx.x] = ag;
    sh[threadIdx.x] = ah;
    __syncthreads();
    for (int s = kThreads / 2; s > 0; s >>= 1) {
        if (threadIdx.x < s) {
            sg[threadIdx.x] = fmax(sg[threadIdx.x], sg[threadIdx.x + s]);
            sh[threadIdx.x] = fmax(sh[threadIdx.x], sh[threadIdx.x + s]);
        }
        __syncthreads();
    }
    if (threadIdx.x < 2) {
        const double a = threadIdx.x == 0 ? sg[0] : sh[0];
        int e = 0;
        if (a > 0.0) {
            int E;
            frexp(a, &E);
            e = 62 - ceil_log2(N > 0 ? N : 1) - E;
        }
        w.exps[threadIdx.x] = e;
    }
}

__global__ __launch_bounds__(kThreads) void k_gb_row_q(const int32_t *__restrict__ prog_ptr, int P, Ws w) {
    const int p = blockIdx.x * kThreads + threadIdx.x;
    if (p >= P) return;
    const int eg = w.exps[0], eh = w.exps[1];
    const int64_t qg = (int64_t)rint(ldexp(w.gp[p], eg)), qh = (int64_t)rint(ldexp(w.hp[p], eh));
    for (int r = prog_ptr[p]; r < prog_ptr[p + 1]; ++r) {
        w.qg[r] = qg;
        w.qh[r] = qh;
    }
}

// tree arrays to unreached-node defaults, node state cleared, rows in the root
__global__ __launch_bounds__(kThreads) void k_gb_init(Ws w, int n_nodes, int N, int32_t *feature, float *threshold,
                                                      int32_t *left, int32_t *right, uint8_t *default_left,
                                                      float *leaf_value) {
    const int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    if (i < n_nodes) {
        feature[i] = -1;
        threshold[i] = 0.f;
        left[i] = 0;
        right[i] = 0;
        default_left[i] = 0;
        leaf_value[i] = 0.f;
        w.alive[i] = i == 0;
        w.sf[i] = -1;
        w.start[i] = 0;
        w.cnt[i] = i == 0 ? N : 0;
        w.Gt[i] = 0;
        w.Ht[i] = 0;
    }
    if (i < N) {
        w.order[i] = (int32_t)i;
        w.nid[i] = 0;
    }
}

// ------------------------------------------------------------------------------------------
// one depth level
// ------------------------------------------------------------------------------------------

// Node ranges of level d from the parents' partition (X is the previous level's scan), the chunk
// list and the slots of nodes that span several chunks.  One workgroup.
__global__ __launch_bounds__(1024) void k_gb_level(Ws w, int d, int max_slots) {
    __shared__ int32_t sc[1024], ss[1024];
    const int L = 1 << d, base = L - 1;
    const int per = (L + 1023) / 1024;  // consecutive nodes per thread
    const int t = threadIdx.x;
    int chunks = 0, slots = 0;
    for (int q = 0; q < per; ++q) {
        const int j = t * per + q;
        if (j >= L) break;
        const int k = base + j;
        if (d > 0 && w.alive[k]) {
            const int p = (k - 1) / 2;
            const int s = w.start[p], n = w.cnt[p];
            const int nl = w.X[s + n] - w.X[s];
            if (k == 2 * p + 1) {
                w.start[k] = s;
                w.cnt[k] = nl;
            } else {
                w.start[k] = s + nl;
                w.cnt[k] = n - nl;
            }
        }
        const int c = w.alive[k] ? max(1, (w.cnt[k] + kChunk - 1) / kChunk) : 0;
        chunks += c;
        slots += c > 1;
    }
    sc[t] = chunks;
    ss[t] = slots;
    __syncthreads();
    for (int off = 1; off < 1024; off <<= 1) {  // inclusive scans
        const int a = t >= off ? sc[t - off] : 0, b = t >= off ? ss[t - off] : 0;
        __syncthreads();
        sc[t] += a;
        ss[t] += b;
        __syncthreads();
    }
    int c0 = sc[t] - chunks, s0 = ss[t] - slots;
    for (int q = 0; q < per; ++q) {
        const int j = t * per + q;
        if (j >= L) break;
        const int k = base + j;
        const int c = w.alive[k] ? max(1, (w.cnt[k] + kChunk - 1) / kChunk) : 0;
        w.cp[j] = c0;
        w.slot[j] = -1;
        if (c > 1 && s0 < max_slots) {
            w.slot[j] = s0;
            w.slot_node[s0] = j;
        }
        c0 += c;
        s0 += c > 1;
    }
    if (t == 1023) {
        w.cp[L] = sc[1023];
        w.lvl[0] = sc[1023];
        w.lvl[1] = ss[1023];
    }
}

__global__ __launch_bounds__(kThreads) void k_gb_zero_slots(Ws w, int n_fg) {
    const int64_t per_slot = (int64_t)n_fg * 2 * kGroup * kBins;
    const int64_t n = (int64_t)w.lvl[1] * per_slot;
    for (int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x; i < n; i += (int64_t)gridDim.x * kThreads)
        w.hist[i] = 0;
}

// Evaluate the splits of features f0 .. f0 + 7 of one node from its histogram h[2][8][256] (LDS
// or global memory); thread = (feature j = t / 32, bins 8 (t % 32) ..).  Result in *out.
__device__ void evaluate(const int64_t *h, int f0, int F, const float *cuts, int cut_stride,
                         const int32_t *n_cuts, const Params &prm, int eg, int eh, Best *out, Best *red) {
    const int t = threadIdx.x, j = t / 32, q = t % 32, f = f0 + j;
    int64_t pg[8], ph[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        pg[e] = h[(0 * kGroup + j) * kBins + 8 * q + e];
        ph[e] = h[(1 * kGroup + j) * kBins + 8 * q + e];
    }
    const int64_t mg = pg[7], mh = ph[7];  // bin 8q + 7 (bin 255 on lane 31)
#pragma unroll
    for (int e = 1; e < 8; ++e) {
        pg[e] += pg[e - 1];
        ph[e] += ph[e - 1];
    }
    int64_t ig = pg[7], ih = ph[7];  // inclusive scan over the 32 lanes of this feature
#pragma unroll
    for (int off = 1; off < 32; off <<= 1) {
        const int64_t ag = __shfl_up(ig, off, 32), ah = __shfl_up(ih, off, 32);
        if (q >= off) {
            ig += ag;
            ih += ah;
        }
    }
    const int64_t xg = ig - pg[7], xh = ih - ph[7];
    const int64_t Gi = __shfl(ig, 31, 32), Hi = __shfl(ih, 31, 32);
    const int64_t Gm = __shfl(mg, 31, 32), Hm = __shfl(mh, 31, 32);
    Best b;
    b.valid = 0;
    b.gain = 0.0;
    b.key = 0;
    b.GL = b.HL = 0;
    b.G = Gi;
    b.H = Hi;
    if (f < F) {
        const int nc = clamp_cuts(n_cuts, f, cut_stride);
        const double G = ldexp((double)Gi, -eg), H = ldexp((double)Hi, -eh);
        const double parent = node_score(G, H, prm.lambda);
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const int tt = 8 * q + e + 1;
            if (tt > nc) break;
            for (int dir = 1; dir >= 0; --dir) {
                const int64_t gl = xg + pg[e] + (dir ? Gm : 0), hl = xh + ph[e] + (dir ? Hm : 0);
                const double GL = ldexp((double)gl, -eg), HL = ldexp((double)hl, -eh);
                const double GR = ldexp((double)(Gi - gl), -eg), HR = ldexp((double)(Hi - hl), -eh);
                if (!(HL >= prm.mcw) || !(HR >= prm.mcw)) continue;
                const double gain = (node_score(GL, HL, prm.lambda) + node_score(GR, HR, prm.lambda)) - parent;
                if (!b.valid || gain > b.gain) {
                    b.valid = 1;
                    b.gain = gain;
                    b.key = (f * 256 + tt) * 2 + (1 - dir);
                    b.GL = gl;
                    b.HL = hl;
                }
            }
        }
    }
    // best over the 32 lanes of the feature
#pragma unroll
    for (int off = 16; off > 0; off >>= 1) {
        Best o;
        o.gain = __shfl_xor(b.gain, off, 32);
        o.key = __shfl_xor(b.key, off, 32);
        o.valid = __shfl_xor(b.valid, off, 32);
        o.GL = __shfl_xor(b.GL, off, 32);
        o.HL = __shfl_xor(b.HL, off, 32);
        o.G = b.G;
        o.H = b.H;
        if (better(o, b)) b = o;
    }
    if (q == 0) red[j] = b;
    __syncthreads();
    if (t == 0) {
        Best r = red[0];
        for (int i = 1; i < kGroup; ++i)
            if (better(red[i], r)) r = red[i];
        r.G = red[0].G;
        r.H = red[0].H;
        *out = r;
    }
}

struct HistArgs {
    const uint8_t *bins;
    int64_t ld;
    int F, n_fg, d;
    const float *cuts;
    int cut_stride;
    const int32_t *n_cuts;
    Params prm;
};

__global__ __launch_bounds__(kThreads) void k_gb_hist(HistArgs a, Ws w) {
    __shared__ int64_t h[2 * kGroup * kBins];  // 32 KB
    __shared__ Best red[kGroup];
    const int c = blockIdx.x, fg = blockIdx.y, t = threadIdx.x;
    if (c >= w.lvl[0]) return;
    const int L = 1 << a.d, base = L - 1;
    int lo = 0, hi = L - 1;  // the node j with cp[j] <= c < cp[j + 1]
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (w.cp[mid] <= c) lo = mid;
        else hi = mid - 1;
    }
    const int j = lo, k = base + j;
    const int nch = w.cp[j + 1] - w.cp[j];
    const int s = w.start[k], n = w.cnt[k];
    const int i0 = s + (c - w.cp[j]) * kChunk, i1 = std::min(s + n, i0 + kChunk);
    for (int e = t; e < 2 * kGroup * kBins; e += kThreads) h[e] = 0;
    __syncthreads();
    const int f0 = fg * kGroup;
    const int nf = std::min(kGroup, a.F - f0);
    for (int i = i0 + t; i < i1; i += kThreads) {
        const int r = w.order[i];
        const uint64_t word = *reinterpret_cast<const uint64_t *>(a.bins + (int64_t)r * a.ld + f0);
        const unsigned long long qg = (unsigned long long)w.qg[r], qh = (unsigned long long)w.qh[r];
        for (int jj = 0; jj < nf; ++jj) {
            const int b = (int)((word >> (8 * jj)) & 255u);
            atomicAdd(reinterpret_cast<unsigned long long *>(&h[(0 * kGroup + jj) * kBins + b]), qg);
            atomicAdd(reinterpret_cast<unsigned long long *>(&h[(1 * kGroup + jj) * kBins + b]), qh);
        }
    }
    __syncthreads();
    if (nch == 1) {
        evaluate(h, f0, a.F, a.cuts, a.cut_stride, a.n_cuts, a.prm, w.exps[0], w.exps[1],
                 &w.best[(int64_t)j * a.n_fg + fg], red);
        return;
    }
    if (w.slot[j] < 0) return;  // cannot happen: every multi-chunk node has a slot
    int64_t *g = w.hist + ((int64_t)w.slot[j] * a.n_fg + fg) * (2 * kGroup * kBins);
    for (int e = t; e < 2 * kGroup * kBins; e += kThreads) {
        const int64_t v = h[e];
        if (v != 0) atomicAdd(reinterpret_cast<unsigned long long *>(&g[e]), (unsigned long long)v);
    }
}

__global__ __launch_bounds__(kThreads) void k_gb_split(HistArgs a, Ws w) {
    __shared__ Best red[kGroup];
    const int sidx = blockIdx.x, fg = blockIdx.y;
    if (sidx >= w.lvl[1]) return;
    const int j = w.slot_node[sidx];
    const int64_t *g = w.hist + ((int64_t)sidx * a.n_fg + fg) * (2 * kGroup * kBins);
    evaluate(g, fg * kGroup, a.F, a.cuts, a.cut_stride, a.n_cuts, a.prm, w.exps[0], w.exps[1],
             &w.best[(int64_t)j * a.n_fg + fg], red);
}

__device__ __forceinline__ float leaf_weight(int64_t Gi, int64_t Hi, int eg, int eh, const Params &prm) {
    const double G = ldexp((double)Gi, -eg), H = ldexp((double)Hi, -eh);
    return (float)(-(G / (H + prm.lambda)) * prm.eta);
}

struct TreeOut {
    int32_t *feature;
    float *threshold;
    int32_t *left, *right;
    uint8_t *default_left;
    float *leaf_value;
};

__global__ __launch_bounds__(kThreads) void k_gb_decide(Ws w, int d, int n_fg, const float *__restrict__ cuts,
                                                        int cut_stride, Params prm, TreeOut tr) {
    const int j = blockIdx.x * kThreads + threadIdx.x, L = 1 << d;
    if (j >= L) return;
    const int k = L - 1 + j;
    if (!w.alive[k]) return;
    const Best *bs = w.best + (int64_t)j * n_fg;
    Best b = bs[0];
    for (int i = 1; i < n_fg; ++i)
        if (better(bs[i], b)) b = bs[i];
    const int64_t G = bs[0].G, H = bs[0].H;
    w.Gt[k] = G;
    w.Ht[k] = H;
    if (b.valid && b.gain > prm.gamma) {
        const int f = b.key / 512, tt = (b.key / 2) % 256, dir = 1 - (b.key & 1);
        tr.feature[k] = f;
        tr.threshold[k] = cuts[(int64_t)f * cut_stride + tt - 1];
        tr.left[k] = 2 * k + 1;
        tr.right[k] = 2 * k + 2;
        tr.default_left[k] = (uint8_t)dir;
        w.sf[k] = f;
        w.st[k] = tt;
        w.sd[k] = dir;
        w.alive[2 * k + 1] = 1;
        w.alive[2 * k + 2] = 1;
        w.Gt[2 * k + 1] = b.GL;
        w.Ht[2 * k + 1] = b.HL;
        w.Gt[2 * k + 2] = G - b.GL;
        w.Ht[2 * k + 2] = H - b.HL;
    } else {
        tr.leaf_value[k] = leaf_weight(G, H, w.exps[0], w.exps[1], prm);
    }
}

__global__ __launch_bounds__(kThreads) void k_gb_flags(Ws w, int N, const uint8_t *__restrict__ bins, int64_t ld) {
    const int i = blockIdx.x * kThreads + threadIdx.x;
    if (i >= N) return;
    const int r = w.order[i], k = w.nid[r];
    const int f = w.sf[k];
    if (f < 0) {
        w.flag[i] = 1;
        w.spn[i] = -1;
        return;
    }
    const int b = bins[(int64_t)r * ld + f];
    const int go_left = b == 255 ? w.sd[k] : b < w.st[k];
    w.nid[r] = go_left ? 2 * k + 1 : 2 * k + 2;
    w.flag[i] = go_left;
    w.spn[i] = k;
}

// exclusive scan of flag[0..N) into X[0..N]: block sums, a one-workgroup scan of them, the final pass
__global__ __launch_bounds__(kThreads) void k_gb_scan_sum(Ws w, int N) {
    __shared__ int32_t s[kThreads];
    const int b0 = blockIdx.x * kScanBlock;
    int acc = 0;
    for (int i = b0 + threadIdx.x; i < std::min(N, b0 + kScanBlock); i += kThreads) acc += w.flag[i];
    s[threadIdx.x] = acc;
    __syncthreads();
    for (int off = kThreads / 2; off > 0; off >>= 1) {
        if (threadIdx.x < off) s[threadIdx.x] += s[threadIdx.x + off];
        __syncthreads();
    }
    if (threadIdx.x == 0) w.bsum[blockIdx.x] = s[0];
}

__global__ __launch_bounds__(1024) void k_gb_scan_top(Ws w, int nb) {
    __shared__ int32_t s[1024];
    __shared__ int32_t carry;
    if (threadIdx.x == 0) carry = 0;
    __syncthreads();
    for (int b0 = 0; b0 < nb; b0 += 1024) {
        const int i = b0 + threadIdx.x;
        const int v = i < nb ? w.bsum[i] : 0;
        s[threadIdx.x] = v;
        __syncthreads();
        for (int off = 1; off < 1024; off <<= 1) {
            const int a = threadIdx.x >= off ? s[threadIdx.x - off] : 0;
            __syncthreads();
            s[threadIdx.x] += a;
            __syncthreads();
        }
        if (i < nb) w.bsum[i] = carry + s[threadIdx.x] - v;
        __syncthreads();
        if (threadIdx.x == 1023) carry += s[1023];
        __syncthreads();
    }
    if (threadIdx.x == 0) w.bsum[nb] = carry;
}

__global__ __launch_bounds__(kThreads) void k_gb_scan_final(Ws w, int N, int nb) {
    __shared__ int32_t s[kThreads];
    const int b0 = blockIdx.x * kScanBlock;
    constexpr int per = kScanBlock / kThreads;  // 8 consecutive flags per thread
    const int i0 = b0 + threadIdx.x * per;
    int v[per], acc = 0;
#pragma unroll
    for (int e = 0; e < per; ++e) {
        v[e] = i0 + e < N ? w.flag[i0 + e] : 0;
        acc += v[e];
    }
    s[threadIdx.x] = acc;
    __syncthreads();
    for (int off = 1; off < kThreads; off <<= 1) {
        const int a = threadIdx.x >= off ? s[threadIdx.x - off] : 0;
        __syncthreads();
        s[threadIdx.x] += a;
        __syncthreads();
    }
    int run = w.bsum[blockIdx.x] + s[threadIdx.x] - acc;
#pragma unroll
    for (int e = 0; e < per; ++e) {
        if (i0 + e < N) w.X[i0 + e] = run;
        run += v[e];
    }
    if (blockIdx.x == nb - 1 && threadIdx.x == 0) w.X[N] = w.bsum[nb];
}

__global__ __launch_bounds__(kThreads) void k_gb_scatter(Ws w, int N) {
    const int i = blockIdx.x * kThreads + threadIdx.x;
    if (i >= N) return;
    const int k = w.spn[i];
    if (k < 0) {
        w.order2[i] = w.order[i];
        return;
    }
    const int s = w.start[k], n = w.cnt[k];
    const int xs = w.X[s], xi = w.X[i], nl = w.X[s + n] - xs;
    const int pos = w.flag[i] ? s + (xi - xs) : s + nl + (i - s) - (xi - xs);
    w.order2[pos] = w.order[i];
}

__global__ __launch_bounds__(kThreads) void k_gb_leaves(Ws w, int d, Params prm, float *leaf_value) {
    const int j = blockIdx.x * kThreads + threadIdx.x, L = 1 << d;
    if (j >= L) return;
    const int k = L - 1 + j;
    if (!w.alive[k]) return;
    leaf_value[k] = leaf_weight(w.Gt[k], w.Ht[k], w.exps[0], w.exps[1], prm);
}

__global__ __launch_bounds__(kThreads) void k_gb_margin(Ws w, int N, const float *__restrict__ leaf_value,
                                                        float *__restrict__ margin) {
    const int r = blockIdx.x * kThreads + threadIdx.x;
    if (r >= N) return;
    margin[r] = margin[r] + leaf_value[w.nid[r]];
}

// ------------------------------------------------------------------------------------------
// workspace
// ------------------------------------------------------------------------------------------
struct Layout {
    size_t off[32];
    size_t total;
};

int max_slots_for(int N, int depth) {
    const int64_t by_rows = (int64_t)N / (kChunk + 1);
    const int64_t by_nodes = (int64_t)1 << (depth - 1);
    return (int)std::min(by_rows, by_nodes);
}

Ws carve(void *base, int F, int N, int P, int depth, size_t *total) {
    const int n_fg = (F + kGroup - 1) / kGroup;
    const int64_t n_nodes = ((int64_t)1 << (depth + 1)) - 1;
    const int64_t Lmax = (int64_t)1 << (depth - 1);  // widest level that builds histograms
    const int64_t nblk = ceil_div(std::max(P, 1), kThreads);
    const int64_t nb = ceil_div(std::max(N, 1), kScanBlock);
    const int S = max_slots_for(N, depth);
    char *p = static_cast<char *>(base);
    size_t o = 0;
    auto take = [&](size_t bytes) {
        char *r = p ? p + o : nullptr;
        o += (bytes + 255) / 256 * 256;
        return r;
    };
    Ws w;
    w.gp = reinterpret_cast<double *>(take(sizeof(double) * std::max(P, 1)));
    w.hp = reinterpret_cast<double *>(take(sizeof(double) * std::max(P, 1)));
    w.bmax = reinterpret_cast<double *>(take(sizeof(double) * 2 * nblk));
    w.exps = reinterpret_cast<int32_t *>(take(sizeof(int32_t) * 2));
    w.qg = reinterpret_cast<int64_t *>(take(sizeof(int64_t) * std::max(N, 1)));
    w.qh = reinterpret_cast<int64_t *>(take(sizeof(int64_t) * std::max(N, 1)));
    w.order = reinterpret_cast<int32_t *>(take(sizeof(int32_t) * std::max(N, 1)));
    w.order2 = reinterpret_cast<int32_t *>(take(sizeof(int32_t) * std::max(N, 1)));
    w.nid = reinterpret_cast<int32_t *>(take(sizeof(int32_t) * std::max(N, 1)));
    w.flag = reinterpret_cast<int32_t *>(take(sizeof(int32_t) * std::max(N, 1)));
    w.spn = reinterpret_cast<int32_t *>(take(sizeof(int32_t) * std::max(N, 1)));
    w.X = reinterpret_cast<int32_t *>(take(sizeof(int32_t) * (N + 1)));
    w.bsum = reinterpret_cast<int32_t *>(take(sizeof(int32_t) * (nb + 1)));
    w.start = reinterpret_cast<int32_t *>(take(sizeof(int32_t) * n_nodes));
    w.cnt = reinterpret_cast<int32_t *>(take(sizeof(int32_t) * n_nodes));
    w.alive = reinterpret_cast<int32_t *>(take(sizeof(int32_t) * n_nodes));
    w.sf = reinterpret_cast<int32_t *>(take(sizeof(int32_t) * n_nodes));
    w.st = reinterpret_cast<int32_t *>(take(sizeof(int32_t) * n_nodes));
    w.sd = reinterpret_cast<int32_t *>(take(sizeof(int32_t) * n_nodes));
    w.Gt = reinterpret_cast<int64_t *>(take(sizeof(int64_t) * n_nodes));
    w.Ht = reinterpret_cast<int64_t *>(take(sizeof(int64_t) * n_nodes));
    w.cp = reinterpret_cast<int32_t *>(take(sizeof(int32_t) * (Lmax + 1)));
    w.slot = reinterpret_cast<int32_t *>(take(sizeof(int32_t) * Lmax));
    w.slot_node = reinterpret_cast<int32_t *>(take(sizeof(int32_t) * std::max(S, 1)));
    w.lvl = reinterpret_cast<int32_t *>(take(sizeof(int32_t) * 2));
    w.best = reinterpret_cast<Best *>(take(sizeof(Best) * Lmax * n_fg));
    w.hist = reinterpret_cast<int64_t *>(take(sizeof(int64_t) * (size_t)std::max(S, 1) * n_fg * 2 * kGroup * kBins));
    *total = o;
    return w;
}

}  // namespace

size_t gbdt_ws_bytes(int32_t F, int32_t N, int32_t P, int32_t depth) {
    size_t total = 0;
    carve(nullptr, F, N, P, depth, &total);
    return total;
}

int gbdt_bin_launch(const float *x, int64_t ldx, int32_t F, int32_t N, const float *cuts, int32_t cut_stride,
                    const int32_t *n_cuts, uint8_t *bins, int64_t ld, hipStream_t stream) {
    if (N == 0) return HARL_OK;
    // padding bytes of the row: groups past F write zeros (every lane of a group past F skips)
    const dim3 grid((unsigned)ceil_div(N, kThreads), (unsigned)(ld / kGroup));
    hipLaunchKernelGGL(k_gb_bin, grid, dim3(kThreads), 0, stream, x, ldx, F, N, cuts, cut_stride, n_cuts, bins, ld);
    HARL_HIP_CHECK(hipGetLastError());
    return HARL_OK;
}

int gbdt_round_launch(const harl_gbdt_params *prm_in, const uint8_t *bins, int64_t ld, int32_t F, int32_t N,
                      const float *cuts, int32_t cut_stride, const int32_t *n_cuts, const int32_t *prog_ptr,
                      int32_t P, const float *label, const float *weight, float *margin, int32_t *feature,
                      float *threshold, int32_t *left, int32_t *right, uint8_t *default_left, float *leaf_value,
                      void *ws, hipStream_t stream) {
    Params prm{prm_in->eta, prm_in->reg_lambda, prm_in->gamma, prm_in->min_child_weight, prm_in->base_score,
               prm_in->max_depth};
    const int D = prm.depth;
    const int n_fg = (F + kGroup - 1) / kGroup;
    const int n_nodes = (1 << (D + 1)) - 1;
    size_t total = 0;
    Ws w = carve(ws, F, N, P, D, &total);
    const int S = max_slots_for(N, D);
    TreeOut tr{feature, threshold, left, right, default_left, leaf_value};
    const int init_n = std::max(n_nodes, N);
    hipLaunchKernelGGL(k_gb_init, dim3((unsigned)ceil_div(init_n, kThreads)), dim3(kThreads), 0, stream, w, n_nodes, N,
                       feature, threshold, left, right, default_left, leaf_value);
    const int nblk = (int)ceil_div(std::max(P, 1), kThreads);
    hipLaunchKernelGGL(k_gb_prog_grad, dim3(nblk), dim3(kThreads), 0, stream, margin, prog_ptr, P, label, weight,
                       prm.base, w);
    hipLaunchKernelGGL(k_gb_exps, dim3(1), dim3(kThreads), 0, stream, w, nblk, (int64_t)N);
    hipLaunchKernelGGL(k_gb_row_q, dim3(nblk), dim3(kThreads), 0, stream, prog_ptr, P, w);
    HARL_HIP_CHECK(hipGetLastError());
    HistArgs ha{bins, ld, F, n_fg, 0, cuts, cut_stride, n_cuts, prm};
    const unsigned rows_grid = (unsigned)ceil_div(std::max(N, 1), kThreads);
    const int nb = (int)ceil_div(std::max(N, 1), kScanBlock);
    for (int d = 0; d < D; ++d) {
        const int L = 1 << d;
        hipLaunchKernelGGL(k_gb_level, dim3(1), dim3(1024), 0, stream, w, d, S);
        const int slots = std::min(S, L);
        if (slots > 0) {
            const int64_t words = (int64_t)slots * n_fg * 2 * kGroup * kBins;
            const unsigned zg = (unsigned)std::min<int64_t>(ceil_div(words, kThreads), 4096);
            hipLaunchKernelGGL(k_gb_zero_slots, dim3(zg), dim3(kThreads), 0, stream, w, n_fg);
        }
        ha.d = d;
        const unsigned chunk_bound = (unsigned)(ceil_div(N, kChunk) + L);
        hipLaunchKernelGGL(k_gb_hist, dim3(chunk_bound, (unsigned)n_fg), dim3(kThreads), 0, stream, ha, w);
        if (slots > 0)
            hipLaunchKernelGGL(k_gb_split, dim3((unsigned)slots, (unsigned)n_fg), dim3(kThreads), 0, stream, ha, w);
        hipLaunchKernelGGL(k_gb_decide, dim3((unsigned)ceil_div(L, kThreads)), dim3(kThreads), 0, stream, w, d, n_fg,
                           cuts, cut_stride, prm, tr);
        if (N > 0) {
            hipLaunchKernelGGL(k_gb_flags, dim3(rows_grid), dim3(kThreads), 0, stream, w, N, bins, ld);
            hipLaunchKernelGGL(k_gb_scan_sum, dim3((unsigned)nb), dim3(kThreads), 0, stream, w, N);
            hipLaunchKernelGGL(k_gb_scan_top, dim3(1), dim3(1024), 0, stream, w, nb);
            hipLaunchKernelGGL(k_gb_scan_final, dim3((unsigned)nb), dim3(kThreads), 0, stream, w, N, nb);
            hipLaunchKernelGGL(k_gb_scatter, dim3(rows_grid), dim3(kThreads), 0, stream, w, N);
            std::swap(w.order, w.order2);
        }
        HARL_HIP_CHECK(hipGetLastError());
    }
    hipLaunchKernelGGL(k_gb_leaves, dim3((unsigned)ceil_div(1 << D, kThreads)), dim3(kThreads), 0, stream, w, D, prm,
                       leaf_value);
    if (N > 0)
        hipLaunchKernelGGL(k_gb_margin, dim3(rows_grid), dim3(kThreads), 0, stream, w, N, leaf_value, margin);
    HARL_HIP_CHECK(hipGetLastError());
    return HARL_OK;
}

}  // namespace harl
