// Refit of the cost model on measured programs (Algorithm 1: the top-K states are measured and
// the cost model is trained on (S^, P); Section 6.1 and Appendix A.1: XGBoost with Ansor's
// settings).  One boosting round of histogram-based gradient boosting under the pack-sum squared
// error 1/2 sum_p w_p (s_p - y_p)^2, s_p = base + the sum of program p's statement margins; the
// gain, leaf weight and learned missing direction follow Chen and Guestrin (KDD'16, Sections 3
// and 3.4).
//
//   k_gb_bin        bin of feature f of row r = number of cut points <= x (upper bound), 255 for NaN,
//                   stored in 8-feature groups: byte ((f / 8) ld + r) 8 + f % 8, so that a
//                   workgroup of one group reads its rows' 8 bytes from one contiguous plane
//   k_gb_prog_grad  per program: s_p (fp64, statements in order), g_p = w_p (s_p - y_p), h_p = w_p,
//                   per-block maxima of |g|, |h|
//   k_gb_exps       the fixed-point exponents: |v 2^e| <= 2^(62 - ceil(log2 N)), so sums of N rows
//                   of 64-bit integers are exact, and no result depends on summation order
//   k_gb_row_q      each statement row's integer gradient and hessian; rows start in the root
//   per depth d < max_depth (rows kept grouped by node in `order`):
//     k_gb_level    one workgroup: node ranges from the parent's partition, the chunk list
//                   (4096 rows per chunk, more for large sets) and the shared-histogram slots
//                   of multi-chunk nodes
//     k_gb_hist     workgroup = (chunk, 8 features): a [2][8][256] int64 histogram in LDS (ds_add
//                   of integers; the lanes of one add instruction are spread over the 8 features,
//                   so at most 8 meet on one bin; the bin of 0.0 is the total minus the others); a
//                   one-chunk node evaluates its splits at once, a larger one stores its partial
//     k_gb_reduce   a multi-chunk node's histogram: its partials summed in chunk order
//     k_gb_split    the multi-chunk nodes' split evaluation
//     k_gb_decide   per node: best over feature groups, split or leaf, tree arrays, children sums
//     k_gb_flags / scan / k_gb_scatter   stable partition of each split node's rows
//   k_gb_finish     the last level's leaves and margin[r] += the weight of the row's leaf
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
constexpr int kChunk = 2048;        // rows a histogram workgroup loads in one batch
constexpr int kGroup = 8;           // features per histogram workgroup (one 8-byte load per row)
constexpr int kBins = 256;          // bin 255 holds the missing values
constexpr int kBinStride = 257;     // int64 words per (feature, G|H) histogram row: odd, so that
                                    // the 8 features' rows fall on different LDS banks
constexpr int kHistWords = 2 * kGroup * kBinStride;
constexpr int kScanBlock = kThreads; // flags per scan block (one per thread)
constexpr int kBinRowBlocks = 8;     // at most this many 256-row blocks per binning workgroup

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
    int32_t *zb;                                             // [F] the bin of 0.0 per feature
    int32_t *pbase;                                          // [L] first partial of a multi-chunk node
    int64_t *part;                                           // [Pmax][n_fg][2][8][kBinStride]
    int pmax;
    Best *best;                                              // [L][n_fg]
    int64_t *hist;                                           // [S][n_fg][2][8][kBinStride]
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
// Thread = (row, 8-feature group); the group's cut points are staged in LDS first, so the binary
// searches run on LDS, and each workgroup then bins rb_per blocks of 256 rows with them.
__global__ __launch_bounds__(kThreads) void k_gb_bin(const float *__restrict__ x, int64_t ldx, int F, int N,
                                                     const float *__restrict__ cuts, int cut_stride,
                                                     const int32_t *__restrict__ n_cuts, uint8_t *__restrict__ bins,
                                                     int64_t ld, int rb_per) {
    __shared__ float sc[kGroup][256];
    __shared__ int snc[kGroup];
    const int g = blockIdx.y, t = threadIdx.x;
    if (t < kGroup) snc[t] = g * kGroup + t < F ? clamp_cuts(n_cuts, g * kGroup + t, cut_stride) : 0;
    __syncthreads();
    for (int e = t; e < kGroup * 256; e += kThreads) {
        const int j = e / 256, i = e % 256;
        if (i < snc[j]) sc[j][i] = cuts[(int64_t)(g * kGroup + j) * cut_stride + i];
    }
    __syncthreads();
    for (int rb = 0; rb < rb_per; ++rb) {
        const int r = (blockIdx.x * rb_per + rb) * kThreads + t;
        if (r >= N) return;
        uint64_t word = 0;
#pragma unroll
        for (int j = 0; j < kGroup; ++j) {
            const int f = g * kGroup + j;
            if (f >= F) break;
            const float v = x[(int64_t)f * ldx + r];
            int lo = 0, hi = snc[j];
            while (lo < hi) {  // number of cut points <= v
                const int mid = (lo + hi) >> 1;
                if (sc[j][mid] <= v) lo = mid + 1;
                else hi = mid;
            }
            const uint64_t b = v != v ? 255u : (uint64_t)lo;
            word |= b << (8 * j);
        }
        *reinterpret_cast<uint64_t *>(bins + ((int64_t)g * ld + r) * kGroup) = word;
    }
}

// ------------------------------------------------------------------------------------------
// gradients
// ------------------------------------------------------------------------------------------
__global__ __launch_bounds__(kThreads) void k_gb_prog_grad(const float *__restrict__ margin,
                                                           const int32_t *__restrict__ prog_ptr, int P,
                                                           const float *__restrict__ label,
                                                           const float *__restrict__ weight, double base, int N,
                                                           Ws w) {
    __shared__ double sg[kThreads], sh[kThreads];
    const int p = blockIdx.x * kThreads + threadIdx.x;
    double ag = 0.0, ah = 0.0;
    if (p < P) {
        const int r0 = min(max(prog_ptr[p], 0), N), r1 = min(max(prog_ptr[p + 1], r0), N);
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

__global__ __launch_bounds__(kThreads) void k_gb_row_q(const int32_t *__restrict__ prog_ptr, int P, int N, Ws w) {
    const int p = blockIdx.x * kThreads + threadIdx.x;
    if (p >= P) return;
    const int eg = w.exps[0], eh = w.exps[1];
    const int64_t qg = (int64_t)rint(ldexp(w.gp[p], eg)), qh = (int64_t)rint(ldexp(w.hp[p], eh));
    const int r0 = min(max(prog_ptr[p], 0), N), r1 = min(max(prog_ptr[p + 1], r0), N);  // clamped
    for (int r = r0; r < r1; ++r) {
        w.qg[r] = qg;
        w.qh[r] = qh;
    }
}

// tree arrays to unreached-node defaults, node state cleared, rows in the root
__global__ __launch_bounds__(kThreads) void k_gb_init(Ws w, int n_nodes, int N, int F, const float *__restrict__ cuts,
                                                      int cut_stride, const int32_t *__restrict__ n_cuts,
                                                      int32_t *feature, float *threshold, int32_t *left,
                                                      int32_t *right, uint8_t *default_left, float *leaf_value) {
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
    if (i < F) {  // the bin of 0.0: the number of cut points <= 0
        const float *cf = cuts + i * cut_stride;
        int lo = 0, hi = clamp_cuts(n_cuts, (int)i, cut_stride);
        while (lo < hi) {
            const int mid = (lo + hi) >> 1;
            if (cf[mid] <= 0.f) lo = mid + 1;
            else hi = mid;
        }
        w.zb[i] = lo;
    }
}

// ------------------------------------------------------------------------------------------
// one depth level
// ------------------------------------------------------------------------------------------

// Node ranges of level d from the parents' partition (X is the previous level's scan), the chunk
// list and the slots of nodes that span several chunks.  One workgroup.
__global__ __launch_bounds__(1024) void k_gb_level(Ws w, int d, int max_slots, int chunk) {
    __shared__ int32_t sc[1024], ss[1024], sp[1024];
    const int L = 1 << d, base = L - 1;
    const int per = (L + 1023) / 1024;  // consecutive nodes per thread
    const int t = threadIdx.x;
    int chunks = 0, slots = 0, parts = 0;
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
        const int c = w.alive[k] ? max(1, (w.cnt[k] + chunk - 1) / chunk) : 0;
        chunks += c;
        slots += c > 1;
        parts += c > 1 ? c : 0;
    }
    sc[t] = chunks;
    ss[t] = slots;
    sp[t] = parts;
    __syncthreads();
    for (int off = 1; off < 1024; off <<= 1) {  // inclusive scans
        const int a = t >= off ? sc[t - off] : 0, b = t >= off ? ss[t - off] : 0, e = t >= off ? sp[t - off] : 0;
        __syncthreads();
        sc[t] += a;
        ss[t] += b;
        sp[t] += e;
        __syncthreads();
    }
    int c0 = sc[t] - chunks, s0 = ss[t] - slots, p0 = sp[t] - parts;
    for (int q = 0; q < per; ++q) {
        const int j = t * per + q;
        if (j >= L) break;
        const int k = base + j;
        const int c = w.alive[k] ? max(1, (w.cnt[k] + chunk - 1) / chunk) : 0;
        w.cp[j] = c0;
        w.slot[j] = -1;
        w.pbase[j] = -1;
        if (c > 1 && s0 < max_slots && p0 + c <= w.pmax) {
            w.slot[j] = s0;
            w.slot_node[s0] = j;
            w.pbase[j] = p0;
        }
        c0 += c;
        s0 += c > 1;
        p0 += c > 1 ? c : 0;
    }
    if (t == 1023) {
        w.cp[L] = sc[1023];
        w.lvl[0] = sc[1023];
        w.lvl[1] = ss[1023];
    }
}

// Evaluate the splits of features f0 .. f0 + 7 of one node from its histogram h[2][8][kBinStride]
// (LDS or global memory); thread = (feature j = t / 32, bins 8 (t % 32) ..).  Result in *out.
__device__ __forceinline__ void evaluate(const int64_t *h, int f0, int F, const float *cuts, int cut_stride,
                         const int32_t *n_cuts, const Params &prm, int eg, int eh, Best *out, Best *red) {
    const int t = threadIdx.x, j = t / 32, q = t % 32, f = f0 + j;
    int64_t pg[8], ph[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        pg[e] = h[(0 * kGroup + j) * kBinStride + 8 * q + e];
        ph[e] = h[(1 * kGroup + j) * kBinStride + 8 * q + e];
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
    // this lane's best candidate, kept in scalars (a struct copied under a condition spills)
    int bv = 0, bk = 0;
    double bg = 0.0;
    int64_t bGL = 0, bHL = 0;
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
                if (!bv || gain > bg) {
                    bv = 1;
                    bg = gain;
                    bk = (f * 256 + tt) * 2 + (1 - dir);
                    bGL = gl;
                    bHL = hl;
                }
            }
        }
    }
    // best over the 32 lanes of the feature: larger gain, then smaller key
#pragma unroll
    for (int off = 16; off > 0; off >>= 1) {
        const double og = __shfl_xor(bg, off, 32);
        const int ok = __shfl_xor(bk, off, 32), ov = __shfl_xor(bv, off, 32);
        const int64_t oGL = __shfl_xor(bGL, off, 32), oHL = __shfl_xor(bHL, off, 32);
        const bool take = ov && (!bv || og > bg || (og == bg && ok < bk));
        if (take) {
            bv = ov;
            bg = og;
            bk = ok;
            bGL = oGL;
            bHL = oHL;
        }
    }
    if (q == 0) {
        red[j].valid = bv;
        red[j].gain = bg;
        red[j].key = bk;
        red[j].GL = bGL;
        red[j].HL = bHL;
        red[j].G = Gi;
        red[j].H = Hi;
    }
    __syncthreads();
    if (t == 0) {
        int ri = 0;
        for (int i = 1; i < kGroup; ++i)
            if (better(red[i], red[ri])) ri = i;
        out->valid = red[ri].valid;
        out->gain = red[ri].gain;
        out->key = red[ri].key;
        out->GL = red[ri].GL;
        out->HL = red[ri].HL;
        out->G = red[0].G;
        out->H = red[0].H;
    }
}

struct HistArgs {
    const uint8_t *bins;
    int64_t ld;
    int F, n_fg, d, chunk;
    const float *cuts;
    int cut_stride;
    const int32_t *n_cuts;
    Params prm;
};

__global__ __launch_bounds__(kThreads) void k_gb_hist(HistArgs a, Ws w) {
    __shared__ int64_t h[kHistWords];  // 32.1 KB
    __shared__ int64_t tot[2][kThreads];
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
    const int i0 = s + (c - w.cp[j]) * a.chunk, i1 = std::min(s + n, i0 + a.chunk);
    for (int e = t; e < kHistWords; e += kThreads) h[e] = 0;
    const int f0 = fg * kGroup;
    const int nf = std::min(kGroup, a.F - f0);
    // the bin of 0.0 (statement features are mostly zeros) is not added row by row: it is the
    // chunk's total minus the other bins, exact in integers.  At add step e lane l adds feature
    // (e + l) % 8, so one instruction spreads its lanes over the 8 features and at most 8 of
    // them can meet on one bin.
    int zb[kGroup];
#pragma unroll
    for (int e = 0; e < kGroup; ++e) {
        const int jj = (e + t) % kGroup;
        zb[e] = jj < nf ? w.zb[f0 + jj] : -1;
    }
    __syncthreads();
    int64_t sg = 0, sh = 0;
    constexpr int U = kChunk / kThreads;
    for (int b0 = i0; b0 < i1; b0 += kChunk) {  // 2048 rows at a time, every load issued before the adds
        int rr[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int i = b0 + t + kThreads * u;
            rr[u] = i < i1 ? w.order[i] : -1;
        }
        uint64_t word[U];
        int64_t qg[U], qh[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int r = rr[u] < 0 ? 0 : rr[u];
            word[u] = *reinterpret_cast<const uint64_t *>(a.bins + ((int64_t)fg * a.ld + r) * kGroup);
            qg[u] = w.qg[r];
            qh[u] = w.qh[r];
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            if (rr[u] < 0) break;
            sg += qg[u];
            sh += qh[u];
#pragma unroll
            for (int e = 0; e < kGroup; ++e) {
                const int jj = (e + t) % kGroup;
                const int b = (int)((word[u] >> (8 * jj)) & 255u);
                if (zb[e] >= 0 && b != zb[e]) {
                    atomicAdd(reinterpret_cast<unsigned long long *>(&h[(0 * kGroup + jj) * kBinStride + b]),
                              (unsigned long long)qg[u]);
                    atomicAdd(reinterpret_cast<unsigned long long *>(&h[(1 * kGroup + jj) * kBinStride + b]),
                              (unsigned long long)qh[u]);
                }
            }
        }
    }
    tot[0][t] = sg;
    tot[1][t] = sh;
    __syncthreads();
    for (int off = kThreads / 2; off > 0; off >>= 1) {
        if (t < off) {
            tot[0][t] += tot[0][t + off];
            tot[1][t] += tot[1][t + off];
        }
        __syncthreads();
    }
    {  // zero bin = total - the other bins: 16 threads per (G|H, feature) row, 16 bins each
        const int row = t / 16, part = t % 16, gh = row / kGroup, jj = row % kGroup;
        const int b0 = jj < nf ? w.zb[f0 + jj] : -1;
        int64_t *hr = &h[(gh * kGroup + jj) * kBinStride];
        int64_t rest = 0;
#pragma unroll
        for (int e = 0; e < 16; ++e) {
            const int b = part * 16 + e;
            rest += b == b0 ? 0 : hr[b];
        }
#pragma unroll
        for (int off = 8; off > 0; off >>= 1) rest += __shfl_xor(rest, off, 16);
        __syncthreads();
        if (part == 0 && b0 >= 0) hr[b0] = tot[gh][0] - rest;
    }
    __syncthreads();
    if (nch == 1) {
        evaluate(h, f0, a.F, a.cuts, a.cut_stride, a.n_cuts, a.prm, w.exps[0], w.exps[1],
                 &w.best[(int64_t)j * a.n_fg + fg], red);
        return;
    }
    if (w.pbase[j] < 0) return;  // cannot happen: every multi-chunk node has its partials
    int64_t *g = w.part + ((int64_t)(w.pbase[j] + c - w.cp[j]) * a.n_fg + fg) * kHistWords;
    for (int e = t; e < kHistWords; e += kThreads) g[e] = h[e];
}

// The histogram of a multi-chunk node: the sum of its chunks' partial histograms, in chunk
// order (integers: exact).  Workgroup = (slot, feature group, 1/8 of the words).
__global__ __launch_bounds__(kThreads) void k_gb_reduce(HistArgs a, Ws w) {
    const int sidx = blockIdx.x, fg = blockIdx.y;
    if (sidx >= w.lvl[1]) return;
    const int j = w.slot_node[sidx];
    const int nch = w.cp[j + 1] - w.cp[j], pb = w.pbase[j];
    const int64_t stride = (int64_t)a.n_fg * kHistWords;
    const int64_t *src = w.part + ((int64_t)pb * a.n_fg + fg) * kHistWords;
    int64_t *dst = w.hist + ((int64_t)sidx * a.n_fg + fg) * kHistWords;
    constexpr int per = (kHistWords + 7) / 8;
    for (int e = blockIdx.z * per + threadIdx.x; e < std::min(kHistWords, (int)(blockIdx.z + 1) * per); e += kThreads) {
        int64_t acc = 0;
        int q = 0;
        for (; q + 8 <= nch; q += 8) {  // eight loads in flight, added in chunk order
            int64_t v[8];
#pragma unroll
            for (int u = 0; u < 8; ++u) v[u] = src[(int64_t)(q + u) * stride + e];
#pragma unroll
            for (int u = 0; u < 8; ++u) acc += v[u];
        }
        for (; q < nch; ++q) acc += src[(int64_t)q * stride + e];
        dst[e] = acc;
    }
}

__global__ __launch_bounds__(kThreads) void k_gb_split(HistArgs a, Ws w) {
    __shared__ Best red[kGroup];
    const int sidx = blockIdx.x, fg = blockIdx.y;
    if (sidx >= w.lvl[1]) return;
    const int j = w.slot_node[sidx];
    const int64_t *g = w.hist + ((int64_t)sidx * a.n_fg + fg) * kHistWords;
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

// One wave per node: lane i < n_fg holds feature group i's record; the best (larger gain, then the
// smaller key, as in the evaluation) is found by a shuffle reduction, then lane 0 writes.
__global__ __launch_bounds__(kThreads) void k_gb_decide(Ws w, int d, int n_fg, const float *__restrict__ cuts,
                                                        int cut_stride, Params prm, TreeOut tr) {
    const int j = blockIdx.x * (kThreads / 64) + threadIdx.x / 64, lane = threadIdx.x % 64, L = 1 << d;
    if (j >= L) return;
    const int k = L - 1 + j;
    if (!w.alive[k]) return;
    const Best *bs = w.best + (int64_t)j * n_fg;
    int bv = 0, bk = 0;
    double bg = 0.0;
    int64_t bGL = 0, bHL = 0;
    for (int i = lane; i < n_fg; i += 64) {  // n_fg <= 512: records i, i + 64, ... in order
        const Best &o = bs[i];
        if (o.valid && (!bv || o.gain > bg || (o.gain == bg && o.key < bk))) {
            bv = 1;
            bg = o.gain;
            bk = o.key;
            bGL = o.GL;
            bHL = o.HL;
        }
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
        const double og = __shfl_xor(bg, off);
        const int ok = __shfl_xor(bk, off), ov = __shfl_xor(bv, off);
        const int64_t oGL = __shfl_xor(bGL, off), oHL = __shfl_xor(bHL, off);
        if (ov && (!bv || og > bg || (og == bg && ok < bk))) {
            bv = ov;
            bg = og;
            bk = ok;
            bGL = oGL;
            bHL = oHL;
        }
    }
    if (lane != 0) return;
    const int64_t G = bs[0].G, H = bs[0].H;
    w.Gt[k] = G;
    w.Ht[k] = H;
    if (bv && bg > prm.gamma) {
        const int f = bk / 512, tt = (bk / 2) % 256, dir = 1 - (bk & 1);
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
        w.Gt[2 * k + 1] = bGL;
        w.Ht[2 * k + 1] = bHL;
        w.Gt[2 * k + 2] = G - bGL;
        w.Ht[2 * k + 2] = H - bHL;
    } else {
        tr.leaf_value[k] = leaf_weight(G, H, w.exps[0], w.exps[1], prm);
    }
}

// Direction of every row of a node split at this level (left = 1; rows of other nodes stay, as
// "left"), the row's new node, and the number of lefts per block of kScanBlock positions.
__global__ __launch_bounds__(kThreads) void k_gb_flags(Ws w, int N, const uint8_t *__restrict__ bins, int64_t ld) {
    __shared__ int32_t s[kThreads];
    const int i = blockIdx.x * kScanBlock + threadIdx.x;
    int go_left = 0;
    if (i < N) {
        const int r = w.order[i], k = w.nid[r];
        const int f = w.sf[k];
        int sp = -1;
        go_left = 1;
        if (f >= 0) {
            const int b = bins[((int64_t)(f / kGroup) * ld + r) * kGroup + f % kGroup];
            go_left = b == 255 ? w.sd[k] : b < w.st[k];
            w.nid[r] = go_left ? 2 * k + 1 : 2 * k + 2;
            sp = k;
        }
        w.flag[i] = go_left;
        w.spn[i] = sp;
    }
    s[threadIdx.x] = go_left;
    __syncthreads();
    for (int off = kThreads / 2; off > 0; off >>= 1) {
        if (threadIdx.x < off) s[threadIdx.x] += s[threadIdx.x + off];
        __syncthreads();
    }
    if (threadIdx.x == 0) w.bsum[blockIdx.x] = s[0];
}

// exclusive scan of flag[0..N) into X[0..N]: block sums (k_gb_flags), a one-workgroup scan of
// them, the final pass
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
    const int i = blockIdx.x * kScanBlock + threadIdx.x;
    const int v = i < N ? w.flag[i] : 0;
    s[threadIdx.x] = v;
    __syncthreads();
    for (int off = 1; off < kThreads; off <<= 1) {
        const int a = threadIdx.x >= off ? s[threadIdx.x - off] : 0;
        __syncthreads();
        s[threadIdx.x] += a;
        __syncthreads();
    }
    if (i < N) w.X[i] = w.bsum[blockIdx.x] + s[threadIdx.x] - v;
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

// The last level's leaves (threads j < 2^D) and every row's margin update (threads r < N): a row in
// a last-level leaf takes that leaf's weight directly, a row in an earlier leaf reads it.
__global__ __launch_bounds__(kThreads) void k_gb_finish(Ws w, int D, Params prm, int N, float *leaf_value,
                                                        float *__restrict__ margin) {
    const int i = blockIdx.x * kThreads + threadIdx.x, L = 1 << D;
    const int eg = w.exps[0], eh = w.exps[1];
    if (i < L && w.alive[L - 1 + i]) leaf_value[L - 1 + i] = leaf_weight(w.Gt[L - 1 + i], w.Ht[L - 1 + i], eg, eh, prm);
    if (i < N) {
        const int k = w.nid[i];
        const float v = k >= L - 1 ? leaf_weight(w.Gt[k], w.Ht[k], eg, eh, prm) : leaf_value[k];
        margin[i] = margin[i] + v;
    }
}

// ------------------------------------------------------------------------------------------
// workspace
// ------------------------------------------------------------------------------------------
struct Layout {
    size_t off[32];
    size_t total;
};

// Rows per histogram workgroup: at least 4096 (fewer multi-chunk nodes, each with fewer partials:
// 737 -> 637 us per round on 66,923 rows against 2048; 8192 measured 657 us), more for large sets,
// so that a level launches about 4,096 (chunk, feature group) workgroups and stores that many
// partial histograms at most.
int chunk_rows(int N, int F) {
    const int n_fg = (F + kGroup - 1) / kGroup;
    const int64_t m = (int64_t)N * n_fg / ((int64_t)4096 * kChunk);
    return kChunk * (int)std::max<int64_t>(2, std::min<int64_t>(m, 64));
}

int max_slots_for(int N, int F, int depth) {
    const int64_t by_rows = (int64_t)N / (chunk_rows(N, F) + 1);
    const int64_t by_nodes = (int64_t)1 << (depth - 1);
    return (int)std::min(by_rows, by_nodes);
}

Ws carve(void *base, int F, int N, int P, int depth, size_t *total) {
    const int n_fg = (F + kGroup - 1) / kGroup;
    const int64_t n_nodes = ((int64_t)1 << (depth + 1)) - 1;
    const int64_t Lmax = (int64_t)1 << (depth - 1);  // widest level that builds histograms
    const int64_t nblk = ceil_div(std::max(P, 1), kThreads);
    const int64_t nb = ceil_div(std::max(N, 1), kScanBlock);
    const int S = max_slots_for(N, F, depth);
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
    w.zb = reinterpret_cast<int32_t *>(take(sizeof(int32_t) * F));
    w.pbase = reinterpret_cast<int32_t *>(take(sizeof(int32_t) * Lmax));
    // a multi-chunk node of n > CH rows has ceil(n / CH) < 2 n / CH chunks: fewer than 2 N / CH in all
    w.pmax = (int)(2 * ceil_div(std::max(N, 1), chunk_rows(N, F)));
    w.part = reinterpret_cast<int64_t *>(take(sizeof(int64_t) * (size_t)w.pmax * n_fg * kHistWords));
    w.best = reinterpret_cast<Best *>(take(sizeof(Best) * Lmax * n_fg));
    w.hist = reinterpret_cast<int64_t *>(take(sizeof(int64_t) * (size_t)std::max(S, 1) * n_fg * kHistWords));
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
    // bytes of features past F in the last group are written as zeros
    // several row blocks per cut staging on large sets, while keeping about 2,048 workgroups
    const int64_t n_g = ceil_div(F, kGroup);
    const int rb_per = (int)std::max<int64_t>(1, std::min<int64_t>(kBinRowBlocks, ceil_div(N, kThreads) * n_g / 2048));
    const dim3 grid((unsigned)ceil_div(N, kThreads * rb_per), (unsigned)n_g);
    hipLaunchKernelGGL(k_gb_bin, grid, dim3(kThreads), 0, stream, x, ldx, F, N, cuts, cut_stride, n_cuts, bins, ld,
                       rb_per);
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
    const int S = max_slots_for(N, F, D);
    const int CH = chunk_rows(N, F);
    TreeOut tr{feature, threshold, left, right, default_left, leaf_value};
    const int init_n = std::max(std::max(n_nodes, N), F);
    hipLaunchKernelGGL(k_gb_init, dim3((unsigned)ceil_div(init_n, kThreads)), dim3(kThreads), 0, stream, w, n_nodes, N,
                       F, cuts, cut_stride, n_cuts, feature, threshold, left, right, default_left, leaf_value);
    const int nblk = (int)ceil_div(std::max(P, 1), kThreads);
    hipLaunchKernelGGL(k_gb_prog_grad, dim3(nblk), dim3(kThreads), 0, stream, margin, prog_ptr, P, label, weight,
                       prm.base, N, w);
    hipLaunchKernelGGL(k_gb_exps, dim3(1), dim3(kThreads), 0, stream, w, nblk, (int64_t)N);
    hipLaunchKernelGGL(k_gb_row_q, dim3(nblk), dim3(kThreads), 0, stream, prog_ptr, P, N, w);
    HARL_HIP_CHECK(hipGetLastError());
    HistArgs ha{bins, ld, F, n_fg, 0, CH, cuts, cut_stride, n_cuts, prm};
    const unsigned rows_grid = (unsigned)ceil_div(std::max(N, 1), kThreads);
    const int nb = (int)ceil_div(std::max(N, 1), kScanBlock);
    for (int d = 0; d < D; ++d) {
        const int L = 1 << d;
        hipLaunchKernelGGL(k_gb_level, dim3(1), dim3(1024), 0, stream, w, d, S, CH);
        const int slots = std::min(S, L);
        ha.d = d;
        const unsigned chunk_bound = (unsigned)(ceil_div(N, CH) + L);
        hipLaunchKernelGGL(k_gb_hist, dim3(chunk_bound, (unsigned)n_fg), dim3(kThreads), 0, stream, ha, w);
        if (slots > 0) {
            hipLaunchKernelGGL(k_gb_reduce, dim3((unsigned)slots, (unsigned)n_fg, 8), dim3(kThreads), 0, stream, ha, w);
            hipLaunchKernelGGL(k_gb_split, dim3((unsigned)slots, (unsigned)n_fg), dim3(kThreads), 0, stream, ha, w);
        }
        hipLaunchKernelGGL(k_gb_decide, dim3((unsigned)ceil_div(L, kThreads / 64)), dim3(kThreads), 0, stream, w, d, n_fg,
                           cuts, cut_stride, prm, tr);
        if (N > 0) {
            hipLaunchKernelGGL(k_gb_flags, dim3((unsigned)nb), dim3(kThreads), 0, stream, w, N, bins, ld);
            hipLaunchKernelGGL(k_gb_scan_top, dim3(1), dim3(1024), 0, stream, w, nb);
            hipLaunchKernelGGL(k_gb_scan_final, dim3((unsigned)nb), dim3(kThreads), 0, stream, w, N, nb);
            hipLaunchKernelGGL(k_gb_scatter, dim3(rows_grid), dim3(kThreads), 0, stream, w, N);
            std::swap(w.order, w.order2);
        }
        HARL_HIP_CHECK(hipGetLastError());
    }
    hipLaunchKernelGGL(k_gb_finish, dim3((unsigned)ceil_div(std::max(1 << D, N), kThreads)), dim3(kThreads), 0, stream,
                       w, D, prm, N, leaf_value, margin);
    HARL_HIP_CHECK(hipGetLastError());
    return HARL_OK;
}

}  // namespace harl
