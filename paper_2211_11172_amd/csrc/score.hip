// Cost-model scoring of one search round: C(S') for every candidate (Algorithm 1 of the HARL
// paper; the cost model is an XGBoost ensemble, Section 6.1 and Appendix A.2).  A candidate is a
// program of statements; each statement row has F fp32 features; the program score is the base
// score plus the sum over its statements of the ensemble's leaf sum.
//
// K1 tree traversal.  A workgroup owns a tile of statement rows and one group of trees.  The
//   tile's features are staged once into LDS, feature-major ([F][rows] fp32, so a lane's gather
//   of any feature of its own row hits bank = lane: conflict-free whatever feature a node asks
//   for).  Lane = row.  Each level of a walk issues the current node's feature read together with
//   the read of both its children (16 bytes) and picks the child in registers, so a level costs
//   one LDS round trip; the leaf pair comes with the last level.  Row sums are accumulated in fp64
//   and combined over the waves in a fixed order.  Two variants:
//   k_tree_score_wp (depth <= 8): every wave streams its own trees (tree t + k*TW) through a
//     private two-slot LDS ring -- the next tree is fetched into registers while the current one
//     is walked -- so waves never wait on each other between the feature staging and the final
//     reduction.  Each lane walks RPL rows per tree (ILP across rows; the staged tree serves
//     64*RPL rows).
//   k_tree_score_ch (deeper trees, whose 2^depth-node trees are too big for per-wave rings): the
//     workgroup stages chunks of TW*ILP trees shared by all waves, the next chunk fetched into
//     registers during the walk of the current one.
// K2 k_segsum: one wave per program sums its rows' partial slots in a fixed order (fp64).
//
// Grid mapping is XCD-aware: workgroup b takes tree group b % G and row tile b / G; workgroups
// are dealt to the 8 XCDs round-robin, so with G in {2,4,8} every XCD's L2 only ever holds its
// own share of the ensemble.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <vector>

#include "internal.hpp"

namespace harl {
namespace {

constexpr int kWave = 64;
constexpr int kLdsBytes = 160 * 1024;

constexpr int tree_stride_bytes(int D) { return ((1 << D) * 12 + 15) / 16 * 16; }

// Packed tree (1-based breadth-first): byte 8*i holds internal node i (i = 1 .. 2^D - 1; bytes 0..7
// are padding), so the two children of node i sit together, 16-byte aligned, at byte 16*i; the
// 2^D leaves follow at byte 8 * 2^D, the two leaves below a last-level node i at
// 8 * 2^D + 8*i - 4 * 2^D.
template <bool NAN_AWARE>
__device__ __forceinline__ uint32_t go_right(float x, float thr, uint32_t word) {
    uint32_t right = x >= thr ? 1u : 0u;
    if (NAN_AWARE) right |= (x != x && !(word & kNodeDefaultLeft)) ? 1u : 0u;
    return right;
}

// Walk NT_ trees at LDS byte offsets tb[] for R rows of this lane (feature tile row stride RT4
// bytes per feature; lane_off[r] = byte offset of the lane's r-th row).  Every (tree, row) pair is
// an independent chain; all chains of a level are issued together.
template <int D, int NT_, int R, uint32_t RT4, bool NAN_AWARE>
__device__ __forceinline__ void walk_trees(const char *smem, const uint32_t (&tb)[NT_], const uint32_t (&lane_off)[R],
                                           double (&acc)[R]) {
    constexpr uint32_t kLeafBase = 8u << D;
    uint32_t idx[NT_][R], word[NT_][R];
    float thr[NT_][R];
#pragma unroll
    for (int i = 0; i < NT_; ++i) {
        const uint2 root = *reinterpret_cast<const uint2 *>(smem + tb[i] + 8u);
#pragma unroll
        for (int r = 0; r < R; ++r) {
            word[i][r] = root.x;
            thr[i][r] = __uint_as_float(root.y);
            idx[i][r] = 1;
        }
    }
#pragma unroll
    for (int lvl = 0; lvl + 1 < D; ++lvl) {
        float x[NT_][R];
        uint4 kids[NT_][R];
#pragma unroll
        for (int i = 0; i < NT_; ++i)
#pragma unroll
            for (int r = 0; r < R; ++r) {
                x[i][r] = *reinterpret_cast<const float *>(smem + __umul24(word[i][r], RT4) + lane_off[r]);
                kids[i][r] = *reinterpret_cast<const uint4 *>(smem + tb[i] + idx[i][r] * 16u);
            }
#pragma unroll
        for (int i = 0; i < NT_; ++i)
#pragma unroll
            for (int r = 0; r < R; ++r) {
                const uint32_t g = go_right<NAN_AWARE>(x[i][r], thr[i][r], word[i][r]);
                idx[i][r] = 2u * idx[i][r] + g;
                word[i][r] = g ? kids[i][r].z : kids[i][r].x;
                thr[i][r] = __uint_as_float(g ? kids[i][r].w : kids[i][r].y);
            }
    }
    float x[NT_][R];
    float2 lv[NT_][R];
#pragma unroll
    for (int i = 0; i < NT_; ++i)
#pragma unroll
        for (int r = 0; r < R; ++r) {
            x[i][r] = *reinterpret_cast<const float *>(smem + __umul24(word[i][r], RT4) + lane_off[r]);
            lv[i][r] = *reinterpret_cast<const float2 *>(smem + tb[i] + kLeafBase + idx[i][r] * 8u - (4u << D));
        }
#pragma unroll
    for (int i = 0; i < NT_; ++i)
#pragma unroll
        for (int r = 0; r < R; ++r)
            acc[r] += (double)(go_right<NAN_AWARE>(x[i][r], thr[i][r], word[i][r]) ? lv[i][r].y : lv[i][r].x);
}

// Stage rows [row0, row0 + RT) of every feature into LDS ([F][RT] fp32, zero past n_rows), with
// 8 loads in flight per thread; returns (block-wide) whether any staged value is NaN.
template <int RT, int NT>
__device__ __forceinline__ int stage_features(char *smem, const float *__restrict__ X, int64_t ld, int n_rows, int F,
                                              int vec_ok, int row0) {
    constexpr int V = RT / 4;  // float4 per feature row of the tile
    constexpr int B = 8;
    int has_nan = 0;
    const int total = F * V;
    float4 *dst = reinterpret_cast<float4 *>(smem);
    for (int i0 = threadIdx.x; i0 < total; i0 += B * NT) {
        float4 v[B];
#pragma unroll
        for (int j = 0; j < B; ++j) {
            const int i = i0 + j * NT;
            v[j] = make_float4(0.f, 0.f, 0.f, 0.f);
            if (i < total) {
                const int f = i / V, r = row0 + 4 * (i % V);
                const float *src = X + (int64_t)f * ld + r;
                if (vec_ok && r + 3 < n_rows) {
                    v[j] = *reinterpret_cast<const float4 *>(src);
                } else {
                    if (r + 0 < n_rows) v[j].x = src[0];
                    if (r + 1 < n_rows) v[j].y = src[1];
                    if (r + 2 < n_rows) v[j].z = src[2];
                    if (r + 3 < n_rows) v[j].w = src[3];
                }
            }
        }
#pragma unroll
        for (int j = 0; j < B; ++j) {
            const int i = i0 + j * NT;
            if (i < total) {
                has_nan |= (v[j].x != v[j].x) | (v[j].y != v[j].y) | (v[j].z != v[j].z) | (v[j].w != v[j].w);
                dst[i] = v[j];
            }
        }
    }
    return __syncthreads_or(has_nan);
}

// Fixed-order combination of the per-wave row sums (acc[r] of wave w for tile row r*64 + lane),
// written as fp32 partials out[t] for tile rows t with row0 + t < n_rows.  `red` must not overlap
// live data.
template <int RPL, int NW>
__device__ __forceinline__ void reduce_rows(double *red, const double (&acc)[RPL], int wid, int lane, int row0, int n_rows,
                                            float *__restrict__ out) {
    constexpr int RT = 64 * RPL;
#pragma unroll
    for (int r = 0; r < RPL; ++r) red[wid * RT + r * 64 + lane] = acc[r];
    __syncthreads();
    for (int t = threadIdx.x; t < RT; t += NW * kWave) {
        double s = 0.0;
#pragma unroll
        for (int w = 0; w < NW; ++w) s += red[w * RT + t];
        if (row0 + t < n_rows) out[t] = (float)s;
    }
}

// Per-wave tree staging: lane l moves uint4 j*64 + l of a packed tree (S16 uint4 in all).
template <int S16, int PF>
__device__ __forceinline__ void wave_fetch(uint4 (&pf)[PF], const uint4 *__restrict__ src, int lane) {
#pragma unroll
    for (int j = 0; j < PF; ++j)
        if (S16 % kWave == 0 || j * kWave + lane < S16) pf[j] = src[j * kWave + lane];
}

template <int S16, int PF>
__device__ __forceinline__ void wave_commit(const uint4 (&pf)[PF], uint4 *dst, int lane) {
#pragma unroll
    for (int j = 0; j < PF; ++j)
        if (S16 % kWave == 0 || j * kWave + lane < S16) dst[j * kWave + lane] = pf[j];
}

// ---- K1, depth <= 8: persistent workgroups with per-wave private tree rings ----
// The work is the space of (row tile, tree) pairs, tile-major: v = tile * T + tree.  Workgroup b
// owns the contiguous slice [b*L, (b+1)*L), so every workgroup walks the same number of trees and
// the machine is busy to the end.  The partial sums of the piece of tile i walked by workgroup b are
// stored at block (i + b) of RT floats: a workgroup covers a contiguous run of tiles, so i + b
// grows strictly along the (workgroup, tile) pieces and (tiles + workgroups) blocks hold them all;
// a tile's pieces are summed later in workgroup order.
template <int D, int RPL, int TW>
__global__ __launch_bounds__(64 * TW) void k_tree_score_wp(
    const float *__restrict__ X, int64_t ld, int n_rows, int F, int vec_ok, const uint4 *__restrict__ trees,
    int T, int64_t V, int64_t L, float *__restrict__ partial) {
    constexpr int RT = 64 * RPL;
    constexpr int S16 = tree_stride_bytes(D) / 16;  // uint4 per packed tree
    constexpr int PF = (S16 + kWave - 1) / kWave;   // uint4 per lane per tree
    extern __shared__ __align__(16) char smem[];

    const int64_t v_begin = (int64_t)blockIdx.x * L;
    const int64_t v_end = v_begin + L < V ? v_begin + L : V;
    if (v_begin >= v_end) return;  // whole workgroup: no barrier is skipped by part of it
    const int wid = threadIdx.x / kWave, lane = threadIdx.x % kWave;
    const uint32_t ring_off = (uint32_t)F * RT * 4u;
    char *const ring = smem + ring_off + (uint32_t)wid * 2u * (S16 * 16);

    uint4 pf[PF];
#pragma unroll
    for (int j = 0; j < PF; ++j) pf[j] = make_uint4(0, 0, 0, 0);
    uint32_t lane_off[RPL];
#pragma unroll
    for (int r = 0; r < RPL; ++r) lane_off[r] = (uint32_t)(r * 64 + lane) * 4u;

    int64_t v = v_begin;
    int tile = (int)(v / T);
    int t0 = (int)(v % T);
    int t1 = (int)(T - t0 < v_end - v ? T : t0 + (v_end - v));
    int t = t0 + wid;
    if (t < t1) wave_fetch<S16>(pf, trees + (int64_t)t * S16, lane);   // overlaps the feature staging
    while (true) {
        const int row0 = tile * RT;
        const int has_nan = stage_features<RT, 64 * TW>(smem, X, ld, n_rows, F, vec_ok, row0);
        if (t < t1) wave_commit<S16>(pf, reinterpret_cast<uint4 *>(ring), lane);
        if (t + TW < t1) wave_fetch<S16>(pf, trees + (int64_t)(t + TW) * S16, lane);
        double acc[RPL];
#pragma unroll
        for (int r = 0; r < RPL; ++r) acc[r] = 0.0;
        int s = 0;
        for (; t < t1; t += TW) {
            const uint32_t tb[1] = {ring_off + (uint32_t)wid * 2u * (S16 * 16) + (uint32_t)s * (S16 * 16)};
            if (has_nan)
                walk_trees<D, 1, RPL, (uint32_t)RT * 4u, true>(smem, tb, lane_off, acc);
            else
                walk_trees<D, 1, RPL, (uint32_t)RT * 4u, false>(smem, tb, lane_off, acc);
            if (t + TW < t1) {                 // LDS ops of a wave run in order: the walk's reads of
                                               // slot s complete before the next commit overwrites it
                wave_commit<S16>(pf, reinterpret_cast<uint4 *>(ring + (uint32_t)(s ^ 1) * (S16 * 16)), lane);
                if (t + 2 * TW < t1) wave_fetch<S16>(pf, trees + (int64_t)(t + 2 * TW) * S16, lane);
            }
            s ^= 1;
        }
        // the next piece (if any) starts at tree 0 of the next tile: prefetch its first tree now
        v += t1 - t0;
        const bool next = v < v_end;
        const int nt1 = next ? (int)(T < v_end - v ? T : v_end - v) : 0;
        if (next && wid < nt1) wave_fetch<S16>(pf, trees + (int64_t)wid * S16, lane);
        __syncthreads();  // every wave is done with its ring: reuse the ring region for the reduction
        reduce_rows<RPL, TW>(reinterpret_cast<double *>(smem + ring_off), acc, wid, lane, row0, n_rows,
                             partial + ((int64_t)tile + blockIdx.x) * RT);
        if (!next) break;
        ++tile;
        t0 = 0;
        t1 = nt1;
        t = wid;
    }
}

// Workgroup chunk staging: thread t moves uint4 t + j*NT of C consecutive packed trees starting
// at tree t0; slots past t_end are zero (a zero tree reaches a 0.0 leaf).
template <int C, int S16, int NT, int NPF>
__device__ __forceinline__ void block_fetch(uint4 (&pf)[NPF], const uint4 *__restrict__ trees, int t0, int t_end) {
    const int valid16 = min(C, t_end - t0) * S16;
    const uint4 *src = trees + (int64_t)t0 * S16;
#pragma unroll
    for (int j = 0; j < NPF; ++j) {
        const int i = threadIdx.x + j * NT;
        pf[j] = i < valid16 ? src[i] : make_uint4(0, 0, 0, 0);
    }
}

template <int C, int S16, int NT, int NPF>
__device__ __forceinline__ void block_commit(const uint4 (&pf)[NPF], uint4 *dst) {
#pragma unroll
    for (int j = 0; j < NPF; ++j) {
        const int i = threadIdx.x + j * NT;
        if (i < C * S16) dst[i] = pf[j];
    }
}

// ---- K1, deeper trees: chunks of TW*ILP trees shared by the workgroup ----
template <int D, int TW, int ILP>
__global__ __launch_bounds__(64 * TW) void k_tree_score_ch(
    const float *__restrict__ X, int64_t ld, int n_rows, int F, int vec_ok, const uint4 *__restrict__ trees,
    int n_trees, int trees_per_group, int n_groups, float *__restrict__ partial, int64_t ldp) {
    constexpr int RT = 64;
    constexpr int NT = 64 * TW;
    constexpr int C = TW * ILP;                       // trees per chunk
    constexpr int S16 = tree_stride_bytes(D) / 16;    // uint4 per packed tree
    constexpr int CH16 = C * S16;                     // uint4 per chunk
    constexpr int NPF = (CH16 + NT - 1) / NT;         // uint4 prefetched per thread
    extern __shared__ __align__(16) char smem[];

    const int g = blockIdx.x % n_groups;
    const int row0 = (blockIdx.x / n_groups) * RT;
    const int t_begin = g * trees_per_group;
    const int t_end = min(n_trees, t_begin + trees_per_group);
    const uint32_t chunk_off = (uint32_t)F * RT * 4u;

    uint4 pf[NPF];
    if (t_begin < t_end) block_fetch<C, S16, NT>(pf, trees, t_begin, t_end);
    const int has_nan = stage_features<RT, NT>(smem, X, ld, n_rows, F, vec_ok, row0);
    if (t_begin < t_end) block_commit<C, S16, NT>(pf, reinterpret_cast<uint4 *>(smem + chunk_off));
    __syncthreads();

    const int wid = threadIdx.x / kWave, lane = threadIdx.x % kWave;
    const uint32_t lane_off[1] = {(uint32_t)lane * 4u};
    double acc[1] = {0.0};
    for (int t0 = t_begin; t0 < t_end; t0 += C) {
        const bool more = t0 + C < t_end;
        if (more) block_fetch<C, S16, NT>(pf, trees, t0 + C, t_end);
        uint32_t tb[ILP];
#pragma unroll
        for (int i = 0; i < ILP; ++i) tb[i] = chunk_off + (uint32_t)(wid * ILP + i) * (S16 * 16);
        if (has_nan)
            walk_trees<D, ILP, 1, (uint32_t)RT * 4u, true>(smem, tb, lane_off, acc);
        else
            walk_trees<D, ILP, 1, (uint32_t)RT * 4u, false>(smem, tb, lane_off, acc);
        __syncthreads();
        if (more) {
            block_commit<C, S16, NT>(pf, reinterpret_cast<uint4 *>(smem + chunk_off));
            __syncthreads();
        }
    }
    reduce_rows<1, TW>(reinterpret_cast<double *>(smem + chunk_off), acc, wid, lane, row0, n_rows,
                       partial + (int64_t)g * ldp + row0);
}

// K2: one wave per program (lane = statement row, looping for programs of more than 64 rows).
// Each row sums its partials in a fixed order (fp64) -- grouped layout (L == 0): `groups` slots
// partial[g * ldp + r]; sliced layout: the workgroups b = first..last whose slices cut the row's
// tile i (RT rows, T trees), at partial[(i + b) * RT + r % RT] -- and the wave then sums its rows
// with a fixed xor-butterfly, so the result does not depend on scheduling.
__global__ __launch_bounds__(256) void k_segsum(const float *__restrict__ partial, int64_t ldp, int rt_shift, int T,
                                                int64_t L, int groups, const int32_t *__restrict__ prog_ptr, int n_prog,
                                                int n_rows, float base_score, float *__restrict__ prog_score,
                                                float *__restrict__ stmt_score) {
    const int p = blockIdx.x * 4 + threadIdx.x / kWave;
    const int lane = threadIdx.x % kWave;
    if (p >= n_prog) return;  // whole wave
    const int b = min(max(prog_ptr[p], 0), n_rows);
    const int e = min(max(prog_ptr[p + 1], b), n_rows);
    double acc = 0.0;
    for (int r = b + lane; r < e; r += kWave) {
        double s = 0.0;
        if (L == 0) {
            for (int gi = 0; gi < groups; ++gi) s += (double)partial[(int64_t)gi * ldp + r];
        } else {
            const int64_t tile = r >> rt_shift;
            const int64_t first = tile * T / L, last = ((tile + 1) * T - 1) / L;
            const float *src = partial + (tile << rt_shift) + (r & ((1 << rt_shift) - 1));
            for (int64_t wb = first; wb <= last; ++wb) s += (double)src[wb << rt_shift];
        }
        if (stmt_score) stmt_score[r] = (float)s;
        acc += s;
    }
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) acc += __shfl_xor(acc, m, kWave);
    if (lane == 0) prog_score[p] = (float)((double)base_score + acc);
}

// ---------------------------------------------------------------------------------------------
// launch configuration
// ---------------------------------------------------------------------------------------------
using ChKernel = void (*)(const float *, int64_t, int, int, int, const uint4 *, int, int, int, float *, int64_t);
using WpKernel = void (*)(const float *, int64_t, int, int, int, const uint4 *, int, int64_t, int64_t, float *);

struct ScoreCfg {
    bool wp;            // persistent per-wave rings (else grid of shared chunks)
    int a, b;           // wp: RPL, TW;  ch: TW, ILP
    const void *kern;
    int rows_per_tile, threads;
    size_t lds;
};

template <int D>
const void *pick_wp(int rpl, int tw) {
    if constexpr (D <= 8) {
#define HARL_WP(R, T) \
    if (rpl == R && tw == T) return reinterpret_cast<const void *>(k_tree_score_wp<D, R, T>);
        HARL_WP(1, 4) HARL_WP(1, 8) HARL_WP(1, 16) HARL_WP(2, 4) HARL_WP(2, 8) HARL_WP(2, 12)
#undef HARL_WP
    }
    return nullptr;
}

template <int D>
const void *pick_ch(int tw, int ilp) {
#define HARL_CH(T, I) \
    if (tw == T && ilp == I) return reinterpret_cast<const void *>(k_tree_score_ch<D, T, I>);
    HARL_CH(2, 1) HARL_CH(4, 1) HARL_CH(8, 1) HARL_CH(4, 2)
#undef HARL_CH
    return nullptr;
}

template <int... Ds>
const void *pick_depth(int depth, bool wp, int a, int b, std::integer_sequence<int, Ds...>) {
    const void *k = nullptr;
    ((depth == Ds + 1 ? (void)(k = wp ? pick_wp<Ds + 1>(a, b) : pick_ch<Ds + 1>(a, b)) : (void)0), ...);
    return k;
}

ScoreCfg make_cfg(const harl_ensemble *E, bool wp, int a, int b) {
    ScoreCfg c{wp, a, b, pick_depth(E->depth, wp, a, b, std::make_integer_sequence<int, kMaxDepth>{}), 0, 0, 0};
    const size_t stride = (size_t)E->tree_stride;
    if (wp) {
        c.rows_per_tile = 64 * a;
        c.threads = 64 * b;
        const size_t ring = (size_t)b * 2 * stride, red = (size_t)b * c.rows_per_tile * 8;
        c.lds = (size_t)E->n_features * c.rows_per_tile * 4 + (ring > red ? ring : red);
    } else {
        c.rows_per_tile = 64;
        c.threads = 64 * a;
        const size_t chunk = (size_t)a * b * stride, red = (size_t)a * 64 * 8;
        c.lds = (size_t)E->n_features * 64 * 4 + (chunk > red ? chunk : red);
    }
    return c;
}

// Preferred shapes, best first; the first whose LDS fits is used.  HARL_SCORE_CFG="wp,RPL,TW" or
// "ch,TW,ILP" puts a shape first (tuning sweeps).
ScoreCfg choose_cfg(const harl_ensemble *E) {
    std::vector<ScoreCfg> cands;
    if (const char *env = std::getenv("HARL_SCORE_CFG")) {
        char kind[3] = {0, 0, 0};
        int a = 0, b = 0;
        if (std::sscanf(env, "%2[a-z],%d,%d", kind, &a, &b) == 3) cands.push_back(make_cfg(E, kind[0] == 'w', a, b));
    }
    const int wp_pref[][2] = {{2, 12}, {1, 16}, {2, 8}, {2, 4}, {1, 8}, {1, 4}};
    for (auto &p : wp_pref) cands.push_back(make_cfg(E, true, p[0], p[1]));
    const int ch_pref[][2] = {{8, 1}, {4, 2}, {4, 1}, {2, 1}};
    for (auto &p : ch_pref) cands.push_back(make_cfg(E, false, p[0], p[1]));
    for (const ScoreCfg &c : cands)
        if (c.kern && c.lds <= (size_t)kLdsBytes) return c;
    return cands.back();  // nothing fits: the launch reports HARL_E_UNSUPPORTED
}

int device_cus(int device) {
    static int cached[64] = {0};
    if (device < 0 || device >= 64) return 256;
    if (!cached[device]) {
        int n = 0;
        if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, device) != hipSuccess || n <= 0) n = 256;
        cached[device] = n;
    }
    return cached[device];
}

// Work split of the persistent kernel: nb workgroups, each a slice of L (tile, tree) pairs; at
// least 2 trees per wave per slice so the feature staging stays amortised.
struct WpSplit {
    int64_t V, L, tiles;
    int nb;
};

WpSplit wp_split(const harl_ensemble *E, const ScoreCfg &c, int32_t n_rows) {
    WpSplit w{};
    const int64_t tiles = ceil_div(n_rows > 0 ? n_rows : 1, c.rows_per_tile);
    w.tiles = tiles;
    w.V = tiles * E->n_trees;
    const int per_cu = (int)(kLdsBytes / c.lds) > 0 ? (int)(kLdsBytes / c.lds) : 1;
    int64_t nb = (int64_t)device_cus(E->device) * per_cu;
    const int64_t min_l = 2LL * c.b;
    if (ceil_div(w.V, nb) < min_l) nb = ceil_div(w.V, min_l);
    w.L = ceil_div(w.V, nb);
    w.nb = (int)ceil_div(w.V, w.L);
    return w;
}

// Number of tree groups G of the grid kernel.  Each group's share of the ensemble should stay
// L2-resident (about 2 MB per XCD), and the work items (row tile x group) should fill whole waves
// of the machine: G minimises (rounds of co-resident workgroups) x (walk time + staging time per
// item).  HARL_SCORE_GROUPS overrides.
int choose_groups(const harl_ensemble *E, int32_t n_rows, const ScoreCfg &c) {
    const int64_t tiles = ceil_div(n_rows > 0 ? n_rows : 1, c.rows_per_tile);
    const int64_t bytes = (int64_t)E->n_trees * E->tree_stride;
    const int per_cu = c.lds > 0 ? (int)(kLdsBytes / c.lds) : 1;
    const int64_t slots = (int64_t)device_cus(E->device) * (per_cu > 0 ? per_cu : 1);
    const double walk = (double)E->n_trees * c.rows_per_tile * E->depth / 8.0;
    const double stage = (double)E->n_features * c.rows_per_tile * 4 / 32.0 + 2000.0;
    int best = 1;
    double best_cost = 1e300;
    for (int g = 1; g <= 8 && g <= E->n_trees; g *= 2) {
        if (g < 8 && bytes / g > (3 << 20)) continue;
        const double cost = (double)ceil_div(tiles * g, slots) * (walk / g + stage);
        if (cost < best_cost * 0.97) {
            best_cost = cost;
            best = g;
        }
    }
    if (const char *env = std::getenv("HARL_SCORE_GROUPS")) {
        const int o = std::atoi(env);
        if (o >= 1 && o <= E->n_trees && o <= 64) best = o;
    }
    return best;
}

// Floats of partial sums: sliced layout (tiles + workgroups) blocks of RT rows; grouped layout
// G rows-long slots.
size_t partial_floats(const harl_ensemble *E, const ScoreCfg &c, int32_t n_rows) {
    const int64_t ldp = round_up(n_rows > 0 ? n_rows : 1, 64);
    if (c.wp) {
        const WpSplit w = wp_split(E, c, n_rows);
        return (size_t)(w.tiles + w.nb) * c.rows_per_tile;
    }
    return (size_t)choose_groups(E, n_rows, c) * ldp;
}

}  // namespace

size_t score_round_ws_bytes(const harl_ensemble *E, int32_t n_rows) {
    const ScoreCfg c = choose_cfg(E);
    return partial_floats(E, c, n_rows) * sizeof(float) + 256;
}

int score_round_launch(const harl_ensemble *E, const float *X, int64_t ld, int32_t n_rows,
                       const int32_t *prog_ptr, int32_t n_prog, float *prog_score, float *stmt_score,
                       void *ws, size_t ws_bytes, hipStream_t stream) {
    const ScoreCfg c = choose_cfg(E);
    const int64_t ldp = round_up(n_rows > 0 ? n_rows : 1, 64);
    if (ws_bytes < partial_floats(E, c, n_rows) * sizeof(float))
        return fail(HARL_E_WORKSPACE, "harl_score_round: workspace too small");
    float *partial = static_cast<float *>(ws);
    const unsigned seg_grid = (unsigned)ceil_div(n_prog, 4);  // one wave per program
    const int rt_shift = c.rows_per_tile == 128 ? 7 : 6;
    if (n_rows == 0) {
        hipLaunchKernelGGL(k_segsum, dim3(seg_grid), dim3(256), 0, stream, partial, ldp, 6, 1, (int64_t)0, 0, prog_ptr,
                           n_prog, 0, E->base_score, prog_score, stmt_score);
        HARL_HIP_CHECK(hipGetLastError());
        return HARL_OK;
    }
    if (!c.kern || c.lds > (size_t)kLdsBytes)
        return fail(HARL_E_UNSUPPORTED, "harl_score_round: no kernel shape fits this ensemble in LDS");
    if (const int rc = ensure_dynamic_lds(c.kern, c.lds)) return rc;
    const int vec_ok = (ld % 4 == 0) && aligned(X, 16);
    const uint4 *trees = static_cast<const uint4 *>(E->d_trees);
    if (c.wp) {
        const WpSplit w = wp_split(E, c, n_rows);
        hipLaunchKernelGGL(reinterpret_cast<WpKernel>(const_cast<void *>(c.kern)), dim3((unsigned)w.nb), dim3(c.threads),
                           c.lds, stream, X, ld, n_rows, E->n_features, vec_ok, trees, E->n_trees, w.V, w.L, partial);
        HARL_HIP_CHECK(hipGetLastError());
        hipLaunchKernelGGL(k_segsum, dim3(seg_grid), dim3(256), 0, stream, partial, ldp, rt_shift, E->n_trees, w.L, 0,
                           prog_ptr, n_prog, n_rows, E->base_score, prog_score, stmt_score);
    } else {
        const int G = choose_groups(E, n_rows, c);
        const int tiles = (int)ceil_div(n_rows, c.rows_per_tile);
        const int tpg = (int)ceil_div(E->n_trees, G);
        const int groups = (int)ceil_div(E->n_trees, tpg);
        hipLaunchKernelGGL(reinterpret_cast<ChKernel>(const_cast<void *>(c.kern)), dim3((unsigned)tiles * groups),
                           dim3(c.threads), c.lds, stream, X, ld, n_rows, E->n_features, vec_ok, trees, E->n_trees,
                           tpg, groups, partial, ldp);
        HARL_HIP_CHECK(hipGetLastError());
        hipLaunchKernelGGL(k_segsum, dim3(seg_grid), dim3(256), 0, stream, partial, ldp, rt_shift, E->n_trees,
                           (int64_t)0, groups, prog_ptr, n_prog, n_rows, E->base_score, prog_score, stmt_score);
    }
    HARL_HIP_CHECK(hipGetLastError());
    return HARL_OK;
}

// ---------------------------------------------------------------------------------------------
// ensemble packing (host)
// ---------------------------------------------------------------------------------------------
int pack_ensemble(const harl_ensemble_desc *d, harl_ensemble **out, hipStream_t stream) {
    const int T = d->n_trees, F = d->n_features, N = d->n_nodes;
    if (T < 1 || N < 1 || F < 1) return fail(HARL_E_INVALID_ARG, "harl_ensemble_create: n_trees, n_nodes, n_features must be >= 1");
    if (F > kMaxFeatures)
        return fail(HARL_E_UNSUPPORTED, "harl_ensemble_create: n_features above " + std::to_string(kMaxFeatures));
    if (!d->root || !d->feature || !d->threshold || !d->left || !d->right || !d->default_left || !d->leaf_value)
        return fail(HARL_E_INVALID_ARG, "harl_ensemble_create: null node array");
    // depth of every tree, with range and cycle checks (iterative DFS, depth-bounded)
    int depth = 1;
    std::vector<std::pair<int32_t, int>> stack;
    for (int t = 0; t < T; ++t) {
        const int32_t r = d->root[t];
        if (r < 0 || r >= N) return fail(HARL_E_INVALID_ARG, "harl_ensemble_create: root out of range in tree " + std::to_string(t));
        stack.assign(1, {r, 0});
        int64_t visits = 0;
        while (!stack.empty()) {
            auto [n, dep] = stack.back();
            stack.pop_back();
            if (++visits > N) return fail(HARL_E_INVALID_ARG, "harl_ensemble_create: tree " + std::to_string(t) + " is cyclic");
            if (d->feature[n] < 0) {
                depth = dep > depth ? dep : depth;
                continue;
            }
            if (d->feature[n] >= F)
                return fail(HARL_E_INVALID_ARG, "harl_ensemble_create: split feature out of range at node " + std::to_string(n));
            if (dep + 1 > kMaxDepth)
                return fail(HARL_E_UNSUPPORTED, "harl_ensemble_create: tree " + std::to_string(t) + " deeper than 12 (or cyclic)");
            const int32_t L = d->left[n], R = d->right[n];
            if (L < 0 || L >= N || R < 0 || R >= N)
                return fail(HARL_E_INVALID_ARG, "harl_ensemble_create: child out of range at node " + std::to_string(n));
            stack.push_back({L, dep + 1});
            stack.push_back({R, dep + 1});
        }
    }
    const int D = depth;
    const int n_leaf = 1 << D;
    const int stride = tree_stride_bytes(D);
    std::vector<uint8_t> host((size_t)T * stride, 0);
    std::vector<int32_t> map(2 * (size_t)n_leaf);  // complete-tree slot (1-based) -> original node
    for (int t = 0; t < T; ++t) {
        uint8_t *tb = host.data() + (size_t)t * stride;
        uint32_t *words = reinterpret_cast<uint32_t *>(tb);
        float *leaves = reinterpret_cast<float *>(tb + (size_t)n_leaf * 8);
        map[1] = d->root[t];
        for (int s = 1; s < n_leaf; ++s) {
            const int32_t n = map[s];
            uint32_t word = 0;
            float thr = 0.f;
            if (d->feature[n] >= 0) {
                word = (uint32_t)d->feature[n] | (d->default_left[n] ? kNodeDefaultLeft : 0u);
                thr = d->threshold[n];
                if (std::isnan(thr)) thr = -INFINITY;   // no value is < NaN: everything present goes right
                map[2 * s] = d->left[n];
                map[2 * s + 1] = d->right[n];
            } else {                                    // early leaf: dummy split, both sides repeat it
                map[2 * s] = n;
                map[2 * s + 1] = n;
            }
            words[2 * s] = word;
            std::memcpy(&words[2 * s + 1], &thr, 4);
        }
        for (int j = 0; j < n_leaf; ++j) leaves[j] = d->leaf_value[map[n_leaf + j]];
    }
    harl_ensemble *E = new (std::nothrow) harl_ensemble{};
    if (!E) return fail(HARL_E_NOMEM, "harl_ensemble_create: host allocation failed");
    E->n_trees = T;
    E->n_features = F;
    E->depth = D;
    E->tree_stride = stride;
    E->base_score = d->base_score;
    if (hipGetDevice(&E->device) != hipSuccess) {
        delete E;
        return fail(HARL_E_HIP, "harl_ensemble_create: hipGetDevice failed");
    }
    if (hipMalloc(&E->d_trees, host.size()) != hipSuccess) {
        delete E;
        return fail(HARL_E_NOMEM, "harl_ensemble_create: device allocation failed");
    }
    hipError_t e = hipMemcpyAsync(E->d_trees, host.data(), host.size(), hipMemcpyHostToDevice, stream);
    if (e == hipSuccess) e = hipStreamSynchronize(stream);
    if (e != hipSuccess) {
        (void)hipFree(E->d_trees);
        delete E;
        return hip_fail(e, "harl_ensemble_create: upload");
    }
    *out = E;
    return HARL_OK;
}

}  // namespace harl
