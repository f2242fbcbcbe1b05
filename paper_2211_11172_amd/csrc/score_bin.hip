// Cost-model scoring on binned feature codes: the path harl_score_round takes for ensembles of 9 or
// 10 split levels, and of 8 on rounds of at least kB16MinRowsDepth8 statement rows, of up to 256
// features with at most 65,534 distinct thresholds per feature (Algorithm 1's cost model C(S'), an
// XGBoost ensemble: Section 6.1 and Appendix A.1).  Other rounds use the fp32 walk of score.hip,
// whose 3 KB depth-8 trees leave room for 16 waves per CU (at depth 10 its 12 KB trees leave room
// for 6); on small depth-8 rounds the binning pass costs more than the binned walk saves.
//
// A split sends x left iff x < threshold, so a node's decision depends only on where x falls among
// the thresholds its feature is split on.  With t_f[0] < ... < t_f[m_f - 1] the distinct thresholds
// of feature f over the whole ensemble, a present value gets the code
//     b(x) = #{ j : t_f[j] <= x }        (IEEE compares, so -0 and +0 are one value)
// and for a node splitting f at t_f[j]:  x < t_f[j]  <=>  b(x) <= j  <=>  b(x) < theta, theta = j + 1.
// A missing value (NaN) gets the code 0xFFFF.  Each node stores theta and U = 0xFFFF - theta when
// missing values go right, 0xFFFE - theta when they go left; a code c goes right iff
// (c - theta) mod 2^32 <= U.  This reproduces the fp32 comparison exactly, missing values included,
// with one subtraction and one compare per node visit.  A NaN threshold (every present value goes
// right) gets theta = 0.
//
// K0 k_bin16: one pass over the round's fp32 features [F][ld] writes the codes into the workspace:
//   per 256-row tile and feature, 128 dwords {code(row p), code(row p + 128)}.
// K1 k_tree_score_b16: persistent workgroups over slices of the (row tile, tree) space as the fp32
//   walk (XCD-aware slices, tree groups that stay L2-resident, per-wave tree slots streamed through
//   registers).  A tile holds 256 rows, 512 bytes per feature (84 KB for 164 features, the size of
//   a 128-row fp32 tile); each lane walks 4 rows of every tree: twice the row-tree chains per wave
//   of the fp32 walk, and half the tree bytes streamed per row.
//
// Tile in LDS: row group g (rows 64g .. 64g + 63 and 128 + 64g .. 191 + 64g) at byte 65536 g, its
// feature f at 65536 g + 256 f: dword l = {code(row 64g + l), code(row 128 + 64g + l)}.  The code of
// lane l's row 64j + l for feature f is then half j >> 1 of the dword at byte 65536 (j & 1) + 256 f
// + 4 l, which a walk reads whole (a decision takes the half by an SDWA select): the lane and row
// bits of the address never change, and a decision writes the child's feature straight into its
// second byte.  Lanes read distinct banks whatever features their nodes ask for.  Tree slots fill
// the LDS around the two row groups.
//
// Packed tree (D split levels, M = 2^D leaves, nodes numbered breadth-first from 1), 2M bytes: the
// 8-byte records of levels 0 .. D-3, record 0 = {feature(1), 0}, record i (1 <= i < M/4) =
// {theta(i) | U(i) << 16, feature(2i) | feature(2i+1) << 8}.  Its tail in global memory, 8M bytes
// per tree (L2-resident with the trees): the 16-byte records of level D-2, node i = M/4 + k's
// {theta(i) | U(i) << 16, feature(2i) | feature(2i+1) << 8, word(2i), word(2i+1)} at 16k (word(n)
// = theta(n) | U(n) << 16 of a last-level node n), then the leaves, node M/2 + k's at 4M + 8k and
// 4M + 8k + 4.  A level of a walk reads the current node's code and record together (one LDS round
// trip); the record carries both children's features, so the child's code is read with the child's
// record.  A depth-10 slot is 2 KB, and 16 waves fit beside the tile.  A chain loads its level D-2
// record from the tail at the end of a tree's walk and takes that level during the next tree's walk,
// after the root level, and the last level (whose word came with the record) after level 1; its leaf
// is added during the walk after that.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstring>
#include <limits>
#include <vector>

#include "internal.hpp"
#include "walk_b16.hpp"

namespace harl {
namespace {

using namespace b16;
constexpr int kLdsBytes = 160 * 1024;
constexpr int kPrefetchFeatures = 192;          // features per tile held in the register prefetch

// ---- K0: codes of every (row, feature) ----
// The order-preserving 32-bit key of a present value is its bit pattern with the sign bit set for
// +-values >= +0 and all bits inverted for negatives.  Per feature, a window of keys is cut into
// 4,094 buckets of 2^sh keys (sh >= 1): bucket b = clamp((key >> sh) - base, 0, 4095), so keys
// below the window fall in bucket 0 and keys above it in bucket 4095.  The window (and sh) is chosen
// when the ensemble is packed to cover the feature's thresholds, but for up to three outliers at
// either end, with the fewest thresholds in the fullest bucket.  lut[b] = number of thresholds in
// lower buckets, and every bucket holds fewer than 2^steps - 1 thresholds.  A value in bucket b has a
// code between lut[b] and lut[b] + 2^steps - 1: a branch-free binary search of `steps` probes,
// starting at lut[b], finds it.  Probes past the bucket land on larger thresholds (or on the table's
// NaN padding), which never compare <= x, so no bound check is needed; -0 and +0 compare equal, and
// the thresholds hold one zero (+0), which a -0 in the bucket below reaches in the same way (hence
// the one threshold of slack).
// Workgroup (feature f, range of tiles): stages lut and the thresholds of f in LDS (or searches
// them in global memory when they do not fit), then each thread codes two row quads at a time: rows
// 4q .. 4q + 3 and 128 + 4q .. 131 + 4q of a tile, read as two 16-byte loads when the feature rows
// are 16-byte aligned (VEC), written as one 16-byte store.  Rows at or past n_rows get code 0 (never
// summed).
constexpr int kBinThreads = 256;
constexpr int kLutBuckets = 4096;
constexpr int kLutStride = 4104;                  // u16 per feature's lut (4,097 used), 16-byte rows
constexpr int kBinLdsThresholds = 10240;          // 40 KB, padding included
constexpr int kBinQuads = 2;                      // row quads per thread and iteration
constexpr int kQuadsPerTile = kRT / 8;            // 32

__device__ __forceinline__ uint32_t order_key(float x) {
    const uint32_t u = __float_as_uint(x);
    return u ^ ((uint32_t)((int32_t)u >> 31) | 0x80000000u);
}

__device__ __forceinline__ int key_bucket(float x, int sh, uint32_t base) {
    const int b = (int)((order_key(x) >> sh) - base);
    return b < 0 ? 0 : (b > kLutBuckets - 1 ? kLutBuckets - 1 : b);
}

// Codes of N values at once: the probes of the N searches are independent and overlap.  With the
// probe count a compile-time STEPS and the thresholds in LDS, each search carries a pointer whose
// probe offsets are immediates of the LDS reads; otherwise (STEPS = 0) an index and `steps` probes.
typedef __attribute__((address_space(3))) const float lds_float;
template <int N, int STEPS>
__device__ __forceinline__ void codes_of(const float (&x)[N], uint32_t (&c)[N], const uint16_t *lut, const float *tf,
                                         int steps, int sh, uint32_t base) {
    if constexpr (STEPS > 0) {
        lds_float *const t0 = (lds_float *)tf;  // tf points into LDS on this path
        lds_float *p[N];
#pragma unroll
        for (int e = 0; e < N; ++e) p[e] = t0 + lut[key_bucket(x[e], sh, base)];
#pragma unroll
        for (int k = STEPS - 1; k >= 0; --k) {
            float t[N];
#pragma unroll
            for (int e = 0; e < N; ++e) t[e] = p[e][(1 << k) - 1];
            __builtin_amdgcn_sched_barrier(0);  // all N reads in flight before the first compare
#pragma unroll
            for (int e = 0; e < N; ++e)
                if (t[e] <= x[e]) p[e] += 1 << k;
        }
#pragma unroll
        for (int e = 0; e < N; ++e) c[e] = (uint32_t)(p[e] - t0);
    } else {
#pragma unroll
        for (int e = 0; e < N; ++e) c[e] = lut[key_bucket(x[e], sh, base)];
        for (int k = steps - 1; k >= 0; --k) {
            const uint32_t s = 1u << k;
#pragma unroll
            for (int e = 0; e < N; ++e)
                if (tf[c[e] + s - 1] <= x[e]) c[e] += s;
        }
    }
#pragma unroll
    for (int e = 0; e < N; ++e)
        if (x[e] != x[e]) c[e] = kMissing;
}

template <bool VEC, int STEPS>
__global__ __launch_bounds__(kBinThreads) void k_bin16(const float *__restrict__ X, int64_t ld, int n_rows,
                                                       const float *__restrict__ thr, const int32_t *__restrict__ t_off,
                                                       const int32_t *__restrict__ t_len,
                                                       const uint16_t *__restrict__ luts,
                                                       const int32_t *__restrict__ search_f, uint32_t *__restrict__ codes,
                                                       int64_t ldw, int tiles, int tiles_per_block, int blocks_per_f) {
    __shared__ float st[kBinLdsThresholds];
    __shared__ uint16_t sl[kLutStride];
    const int f = blockIdx.x / blocks_per_f;
    const int tile0 = (blockIdx.x % blocks_per_f) * tiles_per_block;
    const int tile1 = min(tiles, tile0 + tiles_per_block);
    if (tile0 >= tile1) return;  // whole workgroup
    const int len = t_len[f], steps = search_f[2 * f] & 0xFF, sh = search_f[2 * f] >> 8;
    const uint32_t base = (uint32_t)search_f[2 * f + 1];
    const float *__restrict__ tg = thr + t_off[f];
    const bool in_lds = len <= kBinLdsThresholds;
    {
        const uint4 *src = reinterpret_cast<const uint4 *>(luts + (int64_t)f * kLutStride);
        uint4 *dst = reinterpret_cast<uint4 *>(sl);
        for (int i = threadIdx.x; i < kLutStride / 8; i += kBinThreads) dst[i] = src[i];
        if (in_lds)
            for (int i = threadIdx.x; i < len; i += kBinThreads) st[i] = tg[i];
    }
    __syncthreads();
    const float *__restrict__ xf = X + (int64_t)f * ld;
    uint32_t *__restrict__ out = codes + (int64_t)f * ldw;
    constexpr int kPass = kBinQuads * kBinThreads;  // quads per pass: 16 tiles
    const int n_quads = (tile1 - tile0) * kQuadsPerTile;
    auto code = [&](const float (&x)[8 * kBinQuads], uint32_t (&c)[8 * kBinQuads]) {
        if (STEPS > 0 && in_lds && steps == STEPS)
            codes_of<8 * kBinQuads, STEPS>(x, c, sl, st, steps, sh, base);
        else if (in_lds)
            codes_of<8 * kBinQuads, 0>(x, c, sl, st, steps, sh, base);
        else
            codes_of<8 * kBinQuads, 0>(x, c, sl, tg, steps, sh, base);
    };
    // quad i of the range: rows 4q .. 4q + 3 and 128 + 4q .. 131 + 4q of tile tile0 + i / 32, whose codes
    // go to dwords 4q .. 4q + 3 of that tile
    auto quad_row = [&](int i) { return (tile0 + i / kQuadsPerTile) * kRT + 4 * (i % kQuadsPerTile); };
    auto store = [&](int r, const uint32_t *c) {
        *reinterpret_cast<uint4 *>(out + (int64_t)(r / kRT) * (kRT / 2) + r % kRT) =
            make_uint4(c[0] | c[4] << 16, c[1] | c[5] << 16, c[2] | c[6] << 16, c[3] | c[7] << 16);
    };
    // Passes over whole tiles of rows below n_rows need no bounds checks; their features are read one
    // pass ahead, so that the next pass's loads are in flight while this one is coded (every pass
    // issues the same loads and stores, the last one re-reading its own features, so the wait for the
    // features counts only the stores issued after them).
    const int full_tiles = min(tile1, n_rows / kRT) - tile0;
    const int n_full = VEC && full_tiles > 0 ? full_tiles * kQuadsPerTile / kPass : 0;
    if (n_full > 0) {
        auto load = [&](int pass, float (&x)[8 * kBinQuads]) {
#pragma unroll
            for (int j = 0; j < kBinQuads; ++j) {
                const int r = quad_row(pass * kPass + j * kBinThreads + threadIdx.x);
                const float4 a = *reinterpret_cast<const float4 *>(xf + r);
                const float4 b = *reinterpret_cast<const float4 *>(xf + r + kRT / 2);
                x[8 * j + 0] = a.x, x[8 * j + 1] = a.y, x[8 * j + 2] = a.z, x[8 * j + 3] = a.w;
                x[8 * j + 4] = b.x, x[8 * j + 5] = b.y, x[8 * j + 6] = b.z, x[8 * j + 7] = b.w;
            }
        };
        float xn[8 * kBinQuads];
        load(0, xn);
        for (int pass = 0; pass < n_full; ++pass) {
            float x[8 * kBinQuads];
#pragma unroll
            for (int e = 0; e < 8 * kBinQuads; ++e) x[e] = xn[e];
            load(min(pass + 1, n_full - 1), xn);
            uint32_t c[8 * kBinQuads];
            code(x, c);
#pragma unroll
            for (int j = 0; j < kBinQuads; ++j) store(quad_row(pass * kPass + j * kBinThreads + threadIdx.x), c + 8 * j);
        }
    }
    // the rest of the range (its last tiles, a partial last tile): bounds-checked, rows at or past
    // n_rows read as 0 and coded 0
    for (int i0 = n_full * kPass + threadIdx.x; i0 < n_quads; i0 += kPass) {
        float x[8 * kBinQuads];
        int row[kBinQuads];
#pragma unroll
        for (int j = 0; j < kBinQuads; ++j) {
            const int i = i0 + j * kBinThreads;
            const int r = i < n_quads ? quad_row(i) : -1;
            row[j] = r;
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const int rr = r + (e & 3) + (e >> 2) * (kRT / 2);
                const float v = xf[rr < 0 ? 0 : (rr < n_rows ? rr : n_rows - 1)];  // n_rows >= 1
                x[8 * j + e] = r >= 0 && rr < n_rows ? v : 0.f;
            }
        }
        uint32_t c[8 * kBinQuads];
        code(x, c);
#pragma unroll
        for (int j = 0; j < kBinQuads; ++j) {
            const int r = row[j];
            if (r < 0) continue;
#pragma unroll
            for (int e = 0; e < 8; ++e)
                if (r + (e & 3) + (e >> 2) * (kRT / 2) >= n_rows) c[8 * j + e] = 0u;
            store(r, c + 8 * j);
        }
    }
}

// ---- K1 ----
// Slices of the (tile, tree) space, XCD-aware: workgroup b runs on XCD b % 8, walks tree group
// (b % 8) % G and slice ((b % 8) / G) * (nb / 8) + b / 8 of that group; consecutive slices share
// their boundary tile and stage it at about the same time, on one XCD (even slices walk their tiles
// last to first, odd ones first to last).
__device__ __forceinline__ void block_slice(int b, int nb, int G, int &g, int &r) {
    const int x = b % 8, j = b / 8;  // nb is a multiple of 8
    g = x % G;
    r = (x / G) * (nb / 8) + j;
}
__host__ __device__ __forceinline__ int group_trees(int T, int G, int g) {
    const int tg = (T + G - 1) / G;
    return T - g * tg < tg ? T - g * tg : tg;
}
__host__ __device__ __forceinline__ int64_t group_slice_len(int64_t tiles, int tc, int nbg) {
    return (tiles * tc + nbg - 1) / nbg;
}

// A wave's tree: lane l moves uint4 j*64 + l (S16 uint4 per tree, PF per lane at most; EXACT: the
// tree is exactly PF * 64 uint4, and the loads need no guard).
template <int PF, bool EXACT>
__device__ __forceinline__ void tree_fetch(uint4 (&pf)[PF], const uint4 *__restrict__ src, int S16, int lane) {
#pragma unroll
    for (int j = 0; j < PF; ++j)
        if (EXACT || j * kWave + lane < S16) pf[j] = src[j * kWave + lane];
}
template <int PF, bool EXACT>
__device__ __forceinline__ void tree_commit(const uint4 (&pf)[PF], uint4 *dst, int S16, int lane, Head &h) {
#pragma unroll
    for (int j = 0; j < PF; ++j)
        if (EXACT || j * kWave + lane < S16) dst[j * kWave + lane] = pf[j];
    h.f = __builtin_amdgcn_readlane(pf[0].x, 0);
    h.w = __builtin_amdgcn_readlane(pf[0].z, 0);
    h.p = __builtin_amdgcn_readlane(pf[0].w, 0);
}

// Tile staging.  uint4 i of a tile is part i % 32 of feature i / 32 in the codes (global: feature
// f's 128 dwords of tile t at f * ldw + 128 t) and goes to LDS uint4 4096 g + 16 f + q, where
// (g, q) = (part / 16, part % 16): row group g, dwords 4q .. 4q + 3.  With NT a multiple of 32,
// thread t holds parts t % 32 of features t / 32 + j * NT / 32.
__device__ __forceinline__ int tile_lds_index(int i) {
    const int part = i % kTileU4;
    return (part / 16) * (int)(kGroupStride / 16) + (i / kTileU4) * 16 + part % 16;
}
// A code tile is read once per tree group and not again soon: a streaming (non-temporal) load, so
// that the code stream does not push the ensemble's node records out of the L2.
typedef unsigned u32x4_nt __attribute__((ext_vector_type(4)));
__device__ __forceinline__ uint4 load_stream(const uint4 *p) {
    const u32x4_nt v = __builtin_nontemporal_load(reinterpret_cast<const u32x4_nt *>(p));
    return make_uint4(v.x, v.y, v.z, v.w);
}
template <int NT, int NPX>
__device__ __forceinline__ void tile_fetch(uint4 (&xf)[NPX], const uint4 *__restrict__ codes, int64_t ldw4, int F,
                                           int tile) {
    const int total = F * kTileU4;
    const uint4 *p = codes + (int64_t)(threadIdx.x / kTileU4) * ldw4 + (int64_t)tile * kTileU4 + threadIdx.x % kTileU4;
    const int64_t step = (int64_t)(NT / kTileU4) * ldw4;
    // every element is assigned (a guarded assignment would leave xf to the stack)
#pragma unroll
    for (int j = 0; j < NPX; ++j) {
        xf[j] = (int)threadIdx.x + j * NT < total ? load_stream(p) : make_uint4(0, 0, 0, 0);
        p += step;
    }
}
template <int NT, int NPX>
__device__ __forceinline__ void tile_commit(const uint4 (&xf)[NPX], uint4 *tile_lds, int F) {
    const int total = F * kTileU4;
    uint4 *dst = tile_lds + tile_lds_index(threadIdx.x);
#pragma unroll
    for (int j = 0; j < NPX; ++j)
        if ((int)threadIdx.x + j * NT < total) dst[j * (NT / kTileU4) * 16] = xf[j];
}
// Direct staging (tiles too wide for the register prefetch), 4 loads in flight per thread.
template <int NT>
__device__ __forceinline__ void tile_stage(uint4 *tile_lds, const uint4 *__restrict__ codes, int64_t ldw4, int F,
                                           int tile) {
    const int total = F * kTileU4;
    for (int i0 = threadIdx.x; i0 < total; i0 += 4 * NT) {
        uint4 v[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int i = i0 + j * NT;
            v[j] = i < total ? load_stream(codes + (int64_t)(i / kTileU4) * ldw4 + (int64_t)tile * kTileU4 + (i % kTileU4))
                             : make_uint4(0, 0, 0, 0);
        }
#pragma unroll
        for (int j = 0; j < 4; ++j)
            if (i0 + j * NT < total) tile_lds[tile_lds_index(i0 + j * NT)] = v[j];
    }
}

template <int TW, int PF, bool EXACT>
__global__ __launch_bounds__(64 * TW) void k_tree_score_b16(const uint4 *__restrict__ codes, int64_t ldw4, int n_rows,
                                                           int F, const uint4 *__restrict__ trees_all, int S16, int D,
                                                           int T_all, int G, int tiles, float *__restrict__ partial_all,
                                                           const float *__restrict__ leaves_all) {
    constexpr int NT = 64 * TW;
    constexpr int NPX = (kPrefetchFeatures * kTileU4 + NT - 1) / NT;
    extern __shared__ __align__(16) char smem[];
    int g, s;
    block_slice(blockIdx.x, gridDim.x, G, g, s);
    const int nbg = gridDim.x / G;
    const int T = group_trees(T_all, G, g);
    if (T <= 0) return;  // whole workgroup
    const int64_t g_tree0 = (int64_t)g * ((T_all + G - 1) / G);
    const uint4 *__restrict__ trees = trees_all + g_tree0 * S16;
    const int M = 1 << D;
    const float *__restrict__ leaves = leaves_all + g_tree0 * (2 * M);  // tails
    const float *const zero = leaves_all + (int64_t)T_all * (2 * M);     // two 0s after them
    float *__restrict__ partial = partial_all + (int64_t)g * (tiles + nbg) * kRT;
    const int64_t V = (int64_t)tiles * T, L = group_slice_len(tiles, T, nbg);
    const int64_t v_begin = (int64_t)s * L;
    const int64_t v_end = v_begin + L < V ? v_begin + L : V;
    if (v_begin >= v_end) return;  // whole workgroup: no barrier is skipped by part of it
    const int tile_first = (int)(v_begin / T), tile_last = (int)((v_end - 1) / T);
    const int dir = (s & 1) ? 1 : -1;
    const int n_pieces = tile_last - tile_first + 1;
    auto piece_lo = [&](int i) { return (int)(v_begin - (int64_t)i * T > 0 ? v_begin - (int64_t)i * T : 0); };
    auto piece_hi = [&](int i) { return (int)(v_end - (int64_t)i * T < T ? v_end - (int64_t)i * T : T); };

    const int wid = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave), lane = threadIdx.x % kWave;
    const uint32_t sb = (uint32_t)S16 * 16u;
    const SlotPlan plan = slot_plan(F, TW, sb);
    const uint32_t slot_off = wid < plan.n_a ? plan.a0 + (uint32_t)wid * sb : plan.b0 + (uint32_t)(wid - plan.n_a) * sb;
    uint4 *const slot = reinterpret_cast<uint4 *>(smem + slot_off);
    unsigned int *const progress = reinterpret_cast<unsigned int *>(smem + plan.progress);
    if (threadIdx.x == 0) progress[0] = progress[1] = 0;

    // the dynamic LDS starts at address 0 (the kernel has no static LDS), so the code addresses
    // carry the row bits alone outside byte 1
    const uint32_t tb = lds_addr(smem) + slot_off;
    const SlotConsts sk = slot_consts(tb, (uint32_t)M);
    uint32_t xa[kRPL];
#pragma unroll
    for (int j = 0; j < kRPL; ++j) xa[j] = lds_addr(smem) + kGroupStride * (j & 1) + 4u * (uint32_t)lane;

    // EXACT: a slot (2M bytes) is exactly PF * 64 uint4 (host-checked); else (depth 8) fewer
    uint4 pf[PF];
#pragma unroll
    for (int j = 0; j < PF; ++j) pf[j] = make_uint4(0, 0, 0, 0);
    Head hd{0, 0, 0};
    float pend[kRPL];
#pragma unroll
    for (int r = 0; r < kRPL; ++r) pend[r] = 0.f;
    const bool x_regs = F <= kPrefetchFeatures;
    uint4 xf[NPX];
    uint4 *const tile_lds = reinterpret_cast<uint4 *>(smem);
    double *const red = reinterpret_cast<double *>(smem + plan.b0);

    int tile = dir > 0 ? tile_first : tile_last;
    int t1 = piece_hi(tile);
    int t = piece_lo(tile) + wid;
    if (t < t1) tree_fetch<PF, EXACT>(pf, trees + (int64_t)t * S16, S16, lane);   // overlaps the tile staging
    if (x_regs) {
        tile_fetch<NT, NPX>(xf, codes, ldw4, F, tile);
        tile_commit<NT, NPX>(xf, tile_lds, F);
        __syncthreads();
        if (n_pieces > 1) tile_fetch<NT, NPX>(xf, codes, ldw4, F, tile + dir);
    } else {
        tile_stage<NT>(tile_lds, codes, ldw4, F, tile);
        __syncthreads();
    }
    for (int piece = 0;; ++piece) {
        const int row0 = tile * kRT;
        if (threadIdx.x == 0) progress[(piece + 1) & 1] = 0;
        uint32_t my_done = 0;
        if (t < t1) tree_commit<PF, EXACT>(pf, slot, S16, lane, hd);
        if (t + TW < t1) tree_fetch<PF, EXACT>(pf, trees + (int64_t)(t + TW) * S16, S16, lane);
        const bool next = piece + 1 < n_pieces;
        const int ntile = tile + dir;
        // this wave's leaves of the piece per row: at most 16 summed in fp32 (acc), then added to
        // the fp64 row sum (acc64)
        float acc[kRPL];
        double acc64[kRPL];
#pragma unroll
        for (int r = 0; r < kRPL; ++r) acc[r] = 0.f, acc64[r] = 0.0;
        Deferred last;
        no_deferred(last, zero);
        for (; t < t1; t += TW) {
            walk(tb, D, sk, hd, xa, acc, leaves + (int64_t)t * (2 * M), pend, last);
            if (t + TW < t1) tree_commit<PF, EXACT>(pf, slot, S16, lane, hd);  // LDS operations of a wave run in order
            // unconditional, past the piece's last tree clamped to it: every pass issues the same
            // loads, so the wait for a pending leaf counts only what was issued after it (with the
            // fetch conditional, the compiler's count assumed no fetch and waited for this one)
            tree_fetch<PF, EXACT>(pf, trees + (int64_t)min(t + 2 * TW, t1 - 1) * S16, S16, lane);
            // fair progress, every second tree: a wave behind its workgroup's average takes the top
            // issue priority
            my_done += 1;
            if (!(my_done & 15)) {
#pragma unroll
                for (int r = 0; r < kRPL; ++r) acc64[r] += (double)acc[r], acc[r] = 0.f;
            }
            if (!(my_done & 1)) {
                uint32_t total = 0;
                if (lane == 0) total = atomicAdd(progress + (piece & 1), 2u) + 2u;
                total = __builtin_amdgcn_readfirstlane(total);
                if (my_done * TW < total)
                    __builtin_amdgcn_s_setprio(3);
                else
                    __builtin_amdgcn_s_setprio(0);
            }
        }
        __builtin_amdgcn_s_setprio(0);
        finish(last, xa, acc, pend);
        const int nt0 = next ? piece_lo(ntile) : 0, nt1 = next ? piece_hi(ntile) : 0;
        // the next piece's first tree, fetched unconditionally (clamped to a tree of the group; a wave
        // with no tree there never commits it), so that the wait for the last leaves counts the same
        // loads on every path: with the fetch conditional, the compiler's count waited for it too.
        // The leaves are added after B1, their loads in flight meanwhile.
        tree_fetch<PF, EXACT>(pf, trees + (int64_t)min(nt0 + wid, T - 1) * S16, S16, lane);
        __syncthreads();  // B1: every wave is done with the tile and its slot
#pragma unroll
        for (int r = 0; r < kRPL; ++r) {
            acc64[r] += (double)(acc[r] + pend[r]);
            pend[r] = 0.f;
            red[wid * kRT + r * 64 + lane] = acc64[r];
        }
        if (next && x_regs) {
            tile_commit<NT, NPX>(xf, tile_lds, F);
            if (piece + 2 < n_pieces) tile_fetch<NT, NPX>(xf, codes, ldw4, F, ntile + dir);
        }
        __syncthreads();  // B2: row sums (and the next tile) are in LDS
        float *__restrict__ out = partial + ((int64_t)tile + s) * kRT;
        for (int r = threadIdx.x; r < kRT; r += NT) {
            double sum = 0.0;
#pragma unroll
            for (int w = 0; w < TW; ++w) sum += red[w * kRT + r];
            if (row0 + r < n_rows) out[r] = (float)sum;
        }
        if (!next) break;
        __syncthreads();  // B3: the sums are read before the next trees overwrite the slots
        if (!x_regs) {
            tile_stage<NT>(tile_lds, codes, ldw4, F, ntile);
            __syncthreads();
        }
        tile = ntile;
        t1 = nt1;
        t = nt0 + wid;
    }
}

// ---------------------------------------------------------------------------------------------
// launch configuration
// ---------------------------------------------------------------------------------------------
using B16Kernel = void (*)(const uint4 *, int64_t, int, int, const uint4 *, int, int, int, int, int, float *,
                           const float *);

struct B16Shape {
    int tw, pf;
    bool exact;
    B16Kernel kern;
};
// Shapes, most waves first: the first whose tree prefetch is one tree per lane group (exactly, or
// half of it at depth 8) and whose slots fit beside the tile is used (depth 8: 512 B slots; depth 9:
// 1 KB, 1 uint4 per lane; depth 10: 2 KB, 2).
const B16Shape kShapes[] = {
    {16, 1, false, k_tree_score_b16<16, 1, false>}, {8, 1, false, k_tree_score_b16<8, 1, false>},
    {16, 1, true, k_tree_score_b16<16, 1, true>},   {8, 1, true, k_tree_score_b16<8, 1, true>},
    {4, 1, true, k_tree_score_b16<4, 1, true>},     {16, 2, true, k_tree_score_b16<16, 2, true>},
    {8, 2, true, k_tree_score_b16<8, 2, true>},     {4, 2, true, k_tree_score_b16<4, 2, true>},
};

size_t b16_lds(const harl_ensemble *E, int tw) { return slot_plan(E->n_features, tw, (uint32_t)E->b16_stride).lds; }

const B16Shape *b16_shape(const harl_ensemble *E) {
    const int s16 = E->b16_stride / 16;
    for (const B16Shape &sh : kShapes)
        if ((sh.exact ? sh.pf * kWave == s16 : 2 * s16 == sh.pf * kWave) && b16_lds(E, sh.tw) <= (size_t)kLdsBytes)
            return &sh;
    return nullptr;
}

int device_cus_b16(int device) {
    static int cached[64] = {0};
    if (device < 0 || device >= 64) return 256;
    if (!cached[device]) {
        int n = 0;
        if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, device) != hipSuccess || n <= 0) n = 256;
        cached[device] = n;
    }
    return cached[device];
}

struct B16Split {
    int64_t tiles;
    int nb, G;
};

B16Split b16_split(const harl_ensemble *E, const B16Shape &sh, int32_t n_rows) {
    B16Split w{};
    w.tiles = ceil_div(n_rows > 0 ? n_rows : 1, kRT);
    w.G = E->tree_groups_b16;
    int64_t nb = device_cus_b16(E->device);  // one workgroup per CU (the tile and slots fill the LDS)
    const int64_t min_l = 2LL * sh.tw;        // at least 2 trees per wave per slice
    const int64_t vg = w.tiles * ceil_div(E->n_trees, w.G);
    if (ceil_div(vg, nb / w.G > 0 ? nb / w.G : 1) < min_l) nb = ceil_div(vg, min_l) * w.G;
    w.nb = (int)round_up(nb < 8 ? 8 : nb, 8);
    return w;
}

int bin_tiles_per_block(int64_t tiles) { return tiles >= 128 ? 128 : (int)tiles; }

}  // namespace

// Workspace: the codes ([F][tiles * 128] dwords, 256-byte aligned) followed by the partial sums.
size_t score_b16_ws_bytes(const harl_ensemble *E, int32_t n_rows) {
    const B16Shape *sh = b16_shape(E);
    if (!sh) return 0;
    const B16Split w = b16_split(E, *sh, n_rows);
    const size_t codes = (size_t)E->n_features * (size_t)w.tiles * kRowBytes;
    const size_t partial = (size_t)w.G * (size_t)(w.tiles + w.nb / w.G) * kRT * sizeof(float);
    return round_up((int64_t)codes, 256) + partial + 256;
}

bool score_b16_packed(const harl_ensemble *E) { return E->d_trees_b16 != nullptr && b16_shape(E) != nullptr; }
bool score_b16_usable(const harl_ensemble *E, int32_t n_rows) { return score_b16_packed(E) && n_rows >= E->b16_min_rows; }

int score_b16_launch(const harl_ensemble *E, const float *X, int64_t ld, int32_t n_rows, float **partial_out,
                     int *groups_out, int *tiles_out, int *nbg_out, void *ws, size_t ws_bytes, hipStream_t stream) {
    const B16Shape *sh = b16_shape(E);
    if (!sh) return fail(HARL_E_UNSUPPORTED, "harl_score_round: no binned kernel shape fits this ensemble");
    const B16Split w = b16_split(E, *sh, n_rows);
    if (ws_bytes < score_b16_ws_bytes(E, n_rows)) return fail(HARL_E_WORKSPACE, "harl_score_round: workspace too small");
    const size_t codes_bytes = round_up((int64_t)E->n_features * w.tiles * kRowBytes, 256);
    uint32_t *codes = static_cast<uint32_t *>(ws);
    float *partial = reinterpret_cast<float *>(static_cast<char *>(ws) + codes_bytes);
    const int64_t ldw = w.tiles * (kRT / 2);
    const int tpb = bin_tiles_per_block(w.tiles);
    const int bpf = (int)ceil_div(w.tiles, tpb);
    // 16-byte feature loads when every feature row starts on a 16-byte boundary; probe offsets as
    // immediates for the workgroups of features searched with the ensemble's most common probe count
    const bool vec = (reinterpret_cast<uintptr_t>(X) % 16) == 0 && ld % 4 == 0;
    using BinKernel = void (*)(const float *, int64_t, int, const float *, const int32_t *, const int32_t *,
                               const uint16_t *, const int32_t *, uint32_t *, int64_t, int, int, int);
    static const BinKernel kBin[2][6] = {
        {k_bin16<false, 0>, k_bin16<false, 1>, k_bin16<false, 2>, k_bin16<false, 3>, k_bin16<false, 4>, k_bin16<false, 5>},
        {k_bin16<true, 0>, k_bin16<true, 1>, k_bin16<true, 2>, k_bin16<true, 3>, k_bin16<true, 4>, k_bin16<true, 5>}};
    const int ms = E->b16_common_steps >= 1 && E->b16_common_steps <= 5 ? E->b16_common_steps : 0;
    hipLaunchKernelGGL(kBin[vec ? 1 : 0][ms], dim3((unsigned)(E->n_features * bpf)), dim3(kBinThreads), 0, stream, X,
                       ld, n_rows, E->d_thr_b16, E->d_thr_off_b16, E->d_thr_len_b16, E->d_lut_b16, E->d_search_b16,
                       codes, ldw, (int)w.tiles, tpb, bpf);
    HARL_HIP_CHECK(hipGetLastError());
    const size_t lds = b16_lds(E, sh->tw);
    if (const int rc = ensure_dynamic_lds(reinterpret_cast<const void *>(sh->kern), lds)) return rc;
    hipLaunchKernelGGL(sh->kern, dim3((unsigned)w.nb), dim3(64 * sh->tw), lds, stream,
                       reinterpret_cast<const uint4 *>(codes), ldw / 4, n_rows, E->n_features,
                       static_cast<const uint4 *>(E->d_trees_b16), E->b16_stride / 16, E->depth, E->n_trees, w.G,
                       (int)w.tiles, partial, E->d_leaves_b16);
    HARL_HIP_CHECK(hipGetLastError());
    *partial_out = partial;
    *groups_out = w.G;
    *tiles_out = (int)w.tiles;
    *nbg_out = w.nb / w.G;
    return HARL_OK;
}

// ---------------------------------------------------------------------------------------------
// packing (host): threshold tables and the binned tree format, from the complete-tree form
// ---------------------------------------------------------------------------------------------
// `feat`, `thr`, `dleft` per complete-tree slot 1 .. M-1 of every tree (T x M, slot 0 unused;
// feature -1 marks a dummy split below an early leaf), `leaf` per leaf slot (T x M).  Returns
// HARL_OK with E's binned fields set, or HARL_OK with them left empty when the ensemble does not
// qualify (the fp32 path is then used).
int pack_b16(harl_ensemble *E, const std::vector<int32_t> &feat, const std::vector<float> &thr,
             const std::vector<uint8_t> &dleft, const std::vector<float> &leaf, hipStream_t stream) {
    const int T = E->n_trees, F = E->n_features, D = E->depth;
    if (F > 256 || D < kMinB16Depth || D > kMaxB16Depth) return HARL_OK;
    const int M = 1 << D;
    // distinct thresholds per feature (NaN thresholds need none: theta = 0), with -0 stored as +0
    std::vector<std::vector<float>> tab(F);
    for (int t = 0; t < T; ++t)
        for (int s = 1; s < M; ++s) {
            const int32_t f = feat[(size_t)t * M + s];
            const float v = thr[(size_t)t * M + s];
            if (f >= 0 && !std::isnan(v)) tab[f].push_back(v == 0.f ? 0.f : v);
        }
    auto key_of = [](float v) {
        uint32_t u;
        std::memcpy(&u, &v, 4);
        return u ^ ((uint32_t)((int32_t)u >> 31) | 0x80000000u);
    };
    // per feature: the sorted thresholds padded with 2^steps NaNs, the bucket window and table, and
    // the probe count
    std::vector<int32_t> off(F), len(F), search(2 * (size_t)F);
    std::vector<uint16_t> lut((size_t)F * kLutStride, 0);
    std::vector<float> flat;
    std::vector<int32_t> per(kLutBuckets);
    for (int f = 0; f < F; ++f) {
        auto &v = tab[f];
        std::sort(v.begin(), v.end());
        v.erase(std::unique(v.begin(), v.end()), v.end());
        if (v.size() > 65534) return HARL_OK;
        const int n = (int)v.size();
        std::vector<uint32_t> k(n);
        for (int i = 0; i < n; ++i) k[i] = key_of(v[i]);
        auto bucket = [](uint32_t key, int sh, uint32_t base) {
            const int b = (int)((key >> sh) - base);
            return b < 0 ? 0 : (b > kLutBuckets - 1 ? kLutBuckets - 1 : b);
        };
        // window [k[lo], k[n - 1 - hi]] in buckets 1 .. 4094; the fewest probes, then the fewest outliers
        int best_steps = 99, best_sh = 1;
        uint32_t best_base = 0;
        for (int drop = 0; drop <= 6; ++drop)
            for (int lo = 0; lo <= drop && lo <= 3; ++lo) {
                const int hi = drop - lo;
                if (hi > 3 || lo + hi >= n) continue;
                const uint32_t klo = k[lo], khi = k[n - 1 - hi];
                int sh = 1;
                while (sh < 31 && (khi >> sh) - (klo >> sh) > (uint32_t)(kLutBuckets - 3)) ++sh;
                const uint32_t base = (klo >> sh) - 1u;
                std::fill(per.begin(), per.end(), 0);
                int max_b = 0;
                for (int i = 0; i < n; ++i) max_b = std::max(max_b, ++per[bucket(k[i], sh, base)]);
                int st = 0;
                while ((1 << st) < max_b + 2) ++st;  // a -0 in the bucket below +0 may count one more
                if (st < best_steps) best_steps = st, best_sh = sh, best_base = base;
            }
        if (n == 0) best_steps = 1, best_sh = 1, best_base = 0;
        std::fill(per.begin(), per.end(), 0);
        for (int i = 0; i < n; ++i) ++per[bucket(k[i], best_sh, best_base)];
        uint16_t *lf = lut.data() + (size_t)f * kLutStride;
        int run = 0;
        for (int b = 0; b < kLutBuckets; ++b) {
            lf[b] = (uint16_t)run;
            run += per[b];
        }
        lf[kLutBuckets] = (uint16_t)run;
        off[f] = (int32_t)flat.size();
        flat.insert(flat.end(), v.begin(), v.end());
        flat.insert(flat.end(), (size_t)1 << best_steps, std::numeric_limits<float>::quiet_NaN());
        len[f] = (int32_t)(flat.size() - off[f]);
        search[2 * f] = best_steps | best_sh << 8;
        search[2 * f + 1] = (int32_t)best_base;
    }
    int common_steps = 0;
    {
        int count[17] = {0};
        for (int f = 0; f < F; ++f) ++count[std::min(search[2 * f] & 0xFF, 16)];
        for (int st = 1; st <= 16; ++st)
            if (count[st] > count[common_steps]) common_steps = st;
    }
    auto word = [&](int32_t f, float v, uint8_t dl) -> uint32_t {
        uint32_t theta = 0;  // dummy split (f < 0) or NaN threshold: every present value goes right
        if (f >= 0 && !std::isnan(v)) {
            const auto &tv = tab[f];
            theta = (uint32_t)(std::lower_bound(tv.begin(), tv.end(), v == 0.f ? 0.f : v) - tv.begin()) + 1u;
        }
        const uint32_t U = (f >= 0 && dl ? 0xFFFEu : 0xFFFFu) - theta;
        return theta | U << 16;
    };
    const int stride = 2 * M;  // the slot: records of levels 0 .. D-3
    std::vector<uint8_t> host((size_t)T * stride, 0);
    std::vector<uint32_t> tails((size_t)T * (2 * M) + 2, 0u);  // level D-2 records, leaves; then two 0s
    auto put = [](uint8_t *dst, uint32_t w) { std::memcpy(dst, &w, 4); };
    for (int t = 0; t < T; ++t) {
        uint8_t *tb = host.data() + (size_t)t * stride;
        uint32_t *tail = tails.data() + (size_t)t * (2 * M);
        const int32_t *ft = feat.data() + (size_t)t * M;
        const float *th = thr.data() + (size_t)t * M;
        const uint8_t *dl = dleft.data() + (size_t)t * M;
        const float *lf = leaf.data() + (size_t)t * M;
        auto fcode = [&](int s) { return (uint32_t)(ft[s] >= 0 ? ft[s] : 0); };
        put(tb, fcode(1));
        for (int s = 1; s < M / 4; ++s) {
            put(tb + 8 * s, word(ft[s], th[s], dl[s]));
            put(tb + 8 * s + 4, fcode(2 * s) | fcode(2 * s + 1) << 8);
        }
        for (int s = M / 4; s < M / 2; ++s) {
            uint32_t *r = tail + 4 * (s - M / 4);
            r[0] = word(ft[s], th[s], dl[s]);
            r[1] = fcode(2 * s) | fcode(2 * s + 1) << 8;
            r[2] = word(ft[2 * s], th[2 * s], dl[2 * s]);
            r[3] = word(ft[2 * s + 1], th[2 * s + 1], dl[2 * s + 1]);
        }
        for (int s = M / 2; s < M; ++s) {
            const int k = s - M / 2;
            std::memcpy(tail + M + 2 * k, lf + (2 * s - M), 4);
            std::memcpy(tail + M + 2 * k + 1, lf + (2 * s + 1 - M), 4);
        }
    }
    // tree groups: the fewest (a power of 2 up to 8) whose share of the records a tile walk reads
    // (the slots and the level D-2 records, 6M bytes per tree) fits in about 4.5 MB, a little over an
    // XCD's 4 MB L2
    int G = 1;
    while (G < 8 && 2 * G <= T && (int64_t)T * 6 * M / G > (9 << 19)) G *= 2;
    if (E->tree_groups_override > 0 && E->tree_groups_override <= T) G = E->tree_groups_override;
    void *d_trees = nullptr, *d_thr = nullptr, *d_off = nullptr, *d_len = nullptr, *d_search = nullptr, *d_lut = nullptr,
         *d_gl = nullptr;
    auto cleanup = [&]() {
        for (void *p : {d_trees, d_thr, d_off, d_len, d_search, d_lut, d_gl})
            if (p) (void)hipFree(p);
    };
    if (hipMalloc(&d_trees, host.size()) != hipSuccess || hipMalloc(&d_thr, flat.size() * 4) != hipSuccess ||
        hipMalloc(&d_off, (size_t)F * 4) != hipSuccess || hipMalloc(&d_len, (size_t)F * 4) != hipSuccess ||
        hipMalloc(&d_search, search.size() * 4) != hipSuccess || hipMalloc(&d_lut, lut.size() * 2) != hipSuccess ||
        hipMalloc(&d_gl, tails.size() * 4) != hipSuccess) {
        cleanup();
        return fail(HARL_E_NOMEM, "harl_ensemble_create: device allocation failed");
    }
    hipError_t e = hipMemcpyAsync(d_trees, host.data(), host.size(), hipMemcpyHostToDevice, stream);
    if (e == hipSuccess) e = hipMemcpyAsync(d_thr, flat.data(), flat.size() * 4, hipMemcpyHostToDevice, stream);
    if (e == hipSuccess) e = hipMemcpyAsync(d_off, off.data(), (size_t)F * 4, hipMemcpyHostToDevice, stream);
    if (e == hipSuccess) e = hipMemcpyAsync(d_len, len.data(), (size_t)F * 4, hipMemcpyHostToDevice, stream);
    if (e == hipSuccess) e = hipMemcpyAsync(d_search, search.data(), search.size() * 4, hipMemcpyHostToDevice, stream);
    if (e == hipSuccess) e = hipMemcpyAsync(d_lut, lut.data(), lut.size() * 2, hipMemcpyHostToDevice, stream);
    if (e == hipSuccess) e = hipMemcpyAsync(d_gl, tails.data(), tails.size() * 4, hipMemcpyHostToDevice, stream);
    if (e == hipSuccess) e = hipStreamSynchronize(stream);
    if (e != hipSuccess) {
        cleanup();
        return hip_fail(e, "harl_ensemble_create: upload");
    }
    E->d_trees_b16 = d_trees;
    E->d_thr_b16 = static_cast<float *>(d_thr);
    E->d_thr_off_b16 = static_cast<int32_t *>(d_off);
    E->d_thr_len_b16 = static_cast<int32_t *>(d_len);
    E->d_search_b16 = static_cast<int32_t *>(d_search);
    E->d_lut_b16 = static_cast<uint16_t *>(d_lut);
    E->d_leaves_b16 = static_cast<float *>(d_gl);
    E->b16_stride = stride;
    E->tree_groups_b16 = G;
    E->b16_common_steps = common_steps;
    E->b16_min_rows = E->b16_min_rows_override >= 0 ? E->b16_min_rows_override : (D <= 8 ? kB16MinRowsDepth8 : 0);
    return HARL_OK;
}

void free_b16(harl_ensemble *E) {
    for (void *p : {E->d_trees_b16, (void *)E->d_thr_b16, (void *)E->d_thr_off_b16, (void *)E->d_thr_len_b16,
                    (void *)E->d_search_b16, (void *)E->d_lut_b16, (void *)E->d_leaves_b16})
        if (p) (void)hipFree(p);
    E->d_trees_b16 = nullptr;
    E->d_leaves_b16 = nullptr;
    E->d_thr_b16 = nullptr;
    E->d_thr_off_b16 = E->d_thr_len_b16 = E->d_search_b16 = nullptr;
    E->d_lut_b16 = nullptr;
}

}  // namespace harl
