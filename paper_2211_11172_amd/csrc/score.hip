// Cost-model scoring of one search round: C(S') for every candidate (Algorithm 1 of the HARL
// paper; the cost model is an XGBoost ensemble, Section 6.1 and Appendix A.2).  A candidate is a
// program of statements; each statement row has F fp32 features; the program score is the base
// score plus the sum over its statements of the ensemble's leaf sum.
//
// K1 k_tree_score: one workgroup owns a tile of 64*RW statement rows and one group of trees.
//   The row tile's features are staged once into LDS, feature-major ([F][64*RW] fp32: a lane's
//   feature gather hits bank = lane for every feature, so it is conflict-free whatever feature a
//   node asks for).  The group's trees stream through LDS in chunks of TW*ILP packed complete
//   trees (the next chunk is fetched into registers while the current one is walked).  Wave
//   (rw, tw) walks ILP trees of each chunk at once for its 64 rows (lane = row); each level issues
//   the current node's feature read together with the read of both its children (16 bytes) and
//   picks the child in registers, so a level costs one LDS round trip.  Row sums are accumulated
//   in fp64 and combined over the TW waves in a fixed order.
// K2 k_segsum: one thread per program sums its rows' per-group partials in a fixed order (fp64).
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

// Packed tree (1-based breadth-first): byte 8*i holds internal node i (i = 1 .. 2^D - 1; bytes 0..7
// are padding), so the two children of node i sit together, 16-byte aligned, at byte 16*i; the
// 2^D leaves follow at byte 8 * 2^D, and the two leaves below a last-level node i at
// 8 * 2^D + 8*i - 4 * 2^D.  One level of the walk therefore issues the feature read of the current
// node and the read of both its children at once, and selects the child in registers: one LDS
// round trip per level, the leaf pair coming with the last level.
template <bool NAN_AWARE>
__device__ __forceinline__ uint32_t go_right(float x, float thr, uint32_t word) {
    uint32_t right = x >= thr ? 1u : 0u;
    if (NAN_AWARE) right |= (x != x && !(word & kNodeDefaultLeft)) ? 1u : 0u;
    return right;
}

template <int D, int RW, int TW, int ILP, bool NAN_AWARE>
__device__ __forceinline__ void walk_chunk(const char *smem, uint32_t chunk_off, uint32_t stride,
                                           int tw, uint32_t lane_off, double &acc) {
    constexpr uint32_t RT4 = 64u * RW * 4u;
    constexpr uint32_t kLeafBase = 8u << D;
    uint32_t base[ILP], idx[ILP], word[ILP];
    float thr[ILP];
#pragma unroll
    for (int i = 0; i < ILP; ++i) {
        base[i] = chunk_off + (uint32_t)(tw * ILP + i) * stride;
        const uint2 root = *reinterpret_cast<const uint2 *>(smem + base[i] + 8u);
        word[i] = root.x;
        thr[i] = __uint_as_float(root.y);
        idx[i] = 1;
    }
#pragma unroll
    for (int lvl = 0; lvl + 1 < D; ++lvl) {
        float x[ILP];
        uint4 kids[ILP];
#pragma unroll
        for (int i = 0; i < ILP; ++i) {
            x[i] = *reinterpret_cast<const float *>(smem + __umul24(word[i], RT4) + lane_off);
            kids[i] = *reinterpret_cast<const uint4 *>(smem + base[i] + idx[i] * 16u);
        }
#pragma unroll
        for (int i = 0; i < ILP; ++i) {
            const uint32_t r = go_right<NAN_AWARE>(x[i], thr[i], word[i]);
            idx[i] = 2u * idx[i] + r;
            word[i] = r ? kids[i].z : kids[i].x;
            thr[i] = __uint_as_float(r ? kids[i].w : kids[i].y);
        }
    }
    float x[ILP];
    float2 lv[ILP];
#pragma unroll
    for (int i = 0; i < ILP; ++i) {
        x[i] = *reinterpret_cast<const float *>(smem + __umul24(word[i], RT4) + lane_off);
        lv[i] = *reinterpret_cast<const float2 *>(smem + base[i] + kLeafBase + idx[i] * 8u - (4u << D));
    }
#pragma unroll
    for (int i = 0; i < ILP; ++i) acc += (double)(go_right<NAN_AWARE>(x[i], thr[i], word[i]) ? lv[i].y : lv[i].x);
}

constexpr int tree_stride_bytes(int D) { return ((1 << D) * 12 + 15) / 16 * 16; }

template <int D, int RW, int TW, int ILP>
__global__ __launch_bounds__(64 * RW * TW) void k_tree_score(
    const float *__restrict__ X, int64_t ld, int n_rows, int F, int vec_ok, const uint4 *__restrict__ trees,
    int n_trees, int trees_per_group, int n_groups, float *__restrict__ partial, int64_t ldp) {
    constexpr int RT = 64 * RW;
    constexpr int NT = 64 * RW * TW;
    constexpr int C = TW * ILP;                       // trees per chunk
    constexpr int S16 = tree_stride_bytes(D) / 16;    // uint4 per packed tree
    constexpr int CH16 = C * S16;                     // uint4 per chunk
    constexpr int NPF = (CH16 + NT - 1) / NT;         // uint4 prefetched per thread
    extern __shared__ __align__(16) char smem[];

    const int g = blockIdx.x % n_groups;
    const int tile = blockIdx.x / n_groups;
    const int row0 = tile * RT;
    const int t_begin = g * trees_per_group;
    const int t_end = min(n_trees, t_begin + trees_per_group);
    const uint32_t chunk_off = (uint32_t)F * RT * 4u;

    // The next chunk of trees is fetched into registers while the current one is walked.
    uint4 pf[NPF];
    auto fetch = [&](int t0) {
        const int valid16 = min(C, t_end - t0) * S16;
        const uint4 *src = trees + (int64_t)t0 * S16;
#pragma unroll
        for (int j = 0; j < NPF; ++j) {
            const int i = threadIdx.x + j * NT;
            pf[j] = i < valid16 ? src[i] : make_uint4(0, 0, 0, 0);   // slots past the group: leaf 0.0
        }
    };
    auto commit = [&]() {
        uint4 *dst = reinterpret_cast<uint4 *>(smem + chunk_off);
#pragma unroll
        for (int j = 0; j < NPF; ++j) {
            const int i = threadIdx.x + j * NT;
            if (i < CH16) dst[i] = pf[j];
        }
    };
    if (t_begin < t_end) fetch(t_begin);

    // ---- stage the row tile's features (feature-major), 8 loads in flight per thread ----
    int has_nan = 0;
    {
        constexpr int V = RT / 4;  // float4 per feature row of the tile
        constexpr int B = 8;
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
    }
    if (t_begin < t_end) commit();
    has_nan = __syncthreads_or(has_nan);

    const int wid = threadIdx.x / kWave, lane = threadIdx.x % kWave;
    const int rw = wid / TW, tw = wid % TW;
    const uint32_t lane_off = (uint32_t)(rw * 64 + lane) * 4u;
    double acc = 0.0;

    for (int t0 = t_begin; t0 < t_end; t0 += C) {
        const bool more = t0 + C < t_end;
        if (more) fetch(t0 + C);
        if (has_nan)
            walk_chunk<D, RW, TW, ILP, true>(smem, chunk_off, (uint32_t)(S16 * 16), tw, lane_off, acc);
        else
            walk_chunk<D, RW, TW, ILP, false>(smem, chunk_off, (uint32_t)(S16 * 16), tw, lane_off, acc);
        __syncthreads();
        if (more) {
            commit();
            __syncthreads();
        }
    }

    // ---- combine the TW partial sums of each row in a fixed order ----
    double *red = reinterpret_cast<double *>(smem + chunk_off);
    red[tw * RT + rw * 64 + lane] = acc;
    __syncthreads();
    if (tw == 0) {
        double s = 0.0;
#pragma unroll
        for (int w = 0; w < TW; ++w) s += red[w * RT + rw * 64 + lane];
        const int r = row0 + rw * 64 + lane;
        if (r < n_rows) partial[(int64_t)g * ldp + r] = (float)s;
    }
}

__global__ __launch_bounds__(256) void k_segsum(const float *__restrict__ partial, int64_t ldp, int n_groups,
                                                const int32_t *__restrict__ prog_ptr, int n_prog, int n_rows,
                                                float base_score, float *__restrict__ prog_score,
                                                float *__restrict__ stmt_score) {
    const int p = blockIdx.x * blockDim.x + threadIdx.x;
    if (p >= n_prog) return;
    const int b = min(max(prog_ptr[p], 0), n_rows);
    const int e = min(max(prog_ptr[p + 1], b), n_rows);
    double acc = (double)base_score;
    constexpr int B = 8;  // rows loaded per batch, all loads issued before the first add
    for (int r0 = b; r0 < e; r0 += B) {
        double s[B];
#pragma unroll
        for (int j = 0; j < B; ++j) s[j] = 0.0;
        for (int gi = 0; gi < n_groups; ++gi) {
            float v[B];
#pragma unroll
            for (int j = 0; j < B; ++j) v[j] = r0 + j < e ? partial[(int64_t)gi * ldp + r0 + j] : 0.f;
#pragma unroll
            for (int j = 0; j < B; ++j) s[j] += (double)v[j];
        }
#pragma unroll
        for (int j = 0; j < B; ++j) {
            if (r0 + j < e) {
                if (stmt_score) stmt_score[r0 + j] = (float)s[j];
                acc += s[j];
            }
        }
    }
    prog_score[p] = (float)acc;
}

// ---------------------------------------------------------------------------------------------
// launch configuration
// ---------------------------------------------------------------------------------------------
struct ScoreCfg {
    int rw, tw, ilp;
};

using ScoreKernel = void (*)(const float *, int64_t, int, int, int, const uint4 *, int, int, int, float *, int64_t);

template <int D>
ScoreKernel pick_for_depth(ScoreCfg c) {
#define HARL_CFG(RW, TW, ILP) \
    if (c.rw == RW && c.tw == TW && c.ilp == ILP) return k_tree_score<D, RW, TW, ILP>;
    HARL_CFG(1, 4, 1)
    HARL_CFG(1, 4, 2)
    HARL_CFG(1, 2, 1)
    HARL_CFG(1, 2, 2)
    if constexpr (D == 6 || D == 8 || D == 10) {
        HARL_CFG(1, 4, 3)
        HARL_CFG(1, 4, 4)
        HARL_CFG(1, 8, 1)
        HARL_CFG(1, 8, 2)
        HARL_CFG(2, 4, 1)
        HARL_CFG(2, 4, 2)
        HARL_CFG(2, 2, 2)
        HARL_CFG(2, 2, 4)
        HARL_CFG(1, 16, 1)
        HARL_CFG(1, 16, 2)
        HARL_CFG(2, 8, 1)
    }
#undef HARL_CFG
    return nullptr;
}

ScoreKernel pick_kernel(int depth, ScoreCfg c) {
    switch (depth) {
        case 1: return pick_for_depth<1>(c);
        case 2: return pick_for_depth<2>(c);
        case 3: return pick_for_depth<3>(c);
        case 4: return pick_for_depth<4>(c);
        case 5: return pick_for_depth<5>(c);
        case 6: return pick_for_depth<6>(c);
        case 7: return pick_for_depth<7>(c);
        case 8: return pick_for_depth<8>(c);
        case 9: return pick_for_depth<9>(c);
        case 10: return pick_for_depth<10>(c);
        case 11: return pick_for_depth<11>(c);
        case 12: return pick_for_depth<12>(c);
        default: return nullptr;
    }
}

size_t lds_need(const harl_ensemble *E, ScoreCfg c) {
    const size_t rt = 64 * c.rw;
    const size_t feat = (size_t)E->n_features * rt * 4;
    const size_t chunk = (size_t)c.tw * c.ilp * E->tree_stride;
    const size_t red = (size_t)c.tw * rt * 8;
    return feat + (chunk > red ? chunk : red);
}

// Default shape per depth; HARL_SCORE_CFG="rw,tw,ilp" overrides it (tuning sweeps).  The first
// candidate whose feature tile and tree chunk fit in LDS is used.
ScoreCfg choose_cfg(const harl_ensemble *E) {
    ScoreCfg pref{1, 4, 2};
    if (E->depth <= 6) pref = ScoreCfg{1, 4, 4};
    else if (E->depth <= 8) pref = ScoreCfg{1, 4, 3};
    else if (E->depth <= 10) pref = ScoreCfg{1, 4, 1};
    else pref = ScoreCfg{1, 2, 1};
    if (const char *env = std::getenv("HARL_SCORE_CFG")) {
        ScoreCfg o{};
        if (std::sscanf(env, "%d,%d,%d", &o.rw, &o.tw, &o.ilp) == 3 && pick_kernel(E->depth, o)) pref = o;
    }
    const ScoreCfg cands[] = {pref, {1, 4, 2}, {1, 4, 1}, {1, 2, 2}, {1, 2, 1}};
    for (const ScoreCfg &c : cands)
        if (pick_kernel(E->depth, c) && lds_need(E, c) <= (size_t)kLdsBytes) return c;
    return pref;  // does not fit: the launch reports HARL_E_UNSUPPORTED
}

// Number of tree groups: the ensemble share per group should stay L2-resident (about 2 MB per
// XCD) and the grid should hold enough workgroups to fill 256 CUs.  HARL_SCORE_GROUPS overrides.
int choose_groups(const harl_ensemble *E, int32_t n_rows, ScoreCfg c) {
    const int64_t tiles = ceil_div(n_rows > 0 ? n_rows : 1, 64 * c.rw);
    const int64_t bytes = (int64_t)E->n_trees * E->tree_stride;
    int g = 1;
    while (g < 8 && g < E->n_trees && (bytes / g > (2 << 20) || tiles * g < 1024)) g *= 2;
    if (const char *env = std::getenv("HARL_SCORE_GROUPS")) {
        const int o = std::atoi(env);
        if (o >= 1 && o <= E->n_trees && o <= 64) g = o;
    }
    return g;
}

}  // namespace

size_t score_round_ws_bytes(const harl_ensemble *E, int32_t n_rows) {
    const ScoreCfg c = choose_cfg(E);
    const int g = choose_groups(E, n_rows, c);
    return (size_t)g * (size_t)round_up(n_rows > 0 ? n_rows : 1, 64) * sizeof(float) + 256;
}

int score_round_launch(const harl_ensemble *E, const float *X, int64_t ld, int32_t n_rows,
                       const int32_t *prog_ptr, int32_t n_prog, float *prog_score, float *stmt_score,
                       void *ws, size_t ws_bytes, hipStream_t stream) {
    const ScoreCfg c = choose_cfg(E);
    const int G = choose_groups(E, n_rows, c);
    const int64_t ldp = round_up(n_rows > 0 ? n_rows : 1, 64);
    if (ws_bytes < (size_t)G * ldp * sizeof(float))
        return fail(HARL_E_WORKSPACE, "harl_score_round: workspace too small");
    float *partial = static_cast<float *>(ws);
    if (n_rows > 0) {
        ScoreKernel kern = pick_kernel(E->depth, c);
        const size_t lds = lds_need(E, c);
        if (!kern || lds > (size_t)kLdsBytes)
            return fail(HARL_E_UNSUPPORTED, "harl_score_round: no kernel shape fits this ensemble in LDS");
        const int tiles = (int)ceil_div(n_rows, 64 * c.rw);
        const int tpg = (int)ceil_div(E->n_trees, G);
        const int groups = (int)ceil_div(E->n_trees, tpg);
        HARL_HIP_CHECK(hipFuncSetAttribute(reinterpret_cast<const void *>(kern),
                                           hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds));
        const int vec_ok = (ld % 4 == 0) && aligned(X, 16);
        hipLaunchKernelGGL(kern, dim3((unsigned)tiles * groups), dim3(64 * c.rw * c.tw), lds, stream, X, ld,
                           n_rows, E->n_features, vec_ok, static_cast<const uint4 *>(E->d_trees), E->n_trees, tpg,
                           groups, partial, ldp);
        HARL_HIP_CHECK(hipGetLastError());
        hipLaunchKernelGGL(k_segsum, dim3((unsigned)ceil_div(n_prog, 256)), dim3(256), 0, stream, partial, ldp,
                           groups, prog_ptr, n_prog, n_rows, E->base_score, prog_score, stmt_score);
    } else {
        hipLaunchKernelGGL(k_segsum, dim3((unsigned)ceil_div(n_prog, 256)), dim3(256), 0, stream, partial, ldp, 0,
                           prog_ptr, n_prog, 0, E->base_score, prog_score, stmt_score);
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
