// Cost-model scoring of one search round: C(S') for every candidate (Algorithm 1 of the HARL
// paper; the cost model is an XGBoost ensemble, Section 6.1 and Appendix A.1).  A candidate is a
// program of statements; each statement row has F fp32 features; the program score is the base
// score plus the sum over its statements of the ensemble's leaf sum.
//
// K1 tree traversal.  A workgroup owns a tile of statement rows and one group of trees.  The
//   tile's features are staged once into LDS, feature-major ([F][rows] fp32, so a lane's gather
//   of any feature of its own row hits bank = lane: conflict-free whatever feature a node asks
//   for).  Lane = row.  Each level of a walk issues the current node's feature read together with
//   the read of the node's record (threshold and both children's feature codes), so a level costs
//   one LDS round trip; the last level's record carries both leaves.  Row sums are accumulated in
//   fp64 and combined over the waves in a fixed order.  Two variants:
//   k_tree_score_wp (depth <= 10): every wave streams its own trees (tree t + k*TW) through
//     private LDS slots, NTW trees walked at once, the next ones fetched into registers while the
//     current ones are walked -- so waves never wait on each other between the feature staging
//     and the final reduction.  Each lane walks RPL rows per tree (ILP across rows and trees; the
//     staged tree serves 64*RPL rows).
//   k_tree_score_ch (deeper trees, whose 2^depth-node trees are too big for per-wave slots): the
//     workgroup stages chunks of TW*ILP trees shared by all waves, the next chunk fetched into
//     registers during the walk of the current one.
// K2 k_segsum: a workgroup owns consecutive programs; every thread forms its rows' sums from their
//     slice partials, and one thread per program adds its rows in row order (fp64, fixed order).
// Ensembles of 9 or 10 split levels (at most 256 features, 65,534 distinct thresholds per feature)
// are scored on 16-bit bin codes instead (score_bin.hip); K2 then sums that path's partials.
//
// Grid mapping is XCD-aware: workgroup b takes tree group b % G and row tile b / G; workgroups
// are dealt to the 8 XCDs round-robin, so with G in {2,4,8} every XCD's L2 only ever holds its
// own share of the ensemble.
#include <hip/hip_runtime.h>

#include <algorithm>

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
constexpr int kMaxWpDepth = 10;  // deeper trees (up to 48 KB each) use the shared-chunk kernel
constexpr int kRegTileFeatures = 192;  // features per row of a register-prefetched tile

// Packed tree of D split levels (M = 2^D leaves), nodes numbered breadth-first from 1:
//   bytes 0..7      record 0: {0, code(1)} -- the root's feature code
//   byte 8*i        record i, 1 <= i < M/2 (levels 0 .. D-2): {threshold(i), code(2i) | code(2i+1) << 16}
//   byte LL+16*j    last-level node i = M/2 + j: {threshold(i), leaf(2i - M), leaf(2i + 1 - M), 0}
// with LL = max(4M, 16) and code(n) = feature(n) | 0x8000 when missing values go left at n.  A
// level of a walk reads the feature value of the current node and the current node's record
// (threshold + both children's codes, 8 bytes) -- both addresses are known when the level starts,
// so a level is one LDS round trip of 12 bytes -- and the last level reads its threshold and both
// leaves in one 16-byte record.  The first 16 bytes {0, code(1), threshold(1), codes(2, 3)} are
// the same for every row and are taken as wave-uniform values.
constexpr uint32_t tree_ll_bytes(int D) { return (4u << D) > 16u ? (4u << D) : 16u; }
constexpr int tree_stride_bytes(int D) { return (int)((tree_ll_bytes(D) + (8u << D) + 15u) / 16u * 16u); }
constexpr uint32_t kCodeDefaultLeft = 0x8000u;
constexpr uint32_t kCodeFeature = 0x7FFFu;
// Up to this many features a code's feature fits its low byte, so a child's feature is selected
// with one byte-select instruction; wider ensembles select the 16-bit code and mask the flag.
constexpr int kNarrowFeatures = 256;

// Wave-uniform head of a packed tree (its bytes 4..15): root code, root threshold, codes of 2 and 3.
struct TreeHead {
    uint32_t code, thr, pair;
};

// Per-slot address constants of the walk (VGPR copies of wave-uniform values, so that one
// v_cndmask can pick between two of them).  With a = the LDS address of the current record:
//   inner level:           next record  = 2a + (go right ? r : l),            l = -tb,  r = 8 - tb
//   into the last level:   next record  = 4a + (go right ? r_last : l_last),   l_last = LL - 8M - 3tb
//   from the root:         next record  = go right ? r0 : l0 (absolute)
struct WalkConst {
    uint32_t l, r, l_last, r_last, l0, r0;
};

// An opaque VGPR copy of a wave-uniform value.
__device__ __forceinline__ uint32_t in_vgpr(uint32_t v) {
    asm("" : "+v"(v));
    return v;
}

template <int D>
__device__ __forceinline__ WalkConst walk_const(uint32_t tb) {
    constexpr uint32_t M = 1u << D, LL = tree_ll_bytes(D);
    WalkConst w;
    w.l = in_vgpr(0u - tb);
    w.r = in_vgpr(8u - tb);
    w.l_last = in_vgpr(LL - 8u * M - 3u * tb);
    w.r_last = in_vgpr(LL - 8u * M - 3u * tb + 16u);
    w.l0 = in_vgpr(D > 2 ? tb + 16u : tb + LL);
    w.r0 = in_vgpr(D > 2 ? tb + 24u : tb + LL + 16u);
    return w;
}

// LDS accesses by absolute LDS byte address (the walk carries addresses as plain integers).
typedef __attribute__((address_space(3))) char lds_char;
__device__ __forceinline__ uint32_t lds_addr(const char *p) { return (uint32_t)(uintptr_t)(const lds_char *)p; }
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
template <class T>
__device__ __forceinline__ T lds_ld(uint32_t a);
template <>
__device__ __forceinline__ float lds_ld<float>(uint32_t a) {
    return *(const __attribute__((address_space(3))) float *)(uintptr_t)a;
}
template <>
__device__ __forceinline__ uint2 lds_ld<uint2>(uint32_t a) {
    const u32x2 v = *(const __attribute__((address_space(3))) u32x2 *)(uintptr_t)a;
    return make_uint2(v.x, v.y);
}
template <>
__device__ __forceinline__ uint4 lds_ld<uint4>(uint32_t a) {
    const u32x4 v = *(const __attribute__((address_space(3))) u32x4 *)(uintptr_t)a;
    return make_uint4(v.x, v.y, v.z, v.w);
}

// One decision of a walk.  Given this lane's feature value x at the current node, the node's
// threshold and the packed codes `pair` of its children: the child's feature index `feat`, the
// child's 16-bit code moved to the upper half of `fw` (its missing-goes-left flag is then the sign
// bit; NaN-aware walk only) and `sel` = go right ? r : l.  A node sends x left iff x < threshold,
// or x is missing (NaN) and the node's own flag (the sign of `fw_cur`) is set.  The children's
// codes are picked with SDWA byte/word selects: one instruction instead of a shift, a mask and a
// select (the compare writes VCC, which the selects read; two wait states separate a VALU write
// of VCC from a VALU read of it as a mask).
template <bool NAN_AWARE, bool NARROW>
__device__ __forceinline__ void decide(float x, uint32_t thr, uint32_t pair, int32_t fw_cur, uint32_t l, uint32_t r,
                                       uint32_t &feat, int32_t &fw, uint32_t &sel) {
    if constexpr (!NAN_AWARE) {
        if constexpr (NARROW) {
            asm("v_cmp_ge_f32 vcc, %2, %3\n\t"
                "s_nop 1\n\t"
                "v_cndmask_b32_sdwa %0, %4, %4, vcc dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_0 src1_sel:BYTE_2\n\t"
                "v_cndmask_b32 %1, %5, %6, vcc"
                : "=&v"(feat), "=&v"(sel)
                : "v"(x), "v"(thr), "v"(pair), "v"(l), "v"(r)
                : "vcc");
        } else {
            asm("v_cmp_ge_f32 vcc, %2, %3\n\t"
                "s_nop 1\n\t"
                "v_cndmask_b32_sdwa %0, %4, %4, vcc dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:WORD_0 src1_sel:WORD_1\n\t"
                "v_cndmask_b32 %1, %5, %6, vcc"
                : "=&v"(feat), "=&v"(sel)
                : "v"(x), "v"(thr), "v"(pair), "v"(l), "v"(r)
                : "vcc");
            feat &= kCodeFeature;
        }
        fw = 0;
        (void)fw_cur;
    } else {
        uint64_t t0, t1;
        // vcc = go left = x < thr || (isnan(x) && flag)
        if constexpr (NARROW) {
            asm("v_cmp_u_f32 %[t0], %[x], %[x]\n\t"
                "v_cmp_gt_i32 %[t1], 0, %[fc]\n\t"
                "s_and_b64 %[t0], %[t0], %[t1]\n\t"
                "v_cmp_lt_f32 vcc, %[x], %[th]\n\t"
                "s_or_b64 vcc, vcc, %[t0]\n\t"
                "v_cndmask_b32_sdwa %[ft], %[p], %[p], vcc dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_2 src1_sel:BYTE_0\n\t"
                "v_cndmask_b32_sdwa %[fw], %[p], %[p], vcc dst_sel:WORD_1 dst_unused:UNUSED_PAD src0_sel:WORD_1 src1_sel:WORD_0\n\t"
                "v_cndmask_b32 %[sl], %[r], %[l], vcc"
                : [ft] "=&v"(feat), [fw] "=&v"(fw), [sl] "=&v"(sel), [t0] "=&s"(t0), [t1] "=&s"(t1)
                : [x] "v"(x), [th] "v"(thr), [p] "v"(pair), [fc] "v"(fw_cur), [l] "v"(l), [r] "v"(r)
                : "vcc");
        } else {
            asm("v_cmp_u_f32 %[t0], %[x], %[x]\n\t"
                "v_cmp_gt_i32 %[t1], 0, %[fc]\n\t"
                "s_and_b64 %[t0], %[t0], %[t1]\n\t"
                "v_cmp_lt_f32 vcc, %[x], %[th]\n\t"
                "s_or_b64 vcc, vcc, %[t0]\n\t"
                "v_cndmask_b32_sdwa %[ft], %[p], %[p], vcc dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:WORD_1 src1_sel:WORD_0\n\t"
                "v_cndmask_b32_sdwa %[fw], %[p], %[p], vcc dst_sel:WORD_1 dst_unused:UNUSED_PAD src0_sel:WORD_1 src1_sel:WORD_0\n\t"
                "v_cndmask_b32 %[sl], %[r], %[l], vcc"
                : [ft] "=&v"(feat), [fw] "=&v"(fw), [sl] "=&v"(sel), [t0] "=&s"(t0), [t1] "=&s"(t1)
                : [x] "v"(x), [th] "v"(thr), [p] "v"(pair), [fc] "v"(fw_cur), [l] "v"(l), [r] "v"(r)
                : "vcc");
            feat &= kCodeFeature;
        }
    }
}

// Last level: the leaf reached from a last-level record {threshold, left leaf, right leaf, 0}.
template <bool NAN_AWARE>
__device__ __forceinline__ float leaf_of(float x, const uint4 &lv, int32_t fw_cur) {
    bool left = x < __uint_as_float(lv.x);
    if (NAN_AWARE) left = left || (x != x && fw_cur < 0);
    return __uint_as_float(left ? lv.y : lv.z);
}

// Walk NT_ trees at LDS addresses tb[] (heads hd[], address constants wc[]) for R rows of this
// lane (feature tile row stride RT4 bytes per feature; lane_off[r] = LDS address of the lane's
// r-th row of feature 0).  Every (tree, row) pair is an independent chain c = tree * R + row.  A
// chain's step at one level decides the child, then at once issues the child's two LDS reads
// (feature value, record); the chains take their steps in turn, so while one chain decides, the
// reads of all the others are in flight (LDS reads of a wave return in order, and the scheduling
// barriers keep that order).  Per chain and inner level: a compare, two selects and two address
// computations.
template <int D, int NT_, int R, uint32_t RT4, bool NAN_AWARE, bool NARROW>
__device__ __forceinline__ void walk_trees(const uint32_t (&tb)[NT_], const TreeHead (&hd)[NT_],
                                           const WalkConst (&wc)[NT_], const uint32_t (&lane_off)[R],
                                           double (&acc)[R]) {
    constexpr int NC = NT_ * R;
    uint32_t thr0[NT_], pair0[NT_];
    int32_t fw0[NT_];
#pragma unroll
    for (int i = 0; i < NT_; ++i) {
        thr0[i] = in_vgpr(hd[i].thr);
        pair0[i] = in_vgpr(hd[i].pair);
        fw0[i] = NAN_AWARE ? (int32_t)in_vgpr(hd[i].code << 16) : 0;
    }
    float x[NC];
    uint32_t a[NC];
    int32_t fw[NC];
    uint2 rec[NC];
    uint4 lv[NC];
    // level 0: the root is the same node for every row of a tree
#pragma unroll
    for (int c = 0; c < NC; ++c) x[c] = lds_ld<float>((hd[c / R].code & kCodeFeature) * RT4 + lane_off[c % R]);
    if constexpr (D == 1) {
#pragma unroll
        for (int c = 0; c < NC; ++c) {
            lv[c] = lds_ld<uint4>(tb[c / R] + 16u);
            fw[c] = fw0[c / R];
        }
    } else {
#pragma unroll
        for (int c = 0; c < NC; ++c) {
            const int i = c / R;
            uint32_t f, sel;
            decide<NAN_AWARE, NARROW>(x[c], thr0[i], pair0[i], fw0[i], wc[i].l0, wc[i].r0, f, fw[c], sel);
            x[c] = lds_ld<float>(f * RT4 + lane_off[c % R]);
            a[c] = sel;
            if constexpr (D > 2)
                rec[c] = lds_ld<uint2>(sel);
            else
                lv[c] = lds_ld<uint4>(sel);
            __builtin_amdgcn_sched_barrier(0);
        }
        // levels 1 .. D-2
#pragma unroll
        for (int lvl = 1; lvl + 1 < D; ++lvl) {
#pragma unroll
            for (int c = 0; c < NC; ++c) {
                const int i = c / R;
                const bool to_last = lvl + 2 == D;
                uint32_t f, sel;
                decide<NAN_AWARE, NARROW>(x[c], rec[c].x, rec[c].y, fw[c], to_last ? wc[i].l_last : wc[i].l,
                                          to_last ? wc[i].r_last : wc[i].r, f, fw[c], sel);
                x[c] = lds_ld<float>(f * RT4 + lane_off[c % R]);
                if (!to_last) {
                    a[c] = 2u * a[c] + sel;
                    rec[c] = lds_ld<uint2>(a[c]);
                } else {
                    a[c] = 4u * a[c] + sel;
                    lv[c] = lds_ld<uint4>(a[c]);
                }
                __builtin_amdgcn_sched_barrier(0);
            }
        }
    }
    // last level: threshold and both leaves
#pragma unroll
    for (int c = 0; c < NC; ++c) acc[c % R] += (double)leaf_of<NAN_AWARE>(x[c], lv[c], fw[c]);
}
// Item i of a row tile ([F][RT] fp32 in LDS, RT/4 float4 per feature): rows row0 + 4*(i % V) ..
// + 3 of feature i / V.  tile_item_vec: one 16-byte load (the tile lies below n_rows and ld, the
// base are 16-byte aligned); tile_item_any: four loads at row indices clamped to n_rows - 1
// (n_rows >= 1), zero past n_rows -- branch-free, for the ragged last tile or an unaligned ld.
// Which one is used is decided once per tile, so full tiles compile to plain vector loads.
template <int V>
__device__ __forceinline__ float4 tile_item_vec(const float *__restrict__ X, int64_t ld, int row0, int i) {
    const int f = i / V, r = row0 + 4 * (i % V);
    return *reinterpret_cast<const float4 *>(X + (int64_t)f * ld + r);
}

template <int V>
__device__ __forceinline__ float4 tile_item_any(const float *__restrict__ X, int64_t ld, int n_rows, int row0, int i) {
    const int f = i / V, r = row0 + 4 * (i % V);
    const float *src = X + (int64_t)f * ld;
    const int last = n_rows - 1;
    const float x = src[min(r, last)], y = src[min(r + 1, last)], z = src[min(r + 2, last)], w = src[min(r + 3, last)];
    return make_float4(r < n_rows ? x : 0.f, r + 1 < n_rows ? y : 0.f, r + 2 < n_rows ? z : 0.f, r + 3 < n_rows ? w : 0.f);
}

__device__ __forceinline__ int any_nan(float4 v) {
    return (v.x != v.x) | (v.y != v.y) | (v.z != v.z) | (v.w != v.w);
}

// Stage rows [row0, row0 + RT) of every feature into LDS, with 4 loads in flight per thread;
// returns (block-wide) whether any staged value is NaN.  `flag` is an LDS word that is 0 on entry
// (ordered before this call by a barrier); threads that see a NaN set it, and the barrier at the
// end publishes it.
template <int RT, int NT>
__device__ __forceinline__ int stage_features(char *smem, const float *__restrict__ X, int64_t ld, int n_rows, int F,
                                              int vec_ok, int row0, volatile int *flag) {
    constexpr int V = RT / 4;  // float4 per feature row of the tile
    constexpr int B = 4;
    int has_nan = 0;
    const int total = F * V;
    const bool full = vec_ok && row0 + RT <= n_rows;
    float4 *dst = reinterpret_cast<float4 *>(smem);
    for (int i0 = threadIdx.x; i0 < total; i0 += B * NT) {
        float4 v[B];
        if (full) {
#pragma unroll
            for (int j = 0; j < B; ++j) {
                const int i = i0 + j * NT;
                v[j] = i < total ? tile_item_vec<V>(X, ld, row0, i) : make_float4(0.f, 0.f, 0.f, 0.f);
            }
        } else {
#pragma unroll
            for (int j = 0; j < B; ++j) {
                const int i = i0 + j * NT;
                v[j] = i < total ? tile_item_any<V>(X, ld, n_rows, row0, i) : make_float4(0.f, 0.f, 0.f, 0.f);
            }
        }
#pragma unroll
        for (int j = 0; j < B; ++j) {
            const int i = i0 + j * NT;
            if (i < total) {
                has_nan |= any_nan(v[j]);
                dst[i] = v[j];
            }
        }
    }
    if (has_nan) *flag = 1;
    __syncthreads();
    return *flag;
}

// Register prefetch of a whole row tile (used when F * RT/4 <= NPF * NT): thread t holds items
// t + j*NT.  The commit writes them to LDS and sets `flag` if any is NaN; the caller's next barrier
// publishes both.
template <int RT, int NT, int NPF>
__device__ __forceinline__ void tile_fetch(float4 (&xf)[NPF], const float *__restrict__ X, int64_t ld, int n_rows,
                                           int F, int vec_ok, int row0) {
    constexpr int V = RT / 4;
    const int total = F * V;
    if (vec_ok && row0 + RT <= n_rows) {
#pragma unroll
        for (int j = 0; j < NPF; ++j) {
            const int i = threadIdx.x + j * NT;
            xf[j] = i < total ? tile_item_vec<V>(X, ld, row0, i) : make_float4(0.f, 0.f, 0.f, 0.f);
        }
    } else {
#pragma unroll
        for (int j = 0; j < NPF; ++j) {
            const int i = threadIdx.x + j * NT;
            xf[j] = i < total ? tile_item_any<V>(X, ld, n_rows, row0, i) : make_float4(0.f, 0.f, 0.f, 0.f);
        }
    }
}

template <int RT, int NT, int NPF>
__device__ __forceinline__ void tile_commit(const float4 (&xf)[NPF], char *smem, int F, volatile int *flag) {
    const int total = F * (RT / 4);
    float4 *dst = reinterpret_cast<float4 *>(smem);
    int has_nan = 0;
#pragma unroll
    for (int j = 0; j < NPF; ++j) {
        const int i = threadIdx.x + j * NT;
        if (i < total) {
            has_nan |= any_nan(xf[j]);
            dst[i] = xf[j];
        }
    }
    if (has_nan) *flag = 1;
}

// Fixed-order combination of the per-wave row sums (acc[r] of wave w for tile row r*64 + lane):
// reduce_put stores them to `red`; after a barrier, reduce_sum writes the fp32 partials out[t] for
// tile rows t with row0 + t < n_rows.  `red` must not overlap live data.
template <int RPL>
__device__ __forceinline__ void reduce_put(double *red, const double (&acc)[RPL], int wid, int lane) {
#pragma unroll
    for (int r = 0; r < RPL; ++r) red[wid * 64 * RPL + r * 64 + lane] = acc[r];
}

template <int RPL, int NW>
__device__ __forceinline__ void reduce_sum(const double *red, int row0, int n_rows, float *__restrict__ out) {
    constexpr int RT = 64 * RPL;
    for (int t = threadIdx.x; t < RT; t += NW * kWave) {
        double s = 0.0;
#pragma unroll
        for (int w = 0; w < NW; ++w) s += red[w * RT + t];
        if (row0 + t < n_rows) out[t] = (float)s;
    }
}

template <int RPL, int NW>
__device__ __forceinline__ void reduce_rows(double *red, const double (&acc)[RPL], int wid, int lane, int row0, int n_rows,
                                            float *__restrict__ out) {
    reduce_put<RPL>(red, acc, wid, lane);
    __syncthreads();
    reduce_sum<RPL, NW>(red, row0, n_rows, out);
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

// Trees t + j*TW (j < NTW, t + j*TW < t_end) of a wave: fetch into registers, commit to the wave's
// LDS slots (slot j) and take their wave-uniform heads (lane l holds uint4 l of each tree).
template <int S16, int PF, int NTW, int TW>
__device__ __forceinline__ void group_fetch(uint4 (&pf)[NTW][PF], const uint4 *__restrict__ trees, int t, int t_end,
                                            int lane) {
#pragma unroll
    for (int j = 0; j < NTW; ++j)
        if (t + j * TW < t_end) wave_fetch<S16>(pf[j], trees + (int64_t)(t + j * TW) * S16, lane);
}

template <int S16, int PF, int NTW, int TW>
__device__ __forceinline__ void group_commit(const uint4 (&pf)[NTW][PF], char *slots, TreeHead (&hd)[NTW], int t,
                                             int t_end, int lane) {
#pragma unroll
    for (int j = 0; j < NTW; ++j)
        if (t + j * TW < t_end) {
            wave_commit<S16>(pf[j], reinterpret_cast<uint4 *>(slots + (uint32_t)j * (S16 * 16)), lane);
            hd[j].code = __builtin_amdgcn_readlane(pf[j][0].y, 0);
            hd[j].thr = __builtin_amdgcn_readlane(pf[j][0].z, 0);
            hd[j].pair = __builtin_amdgcn_readlane(pf[j][0].w, 0);
        }
}

// ---- K1, depth <= 10: persistent workgroups with per-wave private tree slots ----
// The work is the space of (row tile, tree) pairs, tile-major: v = tile * T + tree.  Slice s owns
// the contiguous range [s*L, (s+1)*L), so every workgroup walks the same number of trees and the
// machine is busy to the end.  A slice covers whole tiles plus, at each end, possibly part of a
// tile that the neighbouring slice also covers; both must stage that tile's features.  So that
// the second staging hits L2: consecutive slices run on the same XCD (workgroups are dealt to the
// 8 XCDs round-robin, so workgroup b takes slice (b % 8) * (grid / 8) + b / 8), and even slices
// walk their tiles last to first while odd slices walk first to last -- a shared tile is then the
// first tile of both slices or the last tile of both.  Wave w walks trees w, w + TW, ... of each
// piece, NTW at a time from its NTW LDS slots; the next NTW trees are fetched into registers
// meanwhile and committed over the slots after the walk (LDS operations of one wave execute in
// order, so the walk's reads are served before the commit's writes).  The partial sums of the
// piece of tile i walked by slice s are stored at block (i + s) of RT floats: a slice covers a
// contiguous run of tiles, so i + s grows strictly along the (slice, tile) pieces and (tiles +
// slices) blocks hold them all; a tile's pieces are summed later in slice order.
// Tree groups: an ensemble too large for one XCD's L2 is split into G groups of consecutive trees
// (G divides 8); the workgroups of XCD x all walk group x % G, so every XCD keeps only its group
// L2-resident and a tile's features are staged once per group.  Within a group the work is sliced
// as above.  Group g: trees [g Tg, g Tg + Tc) with Tg = ceil(T / G); its slices r = 0 .. nb/G - 1.
__device__ __forceinline__ void block_slice(int b, int nb, int G, int &g, int &r) {
    const int x = b % 8, j = b / 8;  // nb is a multiple of 8
    g = x % G;
    r = (x / G) * (nb / 8) + j;
}

// Trees of group g, its (tile, tree) pairs per slice, and the offset of its partial-sum blocks.
__host__ __device__ __forceinline__ int group_trees(int T, int G, int g) {
    const int tg = (T + G - 1) / G;
    return T - g * tg < tg ? T - g * tg : tg;
}
__host__ __device__ __forceinline__ int64_t group_slice_len(int64_t tiles, int tc, int nbg) {
    return (tiles * tc + nbg - 1) / nbg;
}

template <int D, int RPL, int TW, int NTW, bool NARROW>
__global__ __launch_bounds__(64 * TW) void k_tree_score_wp(
    const float *__restrict__ X, int64_t ld, int n_rows, int F, int vec_ok, const uint4 *__restrict__ trees_all,
    int T_all, int G, int tiles, float *__restrict__ partial_all) {
    constexpr int RT = 64 * RPL;
    constexpr int S16 = tree_stride_bytes(D) / 16;  // uint4 per packed tree
    constexpr int PF = (S16 + kWave - 1) / kWave;   // uint4 per lane per tree
    constexpr int STEP = NTW * TW;                  // trees between a wave's consecutive groups
    extern __shared__ __align__(16) char smem[];
    int g, s;
    block_slice(blockIdx.x, gridDim.x, G, g, s);
    const int nbg = gridDim.x / G;
    const int T = group_trees(T_all, G, g);
    if (T <= 0) return;  // whole workgroup
    const uint4 *__restrict__ trees = trees_all + (int64_t)g * ((T_all + G - 1) / G) * S16;
    float *__restrict__ partial = partial_all + (int64_t)g * (tiles + nbg) * RT;
    const int64_t V = (int64_t)tiles * T, L = group_slice_len(tiles, T, nbg);
    const int64_t v_begin = (int64_t)s * L;
    const int64_t v_end = v_begin + L < V ? v_begin + L : V;
    if (v_begin >= v_end) return;  // whole workgroup: no barrier is skipped by part of it
    const int tile_first = (int)(v_begin / T), tile_last = (int)((v_end - 1) / T);
    const int dir = (s & 1) ? 1 : -1;
    const int n_pieces = tile_last - tile_first + 1;
    // trees [lo, hi) of tile i that belong to this slice
    auto piece_lo = [&](int i) { return (int)(v_begin - (int64_t)i * T > 0 ? v_begin - (int64_t)i * T : 0); };
    auto piece_hi = [&](int i) { return (int)(v_end - (int64_t)i * T < T ? v_end - (int64_t)i * T : T); };

    const int wid = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave), lane = threadIdx.x % kWave;
    const uint32_t ring_off = (uint32_t)F * RT * 4u;
    const uint32_t slot0 = ring_off + (uint32_t)wid * NTW * (S16 * 16);
    char *const slots = smem + slot0;
    // four words past the slot / reduction region: two NaN flags and two tree-progress counters,
    // alternating between pieces; thread 0 clears the next piece's pair once every thread is done
    // with its previous use
    constexpr uint32_t kSlots = (uint32_t)TW * NTW * S16 * 16, kRed = (uint32_t)TW * RT * 8;
    volatile int *const flags = reinterpret_cast<volatile int *>(smem + ring_off + (kSlots > kRed ? kSlots : kRed));
    unsigned int *const progress = const_cast<unsigned int *>(reinterpret_cast<volatile unsigned int *>(flags)) + 2;
    if (threadIdx.x == 0) flags[0] = flags[1] = flags[2] = flags[3] = 0;
    __syncthreads();

    uint4 pf[NTW][PF];
#pragma unroll
    for (int j = 0; j < NTW; ++j)
#pragma unroll
        for (int k = 0; k < PF; ++k) pf[j][k] = make_uint4(0, 0, 0, 0);
    TreeHead hd[NTW];
#pragma unroll
    for (int j = 0; j < NTW; ++j) hd[j] = TreeHead{0, 0, 0};
    const uint32_t base = lds_addr(smem);
    uint32_t lane_off[RPL];
#pragma unroll
    for (int r = 0; r < RPL; ++r) lane_off[r] = base + (uint32_t)(r * 64 + lane) * 4u;
    // slot addresses and walk constants (both entries the same slot when NTW == 1)
    const uint32_t tb[2] = {base + slot0, base + slot0 + (NTW > 1 ? S16 * 16 : 0)};
    WalkConst wc[2];
    wc[0] = walk_const<D>(tb[0]);
    wc[1] = NTW > 1 ? walk_const<D>(tb[1]) : wc[0];

    // the next tile's features are loaded into registers during the walk of the current one when
    // they fit (F <= kRegTileFeatures, and the tree and tile prefetch registers within what the
    // shape's occupancy leaves beside the walk), else staged between the pieces
    constexpr int NT = 64 * TW;
    constexpr int kNpx = (kRegTileFeatures * (RT / 4) + NT - 1) / NT;
    constexpr int kWavesPerSimd = (TW + 3) / 4;
    constexpr int kVgprBudget = (512 / kWavesPerSimd < 256 ? 512 / kWavesPerSimd : 256) - 80 - 2 * PF * NTW;  // walk
    constexpr bool kRegTile = RPL <= 2 && 4 * (PF * NTW + kNpx) <= kVgprBudget;
    constexpr int NPX = kRegTile ? kNpx : 1;
    const bool x_regs = kRegTile && F * (RT / 4) <= NPX * NT;
    float4 xf[NPX];
    double *const red = reinterpret_cast<double *>(smem + ring_off);

    int tile = dir > 0 ? tile_first : tile_last;
    int t0 = piece_lo(tile), t1 = piece_hi(tile);
    int t = t0 + wid;
    group_fetch<S16, PF, NTW, TW>(pf, trees, t, t1, lane);   // overlaps the feature staging
    int has_nan;
    if (x_regs) {  // the whole first tile in one batch of loads
        tile_fetch<RT, NT, NPX>(xf, X, ld, n_rows, F, vec_ok, tile * RT);
        tile_commit<RT, NT, NPX>(xf, smem, F, flags);
        __syncthreads();
        has_nan = __builtin_amdgcn_readfirstlane(flags[0]);
        if (n_pieces > 1) tile_fetch<RT, NT, NPX>(xf, X, ld, n_rows, F, vec_ok, (tile + dir) * RT);
    } else {
        has_nan = __builtin_amdgcn_readfirstlane(stage_features<RT, NT>(smem, X, ld, n_rows, F, vec_ok, tile * RT, flags));
    }
    // With x_regs, xf holds the loads of the next tile from the commit of the current one on (its
    // fetch is issued as soon as the registers are free), so the stream of feature tiles keeps a
    // tile in flight through the barriers and row-sum reduction between pieces.
    for (int piece = 0;; ++piece) {
        const int row0 = tile * RT;
        if (threadIdx.x == 0) {
            flags[(piece + 1) & 1] = 0;      // NaN flag of the next tile (set at its staging, after B1)
            flags[2 + ((piece + 1) & 1)] = 0;  // progress count of the next piece
        }
        uint32_t my_done = 0;
        group_commit<S16, PF, NTW, TW>(pf, slots, hd, t, t1, lane);
        group_fetch<S16, PF, NTW, TW>(pf, trees, t + STEP, t1, lane);
        const bool next = piece + 1 < n_pieces;
        const int ntile = tile + dir;
        double acc[RPL];
#pragma unroll
        for (int r = 0; r < RPL; ++r) acc[r] = 0.0;
        for (; t < t1; t += STEP) {
            if (NTW == 2 && t + TW < t1) {
                const TreeHead h2[2] = {hd[0], hd[NTW - 1]};
                if (has_nan)
                    walk_trees<D, 2, RPL, (uint32_t)RT * 4u, true, NARROW>(tb, h2, wc, lane_off, acc);
                else
                    walk_trees<D, 2, RPL, (uint32_t)RT * 4u, false, NARROW>(tb, h2, wc, lane_off, acc);
            } else {
                const uint32_t tb1[1] = {tb[0]};
                const TreeHead h1[1] = {hd[0]};
                const WalkConst w1[1] = {wc[0]};
                if (has_nan)
                    walk_trees<D, 1, RPL, (uint32_t)RT * 4u, true, NARROW>(tb1, h1, w1, lane_off, acc);
                else
                    walk_trees<D, 1, RPL, (uint32_t)RT * 4u, false, NARROW>(tb1, h1, w1, lane_off, acc);
            }
            if (t + STEP < t1) {
                group_commit<S16, PF, NTW, TW>(pf, slots, hd, t + STEP, t1, lane);
                group_fetch<S16, PF, NTW, TW>(pf, trees, t + 2 * STEP, t1, lane);
            }
            // Fair progress: the SIMD arbiter favours older waves, and a piece ends at a barrier,
            // so a wave that has walked fewer trees than its workgroup's average takes the top
            // issue priority until it catches up.
            const uint32_t walked = (NTW == 2 && t + TW < t1) ? 2u : 1u;
            my_done += walked;
            uint32_t total = 0;
            if (lane == 0) total = atomicAdd(progress + (piece & 1), walked) + walked;
            total = __builtin_amdgcn_readfirstlane(total);
            if (my_done * TW < total)
                __builtin_amdgcn_s_setprio(3);
            else
                __builtin_amdgcn_s_setprio(0);
        }
        __builtin_amdgcn_s_setprio(0);
        const int nt0 = next ? piece_lo(ntile) : 0, nt1 = next ? piece_hi(ntile) : 0;
        if (next) group_fetch<S16, PF, NTW, TW>(pf, trees, nt0 + wid, nt1, lane);  // first trees of the next piece
        __syncthreads();  // B1: every wave is done with the tile and its slots
        reduce_put<RPL>(red, acc, wid, lane);
        if (next && x_regs) {
            tile_commit<RT, NT, NPX>(xf, smem, F, flags + ((piece + 1) & 1));
            if (piece + 2 < n_pieces) tile_fetch<RT, NT, NPX>(xf, X, ld, n_rows, F, vec_ok, (ntile + dir) * RT);
        }
        __syncthreads();  // B2: row sums and the next tile are in LDS
        reduce_sum<RPL, TW>(red, row0, n_rows, partial + ((int64_t)tile + s) * RT);
        if (!next) break;
        if (x_regs) {
            __syncthreads();  // B3: the sums are read before the next trees overwrite the slots
            has_nan = __builtin_amdgcn_readfirstlane(flags[(piece + 1) & 1]);
        } else {
            has_nan = __builtin_amdgcn_readfirstlane(
                stage_features<RT, NT>(smem, X, ld, n_rows, F, vec_ok, ntile * RT, flags + ((piece + 1) & 1)));
        }
        tile = ntile;
        t0 = nt0;
        t1 = nt1;
        t = t0 + wid;
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
template <int D, int TW, int ILP, bool NARROW>
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
    constexpr uint32_t kChunk = (uint32_t)CH16 * 16, kRed = (uint32_t)TW * RT * 8;
    volatile int *const flag = reinterpret_cast<volatile int *>(smem + chunk_off + (kChunk > kRed ? kChunk : kRed));
    if (threadIdx.x == 0) *flag = 0;
    __syncthreads();
    const int has_nan = stage_features<RT, NT>(smem, X, ld, n_rows, F, vec_ok, row0, flag);
    if (t_begin < t_end) block_commit<C, S16, NT>(pf, reinterpret_cast<uint4 *>(smem + chunk_off));
    __syncthreads();

    const int wid = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave), lane = threadIdx.x % kWave;
    const uint32_t base = lds_addr(smem);
    const uint32_t lane_off[1] = {base + (uint32_t)lane * 4u};
    double acc[1] = {0.0};
    for (int t0 = t_begin; t0 < t_end; t0 += C) {
        const bool more = t0 + C < t_end;
        if (more) block_fetch<C, S16, NT>(pf, trees, t0 + C, t_end);
        uint32_t tb[ILP];
        TreeHead hd[ILP];
        WalkConst wc[ILP];
#pragma unroll
        for (int i = 0; i < ILP; ++i) {
            tb[i] = base + chunk_off + (uint32_t)(wid * ILP + i) * (S16 * 16);
            const uint4 h = lds_ld<uint4>(tb[i]);
            hd[i] = TreeHead{(uint32_t)__builtin_amdgcn_readfirstlane(h.y), (uint32_t)__builtin_amdgcn_readfirstlane(h.z),
                             (uint32_t)__builtin_amdgcn_readfirstlane(h.w)};
            wc[i] = walk_const<D>(tb[i]);
        }
        if (has_nan)
            walk_trees<D, ILP, 1, (uint32_t)RT * 4u, true, NARROW>(tb, hd, wc, lane_off, acc);
        else
            walk_trees<D, ILP, 1, (uint32_t)RT * 4u, false, NARROW>(tb, hd, wc, lane_off, acc);
        __syncthreads();
        if (more) {
            block_commit<C, S16, NT>(pf, reinterpret_cast<uint4 *>(smem + chunk_off));
            __syncthreads();
        }
    }
    reduce_rows<1, TW>(reinterpret_cast<double *>(smem + chunk_off), acc, wid, lane, row0, n_rows,
                       partial + (int64_t)g * ldp + row0);
}

// K2: per-program sums.  A workgroup owns `ppw` (<= 64) consecutive programs and walks the rows
// they cover in chunks of kSegChunk rows.  Every thread forms the sums s_r of its rows of a chunk
// into LDS, in a fixed order in fp64 -- grouped layout: the `groups` slots partial[g * ldp + r];
// sliced layout: per tree group g, the slices b = first..last that cut the row's tile i, at block
// (i + b) of the group's region, with (first, last) computed once per (tile, group) of the chunk.
// Thread j then adds the rows of program j that lie in the chunk, in row order.  No sum depends on
// scheduling.  A row's first two slices are loaded for all of a thread's rows at once; a tile cut
// by more than two slices of one group (small rounds) takes the remaining ones in a loop.
constexpr int kSegThreads = 256, kSegChunk = 2048, kSegRows = kSegChunk / kSegThreads;
constexpr int kSegMaxProg = 64, kSegMaxGroups = 8, kSegMaxTiles = kSegChunk / 64 + 1;

__global__ __launch_bounds__(kSegThreads) void k_segsum(const float *__restrict__ partial, int64_t ldp, int rt_shift,
                                                        int T, int sliced, int groups, int tiles, int nbg,
                                                        const int32_t *__restrict__ prog_ptr, int n_prog, int n_rows,
                                                        int ppw, float base_score, float *__restrict__ prog_score,
                                                        float *__restrict__ stmt_score) {
    __shared__ double srow[kSegChunk];
    __shared__ int2 span[kSegMaxGroups * kSegMaxTiles];
    __shared__ int pb[kSegMaxProg], pe[kSegMaxProg], range[2];
    const int t = threadIdx.x;
    const int p0 = blockIdx.x * ppw;
    const int np = min(ppw, n_prog - p0);
    const int RT = 1 << rt_shift;
    if (t < kWave) {  // wave 0: the programs' clamped bounds and the rows they cover
        int b = n_rows, e = 0;
        if (t < np) {
            b = min(max(prog_ptr[p0 + t], 0), n_rows);
            e = min(max(prog_ptr[p0 + t + 1], b), n_rows);
            pb[t] = b;
            pe[t] = e;
        }
        int lo = b, hi = e;
#pragma unroll
        for (int m = 32; m >= 1; m >>= 1) {
            lo = min(lo, __shfl_xor(lo, m, kWave));
            hi = max(hi, __shfl_xor(hi, m, kWave));
        }
        if (t == 0) {
            range[0] = lo;
            range[1] = hi;
        }
    }
    __syncthreads();
    const int lo = range[0], hi = range[1];
    double acc = 0.0;
    for (int c0 = lo; c0 < hi; c0 += kSegChunk) {
        const int c1 = min(c0 + kSegChunk, hi);
        const int tile0 = c0 >> rt_shift;
        if (sliced) {
            const int ntc = ((c1 - 1) >> rt_shift) - tile0 + 1;
            const bool narrow = (int64_t)(tiles + 1) * T <= (int64_t)UINT32_MAX;  // 32-bit divisions suffice
            for (int i = t; i < ntc * groups; i += kSegThreads) {
                const int gi = i / ntc, ti = i - gi * ntc;
                const int64_t tile = tile0 + ti;
                const int tc = group_trees(T, groups, gi);
                int2 sp = make_int2(0, -1);
                if (tc > 0) {
                    const int64_t L = group_slice_len(tiles, tc, nbg);
                    if (narrow)
                        sp = make_int2((int)((uint32_t)(tile * tc) / (uint32_t)L),
                                       (int)((uint32_t)((tile + 1) * tc - 1) / (uint32_t)L));
                    else
                        sp = make_int2((int)(tile * tc / L), (int)(((tile + 1) * tc - 1) / L));
                }
                span[gi * kSegMaxTiles + ti] = sp;
            }
            __syncthreads();
        }
        double s[kSegRows];
#pragma unroll
        for (int k = 0; k < kSegRows; ++k) s[k] = 0.0;
        for (int gi = 0; gi < groups; ++gi) {
            const float *__restrict__ src = sliced ? partial + (int64_t)gi * (tiles + nbg) * RT : partial + (int64_t)gi * ldp;
            float v0[kSegRows], v1[kSegRows];
            int2 sp[kSegRows];
#pragma unroll
            for (int k = 0; k < kSegRows; ++k) {
                const int r = c0 + t + k * kSegThreads;
                v0[k] = v1[k] = 0.f;
                sp[k] = make_int2(0, 0);
                if (r < c1) {
                    if (sliced) {
                        sp[k] = span[gi * kSegMaxTiles + ((r >> rt_shift) - tile0)];
                        // slice b's piece of row r (tile i) is at block (i + b): src + r + b * RT
                        const float *q = src + r + (int64_t)sp[k].x * RT;
                        if (sp[k].y >= sp[k].x) v0[k] = q[0];
                        if (sp[k].y > sp[k].x) v1[k] = q[RT];
                    } else {
                        v0[k] = src[r];
                    }
                }
            }
#pragma unroll
            for (int k = 0; k < kSegRows; ++k) {
                s[k] += (double)v0[k];
                s[k] += (double)v1[k];
                const int r = c0 + t + k * kSegThreads;
                if (sliced && r < c1 && sp[k].y > sp[k].x + 1) {
                    const float *q = src + r + (int64_t)sp[k].x * RT;
                    for (int j = 2; j <= sp[k].y - sp[k].x; ++j) s[k] += (double)q[(int64_t)j * RT];
                }
            }
        }
#pragma unroll
        for (int k = 0; k < kSegRows; ++k) {
            const int r = c0 + t + k * kSegThreads;
            if (r < c1) {
                srow[r - c0] = s[k];
                if (stmt_score) stmt_score[r] = (float)s[k];
            }
        }
        __syncthreads();
        if (t < np) {
            const int b = max(pb[t], c0) - c0, e = min(pe[t], c1) - c0;
            int r = b;
            for (; r + 4 <= e; r += 4) {
                const double a0 = srow[r], a1 = srow[r + 1], a2 = srow[r + 2], a3 = srow[r + 3];
                acc += a0;
                acc += a1;
                acc += a2;
                acc += a3;
            }
            for (; r < e; ++r) acc += srow[r];
        }
        __syncthreads();  // srow and span are rewritten by the next chunk
    }
    if (t < np) prog_score[p0 + t] = (float)((double)base_score + acc);
}

// Programs per workgroup of K2: enough workgroups to cover the machine at every batch size.
int segsum_ppw(int32_t n_prog) { return n_prog >= 32768 ? 64 : 16; }

// ---------------------------------------------------------------------------------------------
// launch configuration
// ---------------------------------------------------------------------------------------------
using ChKernel = void (*)(const float *, int64_t, int, int, int, const uint4 *, int, int, int, float *, int64_t);
using WpKernel = void (*)(const float *, int64_t, int, int, int, const uint4 *, int, int, int, float *);

struct ScoreCfg {
    bool wp;            // persistent per-wave tree slots (else grid of shared chunks)
    int a, b, c;        // wp: RPL, TW, NTW;  ch: TW, ILP, -
    const void *kern;
    int rows_per_tile, threads;
    size_t lds;
};

// A per-wave-slot shape is instantiated for depth D only if its tree slots alone fit in LDS.
template <int D, int RPL, int TW, int NTW>
constexpr bool wp_fits() {
    return D <= kMaxWpDepth && (size_t)TW * NTW * tree_stride_bytes(D) + 64 * RPL * 4 <= (size_t)kLdsBytes;
}

template <int D, bool NARROW>
const void *pick_wp(int rpl, int tw, int ntw) {
#define HARL_WP(R, T, N)                                                                          \
    if constexpr (wp_fits<D, R, T, N>())                                                          \
        if (rpl == R && tw == T && ntw == N)                                                      \
            return reinterpret_cast<const void *>(k_tree_score_wp<D, R, T, N, NARROW>);
    HARL_WP(2, 16, 1) HARL_WP(2, 12, 2) HARL_WP(2, 12, 1) HARL_WP(2, 8, 1) HARL_WP(2, 6, 1) HARL_WP(2, 4, 1)
    HARL_WP(1, 16, 2) HARL_WP(1, 8, 1) HARL_WP(1, 4, 1)
#undef HARL_WP
    return nullptr;
}

template <int D, bool NARROW>
const void *pick_ch(int tw, int ilp) {
#define HARL_CH(T, I)                                                                           \
    if constexpr ((size_t)T * I * tree_stride_bytes(D) + 64 * 4 <= (size_t)kLdsBytes)          \
        if (tw == T && ilp == I) return reinterpret_cast<const void *>(k_tree_score_ch<D, T, I, NARROW>);
    HARL_CH(2, 1) HARL_CH(4, 1) HARL_CH(8, 1) HARL_CH(4, 2)
#undef HARL_CH
    return nullptr;
}

template <bool NARROW, int... Ds>
const void *pick_depth(int depth, bool wp, int a, int b, int c, std::integer_sequence<int, Ds...>) {
    const void *k = nullptr;
    ((depth == Ds + 1 ? (void)(k = wp ? pick_wp<Ds + 1, NARROW>(a, b, c) : pick_ch<Ds + 1, NARROW>(a, b)) : (void)0), ...);
    return k;
}

ScoreCfg make_cfg(const harl_ensemble *E, bool wp, int a, int b, int n) {
    const bool narrow = E->n_features <= kNarrowFeatures;
    ScoreCfg c{wp, a, b, n,
               narrow ? pick_depth<true>(E->depth, wp, a, b, n, std::make_integer_sequence<int, kMaxDepth>{})
                      : pick_depth<false>(E->depth, wp, a, b, n, std::make_integer_sequence<int, kMaxDepth>{}),
               0, 0, 0};
    const size_t stride = (size_t)E->tree_stride;
    if (wp) {
        c.rows_per_tile = 64 * a;
        c.threads = 64 * b;
        const size_t ring = (size_t)b * n * stride, red = (size_t)b * c.rows_per_tile * 8;
        c.lds = (size_t)E->n_features * c.rows_per_tile * 4 + (ring > red ? ring : red) + 16;  // + NaN flags, progress counters
    } else {
        c.rows_per_tile = 64;
        c.threads = 64 * a;
        const size_t chunk = (size_t)a * b * stride, red = (size_t)a * 64 * 8;
        c.lds = (size_t)E->n_features * 64 * 4 + (chunk > red ? chunk : red) + 16;  // + NaN flag
    }
    return c;
}

// Preferred shapes, best first; the first whose LDS fits is used.
ScoreCfg choose_cfg(const harl_ensemble *E) {
    std::vector<ScoreCfg> cands;
    const int wp_pref[][3] = {{2, 16, 1}, {2, 12, 2}, {2, 12, 1}, {2, 8, 1}, {2, 6, 1}, {2, 4, 1},
                              {1, 16, 2}, {1, 8, 1}, {1, 4, 1}};
    for (auto &p : wp_pref) cands.push_back(make_cfg(E, true, p[0], p[1], p[2]));
    const int ch_pref[][2] = {{8, 1}, {4, 2}, {4, 1}, {2, 1}};
    for (auto &p : ch_pref) cands.push_back(make_cfg(E, false, p[0], p[1], 1));
    for (const ScoreCfg &c : cands)
        if (c.kern && c.lds <= (size_t)kLdsBytes) return c;
    return cands.back();  // nothing fits: the launch reports HARL_E_UNSUPPORTED
}

// The shape chosen at create.
ScoreCfg stored_cfg(const harl_ensemble *E) { return make_cfg(E, E->cfg_wp != 0, E->cfg_a, E->cfg_b, E->cfg_c); }

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
// least 2 trees per wave per slice so the feature staging stays amortised.  The grid is a whole
// number of XCD rounds (a multiple of 8); slices past the work are empty.
struct WpSplit {
    int64_t tiles;
    int nb, G;  // workgroups (a multiple of 8) and tree groups
};

// Tree groups: the fewest (a power of 2 up to 8) whose share of the packed ensemble fits in about
// 3 MB of an XCD's 4 MB L2 (or the count forced at create).
int tree_groups(const harl_ensemble *E) {
    int G = 1;
    const int64_t bytes = (int64_t)E->n_trees * E->tree_stride;
    while (G < 8 && 2 * G <= E->n_trees && bytes / G > (3 << 20)) G *= 2;
    if (E->tree_groups_override > 0 && E->tree_groups_override <= E->n_trees) G = E->tree_groups_override;
    return G;
}

WpSplit wp_split(const harl_ensemble *E, const ScoreCfg &c, int32_t n_rows) {
    WpSplit w{};
    w.tiles = ceil_div(n_rows > 0 ? n_rows : 1, c.rows_per_tile);
    w.G = tree_groups(E);
    const int per_cu = (int)(kLdsBytes / c.lds) > 0 ? (int)(kLdsBytes / c.lds) : 1;
    int64_t nb = (int64_t)device_cus(E->device) * per_cu;
    // at least 2 trees per wave per slice, so the feature staging stays amortised
    const int64_t min_l = 2LL * c.b * c.c;
    const int64_t vg = w.tiles * ceil_div(E->n_trees, w.G);  // pairs of the largest group
    if (ceil_div(vg, nb / w.G > 0 ? nb / w.G : 1) < min_l) nb = ceil_div(vg, min_l) * w.G;
    w.nb = (int)round_up(nb < 8 ? 8 : nb, 8);
    return w;
}

// Number of tree groups G of the grid kernel.  Each group's share of the ensemble should stay
// L2-resident (about 2 MB per XCD), and the work items (row tile x group) should fill whole waves
// of the machine: G minimises (rounds of co-resident workgroups) x (walk time + staging time per
// item).
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
    return best;
}

// Floats of partial sums: sliced layout (tiles + workgroups) blocks of RT rows; grouped layout
// G rows-long slots.
size_t partial_floats(const harl_ensemble *E, const ScoreCfg &c, int32_t n_rows) {
    const int64_t ldp = round_up(n_rows > 0 ? n_rows : 1, 64);
    if (c.wp) {
        const WpSplit w = wp_split(E, c, n_rows);
        return (size_t)w.G * (w.tiles + w.nb / w.G) * c.rows_per_tile;
    }
    return (size_t)choose_groups(E, n_rows, c) * ldp;
}

}  // namespace

size_t score_round_ws_bytes(const harl_ensemble *E, int32_t n_rows) {
    const ScoreCfg c = stored_cfg(E);
    const size_t fp32 = partial_floats(E, c, n_rows) * sizeof(float) + 256;
    // an ensemble with both forms takes either walk by the round's size: enough for both, so that a
    // workspace sized for n_rows serves every smaller round too
    if (score_b16_packed(E)) return std::max(fp32, score_b16_ws_bytes(E, n_rows));
    return fp32;
}

int score_round_launch(const harl_ensemble *E, const float *X, int64_t ld, int32_t n_rows,
                       const int32_t *prog_ptr, int32_t n_prog, float *prog_score, float *stmt_score,
                       void *ws, size_t ws_bytes, hipStream_t stream) {
    const bool b16 = score_b16_usable(E, n_rows);
    const ScoreCfg c = stored_cfg(E);
    const int64_t ldp = round_up(n_rows > 0 ? n_rows : 1, 64);
    if (ws_bytes < score_round_ws_bytes(E, n_rows)) return fail(HARL_E_WORKSPACE, "harl_score_round: workspace too small");
    float *partial = static_cast<float *>(ws);
    if (n_prog <= 0) return HARL_OK;
    const int ppw = segsum_ppw(n_prog);
    const unsigned seg_grid = (unsigned)ceil_div(n_prog, ppw);
    if (n_rows > 0 && b16) {
        int groups = 0, tiles = 0, nbg = 0;
        if (const int rc = score_b16_launch(E, X, ld, n_rows, &partial, &groups, &tiles, &nbg, ws, ws_bytes, stream))
            return rc;
        hipLaunchKernelGGL(k_segsum, dim3(seg_grid), dim3(kSegThreads), 0, stream, partial, ldp, 8, E->n_trees, 1,
                           groups, tiles, nbg, prog_ptr, n_prog, n_rows, ppw, E->base_score, prog_score, stmt_score);
        HARL_HIP_CHECK(hipGetLastError());
        return HARL_OK;
    }
    if (n_rows == 0) {
        hipLaunchKernelGGL(k_segsum, dim3(seg_grid), dim3(kSegThreads), 0, stream, partial, ldp, 6, 1, 0, 0, 1, 8,
                           prog_ptr, n_prog, 0, ppw, E->base_score, prog_score, stmt_score);
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
                           c.lds, stream, X, ld, n_rows, E->n_features, vec_ok, trees, E->n_trees, w.G, (int)w.tiles,
                           partial);
        HARL_HIP_CHECK(hipGetLastError());
        hipLaunchKernelGGL(k_segsum, dim3(seg_grid), dim3(kSegThreads), 0, stream, partial, ldp,
                           __builtin_ctz((unsigned)c.rows_per_tile), E->n_trees, 1, w.G, (int)w.tiles, w.nb / w.G,
                           prog_ptr, n_prog, n_rows, ppw, E->base_score, prog_score, stmt_score);
    } else {
        const int G = choose_groups(E, n_rows, c);
        const int tiles = (int)ceil_div(n_rows, c.rows_per_tile);
        const int tpg = (int)ceil_div(E->n_trees, G);
        const int groups = (int)ceil_div(E->n_trees, tpg);
        hipLaunchKernelGGL(reinterpret_cast<ChKernel>(const_cast<void *>(c.kern)), dim3((unsigned)tiles * groups),
                           dim3(c.threads), c.lds, stream, X, ld, n_rows, E->n_features, vec_ok, trees, E->n_trees,
                           tpg, groups, partial, ldp);
        HARL_HIP_CHECK(hipGetLastError());
        hipLaunchKernelGGL(k_segsum, dim3(seg_grid), dim3(kSegThreads), 0, stream, partial, ldp,
                           __builtin_ctz((unsigned)c.rows_per_tile), E->n_trees, 0, groups, tiles, 8, prog_ptr, n_prog,
                           n_rows, ppw, E->base_score, prog_score, stmt_score);
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
    const int M = 1 << D;
    const uint32_t LL = tree_ll_bytes(D);
    const int stride = tree_stride_bytes(D);
    std::vector<uint8_t> host((size_t)T * stride, 0);
    std::vector<int32_t> map(2 * (size_t)M);      // complete-tree slot (1-based) -> original node
    std::vector<uint32_t> code(M), thr_bits(M);   // per internal slot 1 .. M-1
    // the complete-tree form of every tree, for the binned packing: per split slot its feature (-1
    // for a dummy split below an early leaf), threshold and missing direction; per leaf slot its value
    std::vector<int32_t> c_feat((size_t)T * M, -1);
    std::vector<float> c_thr((size_t)T * M, 0.f), c_leaf((size_t)T * M, 0.f);
    std::vector<uint8_t> c_dl((size_t)T * M, 0);
    auto put = [](uint8_t *dst, uint32_t w) { std::memcpy(dst, &w, 4); };
    for (int t = 0; t < T; ++t) {
        uint8_t *tb = host.data() + (size_t)t * stride;
        map[1] = d->root[t];
        for (int s = 1; s < M; ++s) {
            const int32_t n = map[s];
            float thr = 0.f;
            code[s] = 0;
            if (d->feature[n] >= 0) {
                code[s] = (uint32_t)d->feature[n] | (d->default_left[n] ? kCodeDefaultLeft : 0u);
                thr = d->threshold[n];
                c_feat[(size_t)t * M + s] = d->feature[n];
                c_thr[(size_t)t * M + s] = thr;
                c_dl[(size_t)t * M + s] = d->default_left[n] ? 1 : 0;
                if (std::isnan(thr)) thr = -INFINITY;   // no value is < NaN: everything present goes right
                map[2 * s] = d->left[n];
                map[2 * s + 1] = d->right[n];
            } else {                                    // early leaf: dummy split, both sides repeat it
                map[2 * s] = n;
                map[2 * s + 1] = n;
            }
            std::memcpy(&thr_bits[s], &thr, 4);
        }
        for (int j = 0; j < M; ++j) c_leaf[(size_t)t * M + j] = d->leaf_value[map[M + j]];
        put(tb + 4, code[1]);
        for (int s = 1; s < M / 2; ++s) {
            put(tb + 8 * s, thr_bits[s]);
            put(tb + 8 * s + 4, code[2 * s] | code[2 * s + 1] << 16);
        }
        for (int s = M / 2; s < M; ++s) {
            uint8_t *rec = tb + LL + 16 * (s - M / 2);
            const float l0 = d->leaf_value[map[2 * s]], l1 = d->leaf_value[map[2 * s + 1]];
            put(rec, thr_bits[s]);
            std::memcpy(rec + 4, &l0, 4);
            std::memcpy(rec + 8, &l1, 4);
        }
    }
    harl_ensemble *E = new (std::nothrow) harl_ensemble{};
    if (!E) return fail(HARL_E_NOMEM, "harl_ensemble_create: host allocation failed");
    E->n_trees = T;
    E->n_features = F;
    E->depth = D;
    E->tree_stride = stride;
    E->base_score = d->base_score;
    // the tree-group count may be forced (a power of 2 up to 8) to test the grouped layout on small
    // ensembles; read once here, so that every call on the handle uses the same layout
    if (const char *env = std::getenv("HARL_SCORE_TREE_GROUPS")) {
        const int o = std::atoi(env);
        if ((o == 1 || o == 2 || o == 4 || o == 8) && o <= T) E->tree_groups_override = o;
    }
    // likewise the row count from which a depth-8 ensemble takes the binned walk
    E->b16_min_rows_override = -1;
    if (const char *env = std::getenv("HARL_SCORE_BINNED_MIN_ROWS")) {
        const long o = std::atol(env);
        if (o >= 0 && o <= INT32_MAX) E->b16_min_rows_override = (int32_t)o;
    }
    {
        const ScoreCfg c = choose_cfg(E);
        E->cfg_wp = c.wp ? 1 : 0;
        E->cfg_a = c.a;
        E->cfg_b = c.b;
        E->cfg_c = c.c;
    }
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
    if (const int rc = pack_b16(E, c_feat, c_thr, c_dl, c_leaf, stream)) {
        (void)hipFree(E->d_trees);
        delete E;
        return rc;
    }
    *out = E;
    return HARL_OK;
}

void free_ensemble(harl_ensemble *E) {
    free_b16(E);
    (void)hipFree(E->d_trees);
    delete E;
}

}  // namespace harl
