// The binned tree walk (the hot loop of k_tree_score_b16 in score_bin.hip), shared with the
// visit-loop microbenchmark (probe/visit_probe.hip) so that both run the same instructions.  Layouts
// of the code tile and of the packed trees are described in score_bin.hip.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace harl {
namespace b16 {


constexpr int kWave = 64;
constexpr int kRT = 256;                        // rows per tile
constexpr int kRPL = 4;                         // rows per lane
constexpr uint32_t kRowBytes = kRT * 2;         // bytes per feature row of a tile
constexpr int kTileU4 = kRowBytes / 16;         // uint4 per feature row of a tile (32)
constexpr uint32_t kMissing = 0xFFFFu;
constexpr uint32_t kGroupStride = 65536;        // LDS bytes between the tile's two row groups

// LDS accesses by absolute byte address.
__device__ __forceinline__ uint32_t lds_b32(uint32_t a) {
    return *(const __attribute__((address_space(3))) uint32_t *)(uintptr_t)a;
}
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint2 lds_b64(uint32_t a) {
    const u32x2 v = *(const __attribute__((address_space(3))) u32x2 *)(uintptr_t)a;
    return make_uint2(v.x, v.y);
}
typedef __attribute__((address_space(3))) char lds_char;
__device__ __forceinline__ uint32_t lds_addr(const char *p) { return (uint32_t)(uintptr_t)(const lds_char *)p; }

// An opaque VGPR copy of a wave-uniform value (so that one v_cndmask can select between two).
__device__ __forceinline__ uint32_t in_vgpr(uint32_t v) {
    asm("" : "+v"(v));
    return v;
}

// One inner decision: code c at a node with word w = theta | U << 16 and child features p (byte 0
// left, byte 1 right).  Writes the child's feature into byte 1 of the code address xa (the other
// bytes, the lane's row, are kept) and returns sel = go right ? r : l.  The compare writes VCC and
// the SDWA select reads it (two wait states between them).  CSEL picks the code from c: the whole
// register (0), or its low (1) or high (2) half, for two rows' codes read as one dword.
#define HARL_B16_DECIDE(CSEL)                                                                                       \
    asm("v_sub_u32_sdwa %[d], %[c], %[w] dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:" CSEL " src1_sel:WORD_0\n\t" \
        "v_cmp_le_u32_sdwa vcc, %[d], %[w] src0_sel:DWORD src1_sel:WORD_1\n\t"                                     \
        "s_nop 1\n\t"                                                                                               \
        "v_cndmask_b32_sdwa %[xa], %[p], %[p], vcc dst_sel:BYTE_1 dst_unused:UNUSED_PRESERVE src0_sel:BYTE_0 "      \
        "src1_sel:BYTE_1\n\t"                                                                                       \
        "v_cndmask_b32 %[s], %[l], %[r], vcc"                                                                       \
        : [d] "=&v"(d), [xa] "+v"(xa), [s] "=&v"(sel)                                                               \
        : [c] "v"(c), [w] "v"(w), [p] "v"(p), [l] "v"(l), [r] "v"(r)                                                \
        : "vcc")
template <int CSEL = 0>
__device__ __forceinline__ void decide(uint32_t c, uint32_t w, uint32_t p, uint32_t l, uint32_t r, uint32_t &xa,
                                       uint32_t &sel) {
    uint32_t d;
    if constexpr (CSEL == 0)
        HARL_B16_DECIDE("DWORD");
    else if constexpr (CSEL == 1)
        HARL_B16_DECIDE("WORD_0");
    else
        HARL_B16_DECIDE("WORD_1");
}
#undef HARL_B16_DECIDE

// acc + leaf, kept where it stands (before the next leaf load into the same register): moved to the
// end of a tree's walk, it kept the previous leaf alive past the new load, and the register copy at
// the loop's back edge then waited for every load in flight, the next trees' prefetch included.
__device__ __forceinline__ float add_pinned(float acc, float leaf) {
    float r;
    asm volatile("v_add_f32 %0, %1, %2" : "=v"(r) : "v"(acc), "v"(leaf));
    return r;
}

// Writes feature fv (its byte 0) into byte 1 of the code address xa, keeping the row bits.
__device__ __forceinline__ void set_feature(uint32_t &xa, uint32_t fv) {
    asm("v_mov_b32_sdwa %[xa], %[f] dst_sel:BYTE_1 dst_unused:UNUSED_PRESERVE src0_sel:BYTE_0" : [xa] "+v"(xa)
        : [f] "v"(fv));
}

// The decision at a node of level D-2 from its tail record r = {word, children's features, left
// child's word, right child's word}: writes the child's feature into byte 1 of xa, returns the
// child's word in cw and j' = jj + (go right) in cj (jj = 2j for the level D-2 node j, so that j' is
// the child's index in the last level).  The carry of the add is the decision itself.  CSEL as for
// decide.
#define HARL_B16_DECIDE_D2(CSEL)                                                                                    \
    asm("v_sub_u32_sdwa %[d], %[c], %[w] dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:" CSEL " src1_sel:WORD_0\n\t" \
        "v_cmp_le_u32_sdwa vcc, %[d], %[w] src0_sel:DWORD src1_sel:WORD_1\n\t"                                     \
        "s_nop 1\n\t"                                                                                               \
        "v_cndmask_b32_sdwa %[xa], %[p], %[p], vcc dst_sel:BYTE_1 dst_unused:UNUSED_PRESERVE src0_sel:BYTE_0 "      \
        "src1_sel:BYTE_1\n\t"                                                                                       \
        "v_cndmask_b32 %[cw], %[l], %[r], vcc\n\t"                                                                  \
        "v_addc_co_u32 %[cj], vcc, 0, %[jj], vcc"                                                                   \
        : [d] "=&v"(d), [xa] "+v"(xa), [cw] "=&v"(cw), [cj] "=&v"(cj)                                               \
        : [c] "v"(c), [w] "v"(r.x), [p] "v"(r.y), [l] "v"(r.z), [r] "v"(r.w), [jj] "v"(jj)                          \
        : "vcc")
template <int CSEL>
__device__ __forceinline__ void decide_d2(uint32_t c, const uint4 &r, uint32_t jj, uint32_t &xa, uint32_t &cw,
                                          uint32_t &cj) {
    uint32_t d;
    if constexpr (CSEL == 1)
        HARL_B16_DECIDE_D2("WORD_0");
    else
        HARL_B16_DECIDE_D2("WORD_1");
}
#undef HARL_B16_DECIDE_D2

// Last level: 8 j + (go right ? 4 : 0), the byte offset of the leaf reached from last-level node j
// (code c, word w) among the tree's leaves.  CSEL as for decide.
#define HARL_B16_LEAF(CSEL)                                                                                         \
    asm("v_sub_u32_sdwa %[d], %[c], %[w] dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:" CSEL " src1_sel:WORD_0\n\t" \
        "v_cmp_le_u32_sdwa vcc, %[d], %[w] src0_sel:DWORD src1_sel:WORD_1\n\t"                                     \
        "s_nop 1\n\t"                                                                                               \
        "v_cndmask_b32_e64 %[s], 0, 4, vcc"                                                                         \
        : [d] "=&v"(d), [s] "=&v"(s)                                                                                \
        : [c] "v"(c), [w] "v"(w)                                                                                    \
        : "vcc")
template <int CSEL>
__device__ __forceinline__ uint32_t leaf_off(uint32_t c, uint32_t w, uint32_t j) {
    uint32_t d, s;
    if constexpr (CSEL == 1)
        HARL_B16_LEAF("WORD_0");
    else
        HARL_B16_LEAF("WORD_1");
    return 8u * j + s;
}
#undef HARL_B16_LEAF

struct Head {
    uint32_t f, w, p;  // root feature, root word, root's children's features (D >= 2)
};

// Address constants of a wave's slot (tb) for trees of depth D (M = 2^D): the root's children's
// records at tb + 16 and tb + 24; child 2n + g of a record at a is at 2a - tb + 8g; the tail record of
// child g of the level D-3 record at a is at tail byte 4a + 16g - 4 (tb + M).  The walk's v_cndmask
// selects between two VGPR copies: those of the inner levels are made once per kernel, the others
// where they are used (fewer registers live through the walk).
struct SlotConsts {
    uint32_t tb, lt, li, ri;
};
__device__ __forceinline__ SlotConsts slot_consts(uint32_t tb, uint32_t M) {
    return SlotConsts{tb, 0u - 4u * (tb + M), in_vgpr(0u - tb), in_vgpr(8u - tb)};
}

// A tree's last two levels, left for the next walk: per chain the code of its level D-2 node, that
// node's tail record (loaded from global memory, in flight) and jj = 2j for the node's index j in
// its level; lb locates the tree's leaves.
struct Deferred {
    uint32_t x[kRPL], jj[kRPL];
    uint4 r[kRPL];
    const char *lb;
};

// A deferred tree whose leaves are the two floats at `zero` (both 0): the one left before a piece's
// first tree.  Its record {theta 1, U 0 | features 0 | two such words} sends code 0 left, and the
// last level's word sends any code to leaf 0 or 1.
__device__ __forceinline__ void no_deferred(Deferred &d, const float *zero) {
#pragma unroll
    for (int c = 0; c < kRPL; ++c) d.x[c] = 0u, d.jj[c] = 0u, d.r[c] = make_uint4(1u, 0u, 1u, 1u);
    d.lb = reinterpret_cast<const char *>(zero);
}

// The last level of a deferred tree, as left by step_d2: per chain the code and word of its last
// level node and that node's index.
struct LastLevel {
    uint32_t x[kRPL], w[kRPL], j[kRPL];
};

// Level D-2 of the deferred tree d: each chain decides with its record and reads the code of its
// last-level node.
__device__ __forceinline__ void step_d2(const Deferred &d, uint32_t (&xa)[kRPL], LastLevel &e) {
#pragma unroll
    for (int c = 0; c < kRPL; ++c) {
        if (c < 2)
            decide_d2<1>(d.x[c], d.r[c], d.jj[c], xa[c], e.w[c], e.j[c]);
        else
            decide_d2<2>(d.x[c], d.r[c], d.jj[c], xa[c], e.w[c], e.j[c]);
        e.x[c] = lds_b32(xa[c]);
        __builtin_amdgcn_sched_barrier(0);
    }
}

// The last level: each chain's leaf (leaves at lb) is loaded into pend[] after the leaf pending from
// the tree before has been added to acc[].
__device__ __forceinline__ void step_leaf(const LastLevel &e, const char *lb, float (&acc)[kRPL], float (&pend)[kRPL]) {
#pragma unroll
    for (int c = 0; c < kRPL; ++c) {
        const uint32_t o = c < 2 ? leaf_off<1>(e.x[c], e.w[c], e.j[c]) : leaf_off<2>(e.x[c], e.w[c], e.j[c]);
        acc[c] = add_pinned(acc[c], pend[c]);
        __builtin_amdgcn_sched_barrier(0);
        pend[c] = *reinterpret_cast<const float *>(lb + o);
    }
}

// Finish the deferred tree d (the last one of a piece): its last two levels.
__device__ __forceinline__ void finish(const Deferred &d, uint32_t (&xa)[kRPL], float (&acc)[kRPL],
                                       float (&pend)[kRPL]) {
    LastLevel e;
    step_d2(d, xa, e);
    step_leaf(e, d.lb, acc, pend);
}

// Walk one tree (slot at LDS address tb, depth D >= 5 at run time) for this lane's kRPL rows, down
// to level D-3, the last level whose records the slot holds; xa[j] is the LDS address of the dword
// that holds row j's code (its low half for j < 2, its high half for j >= 2), whose byte 1 (the
// feature) each level rewrites.  The rows are independent chains: each takes
// its step of a level in turn, so the reads of the others are in flight while one decides.  The
// tree's tail is at gl: M/4 records of 16 bytes for level D-2, then the M leaves.  Level D-2 and the
// last level are left in d for the next walk: it first takes the previous tree's (or
// no_deferred's) level D-2 after its own root level and that tree's last level after its own level
// 1, so that the records and leaves loaded from the tails have a whole walk to arrive.
__device__ __forceinline__ void walk(uint32_t tb, int D, const SlotConsts &k, const Head &h, uint32_t (&xa)[kRPL],
                                     float (&acc)[kRPL], const float *__restrict__ gl, float (&pend)[kRPL],
                                     Deferred &d) {
    const uint32_t M = 1u << D;
    uint32_t x[kRPL], a[kRPL];
    uint2 rec[kRPL];
    // the root: chains j and j + 2 read the two halves of one dword of the root's feature
    const uint32_t hf = in_vgpr(h.f);
    uint32_t x01[2];
#pragma unroll
    for (int c = 0; c < 2; ++c) {
        set_feature(xa[c], hf);
        x01[c] = lds_b32(xa[c]);
    }
    const uint32_t hw = in_vgpr(h.w), hp = in_vgpr(h.p), l0 = in_vgpr(k.tb + 16u), r0 = in_vgpr(k.tb + 24u);
#pragma unroll
    for (int c = 0; c < kRPL; ++c) {
        uint32_t s;
        if (c < 2)
            decide<1>(x01[c & 1], hw, hp, l0, r0, xa[c], s);
        else
            decide<2>(x01[c & 1], hw, hp, l0, r0, xa[c], s);
        x[c] = lds_b32(xa[c]);
        a[c] = s;
        rec[c] = lds_b64(s);
        __builtin_amdgcn_sched_barrier(0);
    }
    LastLevel e;
    step_d2(d, xa, e);
    // levels 1 .. D-4, the previous tree's last level after level 1
    auto inner = [&]() {
#pragma unroll
        for (int c = 0; c < kRPL; ++c) {
            uint32_t s;
            if (c < 2)
                decide<1>(x[c], rec[c].x, rec[c].y, k.li, k.ri, xa[c], s);
            else
                decide<2>(x[c], rec[c].x, rec[c].y, k.li, k.ri, xa[c], s);
            x[c] = lds_b32(xa[c]);
            a[c] = 2u * a[c] + s;
            rec[c] = lds_b64(a[c]);
            __builtin_amdgcn_sched_barrier(0);
        }
    };
    inner();
    step_leaf(e, d.lb, acc, pend);
    for (int lvl = 2; lvl + 3 < D; ++lvl) inner();
    // level D-3 into level D-2: the D-3 record of node m at a = tb + 8m, its child n = 2m + g has its
    // tail record at byte 16 (n - M/4) = 4a + 16g - 4 (tb + M)
    const char *__restrict__ tail = reinterpret_cast<const char *>(gl);
    const uint32_t lt = in_vgpr(k.lt), rt = in_vgpr(k.lt + 16u);
#pragma unroll
    for (int c = 0; c < kRPL; ++c) {
        uint32_t s;
        if (c < 2)
            decide<1>(x[c], rec[c].x, rec[c].y, lt, rt, xa[c], s);
        else
            decide<2>(x[c], rec[c].x, rec[c].y, lt, rt, xa[c], s);
        d.x[c] = lds_b32(xa[c]);
        const uint32_t o = 4u * a[c] + s;
        d.r[c] = *reinterpret_cast<const uint4 *>(tail + o);
        d.jj[c] = o >> 3;
        __builtin_amdgcn_sched_barrier(0);
    }
    d.lb = tail + 4u * M;  // the leaves follow the M/4 records of 16 bytes
}

// LDS placement of a workgroup's tree slots: n_a slots of `sb` bytes after row group 0 (from byte
// 256 F up to 65536), the rest after row group 1 (from 65536 + 256 F); the row sums of a piece
// reuse the second area, and two progress counters follow whichever of slots and sums is longer.
struct SlotPlan {
    int n_a;
    uint32_t a0, b0, progress, lds;
};
__host__ __device__ __forceinline__ SlotPlan slot_plan(int F, int tw, uint32_t sb) {
    SlotPlan p{};
    p.a0 = 256u * (uint32_t)F;
    p.b0 = kGroupStride + 256u * (uint32_t)F;
    const int fit_a = (int)((kGroupStride - p.a0) / sb);
    p.n_a = fit_a < tw ? fit_a : tw;
    const uint32_t slots_b = (uint32_t)(tw - p.n_a) * sb, red = (uint32_t)tw * kRT * 8u;
    p.progress = p.b0 + (slots_b > red ? slots_b : red);
    p.lds = p.progress + 16u;
    return p;
}

}  // namespace b16
}  // namespace harl
