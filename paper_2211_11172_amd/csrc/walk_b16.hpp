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
__device__ __forceinline__ uint32_t lds_u16(uint32_t a) {
    return *(const __attribute__((address_space(3))) uint16_t *)(uintptr_t)a;
}
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
// the SDWA select reads it (two wait states between them).
__device__ __forceinline__ void decide(uint32_t c, uint32_t w, uint32_t p, uint32_t l, uint32_t r, uint32_t &xa,
                                       uint32_t &sel) {
    uint32_t d;
    asm("v_sub_u32_sdwa %[d], %[c], %[w] dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:DWORD src1_sel:WORD_0\n\t"
        "v_cmp_le_u32_sdwa vcc, %[d], %[w] src0_sel:DWORD src1_sel:WORD_1\n\t"
        "s_nop 1\n\t"
        "v_cndmask_b32_sdwa %[xa], %[p], %[p], vcc dst_sel:BYTE_1 dst_unused:UNUSED_PRESERVE src0_sel:BYTE_0 src1_sel:BYTE_1\n\t"
        "v_cndmask_b32 %[s], %[l], %[r], vcc"
        : [d] "=&v"(d), [xa] "+v"(xa), [s] "=&v"(sel)
        : [c] "v"(c), [w] "v"(w), [p] "v"(p), [l] "v"(l), [r] "v"(r)
        : "vcc");
}

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

// Last level: 2 a + (go right ? 4 : 0) for the last-level node whose word is at tail byte
// a - tb - 2M (walk).
__device__ __forceinline__ uint32_t leaf_off(uint32_t c, uint32_t w, uint32_t a) {
    uint32_t d, s;
    asm("v_sub_u32_sdwa %[d], %[c], %[w] dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:DWORD src1_sel:WORD_0\n\t"
        "v_cmp_le_u32_sdwa vcc, %[d], %[w] src0_sel:DWORD src1_sel:WORD_1\n\t"
        "s_nop 1\n\t"
        "v_cndmask_b32_e64 %[s], 0, 4, vcc"
        : [d] "=&v"(d), [s] "=&v"(s)
        : [c] "v"(c), [w] "v"(w)
        : "vcc");
    return 2u * a + s;
}

struct Head {
    uint32_t f, w, p;  // root feature, root word, root's children's features (D >= 2)
};

// Address constants of a wave's slot (tb) for trees of depth D, as VGPR copies made once per kernel
// (the walk's v_cndmask selects between two of them): the root's children's records at tb + 16 and
// tb + 24; child 2n + g of a record at a is at 2a - tb + 8g; the last-level word of the child g of
// the level D-2 record at a is at byte a + 4g of the tree's tail shifted back by tb + 2M.
struct SlotConsts {
    uint32_t l0, r0, li, ri, lt, rt;
};
__device__ __forceinline__ SlotConsts slot_consts(uint32_t tb) {
    return SlotConsts{in_vgpr(tb + 16u), in_vgpr(tb + 24u), in_vgpr(0u - tb), in_vgpr(8u - tb), in_vgpr(0u), in_vgpr(4u)};
}

// A tree's last level, left for the next walk: per chain the code of the last-level node, its word
// (loaded from the tail, in flight) and a, its word's tail byte plus tb + 2M; lb locates the
// leaves (leaf byte lb + 2a + 4g).
struct LastLevel {
    uint32_t x[kRPL], w[kRPL], a[kRPL];
    const char *lb;
};

// A last level that loads the float at `zero` (which holds 0) for every chain: the one left before
// a piece's first tree.
__device__ __forceinline__ void no_last_level(LastLevel &d, const float *zero) {
#pragma unroll
    for (int c = 0; c < kRPL; ++c) d.x[c] = 0u, d.w[c] = 1u, d.a[c] = 0u;  // code 0 < theta 1: offset 0
    d.lb = reinterpret_cast<const char *>(zero);
}

// The last level of tree d: each chain's leaf is loaded into pend[] after the leaf pending from the
// tree before has been added to acc[].
__device__ __forceinline__ void finish(const LastLevel &d, float (&acc)[kRPL], float (&pend)[kRPL]) {
#pragma unroll
    for (int c = 0; c < kRPL; ++c) {
        const uint32_t o = leaf_off(d.x[c], d.w[c], d.a[c]);
        acc[c] = add_pinned(acc[c], pend[c]);
        __builtin_amdgcn_sched_barrier(0);
        pend[c] = *reinterpret_cast<const float *>(d.lb + o);
    }
}

// Walk one tree (slot at LDS address tb, depth D >= 3 at run time) for this lane's kRPL rows, down
// to its last split level; xa[j] is the LDS address of row j's code, whose byte 1 (the feature) each
// level rewrites.  The rows are independent chains: each takes its step of a level in turn, so the
// reads of the others are in flight while one decides.  The tree's tail is at gl (the M/2 last-level
// words, then the M leaves).  The last level's words are loaded from the tail and the level itself
// is left in d: the walk first finishes the previous tree's (or no_last_level's), after its own
// root level, so that the words have a whole walk to arrive.
__device__ __forceinline__ void walk(uint32_t tb, int D, const SlotConsts &k, const Head &h, uint32_t (&xa)[kRPL],
                                     float (&acc)[kRPL], const float *__restrict__ gl, float (&pend)[kRPL],
                                     LastLevel &d) {
    const uint32_t M = 1u << D;
    uint32_t x[kRPL], a[kRPL];
    uint2 rec[kRPL];
    const uint32_t hf = in_vgpr(h.f);
#pragma unroll
    for (int c = 0; c < kRPL; ++c) {
        set_feature(xa[c], hf);
        x[c] = lds_u16(xa[c]);
    }
    const uint32_t hw = in_vgpr(h.w), hp = in_vgpr(h.p);
#pragma unroll
    for (int c = 0; c < kRPL; ++c) {
        uint32_t s;
        decide(x[c], hw, hp, k.l0, k.r0, xa[c], s);
        x[c] = lds_u16(xa[c]);
        a[c] = s;
        rec[c] = lds_b64(s);
        __builtin_amdgcn_sched_barrier(0);
    }
    finish(d, acc, pend);
    // levels 1 .. D-3
    for (int lvl = 1; lvl + 2 < D; ++lvl) {
#pragma unroll
        for (int c = 0; c < kRPL; ++c) {
            uint32_t s;
            decide(x[c], rec[c].x, rec[c].y, k.li, k.ri, xa[c], s);
            x[c] = lds_u16(xa[c]);
            a[c] = 2u * a[c] + s;
            rec[c] = lds_b64(a[c]);
            __builtin_amdgcn_sched_barrier(0);
        }
    }
    // level D-2 into the last level: the D-2 record of node i at a = tb + 8i, its child M/2 + j
    // (j = 2i + g - M/2) has its word at tail byte 4j = a + 4g - tb - 2M
    const char *__restrict__ wb = reinterpret_cast<const char *>(gl) - (tb + 2u * M);
#pragma unroll
    for (int c = 0; c < kRPL; ++c) {
        uint32_t s;
        decide(x[c], rec[c].x, rec[c].y, k.lt, k.rt, xa[c], s);
        d.x[c] = lds_u16(xa[c]);
        d.a[c] = a[c] + s;
        d.w[c] = *reinterpret_cast<const uint32_t *>(wb + d.a[c]);
        __builtin_amdgcn_sched_barrier(0);
    }
    // last-level node M/2 + j's leaves are at tail byte 2M + 8j, and 2 (a + 4g) = 8j + 2tb + 4M:
    // leaf byte = lb + 2 (a + 4g) + 4g' with lb = tail - 2tb - 2M
    d.lb = reinterpret_cast<const char *>(gl) - (2u * tb + 2u * M);
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
