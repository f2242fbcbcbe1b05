// Actor/critic forward of one search round (HARL paper, Algorithm 1: select the modifications M
// with pi_theta(M|S); the critic V(S) of Eq. 6; Section 4.3).  Shared trunk
// h1 = ReLU(W1 s + b1), h2 = ReLU(W2 h1 + b2); actor head logits = Wa h2 + ba; value head
// v = wv . h2 + bv; action = lowest-index argmax of the logits; probs = softmax(logits).
//
// K4 k_policy: the three dense contractions run on MFMA, transposed so that states are the MFMA
// N dimension (H^T = W X^T).  A workgroup holds 16*NSG states and U waves; a wave computes its
// share of each layer's 16-unit tiles in groups of TP tiles.
//   start    every wave issues the global loads its first tile groups need up front (states,
//            biases, the first W1 fragments into a register ring; the first W2 fragments into a
//            second ring during phase 1, behind its MFMAs), so that the kernel waits on memory
//            latency about once rather than once per phase;
//   phase 0  the biases and the states are staged into LDS (activation layout below);
//   phase 1  each wave computes its 1/U of h1's tiles for all states, TP tiles at a time (A =
//            W1 fragments streamed from global memory through the register ring, B = states
//            from LDS, read one k-group ahead), applies bias + ReLU (+ bf16 rounding) and stores
//            the tiles to LDS;
//   phase 2  each wave computes its 1/U of h2's tiles the same way (B = h1 from LDS; every A
//            fragment feeds NSG state groups) and feeds each finished tile straight from its
//            accumulator registers into the head contraction: the MFMA result layout of a tile is
//            re-used as the B operand layout, with the head weights pre-permuted to match;
//   phase 3  each wave takes whole states: the U per-wave partial heads of a state are summed in
//            a fixed order with the bias, and argmax, softmax and value computed and written out.
// fp32 policies use v_mfma_f32_16x16x4_f32, bf16 policies v_mfma_f32_16x16x32_bf16 (fp32
// accumulation; h1, h2 rounded to bf16, nearest even).  Weights are pre-tiled at create time so
// that a lane's operand for one "k-group" is 16 contiguous bytes:
//   fp32: a k-group is 16 input units = 4 MFMAs; lane l, slot j (j < 4) holds unit 16g + 4(l/16) + j
//   bf16: a k-group is 32 input units = 1 MFMA;  lane l, slot j (j < 8) holds unit 32g + 8(l/16) + j
// Fragments are stored k-group-major ([g][tile][lane] x 16 B): the waves of a workgroup, which own
// different tiles, read one contiguous stretch of the layer's weights at a time, spread evenly over
// the cache channels.
//
// Activations in LDS are kept as 16-byte "unit blocks" (4 fp32 or 8 bf16 consecutive units of one
// state), stored [unit block][state]: unit u of state s is at byte ((u / UB) NS + s) 16 + (u % UB) EL
// (UB units per block, NS states per workgroup, EL bytes per element).  The B operand of k-group g
// for the state group sg is then unit block 4g + l/16 of state 16 sg + l%16, so the 64 lanes read
// 1 KB of consecutive bytes (no bank conflicts), and the finished h1 tiles are written back the same
// way.
//
// MFMA operand layouts (lane l of 64; i indexes the 4 accumulator registers):
//   16x16x4  f32 : A[m = l%16][k = l/16],          B[k = l/16][n = l%16]
//   16x16x32 bf16: A[m = l%16][k = 8(l/16) + j],   B[k = 8(l/16) + j][n = l%16],  j = 0..7
//   result       : D[m = 4(l/16) + i][n = l%16]
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <type_traits>
#include <vector>

#include "internal.hpp"

namespace harl {
namespace {

constexpr int kMaxU = 8;      // waves per workgroup (at most)
constexpr int kRing = 4;      // k-groups of W1 fragments in flight per wave (W2: the launch table)
constexpr int kHiddenPad = 256;  // hidden widths padded to whole tile groups of every kernel shape
constexpr int kX32MinBatch = 16384;  // bf16 batches from this size use k_policy_x32 (policy_x32.hip)

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

__device__ __forceinline__ uint32_t bf16_rne(float x) {
    // fp32 -> bf16 bits, nearest even (finite inputs: activations after ReLU)
    uint32_t b = __float_as_uint(x);
    b += 0x7FFFu + ((b >> 16) & 1u);
    return b >> 16;
}

__device__ __forceinline__ bf16x8 as_bf16x8(uint4 v) {
    bf16x8 r;
    __builtin_memcpy(&r, &v, 16);
    return r;
}

// Reductions over groups of 16, 32 or 64 lanes without LDS round trips: DPP moves pair the lanes of
// each row of 16 (xor 1, xor 2, half-row mirror, row mirror), then the gfx950 row swaps pair rows
// 2k and 2k+1 (v_permlane16_swap) and the two halves of the wave (v_permlane32_swap).  Every step
// pairs each lane with one partner and both combine the same two values in the same order, so all
// lanes of a group end with the same bits.
template <int CTRL>
__device__ __forceinline__ unsigned dpp(unsigned v) {
    return __builtin_amdgcn_mov_dpp(v, CTRL, 0xF, 0xF, false);
}
constexpr int kDppXor1 = 0xB1, kDppXor2 = 0x4E, kDppHalfMirror = 0x141, kDppMirror = 0x140;

// (value, index) with the larger value, the lower index among equal values; NaN values never win
__device__ __forceinline__ void argmax_step(float &best, int &best_i, float ov, int oi) {
    const bool take = (ov > best) | ((ov == best) & (oi < best_i));
    best = take ? ov : best;
    best_i = take ? oi : best_i;
}

// the two values a lane sees after the row swap of span 16 or 32: the lower group's, the upper's
template <int SPAN>
__device__ __forceinline__ void swap_pair(unsigned v, unsigned &lo, unsigned &hi) {
    const auto r = SPAN == 16 ? __builtin_amdgcn_permlane16_swap(v, v, false, false)
                              : __builtin_amdgcn_permlane32_swap(v, v, false, false);
    lo = r[0];
    hi = r[1];
}

template <int CTRL>
__device__ __forceinline__ void argmax_dpp(float &best, int &best_i) {
    argmax_step(best, best_i, __uint_as_float(dpp<CTRL>(__float_as_uint(best))), (int)dpp<CTRL>((unsigned)best_i));
}

template <int SPAN>
__device__ __forceinline__ void argmax_swap(float &best, int &best_i) {
    unsigned vl, vh, il, ih;
    swap_pair<SPAN>(__float_as_uint(best), vl, vh);
    swap_pair<SPAN>((unsigned)best_i, il, ih);
    best = __uint_as_float(vl);
    best_i = (int)il;
    argmax_step(best, best_i, __uint_as_float(vh), (int)ih);
}

// lowest-index maximum over each group of `width` lanes (16, 32 or 64; uniform)
__device__ __forceinline__ void group_argmax(float &best, int &best_i, int width) {
    argmax_dpp<kDppXor1>(best, best_i);
    argmax_dpp<kDppXor2>(best, best_i);
    argmax_dpp<kDppHalfMirror>(best, best_i);
    argmax_dpp<kDppMirror>(best, best_i);
    if (width >= 32) argmax_swap<16>(best, best_i);
    if (width >= 64) argmax_swap<32>(best, best_i);
}

template <int SPAN>
__device__ __forceinline__ float sum_swap(float x) {
    unsigned lo, hi;
    swap_pair<SPAN>(__float_as_uint(x), lo, hi);
    return __uint_as_float(lo) + __uint_as_float(hi);
}

// sum over each group of `width` lanes (16, 32 or 64; uniform)
__device__ __forceinline__ float group_sum(float x, int width) {
    x += __uint_as_float(dpp<kDppXor1>(__float_as_uint(x)));
    x += __uint_as_float(dpp<kDppXor2>(__float_as_uint(x)));
    x += __uint_as_float(dpp<kDppHalfMirror>(__float_as_uint(x)));
    x += __uint_as_float(dpp<kDppMirror>(__float_as_uint(x)));
    if (width >= 32) x = sum_swap<16>(x);
    if (width >= 64) x = sum_swap<32>(x);
    return x;
}

__device__ __forceinline__ float word(const uint4 &v, int q) {
    return __uint_as_float(q == 0 ? v.x : q == 1 ? v.y : q == 2 ? v.z : v.w);
}

template <bool BF16>
__device__ __forceinline__ void mfma_group(const uint4 &a, const uint4 &b, f32x4 &acc) {
    if constexpr (BF16) {
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(a), as_bf16x8(b), acc, 0, 0, 0);
    } else {
        acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.x), __uint_as_float(b.x), acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.y), __uint_as_float(b.y), acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.z), __uint_as_float(b.z), acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.w), __uint_as_float(b.w), acc, 0, 0, 0);
    }
}

struct PolicyArgs {
    const void *states;
    int B, S;
    int sp, h1p, h2p, hap, a;
    const uint4 *w1, *w2, *wh;
    const float *b1, *b2, *bh;
    int32_t *action;
    float *value, *probs, *logits;
};

// The weight loads of the layer loops are unconditional (a layer's last round is a separate copy
// that issues none, and the head fragments of absent head tiles are read from a valid tile and
// never used): the compiler then knows how many loads follow each one and waits for exactly the
// one it needs, instead of draining every load in flight.

// The A fragments of a layer's first RING iterations (k-groups 0 .. RING - 1 of the wave's first
// tile group; RING <= KG), loaded before the layer starts so that their latency overlaps the work
// before it.
template <int TP, int RING>
__device__ __forceinline__ void ring_fill(uint4 (&ring)[RING][TP], const uint4 *__restrict__ A, int NT, int t0, int l) {
#pragma unroll
    for (int r = 0; r < RING; ++r) {
        const uint4 *src = A + ((int64_t)r * NT + t0) * 64 + l;
#pragma unroll
        for (int j = 0; j < TP; ++j) ring[r][j] = src[j * 64];
    }
}

// One dense layer for this wave: `n_tiles` output tiles of 16 units starting at tile `t0`, each a
// sum over KG k-groups (KG a multiple of RING), computed TP tiles at a time (TP independent
// accumulator chains sharing every B fragment).  The wave's iterations (tile group, k-group) run
// in order; `ring` holds the A fragments of the first RING iterations (ring_fill), and those of
// iteration it + RING are loaded from `A` (packed [g][tile][lane] x 16 B, NT tiles per k-group)
// into ring slot it % RING as soon as iteration it has issued its MFMAs; the B fragments of the
// next k-group are read from the LDS activation blocks `in` into the other half of a double
// buffer.  done(first_tile, acc[TP][NSG]) consumes each finished group.  side(r) issues part r
// (r < RING) of loads meant for later work: a layer of one round issues part r right behind the
// MFMAs of its iteration r, so that the loads drain through the memory pipeline while the MFMAs run
// (issued all at once, they held the waves' instruction issue back for about 0.8 us); any other
// layer issues all parts before its first round.
template <bool BF16, int NSG, int TP, int RING, bool ONE_ROUND_COPY, typename Done, typename Side>
__device__ __forceinline__ void dense_layer(uint4 (&ring)[RING][TP], const uint4 *__restrict__ A, int NT, int t0,
                                            int n_tiles, int KG, const char *in, int ln, int lq, int l, Done done,
                                            Side side) {
    static_assert(RING % 2 == 0, "the B double buffer alternates with the ring slot");
    constexpr int NS = 16 * NSG;
    const int n_groups = n_tiles / TP;
    auto b_load = [&](int g, uint4 (&b)[NSG]) {
#pragma unroll
        for (int sg = 0; sg < NSG; ++sg)
            b[sg] = *reinterpret_cast<const uint4 *>(in + ((g * 4 + lq) * NS + sg * 16 + ln) * 16);
    };
    uint4 b[2][NSG];
    b_load(0, b[0]);
    f32x4 acc[TP][NSG];
    // One round: RING iterations (k-groups g0 .. g0 + RING - 1 of tile group grp).  Every round but
    // the layer's last refills its ring slots with the fragments of the next round (k-groups
    // g0 + RING + r, or r of the next tile group: KG is a multiple of RING) and reads the B
    // fragments one k-group ahead; the last round issues neither, so that no load is left in
    // flight when the layer ends.  The two cases are separate copies of the round, so that every
    // load in either is unconditional and the compiler knows exactly which one each use waits for.
    auto round = [&](int grp, int g0, auto refill_tag, auto side_tag) {
        constexpr bool REFILL = decltype(refill_tag)::value;
        constexpr bool SIDE = decltype(side_tag)::value;
        const bool wrap = g0 + RING >= KG;
        const uint4 *rsrc = A + ((int64_t)(wrap ? 0 : g0 + RING) * NT + t0 + TP * (grp + wrap)) * 64 + l;
#pragma unroll
        for (int r = 0; r < RING; ++r) {
            const int g = g0 + r;
            if (REFILL || r + 1 < RING) b_load(g + 1 == KG ? 0 : g + 1, b[(r + 1) & 1]);
            // the next k-group's B read stays ahead of this k-group's MFMAs (the double buffer)
            __builtin_amdgcn_sched_barrier(0);
            if constexpr (BF16) {
#pragma unroll
                for (int sg = 0; sg < NSG; ++sg)
#pragma unroll
                    for (int j = 0; j < TP; ++j) mfma_group<true>(ring[r][j], b[r & 1][sg], acc[j][sg]);
            } else {
                // the 4 k-steps outermost: consecutive MFMAs feed different accumulators
#pragma unroll
                for (int q = 0; q < 4; ++q)
#pragma unroll
                    for (int sg = 0; sg < NSG; ++sg)
#pragma unroll
                        for (int j = 0; j < TP; ++j)
                            acc[j][sg] = __builtin_amdgcn_mfma_f32_16x16x4f32(word(ring[r][j], q), word(b[r & 1][sg], q),
                                                                              acc[j][sg], 0, 0, 0);
            }
            if constexpr (REFILL) {
                const uint4 *src = rsrc + (int64_t)r * NT * 64;
#pragma unroll
                for (int j = 0; j < TP; ++j) ring[r][j] = src[j * 64];
            }
            if constexpr (SIDE) side(r);
            // keep each refill right behind the MFMAs of its slot (left alone, the scheduler sinks
            // all refills of a round to its end, and the next round then waits on them at once)
            __builtin_amdgcn_sched_barrier(0);
        }
    };
    auto zero = [&]() {
#pragma unroll
        for (int h = 0; h < TP; ++h)
#pragma unroll
            for (int sg = 0; sg < NSG; ++sg) acc[h][sg] = f32x4{0, 0, 0, 0};
    };
    zero();
    const int n_rounds = n_groups * (KG / RING);
    if (ONE_ROUND_COPY && n_rounds == 1) {
        // a layer of one round gets a copy of its own, whose waits count the loads issued before
        // the layer (after the merge with the loop below, the compiler would assume the fewest and
        // wait for loads issued after the layer's own, such as the next layer's first fragments)
        round(0, 0, std::false_type{}, std::true_type{});
        done(t0, acc);
        return;
    }
#pragma unroll
    for (int r = 0; r < RING; ++r) side(r);
    // all rounds but the last in one loop, the last one peeled off after it
    int grp = 0, g0 = 0;
    for (int rr = n_rounds - 1; rr > 0; --rr) {
        round(grp, g0, std::true_type{}, std::false_type{});
        g0 += RING;
        if (g0 == KG) {
            done(t0 + grp * TP, acc);
            zero();
            g0 = 0;
            ++grp;
        }
    }
    round(grp, g0, std::false_type{}, std::false_type{});
    done(t0 + grp * TP, acc);
}

// U waves per workgroup, 16*NSG states; HTM >= head tiles; layers in groups of TP tiles per wave;
// R1 (R2) k-groups of W1 (W2) fragments in flight per wave.
template <bool BF16, int NSG, int HTM, int U, int TP, int R1, int R2>
__global__ __launch_bounds__(64 * U) void k_policy(PolicyArgs p) {
    extern __shared__ __align__(16) char smem[];
    constexpr int EL = BF16 ? 2 : 4;        // bytes per activation element
    constexpr int UB = 16 / EL;             // units per 16-byte unit block
    constexpr int UPG = 4 * UB;             // input units per k-group
    constexpr int NTH = 64 * U;
    const int wid = threadIdx.x / 64, l = threadIdx.x % 64;
    const int ln = l % 16, lq = l / 16;
    const int s0 = blockIdx.x * 16 * NSG;
    constexpr int NS = 16 * NSG;
    // LDS: the biases (b1, b2, heads), then the activations (states, h1), whose space the partial
    // heads take over in phase 3
    float *b1s = reinterpret_cast<float *>(smem);
    float *b2s = b1s + p.h1p;
    float *bhs = b2s + p.h2p;
    char *acts = smem + (p.h1p + p.h2p + p.hap) * 4;
    char *xs = acts;
    char *h1 = acts + NS * p.sp * EL;
    const int HT = p.hap / 16;
    const int NT1 = p.h1p / 16, NT2 = p.h2p / 16;
    const int mt1 = NT1 / U, mt2 = NT2 / U;
    // The global loads the first tile groups need are issued up front, so that the kernel waits
    // for memory about once: the states and biases (staged by phase 0; issued first, so that phase
    // 0 waits for them alone) and the first W1 fragments (register ring) now, the first W2
    // fragments during phase 1 (see dense_layer's side loads), the first head fragments when phase
    // 2 starts (they are needed when its first tile group ends).
    constexpr int PRE = 4;   // state elements per thread loaded up front (the rest: phase 0 loop)
    constexpr int PREB = 2;  // bias float4s per thread loaded up front
    using SE = typename std::conditional<BF16, uint16_t, float>::type;
    const SE *states = static_cast<const SE *>(p.states);
    const int n_st = NS * p.sp;
    SE sv[PRE];
#pragma unroll
    for (int k = 0; k < PRE; ++k) {
        const int e = threadIdx.x + k * NTH;
        const int r = e % NS, c = e / NS;
        const bool ok = e < n_st && s0 + r < p.B && c < p.S;
        sv[k] = states[ok ? (int64_t)(s0 + r) * p.S + c : 0];
    }
    const int nb4 = (p.h1p + p.h2p + p.hap) / 4;
    auto bias_src = [&](int e4) {
        e4 = e4 < nb4 ? e4 : nb4 - 1;
        const int q1 = p.h1p / 4, q2 = q1 + p.h2p / 4;
        const float *src = e4 < q1 ? p.b1 + 4 * e4 : e4 < q2 ? p.b2 + 4 * (e4 - q1) : p.bh + 4 * (e4 - q2);
        return *reinterpret_cast<const float4 *>(src);
    };
    float4 bv4[PREB];
#pragma unroll
    for (int k = 0; k < PREB; ++k) bv4[k] = bias_src(threadIdx.x + k * NTH);
    uint4 ring1[R1][TP], ring2[R2][TP];
    ring_fill<TP, R1>(ring1, p.w1, NT1, wid * mt1, l);
    // head fragments: fp32 one k-group per h2 tile, bf16 one per pair of tiles
    const int HKG = BF16 ? p.h2p / 32 : p.h2p / 16;
    constexpr int HPG = BF16 ? TP / 2 : TP;  // head k-groups per group of TP tiles
    uint4 hpf[HPG][HTM];
    auto head_fetch = [&](int tile) {
        const int hk0 = BF16 ? tile / 2 : tile;
#pragma unroll
        for (int q = 0; q < HPG; ++q)
#pragma unroll
            for (int ht = 0; ht < HTM; ++ht) {
                const int hk = hk0 + q < HKG ? hk0 + q : HKG - 1, hs = ht < HT ? ht : HT - 1;
                hpf[q][ht] = p.wh[((int64_t)hs * HKG + hk) * 64 + l];
            }
    };

    // ------ phase 0: biases -> LDS; states -> LDS unit blocks (zero beyond S and B), state fastest ------
#pragma unroll
    for (int k = 0; k < PREB; ++k) {
        const int e4 = threadIdx.x + k * NTH;
        if (e4 < nb4) reinterpret_cast<float4 *>(b1s)[e4] = bv4[k];
    }
    for (int e4 = threadIdx.x + PREB * NTH; e4 < nb4; e4 += NTH) reinterpret_cast<float4 *>(b1s)[e4] = bias_src(e4);
    auto put_state = [&](int e, SE v) {
        const int r = e % NS, c = e / NS;
        *reinterpret_cast<SE *>(xs + ((c / UB) * NS + r) * 16 + (c % UB) * EL) = v;
    };
#pragma unroll
    for (int k = 0; k < PRE; ++k) {
        const int e = threadIdx.x + k * NTH;
        const int r = e % NS, c = e / NS;
        if (e < n_st) put_state(e, s0 + r < p.B && c < p.S ? sv[k] : SE(0));
    }
    for (int e = threadIdx.x + PRE * NTH; e < n_st; e += NTH) {
        const int r = e % NS, c = e / NS;
        put_state(e, s0 + r < p.B && c < p.S ? states[(int64_t)(s0 + r) * p.S + c] : SE(0));
    }
    __syncthreads();

    // ---------------- phase 1: h1 = act(W1 s + b1), this wave's share of the tiles ----------------
    {
        const int mt_per = mt1;
        dense_layer<BF16, NSG, TP, R1, true>(ring1, p.w1, NT1, wid * mt_per, mt_per, p.sp / UPG, xs, ln, lq, l,
                                         [&](int mt0, f32x4 (&acc)[TP][NSG]) {
#pragma unroll
                                             for (int h = 0; h < TP; ++h) {
                                                 const int u0 = (mt0 + h) * 16 + lq * 4;
                                                 const float4 bias = *reinterpret_cast<const float4 *>(b1s + u0);
                                                 const float bv[4] = {bias.x, bias.y, bias.z, bias.w};
#pragma unroll
                                                 for (int sg = 0; sg < NSG; ++sg) {
                                                     float v[4];
#pragma unroll
                                                     for (int i = 0; i < 4; ++i) v[i] = fmaxf(acc[h][sg][i] + bv[i], 0.f);
                                                     char *dst = h1 + ((u0 / UB) * NS + sg * 16 + ln) * 16 + (u0 % UB) * EL;
                                                     if constexpr (BF16) {
                                                         *reinterpret_cast<uint2 *>(dst) =
                                                             make_uint2(bf16_rne(v[0]) | (bf16_rne(v[1]) << 16),
                                                                        bf16_rne(v[2]) | (bf16_rne(v[3]) << 16));
                                                     } else {
                                                         *reinterpret_cast<float4 *>(dst) = make_float4(v[0], v[1], v[2], v[3]);
                                                     }
                                                 }
                                             }
                                         },
                                         // the first W2 fragments, issued during layer 1
                                         [&](int r) {
                                             static_assert(R2 % R1 == 0, "W2 ring slots per layer-1 iteration");
#pragma unroll
                                             for (int q = 0; q < R2 / R1; ++q) {
                                                 const int slot = r * (R2 / R1) + q;
                                                 const uint4 *src = p.w2 + ((int64_t)slot * NT2 + wid * mt2) * 64 + l;
#pragma unroll
                                                 for (int j = 0; j < TP; ++j) ring2[slot][j] = src[j * 64];
                                             }
                                         });
    }
    __syncthreads();

    // ------- phase 2: h2 tile groups of this wave, chained into the partial heads (registers) -------
    f32x4 hacc[NSG][HTM];
#pragma unroll
    for (int sg = 0; sg < NSG; ++sg)
#pragma unroll
        for (int ht = 0; ht < HTM; ++ht) hacc[sg][ht] = f32x4{0, 0, 0, 0};
    {
        const int mt_per = mt2;
        const int mt_first = wid * mt_per;
        head_fetch(mt_first);
        dense_layer<BF16, NSG, TP, R2, false>(
            ring2, p.w2, NT2, mt_first, mt_per, p.h1p / UPG, h1, ln, lq, l, [&](int mt0, f32x4 (&acc)[TP][NSG]) {
                float bias[TP][4];
#pragma unroll
                for (int h = 0; h < TP; ++h) {
                    const float4 b = *reinterpret_cast<const float4 *>(b2s + (mt0 + h) * 16 + lq * 4);
                    bias[h][0] = b.x; bias[h][1] = b.y; bias[h][2] = b.z; bias[h][3] = b.w;
                }
#pragma unroll
                for (int sg = 0; sg < NSG; ++sg) {
                    float v[TP][4];
#pragma unroll
                    for (int h = 0; h < TP; ++h)
#pragma unroll
                        for (int i = 0; i < 4; ++i) v[h][i] = fmaxf(acc[h][sg][i] + bias[h][i], 0.f);
                    if constexpr (BF16) {
                        // head k-group of tiles (2q, 2q+1): slots 0..3 tile 2q, 4..7 tile 2q+1 (accumulator layout)
#pragma unroll
                        for (int q = 0; q < HPG; ++q) {
                            uint4 bv;
                            bv.x = bf16_rne(v[2 * q][0]) | (bf16_rne(v[2 * q][1]) << 16);
                            bv.y = bf16_rne(v[2 * q][2]) | (bf16_rne(v[2 * q][3]) << 16);
                            bv.z = bf16_rne(v[2 * q + 1][0]) | (bf16_rne(v[2 * q + 1][1]) << 16);
                            bv.w = bf16_rne(v[2 * q + 1][2]) | (bf16_rne(v[2 * q + 1][3]) << 16);
#pragma unroll
                            for (int ht = 0; ht < HTM; ++ht)
                                if (ht < HT) mfma_group<true>(hpf[q][ht], bv, hacc[sg][ht]);
                        }
                    } else {
#pragma unroll
                        for (int h = 0; h < TP; ++h) {
                            const uint4 bv = make_uint4(__float_as_uint(v[h][0]), __float_as_uint(v[h][1]),
                                                        __float_as_uint(v[h][2]), __float_as_uint(v[h][3]));
#pragma unroll
                            for (int ht = 0; ht < HTM; ++ht)
                                if (ht < HT) mfma_group<false>(hpf[h][ht], bv, hacc[sg][ht]);
                        }
                    }
                }
                if (mt0 + TP < mt_first + mt_per) head_fetch(mt0 + TP);
            },
            [](int) {});
    }
    __syncthreads();  // h1 no longer needed: its LDS takes the partial heads

    // ---------------- phase 3: fixed-order sum of the U partial heads, epilogue ----------------
    // The partial heads are stored [U][state][row], rows padded to hap + 4 floats: a lane writes
    // its 4 rows of a head tile as one 16-byte store, and the 16 lanes of a store cycle (16
    // states, stride (hap + 4) / 4 an odd number of 16-byte units) hit disjoint banks.  The waves then take whole states: each pass of a wave takes 64 / W states, W =
    // 16, 32 or 64 lanes per state (the head rows rounded up); lane l sums row l % W (and l % W + 64
    // when a state has more than 64 rows) over the U waves in wave order, adds the bias, and argmax
    // and the softmax sum are reductions over the lanes of a state.
    float *part = reinterpret_cast<float *>(acts);
    const int rs = p.hap + 4;
    const int nz = NS * rs;
#pragma unroll
    for (int sg = 0; sg < NSG; ++sg)
#pragma unroll
        for (int ht = 0; ht < HTM; ++ht)
            if (ht < HT)
                *reinterpret_cast<float4 *>(part + (int64_t)wid * nz + (sg * 16 + ln) * rs + ht * 16 + lq * 4) =
                    make_float4(hacc[sg][ht][0], hacc[sg][ht][1], hacc[sg][ht][2], hacc[sg][ht][3]);
    __syncthreads();
    constexpr int RC = (HTM * 16 + 63) / 64;  // row chunks of 64 per state
    const int rw = p.hap <= 16 ? 16 : p.hap <= 32 ? 32 : 64;
    const int spp = 64 / rw;
    for (int sb = wid * spp; sb < NS; sb += U * spp) {
        const int sl = sb + l / rw, lr = l % rw;
        const int st = s0 + sl;
        float z[RC];
        float best = -INFINITY;
        int best_i = 0x7FFFFFFF;
#pragma unroll
        for (int c = 0; c < RC; ++c) {
            const int row = c * 64 + lr;
            z[c] = 0.f;
            if (row < p.hap) {
                const int v = sl * rs + row;
                float s = 0.f;
#pragma unroll
                for (int w = 0; w < U; ++w) s += part[(int64_t)w * nz + v];
                z[c] = s + bhs[row];
            }
            if (row < p.a) argmax_step(best, best_i, z[c], row);
        }
        group_argmax(best, best_i, rw);
        if (best_i == 0x7FFFFFFF) best_i = 0;  // only NaN logits: no maximum exists
        float e[RC] = {}, sum = 0.f;
        if (p.probs) {
#pragma unroll
            for (int c = 0; c < RC; ++c) {
                e[c] = c * 64 + lr < p.a ? expf(z[c] - best) : 0.f;
                sum += e[c];
            }
            sum = group_sum(sum, rw);
        }
        if (st < p.B) {
#pragma unroll
            for (int c = 0; c < RC; ++c) {
                const int row = c * 64 + lr;
                if (row < p.a) {
                    if (p.logits) p.logits[(int64_t)st * p.a + row] = z[c];
                    if (p.probs) p.probs[(int64_t)st * p.a + row] = e[c] / sum;
                }
                if (row == p.a) p.value[st] = z[c];
            }
            if (lr == 0) p.action[st] = best_i;
        }
    }
}

// ---------------------------------------------------------------------------------------------
// host: weight pre-tiling
// ---------------------------------------------------------------------------------------------
// Pack the A operand of a [rows x K] row-major weight (fp32 values or bf16 bits) into 16-byte
// per-lane fragments: lane l, slot j of k-group g of tile mt holds W[16 mt + l%16][kmap(g, l/16, j)],
// zero outside the matrix.  Order [g][tile][lane] (k-group-major, the layer weights) or
// [tile][g][lane] (the heads).
template <typename KMap>
std::vector<uint32_t> pack_frags(const void *W, bool bf, int rows, int K, int rows_p, int n_g, bool g_major,
                                 KMap kmap) {
    const int per = bf ? 8 : 4;
    const int n_t = rows_p / 16;
    std::vector<uint32_t> out;
    out.reserve((size_t)n_t * n_g * 64 * 4);
    for (int o = 0; o < n_t * n_g; ++o)
        for (int l = 0; l < 64; ++l) {
            const int mt = g_major ? o % n_t : o / n_g, g = g_major ? o / n_t : o % n_g;
            uint32_t slot[8] = {};
            for (int j = 0; j < per; ++j) {
                const int r = mt * 16 + l % 16, k = kmap(g, l / 16, j);
                if (r >= rows || k < 0 || k >= K) continue;
                if (bf) slot[j] = static_cast<const uint16_t *>(W)[(int64_t)r * K + k];
                else std::memcpy(&slot[j], static_cast<const float *>(W) + (int64_t)r * K + k, 4);
            }
            if (bf)
                for (int w = 0; w < 4; ++w) out.push_back(slot[2 * w] | (slot[2 * w + 1] << 16));
            else
                for (int w = 0; w < 4; ++w) out.push_back(slot[w]);
        }
    return out;
}

template <typename T>
int upload(const std::vector<T> &h, void **d, hipStream_t stream) {
    if (hipMalloc(d, h.size() * sizeof(T) + 16) != hipSuccess) return HARL_E_NOMEM;
    if (hipMemcpyAsync(*d, h.data(), h.size() * sizeof(T), hipMemcpyHostToDevice, stream) != hipSuccess) return HARL_E_HIP;
    return HARL_OK;
}

size_t policy_lds_bytes(const harl_policy *P, int nsg, int u) {
    const bool bf = P->dtype == HARL_BF16;
    const size_t el = bf ? 2 : 4;
    const size_t ns = 16 * (size_t)nsg;
    const size_t acts = ns * P->sp * el + ns * P->h1p * el;
    const size_t part = (size_t)u * ns * (P->hap + 4) * 4;  // partial heads
    const size_t bias = ((size_t)P->h1p + P->h2p + P->hap) * 4;
    return bias + (acts > part ? acts : part);
}

}  // namespace

int pack_policy(const harl_policy_desc *d, harl_policy **out, hipStream_t stream) {
    if (d->dtype != HARL_F32 && d->dtype != HARL_BF16) return fail(HARL_E_INVALID_ARG, "harl_policy_create: bad dtype");
    if (d->s < 1 || d->s > 1024 || d->h1 < 1 || d->h1 > 4096 || d->h2 < 1 || d->h2 > 4096 || d->a < 1 || d->a > 127)
        return fail(HARL_E_INVALID_ARG, "harl_policy_create: sizes out of range");
    if (!d->w1 || !d->b1 || !d->w2 || !d->b2 || !d->wa || !d->ba || !d->wv || !d->bv)
        return fail(HARL_E_INVALID_ARG, "harl_policy_create: null weight or bias");
    const bool bf = d->dtype == HARL_BF16;
    const int UPG = bf ? 32 : 16;
    const int sp = (int)round_up(d->s, UPG * kRing);   // whole rings of k-groups
    const int h1p = (int)round_up(d->h1, kHiddenPad);   // whole tile groups per wave, whole k-groups
    const int h2p = (int)round_up(d->h2, kHiddenPad);
    const int hap = (int)round_up(d->a + 1, 16);
    // heads as one matrix [a+1][h2]: rows 0..a-1 actor, row a value
    const size_t esz = bf ? 2 : 4;
    std::vector<uint8_t> wh((size_t)(d->a + 1) * d->h2 * esz);
    std::memcpy(wh.data(), d->wa, (size_t)d->a * d->h2 * esz);
    std::memcpy(wh.data() + (size_t)d->a * d->h2 * esz, d->wv, (size_t)d->h2 * esz);
    std::vector<uint32_t> w1, w2, whp;
    if (bf) {
        auto kstd = [](int g, int q, int j) { return g * 32 + q * 8 + j; };
        w1 = pack_frags(d->w1, true, d->h1, d->s, h1p, sp / 32, true, kstd);
        w2 = pack_frags(d->w2, true, d->h2, d->h1, h2p, h1p / 32, true, kstd);
        // head k-group p consumes h2 tiles 2p (slots 0..3) and 2p+1 (slots 4..7), each from the
        // accumulator layout: unit 16 t + 4 q + i
        auto khead = [](int pr, int q, int j) { return pr * 32 + (j / 4) * 16 + q * 4 + (j % 4); };
        whp = pack_frags(wh.data(), true, d->a + 1, d->h2, hap, h2p / 32, false, khead);
    } else {
        auto kstd = [](int g, int q, int j) { return g * 16 + q * 4 + j; };
        w1 = pack_frags(d->w1, false, d->h1, d->s, h1p, sp / 16, true, kstd);
        w2 = pack_frags(d->w2, false, d->h2, d->h1, h2p, h1p / 16, true, kstd);
        // head k-group t consumes h2 tile t from the accumulator layout (unit 16 t + 4 q + j): the
        // same map as the standard one
        whp = pack_frags(wh.data(), false, d->a + 1, d->h2, hap, h2p / 16, false, kstd);
    }
    std::vector<float> b1(h1p, 0.f), b2(h2p, 0.f), bh(hap, 0.f);
    std::memcpy(b1.data(), d->b1, (size_t)d->h1 * 4);
    std::memcpy(b2.data(), d->b2, (size_t)d->h2 * 4);
    std::memcpy(bh.data(), d->ba, (size_t)d->a * 4);
    bh[d->a] = d->bv[0];

    harl_policy *P = new (std::nothrow) harl_policy{};
    if (!P) return fail(HARL_E_NOMEM, "harl_policy_create: host allocation failed");
    P->dtype = d->dtype;
    P->s = d->s; P->h1 = d->h1; P->h2 = d->h2; P->a = d->a;
    P->sp = sp; P->h1p = h1p; P->h2p = h2p; P->hap = hap;
    (void)hipGetDevice(&P->device);
    if (policy_lds_bytes(P, 1, kMaxU) > 160 * 1024) {
        delete P;
        return fail(HARL_E_UNSUPPORTED, "harl_policy_create: layers too wide for the LDS-resident activations");
    }
    void *b1d = nullptr, *b2d = nullptr, *bhd = nullptr;
    int rc = upload(w1, &P->d_w1, stream);
    if (rc == HARL_OK) rc = upload(w2, &P->d_w2, stream);
    if (rc == HARL_OK) rc = upload(whp, &P->d_wh, stream);
    if (rc == HARL_OK) rc = upload(b1, &b1d, stream);
    if (rc == HARL_OK) rc = upload(b2, &b2d, stream);
    if (rc == HARL_OK) rc = upload(bh, &bhd, stream);
    P->d_b1 = static_cast<float *>(b1d);
    P->d_b2 = static_cast<float *>(b2d);
    P->d_bh = static_cast<float *>(bhd);
    if (rc == HARL_OK && hipStreamSynchronize(stream) != hipSuccess) rc = HARL_E_HIP;
    if (rc == HARL_OK && policy_x32_eligible(d)) rc = pack_policy_x32(d, P, stream);
    if (rc != HARL_OK) {
        (void)hipFree(P->d_w1); (void)hipFree(P->d_w2); (void)hipFree(P->d_wh);
        (void)hipFree(P->d_b1); (void)hipFree(P->d_b2); (void)hipFree(P->d_bh);
        (void)hipFree(P->x32_stream); (void)hipFree(P->x32_bias);
        delete P;
        return fail(rc, "harl_policy_create: device allocation or upload failed");
    }
    *out = P;
    return HARL_OK;
}

int policy_step_launch(const harl_policy *P, const void *states, int32_t B, int32_t *action, float *value,
                       float *probs, float *logits, hipStream_t stream) {
    if (B == 0) return HARL_OK;
    PolicyArgs a{};
    a.states = states;
    a.B = B;
    a.S = P->s;
    a.sp = P->sp; a.h1p = P->h1p; a.h2p = P->h2p; a.hap = P->hap; a.a = P->a;
    a.w1 = static_cast<const uint4 *>(P->d_w1);
    a.w2 = static_cast<const uint4 *>(P->d_w2);
    a.wh = static_cast<const uint4 *>(P->d_wh);
    a.b1 = P->d_b1; a.b2 = P->d_b2; a.bh = P->d_bh;
    a.action = action; a.value = value; a.probs = probs; a.logits = logits;
    const bool bf = P->dtype == HARL_BF16;
    // Large bf16 batches of the shapes it covers go to the 128-states-per-workgroup kernel
    if (P->x32_stream && B >= kX32MinBatch) return policy_x32_launch(P, states, B, action, value, probs, logits, stream);
    // Large batches share every weight fragment among several state groups (bf16: 4 groups of 16
    // states, 4 waves; fp32: 2 groups, 8 waves -- measured best on 65,536 states); small batches
    // use 16 states per workgroup so that they still spread over every CU.
    int nsg = B >= 16 * 1024 ? (bf ? 4 : 2) : 1;
    int u = nsg == 4 ? 4 : 8;
    if (policy_lds_bytes(P, nsg, u) > 160 * 1024) {
        nsg = 1;
        u = 8;
    }
    const size_t lds = policy_lds_bytes(P, nsg, u);
    const unsigned grid = (unsigned)ceil_div(B, 16 * nsg);
    const int ht = P->hap / 16;
    const int htm = ht <= 2 ? 2 : ht <= 5 ? 5 : 8;
    const void *kern = nullptr;
    // R2 = 8 k-groups of W2 in flight for 16-state workgroups (one per CU on small batches, where
    // each workgroup's memory waits are the kernel's); 4 for the 32- and 64-state shapes of large
    // batches, whose workgroups follow each other on a CU (8 measured 3 % slower at 65,536 fp32
    // states, and more registers spill at 8 head tiles)
#define HARL_POL(BF, NSG, HTM, U, TP, R2)              \
    if (bf == BF && nsg == NSG && htm == HTM && u == U) \
        kern = reinterpret_cast<const void *>(k_policy<BF, NSG, HTM, U, TP, kRing, R2>);
    HARL_POL(false, 1, 2, 8, 2, 8) HARL_POL(false, 1, 5, 8, 2, 8) HARL_POL(false, 1, 8, 8, 2, 8)
    HARL_POL(false, 2, 2, 8, 2, 4) HARL_POL(false, 2, 5, 8, 2, 4) HARL_POL(false, 2, 8, 8, 2, 4)
    HARL_POL(true, 1, 2, 8, 2, 8) HARL_POL(true, 1, 5, 8, 2, 8) HARL_POL(true, 1, 8, 8, 2, 8)
    HARL_POL(true, 4, 2, 4, 4, 4) HARL_POL(true, 4, 5, 4, 4, 4) HARL_POL(true, 4, 8, 4, 4, 4)
#undef HARL_POL
    if (!kern) return fail(HARL_E_UNSUPPORTED, "harl_policy_step: no kernel for this policy shape");
    if (const int rc = ensure_dynamic_lds(kern, lds)) return rc;
    void *args[] = {&a};
    HARL_HIP_CHECK(hipLaunchKernel(kern, dim3(grid), dim3(64 * u), args, lds, stream));
    HARL_HIP_CHECK(hipGetLastError());
    return HARL_OK;
}

}  // namespace harl
