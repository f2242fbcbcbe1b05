// Actor/critic forward of one search round (HARL paper, Algorithm 1: select the modifications M
// with pi_theta(M|S); the critic V(S) of Eq. 6; Section 4.3).  Shared trunk
// h1 = ReLU(W1 s + b1), h2 = ReLU(W2 h1 + b2); actor head logits = Wa h2 + ba; value head
// v = wv . h2 + bv; action = lowest-index argmax of the logits; probs = softmax(logits).
//
// K4 k_policy: the three dense contractions run on MFMA, transposed so that states are the MFMA
// N dimension (H^T = W X^T).  A workgroup holds 16*NSG states and U waves; a wave computes its
// share of each layer's 16-unit tiles in groups of TP tiles.
//   phase 0  the states are staged into LDS ([state][unit], padded rows);
//   phase 1  each wave computes its 1/U of h1's tiles for all states, TP tiles at a time (A =
//            W1 fragments streamed from global memory through a kRing-deep register ring, B =
//            states from LDS, read one k-group ahead), applies bias + ReLU (+ bf16 rounding) and
//            stores the tiles to LDS;
//   phase 2  each wave computes its 1/U of h2's tiles the same way (B = h1 from LDS; every A
//            fragment feeds NSG state groups) and feeds each finished tile straight from its
//            accumulator registers into the head contraction: the MFMA result layout of a tile is
//            re-used as the B operand layout, with the head weights pre-permuted to match;
//   phase 3  the U per-wave partial heads are summed in a fixed order; bias, argmax, softmax
//            and value are computed per state and written out.
// fp32 policies use v_mfma_f32_16x16x4_f32, bf16 policies v_mfma_f32_16x16x32_bf16 (fp32
// accumulation; h1, h2 rounded to bf16, nearest even).  Weights are pre-tiled at create time so
// that a lane's operand for one "k-group" is 16 contiguous bytes:
//   fp32: a k-group is 16 input units = 4 MFMAs; lane l, slot j (j < 4) holds unit 16g + 4(l/16) + j
//   bf16: a k-group is 32 input units = 1 MFMA;  lane l, slot j (j < 8) holds unit 32g + 8(l/16) + j
// so an activation row in LDS ([state][unit]) gives the B operand of k-group g at byte offset
// 64g + 16(l/16) for either dtype.
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
#include <vector>

#include "internal.hpp"

namespace harl {
namespace {

constexpr int kMaxU = 8;      // waves per workgroup (at most)
constexpr int kRing = 4;      // k-groups of weight fragments in flight per wave
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

// The A fragments of a layer's first RING iterations (see dense_layer), loaded before the layer
// starts so that their latency overlaps the work before it.
template <int TP, int RING>
__device__ __forceinline__ void ring_fill(uint4 (&ring)[RING][TP], const uint4 *__restrict__ A, int t0, int n_tiles,
                                          int KG, int l) {
    const int NIT = n_tiles / TP * KG;
    const int64_t tstride = (int64_t)KG * 64;
#pragma unroll
    for (int r = 0; r < RING; ++r) {
        if (r < NIT) {
            const uint4 *src = A + (int64_t)(t0 + TP * (r / KG)) * tstride + (int64_t)(r % KG) * 64 + l;
#pragma unroll
            for (int j = 0; j < TP; ++j) ring[r][j] = src[j * tstride];
        } else {
#pragma unroll
            for (int j = 0; j < TP; ++j) ring[r][j] = make_uint4(0, 0, 0, 0);
        }
    }
}

// One dense layer for this wave: `n_tiles` output tiles of 16 units starting at tile `t0`, each a
// sum over KG k-groups (KG a multiple of RING), computed TP tiles at a time (TP independent
// accumulator chains sharing every B fragment).  The wave's iterations (tile group, k-group) run
// in order; `ring` holds the A fragments of the first RING iterations (ring_fill), and those of
// iteration it + RING are loaded from `A` (packed [tile][g][lane] x 16 B) into ring slot it % RING
// as soon as iteration it has issued its MFMAs; the B fragments of the next k-group are read from
// the LDS activation rows `in` (row stride `in_stride` bytes) into the other half of a double
// buffer.  done(first_tile, acc[TP][NSG]) consumes each finished group.
template <bool BF16, int NSG, int TP, int RING, typename Done>
__device__ __forceinline__ void dense_layer(uint4 (&ring)[RING][TP], const uint4 *__restrict__ A, int t0, int n_tiles,
                                            int KG, const char *in, int in_stride, int ln, int lq, int l, Done done) {
    static_assert(RING % 2 == 0, "the B double buffer alternates with the ring slot");
    const int n_groups = n_tiles / TP;
    const int NIT = n_groups * KG;
    const int64_t tstride = (int64_t)KG * 64;  // uint4 between the same k-group of consecutive tiles
    auto a_src = [&](int it) {
        return A + (int64_t)(t0 + TP * (it / KG)) * tstride + (int64_t)(it % KG) * 64 + l;
    };
    auto b_load = [&](int g, uint4 (&b)[NSG]) {
#pragma unroll
        for (int sg = 0; sg < NSG; ++sg)
            b[sg] = *reinterpret_cast<const uint4 *>(in + (sg * 16 + ln) * in_stride + g * 64 + lq * 16);
    };
    uint4 b[2][NSG];
    b_load(0, b[0]);
    for (int grp = 0; grp < n_groups; ++grp) {
        f32x4 acc[TP][NSG];
#pragma unroll
        for (int h = 0; h < TP; ++h)
#pragma unroll
            for (int sg = 0; sg < NSG; ++sg) acc[h][sg] = f32x4{0, 0, 0, 0};
        for (int g0 = 0; g0 < KG; g0 += RING) {
#pragma unroll
            for (int r = 0; r < RING; ++r) {
                const int g = g0 + r;
                const int it = grp * KG + g;
                if (it + 1 < NIT) b_load(g + 1 == KG ? 0 : g + 1, b[(r + 1) & 1]);
#pragma unroll
                for (int sg = 0; sg < NSG; ++sg)
#pragma unroll
                    for (int j = 0; j < TP; ++j) mfma_group<BF16>(ring[r][j], b[r & 1][sg], acc[j][sg]);
                if (it + RING < NIT) {
                    const uint4 *src = a_src(it + RING);
#pragma unroll
                    for (int j = 0; j < TP; ++j) ring[r][j] = src[j * tstride];
                }
            }
        }
        done(t0 + grp * TP, acc);
    }
}

// U waves per workgroup, 16*NSG states; HTM >= head tiles; layers in groups of TP tiles per wave.
template <bool BF16, int NSG, int HTM, int U, int TP, int RING>
__global__ __launch_bounds__(64 * U) void k_policy(PolicyArgs p) {
    extern __shared__ __align__(16) char smem[];
    constexpr int EL = BF16 ? 2 : 4;        // bytes per activation element
    constexpr int UPG = BF16 ? 32 : 16;     // input units per k-group
    constexpr int NTH = 64 * U;
    const int wid = threadIdx.x / 64, l = threadIdx.x % 64;
    const int ln = l % 16, lq = l / 16;
    const int s0 = blockIdx.x * 16 * NSG;
    constexpr int NS = 16 * NSG;
    const int xs_stride = p.sp * EL + 16;   // bytes per state row (padded against bank conflicts)
    const int h1_stride = p.h1p * EL + 16;
    char *xs = smem;
    char *h1 = smem + NS * xs_stride;
    const int HT = p.hap / 16;
    // the first W1 fragments are loaded while the states are staged
    const int mt1 = p.h1p / 16 / U, mt2 = p.h2p / 16 / U;
    uint4 ring[RING][TP];
    ring_fill<TP, RING>(ring, p.w1, wid * mt1, mt1, p.sp / UPG, l);

    // ---------------- phase 0: states -> LDS [state][unit] (zero beyond S and B) ----------------
    {
        const int row_elems = p.sp;
        for (int e = threadIdx.x; e < NS * row_elems; e += NTH) {
            const int r = e / row_elems, c = e % row_elems;
            const int st = s0 + r;
            if constexpr (BF16) {
                uint16_t v = 0;
                if (st < p.B && c < p.S) v = static_cast<const uint16_t *>(p.states)[(int64_t)st * p.S + c];
                *reinterpret_cast<uint16_t *>(xs + r * xs_stride + c * 2) = v;
            } else {
                float v = 0.f;
                if (st < p.B && c < p.S) v = static_cast<const float *>(p.states)[(int64_t)st * p.S + c];
                *reinterpret_cast<float *>(xs + r * xs_stride + c * 4) = v;
            }
        }
    }
    __syncthreads();

    // ---------------- phase 1: h1 = act(W1 s + b1), this wave's share of the tiles ----------------
    {
        const int mt_per = mt1;
        dense_layer<BF16, NSG, TP, RING>(ring, p.w1, wid * mt_per, mt_per, p.sp / UPG, xs, xs_stride, ln, lq, l,
                                         [&](int mt0, f32x4 (&acc)[TP][NSG]) {
#pragma unroll
                                             for (int h = 0; h < TP; ++h) {
                                                 const int u0 = (mt0 + h) * 16 + lq * 4;
#pragma unroll
                                                 for (int sg = 0; sg < NSG; ++sg) {
                                                     float v[4];
#pragma unroll
                                                     for (int i = 0; i < 4; ++i) v[i] = fmaxf(acc[h][sg][i] + p.b1[u0 + i], 0.f);
                                                     char *dst = h1 + (sg * 16 + ln) * h1_stride + u0 * EL;
                                                     if constexpr (BF16) {
                                                         *reinterpret_cast<uint2 *>(dst) =
                                                             make_uint2(bf16_rne(v[0]) | (bf16_rne(v[1]) << 16),
                                                                        bf16_rne(v[2]) | (bf16_rne(v[3]) << 16));
                                                     } else {
                                                         *reinterpret_cast<float4 *>(dst) = make_float4(v[0], v[1], v[2], v[3]);
                                                     }
                                                 }
                                             }
                                         });
    }
    // the first W2 fragments are loaded before the barrier that publishes h1
    ring_fill<TP, RING>(ring, p.w2, wid * mt2, mt2, p.h1p / UPG, l);
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
                    const int hk = hk0 + q;
                    if (ht < HT && hk < HKG) hpf[q][ht] = p.wh[((int64_t)ht * HKG + hk) * 64 + l];
                }
        };
        head_fetch(mt_first);
        dense_layer<BF16, NSG, TP, RING>(
            ring, p.w2, mt_first, mt_per, p.h1p / UPG, h1, h1_stride, ln, lq, l, [&](int mt0, f32x4 (&acc)[TP][NSG]) {
                float bias[TP][4];
#pragma unroll
                for (int h = 0; h < TP; ++h)
#pragma unroll
                    for (int i = 0; i < 4; ++i) bias[h][i] = p.b2[(mt0 + h) * 16 + lq * 4 + i];
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
                head_fetch(mt0 + TP);
            });
    }
    __syncthreads();  // h1 no longer needed: its LDS takes the partial heads

    // ---------------- phase 3: fixed-order sum of the U partial heads, epilogue ----------------
    // Every thread sums some of the NSG*hap*16 head values over the U waves (in wave order, then
    // the bias) into zs; the waves of the state groups then take argmax, softmax and the value.
    float *part = reinterpret_cast<float *>(smem);  // [U][NSG][hap][16]
    float *zs = part + (int64_t)U * NSG * p.hap * 16;  // [NSG][hap][16]
#pragma unroll
    for (int sg = 0; sg < NSG; ++sg)
#pragma unroll
        for (int ht = 0; ht < HTM; ++ht)
            if (ht < HT)
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    part[(((int64_t)wid * NSG + sg) * p.hap + ht * 16 + lq * 4 + i) * 16 + ln] = hacc[sg][ht][i];
    __syncthreads();
    {
        const int nz = NSG * p.hap * 16;
        for (int v = threadIdx.x; v < nz; v += NTH) {
            const int row = (v / 16) % p.hap;
            float s = 0.f;
#pragma unroll
            for (int w = 0; w < U; ++w) s += part[(int64_t)w * nz + v];
            zs[v] = s + p.bh[row];
        }
    }
    __syncthreads();
    for (int sg = wid; sg < NSG; sg += U) {
        const int st = s0 + sg * 16 + ln;
        float best = -INFINITY;
        int best_i = 0x7FFFFFFF;
        float val = 0.f;
        float z[HTM][4];  // rows owned by this lane: 16*ht + 4*lq + i
#pragma unroll
        for (int ht = 0; ht < HTM; ++ht)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                z[ht][i] = 0.f;
                if (ht >= HT) continue;
                const int row = ht * 16 + lq * 4 + i;
                const float s = zs[((int64_t)sg * p.hap + row) * 16 + ln];
                z[ht][i] = s;
                if (row < p.a && (s > best || (s == best && row < best_i))) {
                    best = s;
                    best_i = row;
                }
                if (row == p.a) val = s;
            }
        // combine over the 4 lanes of this state (xor 16, xor 32)
#pragma unroll
        for (int m = 16; m <= 32; m <<= 1) {
            const float ob = __shfl_xor(best, m, 64);
            const int oi = __shfl_xor(best_i, m, 64);
            if (ob > best || (ob == best && oi < best_i)) {
                best = ob;
                best_i = oi;
            }
            val += __shfl_xor(val, m, 64);
        }
        if (best_i == 0x7FFFFFFF) best_i = 0;  // only NaN logits: no maximum exists
        float sum = 0.f;
        if (p.probs) {
#pragma unroll
            for (int ht = 0; ht < HTM; ++ht)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int row = ht * 16 + lq * 4 + i;
                    if (ht < HT && row < p.a) sum += expf(z[ht][i] - best);
                }
            sum += __shfl_xor(sum, 16, 64);
            sum += __shfl_xor(sum, 32, 64);
        }
        if (st < p.B) {
#pragma unroll
            for (int ht = 0; ht < HTM; ++ht)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int row = ht * 16 + lq * 4 + i;
                    if (ht < HT && row < p.a) {
                        if (p.logits) p.logits[(int64_t)st * p.a + row] = z[ht][i];
                        if (p.probs) p.probs[(int64_t)st * p.a + row] = expf(z[ht][i] - best) / sum;
                    }
                }
            if (lq == 0) {
                p.action[st] = best_i;
                p.value[st] = val;
            }
        }
    }
}

// ---------------------------------------------------------------------------------------------
// host: weight pre-tiling
// ---------------------------------------------------------------------------------------------
// Pack the A operand of a [rows x K] row-major weight (fp32 values or bf16 bits) into 16-byte
// per-lane fragments, order [tile][g][lane]: lane l, slot j of k-group g of tile mt holds
// W[16 mt + l%16][kmap(g, l/16, j)], zero outside the matrix.
template <typename KMap>
std::vector<uint32_t> pack_frags(const void *W, bool bf, int rows, int K, int rows_p, int n_g, KMap kmap) {
    const int per = bf ? 8 : 4;
    std::vector<uint32_t> out;
    out.reserve((size_t)rows_p / 16 * n_g * 64 * 4);
    for (int mt = 0; mt < rows_p / 16; ++mt)
        for (int g = 0; g < n_g; ++g)
            for (int l = 0; l < 64; ++l) {
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
    const size_t acts = ns * (P->sp * el + 16) + ns * (P->h1p * el + 16);
    const size_t part = (size_t)(u + 1) * nsg * P->hap * 16 * 4;  // partial heads and their sums
    return acts > part ? acts : part;
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
        w1 = pack_frags(d->w1, true, d->h1, d->s, h1p, sp / 32, kstd);
        w2 = pack_frags(d->w2, true, d->h2, d->h1, h2p, h1p / 32, kstd);
        // head k-group p consumes h2 tiles 2p (slots 0..3) and 2p+1 (slots 4..7), each from the
        // accumulator layout: unit 16 t + 4 q + i
        auto khead = [](int pr, int q, int j) { return pr * 32 + (j / 4) * 16 + q * 4 + (j % 4); };
        whp = pack_frags(wh.data(), true, d->a + 1, d->h2, hap, h2p / 32, khead);
    } else {
        auto kstd = [](int g, int q, int j) { return g * 16 + q * 4 + j; };
        w1 = pack_frags(d->w1, false, d->h1, d->s, h1p, sp / 16, kstd);
        w2 = pack_frags(d->w2, false, d->h2, d->h1, h2p, h1p / 16, kstd);
        // head k-group t consumes h2 tile t from the accumulator layout (unit 16 t + 4 q + j): the
        // same map as the standard one
        whp = pack_frags(wh.data(), false, d->a + 1, d->h2, hap, h2p / 16, kstd);
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
#define HARL_POL(BF, NSG, HTM, U, TP)                  \
    if (bf == BF && nsg == NSG && htm == HTM && u == U) \
        kern = reinterpret_cast<const void *>(k_policy<BF, NSG, HTM, U, TP, kRing>);
    HARL_POL(false, 1, 2, 8, 2) HARL_POL(false, 1, 5, 8, 2) HARL_POL(false, 1, 8, 8, 2)
    HARL_POL(false, 2, 2, 8, 2) HARL_POL(false, 2, 5, 8, 2) HARL_POL(false, 2, 8, 8, 2)
    HARL_POL(true, 1, 2, 8, 2) HARL_POL(true, 1, 5, 8, 2) HARL_POL(true, 1, 8, 8, 2)
    HARL_POL(true, 4, 2, 4, 4) HARL_POL(true, 4, 5, 4, 4) HARL_POL(true, 4, 8, 4, 4)
#undef HARL_POL
    if (!kern) return fail(HARL_E_UNSUPPORTED, "harl_policy_step: no kernel for this policy shape");
    if (const int rc = ensure_dynamic_lds(kern, lds)) return rc;
    void *args[] = {&a};
    HARL_HIP_CHECK(hipLaunchKernel(kern, dim3(grid), dim3(64 * u), args, lds, stream));
    HARL_HIP_CHECK(hipGetLastError());
    return HARL_OK;
}

}  // namespace harl
