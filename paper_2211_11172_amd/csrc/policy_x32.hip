// Actor/critic forward for large bf16 batches (HARL paper, Algorithm 1: the actor pi_theta(M|S)
// picks each candidate's modification, the critic V(S) of Eq. 6 gives its value; Section 4.3).
// Same function as k_policy in policy.hip -- shared trunk h1 = ReLU(W1 s + b1), h2 = ReLU(W2 h1 +
// b2), heads logits = Wa h2 + ba and v = wv . h2 + bv, lowest-index argmax, softmax -- laid out so
// that every weight byte read from L2 serves 128 states and every MFMA operand read from LDS is
// conflict-free.
//
// K4b k_policy_x32: a workgroup of 8 waves (two per SIMD) owns 128 states.  Waves g and g + 4 take
// the same 32 states (the N dimension of v_mfma_f32_32x32x16_bf16: 32 units x 16 inputs x 32
// states per instruction) and split the hidden layer h1 in halves: wave g + 4k holds, in
// registers, h1 units [k H1/2, (k+1) H1/2) of its 32 states.
//   - A finished 32-unit h1 tile leaves the accumulators, after bias, ReLU and rounding, already in
//     the B-operand layout of two layer-2 k-steps, because W2's input order is permuted at create
//     time to match it; the same holds from each h2 tile into the heads.  So neither h1 nor h2 is
//     stored to memory.
//   - Per 32-unit h2 tile both waves of a pair contract their half of h1; the second hands its
//     partial sums to the first through LDS, which finishes the tile (bias, ReLU, rounding) and
//     feeds it into the heads.  Two waves per SIMD let one wave's epilogue work overlap the other
//     wave's MFMAs.
//   - The weights stream through LDS in chunks shared by all waves, double-buffered: W1 in chunks
//     of 8 tiles (4 per half), then per h2 tile its W2 rows plus the matching head columns and the
//     chunk's biases.  Chunk c + 1 is copied global -> LDS by the DMA path (global_load_lds, 16
//     bytes per lane, no registers) while chunk c is consumed.
//   - Epilogue: head biases, lowest-index argmax over the logits, value, softmax; logits and
//     probabilities are transposed through LDS and written out row by row.
//
// MFMA 32x32x16 operand layouts (lane l of 64, h = l / 32, slot j = 0..7 of 8 bf16 per lane):
//   A[m = l % 32][k-slot (h, j)],  B[k-slot (h, j)][n = l % 32],  the same k for the same (h, j);
//   result register i = 0..15 of lane l: D[m = 8 (i / 4) + 4 h + i % 4][n = l % 32].
// Input order of a k-step of 16 inputs, by (h, j):
//   layer 1 (states, W1):       k = 8 h + j
//   layer 2 and heads (h1, h2): k = 8 (j / 4) + 4 h + j % 4  -- registers 8q .. 8q+7 of a finished
//   32-unit tile t hold, for lane half h, exactly units 32 t + 16 q + that k (q = 0, 1).
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstring>
#include <vector>

#include "internal.hpp"

namespace harl {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4v __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void lds_void;

constexpr int kWaves = 8;
constexpr int kGroups = 4;            // state groups of 32 per workgroup
constexpr int kStatesPerWave = 32;
constexpr int kStatesPerBlock = kGroups * kStatesPerWave;
constexpr int kKs1 = 8;               // layer-1 k-steps: inputs padded to 128
constexpr int kL1TilesPerChunk = 8;   // 32-unit W1 tiles per chunk (8 KB each), 4 per h1 half
constexpr int kFrag = 1024;           // bytes of one operand fragment (64 lanes x 16 B)
constexpr int kRing = 4;              // A fragments in flight per wave
constexpr int kMaxHeadTiles = 3;      // head rows (actions + value) <= 96
constexpr int kSlotBytes = kGroups * 64 * 64;  // exchange slots: one 32x32 fp32 tile per pair

struct X32Args {
    const uint16_t *states;
    int B, S, a, nt2, chunk_bytes;
    const char *stream;  // chunks of chunk_bytes: W1 chunks, then one chunk per h2 tile
    const float4 *bhp;   // head biases [tile][h][16] in accumulator order
    int32_t *action;
    float *value, *probs, *logits;
};

__device__ __forceinline__ uint32_t bf16_rne(float x) {
    // fp32 -> bf16 bits, nearest even (finite inputs: activations after ReLU)
    uint32_t b = __float_as_uint(x);
    b += 0x7FFFu + ((b >> 16) & 1u);
    return b >> 16;
}

__device__ __forceinline__ bf16x8 as_bf(u32x4v v) { return __builtin_bit_cast(bf16x8, v); }

__device__ __forceinline__ f32x16 mfma(const bf16x8 &a, const bf16x8 &b, const f32x16 &c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ bf16x8 lds_frag(const char *base, int frag, int lane) {
    return *reinterpret_cast<const bf16x8 *>(base + frag * kFrag + lane * 16);
}

// Bias, ReLU and bf16 rounding of a finished 32x32 tile; lo / hi are the B operands of the tile's
// first / second 16-input k-step of the next contraction.
__device__ __forceinline__ void act_pack(const f32x16 &acc, const float4 (&bias)[4], bf16x8 &lo, bf16x8 &hi) {
    float v[16];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        v[4 * q + 0] = fmaxf(acc[4 * q + 0] + bias[q].x, 0.f);
        v[4 * q + 1] = fmaxf(acc[4 * q + 1] + bias[q].y, 0.f);
        v[4 * q + 2] = fmaxf(acc[4 * q + 2] + bias[q].z, 0.f);
        v[4 * q + 3] = fmaxf(acc[4 * q + 3] + bias[q].w, 0.f);
    }
    lo = as_bf(u32x4v{bf16_rne(v[0]) | bf16_rne(v[1]) << 16, bf16_rne(v[2]) | bf16_rne(v[3]) << 16,
                      bf16_rne(v[4]) | bf16_rne(v[5]) << 16, bf16_rne(v[6]) | bf16_rne(v[7]) << 16});
    hi = as_bf(u32x4v{bf16_rne(v[8]) | bf16_rne(v[9]) << 16, bf16_rne(v[10]) | bf16_rne(v[11]) << 16,
                      bf16_rne(v[12]) | bf16_rne(v[13]) << 16, bf16_rne(v[14]) | bf16_rne(v[15]) << 16});
}

// Materialise a value here: an empty volatile asm that reads and rewrites its registers, so the
// computation producing it cannot be sunk towards its later uses (a finished h1 tile must leave the
// accumulators at once, or every tile's accumulators would stay live until layer 2).
__device__ __forceinline__ void pin(bf16x8 &v) { asm volatile("" : "+v"(v)); }

// Bias of half h of a tile from a [tile][h][16] block (accumulator order).
__device__ __forceinline__ void load_bias(const float4 *b, int tile, int h, float4 (&out)[4]) {
#pragma unroll
    for (int q = 0; q < 4; ++q) out[q] = b[(tile * 2 + h) * 4 + q];
}

// The last 1 KB of every chunk holds the biases of the chunk's tiles ([tile][h][16] floats).
__device__ __forceinline__ const float4 *chunk_bias(const char *chunk, int chunk_bytes) {
    return reinterpret_cast<const float4 *>(chunk + chunk_bytes - kFrag);
}

// This wave's share of the copy of one chunk: 1 KB pieces w, w + 8, ... by the DMA path.
__device__ __forceinline__ void copy_chunk(const char *__restrict__ src, char *dst, int n_pieces, int wid, int lane) {
    for (int q = wid; q < n_pieces; q += kWaves)
        __builtin_amdgcn_global_load_lds(reinterpret_cast<const void *>(src + (int64_t)q * kFrag + lane * 16),
                                         (lds_void *)(dst + q * kFrag), 16, 0, 0);
}

// Wait for this thread's outstanding global -> LDS copies, then for every wave's (the barrier).
__device__ __forceinline__ void chunk_barrier() {
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
}

// Layer-1 chunk C: its tiles 4k .. 4k+3 belong to h1 half k; this wave (half `kh`) computes its
// four, which are h1 tiles 4C .. 4C+3 of its half, from `cur`, while the next chunk is copied from
// `src` into `nxt`.  `cur` and `nxt` are distinct buffers; saying so (__restrict__) lets the
// compiler see that the LDS reads of `cur` need not wait for the copies into `nxt`.  Tiles are
// finished one at a time: the scheduling barriers and pin() keep the compiler from running several
// tiles' MFMAs ahead of their activations.
template <int C, int KH>
__device__ __forceinline__ void layer1_chunk(const char *__restrict__ cur, char *__restrict__ nxt,
                                             const char *__restrict__ src, int n_pieces, int chunk_bytes, int wid,
                                             int kh, int l, const bf16x8 (&xb)[kKs1], bf16x8 (&h1)[KH]) {
    copy_chunk(src, nxt, n_pieces, wid, l);
    __builtin_amdgcn_sched_barrier(0);
    const float4 *bb = chunk_bias(cur, chunk_bytes);
#pragma unroll
    for (int u = 0; u < 4; ++u) {
        const int slot = 4 * kh + u, t = 4 * C + u;
        float4 bias[4];
        load_bias(bb, slot, l / 32, bias);
        bf16x8 ring[kRing];
#pragma unroll
        for (int r = 0; r < kRing; ++r) ring[r] = lds_frag(cur, slot * kKs1 + r, l);
        f32x16 acc0 = {}, acc1 = {};
#pragma unroll
        for (int s = 0; s < kKs1; s += 2) {
            acc0 = mfma(ring[s % kRing], xb[s], acc0);
            acc1 = mfma(ring[(s + 1) % kRing], xb[s + 1], acc1);
            if (s + kRing < kKs1) {
                ring[s % kRing] = lds_frag(cur, slot * kKs1 + s + kRing, l);
                ring[(s + 1) % kRing] = lds_frag(cur, slot * kKs1 + s + 1 + kRing, l);
            }
            __builtin_amdgcn_sched_barrier(0);
        }
        act_pack(acc0 + acc1, bias, h1[2 * t], h1[2 * t + 1]);
        pin(h1[2 * t]);
        pin(h1[2 * t + 1]);
        __builtin_amdgcn_sched_barrier(0);
    }
}

// Layer-2 step T (T = 0 .. nt2; the last one only finishes tile nt2 - 1).  Chunk layout: W2 rows of
// tile T (one fragment per 16-input k-step), then the head columns and the b2 bias of tile T - 1.
// The two waves of a pair swap roles every step: in step T the wave of half T % 2 is the writer,
// the other the keeper.  In step T:
//   - every wave copies its share of the next chunk into `nxt`;
//   - the writer first finishes tile T - 1, whose keeper it was: its own partial sums plus its
//     partner's from the pair's exchange slot, bias, ReLU, bf16, straight into its head
//     accumulators;
//   - both waves contract their half of h1 with the W2 rows of tile T in `cur`; the writer stores
//     its sums in the exchange slot (after its own read of the slot above: program order), the
//     keeper keeps them for the next step, where it is the writer.
// One workgroup barrier per step (the caller's), and the finishing work of one wave overlaps the
// other wave's MFMAs.  `cur` and `nxt` are distinct buffers (__restrict__: the LDS reads of `cur`
// need not wait for the copies into `nxt`).
template <int KH, int HT>
__device__ __forceinline__ void layer2_step(const char *__restrict__ cur, char *__restrict__ nxt,
                                            const char *__restrict__ src, float4 *__restrict__ slot, int n_pieces,
                                            int chunk_bytes, int wid, bool writer, int kh, int l, bool finish,
                                            bool contract, const bf16x8 (&h1)[KH], f32x16 &own, f32x16 (&hacc)[HT]) {
    copy_chunk(src, nxt, n_pieces, wid, l);
    __builtin_amdgcn_sched_barrier(0);
    if (writer && finish) {
        f32x16 sum = own;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const float4 o = slot[q * 64 + l];
            sum[4 * q] += o.x;
            sum[4 * q + 1] += o.y;
            sum[4 * q + 2] += o.z;
            sum[4 * q + 3] += o.w;
        }
        float4 bias[4];
        load_bias(chunk_bias(cur, chunk_bytes), 0, l / 32, bias);
        bf16x8 hb[2];
        act_pack(sum, bias, hb[0], hb[1]);
#pragma unroll
        for (int ht = 0; ht < HT; ++ht) {
            hacc[ht] = mfma(lds_frag(cur, 2 * KH + 2 * ht, l), hb[0], hacc[ht]);
            hacc[ht] = mfma(lds_frag(cur, 2 * KH + 2 * ht + 1, l), hb[1], hacc[ht]);
        }
    }
    if (contract) {
        // A fragments through a kRing-deep register ring: the read of k-step s + kRing is issued
        // right after the MFMA of k-step s (the scheduling barriers keep the compiler from
        // shrinking the ring, which would expose the LDS latency at every MFMA)
        const int f0 = kh * KH;  // this half's first k-step
        bf16x8 ring[kRing];
#pragma unroll
        for (int r = 0; r < kRing; ++r) ring[r] = lds_frag(cur, f0 + r, l);
        f32x16 acc = {};
#pragma unroll
        for (int s = 0; s < KH; ++s) {
            acc = mfma(ring[s % kRing], h1[s], acc);
            if (s + kRing < KH) ring[s % kRing] = lds_frag(cur, f0 + s + kRing, l);
            __builtin_amdgcn_sched_barrier(0);
        }
        if (writer) {
#pragma unroll
            for (int q = 0; q < 4; ++q) slot[q * 64 + l] = make_float4(acc[4 * q], acc[4 * q + 1], acc[4 * q + 2], acc[4 * q + 3]);
        } else {
            own = acc;
        }
    }
    __builtin_amdgcn_sched_barrier(0);
}

template <int KS2, int HT>
__global__ __launch_bounds__(64 * kWaves) __attribute__((amdgpu_waves_per_eu(2, 2))) void k_policy_x32(X32Args p) {
    extern __shared__ __align__(16) char smem[];
    constexpr int KH = KS2 / 2;                      // layer-2 k-steps (and h1 tiles x 2) per half
    constexpr int NC1 = KS2 / 16;                    // W1 chunks: 4 tiles of each half per chunk
    static_assert(NC1 == 2 || NC1 == 4, "h1 of 512 or 1024 units");
    const int wid = __builtin_amdgcn_readfirstlane(threadIdx.x / 64);
    const int g = wid % kGroups, kh = wid / kGroups;
    const int l = threadIdx.x % 64, n = l % 32, h = l / 32;
    const int s_blk = blockIdx.x * kStatesPerBlock;
    const int s0 = s_blk + g * kStatesPerWave;
    const int st = s0 + n;
    const int CH = p.chunk_bytes, n_pieces = CH / kFrag, n_chunks = NC1 + p.nt2 + 1;
    char *const buf0 = smem;
    char *const buf1 = smem + CH;

    copy_chunk(p.stream, buf0, n_pieces, wid, l);
    // layer-1 B operands: this lane's state, inputs 16 s + 8 h .. + 7 (S % 8 == 0, zero past S)
    bf16x8 xb[kKs1];
#pragma unroll
    for (int s = 0; s < kKs1; ++s) {
        const int k0 = 16 * s + 8 * h;
        xb[s] = as_bf(u32x4v{0, 0, 0, 0});
        if (st < p.B && k0 < p.S) xb[s] = *reinterpret_cast<const bf16x8 *>(p.states + (int64_t)st * p.S + k0);
    }
    chunk_barrier();

    // ---------------- layer 1: this wave's half of h1 into registers ----------------
    bf16x8 h1[KH];
    layer1_chunk<0, KH>(buf0, buf1, p.stream + (int64_t)1 * CH, 1 < n_chunks ? n_pieces : 0, CH, wid, kh, l, xb, h1);
    chunk_barrier();
    layer1_chunk<1, KH>(buf1, buf0, p.stream + (int64_t)2 * CH, 2 < n_chunks ? n_pieces : 0, CH, wid, kh, l, xb, h1);
    chunk_barrier();
    if constexpr (NC1 > 2) {
        layer1_chunk<2, KH>(buf0, buf1, p.stream + (int64_t)3 * CH, 3 < n_chunks ? n_pieces : 0, CH, wid, kh, l, xb, h1);
        chunk_barrier();
        layer1_chunk<3, KH>(buf1, buf0, p.stream + (int64_t)4 * CH, 4 < n_chunks ? n_pieces : 0, CH, wid, kh, l, xb, h1);
        chunk_barrier();
    }

    // ---------------- layer 2: one 32-unit h2 tile per step, finished one step later ----------------
    f32x16 hacc[HT];
#pragma unroll
    for (int ht = 0; ht < HT; ++ht) hacc[ht] = f32x16{};
    f32x16 own = {};
    float4 *const slot = reinterpret_cast<float4 *>(smem + 2 * CH) + g * 4 * 64;  // this pair's exchange slot
    for (int T = 0; T <= p.nt2; ++T) {
        const int c = NC1 + T;
        layer2_step<KH, HT>((c & 1) ? buf1 : buf0, (c & 1) ? buf0 : buf1, p.stream + (int64_t)(c + 1) * CH, slot,
                            c + 1 < n_chunks ? n_pieces : 0, CH, wid, kh == (T & 1), kh, l, T > 0, T < p.nt2, h1, own,
                            hacc);
        chunk_barrier();  // the next chunk and the writers' partial sums are in LDS
    }
    // each wave of a pair accumulated the heads of every other tile: the half-1 wave hands its
    // accumulators to the half-0 wave (chunk buffers are free now)
    {
        float4 *hx = reinterpret_cast<float4 *>(smem) + g * (HT * 4 * 64);
        if (kh == 1) {
#pragma unroll
            for (int ht = 0; ht < HT; ++ht)
#pragma unroll
                for (int q = 0; q < 4; ++q)
                    hx[(ht * 4 + q) * 64 + l] = make_float4(hacc[ht][4 * q], hacc[ht][4 * q + 1], hacc[ht][4 * q + 2], hacc[ht][4 * q + 3]);
        }
        __syncthreads();
        if (kh == 0) {
#pragma unroll
            for (int ht = 0; ht < HT; ++ht)
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const float4 o = hx[(ht * 4 + q) * 64 + l];
                    hacc[ht][4 * q] += o.x;
                    hacc[ht][4 * q + 1] += o.y;
                    hacc[ht][4 * q + 2] += o.z;
                    hacc[ht][4 * q + 3] += o.w;
                }
        }
        __syncthreads();  // hx is read before the epilogue reuses the buffer
    }

    // ---------------- epilogue (the waves of half 0 hold the heads) ----------------
    // head rows of register i of tile ht: 32 ht + 8 (i / 4) + 4 h + i % 4 (actor rows < a, value row a)
    const int AP = p.a + 1;
    float *const tz = reinterpret_cast<float *>(smem);                 // [128 states][AP]
    float *const tmax = tz + kStatesPerBlock * AP, *const tinv = tmax + kStatesPerBlock;
    if (kh == 0) {
        float z[HT][16];
        float best = -INFINITY, val = 0.f;
        int best_i = 0x7FFFFFFF;
#pragma unroll
        for (int ht = 0; ht < HT; ++ht) {
            float4 bias[4];
            load_bias(p.bhp, ht, h, bias);
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const float bb = (i % 4 == 0) ? bias[i / 4].x : (i % 4 == 1) ? bias[i / 4].y : (i % 4 == 2) ? bias[i / 4].z : bias[i / 4].w;
                const int row = 32 * ht + 8 * (i / 4) + 4 * h + i % 4;
                const float v = hacc[ht][i] + bb;
                z[ht][i] = v;
                if (row < p.a && (v > best || (v == best && row < best_i))) {
                    best = v;
                    best_i = row;
                }
                if (row == p.a) val = v;
            }
        }
        {  // the other half of this state's rows sits in lane l ^ 32
            const float ob = __shfl_xor(best, 32, 64);
            const int oi = __shfl_xor(best_i, 32, 64);
            if (ob > best || (ob == best && oi < best_i)) {
                best = ob;
                best_i = oi;
            }
            val += __shfl_xor(val, 32, 64);
        }
        if (best_i == 0x7FFFFFFF) best_i = 0;  // only NaN logits: no maximum exists
        float sum = 0.f;
        if (p.probs) {
#pragma unroll
            for (int ht = 0; ht < HT; ++ht)
#pragma unroll
                for (int i = 0; i < 16; ++i)
                    if (32 * ht + 8 * (i / 4) + 4 * h + i % 4 < p.a) sum += __expf(z[ht][i] - best);
            sum += __shfl_xor(sum, 32, 64);
        }
        if (h == 0 && st < p.B) {
            p.action[st] = best_i;
            p.value[st] = val;
        }
        if (p.logits || p.probs) {
            // both chunk buffers are free after the last barrier
            const int ls = g * kStatesPerWave + n;
#pragma unroll
            for (int ht = 0; ht < HT; ++ht)
#pragma unroll
                for (int i = 0; i < 16; ++i) {
                    const int row = 32 * ht + 8 * (i / 4) + 4 * h + i % 4;
                    if (row < p.a) tz[ls * AP + row] = z[ht][i];
                }
            if (h == 0) {
                tmax[ls] = best;
                tinv[ls] = 1.f / sum;
            }
        }
    }
    if (p.logits || p.probs) {
        __syncthreads();
        // all 8 waves write: wave w takes states w, w + 8, ..., four at a time
        const int nv = p.B - s_blk < kStatesPerBlock ? p.B - s_blk : kStatesPerBlock;
        for (int n0 = wid; n0 < nv; n0 += 4 * kWaves) {
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int nn = n0 + j * kWaves;
                if (nn >= nv) break;
                const float mx = tmax[nn], inv = tinv[nn];
                for (int r = l; r < p.a; r += 64) {
                    const float v = tz[nn * AP + r];
                    const int64_t o = (int64_t)(s_blk + nn) * p.a + r;
                    if (p.logits) p.logits[o] = v;
                    if (p.probs) p.probs[o] = __expf(v - mx) * inv;
                }
            }
        }
    }
}

// ---------------------------------------------------------------------------------------------
// host: packing
// ---------------------------------------------------------------------------------------------
uint16_t wbits(const void *W, int K, int r, int k) { return static_cast<const uint16_t *>(W)[(int64_t)r * K + k]; }

// One 1 KB operand fragment: lane l, slot j = row (row0 + l % 32), input kmap(l / 32, j) of W
// ([rows][K] bf16 bits), zero outside the matrix.
template <typename KMap>
void put_frag(uint8_t *dst, const void *W, int rows, int K, int row0, KMap kmap) {
    for (int l = 0; l < 64; ++l)
        for (int j = 0; j < 8; ++j) {
            const int r = row0 + l % 32, k = kmap(l / 32, j);
            const uint16_t v = (r < rows && k >= 0 && k < K) ? wbits(W, K, r, k) : 0;
            std::memcpy(dst + l * 16 + j * 2, &v, 2);
        }
}

// [tile][h][16] biases in accumulator order: entry i of half h of tile t = b[32 t + 8 (i/4) + 4 h + i % 4]
std::vector<float> pack_bias(const float *b, int n, int tiles, const float *extra = nullptr, int n_extra = 0) {
    std::vector<float> out((size_t)tiles * 32, 0.f);
    for (int t = 0; t < tiles; ++t)
        for (int h = 0; h < 2; ++h)
            for (int i = 0; i < 16; ++i) {
                const int u = 32 * t + 8 * (i / 4) + 4 * h + i % 4;
                float v = 0.f;
                if (u < n) v = b[u];
                else if (u - n < n_extra) v = extra[u - n];
                out[((size_t)t * 2 + h) * 16 + i] = v;
            }
    return out;
}

}  // namespace

bool policy_x32_eligible(const harl_policy_desc *d) {
    return d->dtype == HARL_BF16 && d->s <= 16 * kKs1 && d->s % 8 == 0 && d->h1 <= 1024 &&
           d->a + 1 <= 32 * kMaxHeadTiles;
}

int pack_policy_x32(const harl_policy_desc *d, harl_policy *P, hipStream_t stream) {
    const int KS2 = d->h1 <= 512 ? 32 : 64;
    const int h1p = 16 * KS2, nt1 = h1p / 32, nc1 = nt1 / kL1TilesPerChunk;
    const int nt2 = (int)ceil_div(d->h2, 32), HT = (int)ceil_div(d->a + 1, 32);
    const int CH = (std::max(kL1TilesPerChunk * kKs1, KS2 + 2 * HT) + 1) * kFrag;  // + the bias KB
    std::vector<uint8_t> s((size_t)(nc1 + nt2 + 1) * CH, 0);
    auto k1 = [](int h, int j) { return 8 * h + j; };
    auto k2 = [](int h, int j) { return 8 * (j / 4) + 4 * h + j % 4; };
    // W1 chunk c, slot 4k + u (k = 0, 1; u < 4) holds h1 tile k * nt1/2 + 4c + u
    auto l1_slot = [&](int t, int &chunk, int &slot) {
        const int k = t / (nt1 / 2), lt = t % (nt1 / 2);
        chunk = lt / 4;
        slot = 4 * k + lt % 4;
    };
    for (int t = 0; t < nt1; ++t) {
        int chunk, slot;
        l1_slot(t, chunk, slot);
        for (int k = 0; k < kKs1; ++k)
            put_frag(s.data() + (size_t)chunk * CH + (slot * kKs1 + k) * kFrag, d->w1, d->h1, d->s, 32 * t,
                     [&](int h, int j) { return 16 * k + k1(h, j); });
    }
    // heads as one matrix [a+1][h2]: actor rows, then the value row
    std::vector<uint16_t> wh((size_t)(d->a + 1) * d->h2);
    std::memcpy(wh.data(), d->wa, (size_t)d->a * d->h2 * 2);
    std::memcpy(wh.data() + (size_t)d->a * d->h2, d->wv, (size_t)d->h2 * 2);
    // layer-2 chunk T (T = 0 .. nt2): W2 rows of tile T, then the head columns of tile T - 1 (the
    // kernel finishes each tile one step later)
    for (int T = 0; T <= nt2; ++T) {
        uint8_t *chunk = s.data() + (size_t)(nc1 + T) * CH;
        if (T < nt2)
            for (int k = 0; k < KS2; ++k)
                put_frag(chunk + k * kFrag, d->w2, d->h2, d->h1, 32 * T, [&](int h, int j) { return 16 * k + k2(h, j); });
        if (T > 0)
            for (int ht = 0; ht < HT; ++ht)
                for (int q = 0; q < 2; ++q)
                    put_frag(chunk + (KS2 + 2 * ht + q) * kFrag, wh.data(), d->a + 1, d->h2, 32 * ht,
                             [&](int h, int j) { return 32 * (T - 1) + 16 * q + k2(h, j); });
    }
    // biases: each chunk's last KB holds its tiles' biases in accumulator order (8 W1 tiles of 128 B,
    // or the one h2 tile); the head biases are a separate small array
    const std::vector<float> b1 = pack_bias(d->b1, d->h1, nt1), b2 = pack_bias(d->b2, d->h2, nt2),
                             bh = pack_bias(d->ba, d->a, HT, d->bv, 1);
    for (int t = 0; t < nt1; ++t) {
        int chunk, slot;
        l1_slot(t, chunk, slot);
        std::memcpy(s.data() + (size_t)(chunk + 1) * CH - kFrag + slot * 128, b1.data() + (size_t)t * 32, 128);
    }
    for (int T = 0; T < nt2; ++T)
        std::memcpy(s.data() + (size_t)(nc1 + T + 2) * CH - kFrag, b2.data() + (size_t)T * 32, 128);
    if (hipMalloc(&P->x32_stream, s.size()) != hipSuccess) return fail(HARL_E_NOMEM, "harl_policy_create: device allocation failed");
    if (hipMalloc(&P->x32_bias, bh.size() * 4) != hipSuccess) return fail(HARL_E_NOMEM, "harl_policy_create: device allocation failed");
    hipError_t e = hipMemcpyAsync(P->x32_stream, s.data(), s.size(), hipMemcpyHostToDevice, stream);
    if (e == hipSuccess) e = hipMemcpyAsync(P->x32_bias, bh.data(), bh.size() * 4, hipMemcpyHostToDevice, stream);
    if (e == hipSuccess) e = hipStreamSynchronize(stream);
    if (e != hipSuccess) return hip_fail(e, "harl_policy_create: upload");
    P->x32_ks2 = KS2;
    P->x32_ht = HT;
    P->x32_nt1 = nt1;
    P->x32_nt2 = nt2;
    P->x32_chunk = CH;
    return HARL_OK;
}

int policy_x32_launch(const harl_policy *P, const void *states, int32_t B, int32_t *action, float *value, float *probs,
                      float *logits, hipStream_t stream) {
    X32Args a{};
    a.states = static_cast<const uint16_t *>(states);
    a.B = B;
    a.S = P->s;
    a.a = P->a;
    a.nt2 = P->x32_nt2;
    a.chunk_bytes = P->x32_chunk;
    a.stream = static_cast<const char *>(P->x32_stream);
    a.bhp = static_cast<const float4 *>(P->x32_bias);
    a.action = action;
    a.value = value;
    a.probs = probs;
    a.logits = logits;
    const void *kern = nullptr;
#define HARL_X32(K, H) \
    if (P->x32_ks2 == K && P->x32_ht == H) kern = reinterpret_cast<const void *>(k_policy_x32<K, H>);
    HARL_X32(32, 1) HARL_X32(32, 2) HARL_X32(32, 3)
    HARL_X32(64, 1) HARL_X32(64, 2) HARL_X32(64, 3)
#undef HARL_X32
    if (!kern) return fail(HARL_E_UNSUPPORTED, "harl_policy_step: no large-batch kernel for this policy shape");
    const size_t lds = 2 * (size_t)P->x32_chunk + kSlotBytes;
    if (const int rc = ensure_dynamic_lds(kern, lds)) return rc;
    void *args[] = {&a};
    HARL_HIP_CHECK(hipLaunchKernel(kern, dim3((unsigned)ceil_div(B, kStatesPerBlock)), dim3(64 * kWaves), args, lds, stream));
    HARL_HIP_CHECK(hipGetLastError());
    return HARL_OK;
}

}  // namespace harl
