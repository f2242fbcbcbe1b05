// Schedule tracks between rounds (HARL paper, Algorithm 1 and Section 5): the reward of a
// modification step, its advantage (Eq. 6), and the adaptive-stopping elimination of the tracks
// with the lowest advantages.
//
// K7 k_track_advantage: one thread per track, fp32:
//      r = (C(s') - C(s)) / max(|C(s)|, eps)   -- Algorithm 1's relative score change, with the
//                                                 denominator read as max(|C(s)|, eps)
//      A = r + gamma V(s') - V(s)              -- Eq. 6
// K8 elimination: the n_keep tracks ranked first by (advantage desc, NaN last, -0 ties +0, lower
//    track index first) survive; their indices are written in ascending order (the live set is
//    compacted in place order), optionally with their rows of a per-track matrix.
//    Ranking keys are the 32-bit order keys of the advantages.  The n_keep-th largest key T comes
//    from a 4-pass most-significant-digit radix select (8 bits per pass): k_elim_hist (per-block
//    histograms of the current digit among the keys that match the digits chosen so far) and
//    k_elim_digit (one workgroup: sums the block histograms in block order and picks the digit;
//    the chosen prefix and the ranks still needed live in the workspace).  Every key above T
//    survives, and of the keys equal to T the first `need` in track order: k_elim_count counts both
//    per block, k_elim_scan turns the counts into block offsets, and k_elim_scatter writes each
//    survivor's index at its position in track order.  No atomics leave a workgroup, so the result
//    does not depend on scheduling.  Up to kFusedMax tracks, k_elim_fused does all of it in one
//    workgroup (keys in registers, the histograms in LDS) instead of eleven launches.
#include <hip/hip_runtime.h>

#include "internal.hpp"

namespace harl {
namespace {

constexpr int kAdvThreads = 256;
constexpr int kElimThreads = 256;
constexpr int kElimPer = 16;                            // keys per thread
constexpr int kElimBlock = kElimThreads * kElimPer;     // keys per workgroup
constexpr int kScanThreads = 1024;
constexpr int kGatherThreads = 256;

// ---- K7 ----
__global__ __launch_bounds__(kAdvThreads) void k_track_advantage(const float *__restrict__ c_prev,
                                                                 const float *__restrict__ c_next,
                                                                 const float *__restrict__ v_prev,
                                                                 const float *__restrict__ v_next, int n, float gamma,
                                                                 float eps, float *__restrict__ reward,
                                                                 float *__restrict__ adv) {
    const int i = blockIdx.x * kAdvThreads + threadIdx.x;
    if (i >= n) return;
    const float c = c_prev[i];
    const float r = (c_next[i] - c) / fmaxf(fabsf(c), eps);  // fmaxf(NaN, eps) = eps: r stays NaN
    if (reward) reward[i] = r;
    adv[i] = r + gamma * v_next[i] - v_prev[i];
}

// ---- K8 ----
// Larger key = ranked ahead; NaN -> 0 (behind every number); -0 -> +0.
__device__ __forceinline__ uint32_t order_key(float s) {
    uint32_t b = __float_as_uint(s);
    if (s != s) return 0u;
    if (b == 0x80000000u) b = 0u;
    return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}

struct ElimState {
    uint32_t prefix;  // digits of T chosen so far (higher passes), low bits zero
    uint32_t need;    // ranks still needed among the keys that match the prefix
};

// Per-block histogram of digit `shift` (24, 16, 8, 0) of the keys matching the prefix; block b owns
// keys [b * kElimBlock, (b + 1) * kElimBlock), read with stride kElimThreads (coalesced).
__global__ __launch_bounds__(kElimThreads) void k_elim_hist(const float *__restrict__ adv, int n, int shift,
                                                            const ElimState *__restrict__ st,
                                                            uint32_t *__restrict__ hist) {
    __shared__ uint32_t h[256];
    const int t = threadIdx.x, lane = t % 64;
    h[t] = 0;
    const uint32_t prefix = shift == 24 ? 0u : st->prefix;
    __syncthreads();
    const int64_t base = (int64_t)blockIdx.x * kElimBlock;
#pragma unroll
    for (int j = 0; j < kElimPer; ++j) {
        const int64_t i = base + (int64_t)j * kElimThreads + t;
        const bool in = i < n;
        const uint32_t key = in ? order_key(adv[i]) : 0u;
        const bool alive = in && (shift == 24 || ((key ^ prefix) >> (shift + 8)) == 0);
        const uint32_t bin = (key >> shift) & 255u;
        // lanes sharing the first live lane's bin are counted with one atomic
        const uint64_t live = __ballot(alive);
        if (live) {
            const int first = __builtin_ctzll(live);
            const uint32_t b0 = __builtin_amdgcn_readlane(bin, first);
            const uint64_t same = __ballot(alive && bin == b0);
            if (lane == first) atomicAdd(&h[b0], (uint32_t)__popcll(same));
            if (alive && bin != b0) atomicAdd(&h[bin], 1u);
        }
    }
    __syncthreads();
    hist[(int64_t)blockIdx.x * 256 + t] = h[t];
}

// Sum the block histograms (bins per thread, blocks in order), then pick the digit d of the
// need-th largest key: the keys with a larger digit number fewer than `need`, those with a digit
// >= d at least `need`.
__global__ __launch_bounds__(256) void k_elim_digit(const uint32_t *__restrict__ hist, int n_blocks, int shift,
                                                    uint32_t n_keep, ElimState *__restrict__ st) {
    __shared__ uint32_t h[256];
    const int t = threadIdx.x;
    uint32_t c = 0;
    for (int b = 0; b < n_blocks; ++b) c += hist[(int64_t)b * 256 + t];
    h[t] = c;
    const uint32_t need = shift == 24 ? n_keep : st->need;
    const uint32_t prefix = shift == 24 ? 0u : st->prefix;
    __syncthreads();
    if (t < 64) {
        // lane t holds digits 255-4t .. 252-4t (descending); inclusive prefix over lanes
        const uint32_t h0 = h[255 - 4 * t], h1 = h[254 - 4 * t], h2 = h[253 - 4 * t], h3 = h[252 - 4 * t];
        const uint32_t s = h0 + h1 + h2 + h3;
        uint32_t incl = s;
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
            const uint32_t v = __shfl_up(incl, o, 64);
            if (t >= o) incl += v;
        }
        const uint32_t excl = incl - s;
        if (excl < need && incl >= need) {
            uint32_t above = excl;
            int d;
            if (above + h0 >= need) d = 255 - 4 * t;
            else if (above += h0, above + h1 >= need) d = 254 - 4 * t;
            else if (above += h1, above + h2 >= need) d = 253 - 4 * t;
            else { above += h2; d = 252 - 4 * t; }
            st->prefix = prefix | ((uint32_t)d << shift);
            st->need = need - above;
        }
    }
}

// Keys [b * kElimBlock + kElimPer * t, + kElimPer) of thread t: counts of keys above T (low
// word) and equal to T (high word).
__device__ __forceinline__ uint64_t chunk_counts(const float *__restrict__ adv, int n, int64_t i0, uint32_t T) {
    uint32_t above = 0, eq = 0;
#pragma unroll
    for (int q = 0; q < kElimPer; ++q) {
        const int64_t i = i0 + q;
        if (i < n) {
            const uint32_t key = order_key(adv[i]);
            above += key > T;
            eq += key == T;
        }
    }
    return (uint64_t)above | ((uint64_t)eq << 32);
}

// Exclusive prefix over the threads of a workgroup of NT threads (64-bit, two 32-bit counts that
// never carry into each other); `total` receives the workgroup's sum.
template <int NT>
__device__ __forceinline__ uint64_t block_excl_scan(uint64_t v, uint64_t *wsum, uint64_t &total) {
    const int t = threadIdx.x, lane = t % 64, w = t / 64;
    uint64_t incl = v;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const uint64_t u = __shfl_up(incl, o, 64);
        if (lane >= o) incl += u;
    }
    if (lane == 63) wsum[w] = incl;
    __syncthreads();
    uint64_t before = 0, all = 0;
#pragma unroll
    for (int k = 0; k < NT / 64; ++k) {
        const uint64_t s = wsum[k];
        if (k < w) before += s;
        all += s;
    }
    total = all;
    return before + incl - v;
}

__global__ __launch_bounds__(kElimThreads) void k_elim_count(const float *__restrict__ adv, int n,
                                                             const ElimState *__restrict__ st,
                                                             uint64_t *__restrict__ cnt) {
    __shared__ uint64_t wsum[kElimThreads / 64];
    const uint64_t v = chunk_counts(adv, n, (int64_t)blockIdx.x * kElimBlock + (int64_t)kElimPer * threadIdx.x,
                                    st->prefix);
    uint64_t total;
    (void)block_excl_scan<kElimThreads>(v, wsum, total);
    if (threadIdx.x == 0) cnt[blockIdx.x] = total;
}

// Exclusive prefix of the per-block counts, in block order, by one workgroup.
__global__ __launch_bounds__(kScanThreads) void k_elim_scan(const uint64_t *__restrict__ cnt, int n_blocks,
                                                            uint64_t *__restrict__ off) {
    __shared__ uint64_t wsum[kScanThreads / 64];
    uint64_t carry = 0;
    for (int b0 = 0; b0 < n_blocks; b0 += kScanThreads) {
        const int b = b0 + (int)threadIdx.x;
        const uint64_t v = b < n_blocks ? cnt[b] : 0;
        uint64_t total;
        const uint64_t ex = block_excl_scan<kScanThreads>(v, wsum, total);
        if (b < n_blocks) off[b] = carry + ex;
        carry += total;
        __syncthreads();  // wsum is rewritten by the next chunk
    }
}

// Survivor positions in track order: a key above T at track i goes to (keys above T before i) +
// min(keys equal to T before i, need); a key equal to T survives if fewer than `need` equal keys
// precede it, at the same position formula.
__global__ __launch_bounds__(kElimThreads) void k_elim_scatter(const float *__restrict__ adv, int n,
                                                               const ElimState *__restrict__ st,
                                                               const uint64_t *__restrict__ off, int n_keep,
                                                               int32_t *__restrict__ keep_index) {
    __shared__ uint64_t wsum[kElimThreads / 64];
    const uint32_t T = st->prefix, need = st->need;
    const int64_t i0 = (int64_t)blockIdx.x * kElimBlock + (int64_t)kElimPer * threadIdx.x;
    const uint64_t v = chunk_counts(adv, n, i0, T);
    uint64_t total;
    const uint64_t ex = off[blockIdx.x] + block_excl_scan<kElimThreads>(v, wsum, total);
    uint32_t above = (uint32_t)ex, eq = (uint32_t)(ex >> 32);
#pragma unroll
    for (int q = 0; q < kElimPer; ++q) {
        const int64_t i = i0 + q;
        if (i < n) {
            const uint32_t key = order_key(adv[i]);
            const uint32_t pos = above + (eq < need ? eq : need);
            const bool keep = key > T || (key == T && eq < need);
            if (keep && pos < (uint32_t)n_keep) keep_index[pos] = (int32_t)i;
            above += key > T;
            eq += key == T;
        }
    }
}

constexpr int kFusedThreads = 1024, kFusedPer = 16, kFusedMax = kFusedThreads * kFusedPer;

// The whole elimination of n <= kFusedMax tracks in one workgroup: thread t holds the keys of
// tracks [16t, 16t + 16) in registers; each radix pass histograms the live keys into one of two
// LDS histograms (the other is cleared meanwhile) and wave 0 picks the digit; the survivors'
// positions come from one workgroup-wide prefix sum of the per-thread counts.
__global__ __launch_bounds__(kFusedThreads) void k_elim_fused(const float *__restrict__ adv, int n, int n_keep,
                                                              int32_t *__restrict__ keep_index) {
    __shared__ uint32_t hist[2][256];
    __shared__ uint32_t s_digit, s_above;
    __shared__ uint64_t wsum[kFusedThreads / 64];
    const int t = threadIdx.x, lane = t % 64;
    const int i0 = t * kFusedPer;
    uint32_t key[kFusedPer];
#pragma unroll
    for (int q = 0; q < kFusedPer; ++q) key[q] = i0 + q < n ? order_key(adv[i0 + q]) : 0u;
    if (t < 512) (&hist[0][0])[t] = 0;
    __syncthreads();
    uint32_t prefix = 0, need = (uint32_t)n_keep;
    int hb = 0;
    for (int shift = 24; shift >= 0; shift -= 8) {
#pragma unroll
        for (int q = 0; q < kFusedPer; ++q) {
            const bool alive = i0 + q < n && (shift == 24 || ((key[q] ^ prefix) >> (shift + 8)) == 0);
            const uint32_t bin = (key[q] >> shift) & 255u;
            const uint64_t live = __ballot(alive);
            if (live) {
                const int first = __builtin_ctzll(live);
                const uint32_t b0 = __builtin_amdgcn_readlane(bin, first);
                const uint64_t same = __ballot(alive && bin == b0);
                if (lane == first) atomicAdd(&hist[hb][b0], (uint32_t)__popcll(same));
                if (alive && bin != b0) atomicAdd(&hist[hb][bin], 1u);
            }
        }
        // the other histogram was last read before the previous pass's final barrier
        if (t < 256) hist[hb ^ 1][t] = 0;
        __syncthreads();
        if (t < 64) {
            const uint32_t *h = hist[hb];
            const uint32_t h0 = h[255 - 4 * t], h1 = h[254 - 4 * t], h2 = h[253 - 4 * t], h3 = h[252 - 4 * t];
            const uint32_t sum = h0 + h1 + h2 + h3;
            uint32_t incl = sum;
#pragma unroll
            for (int o = 1; o < 64; o <<= 1) {
                const uint32_t v = __shfl_up(incl, o, 64);
                if (t >= o) incl += v;
            }
            const uint32_t excl = incl - sum;
            if (excl < need && incl >= need) {
                uint32_t above = excl;
                int d;
                if (above + h0 >= need) d = 255 - 4 * t;
                else if (above += h0, above + h1 >= need) d = 254 - 4 * t;
                else if (above += h1, above + h2 >= need) d = 253 - 4 * t;
                else { above += h2; d = 252 - 4 * t; }
                s_digit = (uint32_t)d;
                s_above = above;
            }
        }
        __syncthreads();
        prefix |= s_digit << shift;
        need -= s_above;
        hb ^= 1;
    }
    const uint32_t T = prefix;
    uint32_t above = 0, eq = 0;
#pragma unroll
    for (int q = 0; q < kFusedPer; ++q)
        if (i0 + q < n) {
            above += key[q] > T;
            eq += key[q] == T;
        }
    uint64_t total;
    const uint64_t ex = block_excl_scan<kFusedThreads>((uint64_t)above | ((uint64_t)eq << 32), wsum, total);
    above = (uint32_t)ex;
    eq = (uint32_t)(ex >> 32);
#pragma unroll
    for (int q = 0; q < kFusedPer; ++q)
        if (i0 + q < n) {
            const uint32_t pos = above + (eq < need ? eq : need);
            const bool keep = key[q] > T || (key[q] == T && eq < need);
            if (keep && pos < (uint32_t)n_keep) keep_index[pos] = i0 + q;
            above += key[q] > T;
            eq += key[q] == T;
        }
}

__global__ __launch_bounds__(kGatherThreads) void k_iota(int32_t *__restrict__ out, int n) {
    const int i = blockIdx.x * kGatherThreads + threadIdx.x;
    if (i < n) out[i] = i;
}

// rows_out[m] = rows[keep_index[m]] for m < n_keep, in units of V bytes (row_units per row).
template <typename V>
__global__ __launch_bounds__(kGatherThreads) void k_gather_rows(const V *__restrict__ rows, int64_t row_units,
                                                                const int32_t *__restrict__ keep_index, int n_keep,
                                                                V *__restrict__ rows_out) {
    const int64_t total = (int64_t)n_keep * row_units;
    for (int64_t e = (int64_t)blockIdx.x * kGatherThreads + threadIdx.x; e < total;
         e += (int64_t)gridDim.x * kGatherThreads) {
        const int64_t m = e / row_units, u = e - m * row_units;
        rows_out[e] = rows[(int64_t)keep_index[m] * row_units + u];
    }
}

struct ElimLayout {
    size_t state, hist, cnt, off, total;
};

ElimLayout elim_layout(int32_t n) {
    const int64_t blocks = ceil_div(n > 0 ? n : 1, kElimBlock);
    ElimLayout L{};
    L.state = 0;
    L.hist = 256;
    L.cnt = L.hist + (size_t)round_up(blocks * 256 * 4, 256);
    L.off = L.cnt + (size_t)round_up(blocks * 8, 256);
    L.total = L.off + (size_t)round_up(blocks * 8, 256);
    return L;
}

int gather_launch(const void *rows, int64_t row_bytes, const int32_t *keep_index, int32_t n_keep, void *rows_out,
                  hipStream_t stream) {
    const bool v16 = row_bytes % 16 == 0 && aligned(rows, 16) && aligned(rows_out, 16);
    const bool v4 = row_bytes % 4 == 0 && aligned(rows, 4) && aligned(rows_out, 4);
    const int64_t unit = v16 ? 16 : v4 ? 4 : 1;
    const int64_t units = row_bytes / unit, total = (int64_t)n_keep * units;
    const unsigned grid = (unsigned)(ceil_div(total, kGatherThreads) < 65536 ? ceil_div(total, kGatherThreads) : 65536);
    if (v16)
        hipLaunchKernelGGL(k_gather_rows<uint4>, dim3(grid), dim3(kGatherThreads), 0, stream,
                           static_cast<const uint4 *>(rows), units, keep_index, n_keep, static_cast<uint4 *>(rows_out));
    else if (v4)
        hipLaunchKernelGGL(k_gather_rows<uint32_t>, dim3(grid), dim3(kGatherThreads), 0, stream,
                           static_cast<const uint32_t *>(rows), units, keep_index, n_keep,
                           static_cast<uint32_t *>(rows_out));
    else
        hipLaunchKernelGGL(k_gather_rows<uint8_t>, dim3(grid), dim3(kGatherThreads), 0, stream,
                           static_cast<const uint8_t *>(rows), units, keep_index, n_keep,
                           static_cast<uint8_t *>(rows_out));
    HARL_HIP_CHECK(hipGetLastError());
    return HARL_OK;
}

}  // namespace

int track_advantage_launch(const float *c_prev, const float *c_next, const float *v_prev, const float *v_next, int32_t n,
                           float gamma, float eps, float *reward, float *adv, hipStream_t stream) {
    hipLaunchKernelGGL(k_track_advantage, dim3((unsigned)ceil_div(n, kAdvThreads)), dim3(kAdvThreads), 0, stream, c_prev,
                       c_next, v_prev, v_next, n, gamma, eps, reward, adv);
    HARL_HIP_CHECK(hipGetLastError());
    return HARL_OK;
}

size_t track_eliminate_ws_bytes(int32_t n) { return elim_layout(n).total; }

int track_eliminate_launch(const float *adv, int32_t n, int32_t n_keep, int32_t *keep_index, const void *rows,
                           int64_t row_bytes, void *rows_out, void *ws, hipStream_t stream) {
    if (n_keep == n) {
        hipLaunchKernelGGL(k_iota, dim3((unsigned)ceil_div(n, kGatherThreads)), dim3(kGatherThreads), 0, stream,
                           keep_index, n);
        HARL_HIP_CHECK(hipGetLastError());
    } else if (n <= kFusedMax) {
        hipLaunchKernelGGL(k_elim_fused, dim3(1), dim3(kFusedThreads), 0, stream, adv, n, n_keep, keep_index);
        HARL_HIP_CHECK(hipGetLastError());
    } else {
        const ElimLayout L = elim_layout(n);
        char *w = static_cast<char *>(ws);
        ElimState *st = reinterpret_cast<ElimState *>(w + L.state);
        uint32_t *hist = reinterpret_cast<uint32_t *>(w + L.hist);
        uint64_t *cnt = reinterpret_cast<uint64_t *>(w + L.cnt), *off = reinterpret_cast<uint64_t *>(w + L.off);
        const int blocks = (int)ceil_div(n, kElimBlock);
        for (int shift = 24; shift >= 0; shift -= 8) {
            hipLaunchKernelGGL(k_elim_hist, dim3(blocks), dim3(kElimThreads), 0, stream, adv, n, shift, st, hist);
            HARL_HIP_CHECK(hipGetLastError());
            hipLaunchKernelGGL(k_elim_digit, dim3(1), dim3(256), 0, stream, hist, blocks, shift, (uint32_t)n_keep, st);
            HARL_HIP_CHECK(hipGetLastError());
        }
        hipLaunchKernelGGL(k_elim_count, dim3(blocks), dim3(kElimThreads), 0, stream, adv, n, st, cnt);
        HARL_HIP_CHECK(hipGetLastError());
        hipLaunchKernelGGL(k_elim_scan, dim3(1), dim3(kScanThreads), 0, stream, cnt, blocks, off);
        HARL_HIP_CHECK(hipGetLastError());
        hipLaunchKernelGGL(k_elim_scatter, dim3(blocks), dim3(kElimThreads), 0, stream, adv, n, st, off, n_keep,
                           keep_index);
        HARL_HIP_CHECK(hipGetLastError());
    }
    if (rows_out) return gather_launch(rows, row_bytes, keep_index, n_keep, rows_out, stream);
    return HARL_OK;
}

}  // namespace harl
