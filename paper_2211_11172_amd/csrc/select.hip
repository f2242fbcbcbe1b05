// Per-modification-type action selection (HARL paper, Section 4.3: the actor returns the best
// modification of each modification type; Appendix A.1: num_iters^2 + 1 tile-size actions and 3
// for each other type; Section 6.1: PPO, whose rollouts sample the actions).
//
// K9 k_policy_select: one (state, segment) per thread.  The actor's logits row of a state is cut
// into consecutive segments, one per modification type.  A segment's action is the lowest index
// attaining the maximum of its logits (greedy) or of logit + Gumbel noise (sampling: the
// Gumbel-max draw from the segment's softmax).  The noise of logit i of state b is -log(-log u),
// u = (w + 0.5) 2^-24 from the top 24 bits w of word i % 4 of Philox4x32-10 (Salmon et al., SC'11)
// at counter (i / 4, b, counter_lo, counter_hi) and key (seed_lo, seed_hi); noise and decision are
// fp64, so the choice is a function of the fp32 logits alone.  The segment's softmax and the
// chosen action's log-probability are fp32.
#include <hip/hip_runtime.h>

#include "internal.hpp"

namespace harl {
namespace {

constexpr int kSelectThreads = 256;
constexpr int kSelectLdsFloats = 4096;  // logits staged per workgroup (with fp64 keys: 48 KB of LDS)

struct Segments {
    int32_t off[HARL_SELECT_MAX_SEGMENTS + 1];
};

// Philox4x32 with 10 rounds: each round multiplies counter words 0 and 2 by two constants into
// 64-bit products; the new counter is (hi(M1 c2) ^ c1 ^ k0, lo(M1 c2), hi(M0 c0) ^ c3 ^ k1,
// lo(M0 c0)); the key advances by the Weyl constants between rounds.
__device__ __forceinline__ uint4 philox4x32_10(uint4 c, uint32_t k0, uint32_t k1) {
    constexpr uint32_t M0 = 0xD2511F53u, M1 = 0xCD9E8D57u, W0 = 0x9E3779B9u, W1 = 0xBB67AE85u;
#pragma unroll
    for (int round = 0; round < 10; ++round) {
        const uint32_t hi0 = __umulhi(M0, c.x), lo0 = M0 * c.x;
        const uint32_t hi1 = __umulhi(M1, c.z), lo1 = M1 * c.z;
        c = make_uint4(hi1 ^ c.y ^ k0, lo1, hi0 ^ c.w ^ k1, lo0);
        k0 += W0;
        k1 += W1;
    }
    return c;
}

// A workgroup owns R consecutive states: their logits rows (contiguous) are staged in LDS with
// coalesced loads; with SAMPLE every (row, group of 4 logits) item draws one Philox block and
// stores the fp64 keys logit + noise; then thread p < R * n_seg takes (row p / n_seg, segment
// p % n_seg) from LDS, and the softmax rows are written back with coalesced stores.
template <bool SAMPLE>
__global__ __launch_bounds__(kSelectThreads) void k_policy_select(const float *__restrict__ logits, int B, int a,
                                                                  int R, Segments seg, int n_seg, uint64_t seed,
                                                                  uint64_t counter, int32_t *__restrict__ action,
                                                                  float *__restrict__ logp, float *__restrict__ probs) {
    extern __shared__ __align__(16) char smem[];
    double *keys = reinterpret_cast<double *>(smem);                                  // [R][a] (SAMPLE)
    float *zs = reinterpret_cast<float *>(smem + (SAMPLE ? (size_t)R * a * 8 : 0));  // [R][a]
    const int t = threadIdx.x;
    const int64_t b0 = (int64_t)blockIdx.x * R;
    const int rows = B - b0 < R ? (int)(B - b0) : R;
    const int n = rows * a;
    for (int e = t; e < n; e += kSelectThreads) zs[e] = logits[b0 * a + e];
    __syncthreads();
    if constexpr (SAMPLE) {
        const int groups = (a + 3) / 4;
        for (int q = t; q < rows * groups; q += kSelectThreads) {
            const int r = q / groups, g = q - r * groups;
            const uint4 w = philox4x32_10(make_uint4((uint32_t)g, (uint32_t)(b0 + r), (uint32_t)counter,
                                                     (uint32_t)(counter >> 32)),
                                          (uint32_t)seed, (uint32_t)(seed >> 32));
            const uint32_t word[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int i = 4 * g + j;
                if (i < a) {
                    const double u = ((double)(word[j] >> 8) + 0.5) * (1.0 / 16777216.0);
                    keys[r * a + i] = (double)zs[r * a + i] - log(-log(u));
                }
            }
        }
        __syncthreads();
    }
    for (int p = t; p < rows * n_seg; p += kSelectThreads) {
        const int r = p / n_seg, s = p - r * n_seg;
        const int lo = seg.off[s], hi = seg.off[s + 1];
        const float *z = zs + r * a;
        float m = -INFINITY;
        double best = -INFINITY;
        int pick = lo;
        for (int i = lo; i < hi; ++i) {
            const float v = z[i];
            m = v > m ? v : m;
            const double key = SAMPLE ? keys[r * a + i] : (double)v;
            if (key > best) {
                best = key;
                pick = i;
            }
        }
        float sum = 0.f;
        for (int i = lo; i < hi; ++i) sum += expf(z[i] - m);
        const int64_t b = b0 + r;
        action[b * n_seg + s] = pick;
        if (logp) logp[b * n_seg + s] = (z[pick] - m) - logf(sum);
        // the segment's softmax replaces its logits in LDS (no other thread reads this segment)
        if (probs)
            for (int i = lo; i < hi; ++i) zs[r * a + i] = expf(zs[r * a + i] - m) / sum;
    }
    if (probs) {
        __syncthreads();
        for (int e = t; e < n; e += kSelectThreads) probs[b0 * a + e] = zs[e];
    }
}

}  // namespace

int policy_select_launch(const float *logits, int32_t B, int32_t a, const int32_t *seg_offsets, int32_t n_seg,
                         uint32_t flags, uint64_t seed, uint64_t counter, int32_t *action, float *logp, float *probs,
                         hipStream_t stream) {
    Segments seg{};
    for (int s = 0; s <= n_seg; ++s) seg.off[s] = seg_offsets[s];
    const bool sample = flags & HARL_SELECT_SAMPLE;
    // rows per workgroup: at most 64, kSelectLdsFloats logits in all, and few enough that a
    // batch spreads over about 256 workgroups
    int64_t R = ceil_div(B, 256);
    R = R < 1 ? 1 : R > 64 ? 64 : R;
    if (R * a > kSelectLdsFloats) R = kSelectLdsFloats / a;
    R = R * n_seg > kSelectThreads ? kSelectThreads / n_seg : R;
    const size_t lds = (size_t)R * a * (sample ? 12 : 4);
    const unsigned grid = (unsigned)ceil_div(B, R);
    const void *kern = sample ? reinterpret_cast<const void *>(k_policy_select<true>)
                              : reinterpret_cast<const void *>(k_policy_select<false>);
    if (const int rc = ensure_dynamic_lds(kern, lds)) return rc;
    if (sample)
        hipLaunchKernelGGL(k_policy_select<true>, dim3(grid), dim3(kSelectThreads), lds, stream, logits, B, a, (int)R,
                           seg, n_seg, seed, counter, action, logp, probs);
    else
        hipLaunchKernelGGL(k_policy_select<false>, dim3(grid), dim3(kSelectThreads), lds, stream, logits, B, a, (int)R,
                           seg, n_seg, seed, counter, action, logp, probs);
    HARL_HIP_CHECK(hipGetLastError());
    return HARL_OK;
}

}  // namespace harl
