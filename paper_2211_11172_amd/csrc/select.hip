// Per-modification-type action selection (HARL paper, Section 4.3: the actor returns the best
// modification of each modification type; Appendix A.2: num_iters^2 + 1 tile-size actions and 3
// for each other type; Section 6.1: PPO, whose rollouts sample the actions).
//
// K9 k_policy_select: one thread per (state, segment).  The actor's logits row of a state is cut
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

template <bool SAMPLE>
__global__ __launch_bounds__(kSelectThreads) void k_policy_select(const float *__restrict__ logits, int B, int a,
                                                                  Segments seg, int n_seg, uint64_t seed,
                                                                  uint64_t counter, int32_t *__restrict__ action,
                                                                  float *__restrict__ logp, float *__restrict__ probs) {
    const int64_t tid = (int64_t)blockIdx.x * kSelectThreads + threadIdx.x;
    if (tid >= (int64_t)B * n_seg) return;
    const int64_t b = tid / n_seg;
    const int s = (int)(tid - b * n_seg);
    const int lo = seg.off[s], hi = seg.off[s + 1];
    const float *z = logits + b * a;
    float m = -INFINITY;
    double best = -INFINITY;
    int pick = lo;
    uint4 w = make_uint4(0, 0, 0, 0);
    for (int i = lo; i < hi; ++i) {
        const float v = z[i];
        m = v > m ? v : m;
        double key = v;
        if constexpr (SAMPLE) {
            if (i == lo || (i & 3) == 0)
                w = philox4x32_10(make_uint4((uint32_t)(i >> 2), (uint32_t)b, (uint32_t)counter, (uint32_t)(counter >> 32)),
                                  (uint32_t)seed, (uint32_t)(seed >> 32));
            const uint32_t word = (i & 3) == 0 ? w.x : (i & 3) == 1 ? w.y : (i & 3) == 2 ? w.z : w.w;
            const double u = ((double)(word >> 8) + 0.5) * (1.0 / 16777216.0);
            key += -log(-log(u));
        }
        if (key > best) {
            best = key;
            pick = i;
        }
    }
    float sum = 0.f;
    for (int i = lo; i < hi; ++i) sum += expf(z[i] - m);
    if (probs)
        for (int i = lo; i < hi; ++i) probs[b * a + i] = expf(z[i] - m) / sum;
    action[tid] = pick;
    if (logp) logp[tid] = (z[pick] - m) - logf(sum);
}

}  // namespace

int policy_select_launch(const float *logits, int32_t B, int32_t a, const int32_t *seg_offsets, int32_t n_seg,
                         uint32_t flags, uint64_t seed, uint64_t counter, int32_t *action, float *logp, float *probs,
                         hipStream_t stream) {
    Segments seg{};
    for (int s = 0; s <= n_seg; ++s) seg.off[s] = seg_offsets[s];
    const unsigned grid = (unsigned)ceil_div((int64_t)B * n_seg, kSelectThreads);
    if (flags & HARL_SELECT_SAMPLE)
        hipLaunchKernelGGL(k_policy_select<true>, dim3(grid), dim3(kSelectThreads), 0, stream, logits, B, a, seg, n_seg,
                           seed, counter, action, logp, probs);
    else
        hipLaunchKernelGGL(k_policy_select<false>, dim3(grid), dim3(kSelectThreads), 0, stream, logits, B, a, seg,
                           n_seg, seed, counter, action, logp, probs);
    HARL_HIP_CHECK(hipGetLastError());
    return HARL_OK;
}

}  // namespace harl
