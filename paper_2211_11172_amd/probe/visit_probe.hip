// Visit-loop microbenchmark of the binned tree walk: the walk of k_tree_score_b16 (walk_b16.hpp,
// the same instructions) with the code tile and every wave's tree resident in LDS and nothing
// streamed, repeated `reps` times.  It measures the node-visit rate the walk itself reaches for a
// given number of waves per CU (each wave walks 4 rows per lane of a 256-row tile), i.e. the ceiling
// of the scoring kernel's walk without the tile staging, the tree streaming and the reductions.
// Not part of libharl: it builds into libharl_probe.so, which only the benchmark loads.
#include <hip/hip_runtime.h>

#include "../csrc/walk_b16.hpp"

using namespace harl::b16;

namespace {

template <int TW>
__global__ __launch_bounds__(64 * TW) void k_visit_probe(const uint4 *__restrict__ codes, int F,
                                                        const uint4 *__restrict__ trees, int n_trees, int S16, int D,
                                                        const float *__restrict__ leaves, int reps,
                                                        double *__restrict__ out) {
    extern __shared__ __align__(16) char smem[];
    const int wid = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave), lane = threadIdx.x % kWave;
    const uint32_t sb = (uint32_t)S16 * 16u;
    const SlotPlan plan = slot_plan(F, TW, sb);
    // the tile: row group g's F * 16 uint4 at LDS uint4 4096 g (codes: [2][F][16] uint4)
    for (int i = threadIdx.x; i < 2 * F * 16; i += 64 * TW) {
        const int g = i / (F * 16), r = i % (F * 16);
        reinterpret_cast<uint4 *>(smem)[g * (int)(kGroupStride / 16) + r] = codes[i];
    }
    const int tree = (blockIdx.x * TW + wid) % n_trees;
    const uint32_t slot_off = wid < plan.n_a ? plan.a0 + (uint32_t)wid * sb : plan.b0 + (uint32_t)(wid - plan.n_a) * sb;
    uint4 *slot = reinterpret_cast<uint4 *>(smem + slot_off);
    for (int i = lane; i < S16; i += kWave) slot[i] = trees[(int64_t)tree * S16 + i];
    __syncthreads();
    const uint4 h0 = slot[0];
    Head hd{(uint32_t)__builtin_amdgcn_readfirstlane(h0.x), (uint32_t)__builtin_amdgcn_readfirstlane(h0.z),
            (uint32_t)__builtin_amdgcn_readfirstlane(h0.w)};
    const uint32_t tb = lds_addr(smem) + slot_off;
    uint32_t xa[kRPL];
#pragma unroll
    for (int j = 0; j < kRPL; ++j) xa[j] = lds_addr(smem) + kGroupStride * (j & 1) + 4u * (uint32_t)lane;
    float acc[kRPL] = {0.f, 0.f, 0.f, 0.f};
    float pend[kRPL] = {0.f, 0.f, 0.f, 0.f};
    const float *gl = leaves + (int64_t)tree * (2 << D);  // the tree's tail
    const SlotConsts sk = slot_consts(tb, 1u << D);
    Deferred last;
    no_deferred(last, leaves + (int64_t)n_trees * (2 << D));
    for (int r = 0; r < reps; ++r) walk(tb, D, sk, hd, xa, acc, gl, pend, last);
    finish(last, xa, acc, pend);
    double s = 0.0;
#pragma unroll
    for (int j = 0; j < kRPL; ++j) s += (double)acc[j] + (double)pend[j];
    out[(int64_t)blockIdx.x * 64 * TW + threadIdx.x] = s;
}

using ProbeKernel = void (*)(const uint4 *, int, const uint4 *, int, int, int, const float *, int, double *);

template <int TW>
int launch(int F, const void *codes, const void *trees, int n_trees, int S16, int D, const float *leaves, int reps,
           int n_blocks, double *out, hipStream_t stream) {
    const SlotPlan plan = slot_plan(F, TW, (uint32_t)S16 * 16u);
    if (plan.lds > 160u * 1024u) return -2;
    const ProbeKernel k = k_visit_probe<TW>;
    if (hipFuncSetAttribute(reinterpret_cast<const void *>(k), hipFuncAttributeMaxDynamicSharedMemorySize, (int)plan.lds) !=
        hipSuccess)
        return -4;
    hipLaunchKernelGGL(k, dim3((unsigned)n_blocks), dim3(64 * TW), plan.lds, stream,
                       static_cast<const uint4 *>(codes), F, static_cast<const uint4 *>(trees), n_trees, S16, D,
                       leaves, reps, out);
    return hipGetLastError() == hipSuccess ? 0 : -4;
}

}  // namespace

extern "C" {

// Walk `reps` times, in n_blocks workgroups of `waves` waves (1, 2, 4, 8, 12 or 16), the packed trees
// d_trees ([n_trees][2 * 2^depth] bytes of records, the binned layout, depth 9 or 10; wave w of
// block b walks tree (b * waves + w) % n_trees) over the code tile d_codes ([2][n_features][64]
// dwords, row group major) with the trees' tails d_leaves ([n_trees][2 * 2^depth] dwords: level
// depth-2's 16-byte records, then the leaves as fp32; then two 0.0f); d_out [n_blocks * 64 * waves]
// receives each thread's sum (to keep the work).  Returns 0, -1 on bad arguments, -2 when the tile and slots do not
// fit in LDS, -4 on a launch failure.
int harl_probe_visits(int waves, int depth, int reps, int n_features, int n_blocks, const void *d_codes,
                      const void *d_trees, int n_trees, const float *d_leaves, double *d_out, void *stream) {
    if (depth < 9 || depth > 10 || reps < 1 || n_features < 1 || n_features > 256 || n_blocks < 1 || n_trees < 1 ||
        !d_codes || !d_trees || !d_leaves || !d_out)
        return -1;
    const int S16 = (2 << depth) / 16;  // the slot: records of levels 0 .. depth-3
    hipStream_t s = static_cast<hipStream_t>(stream);
    switch (waves) {
    case 1: return launch<1>(n_features, d_codes, d_trees, n_trees, S16, depth, d_leaves, reps, n_blocks, d_out, s);
    case 2: return launch<2>(n_features, d_codes, d_trees, n_trees, S16, depth, d_leaves, reps, n_blocks, d_out, s);
    case 4: return launch<4>(n_features, d_codes, d_trees, n_trees, S16, depth, d_leaves, reps, n_blocks, d_out, s);
    case 8: return launch<8>(n_features, d_codes, d_trees, n_trees, S16, depth, d_leaves, reps, n_blocks, d_out, s);
    case 12: return launch<12>(n_features, d_codes, d_trees, n_trees, S16, depth, d_leaves, reps, n_blocks, d_out, s);
    case 16: return launch<16>(n_features, d_codes, d_trees, n_trees, S16, depth, d_leaves, reps, n_blocks, d_out, s);
    default: return -1;
    }
}

}  // extern "C"
