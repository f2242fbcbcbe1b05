// Top-K selection of one round (Algorithm 1 of the HARL paper: "select top-K states from the
// heap H"; Section 4.3, Top-K Selection Phase) and the running top-K that plays the heap H
// accumulating candidates across steps.
//
// Ranking: score descending, then global index ascending; -0 ties +0; NaN below every number.
// A score becomes a 32-bit order key (larger key = better); candidate i's 64-bit composite is
// key << 32 | (0xFFFFFFFF - i), so the ranking is the descending order of unique composites and
// every selection below is exact and deterministic.
//
// K3 k_topk_select: a workgroup of 1024 threads owns a segment of up to 8192 candidates, held in
//    registers.  A most-significant-digit radix select (8 bits per pass over the composite,
//    per-wave LDS histograms, early exit once a digit bucket holds exactly the ranks still needed;
//    a segment of at most kk candidates keeps them all) finds the segment's kk best; they are
//    compacted into LDS and sorted (kk <= 128: each key's slot is its rank, counted against all
//    others by several threads per key; larger kk: bitonic, in the last round only, in registers
//    and lane shuffles up to one key per thread).  Lanes of one LDS atomic that hit
//    the same address are serialised, so histogram updates and compaction slots are aggregated per
//    wave first.
//    Segments run in parallel; their selections (unsorted: the next round selects again) form the
//    next round's candidates until one segment is left, whose workgroup writes the final top-k
//    directly (or, sorted, for the merge).
// K5 k_topk_merge: merges the sorted top-k of this call into the sorted running top-k by rank
//    computation (an element's output slot is its own index plus the number of elements of the
//    other list that rank ahead of it).
#include <hip/hip_runtime.h>

#include <mutex>

#include "internal.hpp"

namespace harl {
namespace {

// The candidate buffers of harl_topk_static: a file-scope device array instead of a caller
// workspace.  Every device that runs the library holds its own copy until the process ends.  In host
// code its name is only a host-side stand-in: kernels get the device address that
// hipGetSymbolAddress returns for the current device (topk_scratch below), never the name itself.
static __device__ __align__(256) unsigned char scratch[HARL_TOPK_STATIC_SCRATCH_BYTES];

constexpr int kSelThreads = 1024;
constexpr int kPerThread = 8;
constexpr int kRankSortMax = 128;  // up to this many selected keys are ranked directly, else bitonic
constexpr int kSeg = kSelThreads * kPerThread;  // candidates per workgroup
constexpr int kMergeThreads = 1024;

__device__ __forceinline__ uint32_t order_key(float s) {
    uint32_t b = __float_as_uint(s);
    if (s != s) return 0u;                  // NaN ranks last
    if (b == 0x80000000u) b = 0u;           // -0 ties +0
    return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}

__device__ __forceinline__ uint32_t local_of(uint64_t c) { return 0xFFFFFFFFu - (uint32_t)(c & 0xFFFFFFFFull); }

// Inclusive prefix sum over the 64 lanes of a wave.
__device__ __forceinline__ uint32_t wave_incl_scan(uint32_t v, int lane) {
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const uint32_t u = __shfl_up(v, o, 64);
        if (lane >= o) v += u;
    }
    return v;
}

// FROM_SCORES: round 0 reads fp32 scores (candidate = position); later rounds read composites.
// emit: this is the last round and its (single) workgroup writes io_score / io_index directly.
// sort_out: the kk selected composites are written in rank order (the last round, whose list is
// emitted or merged); the rounds before it feed another selection, which needs no order.
template <bool FROM_SCORES>
__global__ __launch_bounds__(kSelThreads) void k_topk_select(const float *__restrict__ score, const uint64_t *__restrict__ cin,
                                                             int64_t count, int kk, uint64_t *__restrict__ cout, int emit,
                                                             int sort_out, int n, int64_t index_base,
                                                             float *__restrict__ out_score, int64_t *__restrict__ out_index) {
    __shared__ uint32_t hist[2][256];  // digit histograms of consecutive passes (one is cleared meanwhile)
    __shared__ uint64_t sel[HARL_TOPK_MAX_K > kRankSortMax ? HARL_TOPK_MAX_K : kRankSortMax];
    __shared__ uint64_t ranked[kRankSortMax];
    __shared__ uint32_t s_digit, s_above, s_eq, s_cnt;
    const int t = threadIdx.x, lane = t % 64;
    const int64_t base = (int64_t)blockIdx.x * kSeg;
    const int64_t rem = count - base;
    const int n_valid = rem < kSeg ? (int)rem : kSeg;

    uint64_t x[kPerThread];
#pragma unroll
    for (int j = 0; j < kPerThread; ++j) {
        const int64_t i = base + (int64_t)j * kSelThreads + t;
        x[j] = 0;  // padding ranks below every candidate and never enters a histogram
        if (i < count) {
            if constexpr (FROM_SCORES)
                x[j] = ((uint64_t)order_key(score[i]) << 32) | (uint64_t)(0xFFFFFFFFu - (uint32_t)i);
            else
                x[j] = cin[i];
        }
    }
    // register slots j >= jn hold no candidate in any thread: the loops below skip them uniformly
    const int jn = (n_valid + kSelThreads - 1) / kSelThreads;
    auto valid = [&](int j) { return j * kSelThreads + t < n_valid; };
    for (int i = t; i < 2 * 256; i += kSelThreads) (&hist[0][0])[i] = 0;
    if (t == 0) s_cnt = 0;
    __syncthreads();

    // ---- radix select: find the prefix of the kk-th largest composite ----
    uint64_t prefix = 0;
    int shift = 64, hb = 0;
    uint32_t kr = (uint32_t)kk;  // ranks still needed among candidates matching `prefix`
    bool done = n_valid <= kk;   // a short segment keeps every candidate
    while (shift > 0 && !done) {
        shift -= 8;
        // Scores concentrate in few digit values (the leading digits are sign and exponent), and
        // lanes of one atomic instruction that hit the same bin are serialised.  So the lanes that
        // share the first live lane's bin are counted with a single atomic, the rest (few, and
        // spread) with their own.
#pragma unroll
        for (int j = 0; j < kPerThread; ++j) {
            if (j >= jn) break;
            const bool alive = valid(j) && (shift == 56 || ((x[j] ^ prefix) >> (shift + 8)) == 0);
            const uint32_t bin = (uint32_t)(x[j] >> shift) & 255u;
            const uint64_t live = __ballot(alive);
            if (live) {
                const int first = __builtin_ctzll(live);
                const uint32_t b0 = __builtin_amdgcn_readlane(bin, first);
                const uint64_t same = __ballot(alive && bin == b0);
                if (lane == first) atomicAdd(&hist[hb][b0], (uint32_t)__popcll(same));
                if (alive && bin != b0) atomicAdd(&hist[hb][bin], 1u);
            }
        }
        // the other histogram was last read by the previous pass's scan, before its final barrier
        if (t < 256) hist[hb ^ 1][t] = 0;
        __syncthreads();
        if (t < 64) {
            const uint32_t *h = hist[hb];
            const uint32_t h0 = h[255 - 4 * t], h1 = h[254 - 4 * t], h2 = h[253 - 4 * t], h3 = h[252 - 4 * t];
            const uint32_t s = h0 + h1 + h2 + h3;
            const uint32_t incl = wave_incl_scan(s, t);
            const uint32_t excl = incl - s;
            if (excl < kr && incl >= kr) {
                uint32_t above = excl;
                int d;
                if (above + h0 >= kr) d = 255 - 4 * t;
                else if (above += h0, above + h1 >= kr) d = 254 - 4 * t;
                else if (above += h1, above + h2 >= kr) d = 253 - 4 * t;
                else { above += h2; d = 252 - 4 * t; }
                s_digit = (uint32_t)d;
                s_above = above;
                s_eq = h[d];
            }
        }
        __syncthreads();
        const uint32_t d = s_digit;
        kr -= s_above;
        prefix |= (uint64_t)d << shift;
        done = s_eq == kr;
        hb ^= 1;
    }

    // ---- compaction: the composites strictly above the prefix bucket take slots [0, kk - kr), the
    // kr in it slots [kk - kr, kk) (a short segment: all of them, [0, n_valid)).  A lane's slots
    // follow from a prefix sum over the wave of both counts (packed in one word, each < 2^16) and
    // one counter atomic per wave.
    {
        const bool all = n_valid <= kk;
        const uint64_t ptop = all ? 0 : prefix >> shift;
        uint32_t cnt = 0;
#pragma unroll
        for (int j = 0; j < kPerThread; ++j) {
            if (j >= jn) break;
            if (!valid(j)) continue;
            const uint64_t top = all ? 1 : x[j] >> shift;
            cnt += top > ptop ? 1u : (top == ptop ? 0x10000u : 0u);
        }
        const uint32_t incl = wave_incl_scan(cnt, lane);
        const uint32_t total = __builtin_amdgcn_readlane(incl, 63);
        uint32_t wbase = 0;
        if (lane == 63 && total) wbase = atomicAdd(&s_cnt, total);
        wbase = __builtin_amdgcn_readlane(wbase, 63) + (incl - cnt);
        uint32_t a_slot = wbase & 0xFFFFu, e_slot = (uint32_t)kk - kr + (wbase >> 16);
#pragma unroll
        for (int j = 0; j < kPerThread; ++j) {
            if (j >= jn) break;
            if (!valid(j)) continue;
            const uint64_t top = all ? 1 : x[j] >> shift;
            if (top > ptop) {
                sel[a_slot++] = x[j];
            } else if (top == ptop) {
                if (e_slot < (uint32_t)kk) sel[e_slot] = x[j];
                ++e_slot;
            }
        }
        if (all)
            for (int i = n_valid + t; i < kk; i += kSelThreads) sel[i] = 0;
    }
    const uint64_t *out_keys = sel;
    if (kk <= kRankSortMax) {
        // rank sort: an entry's output slot is the number of entries ranking ahead of it (a larger
        // composite, or an equal one -- identical padding only -- at a lower position).  The list
        // is padded to kRankSortMax with zero composites (they rank behind every entry, and only
        // entries below kk are placed); 8 consecutive lanes count one entry's rank over 1/8 of it.
        constexpr int G = kSelThreads / kRankSortMax, PART = kRankSortMax / G;
        for (int i = kk + t; i < kRankSortMax; i += kSelThreads) sel[i] = 0;
        __syncthreads();
        const int i = t / G, part = t % G;
        const uint64_t v = sel[i];
        uint32_t rank = 0;
#pragma unroll
        for (int q = 0; q < PART; ++q) {
            const int j = part * PART + q;
            const uint64_t u = sel[j];
            rank += (u > v) | ((u == v) & (j < i));
        }
#pragma unroll
        for (int m = 1; m < G; m <<= 1) rank += __shfl_xor(rank, m, 64);
        if (part == 0 && i < kk) ranked[rank] = v;
        __syncthreads();
        out_keys = ranked;
    } else if (!sort_out) {
        __syncthreads();  // the selected composites, in compaction order
    } else if (kk <= kSelThreads) {
        // bitonic sort, descending, of the kk selected composites padded with zeros to P (a power of
        // 2, at most one per thread): a thread holds one key; partners fewer than 64 positions away
        // are in its wave and exchange by lane shuffles, the others through LDS (two barriers)
        int P = 1;
        while (P < kk) P <<= 1;
        for (int i = kk + t; i < P; i += kSelThreads) sel[i] = 0;
        __syncthreads();
        uint64_t key = t < P ? sel[t] : 0;
        for (int size = 2; size <= P; size <<= 1) {
            for (int stride = size >> 1; stride > 0; stride >>= 1) {
                uint64_t other;
                if (stride >= 64) {
                    __syncthreads();  // the previous exchange's reads are done
                    if (t < P) sel[t] = key;
                    __syncthreads();
                    other = t < P ? sel[t ^ stride] : 0;
                } else {
                    other = __shfl_xor(key, stride, 64);
                }
                // the lower position of a pair keeps the larger key in a descending block
                const bool keep_max = ((t & stride) == 0) == ((t & size) == 0);
                key = keep_max == (key > other) ? key : other;
            }
        }
        __syncthreads();
        if (t < P) sel[t] = key;
        __syncthreads();
    } else {
        int P = 1;
        while (P < kk) P <<= 1;
        for (int i = kk + t; i < P; i += kSelThreads) sel[i] = 0;
        __syncthreads();
        // bitonic sort of the kk selected composites, descending
        for (int size = 2; size <= P; size <<= 1) {
            for (int stride = size >> 1; stride > 0; stride >>= 1) {
                for (int i = t; i < P / 2; i += kSelThreads) {
                    const int lo = 2 * i - (i & (stride - 1)), hi = lo + stride;
                    const bool desc = (lo & size) == 0;
                    const uint64_t a = sel[lo], b = sel[hi];
                    if (desc ? (a < b) : (a > b)) {
                        sel[lo] = b;
                        sel[hi] = a;
                    }
                }
                __syncthreads();
            }
        }
    }
    for (int i = t; i < kk; i += kSelThreads) {
        const uint64_t key = out_keys[i];
        if (emit) {
            uint32_t l = local_of(key);
            l = l < (uint32_t)n ? l : (uint32_t)(n - 1);
            out_score[i] = score[l];
            out_index[i] = index_base + (int64_t)l;
        } else {
            cout[(int64_t)blockIdx.x * kk + i] = key;
        }
    }
}

// a ranks ahead of b
__device__ __forceinline__ bool ahead(uint32_t ka, int64_t ia, uint32_t kb, int64_t ib) {
    return ka > kb || (ka == kb && ia < ib);
}

// running (k sorted entries in io_*) <- top-k of running U batch (nb sorted composites of this call).
__global__ __launch_bounds__(kMergeThreads) void k_topk_merge(const uint64_t *__restrict__ bkeys, int nb,
                                                              const float *__restrict__ score, int n, int64_t index_base,
                                                              float *__restrict__ io_score, int64_t *__restrict__ io_index,
                                                              int k) {
    __shared__ uint32_t ak[HARL_TOPK_MAX_K], bk[HARL_TOPK_MAX_K];
    __shared__ int64_t ai[HARL_TOPK_MAX_K], bi[HARL_TOPK_MAX_K];
    __shared__ float as[HARL_TOPK_MAX_K], bs[HARL_TOPK_MAX_K];
    for (int i = threadIdx.x; i < k; i += kMergeThreads) {
        as[i] = io_score[i];
        ak[i] = order_key(as[i]);
        ai[i] = io_index[i];
    }
    for (int j = threadIdx.x; j < nb; j += kMergeThreads) {
        uint32_t l = local_of(bkeys[j]);
        l = l < (uint32_t)n ? l : (uint32_t)(n - 1);
        bs[j] = score[l];
        bk[j] = (uint32_t)(bkeys[j] >> 32);
        bi[j] = index_base + (int64_t)l;
    }
    __syncthreads();
    // output slot of running entry i: i + #(batch entries strictly ahead of it)
    for (int i = threadIdx.x; i < k; i += kMergeThreads) {
        int lo = 0, hi = nb;
        while (lo < hi) {
            const int mid = (lo + hi) >> 1;
            if (ahead(bk[mid], bi[mid], ak[i], ai[i])) lo = mid + 1;
            else hi = mid;
        }
        const int pos = i + lo;
        if (pos < k) {
            io_score[pos] = as[i];
            io_index[pos] = ai[i];
        }
    }
    // output slot of batch entry j: j + #(running entries ahead of it or equal to it)
    for (int j = threadIdx.x; j < nb; j += kMergeThreads) {
        int lo = 0, hi = k;
        while (lo < hi) {
            const int mid = (lo + hi) >> 1;
            if (!ahead(bk[j], bi[j], ak[mid], ai[mid])) lo = mid + 1;
            else hi = mid;
        }
        const int pos = j + lo;
        if (pos < k) {
            io_score[pos] = bs[j];
            io_index[pos] = bi[j];
        }
    }
}

__global__ void k_topk_reset(float *__restrict__ s, int64_t *__restrict__ idx, int k) {
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i < k) {
        s[i] = -INFINITY;
        idx[i] = INT64_MAX;
    }
}

struct Plan {
    int rounds;
    int64_t counts[40];  // candidates entering each round
    size_t buf_keys;     // composites per ping-pong buffer
};

Plan make_plan(int32_t n, int32_t k) {
    Plan p{};
    int64_t c = n;
    size_t mx = 0;
    do {
        p.counts[p.rounds++] = c;
        const int64_t segs = ceil_div(c, kSeg);
        c = segs * k;
        if ((size_t)c > mx) mx = (size_t)c;
        if (segs == 1) break;
    } while (p.rounds < 40);
    p.buf_keys = mx;
    return p;
}

}  // namespace

size_t topk_ws_bytes(int32_t n, int32_t k) {
    if (n <= 0 || k <= 0) return 256;
    const Plan p = make_plan(n, k);
    return 2 * round_up((int64_t)p.buf_keys * 8, 256) + 256;
}

int topk_launch(const float *score, int32_t n, int32_t k, int64_t index_base, float *io_score, int64_t *io_index,
                uint32_t flags, void *ws, size_t ws_bytes, hipStream_t stream) {
    if (k == 0 || (n == 0 && (flags & HARL_TOPK_MERGE))) return HARL_OK;
    const Plan p = make_plan(n, k);
    const size_t buf_bytes = round_up((int64_t)p.buf_keys * 8, 256);
    if (ws_bytes < 2 * buf_bytes) return fail(HARL_E_WORKSPACE, "harl_topk: workspace too small");
    uint64_t *buf[2] = {static_cast<uint64_t *>(ws), reinterpret_cast<uint64_t *>(static_cast<char *>(ws) + buf_bytes)};
    const bool merge = flags & HARL_TOPK_MERGE;
    const uint64_t *src = nullptr;
    for (int r = 0; r < p.rounds; ++r) {
        const int64_t c = p.counts[r];
        const unsigned segs = (unsigned)ceil_div(c, kSeg);
        const int last = r == p.rounds - 1 ? 1 : 0;
        const int emit = last && !merge ? 1 : 0;
        uint64_t *dst = buf[r & 1];
        if (r == 0)
            hipLaunchKernelGGL(k_topk_select<true>, dim3(segs), dim3(kSelThreads), 0, stream, score, nullptr, c, k, dst,
                               emit, last, n, index_base, io_score, io_index);
        else
            hipLaunchKernelGGL(k_topk_select<false>, dim3(segs), dim3(kSelThreads), 0, stream, score, src, c, k, dst,
                               emit, last, n, index_base, io_score, io_index);
        HARL_HIP_CHECK(hipGetLastError());
        src = dst;
    }
    if (merge) {
        const int nb = k < n ? k : n;  // real candidates at the head of the final sorted list
        hipLaunchKernelGGL(k_topk_merge, dim3(1), dim3(kMergeThreads), 0, stream, src, nb, score, n, index_base, io_score,
                           io_index, k);
        HARL_HIP_CHECK(hipGetLastError());
    }
    return HARL_OK;
}

// Device address of this device's `scratch`, looked up once per device (with that device current)
// and kept.
int topk_scratch(void **out) {
    static std::mutex mu;
    static void *addr[64] = {nullptr};
    int dev = 0;
    HARL_HIP_CHECK(hipGetDevice(&dev));
    if (dev < 0 || dev >= 64) return fail(HARL_E_UNSUPPORTED, "harl_topk_static: device index above 63");
    std::lock_guard<std::mutex> lock(mu);
    if (!addr[dev]) {
        void *p = nullptr;
        const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !p) return hip_fail(e != hipSuccess ? e : hipErrorInvalidSymbol, "harl_topk_static: scratch address");
        addr[dev] = p;
    }
    *out = addr[dev];
    return HARL_OK;
}

int topk_reset_launch(float *io_score, int64_t *io_index, int32_t k, hipStream_t stream) {
    if (k == 0) return HARL_OK;
    hipLaunchKernelGGL(k_topk_reset, dim3((unsigned)ceil_div(k, 256)), dim3(256), 0, stream, io_score, io_index, k);
    HARL_HIP_CHECK(hipGetLastError());
    return HARL_OK;
}

}  // namespace harl
