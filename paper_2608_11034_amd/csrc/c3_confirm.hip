// Temporal confirmation of C3 results for gfx950.
//
// Input: per-iteration outlier bitmaps of G peer groups (u64 per (t, g)) for
// fingerprints (exact C3) and timings (statistical C3).  Output: one verdict
// per rank, rank = r * G + g.
//
// Pass 1: one thread per (segment, rank); a segment is kSeg consecutive
// iterations.  Consecutive threads take consecutive groups g, so the loads of
// bitmap[t][g] are coalesced.  The thread counts attributed iterations in its
// segment, notes the first attributed fingerprint and any two consecutive
// attributed timings (the pair (t, t + 1) belongs to the segment of t), and
// slides a window of W iterations over the window starts in its segment
// (reading up to W - 1 iterations into the next segment).
// Pass 2: one thread per rank combines its segments in order.
#include "c3_device.h"
#include "c3_internal.h"

namespace c3 {

constexpr int64_t kSeg = 64;
constexpr int kConfThreads = 256;

struct SegVerdict {
    uint32_t flags;          // bit 2: two consecutive slow iterations
    int32_t first_div;       // first attributed fingerprint iteration, -1
    uint32_t div_count;
    uint32_t slow_count;
    uint32_t max_window;
    int32_t first_window;    // first window start over the threshold, -1
};
static_assert(sizeof(SegVerdict) == 24, "segment verdict layout");

__device__ inline uint32_t bit_of(const uint64_t* bm, int64_t t, int64_t G, int64_t g, int r) {
    return (uint32_t)((bm[t * G + g] >> r) & 1ull);
}

__global__ void __launch_bounds__(kConfThreads) confirm_segment_kernel(
    const uint64_t* __restrict__ fpb, const uint64_t* __restrict__ tmb, int R, int64_t G, int64_t T,
    int64_t Wt, int64_t n_seg, SegVerdict* __restrict__ out) {
    const int64_t n_ranks = (int64_t)R * G;
    const int64_t idx = (int64_t)blockIdx.x * kConfThreads + threadIdx.x;
    if (idx >= n_ranks * n_seg) return;
    const int64_t sgi = idx / n_ranks;
    const int64_t rank = idx - sgi * n_ranks;
    const int r = (int)(rank / G);
    const int64_t g = rank - (int64_t)r * G;
    const int64_t t0 = sgi * kSeg;
    const int64_t t1 = min(T, t0 + kSeg);
    SegVerdict v{0u, -1, 0u, 0u, 0u, -1};
    uint32_t prev = 0;
    for (int64_t t = t0; t < t1; ++t) {
        const uint32_t dv = bit_of(fpb, t, G, g, r);
        const uint32_t sl = bit_of(tmb, t, G, g, r);
        if (dv) {
            if (v.first_div < 0) v.first_div = (int32_t)t;
            ++v.div_count;
        }
        v.slow_count += sl;
        if (sl && prev) v.flags |= 4u;
        prev = sl;
    }
    // the pair (t1 - 1, t1) belongs to this segment
    if (t1 < T && prev && bit_of(tmb, t1, G, g, r)) v.flags |= 4u;
    // windows starting in [t0, min(t1, T - Wt + 1))
    const int64_t s_end = min(t1, T - Wt + 1);
    if (Wt > 0 && t0 < s_end) {
        uint32_t c = 0;
        for (int64_t t = t0; t < t0 + Wt; ++t) c += bit_of(tmb, t, G, g, r);
        for (int64_t s = t0;; ++s) {
            if (c > v.max_window) v.max_window = c;
            if (2 * (int64_t)c > Wt && v.first_window < 0) v.first_window = (int32_t)s;
            if (s + 1 >= s_end) break;
            c += bit_of(tmb, s + Wt, G, g, r);
            c -= bit_of(tmb, s, G, g, r);
        }
    }
    out[idx] = v;
}

__global__ void __launch_bounds__(kConfThreads) confirm_combine_kernel(
    const SegVerdict* __restrict__ seg, int64_t n_ranks, int64_t n_seg,
    c3_rank_verdict_t* __restrict__ verdicts) {
    const int64_t rank = (int64_t)blockIdx.x * kConfThreads + threadIdx.x;
    if (rank >= n_ranks) return;
    uint32_t fl = 0, dc = 0, sc = 0, mw = 0;
    int32_t fd = -1, fw = -1;
    for (int64_t s = 0; s < n_seg; ++s) {
        const SegVerdict v = seg[s * n_ranks + rank];
        fl |= v.flags;
        dc += v.div_count;
        sc += v.slow_count;
        mw = max(mw, v.max_window);
        if (fd < 0) fd = v.first_div;
        if (fw < 0) fw = v.first_window;
    }
    if (fw >= 0) fl |= C3_RANK_STRAGGLER;
    if (fd >= 0) fl |= C3_RANK_PROTOCOL;
    c3_rank_verdict_t out;
    out.flags = fl;
    out.first_divergent_iter = fd;
    out.divergent_count = dc;
    out.slow_count = sc;
    out.max_window_slow = mw;
    out.first_straggler_window = fw;
    verdicts[rank] = out;
}

size_t confirm_ws_bytes(int R, int64_t G, int64_t T) {
    const int64_t n_seg = T > 0 ? (T + kSeg - 1) / kSeg : 1;
    return (size_t)(n_seg * (int64_t)R * G * (int64_t)sizeof(SegVerdict)) + 256;
}

hipError_t launch_confirm(const uint64_t* fp_bitmap, const uint64_t* time_bitmap, int R, int64_t G,
                          int64_t T, int window, c3_rank_verdict_t* verdicts, void* ws,
                          hipStream_t stream) {
    const int64_t n_ranks = (int64_t)R * G;
    if (n_ranks == 0) return hipSuccess;
    const int64_t n_seg = T > 0 ? (T + kSeg - 1) / kSeg : 1;
    const int64_t Wt = (int64_t)window < T ? (int64_t)window : T;
    SegVerdict* seg = static_cast<SegVerdict*>(ws);
    const int64_t threads1 = n_ranks * n_seg;
    const int64_t blocks1 = (threads1 + kConfThreads - 1) / kConfThreads;
    if (blocks1 > 0x7FFFFFFF) return hipErrorInvalidValue;
    hipLaunchKernelGGL(confirm_segment_kernel, dim3((unsigned)blocks1), dim3(kConfThreads), 0, stream,
                       fp_bitmap, time_bitmap, R, G, T, Wt, n_seg, seg);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int64_t blocks2 = (n_ranks + kConfThreads - 1) / kConfThreads;
    hipLaunchKernelGGL(confirm_combine_kernel, dim3((unsigned)blocks2), dim3(kConfThreads), 0, stream,
                       seg, n_ranks, n_seg, verdicts);
    return hipGetLastError();
}

}  // namespace c3
