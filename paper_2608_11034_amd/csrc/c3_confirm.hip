// Temporal confirmation of C3 results for gfx950.
//
// Input: per-iteration outlier bitmaps of G peer groups (u64 per (t, g)) for
// fingerprints (exact C3) and timings (statistical C3).  Output: one verdict
// per rank, rank = r * G + g.
//
// Pass 1: one thread per (segment, rank); a segment is kSeg consecutive
// iterations.  Threads are ordered (segment, group, replica), so the R
// threads of one group are adjacent lanes reading the same bitmap word and
// a wave's load touches 64 / R consecutive words.  The thread counts
// attributed iterations in its
// segment, notes the first attributed fingerprint and any two consecutive
// attributed timings (the pair (t, t + 1) belongs to the segment of t), and
// slides a window of W iterations over the window starts in its segment
// (reading up to W - 1 iterations, and at least one, into the next segment).  For W <= 64 the
// thread first gathers its bits of the segment (and the next W - 1
// iterations) into 64-bit masks with independent loads, then works on the
// masks with shifts and popcounts; longer windows walk the bitmaps.
// Pass 2: one thread per rank combines its segments in order.  Partial
// results are stored [segment][group][replica], in pass-1 thread order.
#include "c3_device.h"
#include "c3_internal.h"

namespace c3 {

constexpr int64_t kSeg = 64;
#ifndef C3_CONFIRM_GROUP_SEG
#define C3_CONFIRM_GROUP_SEG 32
#endif
constexpr int kGroupSeg = C3_CONFIRM_GROUP_SEG;   // segment of the per-group kernel
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
    const int64_t gr = idx - sgi * n_ranks;      // g * R + r
    const int64_t g = gr / R;
    const int r = (int)(gr - g * R);
    const int64_t t0 = sgi * kSeg;
    const int64_t t1 = min(T, t0 + kSeg);
    SegVerdict v{0u, -1, 0u, 0u, 0u, -1};
    if (Wt <= 64) {
        // Gather this rank's bits with independent loads: bit i of lo/div is
        // iteration t0 + i (i < 64), bit i of hi is iteration t0 + 64 + i.
        uint64_t div = 0, lo = 0, hi = 0;
#pragma unroll
        for (int i = 0; i < kSeg; ++i) {
            const int64_t t = t0 + i;
            if (t < t1) {
                div |= (uint64_t)bit_of(fpb, t, G, g, r) << i;
                lo |= (uint64_t)bit_of(tmb, t, G, g, r) << i;
            }
        }
        // iterations read past the segment: by its windows, and t1 for the
        // pair (t1 - 1, t1) even when W = 1
        const int64_t t_hi_end = min(T, t1 + (Wt > 1 ? Wt - 1 : 1));
#pragma unroll
        for (int i = 0; i < kSeg - 1; ++i) {
            const int64_t t = t0 + kSeg + i;
            if (t < t_hi_end) hi |= (uint64_t)bit_of(tmb, t, G, g, r) << i;
        }
        v.div_count = (uint32_t)__builtin_popcountll(div);
        v.first_div = div ? (int32_t)(t0 + __builtin_ctzll(div)) : -1;
        v.slow_count = (uint32_t)__builtin_popcountll(lo);
        // pairs (t, t + 1) with t in the segment; bits past T are zero
        if ((lo & (lo >> 1)) != 0 || ((lo >> 63) & hi & 1ull) != 0) v.flags |= 4u;
        const int64_t s_end = min(t1, T - Wt + 1);
        const uint64_t wmask = Wt == 64 ? ~0ull : ((1ull << Wt) - 1);
        for (int64_t s0 = t0; s0 < s_end; ++s0) {
            const int off = (int)(s0 - t0);
            const uint64_t w = off == 0 ? lo : ((lo >> off) | (hi << (64 - off)));
            const uint32_t c = (uint32_t)__builtin_popcountll(w & wmask);
            if (c > v.max_window) v.max_window = c;
            if (2 * (int64_t)c > Wt && v.first_window < 0) v.first_window = (int32_t)s0;
        }
        out[idx] = v;
        return;
    }
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

// Groups of up to RMAX replicas with W <= 64: one thread per (segment,
// group) reads each bitmap word once and transposes it into per-replica
// 64-bit masks over iterations (lo/div: t0 + i; hi: t0 + 64 + i), then
// evaluates every replica's counts and windows with shifts and popcounts.
// Results go to the same [segment][group][replica] slots as the general
// kernel.
template <int RMAX, int SEG>
__global__ void __launch_bounds__(kConfThreads) confirm_group_kernel(
    const uint64_t* __restrict__ fpb, const uint64_t* __restrict__ tmb, int R, int64_t G, int64_t T,
    int64_t Wt, int64_t n_seg, SegVerdict* __restrict__ out) {
    const int64_t idx = (int64_t)blockIdx.x * kConfThreads + threadIdx.x;
    if (idx >= n_seg * G) return;
    const int64_t sgi = idx / G;
    const int64_t g = idx - sgi * G;
    const int64_t t0 = sgi * SEG;
    const int64_t t1 = min(T, t0 + SEG);
    // read past the segment for its windows, and t1 for the pair (t1 - 1, t1)
    const int64_t t_hi_end = min(T, t1 + (Wt > 1 ? Wt - 1 : 1));
    uint64_t div[RMAX], lo[RMAX], hi[RMAX];
#pragma unroll
    for (int r = 0; r < RMAX; ++r) div[r] = lo[r] = hi[r] = 0;
    const uint64_t* fp = fpb + t0 * G + g;
    const uint64_t* tm = tmb + t0 * G + g;
    const int nlo = (int)(t1 - t0);
    if (nlo == SEG) {
        // full segment: fixed trip count, so the loads are issued ahead
#pragma unroll 16
        for (int i = 0; i < SEG; ++i) {
            const uint64_t fw = fp[(int64_t)i * G], tw = tm[(int64_t)i * G];
#pragma unroll
            for (int r = 0; r < RMAX; ++r) {
                div[r] |= ((fw >> r) & 1ull) << i;
                lo[r] |= ((tw >> r) & 1ull) << i;
            }
        }
    } else {
        for (int i = 0; i < nlo; ++i) {
            const uint64_t fw = fp[(int64_t)i * G], tw = tm[(int64_t)i * G];
#pragma unroll
            for (int r = 0; r < RMAX; ++r) {
                div[r] |= ((fw >> r) & 1ull) << i;
                lo[r] |= ((tw >> r) & 1ull) << i;
            }
        }
    }
    const int nhi = t_hi_end > t0 + SEG ? (int)(t_hi_end - t0 - SEG) : 0;
#pragma unroll 8
    for (int i = 0; i < nhi; ++i) {
        const uint64_t tw = tm[(int64_t)(SEG + i) * G];
#pragma unroll
        for (int r = 0; r < RMAX; ++r) hi[r] |= ((tw >> r) & 1ull) << i;
    }
    const int64_t s_end = min(t1, T - Wt + 1);
    const uint64_t wmask = Wt == 64 ? ~0ull : ((1ull << Wt) - 1);
    const uint64_t seg_mask = SEG == 64 ? ~0ull : ((1ull << SEG) - 1);
    SegVerdict* o = out + sgi * (int64_t)R * G + g * R;
#pragma unroll
    for (int r = 0; r < RMAX; ++r) {
        if (r >= R) break;
        // 128-bit run of timing bits: bit i is iteration t0 + i
        const uint64_t b0 = SEG == 64 ? lo[r] : (lo[r] | (hi[r] << (SEG & 63)));
        const uint64_t b1 = SEG == 64 ? hi[r] : (hi[r] >> ((64 - SEG) & 63));
        SegVerdict v{0u, -1, 0u, 0u, 0u, -1};
        v.div_count = (uint32_t)__builtin_popcountll(div[r]);
        v.first_div = div[r] ? (int32_t)(t0 + __builtin_ctzll(div[r])) : -1;
        v.slow_count = (uint32_t)__builtin_popcountll(lo[r]);
        // pairs (t, t + 1) with t in the segment; bits past T are zero
        const uint64_t pairs = b0 & ((b0 >> 1) | (b1 << 63)) & seg_mask;
        if (pairs != 0) v.flags |= 4u;
        for (int64_t s0 = t0; s0 < s_end; ++s0) {
            const int off = (int)(s0 - t0);
            const uint64_t w = off == 0 ? b0 : ((b0 >> off) | (b1 << (64 - off)));
            const uint32_t c = (uint32_t)__builtin_popcountll(w & wmask);
            if (c > v.max_window) v.max_window = c;
            if (2 * (int64_t)c > Wt && v.first_window < 0) v.first_window = (int32_t)s0;
        }
        o[r] = v;
    }
}

__global__ void __launch_bounds__(kConfThreads) confirm_combine_kernel(
    const SegVerdict* __restrict__ seg, int R, int64_t G, int64_t n_ranks, int64_t n_seg,
    c3_rank_verdict_t* __restrict__ verdicts) {
    const int64_t rank = (int64_t)blockIdx.x * kConfThreads + threadIdx.x;
    if (rank >= n_ranks) return;
    const int64_t r = rank / G;
    const int64_t g = rank - r * G;
    const int64_t gr = g * R + r;               // position inside a segment's block
    uint32_t fl = 0, dc = 0, sc = 0, mw = 0;
    int32_t fd = -1, fw = -1;
#pragma unroll 4
    for (int64_t s = 0; s < n_seg; ++s) {
        const SegVerdict v = seg[s * n_ranks + gr];
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
    const int64_t seg_len = kGroupSeg < kSeg ? kGroupSeg : kSeg;
    const int64_t n_seg = T > 0 ? (T + seg_len - 1) / seg_len : 1;
    return (size_t)(n_seg * (int64_t)R * G * (int64_t)sizeof(SegVerdict)) + 256;
}

hipError_t launch_confirm(const uint64_t* fp_bitmap, const uint64_t* time_bitmap, int R, int64_t G,
                          int64_t T, int window, c3_rank_verdict_t* verdicts, void* ws,
                          hipStream_t stream) {
    const int64_t n_ranks = (int64_t)R * G;
    if (n_ranks == 0) return hipSuccess;
    const int64_t Wt = (int64_t)window < T ? (int64_t)window : T;
    SegVerdict* seg = static_cast<SegVerdict*>(ws);
    const bool by_group = R <= 16 && Wt <= 64;
    const int64_t seg_len = by_group ? kGroupSeg : kSeg;
    const int64_t n_seg = T > 0 ? (T + seg_len - 1) / seg_len : 1;
    const int64_t threads1 = (by_group ? G : n_ranks) * n_seg;
    const int64_t blocks1 = (threads1 + kConfThreads - 1) / kConfThreads;
    if (blocks1 > 0x7FFFFFFF) return hipErrorInvalidValue;
    if (by_group && R <= 8)
        hipLaunchKernelGGL((confirm_group_kernel<8, kGroupSeg>), dim3((unsigned)blocks1),
                           dim3(kConfThreads), 0, stream, fp_bitmap, time_bitmap, R, G, T, Wt, n_seg,
                           seg);
    else if (by_group)
        hipLaunchKernelGGL((confirm_group_kernel<16, kGroupSeg>), dim3((unsigned)blocks1),
                           dim3(kConfThreads), 0, stream, fp_bitmap, time_bitmap, R, G, T, Wt, n_seg,
                           seg);
    else
        hipLaunchKernelGGL(confirm_segment_kernel, dim3((unsigned)blocks1), dim3(kConfThreads), 0,
                           stream, fp_bitmap, time_bitmap, R, G, T, Wt, n_seg, seg);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int64_t blocks2 = (n_ranks + kConfThreads - 1) / kConfThreads;
    hipLaunchKernelGGL(confirm_combine_kernel, dim3((unsigned)blocks2), dim3(kConfThreads), 0, stream,
                       seg, R, G, n_ranks, n_seg, verdicts);
    return hipGetLastError();
}

}  // namespace c3
