// Consensus kernels of C3 for gfx950: the decision step of Algorithm 1.
//
// Groups of up to 16 replicas: one thread per unit, the R values in
// registers (128-bit row loads when replicas are adjacent), deciding with
// the per-unit functions of c3_vote_row.h.  Larger groups:
//
// Layout: one lane per (unit, replica).  A unit's R values sit in a group of
// W = next_pow2(R) consecutive lanes of one wave64 (64 / W units per wave),
// so every comparison among peers is a cross-lane shuffle and every set of
// peers is a slice of one 64-bit ballot.  Lanes past R (and past the last
// unit) stay active for the shuffles and are masked out of every ballot.
//
// EXACT (Sec. 5.3): each lane counts the peers whose value equals its own.
// A strict majority exists iff some lane's count c satisfies 2c > R; then
// the majority lanes are exactly those with 2c > R (the value held by more
// than half the peers is unique), the outlier bitmap is the ballot of the
// other valid lanes, and the majority index is the lowest majority lane.
//
// STATISTICAL (Sec. 5.4), in fp64: a lane's stable rank among the finite
// values (value, then replica index) gives every order statistic by one
// ballot and one shuffle: the median, the median absolute deviation, the
// type-7 quartiles and the range, in the fallback order MAD -> IQR / 2 ->
// range / n_finite.  Non-finite values are outliers and take no part in m
// or d.  No floating-point contraction is allowed in this file (the host
// compiles it with -ffp-contract=off), so the decision rounds exactly as the
// plain definition does.
#include "c3_device.h"
#include "c3_internal.h"
#include "c3_vote_row.h"

namespace c3 {

constexpr int kVoteThreads = 256;

__device__ inline double load_ev_f64(const char* p, int kind) {
    if (kind == C3_EV_F32) return (double)*reinterpret_cast<const float*>(p);
    return *reinterpret_cast<const double*>(p);
}

__device__ inline uint64_t group_bits(uint64_t ballot, int gbase, uint64_t gmask) {
    return (ballot >> gbase) & gmask;
}

__global__ void __launch_bounds__(kVoteThreads) exact_vote_kernel(
    const char* __restrict__ ev, int kind, int64_t rstride, int64_t ustride, int R, int gw_log2,
    int64_t n_units, uint8_t* __restrict__ status, uint64_t* __restrict__ bitmap,
    int32_t* __restrict__ majority_idx) {
    const int gw = 1 << gw_log2;
    const int lane = threadIdx.x & 63;
    const int r = lane & (gw - 1);
    const int gbase = lane - r;
    const uint64_t gmask = gw == 64 ? ~0ull : ((1ull << gw) - 1);
    const int64_t units_per_block = (int64_t)(kVoteThreads >> gw_log2);
    const int64_t u = (int64_t)blockIdx.x * units_per_block + (threadIdx.x >> gw_log2);
    const bool valid = u < n_units && r < R;
    const uint64_t e = valid ? load_ev_bits(ev + u * ustride + (int64_t)r * rstride, kind) : 0ull;
    int cnt = 0;
    for (int j = 0; j < R; ++j) cnt += (shfl_u64(e, gbase + j) == e) ? 1 : 0;
    const bool maj = valid && 2 * cnt > R;
    const uint64_t mb = group_bits(ballot64(maj), gbase, gmask);
    const uint64_t ob = group_bits(ballot64(valid && !maj), gbase, gmask);
    if (valid && r == 0) {
        if (mb == 0) {
            status[u] = C3_INCONCLUSIVE;
            bitmap[u] = 0;
            majority_idx[u] = -1;
        } else {
            status[u] = ob ? C3_ATTRIBUTED : C3_AGREE;
            bitmap[u] = ob;
            majority_idx[u] = __builtin_ctzll(mb);
        }
    }
}

// Order statistic k (0-based) of the finite values of a lane group, given
// every lane's stable rank among them.
__device__ inline double order_stat(double x, bool fin, int rank, int k, int gbase, uint64_t gmask) {
    const uint64_t b = group_bits(ballot64(fin && rank == k), gbase, gmask);
    const int src = gbase + (b ? __builtin_ctzll(b) : 0);
    return shfl_f64(x, src);
}

__device__ inline int stable_rank(double x, bool fin, int R, int r, int gbase) {
    int rank = 0;
    for (int j = 0; j < R; ++j) {
        const double y = shfl_f64(x, gbase + j);
        const bool fy = __shfl((int)fin, gbase + j, 64) != 0;
        rank += (fy && (y < x || (y == x && j < r))) ? 1 : 0;
    }
    return rank;
}

__device__ inline double median_of(double x, bool fin, int rank, int nf, int gbase, uint64_t gmask) {
    if (nf & 1) return order_stat(x, fin, rank, (nf - 1) / 2, gbase, gmask);
    const double a = order_stat(x, fin, rank, nf / 2 - 1, gbase, gmask);
    const double b = order_stat(x, fin, rank, nf / 2, gbase, gmask);
    return (a + b) * 0.5;
}

// Hyndman-Fan type 7: h = (n - 1) p; Q = s[floor h] + frac(h) (s[floor h + 1] - s[floor h]).
__device__ inline double quantile7(double x, bool fin, int rank, int nf, double p, int gbase,
                                   uint64_t gmask) {
    const double h = (double)(nf - 1) * p;
    const double fl = floor(h);
    const int lo = (int)fl;
    const double frac = h - fl;
    if (lo + 1 >= nf) return order_stat(x, fin, rank, nf - 1, gbase, gmask);
    const double a = order_stat(x, fin, rank, lo, gbase, gmask);
    const double b = order_stat(x, fin, rank, lo + 1, gbase, gmask);
    const double diff = b - a;
    const double prod = frac * diff;
    return a + prod;
}

__global__ void __launch_bounds__(kVoteThreads) statistical_vote_kernel(
    const char* __restrict__ ev, int kind, int64_t rstride, int64_t ustride, int R, int gw_log2,
    int64_t n_units, double kappa, uint8_t* __restrict__ status, uint64_t* __restrict__ bitmap,
    int32_t* __restrict__ majority_idx) {
    const int gw = 1 << gw_log2;
    const int lane = threadIdx.x & 63;
    const int r = lane & (gw - 1);
    const int gbase = lane - r;
    const uint64_t gmask = gw == 64 ? ~0ull : ((1ull << gw) - 1);
    const int64_t units_per_block = (int64_t)(kVoteThreads >> gw_log2);
    const int64_t u = (int64_t)blockIdx.x * units_per_block + (threadIdx.x >> gw_log2);
    const bool valid = u < n_units && r < R;
    const double x = valid ? load_ev_f64(ev + u * ustride + (int64_t)r * rstride, kind) : 0.0;
    const bool fin = valid && __builtin_isfinite(x);
    const uint64_t finb = group_bits(ballot64(fin), gbase, gmask);
    const uint64_t nonfin = group_bits(ballot64(valid && !fin), gbase, gmask);
    const int nf = __builtin_popcountll(finb);
    if (2 * nf <= R) {  // finite values are not a strict majority
        if (valid && r == 0) {
            status[u] = C3_INCONCLUSIVE;
            bitmap[u] = 0;
            majority_idx[u] = -1;
        }
        return;
    }
    const int rank = stable_rank(x, fin, R, r, gbase);
    const double m = median_of(x, fin, rank, nf, gbase, gmask);
    const double dev = fin ? fabs(x - m) : 0.0;
    const int drank = stable_rank(dev, fin, R, r, gbase);
    double d = median_of(dev, fin, drank, nf, gbase, gmask);
    if (d == 0.0) {
        const double q3 = quantile7(x, fin, rank, nf, 0.75, gbase, gmask);
        const double q1 = quantile7(x, fin, rank, nf, 0.25, gbase, gmask);
        d = (q3 - q1) * 0.5;
    }
    if (d == 0.0) {
        const double hi = order_stat(x, fin, rank, nf - 1, gbase, gmask);
        const double lo = order_stat(x, fin, rank, 0, gbase, gmask);
        d = (hi - lo) / (double)nf;
    }
    bool flag = false;
    if (d != 0.0) {
        const double thr = kappa * d;
        flag = fin && dev > thr;
    }
    const uint64_t B = nonfin | group_bits(ballot64(flag), gbase, gmask);
    const uint64_t medb = group_bits(ballot64(fin && rank == (nf - 1) / 2), gbase, gmask);
    if (valid && r == 0) {
        status[u] = B ? C3_ATTRIBUTED : C3_AGREE;
        bitmap[u] = B;
        majority_idx[u] = medb ? __builtin_ctzll(medb) : -1;
    }
}

// ---------------------------------------------------------------------------
// Small groups (R <= 16): one thread per unit with the R values in registers.
// Cross-lane traffic dominates the lane-per-replica kernels at these sizes;
// here the whole decision is register arithmetic.  NMAX is R rounded up to
// a power of two; slots past R are padding that never takes part.
// ---------------------------------------------------------------------------
template <int NMAX>
__global__ void __launch_bounds__(kVoteThreads) exact_vote_small_kernel(
    const char* __restrict__ ev, int kind, int64_t rstride, int64_t ustride, int R, int64_t n_units,
    bool dense, uint8_t* __restrict__ status, uint64_t* __restrict__ bitmap,
    int32_t* __restrict__ majority_idx) {
    const int64_t u = (int64_t)blockIdx.x * kVoteThreads + threadIdx.x;
    if (u >= n_units) return;
    uint64_t e[NMAX];
    load_row_bits<NMAX>(ev + u * ustride, kind, rstride, R, dense, e);
    const UnitVote v = exact_vote_row<NMAX>(e, R);
    status[u] = v.status;
    bitmap[u] = v.bitmap;
    majority_idx[u] = v.majority;
}

template <int NMAX, int KIND>
__global__ void __launch_bounds__(kVoteThreads) statistical_vote_small_kernel(
    const char* __restrict__ ev, int kind, int64_t rstride, int64_t ustride, int R, int64_t n_units,
    bool dense, double kappa, uint8_t* __restrict__ status, uint64_t* __restrict__ bitmap,
    int32_t* __restrict__ majority_idx) {
    const int64_t u = (int64_t)blockIdx.x * kVoteThreads + threadIdx.x;
    if (u >= n_units) return;
    uint64_t bits[NMAX];
    load_row_bits<NMAX>(ev + u * ustride, kind, rstride, R, dense, bits);
    const UnitVote v = statistical_vote_row<NMAX, KIND>(bits, R, kappa);
    status[u] = v.status;
    bitmap[u] = v.bitmap;
    majority_idx[u] = v.majority;
}

template <int NMAX>
static void launch_small(const char* ev, int kind, int64_t rstride, int64_t ustride, int R,
                         int64_t n_units, int mode, double kappa, uint8_t* status, uint64_t* bitmap,
                         int32_t* majority_idx, hipStream_t stream, unsigned blocks) {
    const int64_t vsize = (kind == C3_EV_U64 || kind == C3_EV_F64) ? 8 : 4;
    const bool dense = rstride == vsize && ((int64_t)R * vsize) % 16 == 0 && ustride % 16 == 0 &&
                       ((uintptr_t)ev & 15) == 0;
    if (mode == C3_EXACT)
        hipLaunchKernelGGL(exact_vote_small_kernel<NMAX>, dim3(blocks), dim3(kVoteThreads), 0, stream,
                           ev, kind, rstride, ustride, R, n_units, dense, status, bitmap,
                           majority_idx);
    else if (kind == C3_EV_F32)
        hipLaunchKernelGGL((statistical_vote_small_kernel<NMAX, C3_EV_F32>), dim3(blocks),
                           dim3(kVoteThreads), 0, stream, ev, kind, rstride, ustride, R, n_units,
                           dense, kappa, status, bitmap, majority_idx);
    else
        hipLaunchKernelGGL((statistical_vote_small_kernel<NMAX, C3_EV_F64>), dim3(blocks),
                           dim3(kVoteThreads), 0, stream, ev, kind, rstride, ustride, R, n_units,
                           dense, kappa, status, bitmap, majority_idx);
}

hipError_t launch_consensus(const void* evidence, int kind, int64_t rstride, int64_t ustride, int R,
                            int64_t n_units, int mode, double kappa, uint8_t* status,
                            uint64_t* bitmap, int32_t* majority_idx, hipStream_t stream) {
    if (n_units <= 0) return hipSuccess;
    if (R <= 16) {
        const int64_t blocks = (n_units + kVoteThreads - 1) / kVoteThreads;
        if (blocks > 0x7FFFFFFF) return hipErrorInvalidValue;
        const char* e = static_cast<const char*>(evidence);
        if (R <= 4)
            launch_small<4>(e, kind, rstride, ustride, R, n_units, mode, kappa, status, bitmap,
                            majority_idx, stream, (unsigned)blocks);
        else if (R <= 8)
            launch_small<8>(e, kind, rstride, ustride, R, n_units, mode, kappa, status, bitmap,
                            majority_idx, stream, (unsigned)blocks);
        else
            launch_small<16>(e, kind, rstride, ustride, R, n_units, mode, kappa, status, bitmap,
                             majority_idx, stream, (unsigned)blocks);
        return hipGetLastError();
    }
    int gw_log2 = 0;
    while ((1 << gw_log2) < R) ++gw_log2;
    const int64_t units_per_block = kVoteThreads >> gw_log2;
    const int64_t blocks = (n_units + units_per_block - 1) / units_per_block;
    if (blocks > 0x7FFFFFFF) return hipErrorInvalidValue;
    if (mode == C3_EXACT) {
        hipLaunchKernelGGL(exact_vote_kernel, dim3((unsigned)blocks), dim3(kVoteThreads), 0, stream,
                           static_cast<const char*>(evidence), kind, rstride, ustride, R, gw_log2,
                           n_units, status, bitmap, majority_idx);
    } else {
        hipLaunchKernelGGL(statistical_vote_kernel, dim3((unsigned)blocks), dim3(kVoteThreads), 0,
                           stream, static_cast<const char*>(evidence), kind, rstride, ustride, R,
                           gw_log2, n_units, kappa, status, bitmap, majority_idx);
    }
    return hipGetLastError();
}

}  // namespace c3
