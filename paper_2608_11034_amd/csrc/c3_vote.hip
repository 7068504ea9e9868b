// Consensus kernels of C3 for gfx950: the decision step of Algorithm 1.
//
// Groups of up to 16 replicas: one thread per unit, the R values in
// registers (128-bit row loads when replicas are adjacent), order
// statistics from min/max bitonic sorting networks, and the lower-median
// replica from counts in the stable (value, replica) order.  Larger groups:
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

namespace c3 {

constexpr int kVoteThreads = 256;

__device__ inline uint64_t load_ev_bits(const char* p, int kind) {
    if (kind == C3_EV_U64 || kind == C3_EV_F64) return *reinterpret_cast<const uint64_t*>(p);
    return *reinterpret_cast<const uint32_t*>(p);
}

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
typedef uint32_t vu32x4 __attribute__((ext_vector_type(4)));

// Raw bits of the R values of one unit (4-byte kinds zero-extended).  With
// `dense` the replicas are adjacent and the row is 16-byte aligned and a
// whole number of 16-byte words, so it is read with 128-bit loads.
template <int NMAX>
__device__ __forceinline__ void load_row_bits(const char* base, int kind, int64_t rstride, int R,
                                              bool dense, uint64_t (&e)[NMAX]) {
    const bool wide = kind == C3_EV_U64 || kind == C3_EV_F64;
    if (dense && wide) {
#pragma unroll
        for (int j = 0; j < NMAX / 2; ++j) {
            vu32x4 v = {0u, 0u, 0u, 0u};
            if (2 * j < R) v = *reinterpret_cast<const vu32x4*>(base + 16 * j);
            e[2 * j] = ((uint64_t)v.y << 32) | v.x;
            e[2 * j + 1] = ((uint64_t)v.w << 32) | v.z;
        }
    } else if (dense && NMAX >= 4) {
#pragma unroll
        for (int j = 0; j < NMAX / 4; ++j) {
            vu32x4 v = {0u, 0u, 0u, 0u};
            if (4 * j < R) v = *reinterpret_cast<const vu32x4*>(base + 16 * j);
            e[4 * j] = v.x;
            e[4 * j + 1] = v.y;
            e[4 * j + 2] = v.z;
            e[4 * j + 3] = v.w;
        }
    } else {
#pragma unroll
        for (int r = 0; r < NMAX; ++r)
            e[r] = r < R ? load_ev_bits(base + (int64_t)r * rstride, kind) : 0ull;
    }
}

template <int NMAX>
__global__ void __launch_bounds__(kVoteThreads) exact_vote_small_kernel(
    const char* __restrict__ ev, int kind, int64_t rstride, int64_t ustride, int R, int64_t n_units,
    bool dense, uint8_t* __restrict__ status, uint64_t* __restrict__ bitmap,
    int32_t* __restrict__ majority_idx) {
    const int64_t u = (int64_t)blockIdx.x * kVoteThreads + threadIdx.x;
    if (u >= n_units) return;
    uint64_t e[NMAX];
    load_row_bits<NMAX>(ev + u * ustride, kind, rstride, R, dense, e);
    uint64_t maj = 0, other = 0;
#pragma unroll
    for (int r = 0; r < NMAX; ++r) {
        int cnt = 0;
#pragma unroll
        for (int j = 0; j < NMAX; ++j) cnt += (j < R && e[j] == e[r]) ? 1 : 0;
        if (r < R) {
            if (2 * cnt > R) maj |= 1ull << r; else other |= 1ull << r;
        }
    }
    if (maj == 0) {
        status[u] = C3_INCONCLUSIVE;
        bitmap[u] = 0;
        majority_idx[u] = -1;
    } else {
        status[u] = other ? C3_ATTRIBUTED : C3_AGREE;
        bitmap[u] = other;
        majority_idx[u] = __builtin_ctzll(maj);
    }
}

// Bitonic sorting network over N register slots (N a power of two, values
// without NaN): each comparator is one min and one max.
template <int N>
__device__ __forceinline__ void bitonic_sort(double (&v)[N]) {
    constexpr int LOG = N == 2 ? 1 : N == 4 ? 2 : N == 8 ? 3 : 4;
    static_assert((1 << LOG) == N, "power of two up to 16");
#pragma unroll
    for (int kk = 1; kk <= LOG; ++kk) {
#pragma unroll
        for (int jj = kk - 1; jj >= 0; --jj) {
#pragma unroll
            for (int i = 0; i < N; ++i) {
                const int l = i ^ (1 << jj);
                if (l > i) {
                    const double lo = fmin(v[i], v[l]), hi = fmax(v[i], v[l]);
                    const bool up = (i & (1 << kk)) == 0;
                    v[i] = up ? lo : hi;
                    v[l] = up ? hi : lo;
                }
            }
        }
    }
}

// v[k] for a run-time k, as an OR of masked slots.  A select chain would be
// turned back into an indexed load, which puts the array in scratch memory.
template <int N>
__device__ __forceinline__ double pick(const double (&v)[N], int k) {
    uint64_t out = 0;
#pragma unroll
    for (int i = 0; i < N; ++i) {
        const uint64_t m = 0ull - (uint64_t)(i == k);
        out |= m & (uint64_t)__double_as_longlong(v[i]);
    }
    return __longlong_as_double((long long)out);
}

template <int N>
__device__ __forceinline__ double median_sorted(const double (&s)[N], int n) {
    if (n & 1) return pick<N>(s, (n - 1) / 2);
    return (pick<N>(s, n / 2 - 1) + pick<N>(s, n / 2)) * 0.5;
}

template <int N>
__device__ __forceinline__ double quantile7_sorted(const double (&s)[N], int n, double p) {
    const double h = (double)(n - 1) * p;
    const double fl = floor(h);
    const int lo = (int)fl;
    const double frac = h - fl;
    if (lo + 1 >= n) return pick<N>(s, n - 1);
    const double a = pick<N>(s, lo);
    const double b = pick<N>(s, lo + 1);
    const double diff = b - a;
    const double prod = frac * diff;
    return a + prod;
}

template <int NMAX>
__global__ void __launch_bounds__(kVoteThreads) statistical_vote_small_kernel(
    const char* __restrict__ ev, int kind, int64_t rstride, int64_t ustride, int R, int64_t n_units,
    bool dense, double kappa, uint8_t* __restrict__ status, uint64_t* __restrict__ bitmap,
    int32_t* __restrict__ majority_idx) {
    const int64_t u = (int64_t)blockIdx.x * kVoteThreads + threadIdx.x;
    if (u >= n_units) return;
    const double inf = __builtin_huge_val();
    uint64_t bits[NMAX];
    load_row_bits<NMAX>(ev + u * ustride, kind, rstride, R, dense, bits);
    double x[NMAX], s[NMAX];
    uint64_t fin = 0;
#pragma unroll
    for (int r = 0; r < NMAX; ++r) {
        x[r] = kind == C3_EV_F32 ? (double)__uint_as_float((uint32_t)bits[r])
                                 : __longlong_as_double((long long)bits[r]);
        const bool f = r < R && __builtin_isfinite(x[r]);
        fin |= (uint64_t)f << r;
        s[r] = f ? x[r] : inf;      // excluded values sort after every finite one
    }
    const uint64_t valid = R == 64 ? ~0ull : ((1ull << R) - 1);
    const uint64_t nonfin = valid & ~fin;
    const int nf = __builtin_popcountll(fin);
    if (2 * nf <= R) {
        status[u] = C3_INCONCLUSIVE;
        bitmap[u] = 0;
        majority_idx[u] = -1;
        return;
    }
    bitonic_sort<NMAX>(s);
    const double m = median_sorted<NMAX>(s, nf);
    double dev[NMAX], ds[NMAX];
#pragma unroll
    for (int r = 0; r < NMAX; ++r) {
        dev[r] = ((fin >> r) & 1ull) ? fabs(x[r] - m) : inf;
        ds[r] = dev[r];
    }
    bitonic_sort<NMAX>(ds);
    double d = median_sorted<NMAX>(ds, nf);
    if (d == 0.0) {
        const double q3 = quantile7_sorted<NMAX>(s, nf, 0.75);
        const double q1 = quantile7_sorted<NMAX>(s, nf, 0.25);
        d = (q3 - q1) * 0.5;
    }
    if (d == 0.0) d = (pick<NMAX>(s, nf - 1) - s[0]) / (double)nf;
    uint64_t B = nonfin;
    if (d != 0.0) {
        const double thr = kappa * d;
#pragma unroll
        for (int r = 0; r < NMAX; ++r)
            if (((fin >> r) & 1ull) && dev[r] > thr) B |= 1ull << r;
    }
    // lower-median replica: stable position (nf - 1) / 2 in (value, replica) order
    const double target = pick<NMAX>(s, (nf - 1) / 2);
    int want = (nf - 1) / 2;
#pragma unroll
    for (int r = 0; r < NMAX; ++r) want -= (((fin >> r) & 1ull) && x[r] < target) ? 1 : 0;
    int med = -1;
#pragma unroll
    for (int r = 0; r < NMAX; ++r) {
        if (((fin >> r) & 1ull) && x[r] == target) {
            if (want == 0 && med < 0) med = r;
            --want;
        }
    }
    status[u] = B ? C3_ATTRIBUTED : C3_AGREE;
    bitmap[u] = B;
    majority_idx[u] = med;
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
    else
        hipLaunchKernelGGL(statistical_vote_small_kernel<NMAX>, dim3(blocks), dim3(kVoteThreads), 0,
                           stream, ev, kind, rstride, ustride, R, n_units, dense, kappa, status,
                           bitmap, majority_idx);
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
