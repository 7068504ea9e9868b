// Consensus kernels of C3 for gfx950: the decision step of Algorithm 1.
//
// Which kernel decides a unit depends on the group size R:
//   R <= 16            one thread per unit, the R values in registers
//                      (128-bit row loads when replicas are adjacent),
//                      deciding with the per-unit functions of c3_vote_row.h;
//   EXACT, R > 16 and  one wave per unit: lane l holds replicas l, l + 64,
//   STATISTICAL,       ... (see the wave kernels below), every peer value
//   R > 32             reaches all lanes by readlane, and bitmap word s is
//                      one ballot;
//   STATISTICAL,       one lane per (unit, replica): a unit's values sit in
//   17 <= R <= 32      32 consecutive lanes, two units per wave, peers
//                      compared by shuffles.
// Measured on 1M-unit rows: the wave kernel's exact vote is 1.5x (R = 17) to
// 7.6x (R = 64) faster than lane-per-replica counting, and its statistical
// vote faster from R = 48, slower at R <= 32 where two units share a wave.
//
// EXACT (Sec. 5.3): a strict majority exists iff some value is held by more
// than R / 2 replicas; those are the majority, the bitmap marks the others
// and the majority index is the lowest majority replica.
//
// STATISTICAL (Sec. 5.4), in fp64: order statistics of the finite values in
// the stable (value, then replica index) order -- from each value's rank in
// the lane-per-replica kernel, from a sort across the wave in the wave
// kernel -- give the median, the median absolute deviation, the type-7
// quartiles and the range, in the fallback order MAD -> IQR / 2 ->
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

// ---------------------------------------------------------------------------
// Wave per unit (EXACT above 16 replicas, STATISTICAL above 32).  Lane l
// holds the values of replicas l, l + 64, l + 128 and l + 192 (NS =
// ceil(R / 64) slots; slot s holds replica 64 s + l), so bitmap word s is the
// ballot of slot s.  The exact vote broadcasts candidate values by readlane
// at a wave-uniform index; the statistical vote sorts the wave's keys.
// ---------------------------------------------------------------------------
constexpr int kWideUnitsPerBlock = kVoteThreads / 64;

__device__ inline uint64_t readlane_u64(uint64_t v, int l) {
    const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)v, l);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(v >> 32), l);
    return ((uint64_t)hi << 32) | lo;
}

__device__ inline double readlane_f64(double v, int l) {
    return __longlong_as_double((long long)readlane_u64((uint64_t)__double_as_longlong(v), l));
}

// Value of replica j (wave-uniform) from the slot registers.
template <int NS>
__device__ inline uint64_t wide_value(const uint64_t (&e)[NS], int j) {
    uint64_t v = 0;
#pragma unroll
    for (int s = 0; s < NS; ++s)
        if (s == (j >> 6)) v = readlane_u64(e[s], j & 63);
    return v;
}

template <int NS>
__device__ inline void wide_write(int64_t u, uint8_t st, const uint64_t (&b)[NS], int32_t mj,
                                  uint8_t* __restrict__ status, uint64_t* __restrict__ bitmap,
                                  int32_t* __restrict__ majority_idx) {
    if ((threadIdx.x & 63) != 0) return;
    status[u] = st;
    majority_idx[u] = mj;
#pragma unroll
    for (int s = 0; s < NS; ++s) bitmap[u * NS + s] = b[s];
}

// EXACT: a strict majority has more than R / 2 members, so one of replicas
// 0 .. floor(R / 2) holds it.  Candidate values are tried from the lowest
// such replica not yet covered, each with one broadcast and NS ballots; a
// failed value marks every replica holding it, so each distinct value is
// tried once.  The usual unit (replica 0 in the majority) needs one try, a
// two-way split two.  A unit whose candidates all fail has no strict
// majority.
template <int NS>
__global__ void __launch_bounds__(kVoteThreads) exact_vote_wide_kernel(
    const char* __restrict__ ev, int kind, int64_t rstride, int64_t ustride, int R, int64_t n_units,
    uint8_t* __restrict__ status, uint64_t* __restrict__ bitmap, int32_t* __restrict__ majority_idx) {
    const int lane = threadIdx.x & 63;
    const int64_t u = (int64_t)blockIdx.x * kWideUnitsPerBlock + (threadIdx.x >> 6);
    if (u >= n_units) return;  // the whole wave leaves together
    uint64_t e[NS];
    bool valid[NS];
#pragma unroll
    for (int s = 0; s < NS; ++s) {
        const int r = 64 * s + lane;
        valid[s] = r < R;
        e[s] = valid[s] ? load_ev_bits(ev + u * ustride + (int64_t)r * rstride, kind) : 0ull;
    }
    uint64_t cand = 0;
    int cnt = 0;
    bool tried[NS];
#pragma unroll
    for (int s = 0; s < NS; ++s) tried[s] = false;
    int j = 0;
    while (true) {  // at most floor(R / 2) + 1 rounds: each covers replica j
        cand = wide_value<NS>(e, j);
        cnt = 0;
#pragma unroll
        for (int s = 0; s < NS; ++s) {
            const bool eq = valid[s] && e[s] == cand;
            cnt += __builtin_popcountll(ballot64(eq));
            tried[s] = tried[s] || eq;
        }
        if (2 * cnt > R) break;
        j = -1;
#pragma unroll
        for (int s = NS - 1; s >= 0; --s) {
            const uint64_t b = ballot64(!tried[s] && 64 * s + lane <= R / 2);
            if (b) j = 64 * s + __builtin_ctzll(b);
        }
        if (j < 0) break;
    }
    uint64_t ob[NS];
#pragma unroll
    for (int s = 0; s < NS; ++s) ob[s] = 0;
    if (2 * cnt <= R) {
        wide_write<NS>(u, C3_INCONCLUSIVE, ob, -1, status, bitmap, majority_idx);
        return;
    }
    int mj = -1;
    bool any = false;
#pragma unroll
    for (int s = NS - 1; s >= 0; --s) {
        const uint64_t mb = ballot64(valid[s] && e[s] == cand);
        ob[s] = ballot64(valid[s] && e[s] != cand);
        if (mb) mj = 64 * s + __builtin_ctzll(mb);
        any = any || ob[s] != 0;
    }
    wide_write<NS>(u, any ? C3_ATTRIBUTED : C3_AGREE, ob, mj, status, bitmap, majority_idx);
}

// Bitonic sort of the wave's 64 * NP (value, replica) keys, ascending by
// value, then replica: position p = 64 s + lane ends up holding the p-th
// smallest key.  Keys are unique (the replica breaks ties), so the order is
// the stable (value, replica) order.  Partners within a slot are 2^i lanes
// apart (xor shuffles); partners 64 and more apart sit in the same lane.
__device__ inline bool key_less(double av, int ai, double bv, int bi) {
    return av < bv || (av == bv && ai < bi);
}

template <int NP>
__device__ inline void wave_sort(double (&v)[NP], int (&id)[NP]) {
    const int lane = threadIdx.x & 63;
#pragma unroll
    for (int k = 2; k <= 64 * NP; k <<= 1) {
#pragma unroll
        for (int j = k >> 1; j > 0; j >>= 1) {
            if (j >= 64) {
#pragma unroll
                for (int s = 0; s < NP; ++s) {
                    const int t = s ^ (j >> 6);
                    if (t < s) continue;                 // each slot pair once
                    const bool asc = ((64 * s) & k) == 0;
                    const bool tl = key_less(v[t], id[t], v[s], id[s]);
                    if (asc ? tl : !tl) {
                        const double w = v[s];
                        v[s] = v[t];
                        v[t] = w;
                        const int q = id[s];
                        id[s] = id[t];
                        id[t] = q;
                    }
                }
            } else {
#pragma unroll
                for (int s = 0; s < NP; ++s) {
                    const double ov = shfl_xor_f64(v[s], j);
                    const int oi = (int)shfl_xor_u32((uint32_t)id[s], j);
                    const bool lower = (lane & j) == 0;
                    const bool asc = ((64 * s + lane) & k) == 0;
                    const bool ol = key_less(ov, oi, v[s], id[s]);
                    if (lower == asc ? ol : !ol) {
                        v[s] = ov;
                        id[s] = oi;
                    }
                }
            }
        }
    }
}

// The key at sorted position k (wave-uniform).
template <int NP>
__device__ inline double sorted_at(const double (&v)[NP], int k) {
    double r = 0.0;
#pragma unroll
    for (int s = 0; s < NP; ++s)
        if (s == (k >> 6)) r = readlane_f64(v[s], k & 63);
    return r;
}

template <int NP>
__device__ inline double sorted_median(const double (&v)[NP], int nf) {
    if (nf & 1) return sorted_at<NP>(v, (nf - 1) / 2);
    const double a = sorted_at<NP>(v, nf / 2 - 1);
    const double b = sorted_at<NP>(v, nf / 2);
    return (a + b) * 0.5;
}

// Hyndman-Fan type 7, as quantile7 above.
template <int NP>
__device__ inline double sorted_quantile7(const double (&v)[NP], int nf, double p) {
    const double h = (double)(nf - 1) * p;
    const double fl = floor(h);
    const int lo = (int)fl;
    const double frac = h - fl;
    if (lo + 1 >= nf) return sorted_at<NP>(v, nf - 1);
    const double a = sorted_at<NP>(v, lo);
    const double b = sorted_at<NP>(v, lo + 1);
    const double diff = b - a;
    const double prod = frac * diff;
    return a + prod;
}

template <int NS>
__global__ void __launch_bounds__(kVoteThreads) statistical_vote_wide_kernel(
    const char* __restrict__ ev, int kind, int64_t rstride, int64_t ustride, int R, int64_t n_units,
    double kappa, uint8_t* __restrict__ status, uint64_t* __restrict__ bitmap,
    int32_t* __restrict__ majority_idx) {
    const int lane = threadIdx.x & 63;
    const int64_t u = (int64_t)blockIdx.x * kWideUnitsPerBlock + (threadIdx.x >> 6);
    if (u >= n_units) return;  // the whole wave leaves together
    double x[NS];
    bool fin[NS];
    uint64_t finb[NS], B[NS];
    int nf = 0;
#pragma unroll
    for (int s = 0; s < NS; ++s) {
        const int r = 64 * s + lane;
        const bool valid = r < R;
        x[s] = valid ? load_ev_f64(ev + u * ustride + (int64_t)r * rstride, kind) : 0.0;
        fin[s] = valid && __builtin_isfinite(x[s]);
        finb[s] = ballot64(fin[s]);
        B[s] = ballot64(valid && !fin[s]);  // a non-finite value is an outlier
        nf += __builtin_popcountll(finb[s]);
    }
    if (2 * nf <= R) {  // finite values are not a strict majority
#pragma unroll
        for (int s = 0; s < NS; ++s) B[s] = 0;
        wide_write<NS>(u, C3_INCONCLUSIVE, B, -1, status, bitmap, majority_idx);
        return;
    }
    // sorted copies (NP slots: NS padded to a power of two); excluded values
    // sort last as +inf
    constexpr int NP = NS == 3 ? 4 : NS;
    const double inf = __builtin_huge_val();
    double sv[NP];
    int si[NP];
#pragma unroll
    for (int s = 0; s < NP; ++s) {
        sv[s] = s < NS && fin[s < NS ? s : 0] ? x[s < NS ? s : 0] : inf;
        si[s] = 64 * s + lane;
    }
    wave_sort<NP>(sv, si);
    const double m = sorted_median<NP>(sv, nf);
    // lower-median replica: stable position (nf - 1) / 2
    int mj = -1;
    const int pm = (nf - 1) / 2;
#pragma unroll
    for (int s = 0; s < NP; ++s)
        if (s == (pm >> 6)) mj = __builtin_amdgcn_readlane(si[s], pm & 63);
    double dev[NS];
#pragma unroll
    for (int s = 0; s < NS; ++s) dev[s] = fin[s] ? fabs(x[s] - m) : 0.0;
    double sd[NP];
    int sdi[NP];
#pragma unroll
    for (int s = 0; s < NP; ++s) {
        sd[s] = s < NS && fin[s < NS ? s : 0] ? dev[s < NS ? s : 0] : inf;
        sdi[s] = 64 * s + lane;
    }
    wave_sort<NP>(sd, sdi);
    double d = sorted_median<NP>(sd, nf);
    if (d == 0.0) {
        const double q3 = sorted_quantile7<NP>(sv, nf, 0.75);
        const double q1 = sorted_quantile7<NP>(sv, nf, 0.25);
        d = (q3 - q1) * 0.5;
    }
    if (d == 0.0) {
        const double hi = sorted_at<NP>(sv, nf - 1);
        const double lo = sorted_at<NP>(sv, 0);
        d = (hi - lo) / (double)nf;
    }
    const double thr = kappa * d;
    bool any = false;
#pragma unroll
    for (int s = 0; s < NS; ++s) {
        const bool flag = d != 0.0 && fin[s] && dev[s] > thr;
        B[s] |= ballot64(flag);
        any = any || B[s] != 0;
    }
    wide_write<NS>(u, any ? C3_ATTRIBUTED : C3_AGREE, B, mj, status, bitmap, majority_idx);
}

template <int NS>
static void launch_wide(const char* e, int kind, int64_t rstride, int64_t ustride, int R,
                        int64_t n_units, int mode, double kappa, uint8_t* status, uint64_t* bitmap,
                        int32_t* majority_idx, hipStream_t stream, unsigned blocks) {
    if (mode == C3_EXACT)
        hipLaunchKernelGGL(exact_vote_wide_kernel<NS>, dim3(blocks), dim3(kVoteThreads), 0, stream,
                           e, kind, rstride, ustride, R, n_units, status, bitmap, majority_idx);
    else
        hipLaunchKernelGGL(statistical_vote_wide_kernel<NS>, dim3(blocks), dim3(kVoteThreads), 0,
                           stream, e, kind, rstride, ustride, R, n_units, kappa, status, bitmap,
                           majority_idx);
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
    if (mode == C3_EXACT || R > 32) {
        const int64_t blocks = (n_units + kWideUnitsPerBlock - 1) / kWideUnitsPerBlock;
        if (blocks > 0x7FFFFFFF || R > C3_MAX_PEERS) return hipErrorInvalidValue;
        const char* e = static_cast<const char*>(evidence);
        const unsigned nb = (unsigned)blocks;
        if (R <= 64)
            launch_wide<1>(e, kind, rstride, ustride, R, n_units, mode, kappa, status, bitmap,
                           majority_idx, stream, nb);
        else if (R <= 128)
            launch_wide<2>(e, kind, rstride, ustride, R, n_units, mode, kappa, status, bitmap,
                           majority_idx, stream, nb);
        else if (R <= 192)
            launch_wide<3>(e, kind, rstride, ustride, R, n_units, mode, kappa, status, bitmap,
                           majority_idx, stream, nb);
        else
            launch_wide<4>(e, kind, rstride, ustride, R, n_units, mode, kappa, status, bitmap,
                           majority_idx, stream, nb);
        return hipGetLastError();
    }
    // STATISTICAL, 17 <= R <= 32: lane groups of 32
    int gw_log2 = 0;
    while ((1 << gw_log2) < R) ++gw_log2;
    const int64_t units_per_block = kVoteThreads >> gw_log2;
    const int64_t blocks = (n_units + units_per_block - 1) / units_per_block;
    if (blocks > 0x7FFFFFFF) return hipErrorInvalidValue;
    hipLaunchKernelGGL(statistical_vote_kernel, dim3((unsigned)blocks), dim3(kVoteThreads), 0,
                       stream, static_cast<const char*>(evidence), kind, rstride, ustride, R,
                       gw_log2, n_units, kappa, status, bitmap, majority_idx);
    return hipGetLastError();
}

}  // namespace c3
