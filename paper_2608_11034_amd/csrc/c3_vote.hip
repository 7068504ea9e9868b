// Consensus kernels of C3 for gfx950: the decision step of Algorithm 1.
//
// Which kernel decides a unit depends on the group size R:
//   R <= 32   one thread per unit, the R values in registers (128-bit row
//             loads when replicas are adjacent), deciding with the per-unit
//             functions of c3_vote_row.h;
//   R > 32    one wave per unit: lane l holds replicas l, l + 64, ... (see
//             the wave kernels below) and bitmap word s is one ballot.  The
//             exact vote broadcasts candidate values by readlane; the
//             statistical vote sorts the wave's values once.
// Per 256K units the wave kernel's statistical vote takes 0.09-0.11 ms at
// R = 33-64 and 0.26-0.37 ms at R = 129-256 (fp32-fp64), 1.8x to 8x faster
// than the rank loops and (value, replica) double sorts it replaced; on 1M-unit
// rows its exact vote was up to 7.6x (R = 64) faster than lane-per-replica
// counting.
//
// EXACT (Sec. 5.3): a strict majority exists iff some value is held by more
// than R / 2 replicas; those are the majority, the bitmap marks the others
// and the majority index is the lowest majority replica.
//
// STATISTICAL (Sec. 5.4), in fp64: order statistics of the finite values in
// the stable (value, then replica index) order give the median, the median
// absolute deviation, the type-7 quartiles and the range, in the fallback
// order MAD -> IQR / 2 -> range / n_finite.  Non-finite values are outliers
// and take no part in m or d.  No floating-point contraction is allowed in
// this file (the host compiles it with -ffp-contract=off), so the decision
// rounds exactly as the plain definition does.
#include "c3_device.h"
#include "c3_internal.h"
#include "c3_vote_row.h"

namespace c3 {

constexpr int kVoteThreads = 256;

// ---------------------------------------------------------------------------
// Small groups (R <= 32): one thread per unit with the R values in registers,
// so the whole decision is register arithmetic.  NMAX is R rounded up to a
// power of two; slots past R are padding that never takes part.
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
// Wave per unit (every group above 32 replicas).  Lane l
// holds the values of replicas l, l + 64, l + 128 and l + 192 (NS =
// ceil(R / 64) slots; slot s holds replica 64 s + l), so bitmap word s is the
// ballot of slot s.  The exact vote broadcasts candidate values by readlane
// at a wave-uniform index; the statistical vote sorts the wave's values.
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

// STATISTICAL over more than 32 replicas: the wave sorts the finite values
// once and reads every order statistic off the sorted copy.
//
// Sorted position p = NP lane + i lives in register i of lane `lane` (NP =
// ceil(R / 64) rounded up to a power of two, excluded values as +inf), so
// the network's shortest distances -- the most frequent ones -- are
// compare-exchanges between a lane's own registers, and the rest pair lane l
// with lane l ^ M.  The network is the bitonic sorter in its one-direction
// form: merging blocks of K, position p first meets p ^ (K - 1) (the
// reversed other half), then p ^ j for j = K / 4 .. 1, the smaller key
// always going to the lower position.  Values only: equal values are
// interchangeable, and the lower-median replica is found afterwards by
// counting.

// Lane l's copy of v from lane l ^ M: DPP where a row of 16 can express the
// pattern (quad permutes, mirrors), ds_swizzle inside 32 lanes, ds_bpermute
// across the halves.
template <int M>
__device__ __forceinline__ uint32_t xor_lane_u32(uint32_t v) {
    const int iv = (int)v;
    if constexpr (M == 1) return (uint32_t)__builtin_amdgcn_mov_dpp(iv, 0xB1, 0xF, 0xF, false);
    else if constexpr (M == 2) return (uint32_t)__builtin_amdgcn_mov_dpp(iv, 0x4E, 0xF, 0xF, false);
    else if constexpr (M == 3) return (uint32_t)__builtin_amdgcn_mov_dpp(iv, 0x1B, 0xF, 0xF, false);
    else if constexpr (M == 7) return (uint32_t)__builtin_amdgcn_mov_dpp(iv, 0x141, 0xF, 0xF, false);
    else if constexpr (M == 15) return (uint32_t)__builtin_amdgcn_mov_dpp(iv, 0x140, 0xF, 0xF, false);
    else if constexpr (M < 32) return (uint32_t)__builtin_amdgcn_ds_swizzle(iv, 0x1F | (M << 10));
    else return (uint32_t)__shfl_xor(iv, M, 64);
}

template <int M>
__device__ __forceinline__ float xor_lane(float v) {
    return __uint_as_float(xor_lane_u32<M>(__float_as_uint(v)));
}

template <int M>
__device__ __forceinline__ double xor_lane(double v) {
    const uint64_t b = (uint64_t)__double_as_longlong(v);
    const uint64_t lo = xor_lane_u32<M>((uint32_t)b), hi = xor_lane_u32<M>((uint32_t)(b >> 32));
    return __longlong_as_double((long long)((hi << 32) | lo));
}

template <typename V>
__device__ __forceinline__ void order_pair(V& a, V& b) {
    const bool sw = b < a;
    const V lo = sw ? b : a, hi = sw ? a : b;
    a = lo;
    b = hi;
}

// Between lanes: a lane in the lower half of the pair keeps the smaller key.
template <typename V>
__device__ __forceinline__ V keep(V mine, V other, bool upper) {
    return ((other < mine) != upper) ? other : mine;
}

template <int NP, int K, typename V>
__device__ __forceinline__ void sort_flip(V (&k)[NP], int lane) {
    if constexpr (K <= NP) {
#pragma unroll
        for (int i = 0; i < NP; ++i)
            if (i < (i ^ (K - 1))) order_pair(k[i], k[i ^ (K - 1)]);
    } else {
        constexpr int M = K / NP - 1;               // (lane, i) meets (lane ^ M, i ^ (NP - 1))
        const bool upper = (lane & (K / NP / 2)) != 0;
        V o[NP];
#pragma unroll
        for (int i = 0; i < NP; ++i) o[i] = xor_lane<M>(k[i ^ (NP - 1)]);
#pragma unroll
        for (int i = 0; i < NP; ++i) k[i] = keep(k[i], o[i], upper);
    }
}

template <int NP, int J, typename V>
__device__ __forceinline__ void sort_halves(V (&k)[NP], int lane) {
    if constexpr (J >= 1) {
        if constexpr (J < NP) {
#pragma unroll
            for (int i = 0; i < NP; ++i)
                if ((i & J) == 0) order_pair(k[i], k[i | J]);
        } else {
            constexpr int M = J / NP;
            const bool upper = (lane & M) != 0;
#pragma unroll
            for (int i = 0; i < NP; ++i) k[i] = keep(k[i], xor_lane<M>(k[i]), upper);
        }
        sort_halves<NP, J / 2>(k, lane);
    }
}

template <int NP, int K, typename V>
__device__ __forceinline__ void wave_sort(V (&k)[NP], int lane) {
    if constexpr (K <= 64 * NP) {
        sort_flip<NP, K>(k, lane);
        sort_halves<NP, K / 4>(k, lane);
        wave_sort<NP, 2 * K>(k, lane);
    }
}

// The key at sorted position p (wave-uniform).
template <int NP, typename V>
__device__ __forceinline__ double sorted_at(const V (&k)[NP], int p) {
    const int l = p / NP, i = p % NP;
    V r = 0;
#pragma unroll
    for (int t = 0; t < NP; ++t)
        if (t == i) {
            if constexpr (sizeof(V) == 4)
                r = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(k[t]), l));
            else
                r = __longlong_as_double((long long)readlane_u64((uint64_t)__double_as_longlong(k[t]), l));
        }
    return (double)r;
}

template <int NP, typename V>
__device__ __forceinline__ double sorted_median(const V (&k)[NP], int nf) {
    if (nf & 1) return sorted_at<NP>(k, (nf - 1) / 2);
    const double a = sorted_at<NP>(k, nf / 2 - 1);
    const double b = sorted_at<NP>(k, nf / 2);
    return (a + b) * 0.5;
}

// Hyndman-Fan type 7: h = (n - 1) p; Q = s[floor h] + frac(h) (s[floor h + 1] - s[floor h]).
template <int NP, typename V>
__device__ __forceinline__ double sorted_quantile7(const V (&k)[NP], int nf, double p) {
    const double h = (double)(nf - 1) * p;
    const double fl = floor(h);
    const int lo = (int)fl;
    const double frac = h - fl;
    if (lo + 1 >= nf) return sorted_at<NP>(k, nf - 1);
    const double a = sorted_at<NP>(k, lo);
    const double b = sorted_at<NP>(k, lo + 1);
    const double diff = b - a;
    const double prod = frac * diff;
    return a + prod;
}

// Median of |s - m| over the nf sorted finite values s, without sorting the
// deviations: the `split` values below m give m - s[split - 1 - i], the
// others s[split + i] - m, two ascending runs (each deviation rounds as
// |s - m| does, since rounding is symmetric).  Order statistic k of their
// union is found by bisecting how many of the k + 1 smallest come from the
// first run.
template <int NP, typename V>
__device__ __forceinline__ double deviation_median(const V (&k)[NP], int nf, int split, double m) {
    const int nl = split, nh = nf - split;
    auto L = [&](int i) { return m - sorted_at<NP>(k, split - 1 - i); };
    auto H = [&](int i) { return sorted_at<NP>(k, split + i) - m; };
    const int q = (nf - 1) / 2;                     // lower middle position
    int lo = q + 1 - nh > 0 ? q + 1 - nh : 0;
    int hi = q + 1 < nl ? q + 1 : nl;
    while (lo < hi) {                               // uniform bisection
        const int mid = (lo + hi) >> 1;
        if (L(mid) < H(q - mid)) lo = mid + 1;
        else hi = mid;
    }
    const int i = lo;                               // q + 1 smallest: i from L, q + 1 - i from H
    double a = -__builtin_huge_val();
    if (i > 0) a = L(i - 1);
    if (q - i >= 0) a = fmax(a, H(q - i));
    if (nf & 1) return a;
    double b = __builtin_huge_val();
    if (i < nl) b = L(i);
    if (q + 1 - i < nh) b = fmin(b, H(q + 1 - i));
    return (a + b) * 0.5;
}

template <int NS, int KIND>
__global__ void __launch_bounds__(kVoteThreads) statistical_vote_wide_kernel(
    const char* __restrict__ ev, int64_t rstride, int64_t ustride, int R, int64_t n_units,
    double kappa, uint8_t* __restrict__ status, uint64_t* __restrict__ bitmap,
    int32_t* __restrict__ majority_idx) {
    // fp32 evidence is ordered and compared in fp32 (the widening to fp64 is
    // exact and monotonic); every arithmetic step is fp64
    using V = typename std::conditional<KIND == C3_EV_F32, float, double>::type;
    const int lane = threadIdx.x & 63;
    const int64_t u = (int64_t)blockIdx.x * kWideUnitsPerBlock + (threadIdx.x >> 6);
    if (u >= n_units) return;  // the whole wave leaves together
    V x[NS];
    bool fin[NS];
    uint64_t B[NS];
    int nf = 0;
#pragma unroll
    for (int s = 0; s < NS; ++s) {
        const int r = 64 * s + lane;
        const bool valid = r < R;
        x[s] = valid ? *reinterpret_cast<const V*>(ev + u * ustride + (int64_t)r * rstride) : (V)0;
        fin[s] = valid && __builtin_isfinite(x[s]);
        nf += __builtin_popcountll(ballot64(fin[s]));
        B[s] = ballot64(valid && !fin[s]);  // a non-finite value is an outlier
    }
    if (2 * nf <= R) {  // finite values are not a strict majority
#pragma unroll
        for (int s = 0; s < NS; ++s) B[s] = 0;
        wide_write<NS>(u, C3_INCONCLUSIVE, B, -1, status, bitmap, majority_idx);
        return;
    }
    constexpr int NP = NS == 3 ? 4 : NS;
    V k[NP];
#pragma unroll
    for (int i = 0; i < NP; ++i)
        k[i] = i < NS && fin[i < NS ? i : 0] ? x[i < NS ? i : 0] : (V)__builtin_huge_val();
    wave_sort<NP, 2>(k, lane);
    const double m = sorted_median<NP>(k, nf);
    int split = 0;                                  // finite values below m
#pragma unroll
    for (int s = 0; s < NS; ++s) split += __builtin_popcountll(ballot64(fin[s] && (double)x[s] < m));
    double d = deviation_median<NP>(k, nf, split, m);
    if (d == 0.0) {
        const double q3 = sorted_quantile7<NP>(k, nf, 0.75);
        const double q1 = sorted_quantile7<NP>(k, nf, 0.25);
        d = (q3 - q1) * 0.5;
    }
    if (d == 0.0) {
        const double hi = sorted_at<NP>(k, nf - 1);
        const double lo = sorted_at<NP>(k, 0);
        d = (hi - lo) / (double)nf;
    }
    const double thr = kappa * d;
    bool any = false;
#pragma unroll
    for (int s = 0; s < NS; ++s) {
        const bool flag = d != 0.0 && fin[s] && fabs((double)x[s] - m) > thr;
        B[s] |= ballot64(flag);
        any = any || B[s] != 0;
    }
    // lower-median replica: position (nf - 1) / 2 of the stable (value,
    // replica) order is the want-th replica, by index, holding the value
    // there, after the replicas holding smaller values
    const int pm = (nf - 1) / 2;
    const V target = (V)sorted_at<NP>(k, pm);
    int want = pm;
#pragma unroll
    for (int s = 0; s < NS; ++s) want -= __builtin_popcountll(ballot64(fin[s] && x[s] < target));
    int mj = -1;
#pragma unroll
    for (int s = 0; s < NS; ++s) {
        uint64_t eq = ballot64(fin[s] && x[s] == target);
        const int c = __builtin_popcountll(eq);
        if (mj < 0 && want < c) {
            for (int w = 0; w < want; ++w) eq &= eq - 1ull;
            mj = 64 * s + __builtin_ctzll(eq);
        }
        want -= c;
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
    else if (kind == C3_EV_F32)
        hipLaunchKernelGGL((statistical_vote_wide_kernel<NS, C3_EV_F32>), dim3(blocks),
                           dim3(kVoteThreads), 0, stream, e, rstride, ustride, R, n_units, kappa,
                           status, bitmap, majority_idx);
    else
        hipLaunchKernelGGL((statistical_vote_wide_kernel<NS, C3_EV_F64>), dim3(blocks),
                           dim3(kVoteThreads), 0, stream, e, rstride, ustride, R, n_units, kappa,
                           status, bitmap, majority_idx);
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
    // Up to 32 replicas one thread decides a unit: against a wave per unit,
    // 0.035-0.044 against 0.092-0.102 ms per 262,144 units of fp32 times at
    // R = 17-32, 0.055-0.072 against 0.106-0.117 for fp64, 0.027-0.046
    // against 0.044-0.046 for 64-bit fingerprints; the same results.
    if (R <= 32) {
        const int64_t blocks = (n_units + kVoteThreads - 1) / kVoteThreads;
        if (blocks > 0x7FFFFFFF) return hipErrorInvalidValue;
        const char* e = static_cast<const char*>(evidence);
        if (R <= 4)
            launch_small<4>(e, kind, rstride, ustride, R, n_units, mode, kappa, status, bitmap,
                            majority_idx, stream, (unsigned)blocks);
        else if (R <= 8)
            launch_small<8>(e, kind, rstride, ustride, R, n_units, mode, kappa, status, bitmap,
                            majority_idx, stream, (unsigned)blocks);
        else if (R <= 16)
            launch_small<16>(e, kind, rstride, ustride, R, n_units, mode, kappa, status, bitmap,
                             majority_idx, stream, (unsigned)blocks);
        else
            launch_small<32>(e, kind, rstride, ustride, R, n_units, mode, kappa, status, bitmap,
                             majority_idx, stream, (unsigned)blocks);
        return hipGetLastError();
    }
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

}  // namespace c3
