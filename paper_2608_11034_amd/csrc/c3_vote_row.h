// Per-unit decisions of Algorithm 1 for groups of up to 32 replicas, one
// thread per unit with the R values in registers.  Used by the consensus
// kernels (c3_vote.hip) and the fused timing-consensus kernel
// (c3_timing.hip), so both decide every unit with the same code.
//
// EXACT (Sec. 5.3): a strict majority exists iff some value is held by
// more than R / 2 replicas; those are the majority, the bitmap marks the
// others and the majority index is the lowest majority replica.  The value
// is found with R compares against replica 0 in the usual case, else with a
// Boyer-Moore pass.
//
// STATISTICAL (Sec. 5.4), in fp64: order statistics from min/max sorting
// networks over the finite values (non-finite ones sort last and are
// outliers), RobustScale in the order MAD -> IQR / 2 (type-7 quartiles) ->
// range / n_finite, strict |x - m| > kappa d, and the lower-median replica in
// the stable (value, replica) order.  Files including this header are
// compiled without floating-point contraction, so the decision rounds
// exactly as the plain definition does.
#pragma once

#include <type_traits>

#include "../../include/c3.h"
#include "c3_device.h"

namespace c3 {

typedef uint32_t vu32x4 __attribute__((ext_vector_type(4)));

struct UnitVote {
    uint64_t bitmap;
    int32_t majority;
    uint8_t status;
};

__device__ inline uint64_t load_ev_bits(const char* p, int kind) {
    if (kind == C3_EV_U64 || kind == C3_EV_F64) return *reinterpret_cast<const uint64_t*>(p);
    return *reinterpret_cast<const uint32_t*>(p);
}

// Raw bits of the R values of one unit (4-byte kinds zero-extended).  With
// `dense` the replicas are adjacent and the row is 16-byte aligned and a
// whole number of 16-byte words, so it is read with 128-bit loads.  Every
// slot is loaded unconditionally (slots past R re-read the row's first word
// and are zeroed afterwards): loads under a branch would each be waited for
// at the branch's join, serializing them.
template <int NMAX>
__device__ __forceinline__ void load_row_bits(const char* base, int kind, int64_t rstride, int R,
                                              bool dense, uint64_t (&e)[NMAX]) {
    const bool wide = kind == C3_EV_U64 || kind == C3_EV_F64;
    if (dense && wide) {
        vu32x4 v[NMAX / 2];
#pragma unroll
        for (int j = 0; j < NMAX / 2; ++j)
            v[j] = *reinterpret_cast<const vu32x4*>(base + (2 * j < R ? 16 * j : 0));
#pragma unroll
        for (int j = 0; j < NMAX / 2; ++j) {
            const bool in = 2 * j < R;
            e[2 * j] = in ? ((uint64_t)v[j].y << 32) | v[j].x : 0ull;
            e[2 * j + 1] = in ? ((uint64_t)v[j].w << 32) | v[j].z : 0ull;
        }
    } else if (dense && NMAX >= 4) {
        vu32x4 v[NMAX / 4];
#pragma unroll
        for (int j = 0; j < NMAX / 4; ++j)
            v[j] = *reinterpret_cast<const vu32x4*>(base + (4 * j < R ? 16 * j : 0));
#pragma unroll
        for (int j = 0; j < NMAX / 4; ++j) {
            const bool in = 4 * j < R;
            e[4 * j] = in ? v[j].x : 0u;
            e[4 * j + 1] = in ? v[j].y : 0u;
            e[4 * j + 2] = in ? v[j].z : 0u;
            e[4 * j + 3] = in ? v[j].w : 0u;
        }
    } else {
#pragma unroll
        for (int r = 0; r < NMAX; ++r) e[r] = load_ev_bits(base + (r < R ? r : 0) * rstride, kind);
#pragma unroll
        for (int r = 0; r < NMAX; ++r) e[r] = r < R ? e[r] : 0ull;
    }
}

template <int NMAX>
__device__ __forceinline__ uint64_t equal_mask(const uint64_t (&e)[NMAX], int R, uint64_t v) {
    uint64_t m = 0;
#pragma unroll
    for (int r = 0; r < NMAX; ++r) m |= (uint64_t)(r < R && e[r] == v) << r;
    return m;
}

// A strict majority value, if any, is unique, so the majority replicas are
// the holders of one candidate value.  The candidate is replica 0's value
// when that already has a majority (the usual case: one pass of R
// compares); otherwise the Boyer-Moore majority candidate, which is the
// majority value whenever there is one.
template <int NMAX>
__device__ __forceinline__ UnitVote exact_vote_row(const uint64_t (&e)[NMAX], int R) {
    UnitVote v;
    // Every replica holding replica 0's value (the usual unit) is settled by
    // R - 1 compares whose results combine as lane masks; the units of a
    // wave that need the general rule below take it together, and a wave
    // with none skips it.
    bool same = true;
#pragma unroll
    for (int r = 1; r < NMAX; ++r) same &= (r >= R) | (e[r] == e[0]);
    if (same) {
        v.status = C3_AGREE;
        v.bitmap = 0;
        v.majority = 0;
        return v;
    }
    uint64_t maj = equal_mask<NMAX>(e, R, e[0]);
    if (2 * __builtin_popcountll(maj) <= R) {
        uint64_t cand = e[0];
        int cnt = 0;
#pragma unroll
        for (int r = 0; r < NMAX; ++r) {
            if (r < R) {
                if (cnt == 0) cand = e[r];
                cnt += e[r] == cand ? 1 : -1;
            }
        }
        maj = equal_mask<NMAX>(e, R, cand);
    }
    if (2 * __builtin_popcountll(maj) <= R) {
        v.status = C3_INCONCLUSIVE;
        v.bitmap = 0;
        v.majority = -1;
    } else {
        const uint64_t valid = R == 64 ? ~0ull : ((1ull << R) - 1);
        v.bitmap = valid & ~maj;
        v.status = v.bitmap ? C3_ATTRIBUTED : C3_AGREE;
        v.majority = __builtin_ctzll(maj);
    }
    return v;
}

// Batcher's odd-even merge sort over N register slots (N a power of two,
// values without NaN): 5, 19, 63 and 191 comparators for 4, 8, 16 and 32
// slots, each one min and one max.  The slots never hold a NaN, so the hardware min and
// max are used as they are: fminf / fmaxf would first quiet each input
// (one more instruction per slot), which only matters for signaling NaNs.
__device__ __forceinline__ float vmin(float a, float b) {
    float r;
    asm("v_min_f32 %0, %1, %2" : "=v"(r) : "v"(a), "v"(b));
    return r;
}
__device__ __forceinline__ float vmax(float a, float b) {
    float r;
    asm("v_max_f32 %0, %1, %2" : "=v"(r) : "v"(a), "v"(b));
    return r;
}
__device__ __forceinline__ double vmin(double a, double b) {
    double r;
    asm("v_min_f64 %0, %1, %2" : "=v"(r) : "v"(a), "v"(b));
    return r;
}
__device__ __forceinline__ double vmax(double a, double b) {
    double r;
    asm("v_max_f64 %0, %1, %2" : "=v"(r) : "v"(a), "v"(b));
    return r;
}
// max(|a|, |b|) of two values without NaN, in one instruction
__device__ __forceinline__ double vmax_abs(double a, double b) {
    double r;
    asm("v_max_f64 %0, |%1|, |%2|" : "=v"(r) : "v"(a), "v"(b));
    return r;
}

template <int N, typename V>
__device__ __forceinline__ void sort_network(V (&v)[N]) {
    static_assert(N >= 2 && (N & (N - 1)) == 0, "power of two");
#pragma unroll
    for (int p = 1; p < N; p <<= 1) {
#pragma unroll
        for (int k = p; k >= 1; k >>= 1) {
#pragma unroll
            for (int j = k % p; j <= N - 1 - k; j += 2 * k) {
#pragma unroll
                for (int i = 0; i < k && i < N - j - k; ++i) {
                    // only pairs inside one block of 2p slots
                    if ((i + j) / (2 * p) == (i + j + k) / (2 * p)) {
                        const V lo = vmin(v[i + j], v[i + j + k]);
                        const V hi = vmax(v[i + j], v[i + j + k]);
                        v[i + j] = lo;
                        v[i + j + k] = hi;
                    }
                }
            }
        }
    }
}

__device__ __forceinline__ uint32_t vbits(float x) { return __float_as_uint(x); }
__device__ __forceinline__ uint64_t vbits(double x) { return (uint64_t)__double_as_longlong(x); }
__device__ __forceinline__ float vfrom(uint32_t b, float) { return __uint_as_float(b); }
__device__ __forceinline__ double vfrom(uint64_t b, double) { return __longlong_as_double((long long)b); }

// v[k] for a run-time k, as an OR of masked slots.  A select chain would be
// turned back into an indexed load, which puts the array in scratch memory.
// With a compile-time k the loop folds to the one slot.
template <int N, typename V>
__device__ __forceinline__ V pick(const V (&v)[N], int k) {
    decltype(vbits(v[0])) out = 0;
#pragma unroll
    for (int i = 0; i < N; ++i) {
        const decltype(out) m = (decltype(out))0 - (decltype(out))(i == k);
        out |= m & vbits(v[i]);
    }
    return vfrom(out, v[0]);
}

// Median of the n smallest slots of s (sorted), in fp64.
template <int N, typename V>
__device__ __forceinline__ double median_sorted(const V (&s)[N], int n) {
    if (n & 1) return (double)pick<N>(s, (n - 1) / 2);
    return ((double)pick<N>(s, n / 2 - 1) + (double)pick<N>(s, n / 2)) * 0.5;
}

// Type-7 quantile p of the n smallest slots of s (sorted), in fp64.
template <int N, typename V>
__device__ __forceinline__ double quantile7_sorted(const V (&s)[N], int n, double p) {
    const double h = (double)(n - 1) * p;
    const double fl = floor(h);
    const int lo = (int)fl;
    const double frac = h - fl;
    if (lo + 1 >= n) return (double)pick<N>(s, n - 1);
    const double a = (double)pick<N>(s, lo);
    const double b = (double)pick<N>(s, lo + 1);
    const double diff = b - a;
    const double prod = frac * diff;
    return a + prod;
}

// Everything after the first sort.  NC > 0 fixes the finite count at
// compile time (every value finite and R == NMAX, the usual case), so every
// order statistic is a plain register and no replica needs a finiteness
// test.  Without MAJ the lower-median replica is not computed (majority is
// -1); callers that keep only the bitmap skip that work.
template <int NMAX, int NC, typename V, bool MAJ>
__device__ __forceinline__ UnitVote statistical_tail(const V (&x)[NMAX], const V (&s)[NMAX],
                                                     uint64_t fin, uint64_t nonfin, int nf_rt,
                                                     double kappa) {
    const int nf = NC > 0 ? NC : nf_rt;
    auto finite = [&](int r) { return NC > 0 || ((fin >> r) & 1ull) != 0; };
    const double m = median_sorted<NMAX>(s, nf);
    // the largest deviation, when known without visiting every replica
    double dmax = __builtin_huge_val();
    double d;
    if constexpr (NC > 0) {
        // m lies between the two middle sorted values, so the deviations of
        // the values below it and of those above it are two ascending runs
        // lo and hi of h each; the two middle deviations are order
        // statistics h - 1 and h of their merge: the minimum, over the ways
        // of taking i from lo and the rest from hi, of the larger last taken.
        constexpr int h = NC / 2;
        const double dlo = (double)s[0] - m, dhi = (double)s[NC - 1] - m;
        double lo[h], hi[h];
#pragma unroll
        for (int k = 0; k < h - 1; ++k) {
            lo[k] = fabs((double)s[h - 1 - k] - m);
            hi[k] = fabs((double)s[h + k] - m);
        }
        lo[h - 1] = fabs(dlo);
        hi[h - 1] = fabs(dhi);
        double a = fmin(hi[h - 1], lo[h - 1]);
#pragma unroll
        for (int i = 1; i < h; ++i) a = fmin(a, fmax(lo[i - 1], hi[h - 1 - i]));
        double b = fmax(lo[0], hi[h - 1]);
#pragma unroll
        for (int i = 2; i <= h; ++i) b = fmin(b, fmax(lo[i - 1], hi[h - i]));
        d = (a + b) * 0.5;
        // lo and hi are the deviations of every value, computed as the flag
        // test computes them, and each run ascends away from m: the largest
        // deviation is the larger run end
        dmax = vmax_abs(dlo, dhi);
    } else {
        double ds[NMAX];
#pragma unroll
        for (int r = 0; r < NMAX; ++r)
            ds[r] = finite(r) ? fabs((double)x[r] - m) : __builtin_huge_val();
        sort_network<NMAX>(ds);
        d = median_sorted<NMAX>(ds, nf);
    }
    // the fallbacks of a zero MAD, skipped by waves where no unit has one
    if (ballot64(d == 0.0) != 0ull) {
        if (d == 0.0) {
            const double q3 = quantile7_sorted<NMAX>(s, nf, 0.75);
            const double q1 = quantile7_sorted<NMAX>(s, nf, 0.25);
            d = (q3 - q1) * 0.5;
        }
        if (d == 0.0) d = ((double)pick<NMAX>(s, nf - 1) - (double)s[0]) / (double)nf;
    }
    uint64_t B = nonfin;
    if (d != 0.0) {
        const double thr = kappa * d;
        // no replica can be flagged when even the largest deviation is not
        // above the threshold (the usual unit): skip the per-replica tests
        if (dmax > thr) {
#pragma unroll
            for (int r = 0; r < NMAX; ++r)
                if (finite(r) && fabs((double)x[r] - m) > thr) B |= 1ull << r;
        }
    }
    UnitVote v;
    v.status = B ? C3_ATTRIBUTED : C3_AGREE;
    v.bitmap = B;
    v.majority = -1;
    if constexpr (!MAJ) return v;
    // lower-median replica: stable position (nf - 1) / 2 in (value, replica) order
    const V target = pick<NMAX>(s, (nf - 1) / 2);
    int want = (nf - 1) / 2;
#pragma unroll
    for (int r = 0; r < NMAX; ++r) want -= (finite(r) && x[r] < target) ? 1 : 0;
    int med = -1;
#pragma unroll
    for (int r = 0; r < NMAX; ++r) {
        if (finite(r) && x[r] == target) {
            if (want == 0 && med < 0) med = r;
            --want;
        }
    }
    v.majority = med;
    return v;
}

// `bits` hold the fp32 (KIND == C3_EV_F32, zero-extended) or fp64 patterns.
// fp32 values are ordered and compared in fp32 (exact: the conversion to
// fp64 is monotonic and exact); every arithmetic step is fp64.
template <int NMAX, int KIND, bool MAJ = true>
__device__ __forceinline__ UnitVote statistical_vote_row(const uint64_t (&bits)[NMAX], int R,
                                                         double kappa) {
    using V = typename std::conditional<KIND == C3_EV_F32, float, double>::type;
    V x[NMAX], s[NMAX];
    // every slot a valid finite value (the usual unit): one class test per
    // slot, combined as lane masks
    bool allfin = true;
#pragma unroll
    for (int r = 0; r < NMAX; ++r) {
        if constexpr (KIND == C3_EV_F32) x[r] = __uint_as_float((uint32_t)bits[r]);
        else x[r] = __longlong_as_double((long long)bits[r]);
        allfin &= (r < R) & __builtin_isfinite(x[r]);
    }
    const uint64_t valid = R == 64 ? ~0ull : ((1ull << R) - 1);
    if (allfin) {
        // sort the values as they are
#pragma unroll
        for (int r = 0; r < NMAX; ++r) s[r] = x[r];
        sort_network<NMAX>(s);
        return statistical_tail<NMAX, NMAX, V, MAJ>(x, s, valid, 0ull, NMAX, kappa);
    }
    uint64_t fin = 0;
#pragma unroll
    for (int r = 0; r < NMAX; ++r) fin |= (uint64_t)(r < R && __builtin_isfinite(x[r])) << r;
    const uint64_t nonfin = valid & ~fin;
    const int nf = __builtin_popcountll(fin);
    if (2 * nf <= R) {
        UnitVote v;
        v.status = C3_INCONCLUSIVE;
        v.bitmap = 0;
        v.majority = -1;
        return v;
    }
#pragma unroll
    for (int r = 0; r < NMAX; ++r)   // excluded values sort last
        s[r] = ((fin >> r) & 1ull) ? x[r] : (V)__builtin_huge_val();
    sort_network<NMAX>(s);
    return statistical_tail<NMAX, 0, V, MAJ>(x, s, fin, nonfin, nf, kappa);
}

}  // namespace c3
