// Single-workgroup localization shared by c3_localize (small inputs) and the
// fused check: one workgroup of NT threads walks the units in rounds of
// NT * PER, each thread owning PER consecutive units, and writes the
// outlier list in (unit ascending, replica ascending) order, the undecided
// units ascending and the three counts.  A unit's bitmap is W = ceil(R / 64)
// words, bit b of word w naming replica 64 w + b.
#pragma once

#include "../../include/c3.h"
#include "c3_device.h"

namespace c3 {

// Set bits of unit u's bitmap.
__device__ inline int unit_popcount(const uint64_t* bitmap, int W, int64_t u) {
    int n = 0;
    for (int w = 0; w < W; ++w) n += __builtin_popcountll(bitmap[u * W + w]);
    return n;
}

// Inclusive prefix sum over the NT threads of a workgroup (fixed order).
template <int NT>
__device__ inline int64_t block_inclusive_scan(int64_t v, int64_t* lds_wave, int64_t& total) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    int64_t x = v;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
        const int64_t y = (int64_t)shfl_u64((uint64_t)x, lane >= d ? lane - d : lane);
        if (lane >= d) x += y;
    }
    if (lane == 63) lds_wave[wave] = x;
    __syncthreads();
    int64_t before = 0;
    total = 0;
    for (int w = 0; w < NT / 64; ++w) {
        if (w < wave) before += lds_wave[w];
        total += lds_wave[w];
    }
    __syncthreads();
    return x + before;
}

// One outlier entry: unit, replica, majority replica and both summaries
// (zeros when no record table is given).
__device__ inline void write_outlier(c3_outlier_t* dst, int64_t u, int r, int32_t mj,
                                     const c3_chunk_record_t* __restrict__ records, int R,
                                     int64_t n_units) {
    c3_outlier_t e;
    e.chunk = u;
    e.replica = r;
    e.majority_replica = mj;
    for (int z = 0; z < 2; ++z) {
        const int rr = z == 0 ? r : mj;
        if (records != nullptr && rr >= 0 && rr < R) {
            const c3_chunk_record_t& rec = records[(int64_t)rr * n_units + u];
            e.nan_count[z] = rec.nan_count;
            e.inf_count[z] = rec.inf_count;
            e.absmax[z] = rec.absmax;
            e.sum[z] = rec.sum;
            e.sumsq[z] = rec.sumsq;
        } else {
            e.nan_count[z] = 0;
            e.inf_count[z] = 0;
            e.absmax[z] = 0.0;
            e.sum[z] = 0.0;
            e.sumsq[z] = 0.0;
        }
    }
    *dst = e;
}

// The per-thread counts of a round travel through a single scan packed into
// one 64-bit word: outliers in the low 24 bits (a round holds at most
// NT * PER units * 256 replicas), undecided and attributed units in 20 bits
// each, so no field overflows for the sizes used (checked below).
constexpr int kOutBits = 24;
constexpr int kUnitBits = 20;
constexpr int64_t kOutMask = (1ll << kOutBits) - 1;
constexpr int64_t kUnitMask = (1ll << kUnitBits) - 1;
static_assert(kOutBits + 2 * kUnitBits <= 64, "fields exceed one word");

template <bool WIDE, int NT, int PER>
__device__ inline void localize_block(
    const uint8_t* __restrict__ status, const uint64_t* __restrict__ bitmap,
    const int32_t* __restrict__ majority_idx, const c3_chunk_record_t* __restrict__ records, int R,
    int W, int64_t n_units, c3_outlier_t* __restrict__ outliers, int64_t out_cap,
    int64_t* __restrict__ undecided, int64_t und_cap, int64_t* __restrict__ counts) {
    static_assert((int64_t)NT * PER * C3_MAX_PEERS <= kOutMask, "outlier field too narrow");
    static_assert((int64_t)NT * PER <= kUnitMask, "unit fields too narrow");
    __shared__ int64_t lds[NT / 64];
    int64_t carry_o = 0, carry_u = 0, carry_a = 0;
    for (int64_t base = 0; base < n_units; base += (int64_t)NT * PER) {
        const int64_t u0 = base + (int64_t)threadIdx.x * PER;
        uint8_t st[PER];
        uint64_t bm[PER];  // the word (one-word bitmaps) or the set-bit count
#pragma unroll
        for (int i = 0; i < PER; ++i) {
            const int64_t u = u0 + i;
            st[i] = u < n_units ? status[u] : (uint8_t)C3_AGREE;
            if constexpr (WIDE)
                bm[i] = u < n_units ? (uint64_t)unit_popcount(bitmap, W, u) : 0ull;
            else
                bm[i] = u < n_units ? bitmap[u] : 0ull;
        }
        int64_t o = 0, un = 0, at = 0;
#pragma unroll
        for (int i = 0; i < PER; ++i) {
            if (st[i] == C3_INCONCLUSIVE) {
                ++un;
            } else if (bm[i]) {
                ++at;
                o += WIDE ? (int64_t)bm[i] : __builtin_popcountll(bm[i]);
            }
        }
        const int64_t packed = o | (un << kOutBits) | (at << (kOutBits + kUnitBits));
        int64_t tot;
        const int64_t excl = block_inclusive_scan<NT>(packed, lds, tot) - packed;
        int64_t po = carry_o + (excl & kOutMask);
        int64_t pu = carry_u + ((excl >> kOutBits) & kUnitMask);
#pragma unroll
        for (int i = 0; i < PER; ++i) {
            const int64_t u = u0 + i;
            if (st[i] == C3_INCONCLUSIVE) {
                if (pu < und_cap) undecided[pu] = u;
                ++pu;
                continue;
            }
            if (!bm[i]) continue;
            const int32_t mj = majority_idx[u];
            for (int w = 0; w < (WIDE ? W : 1); ++w) {
                uint64_t b = WIDE ? bitmap[u * W + w] : bm[i];
                while (b) {
                    const int r = 64 * w + __builtin_ctzll(b);
                    b &= b - 1;
                    if (po < out_cap) write_outlier(&outliers[po], u, r, mj, records, R, n_units);
                    ++po;
                }
            }
        }
        carry_o += tot & kOutMask;
        carry_u += (tot >> kOutBits) & kUnitMask;
        carry_a += (tot >> (kOutBits + kUnitBits)) & kUnitMask;
    }
    if (threadIdx.x == 0) {
        counts[0] = carry_o;
        counts[1] = carry_u;
        counts[2] = carry_a;
    }
}


}  // namespace c3
