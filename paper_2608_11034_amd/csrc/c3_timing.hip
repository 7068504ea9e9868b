// Timing consensus of C3 for gfx950: per (iteration, peer group) an exact
// vote on the ranks' collective fingerprints (Sec. 7: a minority fingerprint
// is a protocol outlier) and a statistical vote on their step times
// (Sec. 5.4), then the per-rank temporal confirmation (Sec. 10: a straggler
// must recur).  The votes are the per-unit decisions of c3_vote_row.h, as in
// c3_consensus; besides the optional per-unit results they OR each outlier
// bit into a per-rank mask (one 32-bit word per rank, kind and 32
// iterations), so the confirmation reads 8 bytes per rank and 32 iterations
// instead of the per-unit bitmaps, and walks them a word at a time.  The
// masks live in the LDS of a single kernel whose workgroups each own a set
// of groups over all iterations (the shapes it takes, with or without
// per-unit results), or else in the workspace (three launches: clear,
// votes, confirmation).
#include "c3_device.h"
#include "c3_internal.h"
#include "c3_vote_row.h"

namespace c3 {

constexpr int kVoteThreads = 256;
constexpr int kSegIters = 32;      // iterations per mask segment (one u32 per rank and kind)
constexpr int kConfirmThreads = 256;
constexpr int kConfirmLanes = 8;   // lanes per rank in the confirmation
constexpr int kPrefetch = 8;       // mask segments fetched at once per lane

// Per-unit outputs of one evidence kind (status null: none) and its masks.
struct VoteOut {
    uint8_t* status;
    uint64_t* bitmap;
    int32_t* majority;
    uint32_t* masks;
};

// Stores one unit's decision: the optional per-unit results, and each
// outlier bit ORed into the per-rank masks [segment][r][g] (bit t mod 32 of
// word t / 32).  Outlier bits are sparse, so the atomics cost little; the
// masks must start zeroed.
__device__ __forceinline__ void store_vote(const UnitVote& v, int R, int64_t G, int64_t n_units,
                                           const VoteOut& o, int64_t u) {
    if (o.status != nullptr) {
        o.status[u] = v.status;
        o.bitmap[u] = v.bitmap;
        o.majority[u] = v.majority;
    }
    if (v.bitmap != 0ull) {
        // 32-bit division when the unit count allows it (uniform per launch)
        const int64_t t = n_units <= 0xFFFFFFFFll ? (int64_t)((uint32_t)u / (uint32_t)G) : u / G;
        const int64_t g = u - t * G;
        const uint32_t bit = 1u << (t & (kSegIters - 1));
        uint32_t* m = o.masks + (t / kSegIters) * R * G + g;
        for (uint64_t b = v.bitmap; b != 0ull; b &= b - 1ull)
            atomicOr(m + (int64_t)__builtin_ctzll(b) * G, bit);
    }
}

// Both votes of one unit u = t * G + g per thread: the fingerprint row
// (exact) and the step-time row (statistical) are loaded together, so their
// memory latency overlaps, and a wave reads 64 consecutive rows of each,
// fully coalesced.  Decisions are the per-unit functions of c3_vote_row.h.
// DENSE (both rows read with 128-bit loads) is a template argument so that
// all loads of both rows sit in one basic block and are issued together.
template <int NMAX, int KIND, bool DENSE>
__global__ void __launch_bounds__(kVoteThreads) timing_votes_kernel(
    const char* __restrict__ fp, const char* __restrict__ tp, int R, int64_t G, int64_t n_units,
    double kappa, bool fp_dense, bool t_dense, VoteOut fo, VoteOut to) {
    constexpr int tsize = KIND == C3_EV_F64 ? 8 : 4;
    const int64_t ub = blockIdx.x;
    const int64_t u = ub * kVoteThreads + threadIdx.x;
    if (u >= n_units) return;
    // the workgroup's rows start at a uniform offset; the lane's offset
    // within them fits 32 bits
    const uint32_t lane_rows = threadIdx.x * (uint32_t)R;
    uint64_t ef[NMAX], et[NMAX];
    load_row_bits<NMAX>(fp + ub * kVoteThreads * R * 8 + lane_rows * 8u, C3_EV_U64, 8, R,
                        DENSE || fp_dense, ef);
    load_row_bits<NMAX>(tp + ub * kVoteThreads * R * tsize + lane_rows * (uint32_t)tsize, KIND,
                        tsize, R, DENSE || t_dense, et);
    store_vote(exact_vote_row<NMAX>(ef, R), R, G, n_units, fo, u);
    store_vote(statistical_vote_row<NMAX, KIND>(et, R, kappa), R, G, n_units, to, u);
}

// Staged variant for R == NMAX with both kinds dense: rows are 32, 64 or
// 128 bytes, read per lane they would take several 16-byte loads per row
// that each touch every cache line of the wave's rows.  Instead each wave
// reads its 64 rows of a kind with contiguous 1 KB loads (lane l, load j:
// bytes 1024 j + 16 l), passes them through its own LDS region and takes
// its row back.  Chunk c of row u sits at slot u * CP + ((c + (u >> s)) &
// (CP - 1)), s = log2(16 / CP), which puts any 16 consecutive lanes on 16
// distinct 16-byte bank groups for the writes and for the reads.  No
// workgroup barrier: a wave only touches its own region, and LDS
// instructions of one wave execute in order.
template <int CP>
__device__ __forceinline__ int stage_slot(int u, int c) {
    constexpr int S = CP == 1 ? 4 : CP == 2 ? 3 : CP == 4 ? 2 : 1;
    return u * CP + ((c + (u >> S)) & (CP - 1));
}

__device__ __forceinline__ void wave_lds_sync() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Loads of one kind: the wave's rows start at wbase, nbytes of them exist
// (non-temporal: every record is read once)
// (whole rows, at least one); loads past them re-read the last 16 bytes.
template <int CP>
__device__ __forceinline__ void stage_load(const char* wbase, int64_t nbytes, int lane,
                                           vu32x4 (&g)[CP]) {
#pragma unroll
    for (int j = 0; j < CP; ++j) {
        int64_t off = 1024 * j + 16 * lane;
        off = off < nbytes - 16 ? off : nbytes - 16;
        g[j] = __builtin_nontemporal_load(reinterpret_cast<const vu32x4*>(wbase + off));
    }
}

template <int CP>
__device__ __forceinline__ void stage_swap(vu32x4* lds, int lane, const vu32x4 (&g)[CP],
                                           vu32x4 (&v)[CP]) {
#pragma unroll
    for (int j = 0; j < CP; ++j) {
        const int b = 1024 * j + 16 * lane;
        lds[stage_slot<CP>(b / (16 * CP), (b / 16) % CP)] = g[j];
    }
    wave_lds_sync();
#pragma unroll
    for (int c = 0; c < CP; ++c) v[c] = lds[stage_slot<CP>(lane, c)];
    wave_lds_sync();   // every lane has read before the region is written again
}

template <int NMAX, int KIND>
__global__ void __launch_bounds__(kVoteThreads) timing_votes_staged_kernel(
    const char* __restrict__ fp, const char* __restrict__ tp, int64_t G, int64_t n_units,
    double kappa, VoteOut fo, VoteOut to) {
    constexpr int R = NMAX;
    constexpr int CPF = NMAX / 2;                                // u64 fingerprints
    constexpr int CPT = KIND == C3_EV_F64 ? NMAX / 2 : NMAX / 4;  // step times
    __shared__ vu32x4 stage[kVoteThreads / 64][64 * CPF];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int64_t wu0 = (int64_t)blockIdx.x * kVoteThreads + wave * 64;
    if (wu0 >= n_units) return;                                  // whole wave past the end
    const int64_t nu = n_units - wu0 < 64 ? n_units - wu0 : 64;
    vu32x4 gf[CPF], gt[CPT], vf[CPF], vt[CPT];
    stage_load<CPF>(fp + wu0 * (16 * CPF), nu * (16 * CPF), lane, gf);
    stage_load<CPT>(tp + wu0 * (16 * CPT), nu * (16 * CPT), lane, gt);
    stage_swap<CPF>(stage[wave], lane, gf, vf);
    stage_swap<CPT>(stage[wave], lane, gt, vt);
    const int64_t u = wu0 + lane;
    if (u >= n_units) return;
    uint64_t ef[NMAX], et[NMAX];
#pragma unroll
    for (int c = 0; c < CPF; ++c) {
        ef[2 * c] = ((uint64_t)vf[c].y << 32) | vf[c].x;
        ef[2 * c + 1] = ((uint64_t)vf[c].w << 32) | vf[c].z;
    }
#pragma unroll
    for (int c = 0; c < CPT; ++c) {
        if constexpr (KIND == C3_EV_F64) {
            et[2 * c] = ((uint64_t)vt[c].y << 32) | vt[c].x;
            et[2 * c + 1] = ((uint64_t)vt[c].w << 32) | vt[c].z;
        } else {
            et[4 * c] = vt[c].x;
            et[4 * c + 1] = vt[c].y;
            et[4 * c + 2] = vt[c].z;
            et[4 * c + 3] = vt[c].w;
        }
    }
    store_vote(exact_vote_row<NMAX>(ef, R), R, G, n_units, fo, u);
    store_vote(statistical_vote_row<NMAX, KIND>(et, R, kappa), R, G, n_units, to, u);
}

// Clears n16 16-byte words (the mask area is a multiple of 256 bytes).
__global__ void __launch_bounds__(256) timing_zero_kernel(uint4* __restrict__ p, int64_t n16) {
    const int64_t step = (int64_t)gridDim.x * 256;
    for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n16; i += step)
        p[i] = make_uint4(0u, 0u, 0u, 0u);
}

// Confirmation: kConfirmLanes adjacent lanes per rank, each over a
// contiguous run of whole segments; a lane also reads up to W - 1 timing
// bits past its run so it sees every window that starts in it.  Lanes
// combine with shuffles.  Positions q = t - t_lo (32 bits): iteration t
// counts if q < len, closes this lane's pair (t - 1, t) if 1 <= q <= len,
// and ends window [t - Wt + 1, t], this lane's if Wt - 1 <= q < len + Wt - 1.
// With Wt <= 32 the window ending at bit i of a segment is a 32-bit field
// of the 64 bits (segment : previous segment), evaluated only where a set
// bit enters; longer windows keep a 64-bit shift register.  Segments whose
// set bits cannot raise the maximum or reach the threshold are skipped.
//
// The masks of the rank's kinds are read at fpm[s * stride], tpm[s * stride]
// for segment s: global memory in the three-launch path, LDS in the
// single-pass kernel.
struct ConfirmAcc {
    uint32_t flags, dc, sc, mw;
    int32_t fd, fw;
};

template <bool SHORT>
__device__ __forceinline__ ConfirmAcc confirm_lane(const uint32_t* fpm, const uint32_t* tpm,
                                                   int64_t stride, int64_t T, int Wt, int part,
                                                   bool live) {
    const int64_t n_seg = (T + kSegIters - 1) / kSegIters;
    const int64_t per = (n_seg + kConfirmLanes - 1) / kConfirmLanes;   // segments per lane
    const int64_t s_lo = part * per;
    const int64_t t_lo = s_lo * kSegIters;
    int64_t t_hi = t_lo + per * kSegIters;
    if (t_hi > T) t_hi = T;
    // Read on to where the last window starting before t_hi ends, and at
    // least one iteration past t_hi for the pair (t_hi - 1, t_hi).
    int64_t t_end = t_hi + (Wt > 1 ? Wt - 1 : 1);
    if (t_end > T) t_end = T;
    ConfirmAcc a{0u, 0u, 0u, 0u, -1, -1};
    if (live && t_lo < t_hi) {
        const uint32_t len = (uint32_t)(t_hi - t_lo);
        const uint32_t wlo = (uint32_t)(Wt - 1);
        const uint64_t wmask = Wt >= 64 ? ~0ull : ((1ull << Wt) - 1ull);
        uint32_t prev = 0;                      // the previous segment's bits
        uint64_t hist = 0;                      // (long windows) bit k: iteration t - k
        for (int64_t s0 = s_lo; s0 * kSegIters < t_end; s0 += kPrefetch) {
            // both kinds' masks of the next kPrefetch segments in one batch
            uint32_t tmv[kPrefetch], fmv[kPrefetch];
#pragma unroll
            for (int j = 0; j < kPrefetch; ++j) {
                tmv[j] = (s0 + j) * kSegIters < t_end ? tpm[(s0 + j) * stride] : 0u;
                fmv[j] = (s0 + j) * kSegIters < t_hi ? fpm[(s0 + j) * stride] : 0u;
            }
#pragma unroll
            for (int j = 0; j < kPrefetch; ++j) {
                // fingerprint bits: counts and the first attributed iteration
                // (bits past T were never set)
                if (fmv[j] != 0u && a.fd < 0)
                    a.fd = (int32_t)((s0 + j) * kSegIters + __builtin_ctz(fmv[j]));
                a.dc += (uint32_t)__builtin_popcount(fmv[j]);
                const int64_t left = t_end - (s0 + j) * kSegIters;
                const uint32_t n = left <= 0 ? 0u : left < kSegIters ? (uint32_t)left : kSegIters;
                if (n == 0u) break;
                const uint32_t q0 = (uint32_t)((s0 + j - s_lo) * kSegIters);
                const uint32_t tm = n < 32u ? tmv[j] & ((1u << n) - 1u) : tmv[j];
                // counts at positions q0 + i < len
                const uint32_t cn = len > q0 ? (len - q0 < n ? len - q0 : n) : 0u;
                a.sc += (uint32_t)__builtin_popcount(cn < 32u ? tm & ((1u << cn) - 1u) : tm);
                // pairs ending at q0 + i with 1 <= q0 + i <= len
                const uint32_t pairs = tm & ((tm << 1) | (prev >> 31));
                const uint32_t p_hi = len + 1u > q0 ? (len + 1u - q0 < n ? len + 1u - q0 : n) : 0u;
                const uint32_t p_mask = (p_hi < 32u ? (1u << p_hi) - 1u : ~0u) & (q0 == 0u ? ~1u : ~0u);
                if (pairs & p_mask) a.flags |= C3_RANK_CONSEC2;
                // windows ending at positions i in [lo_i, hi_i) of this segment
                const uint32_t lo_i = wlo > q0 ? wlo - q0 : 0u;
                const uint32_t hi_q = wlo + len - q0;       // exclusive, may exceed n
                const uint32_t hi_i = wlo + len > q0 ? (hi_q < n ? hi_q : n) : 0u;
                // No window here can raise the maximum or pass the threshold
                // when all set bits of (segment : previous) could not.
                const uint32_t ybits = (uint32_t)__builtin_popcount(tm) + __builtin_popcount(prev);
                if (SHORT) {
                    // a window holds at most Wt iterations
                    const uint32_t ycap = ybits < (uint32_t)Wt ? ybits : (uint32_t)Wt;
                    if ((ycap > a.mw || (2u * ycap > (uint32_t)Wt && a.fw < 0)) && lo_i < hi_i) {
                        // A window count only grows when a set bit enters, so
                        // the maximum and the first window over the threshold
                        // end at a set bit -- or at the lane's first window
                        // end, whose count owes nothing to entering bits.
                        const uint64_t y = ((uint64_t)tm << 32) | prev;
                        const uint32_t wm = (uint32_t)wmask;
                        const uint32_t range = (hi_i >= 32u ? ~0u : (1u << hi_i) - 1u) &
                                               ~((1u << lo_i) - 1u);
                        uint32_t ev = tm & range;
                        if (wlo >= q0 && wlo - q0 < n) ev |= 1u << (wlo - q0);
                        while (ev != 0u) {
                            const uint32_t i = (uint32_t)__builtin_ctz(ev);
                            ev &= ev - 1u;
                            const uint32_t c = (uint32_t)__builtin_popcount(
                                (uint32_t)(y >> (33u + i - (uint32_t)Wt)) & wm);
                            a.mw = c > a.mw ? c : a.mw;
                            if (2u * c > (uint32_t)Wt && a.fw < 0)
                                a.fw = (int32_t)(t_lo + (int64_t)(q0 + i - wlo));
                            // a full window: no later one raises the maximum
                            // or comes first (a rank slow in every iteration)
                            if (a.mw >= (uint32_t)Wt && a.fw >= 0) break;
                        }
                    }
                } else {
                    // once a window is full nothing the windows give can change
                    if ((tm != 0u || hist != 0ull) && !(a.mw >= (uint32_t)Wt && a.fw >= 0)) {
                        for (uint32_t i = 0; i < n; ++i) {
                            hist = (hist << 1) | ((tm >> i) & 1u);
                            if (i >= lo_i && i < hi_i) {
                                const uint32_t c = (uint32_t)__builtin_popcountll(hist & wmask);
                                a.mw = c > a.mw ? c : a.mw;
                                if (2u * c > (uint32_t)Wt && a.fw < 0)
                                    a.fw = (int32_t)(t_lo + (int64_t)(q0 + i - wlo));
                            }
                        }
                    }
                }
                prev = tm;
            }
        }
    }
    return a;
}

// Combines the L lanes of one rank (sums, maxima, first -- smallest
// non-negative -- positions); lane `part` 0 of a live rank writes its
// verdict.  Every lane of the wave must call it.
template <int L = kConfirmLanes>
__device__ __forceinline__ void confirm_store(ConfirmAcc a, bool live, int part,
                                              c3_rank_verdict_t* __restrict__ verdicts,
                                              int64_t rank) {
#pragma unroll
    for (int o = 1; o < L; o <<= 1) {
        a.flags |= (uint32_t)__shfl_xor((int)a.flags, o, L);
        a.dc += (uint32_t)__shfl_xor((int)a.dc, o, L);
        a.sc += (uint32_t)__shfl_xor((int)a.sc, o, L);
        const uint32_t m2 = (uint32_t)__shfl_xor((int)a.mw, o, L);
        a.mw = m2 > a.mw ? m2 : a.mw;
        const int32_t f2 = __shfl_xor(a.fd, o, L);
        a.fd = (a.fd < 0 || (f2 >= 0 && f2 < a.fd)) ? f2 : a.fd;
        const int32_t w2 = __shfl_xor(a.fw, o, L);
        a.fw = (a.fw < 0 || (w2 >= 0 && w2 < a.fw)) ? w2 : a.fw;
    }
    if (!live || part != 0) return;
    if (a.fw >= 0) a.flags |= C3_RANK_STRAGGLER;
    if (a.fd >= 0) a.flags |= C3_RANK_PROTOCOL;
    c3_rank_verdict_t v;
    v.flags = a.flags;
    v.first_divergent_iter = a.fd;
    v.divergent_count = a.dc;
    v.slow_count = a.sc;
    v.max_window_slow = a.mw;
    v.first_straggler_window = a.fw;
    verdicts[rank] = v;
}

// Confirmation of one rank from masks in LDS, windows of at most 32
// iterations, by L lanes: lane `part` owns segments [part * per, part * per
// + per) and evaluates every window that ends in them, so it reads nothing
// past its own segments (the segment before its first gives the bits that
// windows ending early in it reach back to).  Within a segment a window's
// count rises only where a set bit enters, so the windows evaluated are
// those ending at a set bit or at the segment's first position.  A window
// ending before position Wt - 1 is a prefix of the first whole window
// (start 0) and never counts more, so it is evaluated as if whole, with its
// start clamped to 0: it raises the maximum or passes the threshold only
// when the first whole window does.  All arithmetic is 32-bit and the loop
// count is the same on every lane.
template <int L>
__device__ __forceinline__ ConfirmAcc confirm_owned(const uint32_t* fpm, const uint32_t* tpm,
                                                    int stride, int n_seg, int Wt, int part,
                                                    bool live) {
    const int per = (n_seg + L - 1) / L;
    const int s_lo = part * per;
    const uint32_t w = (uint32_t)Wt;
    const uint32_t wm = w >= 32u ? ~0u : (1u << w) - 1u;
    ConfirmAcc a{0u, 0u, 0u, 0u, -1, -1};
    uint32_t pairs = 0u;
    uint32_t prev = live && s_lo > 0 && s_lo <= n_seg ? tpm[(s_lo - 1) * stride] : 0u;
    for (int j = 0; j < per; ++j) {
        const int sg = s_lo + j;
        const bool in = live && sg < n_seg;
        const uint32_t f = in ? fpm[sg * stride] : 0u;
        const uint32_t tm = in ? tpm[sg * stride] : 0u;
        if (f != 0u && a.fd < 0) a.fd = sg * kSegIters + __builtin_ctz(f);
        a.dc += (uint32_t)__builtin_popcount(f);
        const uint32_t nt = (uint32_t)__builtin_popcount(tm);
        a.sc += nt;
        pairs |= tm & ((tm << 1) | (prev >> 31));
        // a window ending here holds at most the set bits of this segment
        // and the previous one, and at most Wt
        const uint32_t yb = nt + (uint32_t)__builtin_popcount(prev);
        const uint32_t ycap = yb < w ? yb : w;
        if (ycap > a.mw || (2u * ycap > w && a.fw < 0)) {
            const uint64_t y = ((uint64_t)tm << 32) | prev;
            const int st0 = sg * kSegIters - Wt + 1;    // start of the window ending at position 0
            auto window = [&](uint32_t i) {
                const uint32_t c = (uint32_t)__builtin_popcount((uint32_t)(y >> (33u + i - w)) & wm);
                a.mw = c > a.mw ? c : a.mw;
                if (2u * c > w && a.fw < 0) a.fw = st0 + (int)i > 0 ? st0 + (int)i : 0;
            };
            // The first position and the two lowest set bits without a
            // branch (a missing bit repeats position 0), so that a wave loops
            // only where a lane has a third set bit in this segment; the
            // windows are taken in ascending order, so the first over the
            // threshold is the one kept.
            window(0u);
            uint32_t ev = tm & ~1u;
            const uint32_t i1 = ev != 0u ? (uint32_t)__builtin_ctz(ev) : 0u;
            ev &= ev - 1u;
            window(i1);
            const uint32_t i2 = ev != 0u ? (uint32_t)__builtin_ctz(ev) : 0u;
            ev &= ev - 1u;
            window(i2);
            // a full window: no later one raises the maximum or comes first
            while (ev != 0u && !(a.mw >= w && a.fw >= 0)) {
                const uint32_t i = (uint32_t)__builtin_ctz(ev);
                ev &= ev - 1u;
                window(i);
            }
        }
        prev = tm;
    }
    if (pairs != 0u) a.flags |= C3_RANK_CONSEC2;
    return a;
}

template <bool SHORT>
__global__ void __launch_bounds__(kConfirmThreads) timing_confirm_kernel(
    const uint32_t* __restrict__ fp_masks, const uint32_t* __restrict__ t_masks, int R, int64_t G,
    int64_t T, int Wt, c3_rank_verdict_t* __restrict__ verdicts) {
    const int64_t idx = (int64_t)blockIdx.x * kConfirmThreads + threadIdx.x;
    const int64_t rank = idx / kConfirmLanes;
    const int part = (int)(idx % kConfirmLanes);
    const bool live = rank < (int64_t)R * G;    // dead lanes still join the shuffles
    const int64_t r = live ? rank / G : 0, g = live ? rank - r * G : 0;
    const ConfirmAcc a = confirm_lane<SHORT>(fp_masks + r * G + g, t_masks + r * G + g,
                                             (int64_t)R * G, T, Wt, part, live);
    confirm_store(a, live, part, verdicts, rank);
}

// ---------------------------------------------------------------------------
// Single-pass timing consensus.  One workgroup owns kPassGroups consecutive
// groups over all T iterations, so every outlier bit of its ranks lands in
// its own LDS: the votes OR the bits into per-rank masks [kind][segment][r]
// [group] there (no global atomics and no clearing launch), and after one
// workgroup barrier the same workgroup confirms its ranks from LDS (windows
// of at most 32 iterations: every rank at once, its segments split among
// the lanes left per rank, confirm_owned).  A
// wave's step is 64 units, kPassIters iterations x kPassGroups groups; the
// step's rows of one kind are kPassIters contiguous runs of kPassGroups
// rows, read with 16-byte loads and passed through the wave's LDS region as
// in the staged kernel (lane l takes back row l: iteration t0 + l /
// kPassGroups, group g0 + l % kPassGroups).  Used with the per-unit results
// of either kind, both or neither, when R equals the group bound, both
// kinds' rows are 16-byte aligned, W <= 64, the masks fit kPassMaskLds
// bytes and there are at least as many workgroups as compute units.
// Per-unit results are written as 16- to 128-byte pieces of each
// iteration's row; on the 32,768-rank workload the pass with those of both
// kinds takes 91.2 us of kernel time against 106.2 us for the three
// launches of the workspace path (clear, votes, confirmation).
// ---------------------------------------------------------------------------
constexpr int kPassGroups = 16;                  // groups per workgroup
constexpr int kPassIters = 64 / kPassGroups;     // iterations per wave step
constexpr int64_t kPassMaskLds = 64 * 1024;      // LDS bytes for the masks

// Eight waves per workgroup, two per SIMD.  On 32,768 ranks x 1,024
// iterations (R = 8, one workgroup per compute unit), per call with HIP
// events, in the build before the one-round confirmation and the step
// counter, verdicts only / with per-unit results: 79.0 / 110.8 us; sixteen
// waves 78.8 / 116.4 (the per-unit form spills at 128 VGPRs); eight groups
// per workgroup, two workgroups per compute unit, 79.7 / 121.2; two steps
// of loads in flight per wave 81.5 us verdicts only.
// Group block of workgroup b: with a grid of a multiple of eight workgroups,
// the blocks that the hardware sends to one XCD (b mod 8) are consecutive,
// so a cache line of per-unit results, which spans the groups of eight
// neighbouring blocks, is written through a single L2 (108.8 against 110.8
// us per call with per-unit results on 32,768 ranks x 1,024 iterations).
__device__ __forceinline__ int64_t pass_group_block(unsigned b, unsigned n) {
    if (n % 8u != 0u) return b;
    return (int64_t)(b % 8u) * (n / 8u) + b / 8u;
}

template <int NMAX>
struct PassShape {
    static constexpr int waves = 8;
    static constexpr int threads = 64 * waves;
};

// Loads of one kind for one wave step: row i of the step (i = 0..63) is unit
// (t0 + i / kPassGroups, g0 + i % kPassGroups), RB = 16 CP bytes long; load j
// of lane l reads the step's bytes 1024 j + 16 l.  Rows outside the T x ng
// block read row (0, g0) instead, whole.  Non-temporal: every record is read
// once.
template <int CP>
__device__ __forceinline__ void pass_load(const char* __restrict__ base, int64_t G, int64_t T,
                                          int64_t g0, int ng, int64_t t0, int lane,
                                          vu32x4 (&g)[CP]) {
    constexpr int RB = 16 * CP;
#pragma unroll
    for (int j = 0; j < CP; ++j) {
        const int b = 1024 * j + 16 * lane;
        const int row = b / RB;
        const int ti = row / kPassGroups, gi = row % kPassGroups;
        const int64_t t = t0 + ti;
        const bool ok = t < T && gi < ng;
        const int64_t off = (ok ? (t * G + g0 + gi) * RB : g0 * RB) + (b % RB);
        g[j] = __builtin_nontemporal_load(reinterpret_cast<const vu32x4*>(base + off));
    }
}

// The same loads when the whole step lies inside the T x G array: the
// step's first row (t0, g0) is a uniform address and every lane adds its
// loop-invariant 32-bit offset (pass_lane_offsets), so no load spends vector
// instructions on its address.
template <int CP>
__device__ __forceinline__ void pass_lane_offsets(int64_t G, int ng, int lane,
                                                  uint32_t (&off)[CP]) {
    constexpr int RB = 16 * CP;
#pragma unroll
    for (int j = 0; j < CP; ++j) {
        const int b = 1024 * j + 16 * lane;
        const int row = b / RB;
        const int ti = row / kPassGroups;
        int gi = row % kPassGroups;
        gi = gi < ng ? gi : 0;                      // groups past the end re-read group g0
        off[j] = (uint32_t)(((int64_t)ti * G + gi) * RB + (b % RB));
    }
}

template <int CP>
__device__ __forceinline__ void pass_load_full(const char* __restrict__ base, int64_t G,
                                               int64_t g0, int64_t t0, const uint32_t (&off)[CP],
                                               vu32x4 (&g)[CP]) {
    constexpr int RB = 16 * CP;
    const char* step = base + (t0 * G + g0) * RB;
#pragma unroll
    for (int j = 0; j < CP; ++j)
        g[j] = __builtin_nontemporal_load(reinterpret_cast<const vu32x4*>(step + off[j]));
}

// PU: per-unit results written, bit 0 those of the fingerprints, bit 1
// those of the step times.
template <int NMAX, int KIND, bool SHORT, int PU>
__global__ void __launch_bounds__(PassShape<NMAX>::threads) timing_pass_kernel(
    const char* __restrict__ fp, const char* __restrict__ tp, int64_t G, int64_t T, double kappa,
    int Wt, c3_rank_verdict_t* __restrict__ verdicts, VoteOut fo, VoteOut to) {
    constexpr int R = NMAX;
    constexpr int NW = PassShape<NMAX>::waves;
    constexpr int CPF = NMAX / 2;                                // u64 fingerprints
    constexpr int CPT = KIND == C3_EV_F64 ? NMAX / 2 : NMAX / 4;  // step times
    constexpr int SEGW = R * kPassGroups;                        // mask words per segment
    __shared__ vu32x4 stage[NW][64 * CPF];
    extern __shared__ uint32_t pass_masks[];                     // [2][n_seg][R][kPassGroups]
    const int lane = threadIdx.x & 63;
    // the wave index, uniform across the wave (keeps the step addresses scalar)
    const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
    // per-unit results: XCD-aware block order (pass_group_block); without
    // them the plain order reads faster (81.2 against 83.4 us per call)
    const int64_t g0 = (PU != 0 ? pass_group_block(blockIdx.x, gridDim.x) : (int64_t)blockIdx.x) *
                       kPassGroups;
    const int ng = G - g0 < kPassGroups ? (int)(G - g0) : kPassGroups;
    const int64_t n_seg = (T + kSegIters - 1) / kSegIters;
    uint32_t* fmask = pass_masks;
    uint32_t* tmask = pass_masks + n_seg * SEGW;
    __shared__ int32_t step_ctr;     // the next step index to hand out

    const int ti = lane / kPassGroups, gi = lane % kPassGroups;
    const int64_t n_steps = (T + kPassIters - 1) / kPassIters;
    // The next step's rows are loaded before this step's results are
    // stored: the vector-memory counter retires loads and stores in issue
    // order, so waiting for loads issued after the stores would wait for
    // the stores too.  A wave's last step loads nothing more: a load left
    // in flight would hold registers that the confirmation reuses.
    uint32_t off_f[CPF], off_t[CPT];
    pass_lane_offsets<CPF>(G, ng, lane, off_f);
    pass_lane_offsets<CPT>(G, ng, lane, off_t);
    auto load_step = [&](int64_t t0, vu32x4 (&gf)[CPF], vu32x4 (&gt)[CPT]) {
        if (t0 + kPassIters <= T) {               // uniform: a whole step
            pass_load_full<CPF>(fp, G, g0, t0, off_f, gf);
            pass_load_full<CPT>(tp, G, g0, t0, off_t, gt);
        } else {                                  // the last, partial step
            pass_load<CPF>(fp, G, T, g0, ng, t0, lane, gf);
            pass_load<CPT>(tp, G, T, g0, ng, t0, lane, gt);
        }
    };
    vu32x4 gf[CPF], gt[CPT];
    auto do_step = [&](int64_t st, int64_t nx) -> int64_t {
        const int64_t t0 = st * kPassIters;
        vu32x4 vf[CPF], vt[CPT];
        stage_swap<CPF>(stage[wave], lane, gf, vf);
        stage_swap<CPT>(stage[wave], lane, gt, vt);
        if (nx < n_steps) load_step(nx * kPassIters, gf, gt);
        int32_t nn = 0;
        if (lane == 0) nn = atomicAdd(&step_ctr, 1);
        const int64_t t = t0 + ti;
        const bool valid = t < T && gi < ng;
        uint64_t ef[NMAX], et[NMAX];
#pragma unroll
        for (int c = 0; c < CPF; ++c) {
            ef[2 * c] = ((uint64_t)vf[c].y << 32) | vf[c].x;
            ef[2 * c + 1] = ((uint64_t)vf[c].w << 32) | vf[c].z;
        }
#pragma unroll
        for (int c = 0; c < CPT; ++c) {
            if constexpr (KIND == C3_EV_F64) {
                et[2 * c] = ((uint64_t)vt[c].y << 32) | vt[c].x;
                et[2 * c + 1] = ((uint64_t)vt[c].w << 32) | vt[c].z;
            } else {
                et[4 * c] = vt[c].x;
                et[4 * c + 1] = vt[c].y;
                et[4 * c + 2] = vt[c].z;
                et[4 * c + 3] = vt[c].w;
            }
        }
        const UnitVote vfp = exact_vote_row<NMAX>(ef, R);
        // without the times' per-unit results only the bitmaps are kept: no
        // lower-median replica
        const UnitVote vtm = statistical_vote_row<NMAX, KIND, (PU & 2) != 0>(et, R, kappa);
        if constexpr (PU != 0) {
            // Every lane stores: a path without the stores would make the
            // wait for the next step's loads cover them.  A lane outside
            // the block holds the row it loaded instead -- (t, g0) in a whole
            // step, (0, g0) in the last one -- and writes that unit's
            // results again, unchanged.
            const int64_t u = valid ? t * G + g0 + gi : (t0 + kPassIters <= T ? t * G + g0 : g0);
            if constexpr ((PU & 1) != 0) {
                fo.status[u] = vfp.status;
                fo.bitmap[u] = vfp.bitmap;
                fo.majority[u] = vfp.majority;
            }
            if constexpr ((PU & 2) != 0) {
                to.status[u] = vtm.status;
                to.bitmap[u] = vtm.bitmap;
                to.majority[u] = vtm.majority;
            }
        }
        if (valid) {
            const uint32_t bit = 1u << (t & (kSegIters - 1));
            const int64_t w0 = (t / kSegIters) * SEGW + gi;
            for (uint64_t b = vfp.bitmap; b != 0ull; b &= b - 1ull)
                atomicOr(fmask + w0 + __builtin_ctzll(b) * kPassGroups, bit);
            for (uint64_t b = vtm.bitmap; b != 0ull; b &= b - 1ull)
                atomicOr(tmask + w0 + __builtin_ctzll(b) * kPassGroups, bit);
        }
        return (int64_t)__builtin_amdgcn_readfirstlane(nn);
    };
    // the first step's rows are requested before the masks are cleared
    if (wave < n_steps) load_step((int64_t)wave * kPassIters, gf, gt);
    for (int64_t i = threadIdx.x; i < 2 * n_seg * SEGW; i += PassShape<NMAX>::threads)
        pass_masks[i] = 0u;
    if (threadIdx.x == 0) step_ctr = 2 * NW;
    __syncthreads();
    if (wave < n_steps) {
        // The first step outside the loop, so that every path into the
        // loop ends with one step's loads and then (with per-unit results)
        // its stores, and the waits for the loads never cover the stores.
        // Wave w takes steps w and w + NW, then steps from the workgroup's
        // counter; the ticket for the step after next is taken during a
        // step, so its latency is hidden.
        int64_t st = wave + NW;
        int64_t nx = do_step(wave, st);
        while (st < n_steps) {
            const int64_t nn = do_step(st, nx);
            st = nx;
            nx = nn;
        }
    }
    __syncthreads();

    // confirmation of the workgroup's ranks (r, g0 + gi)
    if constexpr (SHORT) {
        // every rank at once: CL lanes each, each lane owning whole segments
        constexpr int CL = PassShape<NMAX>::threads / (R * kPassGroups);
        static_assert(CL >= 1 && (CL & (CL - 1)) == 0 && CL <= 64, "lanes per rank");
        const int lr = (int)threadIdx.x / CL;            // r * kPassGroups + gi
        const int part = (int)threadIdx.x % CL;
        const int r = lr / kPassGroups, gr = lr % kPassGroups;
        const bool live = gr < ng;
        const int off = live ? r * kPassGroups + gr : 0;
        const ConfirmAcc a =
            confirm_owned<CL>(fmask + off, tmask + off, SEGW, (int)n_seg, Wt, part, live);
        confirm_store<CL>(a, live, part, verdicts, (int64_t)r * G + g0 + gr);
        return;
    }
    // longer windows: kConfirmLanes lanes per rank, in rounds
    constexpr int per_pass = PassShape<NMAX>::threads / kConfirmLanes;
#pragma unroll 1
    for (int base = 0; base < R * kPassGroups; base += per_pass) {
        const int lr = base + (int)threadIdx.x / kConfirmLanes;    // r * kPassGroups + gi
        const int part = (int)threadIdx.x % kConfirmLanes;
        const int r = lr / kPassGroups, gr = lr % kPassGroups;
        const bool live = lr < R * kPassGroups && gr < ng;
        const int off = live ? r * kPassGroups + gr : 0;
        const ConfirmAcc a = confirm_lane<SHORT>(fmask + off, tmask + off, SEGW, T, Wt, part, live);
        confirm_store(a, live, part, verdicts, (int64_t)r * G + g0 + gr);
    }
}

int64_t timing_masks_bytes(int R, int64_t G, int64_t T) {
    const int64_t n_seg = (T + kSegIters - 1) / kSegIters;
    return 2 * ((n_seg * R * G * 4 + 255) / 256 * 256);
}

template <int NMAX, int KIND>
static hipError_t launch_votes(const uint64_t* fp, const char* tp, int R, int64_t G,
                               int64_t n_units, double kappa, const VoteOut& fo, const VoteOut& to,
                               hipStream_t stream) {
    const int64_t blocks = (n_units + kVoteThreads - 1) / kVoteThreads;
    constexpr int64_t tsize = KIND == C3_EV_F64 ? 8 : 4;
    const bool fp_dense = (R * 8) % 16 == 0 && ((uintptr_t)fp & 15) == 0;
    const bool t_dense = (R * tsize) % 16 == 0 && ((uintptr_t)tp & 15) == 0;
    if (blocks > 0x7FFFFFFF) return hipErrorInvalidValue;
    if (blocks == 0) return hipSuccess;
    if (fp_dense && t_dense && R == NMAX)
        hipLaunchKernelGGL((timing_votes_staged_kernel<NMAX, KIND>), dim3((unsigned)blocks),
                           dim3(kVoteThreads), 0, stream, reinterpret_cast<const char*>(fp), tp, G,
                           n_units, kappa, fo, to);
    else if (fp_dense && t_dense)
        hipLaunchKernelGGL((timing_votes_kernel<NMAX, KIND, true>), dim3((unsigned)blocks),
                           dim3(kVoteThreads), 0, stream, reinterpret_cast<const char*>(fp), tp, R,
                           G, n_units, kappa, fp_dense, t_dense, fo, to);
    else
        hipLaunchKernelGGL((timing_votes_kernel<NMAX, KIND, false>), dim3((unsigned)blocks),
                           dim3(kVoteThreads), 0, stream, reinterpret_cast<const char*>(fp), tp, R,
                           G, n_units, kappa, fp_dense, t_dense, fo, to);
    return hipGetLastError();
}

template <int NMAX>
static hipError_t launch_votes(const uint64_t* fp, const char* tp, int time_kind, int R, int64_t G,
                               int64_t n_units, double kappa, const VoteOut& fo, const VoteOut& to,
                               hipStream_t stream) {
    if (time_kind == C3_EV_F32)
        return launch_votes<NMAX, C3_EV_F32>(fp, tp, R, G, n_units, kappa, fo, to, stream);
    return launch_votes<NMAX, C3_EV_F64>(fp, tp, R, G, n_units, kappa, fo, to, stream);
}

template <int NMAX, int KIND>
static hipError_t launch_pass(const char* fp, const char* tp, int64_t G, int64_t T, double kappa,
                              int Wt, c3_rank_verdict_t* verdicts, const VoteOut& fo,
                              const VoteOut& to, size_t lds, hipStream_t stream) {
    const dim3 grid((unsigned)((G + kPassGroups - 1) / kPassGroups));
    const dim3 block(PassShape<NMAX>::threads);
    const int pu = (fo.status != nullptr ? 1 : 0) | (to.status != nullptr ? 2 : 0);
#define C3_PASS(S, P)                                                                     \
    hipLaunchKernelGGL((timing_pass_kernel<NMAX, KIND, S, P>), grid, block, lds, stream, fp, \
                       tp, G, T, kappa, Wt, verdicts, fo, to)
    if (Wt <= 32) {
        switch (pu) {
            case 0: C3_PASS(true, 0); break;
            case 1: C3_PASS(true, 1); break;
            case 2: C3_PASS(true, 2); break;
            default: C3_PASS(true, 3); break;
        }
    } else {
        switch (pu) {
            case 0: C3_PASS(false, 0); break;
            case 1: C3_PASS(false, 1); break;
            case 2: C3_PASS(false, 2); break;
            default: C3_PASS(false, 3); break;
        }
    }
#undef C3_PASS
    return hipGetLastError();
}

// The single pass applies: R is a group bound with dense 16-byte aligned rows,
// the masks fit in LDS, and the groups give every compute unit a workgroup.
static bool pass_applies(const void* fp, const void* times, int time_kind, int R, int64_t G,
                         int64_t T, int Wt, hipStream_t stream, size_t& lds) {
    if (R != 4 && R != 8 && R != 16) return false;
    const int tsize = time_kind == C3_EV_F64 ? 8 : 4;
    if (((uintptr_t)fp & 15) != 0 || ((uintptr_t)times & 15) != 0 || (R * tsize) % 16 != 0)
        return false;
    if (T < 1 || Wt > 64) return false;
    // the lanes' offsets within a step are 32-bit
    if ((int64_t)kPassIters * G * R * 8 >= ((int64_t)1 << 31)) return false;
    const int64_t n_seg = (T + kSegIters - 1) / kSegIters;
    const int64_t bytes = 2 * n_seg * R * kPassGroups * 4;
    if (bytes > kPassMaskLds) return false;
    const int cus = stream_cu_count(stream);
    if (cus <= 0 || (G + kPassGroups - 1) / kPassGroups < cus) return false;
    lds = (size_t)bytes;
    return true;
}

hipError_t launch_timing_consensus(const uint64_t* fp, const void* times, int time_kind, int R,
                                   int64_t G, int64_t T, double kappa, int window,
                                   uint8_t* fp_status, uint64_t* fp_bitmap, int32_t* fp_majority,
                                   uint8_t* t_status, uint64_t* t_bitmap, int32_t* t_majority,
                                   c3_rank_verdict_t* verdicts, void* ws, hipStream_t stream) {
    const int64_t ranks = (int64_t)R * G;
    if ((ranks * kConfirmLanes + kConfirmThreads - 1) / kConfirmThreads > 0x7FFFFFFF)
        return hipErrorInvalidValue;
    if (ranks == 0) return hipSuccess;
    // the single pass, with the per-unit results of either kind, both or neither
    {
        const int Wt = (int64_t)window < T ? window : (int)T;
        size_t lds = 0;
        if (pass_applies(fp, times, time_kind, R, G, T, Wt, stream, lds)) {
            const char* f = reinterpret_cast<const char*>(fp);
            const char* tp = static_cast<const char*>(times);
            const bool f64 = time_kind == C3_EV_F64;
            const VoteOut fo = {fp_status, fp_bitmap, fp_majority, nullptr};
            const VoteOut to = {t_status, t_bitmap, t_majority, nullptr};
            if (R == 4)
                return f64 ? launch_pass<4, C3_EV_F64>(f, tp, G, T, kappa, Wt, verdicts, fo, to, lds, stream)
                           : launch_pass<4, C3_EV_F32>(f, tp, G, T, kappa, Wt, verdicts, fo, to, lds, stream);
            if (R == 8)
                return f64 ? launch_pass<8, C3_EV_F64>(f, tp, G, T, kappa, Wt, verdicts, fo, to, lds, stream)
                           : launch_pass<8, C3_EV_F32>(f, tp, G, T, kappa, Wt, verdicts, fo, to, lds, stream);
            return f64 ? launch_pass<16, C3_EV_F64>(f, tp, G, T, kappa, Wt, verdicts, fo, to, lds, stream)
                       : launch_pass<16, C3_EV_F32>(f, tp, G, T, kappa, Wt, verdicts, fo, to, lds, stream);
        }
    }
    const int64_t half = timing_masks_bytes(R, G, T) / 2;
    uint32_t* fm = static_cast<uint32_t*>(ws);
    uint32_t* tm = reinterpret_cast<uint32_t*>(static_cast<char*>(ws) + half);
    // the masks collect bits by atomic OR: clear them with a kernel (a memset
    // node would not survive graph capture reliably)
    const int64_t n16 = 2 * half / 16;
    if (n16 > 0) {
        const int64_t blocks = (n16 + 255) / 256 < 4096 ? (n16 + 255) / 256 : 4096;
        hipLaunchKernelGGL(timing_zero_kernel, dim3((unsigned)blocks), dim3(256), 0, stream,
                           reinterpret_cast<uint4*>(fm), n16);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    const char* tp = static_cast<const char*>(times);
    const int64_t n_units = T * G;
    const VoteOut fo = {fp_status, fp_bitmap, fp_majority, fm};
    const VoteOut to = {t_status, t_bitmap, t_majority, tm};
    hipError_t e;
    if (R <= 4)
        e = launch_votes<4>(fp, tp, time_kind, R, G, n_units, kappa, fo, to, stream);
    else if (R <= 8)
        e = launch_votes<8>(fp, tp, time_kind, R, G, n_units, kappa, fo, to, stream);
    else
        e = launch_votes<16>(fp, tp, time_kind, R, G, n_units, kappa, fo, to, stream);
    if (e != hipSuccess) return e;
    const int Wt = (int64_t)window < T ? window : (int)T;
    const int64_t threads = ranks * kConfirmLanes;
    const dim3 grid((unsigned)((threads + kConfirmThreads - 1) / kConfirmThreads));
    if (Wt <= 32)
        hipLaunchKernelGGL(timing_confirm_kernel<true>, grid, dim3(kConfirmThreads), 0, stream, fm,
                           tm, R, G, T, Wt, verdicts);
    else
        hipLaunchKernelGGL(timing_confirm_kernel<false>, grid, dim3(kConfirmThreads), 0, stream, fm,
                           tm, R, G, T, Wt, verdicts);
    return hipGetLastError();
}

}  // namespace c3
