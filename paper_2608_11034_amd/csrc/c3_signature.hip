// Streaming signature kernel of C3 for gfx950.
//
// Per (replica, chunk) it computes the C3SIG-1 signature -- a per-chunk
// reading of the paper's comparable evidence H_w(dtype, shape, bytes)
// (Sec. 5.2) -- and, in the same single pass over HBM, the chunk's NaN/Inf
// counts, absmax and fp64 sum / sum of squares of the finite elements.
//
// C3SIG-1 over a chunk of n bytes: the bytes, zero-padded to a multiple of 16,
// are little-endian u32 words m[0..D-1], D = 4 ceil(n / 16).  Keys K[i] are
// the low 32 bits of SplitMix64 outputs i = 0..257 from a fixed seed.  For
// each word pair p = 2i, with q = p mod 256 and beta = (p div 256) * 0x9E3779B9
// (all u32 arithmetic wraps):
//     A += (m[p] + K[q] + beta) * (m[p+1] + K[q+1] + beta)      (u64, wraps)
//     B += (m[p] + K[q+2] + beta) * (m[p+1] + K[q+3] + beta)
// which is the NH hash of UMAC with a Toeplitz-shifted second key row.  The
// signature is an fmix64 chain over (tag ^ dtype << 32 ^ ndim, shape dims,
// chunk index, n, A, B).  A and B are sums, so any partition of the chunk
// gives the same bits.
//
// Work decomposition: a chunk is cut into tiles of tile_bytes (a power of two
// >= 1 KiB dividing chunk_bytes).  One 256-thread workgroup folds one tile:
// its four waves take the tile's 1 KiB blocks round-robin, every lane loads
// 16 bytes of a block with one 128-bit load, so one wave-wide load covers
// exactly 256 words and lane l always owns key positions 4l .. 4l+5 (held in
// VGPRs for the whole kernel) while beta is wave-uniform.  Lanes reduce with
// xor butterflies, waves combine through LDS in a fixed order, and each tile
// writes one 64-byte partial.  When a chunk is a single tile the workgroup
// writes the chunk record directly; otherwise a finalize kernel combines the
// chunk's partials in tile order.  The per-tile arithmetic never depends on
// which workgroup runs it, so results are independent of the grid size.
//
// Non-finite screen: a lane sums its elements in fp64 without looking at
// them.  A non-finite element is the only way its sum or sum of squares can
// become non-finite (finite fp32/bf16/fp16 values cannot overflow fp64 here),
// so a lane whose sums end non-finite re-reads its own segments and
// classifies every element.  Healthy data never takes that path.
#include "c3_device.h"
#include "c3_internal.h"
#include "c3_vote_row.h"

namespace c3 {

struct LaneKeys {
    uint32_t k0, k1, k2, k3, k4, k5;
};

// beta of block b (wave-uniform, so it stays in a scalar register)
__device__ inline uint32_t block_beta(uint32_t b) { return b * kBlockMul; }

// m + k + beta as one three-input add with beta as the scalar operand.  The
// compiler would otherwise re-associate to m + (k + beta) and spend a
// separate add on each of the six key sums per block.
__device__ inline uint32_t add3(uint32_t m, uint32_t k, uint32_t beta) {
    uint32_t r;
    asm("v_add3_u32 %0, %1, %2, %3" : "=v"(r) : "v"(m), "v"(k), "s"(beta));
    return r;
}

// NH over one 16-byte segment (two word pairs) at key offset 4 * lane.
__device__ inline void nh16(const u32x4 v, const LaneKeys& K, uint32_t beta, uint64_t& A,
                            uint64_t& B) {
    A += (uint64_t)add3(v.x, K.k0, beta) * (uint64_t)add3(v.y, K.k1, beta);
    B += (uint64_t)add3(v.x, K.k2, beta) * (uint64_t)add3(v.y, K.k3, beta);
    A += (uint64_t)add3(v.z, K.k2, beta) * (uint64_t)add3(v.w, K.k3, beta);
    B += (uint64_t)add3(v.z, K.k4, beta) * (uint64_t)add3(v.w, K.k5, beta);
}

__device__ inline double f16_to_f64(uint32_t h) {
    _Float16 x = __builtin_bit_cast(_Float16, (uint16_t)h);
    return (double)(float)x;
}

// ---------------------------------------------------------------------------
// fast statistics: no classification.  `mf` collects the largest magnitude as
// an fp32 value (every fp32, bf16 and fp16 value is one exactly); a NaN or
// Inf may poison it, but such a lane takes the classifying path below, which
// starts over.
// ---------------------------------------------------------------------------
// max(|a|, |b|, |c|) in one instruction (abs source modifiers); NaN
// propagates, which only matters on lanes the classifying path redoes.
__device__ inline float absmax3(float a, float b, float c) {
    float r;
    asm("v_maximum3_f32 %0, |%1|, |%2|, |%3|" : "=v"(r) : "v"(a), "v"(b), "v"(c));
    return r;
}

template <int DT>
__device__ inline void stats_fast(const u32x4 v, double& s, double& q, float& mf) {
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
    if constexpr (DT == C3_F32) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            double d = (double)__uint_as_float(w[i]);
            s += d;
            q = __fma_rn(d, d, q);
        }
        mf = absmax3(mf, absmax3(__uint_as_float(w[0]), __uint_as_float(w[1]), __uint_as_float(w[2])),
                     __uint_as_float(w[3]));
    } else if constexpr (DT == C3_BF16 || DT == C3_F16) {
        float x[8];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            if constexpr (DT == C3_BF16) {
                x[2 * i] = __uint_as_float(w[i] << 16);
                x[2 * i + 1] = __uint_as_float(w[i] & 0xFFFF0000u);
            } else {
                x[2 * i] = (float)__builtin_bit_cast(_Float16, (uint16_t)(w[i] & 0xFFFFu));
                x[2 * i + 1] = (float)__builtin_bit_cast(_Float16, (uint16_t)(w[i] >> 16));
            }
        }
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const double d = (double)x[i];
            s += d;
            q = __fma_rn(d, d, q);
        }
        mf = absmax3(absmax3(x[0], x[1], x[2]), absmax3(x[3], x[4], x[5]), absmax3(x[6], x[7], mf));
    }
}

// magnitude bits of the type from the fp32 value of a finite magnitude
template <int DT>
__device__ inline uint32_t magnitude_bits(float mf) {
    if constexpr (DT == C3_BF16) return __float_as_uint(mf) >> 16;  // exact: a bf16 value
    if constexpr (DT == C3_F16) return (uint32_t)__builtin_bit_cast(uint16_t, (_Float16)mf);
    return __float_as_uint(mf);
}

// slow statistics: classify each element; `mx` is a plain magnitude
template <int DT>
__device__ inline void stats_slow(const u32x4 v, double& s, double& q, uint32_t& mx,
                                  uint32_t& nan_c, uint32_t& inf_c) {
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
    if constexpr (DT == C3_F32) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            uint32_t mag = w[i] & 0x7FFFFFFFu;
            if (mag >= 0x7F800000u) {
                if (mag > 0x7F800000u) ++nan_c; else ++inf_c;
                continue;
            }
            double d = (double)__uint_as_float(w[i]);
            s += d;
            q = __fma_rn(d, d, q);
            mx = max(mx, mag);
        }
    } else {
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            uint32_t h = (i & 1) ? (w[i >> 1] >> 16) : (w[i >> 1] & 0xFFFFu);
            uint32_t mag = h & 0x7FFFu;
            const uint32_t inf_bits = (DT == C3_BF16) ? 0x7F80u : 0x7C00u;
            if (mag >= inf_bits) {
                if (mag > inf_bits) ++nan_c; else ++inf_c;
                continue;
            }
            double d = (DT == C3_BF16) ? (double)__uint_as_float(h << 16) : f16_to_f64(h);
            s += d;
            q = __fma_rn(d, d, q);
            mx = max(mx, mag);
        }
    }
}

// Tail segment of a tile: bytes [0, rem) of a 16-byte segment, rest zero.
__device__ inline u32x4 load_partial(const uint8_t* p, uint32_t rem) {
    uint32_t w[4] = {0u, 0u, 0u, 0u};
    for (uint32_t b = 0; b < rem; ++b) w[b >> 2] |= (uint32_t)p[b] << (8 * (b & 3));
    u32x4 v;
    v.x = w[0];
    v.y = w[1];
    v.z = w[2];
    v.w = w[3];
    return v;
}

struct LaneFold {
    uint64_t A, B;
    double s, q;
    uint32_t mx, nan_c, inf_c;
};

// One wave's share of a tile: blocks wave, wave + 4, ... of `len` bytes.
// Full blocks are read with raw buffer loads: the resource is the tile (a
// wave-uniform base, `len` bytes), the scalar offset the block, the vector
// offset the lane's 16 bytes, so no load spends vector instructions on its
// address.  Each block's beta is pinned in a scalar register, so every key
// sum is one three-input add.
template <int DT, int U>
__device__ inline LaneFold fold_lane(const uint8_t* tile, uint32_t len, uint32_t blk0,
                                     const LaneKeys& K, int wave, int lane) {
    LaneFold f{0, 0, 0.0, 0.0, 0u, 0u, 0u};
    float mf = 0.0f;
    const uint32_t off = (uint32_t)lane * 16u;
    const int nfull = (int)(len >> 10);
    const uint32_t tail = len & 1023u;
    const __amdgpu_buffer_rsrc_t rs = tile_resource(tile, len);
    int k = wave;
    for (; k + 4 * (U - 1) < nfull; k += 4 * U) {
        u32x4 v[U];
#pragma unroll
        for (int u = 0; u < U; ++u) v[u] = load16_buf(rs, off, (uint32_t)(k + 4 * u) << 10);
        // keep all U loads in flight before the first use
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const uint32_t beta = block_beta(blk0 + (uint32_t)(k + 4 * u));
            nh16(v[u], K, beta, f.A, f.B);
            stats_fast<DT>(v[u], f.s, f.q, mf);
        }
    }
    if (k < nfull) {
        // fewer than U blocks left for this wave: one more batch, all loads in
        // flight together; the tests are wave-uniform (scalar branches).
        u32x4 v[U];
#pragma unroll
        for (int u = 0; u < U; ++u)
            if (k + 4 * u < nfull) v[u] = load16_buf(rs, off, (uint32_t)(k + 4 * u) << 10);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int u = 0; u < U; ++u) {
            if (k + 4 * u < nfull) {
                nh16(v[u], K, block_beta(blk0 + (uint32_t)(k + 4 * u)), f.A, f.B);
                stats_fast<DT>(v[u], f.s, f.q, mf);
            }
        }
    }
    const bool has_tail = tail != 0u && (nfull & 3) == wave && off < tail;
    if (has_tail) {
        const uint8_t* seg = tile + ((size_t)nfull << 10) + off;
        u32x4 v = (off + 16u <= tail) ? load16(reinterpret_cast<const u32x4*>(seg))
                                      : load_partial(seg, tail - off);
        nh16(v, K, (blk0 + (uint32_t)nfull) * kBlockMul, f.A, f.B);
        stats_fast<DT>(v, f.s, f.q, mf);
    }
    if constexpr (DT != C3_RAW) {
        if (!__builtin_isfinite(f.s) || !__builtin_isfinite(f.q)) {
            // rare: this lane saw a NaN or Inf; redo its statistics classifying
            f.s = 0.0;
            f.q = 0.0;
            f.mx = 0u;
            for (int kk = wave; kk < nfull; kk += 4)
                stats_slow<DT>(load16(reinterpret_cast<const u32x4*>(tile + ((size_t)kk << 10) + off)),
                               f.s, f.q, f.mx, f.nan_c, f.inf_c);
            if (has_tail) {
                const uint8_t* seg = tile + ((size_t)nfull << 10) + off;
                u32x4 v = (off + 16u <= tail) ? load16(reinterpret_cast<const u32x4*>(seg))
                                              : load_partial(seg, tail - off);
                stats_slow<DT>(v, f.s, f.q, f.mx, f.nan_c, f.inf_c);
            }
        } else {
            f.mx = magnitude_bits<DT>(mf);
        }
    }
    return f;
}

__device__ inline TilePartial wave_reduce(const LaneFold& f) {
    TilePartial p;
    p.A = f.A;
    p.B = f.B;
    p.s = f.s;
    p.sc = 0.0;
    p.q = f.q;
    p.qc = 0.0;
    p.maxbits = f.mx;
    p.nan_count = f.nan_c;
    p.inf_count = f.inf_c;
    p.pad = 0u;
    // Lane sums meet in a fixed six-level butterfly of plain fp64 adds (error
    // at most 6 ulp of the sum of magnitudes); compensation starts at the
    // cross-wave level.
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) {
        p.A += shfl_xor_u64(p.A, m);
        p.B += shfl_xor_u64(p.B, m);
        p.s += shfl_xor_f64(p.s, m);
        p.q += shfl_xor_f64(p.q, m);
        p.maxbits = max(p.maxbits, shfl_xor_u32(p.maxbits, m));
    }
    if (ballot64(f.nan_c != 0u || f.inf_c != 0u) != 0ull) {
#pragma unroll
        for (int m = 32; m >= 1; m >>= 1) {
            p.nan_count += shfl_xor_u32(p.nan_count, m);
            p.inf_count += shfl_xor_u32(p.inf_count, m);
        }
    }
    return p;
}

__device__ inline void partial_add(TilePartial& a, const TilePartial& b) {
    a.A += b.A;
    a.B += b.B;
    comp_add(a.s, a.sc, b.s, b.sc);
    comp_add(a.q, a.qc, b.q, b.qc);
    a.maxbits = max(a.maxbits, b.maxbits);
    a.nan_count += b.nan_count;
    a.inf_count += b.inf_count;
}

__device__ inline int find_segment(const int64_t* base, int n, int64_t j) {
    // largest t in [0, n) with base[t] <= j  (base[0] = 0, base ascending)
    int lo = 0, hi = n;
    while (hi - lo > 1) {
        const int mid = (lo + hi) >> 1;
        if (base[mid] <= j) lo = mid; else hi = mid;
    }
    return lo;
}

__device__ inline double maxbits_to_f64(uint32_t bits, int dtype) {
    if (dtype == C3_F32) return (double)__uint_as_float(bits);
    if (dtype == C3_BF16) return (double)__uint_as_float(bits << 16);
    if (dtype == C3_F16) return f16_to_f64(bits);
    return 0.0;
}

__device__ inline void write_record(c3_chunk_record_t* rec, const TensorInfo* tip, int t,
                                    uint64_t k, uint64_t n, const TilePartial& p) {
    const int dtype = tip->dtype, ndim = tip->ndim;
    uint64_t h = fmix64(kTag ^ ((uint64_t)(uint32_t)dtype << 32) ^ (uint64_t)(uint32_t)ndim);
    for (int d = 0; d < ndim; ++d) h = fmix64(h ^ (uint64_t)tip->shape[d]);
    h = fmix64(h ^ k);
    h = fmix64(h ^ n);
    h = fmix64(h ^ p.A);
    h = fmix64(h ^ p.B);
    const uint64_t es = dtype == C3_F32 ? 4 : (dtype == C3_RAW ? 1 : 2);
    rec->sig = h;
    rec->n_elems = n / es;
    rec->nan_count = p.nan_count;
    rec->inf_count = p.inf_count;
    rec->tensor = (uint32_t)t;
    rec->chunk_in_tensor = (uint32_t)k;
    rec->absmax = maxbits_to_f64(p.maxbits, dtype);
    rec->sum = p.s + p.sc;
    rec->sumsq = p.q + p.qc;
    rec->reserved = 0;
}

// One launch per element type present in the plan.  The plan lists the
// tensors grouped by type (order[], stable in call order) with a tile prefix
// over that order (gtile[]); this launch covers group positions [gk0, gk1)
// of every replica.
template <int DT, int U>
__global__ void __launch_bounds__(kSigThreads, C3_SIG_WAVES_PER_EU)
    signature_kernel(const SigPlan* __restrict__ plan, c3_chunk_record_t* __restrict__ records,
                     int gk0, int gk1, int64_t gtiles) {
    __shared__ TilePartial lds[kSigThreads / 64];
    const int lane = threadIdx.x & 63;
    // the wave index, uniform across the wave (keeps beta and addresses scalar)
    const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
    const char* pb = reinterpret_cast<const char*>(plan);
    const uint64_t* ptrs = reinterpret_cast<const uint64_t*>(pb + plan->off_ptrs);
    const int64_t* tile_base = reinterpret_cast<const int64_t*>(pb + plan->off_tile_base);
    const int64_t* chunk_base = reinterpret_cast<const int64_t*>(pb + plan->off_chunk_base);
    const int32_t* order = reinterpret_cast<const int32_t*>(pb + plan->off_order);
    const int64_t* gtile = reinterpret_cast<const int64_t*>(pb + plan->off_gtile);
    const TensorInfo* tinfo = reinterpret_cast<const TensorInfo*>(pb + plan->off_tmeta);
    TilePartial* partials = reinterpret_cast<TilePartial*>(const_cast<char*>(pb) + plan->off_partials);
    const int T = plan->T;
    const int64_t ntiles = gtiles * plan->R;
    const uint64_t tile_bytes = plan->tile_bytes;
    const uint32_t tpc = plan->tiles_per_chunk;
    const int64_t g0 = gtile[gk0];

    LaneKeys K;
    K.k0 = nh_key(4u * lane + 0u);
    K.k1 = nh_key(4u * lane + 1u);
    K.k2 = nh_key(4u * lane + 2u);
    K.k3 = nh_key(4u * lane + 3u);
    K.k4 = nh_key(4u * lane + 4u);
    K.k5 = nh_key(4u * lane + 5u);

    for (int64_t i = blockIdx.x; i < ntiles; i += gridDim.x) {
        const int64_t r = i / gtiles;
        const int64_t j = g0 + (i - r * gtiles);
        const int k = gk0 + find_segment(gtile + gk0, gk1 - gk0, j);
        const int t = order[k];
        const int64_t lt = j - gtile[k];
        const uint64_t nbytes = tinfo[t].nbytes;
        const uint64_t toff = (uint64_t)lt * tile_bytes;
        const uint32_t len = nbytes > toff ? (uint32_t)min(tile_bytes, nbytes - toff) : 0u;
        const uint32_t blk0 = (uint32_t)(((uint64_t)(lt % tpc) * tile_bytes) >> 10);
        const uint8_t* tile = reinterpret_cast<const uint8_t*>(ptrs[r * T + t]) + toff;

        const LaneFold f = fold_lane<DT, U>(tile, len, blk0, K, wave, lane);
        const TilePartial wp = wave_reduce(f);
        if (lane == 0) lds[wave] = wp;
        __syncthreads();
        if (threadIdx.x == 0) {
            TilePartial p = lds[0];
#pragma unroll
            for (int w = 1; w < kSigThreads / 64; ++w) partial_add(p, lds[w]);
            if (plan->direct) {
                const uint64_t kc = (uint64_t)lt;  // one tile per chunk
                const uint64_t n = nbytes > toff ? min(plan->chunk_bytes, nbytes - toff) : 0;
                write_record(&records[r * plan->C + chunk_base[t] + (int64_t)kc], tinfo + t, t, kc, n, p);
            } else {
                partials[r * plan->tiles_per_replica + tile_base[t] + lt] = p;
            }
        }
        __syncthreads();
    }
}

// Record of (replica r, chunk c) from its tile partials, combined in tile
// order.
__device__ inline void combine_chunk(const SigPlan* __restrict__ plan, int64_t r, int64_t c,
                                     c3_chunk_record_t* out) {
    const char* pb = reinterpret_cast<const char*>(plan);
    const int64_t* tile_base = reinterpret_cast<const int64_t*>(pb + plan->off_tile_base);
    const int64_t* chunk_base = reinterpret_cast<const int64_t*>(pb + plan->off_chunk_base);
    const TensorInfo* tinfo = reinterpret_cast<const TensorInfo*>(pb + plan->off_tmeta);
    const TilePartial* partials = reinterpret_cast<const TilePartial*>(pb + plan->off_partials);
    const int t = find_segment(chunk_base, plan->T, c);
    const uint64_t k = (uint64_t)(c - chunk_base[t]);
    const uint64_t nbytes = tinfo[t].nbytes;
    const int64_t tiles_t = tile_base[t + 1] - tile_base[t];
    const int64_t lt0 = (int64_t)k * plan->tiles_per_chunk;
    const int64_t nt = min((int64_t)plan->tiles_per_chunk, tiles_t - lt0);
    const TilePartial* pp = partials + r * plan->tiles_per_replica + tile_base[t] + lt0;
    TilePartial p = pp[0];
    for (int64_t x = 1; x < nt; ++x) partial_add(p, pp[x]);
    const uint64_t coff = k * plan->chunk_bytes;
    const uint64_t n = nbytes > coff ? min(plan->chunk_bytes, nbytes - coff) : 0;
    write_record(out, tinfo + t, t, k, n, p);
}

// Combine the partials of each (replica, chunk) in tile order.
__global__ void __launch_bounds__(256) finalize_kernel(const SigPlan* __restrict__ plan,
                                                       c3_chunk_record_t* __restrict__ records) {
    const int64_t C = plan->C;
    const int64_t total = C * plan->R;
    for (int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; idx < total;
         idx += (int64_t)gridDim.x * blockDim.x) {
        const int64_t r = idx / C;
        combine_chunk(plan, r, idx - r * C, &records[idx]);
    }
}

// ---------------------------------------------------------------------------
// Finalize, exact vote and localize of a small plan in one workgroup (the
// optimizer-boundary check signs 7 chunks per replica): three launches of a
// few microseconds each become one.  (1) Every record -- combined from its
// tile partials, or as the streaming kernel wrote it when chunks are whole
// tiles -- is written out and kept in LDS.  (2) One thread per chunk votes
// with exact_vote_row, the rule c3_consensus applies, on the signatures.
// (3) One thread lists the outliers (chunk ascending, replica ascending,
// both replicas' summaries) and the undecided chunks, with the counts, as
// c3_localize does.  Needs R * C <= kTailMaxRecords and C <= kTailThreads.
// ---------------------------------------------------------------------------
constexpr int kTailThreads = 256;
constexpr int kTailMaxRecords = 512;

__global__ void __launch_bounds__(kTailThreads) small_tail_kernel(
    const SigPlan* __restrict__ plan, c3_chunk_record_t* __restrict__ records,
    uint8_t* __restrict__ status, uint64_t* __restrict__ bitmap, int32_t* __restrict__ majority,
    c3_outlier_t* __restrict__ outliers, int64_t out_cap, int64_t* __restrict__ undecided,
    int64_t und_cap, int64_t* __restrict__ counts) {
    __shared__ c3_chunk_record_t rec[kTailMaxRecords];
    __shared__ UnitVote votes[kTailThreads];
    const int R = plan->R;
    const int C = (int)plan->C;
    for (int i = threadIdx.x; i < R * C; i += kTailThreads) {
        if (plan->direct) {
            rec[i] = records[i];
        } else {
            combine_chunk(plan, i / C, i % C, &rec[i]);
            records[i] = rec[i];
        }
    }
    __syncthreads();
    if ((int)threadIdx.x < C) {
        const int u = threadIdx.x;
        UnitVote v;
        if (R <= 16) {
            uint64_t e[16];
#pragma unroll
            for (int r = 0; r < 16; ++r) e[r] = r < R ? rec[r * C + u].sig : 0ull;
            v = exact_vote_row<16>(e, R);
        } else {
            uint64_t e[C3_MAX_REPLICAS];
            for (int r = 0; r < C3_MAX_REPLICAS; ++r) e[r] = r < R ? rec[r * C + u].sig : 0ull;
            v = exact_vote_row<C3_MAX_REPLICAS>(e, R);
        }
        status[u] = v.status;
        bitmap[u] = v.bitmap;
        majority[u] = v.majority;
        votes[u] = v;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        int64_t no = 0, nu = 0, na = 0;
        for (int u = 0; u < C; ++u) {
            const UnitVote v = votes[u];
            if (v.status == C3_INCONCLUSIVE) {
                if (nu < und_cap) undecided[nu] = u;
                ++nu;
                continue;
            }
            if (v.bitmap == 0ull) continue;
            ++na;
            for (uint64_t b = v.bitmap; b != 0ull; b &= b - 1ull) {
                const int r = __builtin_ctzll(b);
                if (no < out_cap) {
                    c3_outlier_t o;
                    o.chunk = u;
                    o.replica = r;
                    o.majority_replica = v.majority;
                    const c3_chunk_record_t* s2[2] = {&rec[r * C + u], &rec[v.majority * C + u]};
                    for (int z = 0; z < 2; ++z) {
                        o.nan_count[z] = s2[z]->nan_count;
                        o.inf_count[z] = s2[z]->inf_count;
                        o.absmax[z] = s2[z]->absmax;
                        o.sum[z] = s2[z]->sum;
                        o.sumsq[z] = s2[z]->sumsq;
                    }
                    outliers[no] = o;
                }
                ++no;
            }
        }
        counts[0] = no;
        counts[1] = nu;
        counts[2] = na;
    }
}

bool small_tail_fits(int R, int64_t C) { return C >= 1 && C <= kTailThreads && R * C <= kTailMaxRecords; }

hipError_t launch_small_tail(const SigPlan* dplan, c3_chunk_record_t* records, uint8_t* status,
                             uint64_t* bitmap, int32_t* majority, c3_outlier_t* outliers,
                             int64_t out_cap, int64_t* undecided, int64_t und_cap, int64_t* counts,
                             hipStream_t stream) {
    hipLaunchKernelGGL(small_tail_kernel, dim3(1), dim3(kTailThreads), 0, stream, dplan, records,
                       status, bitmap, majority, outliers, out_cap, undecided, und_cap, counts);
    return hipGetLastError();
}

// Copies the staged plan from pinned host memory into the workspace on the
// compute queue (no copy engine, so no cross-engine synchronization).
__global__ void __launch_bounds__(256) plan_fetch_kernel(const u32x4* __restrict__ src,
                                                         u32x4* __restrict__ dst, int64_t n16) {
    for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n16; i += (int64_t)gridDim.x * 256)
        dst[i] = src[i];
}

hipError_t launch_plan_fetch(const void* host_src, void* dst, size_t bytes, hipStream_t stream) {
    const int64_t n16 = (int64_t)((bytes + 15) / 16);
    const int64_t blocks = (n16 + 255) / 256 < 64 ? (n16 + 255) / 256 : 64;
    if (n16 == 0) return hipSuccess;
    hipLaunchKernelGGL(plan_fetch_kernel, dim3((unsigned)blocks), dim3(256), 0, stream,
                       static_cast<const u32x4*>(host_src), static_cast<u32x4*>(dst), n16);
    return hipGetLastError();
}

template <int DT>
static hipError_t launch_group(const SigPlan* dplan, c3_chunk_record_t* records, int gk0, int gk1,
                               int64_t gtiles, int R, int grid_blocks, hipStream_t stream) {
    const int64_t ntiles = gtiles * R;
    if (ntiles <= 0) return hipSuccess;
    int64_t grid = grid_blocks > 0 ? grid_blocks : ntiles;
    if (grid > ntiles) grid = ntiles;
    if (grid > 0x7FFFFFFF) grid = 0x7FFFFFFF;
    hipLaunchKernelGGL((signature_kernel<DT, kUnroll>), dim3((unsigned)grid), dim3(kSigThreads), 0,
                       stream, dplan, records, gk0, gk1, gtiles);
    return hipGetLastError();
}

hipError_t launch_signature(const SigPlan* dplan, const SigPlan& hplan, const SigGroups& groups,
                            c3_chunk_record_t* records, int grid_blocks, bool finalize,
                            hipStream_t stream, hipEvent_t ev0, hipEvent_t ev1) {
    hipError_t e;
    if (ev0 && (e = hipEventRecord(ev0, stream)) != hipSuccess) return e;
    for (int d = 0; d < 4; ++d) {
        const int gk0 = groups.k0[d], gk1 = groups.k1[d];
        if (gk1 <= gk0) continue;
        const int64_t gt = groups.tiles[d];
        switch (d) {
            case C3_F32: e = launch_group<C3_F32>(dplan, records, gk0, gk1, gt, hplan.R, grid_blocks, stream); break;
            case C3_BF16: e = launch_group<C3_BF16>(dplan, records, gk0, gk1, gt, hplan.R, grid_blocks, stream); break;
            case C3_F16: e = launch_group<C3_F16>(dplan, records, gk0, gk1, gt, hplan.R, grid_blocks, stream); break;
            default: e = launch_group<C3_RAW>(dplan, records, gk0, gk1, gt, hplan.R, grid_blocks, stream); break;
        }
        if (e != hipSuccess) return e;
    }
    if (ev1 && (e = hipEventRecord(ev1, stream)) != hipSuccess) return e;
    if (!hplan.direct && finalize) {
        const int64_t total = hplan.C * hplan.R;
        const int64_t blocks = (total + 255) / 256 < 65536 ? (total + 255) / 256 : 65536;
        hipLaunchKernelGGL(finalize_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, dplan,
                           records);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

}  // namespace c3
