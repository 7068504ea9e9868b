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
// which workgroup runs it, so results are independent of the grid size and
// of the tile order: large launches take their tiles through the XCD map
// (xcd_map_tile), the others in order.
//
// Non-finite screen: a lane sums its elements in fp64 without looking at
// them.  A non-finite element is the only way its sum or sum of squares can
// become non-finite (finite fp32/bf16/fp16 values cannot overflow fp64 here),
// so a lane whose sums end non-finite re-reads its own segments and
// classifies every element.  Healthy data never takes that path.
#include "c3_device.h"
#include "c3_internal.h"
#include "c3_localize_block.h"
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
    // the tensor's description in one batch of loads, so that the chain over
    // the dimensions runs on registers instead of waiting for each in turn
    const TensorInfo ti = *tip;
    const int dtype = ti.dtype, ndim = ti.ndim;
    uint64_t h = fmix64(kTag ^ ((uint64_t)(uint32_t)dtype << 32) ^ (uint64_t)(uint32_t)ndim);
#pragma unroll
    for (int d = 0; d < C3_MAX_NDIM; ++d)
        if (d < ndim) h = fmix64(h ^ (uint64_t)ti.shape[d]);
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
                     int gk0, int gk1, int64_t gtiles, int mapped) {
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

    // a mapped launch: one tile per workgroup, from the XCD map; otherwise
    // tiles blockIdx.x, blockIdx.x + gridDim.x, ...
    for (int64_t i = mapped ? xcd_map_tile(blockIdx.x, ntiles) : (int64_t)blockIdx.x; i < ntiles;
         i += mapped ? ntiles : (int64_t)gridDim.x) {
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
    const int t = reinterpret_cast<const int32_t*>(pb + plan->off_chunk_tensor)[c];
    const uint64_t k = (uint64_t)(c - chunk_base[t]);
    const uint64_t nbytes = tinfo[t].nbytes;
    const int64_t tiles_t = tile_base[t + 1] - tile_base[t];
    const int64_t lt0 = (int64_t)k * plan->tiles_per_chunk;
    const int64_t nt = min((int64_t)plan->tiles_per_chunk, tiles_t - lt0);
    const TilePartial* pp = partials + r * plan->tiles_per_replica + tile_base[t] + lt0;
    TilePartial p = pp[0];
    // in tile order, four partials loaded at a time before they are added
    for (int64_t x0 = 1; x0 < nt; x0 += 4) {
        TilePartial q[4];
#pragma unroll
        for (int j = 0; j < 4; ++j)
            if (x0 + j < nt) q[j] = pp[x0 + j];
#pragma unroll
        for (int j = 0; j < 4; ++j)
            if (x0 + j < nt) partial_add(p, q[j]);
    }
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
// optimizer-boundary check signs 7 chunks per replica; c3_check takes it for
// plans of up to kTailThreads chunks and kTailMaxRecords records): three
// launches of a few microseconds each become one.  (1) Every record --
// combined from its tile partials, or as the streaming kernel wrote it when
// chunks are whole tiles -- is written out and kept in LDS.  (2) One thread
// per chunk votes with exact_vote_row, the rule c3_consensus applies, on the
// signatures.  (3) The lists of c3_localize: a scan over the chunks of their
// outlier and undecided counts gives each chunk's thread the place of its
// entries (chunk ascending, replica ascending within a chunk, both
// replicas' summaries), and thread 0 writes the counts.
// ---------------------------------------------------------------------------
constexpr int kTailThreads = 256;
constexpr int kTailMaxRecords = 1024;

// Inclusive prefix sum over the 64 lanes of a wave.
__device__ inline uint64_t wave_inclusive_scan(uint64_t x, int lane) {
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
        const uint64_t y = shfl_u64(x, lane >= d ? lane - d : lane);
        if (lane >= d) x += y;
    }
    return x;
}

__device__ inline void outlier_from(c3_outlier_t& o, int64_t u, int r, int mj,
                                    const c3_chunk_record_t& a, const c3_chunk_record_t& b) {
    o.chunk = u;
    o.replica = r;
    o.majority_replica = mj;
    o.nan_count[0] = a.nan_count;
    o.nan_count[1] = b.nan_count;
    o.inf_count[0] = a.inf_count;
    o.inf_count[1] = b.inf_count;
    o.absmax[0] = a.absmax;
    o.absmax[1] = b.absmax;
    o.sum[0] = a.sum;
    o.sum[1] = b.sum;
    o.sumsq[0] = a.sumsq;
    o.sumsq[1] = b.sumsq;
}

__global__ void __launch_bounds__(kTailThreads) small_tail_kernel(
    const SigPlan* __restrict__ plan, c3_chunk_record_t* __restrict__ records,
    uint8_t* __restrict__ status, uint64_t* __restrict__ bitmap, int32_t* __restrict__ majority,
    c3_outlier_t* __restrict__ outliers, int64_t out_cap, int64_t* __restrict__ undecided,
    int64_t und_cap, int64_t* __restrict__ counts) {
    __shared__ c3_chunk_record_t rec[kTailMaxRecords];
    __shared__ uint64_t wave_total[kTailThreads / 64];
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
    const int u = threadIdx.x;
    UnitVote v{0ull, -1, (uint8_t)C3_AGREE};
    if (u < C) {
        if (R <= 16) {
            uint64_t e[16];
#pragma unroll
            for (int r = 0; r < 16; ++r) e[r] = r < R ? rec[r * C + u].sig : 0ull;
            v = exact_vote_row<16>(e, R);
        } else if (R <= 32) {
            uint64_t e[32];
#pragma unroll
            for (int r = 0; r < 32; ++r) e[r] = r < R ? rec[r * C + u].sig : 0ull;
            v = exact_vote_row<32>(e, R);
        } else {
            uint64_t e[C3_MAX_REPLICAS];
            for (int r = 0; r < C3_MAX_REPLICAS; ++r) e[r] = r < R ? rec[r * C + u].sig : 0ull;
            v = exact_vote_row<C3_MAX_REPLICAS>(e, R);
        }
        status[u] = v.status;
        bitmap[u] = v.bitmap;
        majority[u] = v.majority;
    }
    // counts packed as outliers (24 bits: at most 256 chunks x 63), undecided
    // and attributed chunks (20 bits each)
    const bool und = u < C && v.status == C3_INCONCLUSIVE;
    const uint64_t n_o = u < C && !und ? (uint64_t)__builtin_popcountll(v.bitmap) : 0ull;
    const uint64_t packed = n_o | ((uint64_t)und << 24) | ((uint64_t)(n_o != 0ull) << 44);
    const int lane = u & 63, wave = u >> 6;
    const uint64_t incl = wave_inclusive_scan(packed, lane);
    if (lane == 63) wave_total[wave] = incl;
    __syncthreads();
    uint64_t before = 0ull, total = 0ull;
#pragma unroll
    for (int w = 0; w < kTailThreads / 64; ++w) {
        const uint64_t t = wave_total[w];
        before += w < wave ? t : 0ull;
        total += t;
    }
    const uint64_t excl = before + incl - packed;
    int64_t po = (int64_t)(excl & 0xFFFFFFull);
    const int64_t pu = (int64_t)((excl >> 24) & 0xFFFFFull);
    for (uint64_t b = n_o ? v.bitmap : 0ull; b != 0ull && po < out_cap; b &= b - 1ull, ++po) {
        const int r = __builtin_ctzll(b);
        c3_outlier_t o;
        outlier_from(o, u, r, v.majority, rec[r * C + u], rec[v.majority * C + u]);
        outliers[po] = o;
    }
    if (und && pu < und_cap) undecided[pu] = u;
    if (u == 0) {
        counts[0] = (int64_t)(total & 0xFFFFFFull);
        counts[1] = (int64_t)((total >> 24) & 0xFFFFFull);
        counts[2] = (int64_t)((total >> 44) & 0xFFFFFull);
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

// ---------------------------------------------------------------------------
// Tail of c3_check: the records of every (replica, chunk) from their tile
// partials (finalize_kernel's combine) or as the streaming kernel wrote
// them, the exact vote of every chunk (exact_vote_row, the rule of
// c3_consensus) and the lists of c3_localize, in two launches.
// check_vote_kernel:
//   - a workgroup of kCheckThreads threads takes CPB = kCheckThreads / N
//     consecutive chunks (a segment), one thread per (chunk, replica slot),
//     so the R records of a chunk are combined in parallel and meet in LDS;
//   - one thread per chunk votes;
//   - with a staging area, the first wave scans the segment's outlier and
//     undecided counts (CPB <= 64 units: one wave) and writes the segment's
//     entries, summaries taken from the records in LDS, into the segment's
//     slots of the staging area, with the three counts.
// check_lists_kernel (one workgroup): scans the segments' counts in segment
// order and copies every staged entry to its place in the caller's lists.
// Segments are in chunk order and entries in (chunk, replica) order inside
// a segment, so the lists come out in c3_localize's order.
// ---------------------------------------------------------------------------
constexpr int kCheckThreads = 256;
constexpr int kCheckMaxListUnits = 8192;   // chunks whose lists go through the staging area
constexpr int kCheckMaxSegments = kCheckMaxListUnits / (kCheckThreads / 32);
// per step of 64 segments: outliers < 64 * CPB * N / 2 = 64 * kCheckThreads / 2,
// units <= 64 * 64
static_assert(64ll * kCheckThreads / 2 < (1ll << 24) && 64 * 64 < (1 << 20), "packed counts");

struct CheckStage {
    int32_t* seg_counts;      // [n_seg][4]: outliers, undecided, attributed units
    c3_outlier_t* out;        // [n_seg][out_per_seg]
    int64_t* und;             // [n_seg][CPB]
    int32_t out_per_seg;
    int32_t cpb;
};

template <int N>
__global__ void __launch_bounds__(kCheckThreads) check_vote_kernel(
    const SigPlan* __restrict__ plan, c3_chunk_record_t* __restrict__ records,
    uint8_t* __restrict__ status, uint64_t* __restrict__ bitmap, int32_t* __restrict__ majority,
    CheckStage stage) {
    constexpr int CPB = kCheckThreads / N;
    static_assert(CPB <= 64, "a segment's units must fit one wave");
    __shared__ c3_chunk_record_t rec[CPB][N];
    __shared__ UnitVote votes[CPB];
    const int R = plan->R;
    const int64_t C = plan->C;
    const int slot = threadIdx.x % N;
    const int cu = threadIdx.x / N;
    const int64_t c = (int64_t)blockIdx.x * CPB + cu;
    if (slot < R && c < C) {
        c3_chunk_record_t* dst = &records[(int64_t)slot * C + c];
        if (plan->direct) {
            rec[cu][slot] = *dst;
        } else {
            c3_chunk_record_t r;
            combine_chunk(plan, slot, c, &r);
            *dst = r;
            rec[cu][slot] = r;
        }
    }
    __syncthreads();
    if ((int)threadIdx.x < CPB) {
        const int64_t u = (int64_t)blockIdx.x * CPB + threadIdx.x;
        if (u < C) {
            uint64_t e[N];
#pragma unroll
            for (int r = 0; r < N; ++r) e[r] = r < R ? rec[threadIdx.x][r].sig : 0ull;
            const UnitVote v = exact_vote_row<N>(e, R);
            status[u] = v.status;
            bitmap[u] = v.bitmap;
            majority[u] = v.majority;
            votes[threadIdx.x] = v;
        }
    }
    if (stage.seg_counts == nullptr) return;
    __syncthreads();
    if (threadIdx.x < 64) {
        // this segment's entries, in (chunk, replica) order, into its slots
        const int lane = threadIdx.x;
        const int64_t u = (int64_t)blockIdx.x * CPB + lane;
        const bool valid = lane < CPB && u < C;
        UnitVote v{0ull, -1, (uint8_t)C3_AGREE};
        if (valid) v = votes[lane];
        const uint64_t n_o =
            valid && v.status != C3_INCONCLUSIVE ? (uint64_t)__builtin_popcountll(v.bitmap) : 0ull;
        const uint64_t n_u = valid && v.status == C3_INCONCLUSIVE ? 1ull : 0ull;
        const uint64_t packed = n_o | (n_u << 32);
        const uint64_t incl = wave_inclusive_scan(packed, lane);
        uint64_t po = (uint32_t)(incl - packed);
        const uint64_t pu = (incl - packed) >> 32;
        c3_outlier_t* so = stage.out + (int64_t)blockIdx.x * stage.out_per_seg;
        for (uint64_t b = n_o ? v.bitmap : 0ull; b != 0ull; b &= b - 1ull) {
            const int r = __builtin_ctzll(b);
            c3_outlier_t o;
            outlier_from(o, u, r, v.majority, rec[lane][r], rec[lane][v.majority]);
            so[po++] = o;
        }
        if (n_u) stage.und[(int64_t)blockIdx.x * CPB + (int64_t)pu] = u;
        const uint64_t tot = shfl_u64(incl, 63);
        const uint64_t n_att = (uint64_t)__builtin_popcountll(ballot64(n_o != 0ull));
        if (lane == 0) {
            int32_t* sc = stage.seg_counts + 4 * (int64_t)blockIdx.x;
            sc[0] = (int32_t)(uint32_t)tot;
            sc[1] = (int32_t)(tot >> 32);
            sc[2] = (int32_t)n_att;
        }
    }
}

__global__ void __launch_bounds__(kCheckThreads) check_lists_kernel(
    CheckStage stage, int n_seg, c3_outlier_t* __restrict__ outliers, int64_t out_cap,
    int64_t* __restrict__ undecided, int64_t und_cap, int64_t* __restrict__ counts) {
    __shared__ int64_t seg_off[2][kCheckMaxSegments];
    __shared__ int32_t seg_n[2][kCheckMaxSegments];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    if (wave == 0) {
        // segment offsets in segment order: one wave, 64 segments per step,
        // the three counts packed into one word (outliers 24 bits, undecided
        // and attributed 20 bits each: a step of 64 segments holds fewer
        // than 64 * kCheckThreads / 2 outliers and at most 64 * 64 units)
        int64_t carry_o = 0, carry_u = 0, carry_a = 0;
        for (int base = 0; base < n_seg; base += 64) {
            const int sgi = base + lane;
            uint64_t o = 0, un = 0, at = 0;
            if (sgi < n_seg) {
                const int32_t* sc = stage.seg_counts + 4 * (int64_t)sgi;
                o = (uint32_t)sc[0];
                un = (uint32_t)sc[1];
                at = (uint32_t)sc[2];
            }
            const uint64_t packed = o | (un << 24) | (at << 44);
            const uint64_t incl = wave_inclusive_scan(packed, lane);
            const uint64_t excl = incl - packed;
            if (sgi < n_seg) {
                seg_off[0][sgi] = carry_o + (int64_t)(excl & 0xFFFFFFull);
                seg_off[1][sgi] = carry_u + (int64_t)((excl >> 24) & 0xFFFFFull);
                seg_n[0][sgi] = (int32_t)o;
                seg_n[1][sgi] = (int32_t)un;
            }
            const uint64_t tot = shfl_u64(incl, 63);
            carry_o += (int64_t)(tot & 0xFFFFFFull);
            carry_u += (int64_t)((tot >> 24) & 0xFFFFFull);
            carry_a += (int64_t)((tot >> 44) & 0xFFFFFull);
        }
        if (lane == 0) {
            counts[0] = carry_o;
            counts[1] = carry_u;
            counts[2] = carry_a;
        }
    }
    __syncthreads();
    for (int sgi = wave; sgi < n_seg; sgi += kCheckThreads / 64) {
        const c3_outlier_t* so = stage.out + (int64_t)sgi * stage.out_per_seg;
        for (int j = lane; j < seg_n[0][sgi]; j += 64) {
            const int64_t d = seg_off[0][sgi] + j;
            if (d < out_cap) outliers[d] = so[j];
        }
        for (int j = lane; j < seg_n[1][sgi]; j += 64) {
            const int64_t d = seg_off[1][sgi] + j;
            if (d < und_cap) undecided[d] = stage.und[(int64_t)sgi * stage.cpb + j];
        }
    }
}

int check_group_bound(int R) { return R <= 4 ? 4 : R <= 8 ? 8 : R <= 16 ? 16 : R <= 32 ? 32 : 0; }

// Staging bytes for the fused lists of C chunks at group bound N (0 when
// the tail leaves the lists to a separate localization).
static uint64_t check_stage_parts(int N, int64_t C, uint64_t& cnt_b, uint64_t& out_b,
                                  uint64_t& und_b, int& out_per_seg) {
    const int64_t cpb = kCheckThreads / N;
    const int64_t n_seg = (C + cpb - 1) / cpb;
    // a strict majority holds more than R / 2 replicas, so a chunk has at
    // most ceil(R / 2) - 1 < N / 2 outliers
    out_per_seg = (int)(cpb * (N / 2));
    cnt_b = (uint64_t)n_seg * 16;
    out_b = (uint64_t)n_seg * out_per_seg * sizeof(c3_outlier_t);
    und_b = (uint64_t)n_seg * cpb * 8;
    return ((cnt_b + 255) / 256 + (out_b + 255) / 256 + (und_b + 255) / 256) * 256;
}

uint64_t check_stage_bytes(int R, int64_t C) {
    const int N = check_group_bound(R);
    if (N == 0 || C > kCheckMaxListUnits) return 0;
    uint64_t a, b, c;
    int o;
    return check_stage_parts(N, C, a, b, c, o);
}

hipError_t launch_check_tail(const SigPlan* dplan, const SigPlan& hplan, c3_chunk_record_t* records,
                             uint8_t* status, uint64_t* bitmap, int32_t* majority,
                             c3_outlier_t* outliers, int64_t out_cap, int64_t* undecided,
                             int64_t und_cap, int64_t* counts, void* stage_ws,
                             hipStream_t stream) {
    const int N = check_group_bound(hplan.R);
    if (N == 0 || hplan.C <= 0) return hipErrorInvalidValue;
    const int64_t cpb = kCheckThreads / N;
    const int64_t blocks = (hplan.C + cpb - 1) / cpb;
    if (blocks > 0x7FFFFFFF) return hipErrorInvalidValue;
    CheckStage st{nullptr, nullptr, nullptr, 0, (int32_t)cpb};
    if (stage_ws != nullptr) {
        if (hplan.C > kCheckMaxListUnits) return hipErrorInvalidValue;
        uint64_t cnt_b, out_b, und_b;
        check_stage_parts(N, hplan.C, cnt_b, out_b, und_b, st.out_per_seg);
        unsigned char* w = static_cast<unsigned char*>(stage_ws);
        st.seg_counts = reinterpret_cast<int32_t*>(w);
        w += (cnt_b + 255) / 256 * 256;
        st.out = reinterpret_cast<c3_outlier_t*>(w);
        w += (out_b + 255) / 256 * 256;
        st.und = reinterpret_cast<int64_t*>(w);
    }
    switch (N) {
        case 4:
            hipLaunchKernelGGL(check_vote_kernel<4>, dim3((unsigned)blocks), dim3(kCheckThreads), 0,
                               stream, dplan, records, status, bitmap, majority, st);
            break;
        case 8:
            hipLaunchKernelGGL(check_vote_kernel<8>, dim3((unsigned)blocks), dim3(kCheckThreads), 0,
                               stream, dplan, records, status, bitmap, majority, st);
            break;
        case 16:
            hipLaunchKernelGGL(check_vote_kernel<16>, dim3((unsigned)blocks), dim3(kCheckThreads), 0,
                               stream, dplan, records, status, bitmap, majority, st);
            break;
        default:
            hipLaunchKernelGGL(check_vote_kernel<32>, dim3((unsigned)blocks), dim3(kCheckThreads), 0,
                               stream, dplan, records, status, bitmap, majority, st);
            break;
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || stage_ws == nullptr) return e;
    hipLaunchKernelGGL(check_lists_kernel, dim3(1), dim3(kCheckThreads), 0, stream, st,
                       (int)blocks, outliers, out_cap, undecided, und_cap, counts);
    return hipGetLastError();
}

// Copies the staged plan from pinned host memory into the workspace on the
// compute queue (no copy engine, so no cross-engine synchronization): up to
// kFetchBlocks workgroups, four 16-byte loads per thread in flight, so a plan
// of up to 128 KiB is one round trip over the host link.  With `seen`, thread
// 0 of workgroup b then stores `seq` into seen[b] (system scope, pinned
// coherent host memory): every load of that workgroup has completed, since
// each thread stored what it loaded before the barrier, so the host may
// reuse the slot once every used word reads `seq`.
constexpr int kFetchThreads = 256;
constexpr int kFetchLoads = 4;

__global__ void __launch_bounds__(kFetchThreads) plan_fetch_kernel(const u32x4* __restrict__ src,
                                                                   u32x4* __restrict__ dst,
                                                                   int64_t n16, uint64_t* seen,
                                                                   uint64_t seq) {
    const int64_t stride = (int64_t)gridDim.x * kFetchThreads;
    for (int64_t i0 = (int64_t)blockIdx.x * kFetchThreads + threadIdx.x; i0 < n16;
         i0 += stride * kFetchLoads) {
        u32x4 v[kFetchLoads];
#pragma unroll
        for (int k = 0; k < kFetchLoads; ++k) {
            const int64_t i = i0 + (int64_t)k * stride;
            if (i < n16) v[k] = src[i];
        }
#pragma unroll
        for (int k = 0; k < kFetchLoads; ++k) {
            const int64_t i = i0 + (int64_t)k * stride;
            if (i < n16) dst[i] = v[k];
        }
    }
    __syncthreads();
    if (threadIdx.x == 0 && seen != nullptr)
        __hip_atomic_store(seen + blockIdx.x, seq, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_SYSTEM);
}

int plan_fetch_blocks(size_t bytes) {
    const int64_t n16 = (int64_t)((bytes + 15) / 16);
    const int64_t per = (int64_t)kFetchThreads * kFetchLoads;
    const int64_t b = (n16 + per - 1) / per;
    return b < 1 ? 1 : b > kFetchBlocks ? kFetchBlocks : (int)b;
}

hipError_t launch_plan_fetch(const void* host_src, void* dst, size_t bytes, hipStream_t stream,
                             uint64_t* seen, uint64_t seq) {
    const int64_t n16 = (int64_t)((bytes + 15) / 16);
    if (n16 == 0 && seen == nullptr) return hipSuccess;
    hipLaunchKernelGGL(plan_fetch_kernel, dim3((unsigned)plan_fetch_blocks(bytes)),
                       dim3(kFetchThreads), 0, stream, static_cast<const u32x4*>(host_src),
                       static_cast<u32x4*>(dst), n16, seen, seq);
    return hipGetLastError();
}

template <int DT>
static hipError_t launch_group(const SigPlan* dplan, c3_chunk_record_t* records, int gk0, int gk1,
                               int64_t gtiles, int R, uint64_t tile_bytes, int grid_blocks,
                               hipStream_t stream) {
    const int64_t ntiles = gtiles * R;
    if (ntiles <= 0) return hipSuccess;
    int64_t grid = grid_blocks > 0 ? grid_blocks : ntiles;
    if (grid > ntiles) grid = ntiles;
    const int mapped = grid_blocks <= 0 && xcd_map_applies(ntiles, tile_bytes);
    if (mapped) grid = xcd_map_grid(ntiles);
    if (grid > 0x7FFFFFFF) grid = 0x7FFFFFFF;
    hipLaunchKernelGGL((signature_kernel<DT, kUnroll>), dim3((unsigned)grid), dim3(kSigThreads), 0,
                       stream, dplan, records, gk0, gk1, gtiles, mapped);
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
            case C3_F32: e = launch_group<C3_F32>(dplan, records, gk0, gk1, gt, hplan.R, hplan.tile_bytes, grid_blocks, stream); break;
            case C3_BF16: e = launch_group<C3_BF16>(dplan, records, gk0, gk1, gt, hplan.R, hplan.tile_bytes, grid_blocks, stream); break;
            case C3_F16: e = launch_group<C3_F16>(dplan, records, gk0, gk1, gt, hplan.R, hplan.tile_bytes, grid_blocks, stream); break;
            default: e = launch_group<C3_RAW>(dplan, records, gk0, gk1, gt, hplan.R, hplan.tile_bytes, grid_blocks, stream); break;
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
