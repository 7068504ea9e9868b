// Plan and partial layouts of the streaming signature kernel, and its
// compile-time tuning knobs.  Shared by the host side (c3_api.cpp), which
// stages the plan, and the kernel (c3_signature.hip), which reads it.
#pragma once

#include <stdint.h>

#include "../../include/c3.h"

namespace c3 {

// ---------------------------------------------------------------------------
// Signature plan.  The host writes one SigPlan header followed by its arrays
// into the workspace; kernels read it through a device pointer.
// ---------------------------------------------------------------------------
struct SigPlan {
    int32_t R;
    int32_t T;
    int64_t C;                  // chunks per replica
    int64_t tiles_per_replica;  // tiles per replica
    uint64_t chunk_bytes;
    uint64_t tile_bytes;        // power-of-two multiple of 1024, divides chunk_bytes
    uint32_t tiles_per_chunk;
    uint32_t direct;            // 1: one tile per chunk, tiles write records
    // byte offsets (from the SigPlan base) of the arrays below
    uint64_t off_ptrs;          // u64  [R*T] replica-major tensor base addresses
    uint64_t off_tile_base;     // i64  [T+1] first tile of each tensor
    uint64_t off_chunk_base;    // i64  [T+1] first chunk of each tensor
    uint64_t off_tmeta;         // TensorInfo [T]
    uint64_t off_order;         // i32  [T] tensor ids grouped by dtype (stable)
    uint64_t off_gtile;         // i64  [T+1] tile prefix in that order
    uint64_t off_chunk_tensor;  // i32  [C] tensor of each chunk
    uint64_t off_partials;      // TilePartial [R * tiles_per_replica]
    uint64_t total_bytes;
};

struct TensorInfo {
    uint64_t nbytes;
    int32_t dtype;
    int32_t ndim;
    int64_t shape[C3_MAX_NDIM];
};

// Fold of one tile (or of a whole chunk when direct): 64 bytes.
struct TilePartial {
    uint64_t A, B;              // NH accumulators (wrapping)
    double s, sc;               // sum and its compensation
    double q, qc;               // sum of squares and its compensation
    uint32_t maxbits;           // magnitude bits of the largest finite element
    uint32_t nan_count, inf_count, pad;
};
static_assert(sizeof(TilePartial) == 64, "partial layout");
static_assert(sizeof(c3_chunk_record_t) == 64, "record layout");

// Tuning knobs of the streaming kernel (compile-time; results do not depend
// on them except for the last bits of the fp64 sums through the tile size).
#ifndef C3_SIG_TILE_MAX
#define C3_SIG_TILE_MAX (256 * 1024)
#endif
#ifndef C3_SIG_UNROLL
#define C3_SIG_UNROLL 16
#endif
#ifndef C3_SIG_WAVES_PER_EU
#define C3_SIG_WAVES_PER_EU 4
#endif
constexpr uint64_t kDefaultTileMax = C3_SIG_TILE_MAX;
constexpr int kSigThreads = 256;
constexpr int kUnroll = C3_SIG_UNROLL;

// Tile map of large launches.  The hardware hands workgroup b to XCD
// b mod 8, and on MI355X XCDs 1, 3, 5 and 7 read about 6% slower than the
// others (the read probe over 4 GiB: 874-930 against 939-981 GB/s each, for
// any pairing of tiles with XCDs), so one tile per workgroup in order lets
// the odd XCDs set the end of the launch.  With the map, tiles go in rounds
// of kXcdRound: within a round an even XCD takes kXcdEven consecutive tiles
// and an odd one kXcdOdd, in XCD order, and every XCD has the same number of
// workgroups, the odd ones' spare workgroups at the end taking no tile.  A
// round of 256 KiB tiles is 64 MiB, and all XCDs stream the same round at
// once.  The read probe over 4 GiB of 256 KiB tiles: 7.16-7.17 TB/s against
// 7.06-7.08 in order (33/31 tiles); 16 or 32 tiles each without a skew
// 7.09-7.12; 64 each 6.68.  The signature kernel gains 1.4-1.6% on the 1B
// bf16 parameters and the 2B fp32 Adam shard (256 KiB tiles) and loses
// 1.2-2.5% on the Llama-layer gradients (128 KiB tiles, where the probe
// still gains), so only launches of tiles of 256 KiB or more use it.
constexpr unsigned kXcdEven = 33, kXcdOdd = 31;
constexpr unsigned kXcdRound = 4 * (kXcdEven + kXcdOdd);
constexpr int64_t kXcdMapMinTiles = 8 * kXcdRound;     // smaller launches keep the order
constexpr uint64_t kXcdMapMinTileBytes = 256 * 1024;

// Workgroups of a mapped launch of n tiles.
inline int64_t xcd_map_grid(int64_t n) { return 8 * ((n + kXcdRound - 1) / kXcdRound) * kXcdEven; }

// Whether a launch of n tiles of tile_bytes with the default grid is mapped.
inline bool xcd_map_applies(int64_t n, uint64_t tile_bytes) {
    return n >= kXcdMapMinTiles && tile_bytes >= kXcdMapMinTileBytes && xcd_map_grid(n) <= 0x7FFFFFFF;
}

// Tile of workgroup b in a mapped launch of n tiles (n when it takes none).
// The last, partial round of m tiles is split in the same proportions: XCD x
// takes [m off_x / R, m (off_x + cnt_x) / R) of it, R the round size.
__device__ __forceinline__ int64_t xcd_map_tile(unsigned b, int64_t n) {
    const unsigned x = b % 8u, k = b / 8u;
    const unsigned cnt = (x & 1u) ? kXcdOdd : kXcdEven;
    const unsigned off = (x / 2u) * (kXcdEven + kXcdOdd) + ((x & 1u) ? kXcdEven : 0u);
    const int64_t full = n / kXcdRound;
    const int64_t round = k / cnt;
    if (round < full) return round * kXcdRound + off + k % cnt;
    const int64_t m = n - full * kXcdRound;
    const int64_t lo = m * off / kXcdRound, hi = m * (off + cnt) / kXcdRound;
    const int64_t j = (int64_t)k - full * cnt;
    return j < hi - lo ? full * kXcdRound + lo + j : n;
}

// Position range [k0, k1) of each dtype in the grouped tensor order and the
// tiles per replica of that group.
struct SigGroups {
    int k0[4], k1[4];
    int64_t tiles[4];
};

}  // namespace c3
