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

// Position range [k0, k1) of each dtype in the grouped tensor order and the
// tiles per replica of that group.
struct SigGroups {
    int k0[4], k1[4];
    int64_t tiles[4];
};

}  // namespace c3
