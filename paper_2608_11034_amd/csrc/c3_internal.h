// Internal declarations of the C3 HIP library (gfx950).  Host entry points
// live in c3_api.cpp; kernels and their launchers live in the .hip files.
#pragma once

#include <hip/hip_runtime.h>
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
static_assert(sizeof(c3_outlier_t) == 80, "outlier layout");
static_assert(sizeof(c3_rank_verdict_t) == 24, "verdict layout");

// Tuning knobs of the streaming kernel (compile-time; results do not depend
// on them except for the last bits of the fp64 sums through the tile size).
#ifndef C3_SIG_TILE_MAX
#define C3_SIG_TILE_MAX (1024 * 1024)
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

hipError_t launch_signature(const SigPlan* dplan, const SigPlan& hplan, const SigGroups& groups,
                            c3_chunk_record_t* records, int grid_blocks, hipStream_t stream,
                            hipEvent_t ev0, hipEvent_t ev1);

// Copies `bytes` (rounded up to 16) from pinned, device-visible host memory
// to device memory with a kernel on `stream`.
hipError_t launch_plan_fetch(const void* host_src, void* dst, size_t bytes, hipStream_t stream);

hipError_t launch_tensor_signature(const c3_chunk_record_t* records, int R, int64_t C, int T,
                                   uint64_t* out, hipStream_t stream);

hipError_t launch_consensus(const void* evidence, int kind, int64_t rstride, int64_t ustride, int R,
                            int64_t n_units, int mode, double kappa, uint8_t* status,
                            uint64_t* bitmap, int32_t* majority_idx, hipStream_t stream);

size_t localize_ws_bytes(int64_t n_units);
hipError_t launch_localize(const uint8_t* status, const uint64_t* bitmap,
                           const int32_t* majority_idx, const c3_chunk_record_t* records, int R,
                           int64_t n_units, c3_outlier_t* outliers, int64_t out_cap,
                           int64_t* undecided, int64_t und_cap, int64_t* counts, void* ws,
                           hipStream_t stream);

size_t confirm_ws_bytes(int R, int64_t G, int64_t T);
hipError_t launch_confirm(const uint64_t* fp_bitmap, const uint64_t* time_bitmap, int R, int64_t G,
                          int64_t T, int window, c3_rank_verdict_t* verdicts, void* ws,
                          hipStream_t stream);

}  // namespace c3
