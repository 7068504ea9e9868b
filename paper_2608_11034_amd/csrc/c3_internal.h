// Internal declarations of the C3 HIP library (gfx950).  Host entry points
// live in c3_api.cpp; kernels and their launchers live in the .hip files.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/c3.h"
#include "c3_sigplan.h"

namespace c3 {

// Compute units of the device `stream` runs on (cached per device; 0 if the
// runtime cannot tell).
int stream_cu_count(hipStream_t stream);

static_assert(sizeof(c3_outlier_t) == 80, "outlier layout");
static_assert(sizeof(c3_rank_verdict_t) == 24, "verdict layout");

// finalize: combine tile partials into records when a chunk spans several
// tiles (false leaves that to launch_small_tail).
hipError_t launch_signature(const SigPlan* dplan, const SigPlan& hplan, const SigGroups& groups,
                            c3_chunk_record_t* records, int grid_blocks, bool finalize,
                            hipStream_t stream, hipEvent_t ev0, hipEvent_t ev1);

// Records (from partials unless chunks are whole tiles), exact votes and
// lists of a small plan in one workgroup: at most 256 chunks and 1,024
// records, R <= 64 (small_tail_fits checks the sizes).
bool small_tail_fits(int R, int64_t C);
hipError_t launch_small_tail(const SigPlan* dplan, c3_chunk_record_t* records, uint8_t* status,
                             uint64_t* bitmap, int32_t* majority, c3_outlier_t* outliers,
                             int64_t out_cap, int64_t* undecided, int64_t und_cap, int64_t* counts,
                             hipStream_t stream);

// Tail of c3_check for R <= 32 (check_group_bound(R) != 0): records from
// partials and exact votes in one kernel; with stage_ws (check_stage_bytes(R,
// C) bytes, 256-byte aligned; C up to 8,192) also the lists of c3_localize,
// staged per segment by that kernel and placed by a one-workgroup kernel.
int check_group_bound(int R);
uint64_t check_stage_bytes(int R, int64_t C);
hipError_t launch_check_tail(const SigPlan* dplan, const SigPlan& hplan, c3_chunk_record_t* records,
                             uint8_t* status, uint64_t* bitmap, int32_t* majority,
                             c3_outlier_t* outliers, int64_t out_cap, int64_t* undecided,
                             int64_t und_cap, int64_t* counts, void* stage_ws,
                             hipStream_t stream);

// Copies `bytes` (rounded up to 16) from pinned, device-visible host memory
// to device memory with a kernel of plan_fetch_blocks(bytes) workgroups on
// `stream`; with `seen` (pinned coherent host memory, kFetchBlocks words)
// workgroup b then stores `seq` into seen[b], which tells the host that its
// part of the source may be reused.
constexpr int kFetchBlocks = 32;
int plan_fetch_blocks(size_t bytes);
hipError_t launch_plan_fetch(const void* host_src, void* dst, size_t bytes, hipStream_t stream,
                             uint64_t* seen = nullptr, uint64_t seq = 0);

hipError_t launch_tensor_signature(const c3_chunk_record_t* records, int R, int64_t C, int T,
                                   uint64_t* out, hipStream_t stream);

// Optimizer-boundary replay: per-replica tensor bases and fp32 factors.
struct AdamwPtrs {
    const float* param[C3_MAX_REPLICAS];
    const float* grad[C3_MAX_REPLICAS];
    const float* exp_avg[C3_MAX_REPLICAS];
    const float* exp_avg_sq[C3_MAX_REPLICAS];
};
struct AdamwConst {
    float decay, w, one_minus_w, beta2, c2, s2, eps, neg_step;
    int lerp_small;
};
// With plan_src set, the same launch also copies plan_bytes (rounded up to
// 16) from plan_src (pinned host memory) to plan_dst.
hipError_t launch_adamw_slice(const AdamwPtrs& ptrs, const AdamwConst& c, int R, bool vec4,
                              int64_t offset, int64_t n, float* out, int64_t stride,
                              hipStream_t stream, const void* plan_src = nullptr,
                              void* plan_dst = nullptr, size_t plan_bytes = 0);

// Fused timing consensus (R <= 16, window <= 64): vote both evidence kinds
// per (iteration, group), collect per-rank outlier bits, confirm per rank.
// Without per-unit results and at a shape that fills the device this is one
// kernel with the bits in LDS; otherwise three launches with the bits in
// the workspace (timing_masks_bytes).
int64_t timing_masks_bytes(int R, int64_t G, int64_t T);
hipError_t launch_timing_consensus(const uint64_t* fp, const void* times, int time_kind, int R,
                                   int64_t G, int64_t T, double kappa, int window,
                                   uint8_t* fp_status, uint64_t* fp_bitmap, int32_t* fp_majority,
                                   uint8_t* t_status, uint64_t* t_bitmap, int32_t* t_majority,
                                   c3_rank_verdict_t* verdicts, void* ws, hipStream_t stream);

hipError_t launch_consensus(const void* evidence, int kind, int64_t rstride, int64_t ustride, int R,
                            int64_t n_units, int mode, double kappa, uint8_t* status,
                            uint64_t* bitmap, int32_t* majority_idx, hipStream_t stream);

// Argument checks shared by c3_localize and c3_localize_noalloc (everything
// but the workspace); C3_OK or an error code.
int localize_check(const uint8_t* status, const uint64_t* bitmap, const int32_t* majority_idx,
                   const c3_chunk_record_t* records, int R, int64_t n_units,
                   const c3_outlier_t* outliers, int64_t out_cap, const int64_t* undecided,
                   int64_t und_cap, const int64_t* counts);

size_t localize_ws_bytes(int64_t n_units);
hipError_t launch_localize(const uint8_t* status, const uint64_t* bitmap,
                           const int32_t* majority_idx, const c3_chunk_record_t* records, int R,
                           int64_t n_units, c3_outlier_t* outliers, int64_t out_cap,
                           int64_t* undecided, int64_t und_cap, int64_t* counts, void* ws,
                           hipStream_t stream);

// Read-only probe over `bytes` (a multiple of 1024) in tiles of tile_bytes;
// writes the xor of each tile's 64-bit words to checksum[tile].
hipError_t launch_read_probe(const void* buf, uint64_t bytes, uint64_t tile_bytes,
                             uint64_t* checksum, hipStream_t stream);

size_t confirm_ws_bytes(int R, int64_t G, int64_t T);
hipError_t launch_confirm(const uint64_t* fp_bitmap, const uint64_t* time_bitmap, int R, int64_t G,
                          int64_t T, int window, c3_rank_verdict_t* verdicts, void* ws,
                          hipStream_t stream);

}  // namespace c3
