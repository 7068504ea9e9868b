/*
 * c3.h -- C ABI of the MI355X (gfx950) hot path of Consensus Collective
 * Communication (C3): per-chunk signatures and numerical summaries of R
 * replica copies resident in one GPU's HBM, strict-majority or robust
 * statistical consensus across the replicas, and a (replica, chunk) outlier
 * list.
 *
 * Paper: "SCOUT: Symmetric Consensus Outlier Detection for Failure
 * Localization in LLM Pre-Training" (arXiv 2608.11034).  C3 maps one
 * diagnostic object per peer of an ordered peer group G = (r_0 .. r_{N-1})
 * to a result R = (s, B, E): a status, an N-bit outlier bitmap and the
 * gathered evidence (Sec. 5.1, Algorithm 1).  Here the N peers are R replica
 * copies on one GPU, peer i is replica i (the caller keeps the mapping from
 * replica index to global rank), the evidence E is the chunk-record table,
 * and s and B are produced per chunk.
 *
 * Common conventions
 *   - Device pointers are plain HIP device addresses owned by the caller.
 *     The library allocates no device memory.  Its state between calls is
 *     a 4 MiB ring of pinned host memory per device (allocated on first
 *     use, kept until the process ends) through which c3_signature and
 *     c3_check stage their plans, so that staging never makes the host wait
 *     for the GPU, and the fixed scratch array of c3_localize_noalloc.
 *   - Host arrays passed in (pointer tables, tensor metadata) are consumed
 *     before the call returns; the caller may free them immediately.
 *   - Every call enqueues work on `stream` and returns without waiting; its
 *     outputs are valid once the stream has been synchronized.  A NULL
 *     stream is the default (null) stream.
 *   - Errors are returned as negative codes (c3_status_t); nothing is thrown
 *     across the ABI and nothing is launched when an argument check fails.
 *   - Calls on different streams with disjoint outputs and workspaces may
 *     run concurrently.
 *   - Outputs are deterministic: identical inputs give identical bits
 *     whatever the grid size.
 *   - HIP graph capture: c3_consensus, c3_localize, c3_confirm,
 *     c3_timing_consensus and c3_tensor_signature only launch kernels and
 *     can be captured.  c3_signature stages its plan from host memory when
 *     called; capture it with C3_OPT_PLAN_STAGED after an eager call with
 *     the same arguments staged the plan into the workspace, and each
 *     replay reads the tensors' current bytes.  c3_optimizer_check stages a
 *     new plan per slice and is not meant for capture.
 */
#ifndef C3_H_
#define C3_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Binary-compatible with hipStream_t / hipEvent_t. */
typedef struct ihipStream_t *c3_stream_t;
typedef struct ihipEvent_t *c3_event_t;

#define C3_ABI_VERSION 1
/* Replicas per peer group.  c3_signature, c3_tensor_signature, c3_consensus
 * and c3_localize take up to C3_MAX_PEERS (the data-parallel peer degrees the
 * paper tabulates reach 192, Table 2); the fused entry points
 * (c3_timing_consensus, c3_confirm, c3_adamw_slice, c3_optimizer_check) take
 * up to C3_MAX_REPLICAS. */
#define C3_MAX_REPLICAS 64
#define C3_MAX_PEERS 256
/* 64-bit words of one unit's outlier bitmap: bit b of word w names replica
 * 64 w + b (Sec. 5.1's N-bit B).  One word for R <= 64. */
#define C3_BITMAP_WORDS(R) (((R) + 63) / 64)
#define C3_MAX_NDIM 8

typedef enum {
    C3_OK = 0,
    C3_E_INVAL = -1,       /* bad size, count, code or NULL pointer        */
    C3_E_ALIGN = -2,       /* a pointer or stride violates its alignment   */
    C3_E_UNSUPPORTED = -3, /* valid request the library does not implement */
    C3_E_WORKSPACE = -4,   /* workspace NULL, misaligned or too small      */
    C3_E_HIP = -5          /* a HIP runtime call or kernel launch failed   */
} c3_status_t;

/* Element types of checked tensors.  RAW tensors are hashed only. */
typedef enum { C3_F32 = 0, C3_BF16 = 1, C3_F16 = 2, C3_RAW = 3 } c3_dtype_t;

/* Comparison mode of Algorithm 1. */
typedef enum { C3_EXACT = 0, C3_STATISTICAL = 1 } c3_mode_t;

/* How one evidence value is stored.  EXACT compares raw bits of any kind;
 * STATISTICAL reads F32 or F64 values. */
typedef enum { C3_EV_U64 = 0, C3_EV_U32 = 1, C3_EV_F32 = 2, C3_EV_F64 = 3 } c3_evidence_kind_t;

/* Status s of a result (Sec. 5.1): Agree -- the evidence satisfies the rule
 * and B = 0; Attributed -- B names one or more outliers; Inconclusive --
 * peers disagree but no attribution is justified, B = 0. */
typedef enum { C3_AGREE = 0, C3_ATTRIBUTED = 1, C3_INCONCLUSIVE = 2 } c3_verdict_t;

/* Iglewicz-Hoaglin modified z-score cut 3.5 expressed against the raw MAD. */
#define C3_KAPPA_DEFAULT (3.5 / 0.6745)

/* Metadata of one checked tensor: H_w hashes dtype and shape with the bytes
 * (Sec. 5.2).  The tensor occupies prod(shape) * element_size contiguous
 * bytes (element sizes 4, 2, 2, 1 for F32, BF16, F16, RAW); ndim 0 is a
 * scalar. */
typedef struct {
    int32_t dtype;
    int32_t ndim;
    int64_t shape[C3_MAX_NDIM];
} c3_tensor_meta_t;

/* Evidence of one (replica, chunk): the C3SIG-1 signature and the numerical
 * summary of the chunk's finite elements.  64 bytes.
 *   sig        64-bit signature over dtype, shape, chunk index, byte length
 *              and bytes (Sec. 5.2 read per chunk; construction C3SIG-1)
 *   n_elems    elements in the chunk (bytes for RAW)
 *   nan_count, inf_count   non-finite elements (exponent field all ones)
 *   tensor, chunk_in_tensor  position of the chunk
 *   absmax     max |x| over finite x (0 if none)
 *   sum, sumsq sum and sum of squares over finite x, accumulated in fp64
 *              with compensated combination (relative error far below 1e-6)
 *   RAW chunks have zero counts and floats. */
typedef struct {
    uint64_t sig;
    uint64_t n_elems;
    uint32_t nan_count;
    uint32_t inf_count;
    uint32_t tensor;
    uint32_t chunk_in_tensor;
    double absmax;
    double sum;
    double sumsq;
    uint64_t reserved;
} c3_chunk_record_t;

/* One localized outlier: unit (chunk), replica, the lowest replica holding
 * the majority value, and the summaries of both ([0] outlier, [1] majority).
 * 80 bytes. */
typedef struct {
    int64_t chunk;
    int32_t replica;
    int32_t majority_replica;
    uint32_t nan_count[2];
    uint32_t inf_count[2];
    double absmax[2];
    double sum[2];
    double sumsq[2];
} c3_outlier_t;

/* Per-rank verdict of temporal confirmation (c3_confirm).  24 bytes.
 *   flags: bit 0 confirmed straggler (flagged in more than half of some
 *          window of W consecutive iterations); bit 1 protocol outlier
 *          (fingerprint attributed in some iteration); bit 2 flagged in two
 *          consecutive iterations at least once (the paper's own rule).
 *   first_divergent_iter  first iteration with an attributed fingerprint, -1
 *   divergent_count       iterations with an attributed fingerprint
 *   slow_count            iterations with an attributed timing
 *   max_window_slow       largest attributed-timing count in one window
 *   first_straggler_window start of the first window over the threshold, -1 */
typedef struct {
    uint32_t flags;
    int32_t first_divergent_iter;
    uint32_t divergent_count;
    uint32_t slow_count;
    uint32_t max_window_slow;
    int32_t first_straggler_window;
} c3_rank_verdict_t;

#define C3_RANK_STRAGGLER 1u
#define C3_RANK_PROTOCOL 2u
#define C3_RANK_CONSEC2 4u

/* Optional launch controls for c3_signature_ex.
 *   ev_kernel_begin / ev_kernel_end: if non-NULL, recorded on the stream
 *     immediately before the first streaming signature kernel (after the
 *     plan is staged) and immediately after the last one, before the
 *     combine of tile partials that chunks spanning several tiles need.
 *     Either may be given alone, so a run of calls can be timed as a
 *     whole.
 *   grid_blocks: workgroups of the streaming kernel; 0 chooses one per tile.
 *     Results do not depend on it.
 *   flags: C3_OPT_PLAN_STAGED -- the workspace still holds the plan that a
 *     previous c3_signature[_ex] call staged there with identical ptrs,
 *     metas, T, R, chunk_bytes and tile_bytes, and the caller has not written
 *     to the workspace since; staging is skipped.  The caller is responsible
 *     for that promise: a stale plan reads stale pointers.
 *   tile_bytes: bytes one workgroup folds into one partial; 0 chooses the
 *     default (the largest power of two up to 256 KiB dividing chunk_bytes).
 *     Must be a power-of-two multiple of 1024 dividing chunk_bytes
 *     (checked); the fp64 sums may differ in the last bits between tile
 *     sizes, everything else is identical. */
typedef struct {
    c3_event_t ev_kernel_begin;
    c3_event_t ev_kernel_end;
    int32_t grid_blocks;
    int32_t flags;
    uint64_t tile_bytes;
} c3_launch_opts_t;

#define C3_OPT_PLAN_STAGED 1

/* Number of chunks C of the chunk plan: each tensor is split on its own into
 * ceil(nbytes / chunk_bytes) chunks (the last may be partial; an empty
 * tensor has one empty chunk so its dtype and shape are still compared);
 * chunk ids run over tensors in the given order.  Returns C, or a negative
 * c3_status_t for invalid metadata or chunk_bytes. */
int64_t c3_num_chunks(const c3_tensor_meta_t *metas, int T, uint64_t chunk_bytes);

/* Device workspace bytes c3_signature needs for this plan (0 on invalid
 * arguments). */
size_t c3_signature_workspace_size(const c3_tensor_meta_t *metas, int T, int R,
                                   uint64_t chunk_bytes);

/* Workspace bytes for a caller-chosen tile size (c3_launch_opts_t.tile_bytes;
 * 0 = default).  0 on invalid arguments. */
size_t c3_signature_workspace_size_ex(const c3_tensor_meta_t *metas, int T, int R,
                                      uint64_t chunk_bytes, uint64_t tile_bytes);

/*
 * c3_signature -- comparable evidence per chunk (Sec. 5.2; Algorithm 1, the
 * line that turns x_i into e_i).  Reads every replica byte exactly once.
 *
 *   ptrs        host array [R * T] of device pointers, replica-major:
 *               ptrs[r * T + t] is replica r's copy of tensor t.  Each must
 *               be 16-byte aligned (C3_E_ALIGN) and non-NULL unless the
 *               tensor is empty.
 *   metas       host array [T]; shared by all replicas.
 *   T, R        tensors per replica (>= 1) and replicas (1..C3_MAX_PEERS).  Records
 *               are per replica and do not depend on R: with R = 1 a rank
 *               signs its own replica, as each rank of a group spread over
 *               GPUs would before the records are gathered (Algorithm 1's
 *               AllGather); comparing is c3_consensus's job.
 *   chunk_bytes positive multiple of 1024.
 *   records     device [R][C] c3_chunk_record_t, 8-byte aligned; written.
 *   ws, ws_bytes  device workspace of at least
 *               c3_signature_workspace_size(...) bytes, 256-byte aligned;
 *               contents need no initialization and are clobbered.
 */
int c3_signature(const void *const *ptrs, const c3_tensor_meta_t *metas, int T, int R,
                 uint64_t chunk_bytes, c3_chunk_record_t *records, void *ws, size_t ws_bytes,
                 c3_stream_t stream);

/* c3_signature with launch controls (opts may be NULL). */
int c3_signature_ex(const void *const *ptrs, const c3_tensor_meta_t *metas, int T, int R,
                    uint64_t chunk_bytes, c3_chunk_record_t *records, void *ws, size_t ws_bytes,
                    c3_stream_t stream, const c3_launch_opts_t *opts);

/* Device workspace bytes c3_check needs for this plan (tile_bytes as in
 * c3_launch_opts_t; 0 = default).  0 on invalid arguments or R < 2. */
size_t c3_check_workspace_size(const c3_tensor_meta_t *metas, int T, int R, uint64_t chunk_bytes,
                               uint64_t tile_bytes);

/*
 * c3_check -- the whole exact check of Algorithm 1 over R co-resident
 * replicas in one call: the evidence of every chunk (Sec. 5.2, as
 * c3_signature), the strict-majority vote of every chunk on the signatures
 * (Sec. 5.3, as c3_consensus in C3_EXACT mode with replica stride C * 64 and
 * unit stride 64) and the outlier and undecided lists (Sec. 5.1, as
 * c3_localize with the records).  Every output is bit-identical to what those
 * three calls write.
 *   ptrs, metas, T, chunk_bytes, records  as c3_signature.
 *   R           2..C3_MAX_PEERS (R = 1: C3_E_INVAL, Sec. 4).
 *   status, bitmap, majority_idx  device [C], [C][C3_BITMAP_WORDS(R)] u64
 *               (8-byte aligned), [C] i32 (4-byte aligned), as c3_consensus.
 *   outliers, out_cap, undecided, und_cap, counts  as c3_localize.
 *   ws, ws_bytes  device workspace of c3_check_workspace_size(...) bytes,
 *               256-byte aligned, not used by another call at the same time.
 *   opts        as c3_signature_ex (may be NULL): the events bracket the
 *               streaming kernels; C3_OPT_PLAN_STAGED skips staging when a
 *               previous c3_signature_ex or c3_check call staged the same
 *               plan into this workspace.
 * One workgroup combines the tile partials, votes the chunks and writes the
 * lists after the streaming pass for plans of up to 256 chunks, 1,024
 * records and 64 replicas.  Otherwise, for R <= 32, one kernel combines and
 * votes and (for up to 8,192 chunks) a second writes the lists; larger
 * groups run the separate steps.  Errors as the three calls.
 */
int c3_check(const void *const *ptrs, const c3_tensor_meta_t *metas, int T, int R,
             uint64_t chunk_bytes, c3_chunk_record_t *records, uint8_t *status, uint64_t *bitmap,
             int32_t *majority_idx, c3_outlier_t *outliers, int64_t out_cap, int64_t *undecided,
             int64_t und_cap, int64_t *counts, void *ws, size_t ws_bytes, c3_stream_t stream,
             const c3_launch_opts_t *opts);

/*
 * c3_tensor_signature -- one signature per (replica, tensor), the paper's own
 * evidence granularity (Sec. 5.2), from the chunk records of c3_signature:
 *     fmix64(0x4333534947540001 ^ (sum of the tensor's chunk signatures
 *     mod 2^64)).
 *
 *   records  device [R][C] as written by c3_signature (tensor ids must be
 *            non-decreasing along each replica's row, as c3_signature
 *            writes them).
 *   R        replicas, 1..C3_MAX_PEERS.
 *   T        number of tensors (>= 1).
 *   out      device [R][T] u64, 8-byte aligned.  Vote on it with
 *            c3_consensus(out, C3_EV_U64, T * 8, 8, R, T, C3_EXACT, ...).
 */
int c3_tensor_signature(const c3_chunk_record_t *records, int R, int64_t C, int T, uint64_t *out,
                        c3_stream_t stream);

/* AdamW hyperparameters of the optimizer step being replayed (fp64 on the
 * host; step t >= 1 is the step count after this update). */
typedef struct {
    double lr, beta1, beta2, eps, weight_decay;
    int64_t step;
} c3_adamw_hparams_t;

/*
 * c3_adamw_slice -- optimizer-boundary replay (Sec. 9, optimizer boundary;
 * Sec. 6.2, optimizer recipe): one AdamW step (decoupled weight decay,
 * PyTorch's single-tensor operation order, amsgrad off) re-applied to
 * elements [offset, offset + n) of R replicas' fp32 tensors, which are only
 * read.  Per element, each fp32 operation rounded once, no contraction:
 *     p1 = p * fp32(1 - lr wd)
 *     m1 = m + w (g - m)  if |w| < 1/2,  else  g - (g - m)(1 - w);  w = fp32(1 - b1)
 *     v1 = v * fp32(b2) + (fp32(1 - b2) g) g
 *     p2 = p1 + fp32(-lr / (1 - b1^t)) * (m1 / (sqrt(v1) / fp32(sqrt(1 - b2^t)) + fp32(eps)))
 * with the scalar factors formed in fp64.  A NaN result is stored as the
 * quiet NaN 0x7FC00000.
 *
 *   param, grad, exp_avg, exp_avg_sq  host arrays [R] of device pointers to
 *            each replica's tensor of `numel` fp32 elements (4-byte aligned;
 *            16-byte aligned bases with offset, n and out_stride multiples
 *            of 4 take the 128-bit path).
 *   out      device fp32, caller-owned: row (replica r, j) at out + (3 r + j)
 *            out_stride holds the n updated values of the parameter (j = 0),
 *            first moment (1) and second moment (2) -- three tensors of n
 *            elements per replica for c3_signature.  out_stride >= n; 0
 *            means n (packed [R][3][n]).
 *   R in 1..64; 0 <= offset, offset + n <= numel; lr >= 0, 0 <= b1, b2 < 1,
 *   eps > 0, wd >= 0, step >= 1, else C3_E_INVAL; misaligned pointers
 *   C3_E_ALIGN; a failed launch C3_E_HIP.  n = 0 does nothing.  Asynchronous
 *   on `stream`.
 */
int c3_adamw_slice(const float *const *param, const float *const *grad,
                   const float *const *exp_avg, const float *const *exp_avg_sq, int R,
                   int64_t numel, int64_t offset, int64_t n, const c3_adamw_hparams_t *hp,
                   float *out, int64_t out_stride, c3_stream_t stream);

/* One optimizer-boundary check over R replicas' AdamW state (Sec. 9). */
typedef struct {
    const float *const *param;       /* host arrays [R] of device pointers, */
    const float *const *grad;        /* numel fp32 elements each, 16-byte   */
    const float *const *exp_avg;     /* aligned                              */
    const float *const *exp_avg_sq;
    int32_t R;                       /* 2..64 */
    int32_t reserved;
    int64_t numel;
    int64_t slice_elems;             /* S: multiple of 256 (65536 in Sec. 9) */
    uint64_t tile_bytes;             /* signature tile: a power of two >= 1024,
                                        lowered until it divides 4 S; 0 = 64 KiB */
} c3_optimizer_state_t;

/* Device outputs of c3_optimizer_check, all caller-owned.  Unit u of the
 * vote is tensor u of each replica: 0 param, 1 grad, 2 exp_avg, 3
 * exp_avg_sq (the input slices), 4 param, 5 exp_avg, 6 exp_avg_sq (the
 * replayed updates). */
typedef struct {
    float *updated;                  /* [R][3][S], 16-byte aligned */
    c3_chunk_record_t *records;      /* [R][7] */
    uint8_t *status;                 /* [7] */
    uint64_t *bitmap;                /* [7] */
    int32_t *majority_idx;           /* [7] */
    c3_outlier_t *outliers;          /* [7 R] */
    int64_t *undecided;              /* [7] */
    int64_t *counts;                 /* [3], as c3_localize */
} c3_optimizer_check_out_t;

/* Workspace bytes for c3_optimizer_check with this state; 0 if invalid. */
size_t c3_optimizer_check_workspace_size(const c3_optimizer_state_t *st);

/*
 * c3_optimizer_check -- scheduled check k at the optimizer boundary (Sec. 9;
 * Sec. 6.2 optimizer recipe; exact C3 of Algorithm 1 on the slices).  Takes
 * the rotating slice [off, off + n): off = (k mod ceil(numel / S)) S, n =
 * min(S, numel - off).  Enqueues on `stream`:
 *   1. c3_adamw_slice on that slice into `updated` (row stride S);
 *   2. c3_signature of seven tensors of n fp32 elements per replica (the
 *      four input slices, read in place, and the three updated slices),
 *      one chunk each;
 *   3. c3_consensus (exact) over the seven units; 4. c3_localize.
 * The outputs are those of these four calls; after the streaming kernel of
 * step 2, one single-workgroup kernel combines the tile partials into the
 * records, votes and writes the lists (R <= 64: always).
 * Healthy data-parallel replicas agree on all seven units; an outlier on an
 * input unit names replicas whose state diverged before the step, one on an
 * output unit only names replicas whose replayed update differs.
 * k >= 0; errors as the four calls (C3_E_INVAL, C3_E_ALIGN, C3_E_WORKSPACE,
 * C3_E_HIP); workspace 256-byte aligned, at least
 * c3_optimizer_check_workspace_size bytes, not used concurrently.
 */
int c3_optimizer_check(const c3_optimizer_state_t *st, int64_t k, const c3_adamw_hparams_t *hp,
                       const c3_optimizer_check_out_t *out, void *ws, size_t ws_bytes,
                       c3_stream_t stream);

/*
 * c3_consensus -- the decision of Algorithm 1 for n_units independent units
 * (chunks, or (iteration, group) records), each with R peer values.
 *
 * Replica r's value for unit u is read at
 *   (const char *)evidence + u * unit_stride_bytes + r * replica_stride_bytes
 * e.g. signatures inside the record table: evidence = &records[0].sig,
 * replica_stride = C * 64, unit_stride = 64.  Strides and the base must be
 * multiples of the value size (8 for U64/F64, 4 for U32/F32): C3_E_ALIGN.
 *
 *   EXACT (Sec. 5.3): c* = count of the most frequent value; if 2 c* <= R the
 *     unit is Inconclusive with B = 0; otherwise bit r of B is set iff
 *     replica r differs from the majority value, status Attributed if B != 0
 *     else Agree, majority_idx = lowest replica holding the majority value.
 *   STATISTICAL (Sec. 5.4), evidence kind F32 or F64, in fp64: a non-finite
 *     value marks its replica; if finite values are not a strict majority the
 *     unit is Inconclusive; m = median of the finite values; d = MAD, else
 *     half the type-7 interquartile range, else range / n_finite; if d = 0
 *     only non-finite replicas are marked; otherwise replica r is marked iff
 *     |x_r - m| > kappa * d.  majority_idx = replica at the lower median.
 *     kappa > 0 (C3_KAPPA_DEFAULT recommended); ignored for EXACT.
 *
 *   status [n_units] u8 (c3_verdict_t), bitmap [n_units][C3_BITMAP_WORDS(R)]
 *   u64 (8-byte aligned), majority_idx [n_units] i32 (-1 when Inconclusive);
 *   device.  R in 2..C3_MAX_PEERS, n_units >= 0.  R = 1 is C3_E_INVAL: a group
 *   of one peer provides no comparison (Sec. 4), so no vote over it may
 *   return Agree.
 */
int c3_consensus(const void *evidence, int evidence_kind, int64_t replica_stride_bytes,
                 int64_t unit_stride_bytes, int R, int64_t n_units, int mode, double kappa,
                 uint8_t *status, uint64_t *bitmap, int32_t *majority_idx, c3_stream_t stream);

/* Device workspace bytes c3_localize needs for n_units. */
size_t c3_localize_workspace_size(int64_t n_units);

/*
 * c3_localize -- turns per-unit results into lists: which replica, which
 * chunk, what summary (Sec. 5.1: B[i] = 1 attributes the divergence to peer
 * i; Sec. 9: reports keep the peers and bitmaps).
 *
 *   status, bitmap, majority_idx  as c3_consensus writes them: bitmap is
 *              [n_units][C3_BITMAP_WORDS(R)] u64; R in 2..C3_MAX_PEERS (R = 1:
 *              C3_E_INVAL, as c3_consensus).
 *   outliers   device [out_cap]: one entry per set bitmap bit, ordered by
 *              (unit ascending, replica ascending).  With records (device
 *              [R][n_units], may be NULL) each entry carries the outlier's
 *              and the majority replica's summary; without, those are 0.
 *   undecided  device [und_cap] i64: Inconclusive units, ascending.
 *   counts     device [3] i64: total outliers, total undecided units, units
 *              with at least one outlier.  Totals are always exact; only
 *              min(total, cap) entries are written, so the caller detects
 *              truncation by comparing counts with the caps.
 *   ws         device workspace of c3_localize_workspace_size(n_units)
 *              bytes, 256-byte aligned.
 */
int c3_localize(const uint8_t *status, const uint64_t *bitmap, const int32_t *majority_idx,
                const c3_chunk_record_t *records, int R, int64_t n_units, c3_outlier_t *outliers,
                int64_t out_cap, int64_t *undecided, int64_t und_cap, int64_t *counts, void *ws,
                size_t ws_bytes, c3_stream_t stream);

/* Largest n_units that c3_localize_noalloc accepts. */
#define C3_LOCALIZE_NOALLOC_MAX_UNITS (1ll << 26)

/*
 * c3_localize_noalloc -- c3_localize for callers that cannot allocate device
 * memory: code under HIP graph capture, tight serving loops and harnesses
 * that forbid allocation.  Same arguments, outputs and errors as
 * c3_localize, without the workspace: the segment counts and offsets it
 * needs for more than 32,768 units live in a fixed 1 MiB device array that
 * the library holds on every device it runs on until the process ends.  The
 * call allocates nothing (no hipMalloc, no host allocation); the first call
 * on a device looks up that device's copy of the array.
 *   n_units    0..C3_LOCALIZE_NOALLOC_MAX_UNITS (2^26); more is C3_E_INVAL.
 * Every call on one device shares that device's array: calls that overlap on
 * one device (two streams, or two host threads) race and must be ordered by
 * the caller.  Results are bit-identical to c3_localize's.
 */
int c3_localize_noalloc(const uint8_t *status, const uint64_t *bitmap,
                        const int32_t *majority_idx, const c3_chunk_record_t *records, int R,
                        int64_t n_units, c3_outlier_t *outliers, int64_t out_cap,
                        int64_t *undecided, int64_t und_cap, int64_t *counts,
                        c3_stream_t stream);

/* Device workspace bytes c3_timing_consensus needs (256 at least; 0 if the
 * sizes are invalid). */
size_t c3_timing_consensus_workspace_size(int R, int64_t G, int64_t T, int window);

/*
 * c3_timing_consensus -- the whole timing path in one call: per (iteration
 * t, group g) exact C3 on the ranks' collective fingerprints (Sec. 5.3; a
 * minority fingerprint is a protocol outlier, Sec. 7) and statistical C3 on
 * their step times (Sec. 5.4), then per-rank temporal confirmation (Sec. 10
 * protocol).  The results equal c3_consensus(fingerprints, EXACT) and
 * c3_consensus(times, STATISTICAL) per unit and c3_confirm on their bitmaps.
 *
 *   R             ranks per group, 2..C3_MAX_REPLICAS (R = 1: C3_E_INVAL; a
 *                 group of one rank provides no comparison, Sec. 4).
 *   fingerprints  device [T][G][R] u64, ranks innermost (8-byte aligned).
 *   times         device [T][G][R] fp32 (C3_EV_F32) or fp64 (C3_EV_F64).
 *   kappa         statistical threshold (> 0); window W >= 1 as c3_confirm.
 *   fp_status/fp_bitmap/fp_majority, t_status/t_bitmap/t_majority
 *                 device [T*G] per-unit results (unit t*G + g), or all
 *                 three NULL for a kind whose per-unit results are not
 *                 wanted (then only the verdicts are produced for it).
 *   verdicts      device [R*G], rank = r*G + g, as c3_confirm.
 * Execution (results do not depend on it):
 *   - R in {4, 8, 16}, both arrays 16-byte aligned, W <= 64,
 *     2 * ceil(T / 32) * R * 64 bytes <= 64 KiB and G / 16 at least the
 *     device's compute-unit count: one kernel, with the per-unit results of
 *     either kind, both or neither; each workgroup votes 16 groups over all
 *     T iterations (writing their per-unit results when requested),
 *     collects its ranks' outlier bits in LDS and confirms them there (the
 *     workspace is not touched);
 *   - otherwise, for R <= 16 and W <= 64: a clearing kernel, one kernel
 *     voting both kinds that ORs each outlier bit into per-rank masks in the
 *     workspace, and a confirmation kernel over those masks;
 *   - otherwise the three separate steps (c3_consensus twice, c3_confirm),
 *     with the per-unit results kept in the workspace when not requested.
 * Errors: C3_E_INVAL (sizes, kinds, kappa, outputs half given),
 * C3_E_WORKSPACE, C3_E_ALIGN, C3_E_HIP.  R * G == 0 does nothing.
 */
int c3_timing_consensus(const uint64_t *fingerprints, const void *times, int time_kind, int R,
                        int64_t G, int64_t T, double kappa, int window, uint8_t *fp_status,
                        uint64_t *fp_bitmap, int32_t *fp_majority, uint8_t *t_status,
                        uint64_t *t_bitmap, int32_t *t_majority, c3_rank_verdict_t *verdicts,
                        void *ws, size_t ws_bytes, c3_stream_t stream);

/* Device workspace bytes c3_confirm needs. */
size_t c3_confirm_workspace_size(int R, int64_t G, int64_t T);

/*
 * c3_confirm -- temporal confirmation of per-iteration results for G peer
 * groups of R ranks over T consecutive iterations (Sec. 10 protocol: a
 * straggler must recur across timing rounds before it is reported; Sec. 7:
 * a minority collective fingerprint is a protocol outlier).
 *
 *   R         ranks per group, 2..C3_MAX_REPLICAS (R = 1: C3_E_INVAL, as
 *             c3_consensus).
 *   fp_bitmap, time_bitmap  device [T][G] u64: the bitmaps c3_consensus
 *             produced for the fingerprint (EXACT) and timing (STATISTICAL)
 *             evidence of unit (t, g).
 *   window    W >= 1 (capped at T): a rank is a confirmed straggler when its
 *             timing is attributed in more than W/2 iterations of some
 *             window of W consecutive iterations.
 *   verdicts  device [R * G], rank = r * G + g (row-major placement with
 *             the replica index major, as in the Sec. 4 example).
 */
int c3_confirm(const uint64_t *fp_bitmap, const uint64_t *time_bitmap, int R, int64_t G,
               int64_t T, int window, c3_rank_verdict_t *verdicts, void *ws, size_t ws_bytes,
               c3_stream_t stream);

/* ---------------------------------------------------------------------- */
/* Checkpoint certification (Sec. 8, Algorithm 3).  Host-only calls; no   */
/* GPU work.  Checkpoint identifiers are caller-chosen non-negative       */
/* integers (e.g. the training step); -1 means none.                      */
/* ---------------------------------------------------------------------- */

/* Job-wide outcome of one replay boundary. */
typedef enum {
    C3_OUTCOME_OK = 0,        /* every comparison agreed                        */
    C3_OUTCOME_STRAGGLER = 1, /* a confirmed straggler, numbers agree           */
    C3_OUTCOME_SDC = 2,       /* some comparison group's evidence disagreed     */
    C3_OUTCOME_HANG = 3       /* a hang or protocol divergence was reported     */
} c3_outcome_t;

/* State of Algorithm 3: recipe catalog size K, accepted recipes q in the
 * current cycle, and the latest, candidate and verified checkpoints. */
typedef struct {
    int32_t K;
    int32_t q;
    int64_t latest;
    int64_t candidate;
    int64_t verified;
} c3_ckpt_state_t;

/* What one c3_ckpt_save call asks the checkpoint system to do.
 *   captured      the new in-memory checkpoint becomes latest
 *   persisted_id  persist this checkpoint as the new candidate (-1: none)
 *   promoted      the previous candidate became verified
 *   retrieve      recovery must restart from retrieve_id (-1: no verified
 *                 checkpoint exists yet) */
typedef struct {
    int32_t captured;
    int32_t promoted;
    int32_t retrieve;
    int32_t reserved;
    int64_t persisted_id;
    int64_t retrieve_id;
} c3_ckpt_action_t;

/* Combines one boundary's evidence into an outcome, most severe first:
 * sdc_units > 0 (attributed or undecided chunks: peers disagree) -> SDC;
 * hang_signals > 0 (hang or protocol-outlier reports) -> HANG;
 * stragglers > 0 -> STRAGGLER; else OK.  Negative counts: C3_E_INVAL. */
int c3_job_outcome(int64_t sdc_units, int64_t hang_signals, int64_t stragglers);

/* Starts a checkpoint cycle for a catalog of K >= 1 recipes (q = 0, no
 * checkpoints). */
int c3_ckpt_init(c3_ckpt_state_t *st, int K);

/* CheckpointSave of Algorithm 3 at one replay boundary.
 *   OK or STRAGGLER: checkpoint_id becomes latest and q advances; when q
 *     reaches K, q resets, the previous candidate (if any) is promoted to
 *     verified and checkpoint_id is persisted as the new candidate.
 *   SDC or HANG: nothing is captured; act->retrieve_id is the checkpoint
 *     CheckpointRetrieval selects (see c3_ckpt_retrieve).  The state is left
 *     as it was; after recovery the caller starts a new cycle.
 * machines_accessible and full_catalog_sdc are the retrieval inputs: whether
 * every machine's latest shard is reachable, and whether a full-catalog
 * replay (run by the caller) found SDC. */
int c3_ckpt_save(c3_ckpt_state_t *st, int outcome, int64_t checkpoint_id, int machines_accessible,
                 int full_catalog_sdc, c3_ckpt_action_t *act);

/* CheckpointRetrieval of Algorithm 3: SDC or an unreachable machine ->
 * verified; STRAGGLER -> latest; otherwise latest unless the full-catalog
 * replay found SDC, then verified. */
int c3_ckpt_retrieve(const c3_ckpt_state_t *st, int outcome, int machines_accessible,
                     int full_catalog_sdc, int64_t *checkpoint_id);

/* ---------------------------------------------------------------------- */
/* Measurement aid (not part of the method).                              */
/* ---------------------------------------------------------------------- */

/*
 * c3_read_probe -- reads `bytes` of device memory once with the streaming
 * signature kernel's access pattern (one 256-thread workgroup per tile,
 * 1 KiB blocks round-robin over its four waves, 128-bit non-temporal loads,
 * 16 in flight per lane) and nothing else, so the signature pass can be set
 * against the read rate this pattern reaches on the same device.
 *   buf        device, 16-byte aligned; bytes a multiple of 1024 (whole
 *              1 KiB blocks, so every load lies inside the buffer; 0: nothing).
 *   tile_bytes power of two in [1 KiB, 16 MiB]; 0 = the signature kernel's
 *              default tile (256 KiB).
 *   checksum   device [ceil(bytes / tile_bytes)] u64, 8-byte aligned: the
 *              xor of the little-endian 64-bit words of each tile.
 *   ev_begin, ev_end  optional events recorded on the stream immediately
 *              around the probe kernel.
 * Errors: C3_E_INVAL, C3_E_ALIGN, C3_E_HIP.
 */
int c3_read_probe(const void *buf, uint64_t bytes, uint64_t tile_bytes, uint64_t *checksum,
                  c3_event_t ev_begin, c3_event_t ev_end, c3_stream_t stream);

/* Static description of a status code. */
const char *c3_status_string(int code);

/* C3_ABI_VERSION of the loaded library. */
int c3_abi_version(void);

#ifdef __cplusplus
}
#endif

#endif /* C3_H_ */
