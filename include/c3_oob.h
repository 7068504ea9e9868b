/*
 * c3_oob.h -- C ABI of out-of-band hang localization for C3 (host only).
 *
 * Paper: "SCOUT: Symmetric Consensus Outlier Detection for Failure
 * Localization in LLM Pre-Training" (arXiv 2608.11034), Sec. 7 (out-of-band
 * hang localization) and Sec. 9 (progress path and communication).
 *
 * A hang stops the trainer and its collectives, so its evidence has to live
 * outside them.  Each trainer rank publishes a monotonic progress coordinate
 * (optimizer step, operation id) and, right before it enters a collective
 * that may block, a fingerprint of that collective (process group, type and
 * the arguments every healthy caller shares) into a lock-free record in
 * POSIX shared memory.  A CPU-only observer process per rank reads the
 * record; once visible progress has been silent beyond a threshold the
 * observers exchange their records (over a communicator of their own) and
 * apply exact C3 to them.  A strict-majority record with a minority of
 * differing ranks localizes a rank-local stall or control-flow divergence
 * (the coordinate differs) or a collective-protocol mismatch (same
 * coordinate, different collective); a record shared by every rank points
 * to a group-scoped runtime or transport stall.
 *
 * This library is plain C++ (no HIP): observers never touch a GPU.  It
 * implements the record, its publication and snapshot, the fingerprints
 * and the classification.  The exchange between observers is the caller's
 * (the Python observer uses a Gloo process group).
 *
 * Conventions: negative return values are C3_OOB_E_* codes; no call blocks
 * except c3_progress_wait_silence, which sleeps at most max_wait_ns.
 */
#ifndef C3_OOB_H_
#define C3_OOB_H_

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define C3_OOB_ABI_VERSION 1
#define C3_OOB_MAX_RANKS 64 /* one 64-bit outlier bitmap */
#define C3_OOB_MAX_NDIM 8

#define C3_OOB_OK 0
#define C3_OOB_E_INVAL (-1) /* bad argument                                  */
#define C3_OOB_E_SYS (-2)   /* shm_open / ftruncate / mmap failed (errno set) */
#define C3_OOB_E_BUSY (-3)  /* no consistent snapshot within the retry bound */
#define C3_OOB_E_FORMAT (-4) /* the segment is not a progress segment of this version */

/* Progress record flags. */
#define C3_OOB_PENDING 1u /* the rank entered the fingerprinted collective and has not left it */

/* Snapshot of one rank's progress record (Sec. 7, comparable progress). */
typedef struct {
    uint64_t step;        /* optimizer step */
    uint64_t op_id;       /* operation identifier within the step */
    uint64_t fingerprint; /* fingerprint of the pending collective; 0 if none */
    uint64_t publish_ns;  /* CLOCK_MONOTONIC time of the latest publication */
    uint64_t publishes;   /* publications so far: the visible progress counter */
    uint32_t flags;       /* C3_OOB_PENDING */
    uint32_t pid;         /* process that mapped the publishing handle */
} c3_progress_t;          /* 48 bytes */

/* Opaque mapping of a progress segment (one record slot per local rank). */
typedef struct c3_progress_seg c3_progress_seg_t;

/* Maps the POSIX shared-memory segment `name` ("/..." as for shm_open) with
 * n_slots record slots (1..C3_OOB_MAX_RANKS).  create != 0 creates it (or
 * reuses an existing segment of the same geometry) and zeroes nothing that
 * already exists; create == 0 attaches to an existing segment and checks
 * its header.  *out receives the handle (caller-owned, c3_progress_close). */
int c3_progress_open(const char *name, int n_slots, int create, c3_progress_seg_t **out);

/* Unmaps the segment; unlink != 0 also removes its name. */
int c3_progress_close(c3_progress_seg_t *seg, int unlink_name);

/* Slots in the segment, or C3_OOB_E_INVAL. */
int c3_progress_slots(const c3_progress_seg_t *seg);

/* Publishes (step, op_id, fingerprint, flags) into `slot`: the slot's single
 * writer (the trainer rank) fills the spare one of two sequence-locked copies
 * and then announces it, wait-free, with no system call beyond reading
 * CLOCK_MONOTONIC.  A writer stopped mid-publication leaves the previous
 * copy readable.  Publish the fingerprint with
 * C3_OOB_PENDING immediately before entering a collective that may block,
 * and the next coordinate (no fingerprint) after it returns. */
int c3_progress_publish(c3_progress_seg_t *seg, int slot, uint64_t step, uint64_t op_id,
                        uint64_t fingerprint, uint32_t flags);

/* Consistent snapshot of the latest complete publication in `slot`
 * (publishes = 0 and zero fields before the first).  Retries only while the
 * writer overtakes the reader by two publications, at most 1<<20 times,
 * then C3_OOB_E_BUSY. */
int c3_progress_read(const c3_progress_seg_t *seg, int slot, c3_progress_t *out);

/* Observer wait: polls `slot` every poll_ns.  Returns 1 with the snapshot in
 * *out once the publication counter has stayed unchanged for silence_ns
 * (silence is measured from the call when nothing was published yet), 0 if
 * max_wait_ns passes first (*out holds the latest snapshot), or a negative
 * code. */
int c3_progress_wait_silence(const c3_progress_seg_t *seg, int slot, uint64_t silence_ns,
                             uint64_t poll_ns, uint64_t max_wait_ns, c3_progress_t *out);

/* Collective types for fingerprints. */
enum {
    C3_COLL_ALL_REDUCE = 1,
    C3_COLL_ALL_GATHER = 2,
    C3_COLL_REDUCE_SCATTER = 3,
    C3_COLL_BROADCAST = 4,
    C3_COLL_REDUCE = 5,
    C3_COLL_ALL_TO_ALL = 6,
    C3_COLL_BARRIER = 7,
    C3_COLL_SEND = 8,
    C3_COLL_RECV = 9
};

/* What healthy callers of one collective must share (Sec. 7).  Fields
 * that do not apply are -1 (reduce_op, root) or ndim = 0.  ndim = -1 marks
 * a legitimately rank-dependent shape (e.g. variable all-to-all splits):
 * the shape is left out of the fingerprint. */
typedef struct {
    uint64_t process_group; /* c3_group_id of the group's ordered member ranks */
    int32_t kind;           /* C3_COLL_* */
    int32_t dtype;          /* the framework's dtype code */
    int32_t reduce_op;      /* the framework's reduction code, or -1 */
    int32_t root;           /* root or peer rank within the group, or -1 */
    int32_t ndim;           /* 0..8, or -1 (shape not compared) */
    int32_t reserved;       /* must be 0 */
    int64_t shape[C3_OOB_MAX_NDIM];
} c3_collective_t;          /* 96 bytes */

/* Identifier of an ordered process group (n >= 1 member ranks):
 *   h = fmix64(0x4333475250000001 ^ n); h = fmix64(h ^ rank) per member. */
uint64_t c3_group_id(const int32_t *ranks, int n);

/* Fingerprint C3FP-1 of a collective (never 0; 0 on invalid input):
 *   h = fmix64(0x4333465000000001 ^ (kind << 32) ^ (uint32)dtype)
 *   h = fmix64(h ^ process_group)
 *   h = fmix64(h ^ ((uint32)reduce_op << 32 | (uint32)root))
 *   h = fmix64(h ^ (uint64)(int64)ndim), then h = fmix64(h ^ shape[d]) per dim
 *   fingerprint = h, or 1 if h = 0.
 * fmix64 is MurmurHash3's 64-bit finalizer. */
uint64_t c3_collective_fingerprint(const c3_collective_t *c);

/* Exact-C3 evidence of a progress record: the coordinate, the pending
 * fingerprint and the pending flag, hashed to 64 bits:
 *   h = fmix64(0x4333505247000001 ^ step); h = fmix64(h ^ op_id);
 *   h = fmix64(h ^ fingerprint); h = fmix64(h ^ (flags & C3_OOB_PENDING)). */
uint64_t c3_progress_evidence(const c3_progress_t *p);

/* Hang classes (Sec. 7, guiding recovery). */
enum {
    C3_HANG_GROUP_STALL = 0,    /* every peer holds the same record */
    C3_HANG_RANK_DIVERGENCE = 1, /* a strict majority record and a minority of outliers */
    C3_HANG_INCONCLUSIVE = 2     /* no strict majority */
};
/* Per-peer reasons. */
enum {
    C3_HANG_REASON_NONE = 0,
    C3_HANG_REASON_PROGRESS = 1, /* its (step, op_id) differs from the majority's */
    C3_HANG_REASON_PROTOCOL = 2  /* same coordinate, other collective or pending state */
};

typedef struct {
    int32_t cls;          /* C3_HANG_* */
    int32_t majority_idx; /* a peer holding the majority record; -1 if inconclusive */
    uint64_t bitmap;      /* bit i: peer i is an outlier (0 unless RANK_DIVERGENCE) */
    uint8_t reason[C3_OOB_MAX_RANKS]; /* C3_HANG_REASON_* per peer */
} c3_hang_verdict_t;      /* 80 bytes */

/* Exact C3 (Algorithm 1, Exact branch) over the R gathered records (peer i
 * = records[i], R in 2..64; a single rank has no peer to compare with,
 * Sec. 4), evidence c3_progress_evidence: the most
 * frequent record with 2 c* > R is the majority, the rest are outliers.
 * Their reasons compare coordinates with the majority record. */
int c3_hang_classify(const c3_progress_t *records, int R, c3_hang_verdict_t *out);

int c3_oob_abi_version(void);

#ifdef __cplusplus
}
#endif

#endif /* C3_OOB_H_ */
