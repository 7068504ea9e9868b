// Out-of-band hang localization of C3 (Sec. 7; Sec. 9 progress path):
// lock-free progress records in POSIX shared memory, collective
// fingerprints, and exact C3 over the records the observers gather.
//
// Segment layout: a 64-byte header (magic, version, slot count, slot size)
// followed by one 128-byte slot per local rank, so writers of different
// slots never share a cache line.  A slot holds two copies of the record,
// each a sequence lock, and the number of the latest complete publication.
// Publication n writes copy n mod 2 (its sequence odd while the fields are
// stored, even afterwards) and then announces n.  A reader takes the copy
// of the announced publication and retries only if that copy's sequence
// moved while it read, which needs two further publications (a copy also
// records which publication it holds, so the snapshot is that one).  A writer
// stopped in the middle of a publication (a frozen trainer is exactly the
// case to observe) therefore never blocks readers: the announced copy stays
// complete.  All fields are atomics (relaxed, ordered by the sequences'
// release/acquire), so a snapshot is never torn.
#include "../../../include/c3_oob.h"

#include <errno.h>
#include <fcntl.h>
#include <string.h>
#include <sys/mman.h>
#include <sys/stat.h>
#include <time.h>
#include <unistd.h>

#include <atomic>
#include <new>

namespace {

constexpr uint64_t kMagic = 0x43334F4F42505247ull;  // "C3OOBPRG"
constexpr uint32_t kVersion = 1;
constexpr uint64_t kTagGroup = 0x4333475250000001ull;
constexpr uint64_t kTagColl = 0x4333465000000001ull;
constexpr uint64_t kTagProgress = 0x4333505247000001ull;
constexpr int kReadRetries = 1 << 20;

struct alignas(64) Header {
    uint64_t magic;
    uint32_t version;
    uint32_t n_slots;
    uint32_t slot_bytes;
    uint32_t pad[11];
};

struct Copy {
    std::atomic<uint64_t> seq;
    std::atomic<uint64_t> number;  // which publication this copy holds
    std::atomic<uint64_t> step;
    std::atomic<uint64_t> op_id;
    std::atomic<uint64_t> fingerprint;
    std::atomic<uint64_t> publish_ns;
    std::atomic<uint32_t> flags;
    std::atomic<uint32_t> pid;
};

struct alignas(64) Slot {
    std::atomic<uint64_t> latest;  // number of the latest complete publication
    Copy copy[2];
    uint64_t pad;
};
static_assert(sizeof(Header) == 64 && sizeof(Slot) == 128, "segment layout");
static_assert(std::atomic<uint64_t>::is_always_lock_free, "lock-free record");
static_assert(sizeof(c3_progress_t) == 48, "snapshot layout");
static_assert(sizeof(c3_collective_t) == 96, "collective layout");
static_assert(sizeof(c3_hang_verdict_t) == 80, "verdict layout");

uint64_t fmix64(uint64_t k) {
    k ^= k >> 33;
    k *= 0xFF51AFD7ED558CCDull;
    k ^= k >> 33;
    k *= 0xC4CEB9FE1A85EC53ull;
    k ^= k >> 33;
    return k;
}

uint64_t now_ns() {
    timespec ts;
    clock_gettime(CLOCK_MONOTONIC, &ts);
    return (uint64_t)ts.tv_sec * 1000000000ull + (uint64_t)ts.tv_nsec;
}

size_t segment_bytes(int n_slots) { return sizeof(Header) + sizeof(Slot) * (size_t)n_slots; }

}  // namespace

struct c3_progress_seg {
    void* base;
    size_t bytes;
    int n_slots;
    uint32_t pid;  // of the process that mapped the segment
    char name[256];
    Header* header() const { return static_cast<Header*>(base); }
    Slot* slot(int i) const {
        return reinterpret_cast<Slot*>(static_cast<char*>(base) + sizeof(Header)) + i;
    }
};

extern "C" {

int c3_oob_abi_version(void) { return C3_OOB_ABI_VERSION; }

int c3_progress_open(const char* name, int n_slots, int create, c3_progress_seg_t** out) {
    if (name == nullptr || out == nullptr || name[0] != '/' || strlen(name) >= 255)
        return C3_OOB_E_INVAL;
    *out = nullptr;
    if (create && (n_slots < 1 || n_slots > C3_OOB_MAX_RANKS)) return C3_OOB_E_INVAL;
    const int fd = shm_open(name, create ? (O_RDWR | O_CREAT) : O_RDWR, 0600);
    if (fd < 0) return C3_OOB_E_SYS;
    struct stat st;
    if (fstat(fd, &st) != 0) {
        close(fd);
        return C3_OOB_E_SYS;
    }
    size_t bytes;
    if (create) {
        bytes = segment_bytes(n_slots);
        if (st.st_size != 0 && (size_t)st.st_size != bytes) {
            close(fd);
            return C3_OOB_E_FORMAT;
        }
        if (st.st_size == 0 && ftruncate(fd, (off_t)bytes) != 0) {
            close(fd);
            return C3_OOB_E_SYS;
        }
    } else {
        if ((size_t)st.st_size < sizeof(Header)) {
            close(fd);
            return C3_OOB_E_FORMAT;
        }
        bytes = (size_t)st.st_size;
    }
    void* base = mmap(nullptr, bytes, PROT_READ | PROT_WRITE, MAP_SHARED, fd, 0);
    close(fd);
    if (base == MAP_FAILED) return C3_OOB_E_SYS;
    Header* h = static_cast<Header*>(base);
    if (create && h->magic == 0) {
        // a fresh segment reads as zeros: fill in the header last
        h->n_slots = (uint32_t)n_slots;
        h->slot_bytes = (uint32_t)sizeof(Slot);
        h->version = kVersion;
        std::atomic_thread_fence(std::memory_order_release);
        reinterpret_cast<std::atomic<uint64_t>*>(&h->magic)->store(kMagic, std::memory_order_release);
    }
    const uint64_t magic =
        reinterpret_cast<std::atomic<uint64_t>*>(&h->magic)->load(std::memory_order_acquire);
    if (magic != kMagic || h->version != kVersion || h->slot_bytes != sizeof(Slot) ||
        h->n_slots < 1 || h->n_slots > (uint32_t)C3_OOB_MAX_RANKS ||
        segment_bytes((int)h->n_slots) > bytes || (create && h->n_slots != (uint32_t)n_slots)) {
        munmap(base, bytes);
        return C3_OOB_E_FORMAT;
    }
    c3_progress_seg* seg = new (std::nothrow) c3_progress_seg;
    if (seg == nullptr) {
        munmap(base, bytes);
        return C3_OOB_E_SYS;
    }
    seg->base = base;
    seg->bytes = bytes;
    seg->n_slots = (int)h->n_slots;
    seg->pid = (uint32_t)getpid();
    strncpy(seg->name, name, sizeof(seg->name) - 1);
    seg->name[sizeof(seg->name) - 1] = '\0';
    *out = seg;
    return C3_OOB_OK;
}

int c3_progress_close(c3_progress_seg_t* seg, int unlink_name) {
    if (seg == nullptr) return C3_OOB_E_INVAL;
    munmap(seg->base, seg->bytes);
    int rc = C3_OOB_OK;
    if (unlink_name && shm_unlink(seg->name) != 0) rc = C3_OOB_E_SYS;
    delete seg;
    return rc;
}

int c3_progress_slots(const c3_progress_seg_t* seg) {
    return seg == nullptr ? C3_OOB_E_INVAL : seg->n_slots;
}

int c3_progress_publish(c3_progress_seg_t* seg, int slot, uint64_t step, uint64_t op_id,
                        uint64_t fingerprint, uint32_t flags) {
    if (seg == nullptr || slot < 0 || slot >= seg->n_slots) return C3_OOB_E_INVAL;
    Slot* s = seg->slot(slot);
    const uint64_t n = s->latest.load(std::memory_order_relaxed) + 1;  // single writer
    Copy& c = s->copy[n & 1];
    const uint64_t seq = c.seq.load(std::memory_order_relaxed);
    c.seq.store(seq | 1u, std::memory_order_relaxed);  // odd: write in progress
    std::atomic_thread_fence(std::memory_order_release);
    c.number.store(n, std::memory_order_relaxed);
    c.step.store(step, std::memory_order_relaxed);
    c.op_id.store(op_id, std::memory_order_relaxed);
    c.fingerprint.store(fingerprint, std::memory_order_relaxed);
    c.flags.store(flags, std::memory_order_relaxed);
    c.pid.store(seg->pid, std::memory_order_relaxed);
    c.publish_ns.store(now_ns(), std::memory_order_relaxed);
    c.seq.store((seq | 1u) + 1u, std::memory_order_release);  // even: complete
    s->latest.store(n, std::memory_order_release);
    return C3_OOB_OK;
}

int c3_progress_read(const c3_progress_seg_t* seg, int slot, c3_progress_t* out) {
    if (seg == nullptr || out == nullptr || slot < 0 || slot >= seg->n_slots)
        return C3_OOB_E_INVAL;
    Slot* s = seg->slot(slot);
    for (int i = 0; i < kReadRetries; ++i) {
        const uint64_t n = s->latest.load(std::memory_order_acquire);
        c3_progress_t p;
        p.publishes = n;
        if (n == 0) {  // nothing published yet
            p.step = p.op_id = p.fingerprint = p.publish_ns = 0;
            p.flags = p.pid = 0;
            *out = p;
            return C3_OOB_OK;
        }
        Copy& c = s->copy[n & 1];
        const uint64_t s0 = c.seq.load(std::memory_order_acquire);
        if (s0 & 1u) continue;  // rewritten already: two publications went by
        p.publishes = c.number.load(std::memory_order_relaxed);
        p.step = c.step.load(std::memory_order_relaxed);
        p.op_id = c.op_id.load(std::memory_order_relaxed);
        p.fingerprint = c.fingerprint.load(std::memory_order_relaxed);
        p.flags = c.flags.load(std::memory_order_relaxed);
        p.pid = c.pid.load(std::memory_order_relaxed);
        p.publish_ns = c.publish_ns.load(std::memory_order_relaxed);
        std::atomic_thread_fence(std::memory_order_acquire);
        if (c.seq.load(std::memory_order_relaxed) == s0) {
            *out = p;
            return C3_OOB_OK;
        }
    }
    return C3_OOB_E_BUSY;
}

int c3_progress_wait_silence(const c3_progress_seg_t* seg, int slot, uint64_t silence_ns,
                             uint64_t poll_ns, uint64_t max_wait_ns, c3_progress_t* out) {
    if (seg == nullptr || out == nullptr || slot < 0 || slot >= seg->n_slots || poll_ns == 0)
        return C3_OOB_E_INVAL;
    const uint64_t t0 = now_ns();
    int rc = c3_progress_read(seg, slot, out);
    if (rc != C3_OOB_OK) return rc;
    uint64_t last_count = out->publishes, last_change = t0;
    for (;;) {
        const uint64_t t = now_ns();
        if (t - last_change >= silence_ns) return 1;
        if (t - t0 >= max_wait_ns) return 0;
        uint64_t nap = poll_ns;
        if (t - t0 + nap > max_wait_ns) nap = max_wait_ns - (t - t0);
        if (last_change + silence_ns - t < nap) nap = last_change + silence_ns - t;
        timespec ts;
        ts.tv_sec = (time_t)(nap / 1000000000ull);
        ts.tv_nsec = (long)(nap % 1000000000ull);
        nanosleep(&ts, nullptr);
        c3_progress_t p;
        rc = c3_progress_read(seg, slot, &p);
        if (rc != C3_OOB_OK) return rc;
        *out = p;
        if (p.publishes != last_count) {
            last_count = p.publishes;
            last_change = now_ns();
        }
    }
}

uint64_t c3_group_id(const int32_t* ranks, int n) {
    if (ranks == nullptr || n < 1) return 0;
    uint64_t h = fmix64(kTagGroup ^ (uint64_t)(uint32_t)n);
    for (int i = 0; i < n; ++i) h = fmix64(h ^ (uint64_t)(uint32_t)ranks[i]);
    return h;
}

uint64_t c3_collective_fingerprint(const c3_collective_t* c) {
    if (c == nullptr || c->ndim < -1 || c->ndim > C3_OOB_MAX_NDIM || c->reserved != 0) return 0;
    uint64_t h = fmix64(kTagColl ^ ((uint64_t)(uint32_t)c->kind << 32) ^ (uint64_t)(uint32_t)c->dtype);
    h = fmix64(h ^ c->process_group);
    h = fmix64(h ^ (((uint64_t)(uint32_t)c->reduce_op << 32) | (uint64_t)(uint32_t)c->root));
    h = fmix64(h ^ (uint64_t)(int64_t)c->ndim);
    for (int d = 0; d < c->ndim; ++d) h = fmix64(h ^ (uint64_t)c->shape[d]);
    return h != 0 ? h : 1;
}

uint64_t c3_progress_evidence(const c3_progress_t* p) {
    if (p == nullptr) return 0;
    uint64_t h = fmix64(kTagProgress ^ p->step);
    h = fmix64(h ^ p->op_id);
    h = fmix64(h ^ p->fingerprint);
    return fmix64(h ^ (uint64_t)(p->flags & C3_OOB_PENDING));
}

int c3_hang_classify(const c3_progress_t* records, int R, c3_hang_verdict_t* out) {
    // a single rank has no peer to be compared with (Sec. 4)
    if (records == nullptr || out == nullptr || R < 2 || R > C3_OOB_MAX_RANKS)
        return C3_OOB_E_INVAL;
    memset(out, 0, sizeof(*out));
    uint64_t e[C3_OOB_MAX_RANKS];
    for (int i = 0; i < R; ++i) e[i] = c3_progress_evidence(&records[i]);
    // most frequent evidence value; the first peer holding it on ties
    int best = 0, best_count = 0;
    for (int i = 0; i < R; ++i) {
        int c = 0;
        for (int j = 0; j < R; ++j) c += e[j] == e[i];
        if (c > best_count) {
            best_count = c;
            best = i;
        }
    }
    if (2 * best_count <= R) {
        out->cls = C3_HANG_INCONCLUSIVE;
        out->majority_idx = -1;
        return C3_OOB_OK;
    }
    out->majority_idx = best;
    const c3_progress_t& m = records[best];
    for (int i = 0; i < R; ++i) {
        if (e[i] == e[best]) continue;
        out->bitmap |= 1ull << i;
        const bool same_coord = records[i].step == m.step && records[i].op_id == m.op_id;
        out->reason[i] = same_coord ? C3_HANG_REASON_PROTOCOL : C3_HANG_REASON_PROGRESS;
    }
    out->cls = out->bitmap ? C3_HANG_RANK_DIVERGENCE : C3_HANG_GROUP_STALL;
    return C3_OOB_OK;
}

}  // extern "C"
